"""GPU parity over the full parameter ranges the ABI accepts, on every launch
path: requantisation shifts over [-31, 31] (17-31 on the 32-bit path too),
negative multipliers, skip exponents 0 and 31, skip numerators up to
2^31 - 1 and negative ones (opposite-sign scales of Eq. 7), on the tiled,
streaming, half-view, short-tile, split-K, fused-projection and direct
kernels and the standalone add. Every skip numerator is bounded so that the
aligned sum u stays inside int32 (the ABI's contract), whatever the inputs.
"""
import numpy as np
import pytest

from gpu_helpers import assert_same, gpu_conv, oracle_conv
from oracle import ref
from paper_2007_06919_amd import aqd, workloads

pytestmark = pytest.mark.gpu

I32 = (1 << 31) - 1


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    return t


def _cmax(d, operand_max, budget):
    """Largest |c| with operand_max * |c| / 2^d + 1 <= budget."""
    return int(min(I32, max(0, (budget - 1) * (1 << d) // max(operand_max, 1))))


def edge_level(rng, cout, v_bound, k_max, fast, sides, base_shift=None):
    """One epilogue table at the edges of the ABI's ranges.

    fast: every shift in [2, 31] (32-bit requantisation), else shifts over
    [-31, 31]; sides: 'random' or 'side0' (every side 0: the skip table);
    |v| <= v_bound and |k| <= k_max bound the skip numerators."""
    mult = rng.integers(1 << 30, 1 << 31, size=cout)
    mult[rng.random(cout) < 0.1] = 1 << 30
    mult[rng.random(cout) < 0.1] = I32
    mult = mult * np.where(rng.random(cout) < 0.3, -1, 1)
    if fast:
        shift = rng.integers(2, 32, size=cout)
        if base_shift is not None:
            keep = rng.random(cout) < 0.5
            shift[keep] = np.clip(base_shift[keep], 2, 31)
        shift[:2] = (2, 31)
    else:
        shift = rng.integers(-31, 32, size=cout)
        if base_shift is not None:
            keep = rng.random(cout) < 0.4
            shift[keep] = np.clip(base_shift[keep], -31, 31)
        shift[:2] = (-31, 1)
    lv = {"bias": rng.integers(-(1 << 12), (1 << 12) + 1, size=cout),
          "mult": mult, "shift": shift}
    if k_max is not None:
        budget = (1 << 30) - (v_bound + k_max + 2)
        assert budget > 0
        side = rng.integers(0, 2, size=cout) if sides == "random" else np.zeros(cout, np.int64)
        d = rng.integers(1, 31, size=cout)
        pick = rng.random(cout)
        d[pick < 0.2] = 0
        d[(pick >= 0.2) & (pick < 0.4)] = 31
        c = np.zeros(cout, np.int64)
        for i in range(cout):
            cm = _cmax(int(d[i]), k_max if side[i] == 0 else v_bound, budget)
            c[i] = cm if rng.random() < 0.25 else rng.integers(0, cm + 1)
            if rng.random() < 0.3:
                c[i] = -c[i]
        lv.update(skip_c=c, skip_d=d, skip_side=side)
    return {k: np.asarray(v, np.int64).astype(np.int32) for k, v in lv.items()}


def edge_case(seed, n, h, w, cin, cout, k, stride, bits_in, bits_w, wenc, bits_out, skip_bits, up2):
    case = workloads.random_conv_case(seed=seed, n=n, h=h, w=w, cin=cin, cout=cout, k=k,
                                      stride=stride, bits_in=bits_in, bits_w=bits_w, wenc=wenc,
                                      bits_out=bits_out, skip_bits=skip_bits, skip_up2=up2)
    rng = np.random.Generator(np.random.PCG64(seed + 500))
    qx = (1 << bits_in) - 1
    wmax = (1 << bits_w) - 1 if wenc == workloads.WENC_PAPER_ODD else 1 << (bits_w - 1)
    v_bound = k * k * cin * qx * wmax + (1 << 12)
    k_max = None
    if skip_bits:
        k_max = int(np.abs(case.skip).max()) if skip_bits == 32 else (1 << skip_bits) - 1
    base = case.levels[0].get("shift")
    levels = []
    if bits_out == 32:
        levels = [{"bias": rng.integers(-(1 << 12), (1 << 12) + 1, size=cout).astype(np.int32)}]
    else:
        for fast in (True, False):
            for sides in (("random", "side0") if skip_bits else ("random",)):
                levels.append(edge_level(rng, cout, v_bound, k_max, fast, sides, base))
    case.levels = levels
    return case


EDGE_CASES = [
    # (n, h, w, cin, cout, k, stride, bits_in, bits_w, wenc, bits_out, skip_bits, up2)
    (1, 19, 23, 64, 256, 3, 1, 4, 4, 1, 4, 4, False),       # 256 x 128 tiles, code skip
    (1, 19, 23, 64, 256, 3, 1, 4, 4, 1, 4, 32, False),      # 256 x 128 tiles, int32 skip
    (1, 17, 21, 64, 128, 3, 1, 2, 2, 0, 2, 2, False),       # 2-bit, 128 x 256 tiles
    (1, 15, 19, 64, 64, 3, 2, 4, 4, 0, 4, 4, True),         # 64 x 512 tiles, upsampled skip
    (2, 33, 37, 64, 256, 1, 1, 4, 4, 1, 4, 4, False),       # streaming 1x1
    (2, 16, 18, 256, 512, 1, 1, 4, 4, 0, 4, 4, True),       # half-view streaming, upsampled
    (1, 25, 31, 256, 288, 1, 1, 4, 4, 0, 4, 4, False),      # 256 x 64 short tiles
    (1, 11, 13, 24, 40, 3, 1, 8, 4, 0, 8, 8, False),        # direct kernel
    (1, 9, 10, 32, 48, 3, 1, 4, 4, 1, 4, 32, True),         # direct kernel, int32 skip
]


@pytest.mark.parametrize("case", EDGE_CASES, ids=lambda c: "x".join(map(str, c)))
def test_edge_ranges_parity(torch, case):
    c = edge_case(hash(case) % 1000 + 31, *case)
    for level, got in enumerate(gpu_conv(c, torch)):
        assert_same(got, oracle_conv(c, level), f"edge ranges {case} level {level}")


SPLIT_EDGE_CASES = [
    (1, 13, 21, 512, 256, 3, 2, 4, 4, 1, 4, 4, False),      # split K, code skip
    (1, 7, 9, 1024, 256, 1, 1, 4, 4, 0, 4, 32, False),      # split K, int32 skip
    (2, 9, 11, 1024, 256, 1, 1, 4, 4, 1, 4, 4, True),       # split K, upsampled skip
]


@pytest.mark.parametrize("case", SPLIT_EDGE_CASES, ids=lambda c: "x".join(map(str, c)))
def test_edge_ranges_split_k(torch, case):
    c = edge_case(hash(case) % 1000 + 37, *case)
    for level, got in enumerate(gpu_conv(c, torch, split=True)):
        assert_same(got, oracle_conv(c, level), f"split edge ranges {case} level {level}")


def test_edge_ranges_fused_projection(torch):
    """qconv_run_proj (tiled and streaming shapes) with the int32 shortcut at
    the edges: the shortcut's int32 output bounds the skip numerators."""
    from test_gpu_conv import _proj_case, _run_proj
    for case, seed in (((2, 14, 15, 256, 14, 15, 64, 1, 512, 3, 1), 41),
                       ((2, 13, 17, 64, 26, 33, 64, 2, 512, 1, 0), 43)):
        main, proj = _proj_case(case, seed)
        rng = np.random.Generator(np.random.PCG64(seed))
        qx, wmax = 15, 15 if main.wenc == workloads.WENC_PAPER_ODD else 8
        v_bound = main.k * main.k * main.cin * qx * wmax + (1 << 12)
        k_max = int(np.abs(main.skip).max())
        for fast in (True, False):
            main.levels = [edge_level(rng, main.cout, v_bound, k_max, fast, "random")]
            assert_same(_run_proj(torch, main, proj), oracle_conv(main),
                        f"fused projection edge ranges {case} fast={fast}")


@pytest.mark.parametrize("bits_a,bits_b,up2", [(4, 4, True), (32, 4, False), (4, 32, True),
                                               (2, 2, False)])
def test_edge_ranges_qadd(torch, bits_a, bits_b, up2):
    dev = torch.device("cuda:0")
    rng = np.random.Generator(np.random.PCG64(bits_a * 7 + bits_b))
    n, h, w, c = 2, 13, 22, 128
    hb, wb = ((h + 1) // 2, (w + 1) // 2) if up2 else (h, w)

    def draw(bits, shape):
        if bits == 32:
            return rng.integers(-(1 << 20), 1 << 20, size=shape)
        return rng.integers(0, 1 << bits, size=shape)

    a, b = draw(bits_a, (n, h, w, c)), draw(bits_b, (n, hb, wb, c))
    a_max, b_max = int(np.abs(a).max()), int(np.abs(b).max())
    for fast, sides in ((True, "random"), (False, "random"), (False, "side0")):
        # the add's "conv operand" is a (side 1 scales it), the skip operand b
        lv = edge_level(rng, c, a_max, b_max, fast, sides)
        p = {k: lv[k] for k in ("skip_c", "skip_d", "skip_side", "mult", "shift")}
        want = ref.pack_codes(ref.qadd(a, b, up2, p["skip_c"], p["skip_d"], p["skip_side"],
                                       p["mult"], p["shift"], 4), 4)

        def dev_t(v, bits):
            if bits == 32:
                return torch.from_numpy(v.astype(np.int32)).to(dev)
            return torch.from_numpy(aqd.pack_codes(v, bits)).to(dev)

        pd = {k: torch.from_numpy(v.astype(np.int32)).to(dev) for k, v in p.items()}
        y = torch.zeros((n, h, w, c // 2), dtype=torch.uint8, device=dev)
        aqd.qadd_run(n, h, w, c, bits_a, bits_b, 4, up2, hb, wb, dev_t(a, bits_a),
                     dev_t(b, bits_b), y, pd)
        torch.cuda.synchronize()
        assert_same(y.cpu().numpy(), want, f"qadd edge ranges {bits_a} {bits_b} {sides}")
