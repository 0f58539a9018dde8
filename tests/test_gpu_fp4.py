"""GPU parity of the 2-bit path on the scaled FP4 MFMA (e2m1 operands, fp32
sums of integers): code outputs with and without 2-bit skips (per-channel
sides, the side-0 table, upsampled), shifts < 2 (64-bit requantisation),
int32 outputs, split K ranges, grouped multi-level launches, and the largest
sums the path admits, all bit-exact against the oracle."""
import numpy as np
import pytest

from gpu_helpers import assert_same, gpu_conv, oracle_conv
from oracle import ref
from paper_2007_06919_amd import aqd, workloads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    return t


def _path(case):
    h = aqd.qconv_create(case.cin, case.cout, case.k, case.stride, case.pad, case.bits_in, case.bits_w,
                         aqd.pack_codes(case.w_fields, case.bits_w), case.levels, wenc=case.wenc,
                         out_mode=aqd.OUT_INT32 if case.bits_out == 32 else aqd.OUT_CODES,
                         bits_out=0 if case.bits_out == 32 else case.bits_out,
                         skip_bits=case.skip_bits, skip_up2=case.skip_up2)
    try:
        return aqd.qconv_path(h)
    finally:
        aqd.qconv_destroy(h)


FP4_CASES = [
    # (n, h, w, cin, cout, k, stride, bits_in, bits_w, wenc, bits_out, skip_bits, up2)
    (2, 50, 84, 256, 256, 3, 1, 2, 2, 1, 2, 0, False),      # head-tower shape, odd-grid weights
    (1, 60, 90, 512, 256, 3, 1, 2, 2, 0, 2, 0, False),      # two stages per tap, two's complement
    (2, 40, 50, 1024, 256, 1, 1, 2, 2, 1, 2, 2, True),      # 1x1, four stages per tap, upsampled skip
    (1, 45, 67, 256, 512, 3, 2, 2, 2, 0, 2, 2, False),      # stride 2, two channel tiles, skip
    (2, 30, 41, 256, 512, 1, 1, 2, 2, 1, 2, 2, False),      # one stage in all (odd count), skip
    (3, 33, 17, 2048, 256, 3, 2, 2, 2, 1, 2, 0, False),     # 72 stages, ragged pixel tail
]


@pytest.mark.parametrize("case", FP4_CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("variant", ["random_sides", "side0", "small_shifts"])
def test_fp4_parity(torch, case, variant):
    n, h, w, cin, cout, k, s, bi, bw, wenc, bo, sb, up2 = case
    c = workloads.random_conv_case(seed=hash(case) % 1000 + 7, n=n, h=h, w=w, cin=cin, cout=cout, k=k,
                                   stride=s, bits_in=bi, bits_w=bw, wenc=wenc, bits_out=bo,
                                   skip_bits=sb, skip_up2=up2)
    assert _path(c) == "fp4-mfma"
    rng = np.random.Generator(np.random.PCG64(37))
    for lv in c.levels:
        if variant == "side0" and sb:
            lv["skip_side"][:] = 0
        if variant == "small_shifts":
            lv["shift"] = rng.integers(-2, 2, size=cout).astype(np.int32)
            lv["mult"] = rng.integers(1 << 24, 1 << 27, size=cout).astype(np.int32)
    for level, got in enumerate(gpu_conv(c, torch)):
        assert_same(got, oracle_conv(c, level), f"fp4 {variant} {case} level {level}")


FP4_INT32_CASES = [
    (1, 30, 50, 256, 256, 3, 1, 2, 2, 1, 32, 0, False),
    (2, 20, 33, 512, 1024, 1, 1, 2, 2, 0, 32, 0, False),
]


@pytest.mark.parametrize("case", FP4_INT32_CASES, ids=lambda c: "x".join(map(str, c)))
def test_fp4_int32_parity(torch, case):
    n, h, w, cin, cout, k, s, bi, bw, wenc, bo, sb, up2 = case
    c = workloads.random_conv_case(seed=hash(case) % 1000 + 11, n=n, h=h, w=w, cin=cin, cout=cout, k=k,
                                   stride=s, bits_in=bi, bits_w=bw, wenc=wenc, bits_out=bo)
    assert _path(c) == "fp4-mfma"
    for level, got in enumerate(gpu_conv(c, torch)):
        assert_same(got, oracle_conv(c, level), f"fp4 int32 {case} level {level}")


FP4_SPLIT_CASES = [
    # few tiles, long K: the split-K parts run on the FP4 kernel
    (1, 13, 21, 1024, 256, 3, 1, 2, 2, 1, 2, 2, False),
    (1, 7, 11, 2048, 512, 3, 2, 2, 2, 0, 2, 0, False),
    (2, 9, 10, 2048, 256, 1, 1, 2, 2, 1, 2, 2, True),
]


@pytest.mark.parametrize("case", FP4_SPLIT_CASES, ids=lambda c: "x".join(map(str, c)))
def test_fp4_split_k_parity(torch, case):
    n, h, w, cin, cout, k, s, bi, bw, wenc, bo, sb, up2 = case
    c = workloads.random_conv_case(seed=hash(case) % 1000 + 13, n=n, h=h, w=w, cin=cin, cout=cout, k=k,
                                   stride=s, bits_in=bi, bits_w=bw, wenc=wenc, bits_out=bo,
                                   skip_bits=sb, skip_up2=up2)
    assert _path(c) == "fp4-mfma"
    for level, got in enumerate(gpu_conv(c, torch, split=True)):
        assert_same(got, oracle_conv(c, level), f"fp4 split {case} level {level}")


@pytest.mark.parametrize("wenc", [workloads.WENC_PAPER_ODD, workloads.WENC_TWOS])
def test_fp4_largest_sums_are_exact(torch, wenc):
    """Every code 3 and every weight at the grid's extreme, one sign per
    channel (K = 9 x 2048: sums of magnitude 165 888 for the odd grid), and
    random extremes: the int32 outputs are the exact integer sums."""
    n, h, w, cin, cout = 1, 12, 20, 2048, 256
    c = workloads.random_conv_case(seed=17 + wenc, n=n, h=h, w=w, cin=cin, cout=cout, k=3,
                                   bits_in=2, bits_w=2, wenc=wenc, bits_out=32)
    c.x[:] = 3
    hi, lo = (3, 0) if wenc == workloads.WENC_PAPER_ODD else (1, 2)   # fields of +max and -max
    c.w_fields[0::2] = hi
    c.w_fields[1::2] = lo
    rng = np.random.Generator(np.random.PCG64(5))
    c.w_fields[cout // 2:] = np.where(rng.random(c.w_fields[cout // 2:].shape) < 0.5, hi, lo)
    assert _path(c) == "fp4-mfma"
    got = gpu_conv(c, torch)[0]
    want = oracle_conv(c)
    assert_same(got, want, f"fp4 extremes wenc={wenc}")
    if wenc == workloads.WENC_PAPER_ODD:
        bias = c.levels[0]["bias"].astype(np.int64)
        assert int(np.abs(want[0, h // 2, w // 2, 0] - bias[0])) == 9 * cin * 3 * 3


def test_fp4_grouped_levels_and_guard_bytes(torch):
    """A grouped launch of two FP4 handles over five pyramid levels, each with
    its own table; outputs between guard bytes that must stay untouched."""
    dev = torch.device("cuda:0")
    n, sizes = 2, [(50, 75), (25, 38), (13, 19), (7, 10), (4, 5)]
    cases = [workloads.random_conv_case(seed=60 + t, n=1, h=8, w=8, cin=256, cout=256, k=3, bits_in=2,
                                        bits_w=2, wenc=1, bits_out=2, num_levels=5) for t in range(2)]
    handles = [aqd.qconv_create(256, 256, 3, 1, 1, 2, 2, aqd.pack_codes(c.w_fields, 2), c.levels,
                                wenc=1, bits_out=2) for c in cases]
    rng = np.random.Generator(np.random.PCG64(29))
    try:
        assert all(aqd.qconv_path(hd) == "fp4-mfma" for hd in handles)
        segs, expect, outs = [], [], []
        for t, c in enumerate(cases):
            for lv, (h, w) in enumerate(sizes):
                x = rng.integers(0, 4, size=(n, h, w, 256))
                xd = torch.from_numpy(aqd.pack_codes(x, 2)).to(dev)
                nbytes = n * h * w * 64
                buf = torch.full((nbytes + 4096,), 0x5A, dtype=torch.uint8, device=dev)
                yd = buf[2048:2048 + nbytes]
                segs.append((handles[t], lv, n, h, w, xd, None, 0, 0, yd))
                outs.append((buf, nbytes))
                L = c.levels[lv]
                want = ref.qconv(x, c.w_fields, 2, 1, 1, L["bias"], wenc=1, mult=L["mult"],
                                 shift=L["shift"], bits_out=2)
                expect.append(ref.pack_codes(want, 2).reshape(-1))
        aqd.qconv_run_group(segs)
        torch.cuda.synchronize()
        for i, ((buf, nbytes), want) in enumerate(zip(outs, expect)):
            host = buf.cpu().numpy()
            assert np.all(host[:2048] == 0x5A) and np.all(host[2048 + nbytes:] == 0x5A), i
            assert_same(host[2048:2048 + nbytes], want, f"fp4 segment {i}")
    finally:
        for hd in handles:
            aqd.qconv_destroy(hd)


def test_two_bit_layers_off_the_fp4_path(torch):
    """2-bit layers the FP4 kernel does not take (cout not a multiple of 256,
    4-bit weights, an int32 skip) report the int8 path and stay exact."""
    for kw in (dict(cin=256, cout=128, bits_w=2, skip_bits=0),
               dict(cin=256, cout=256, bits_w=4, skip_bits=0),
               dict(cin=256, cout=256, bits_w=2, skip_bits=32)):
        c = workloads.random_conv_case(seed=3, n=1, h=17, w=19, k=3, bits_in=2, wenc=1, bits_out=2, **kw)
        assert _path(c) == "i8-mfma", kw
        assert_same(gpu_conv(c, torch)[0], oracle_conv(c), f"int8 path {kw}")
