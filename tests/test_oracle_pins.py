"""Pins of the CPU oracle against what the paper and the mathematics fix.

Every test here checks the oracle against something other than itself: a
library reduction (numpy integer matmul, torch float64 convolution), exact
rational arithmetic, closed forms of the paper's special cases (Eq. 4, Eq. 8,
Eq. 9), invariants and error bounds of the construction (Eq. 5-7), and brute
force on tiny inputs. CPU only.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import ref

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _nearest_half_up(q: Fraction) -> int:
    """Nearest integer to a rational, ties toward +infinity, from the
    definition: the integer n with n - 1/2 <= q < n + 1/2."""
    n = math.floor(q)
    frac = q - n
    return n + 1 if frac >= Fraction(1, 2) else n


# ----------------------------------------------------------------- RSM
def test_rsm_is_round_half_up_of_exact_rational():
    rng = _rng(1)
    a = np.concatenate([rng.integers(-(1 << 31) + 1, 1 << 31, 3000),
                        rng.integers(-300, 300, 1000)])
    c = np.concatenate([rng.integers(-(1 << 31) + 1, 1 << 31, 2000),
                        rng.integers(0, 1 << 31, 1000), rng.integers(1, 9, 1000)])
    d = rng.integers(0, 63, a.size)
    got = ref.rsm_array(a, c, d)
    for ai, ci, di, g in zip(a, c, d, got):
        q = Fraction(int(ai) * int(ci), 1 << int(di))
        assert g == _nearest_half_up(q)
        assert abs(Fraction(g) - q) <= Fraction(1, 2)


def test_rsm_ties_go_up_and_small_cases():
    # a*c/2^d = k + 1/2 exactly -> k + 1, also for negative values
    a = np.array([1, 3, -1, -3, 5, -5, 7, 0])
    c = np.array([1, 1, 1, 1, 1, 1, 3, 123])
    d = np.array([1, 1, 1, 1, 1, 1, 2, 5])
    assert ref.rsm_array(a, c, d) == [1, 2, 0, -1, 3, -2, 5, 0]
    # d = 0 is the plain product
    assert ref.rsm_array([7, -7], [9, 9], [0, 0]) == [63, -63]


# --------------------------------------------------- packing / weight decode
def test_pack_layout_known_bytes():
    assert ref.pack_codes(np.array([[1, 2]]), 4).tolist() == [[0x21]]
    assert ref.pack_codes(np.array([[1, 2, 3, 0]]), 2).tolist() == [[0b00111001]]
    assert ref.pack_codes(np.array([[200, 7]]), 8).tolist() == [[200, 7]]
    # 3-bit codes sit in 4-bit containers
    assert ref.pack_codes(np.array([[1, 7, 5, 0]]), 3).tolist() == [[0x71, 0x05]]


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_pack_roundtrip(bits):
    rng = _rng(bits)
    codes = rng.integers(0, 1 << bits, size=(3, 5, 7, 64))
    packed = ref.pack_codes(codes, bits)
    assert packed.shape == (3, 5, 7, 64 * (4 if bits == 3 else bits) // 8)
    assert np.array_equal(ref.unpack_codes(packed, bits, 64), codes)
    if bits == 3:  # the same bytes as 4-bit codes of the same values
        assert np.array_equal(packed, ref.pack_codes(codes, 4))


def test_weight_decode():
    f = np.arange(16)
    assert ref.decode_weights(f, 4, ref.WENC_TWOS).tolist() == list(range(8)) + list(range(-8, 0))
    assert ref.decode_weights(np.arange(4), 2, ref.WENC_TWOS).tolist() == [0, 1, -2, -1]
    # Eq. 3-4: the paper's odd grid 2*eta - (2^b - 1); b = 2 -> {-3, -1, 1, 3}
    assert ref.decode_weights(np.arange(4), 2, ref.WENC_PAPER_ODD).tolist() == [-3, -1, 1, 3]
    assert ref.decode_weights(f, 4, ref.WENC_PAPER_ODD).tolist() == list(range(-15, 16, 2))
    # 3 bits: {-7, -5, ..., 7} on the odd grid, [-4, 3] in two's complement
    assert ref.decode_weights(np.arange(8), 3, ref.WENC_PAPER_ODD).tolist() == list(range(-7, 8, 2))
    assert ref.decode_weights(np.arange(8), 3, ref.WENC_TWOS).tolist() == [0, 1, 2, 3, -4, -3, -2, -1]


# ------------------------------------------------------ Eq. 2 / 3 / 4
def test_eq2_eq3_quantizers_grid():
    nu = 2.0
    eta, val = ref.quantize_activation(np.array([-1.0, 0.0, 0.66, 1.0, 2.0, 5.0]), nu, 2)
    assert eta.tolist() == [0, 0, 1, 2, 3, 3]
    assert np.allclose(val, eta * nu / 3)
    eta, val = ref.quantize_weight(np.array([-3.0, -1.0, 0.0, 0.4, 1.0]), 1.0, 2)
    # clip to [-1, 1], map to {0..3}: -1 -> 0, 0 -> 1.5 -> 2 (half up), 0.4 -> 2.1 -> 2
    assert eta.tolist() == [0, 0, 2, 2, 3]
    assert np.allclose(val, (2 * eta / 3 - 1) * 1.0)


def test_eq4_identity_scalar():
    """x_bar * w_bar = eta_x (2 eta_w - 2^b + 1) * nu_x nu_w / (2^b - 1)^2 (Eq. 4)."""
    rng = _rng(4)
    for bits in (2, 3, 4, 8):
        q = (1 << bits) - 1
        for _ in range(50):
            x, w = rng.uniform(-1, 3), rng.uniform(-2, 2)
            nux, nuw = rng.uniform(0.5, 3), rng.uniform(0.2, 2)
            ex, xb = ref.quantize_activation(x, nux, bits)
            ew, wb = ref.quantize_weight(w, nuw, bits)
            lhs = float(xb) * float(wb)
            wint = int(ref.decode_weights(ew, bits, ref.WENC_PAPER_ODD))
            rhs = int(ex) * wint * (nux * nuw / q ** 2)
            assert lhs == pytest.approx(rhs, rel=1e-12, abs=1e-15)


# ------------------------------------------------------- accumulation
def _acc(x, w, bits_w, stride, pad, wenc=ref.WENC_TWOS):
    return ref.qconv(x, w, bits_w, stride, pad, np.zeros(w.shape[0], np.int64),
                     wenc=wenc, out_int32=True)


def test_acc_1x1_equals_integer_matmul():
    rng = _rng(11)
    for bits in (2, 4, 8):
        x = rng.integers(0, 1 << bits, size=(2, 7, 9, 48))
        wf = rng.integers(0, 1 << bits, size=(24, 1, 1, 48))
        wv = ref.decode_weights(wf, bits, ref.WENC_TWOS)
        want = (x.reshape(-1, 48).astype(np.int64) @ wv.reshape(24, 48).T).reshape(2, 7, 9, 24)
        assert np.array_equal(_acc(x, wf, bits, 1, 0), want)


@pytest.mark.parametrize("k,stride", [(3, 1), (3, 2), (1, 2), (5, 1), (3, 3)])
@pytest.mark.parametrize("wenc", [ref.WENC_TWOS, ref.WENC_PAPER_ODD])
def test_acc_equals_torch_conv2d_float64(k, stride, wenc):
    rng = _rng(k * 10 + stride + 100 * wenc)
    for bits, (n, h, w, cin, cout) in [(4, (2, 11, 13, 32, 16)), (2, (1, 9, 6, 64, 8)),
                                       (8, (1, 5, 7, 8, 24))]:
        x = rng.integers(0, 1 << bits, size=(n, h, w, cin))
        wf = rng.integers(0, 1 << bits, size=(cout, k, k, cin))
        wv = ref.decode_weights(wf, bits, wenc)
        pad = k // 2
        want = torch.nn.functional.conv2d(
            torch.from_numpy(x.astype(np.float64)).permute(0, 3, 1, 2),
            torch.from_numpy(wv.astype(np.float64)).permute(0, 3, 1, 2),
            stride=stride, padding=pad).permute(0, 2, 3, 1).numpy()
        got = _acc(x, wf, bits, stride, pad, wenc)
        assert got.shape == want.shape
        assert np.array_equal(got, want.astype(np.int64))


def test_acc_brute_force_tiny():
    """Pure-Python loops over one output pixel at a time."""
    rng = _rng(12)
    n, h, w, cin, cout, k, s, p = 1, 4, 5, 8, 3, 3, 2, 1
    x = rng.integers(0, 16, size=(n, h, w, cin))
    wf = rng.integers(0, 16, size=(cout, k, k, cin))
    wv = ref.decode_weights(wf, 4)
    got = _acc(x, wf, 4, s, p)
    ho, wo = (h + 2 * p - k) // s + 1, (w + 2 * p - k) // s + 1
    for oh in range(ho):
        for ow in range(wo):
            for co in range(cout):
                tot = 0
                for r in range(k):
                    for q in range(k):
                        ih, iw = oh * s - p + r, ow * s - p + q
                        if 0 <= ih < h and 0 <= iw < w:
                            tot += sum(int(x[0, ih, iw, ci]) * int(wv[co, r, q, ci])
                                       for ci in range(cin))
                assert got[0, oh, ow, co] == tot


def test_eq4_conv_with_power_of_two_scales_is_exact():
    """Dequantize with power-of-two steps, convolve in float64, divide back:
    the integer accumulator times alpha_conv is the real convolution (Eq. 4)."""
    rng = _rng(13)
    bits = 4
    q = 15
    ax, aw = 2.0 ** -3, 2.0 ** -4          # alpha_x = nu_x / q, alpha_w = nu_w / q
    x = rng.integers(0, 16, size=(1, 8, 8, 16))
    wf = rng.integers(0, 16, size=(8, 3, 3, 16))
    # real tensors that Eq. 2 / Eq. 3 quantize back to exactly these codes
    xb = x * ax
    wb = (2 * wf - q) * aw
    ex, xbq = ref.quantize_activation(xb, q * ax, bits)
    ew, wbq = ref.quantize_weight(wb, q * aw, bits)
    assert np.array_equal(ex, x) and np.array_equal(ew, wf)
    # Eq. 3's restore (2*eta/q - 1)*nu is (2*eta - q)*alpha_w up to float rounding of 1/q
    assert np.allclose(xbq, xb, rtol=0, atol=0) and np.allclose(wbq, wb, rtol=1e-15, atol=0)
    real = torch.nn.functional.conv2d(torch.from_numpy(xb).permute(0, 3, 1, 2),
                                      torch.from_numpy(wb.astype(np.float64)).permute(0, 3, 1, 2),
                                      padding=1).permute(0, 2, 3, 1).numpy()
    acc = _acc(x, wf, bits, 1, 1, ref.WENC_PAPER_ODD)
    assert np.array_equal(real / (ax * aw), acc.astype(np.float64))


# ------------------------------------------------------- epilogue
def _float_epilogue(acc, bias, mult, shift, qm, skip=None, c=None, d=None, side=None):
    """Brute force in float64: y = round(u * M / 2^(31+sh)), clamp; exact while
    every product stays below 2^53 (asserted)."""
    v = acc.astype(np.float64) + bias
    if skip is not None:
        k = skip.astype(np.float64)
        scaled_k = np.floor(k * c / 2.0 ** d + 0.5)
        scaled_v = np.floor(v * c / 2.0 ** d + 0.5)
        assert np.all(np.abs(k * c) < 2.0 ** 53) and np.all(np.abs(v * c) < 2.0 ** 53)
        u = np.where(side == 0, v + scaled_k, scaled_v + k)
    else:
        u = v
    prod = u * mult
    assert np.all(np.abs(prod) < 2.0 ** 53)
    y = np.floor(prod / 2.0 ** (31 + shift) + 0.5)
    return np.clip(y, 0, qm).astype(np.int64)


def _literal(rng, cout, skip=False):
    p = {"bias": rng.integers(-4096, 4097, cout), "mult": rng.integers(1 << 30, 1 << 31, cout),
         "shift": rng.integers(8, 17, cout)}
    if skip:
        p.update(skip_c=rng.integers(1, 1 << 12, cout), skip_d=rng.integers(1, 12, cout),
                 skip_side=rng.integers(0, 2, cout))
    return p


@pytest.mark.parametrize("bits_out", [2, 3, 4, 8])
def test_requant_matches_float_brute_force(bits_out):
    rng = _rng(20 + bits_out)
    x = rng.integers(0, 4, size=(1, 6, 7, 16))
    wf = rng.integers(0, 4, size=(12, 3, 3, 16))
    p = _literal(rng, 12)
    got = ref.qconv(x, wf, 2, 1, 1, p["bias"], mult=p["mult"], shift=p["shift"],
                    bits_out=bits_out)
    acc = _acc(x, wf, 2, 1, 1)
    want = _float_epilogue(acc, p["bias"], p["mult"], p["shift"], (1 << bits_out) - 1)
    assert np.array_equal(got, want)
    assert got.min() >= 0 and got.max() <= (1 << bits_out) - 1


def test_skip_matches_float_brute_force_both_sides_and_upsample():
    rng = _rng(30)
    x = rng.integers(0, 16, size=(2, 7, 9, 16))
    wf = rng.integers(0, 16, size=(8, 3, 3, 16))
    p = _literal(rng, 8, skip=True)
    for up2 in (False, True):
        hs, ws = (4, 5) if up2 else (7, 9)
        sk = rng.integers(0, 16, size=(2, hs, ws, 8))
        got = ref.qconv(x, wf, 4, 1, 1, p["bias"], mult=p["mult"], shift=p["shift"], bits_out=4,
                        skip=sk, skip_up2=up2, skip_c=p["skip_c"], skip_d=p["skip_d"],
                        skip_side=p["skip_side"])
        # nearest 2x upsample by repetition, then crop: a library-level reduction
        full = np.repeat(np.repeat(sk, 2, axis=1), 2, axis=2)[:, :7, :9] if up2 else sk
        acc = _acc(x, wf, 4, 1, 1)
        want = _float_epilogue(acc, p["bias"], p["mult"], p["shift"], 15, full,
                               p["skip_c"], p["skip_d"], p["skip_side"])
        assert np.array_equal(got, want)


def test_power_of_two_scale_is_exact_shift():
    """M = 2^30: the scale is exactly 2^-(sh+1); the requant is rounding of
    u / 2^(sh+1), with ties up."""
    rng = _rng(40)
    x = rng.integers(0, 16, size=(1, 5, 5, 32))
    wf = rng.integers(0, 16, size=(8, 3, 3, 32))
    sh = rng.integers(0, 12, 8)
    bias = rng.integers(-2000, 2000, 8)
    got = ref.qconv(x, wf, 4, 1, 1, bias, mult=np.full(8, 1 << 30), shift=sh, bits_out=8)
    u = _acc(x, wf, 4, 1, 1) + bias
    want = np.clip(np.array([[_nearest_half_up(Fraction(int(v), 1 << (int(s) + 1)))
                              for v, s in zip(row, sh)] for row in u.reshape(-1, 8)]), 0, 255)
    assert np.array_equal(got.reshape(-1, 8), want)


def test_zero_weights_give_bias_only_output():
    rng = _rng(41)
    x = rng.integers(0, 16, size=(1, 6, 6, 16))
    wf = np.zeros((16, 3, 3, 16), np.int64)
    p = _literal(rng, 16)
    p["bias"] = rng.integers(-(1 << 20), 1 << 20, 16)
    p["shift"] = rng.integers(0, 8, 16)
    got = ref.qconv(x, wf, 4, 1, 1, p["bias"], mult=p["mult"], shift=p["shift"], bits_out=4)
    for co in range(16):
        b = int(p["bias"][co])
        y = _nearest_half_up(Fraction(b * int(p["mult"][co]), 1 << (31 + int(p["shift"][co]))))
        assert np.all(got[..., co] == min(max(y, 0), 15))


def test_requant_monotone_and_bounded():
    """For M >= 0 the requant is monotone in u, and before the clamp it is
    within 1/2 of u * M / 2^(31+sh)."""
    u = np.arange(-5000, 5000, 7)
    for M, sh in [(1 << 30, 3), ((1 << 31) - 1, 7), (1518500250, 10), (1 << 30, -2)]:
        y = np.array(ref.rsm_array(u, np.full(u.size, M), np.full(u.size, 31 + sh)))
        assert np.all(np.diff(y) >= 0)
        exact = np.array([Fraction(int(a) * M, 1 << (31 + sh)) for a in u], dtype=object)
        assert all(abs(Fraction(int(a)) - e) <= Fraction(1, 2) for a, e in zip(y, exact))


def test_unit_ratio_skip_is_plain_add():
    """c/2^d = 2/2 (ratio 1): Eq. 7 reduces to eta1 + eta2."""
    rng = _rng(42)
    a = rng.integers(0, 16, size=(1, 4, 4, 8))
    b = rng.integers(0, 16, size=(1, 4, 4, 8))
    ones = np.ones(8, np.int64)
    got = ref.qadd(a, b, False, 2 * ones, ones, 0 * ones, np.full(8, 1 << 30), -ones, 8)
    # M = 2^30, sh = -1: scale exactly 1
    assert np.array_equal(got, a + b)
    got1 = ref.qadd(a, b, False, 2 * ones, ones, ones, np.full(8, 1 << 30), -ones, 8)
    assert np.array_equal(got1, a + b)


def test_eq9_power_of_two_ratio_skip_is_exact():
    """FQN's constraint alpha1/alpha2 = 2^j (Eq. 9) is the case c = 2^(j+1),
    d = 1 of Eq. 8: the aligned add is exact integer arithmetic."""
    rng = _rng(43)
    for j in range(0, 10):
        c, d = ref.approx_ratio(2.0 ** j)
        assert (c, d) == (1 << (j + 1), 1)
        k = rng.integers(0, 256, 100)
        assert ref.rsm_array(k, np.full(100, c), np.full(100, d)) == [int(v) << j for v in k]


def test_skip_alignment_error_bound():
    rng = _rng(44)
    for _ in range(200):
        r = float(rng.uniform(1, 300))
        c, d = ref.approx_ratio(r)
        k = int(rng.integers(0, 1 << 16))
        got = ref.rsm_array([k], [c], [d])[0]
        bound = Fraction(1, 2) + k * abs(Fraction(r) - Fraction(c, 1 << d))
        assert abs(Fraction(got) - k * Fraction(r)) <= bound


def test_qadd_matches_float_brute_force():
    rng = _rng(45)
    a = rng.integers(0, 16, size=(2, 9, 7, 24))
    b = rng.integers(0, 16, size=(2, 5, 4, 24))
    p = _literal(rng, 24, skip=True)
    got = ref.qadd(a, b, True, p["skip_c"], p["skip_d"], p["skip_side"], p["mult"],
                   p["shift"] - 8, 4)
    full = np.repeat(np.repeat(b, 2, axis=1), 2, axis=2)[:, :9, :7]
    want = _float_epilogue(a, 0, p["mult"], p["shift"] - 8, 15, full, p["skip_c"], p["skip_d"],
                           p["skip_side"])
    assert np.array_equal(got, want)


def test_three_bit_output_is_the_four_bit_output_clamped_to_7():
    """Clamping is idempotent and monotone: with the same tables, a 3-bit
    output (Eq. 2, codes in [0, 7]) is min(4-bit output, 7), for convs with
    either skip side and for the standalone add."""
    rng = _rng(47)
    x = rng.integers(0, 8, size=(2, 7, 9, 32))
    wf = rng.integers(0, 8, size=(16, 3, 3, 32))
    skip = rng.integers(0, 8, size=(2, 7, 9, 16))
    p = _literal(rng, 16, skip=True)
    kw = dict(mult=p["mult"], shift=p["shift"] - 4, skip=skip, skip_c=p["skip_c"],
              skip_d=p["skip_d"], skip_side=p["skip_side"], wenc=ref.WENC_PAPER_ODD)
    y3 = ref.qconv(x, wf, 3, 1, 1, p["bias"], bits_out=3, **kw)
    y4 = ref.qconv(x, wf, 3, 1, 1, p["bias"], bits_out=4, **kw)
    assert np.array_equal(y3, np.minimum(y4, 7)) and 0 < (y3 == 7).mean() < 1
    a3 = ref.qadd(x[..., :16], skip, False, p["skip_c"], p["skip_d"], p["skip_side"],
                  p["mult"], p["shift"] - 8, 3)
    a4 = ref.qadd(x[..., :16], skip, False, p["skip_c"], p["skip_d"], p["skip_side"],
                  p["mult"], p["shift"] - 8, 4)
    assert np.array_equal(a3, np.minimum(a4, 7))


def test_int32_range_is_enforced():
    x = np.full((1, 3, 3, 8), 15)
    wf = np.full((2, 3, 3, 8), 7)
    with pytest.raises(ValueError):
        ref.qconv(x, wf, 4, 1, 1, np.array([(1 << 31) - 10, 0]), out_int32=True)


# ------------------------------------------------------- Eq. 8: F
def test_approx_ratio_known_values():
    assert ref.approx_ratio(1.0) == (2, 1)
    assert ref.approx_ratio(1.5) == (3, 1)
    assert ref.approx_ratio(3.0) == (6, 1)
    assert ref.approx_ratio(1.25) == (5, 2)
    assert ref.approx_ratio(math.pi) == (1686629713, 29)
    assert ref.approx_ratio(4.0 / 3.0) == (1431655765, 30)
    with pytest.raises(ValueError):
        ref.approx_ratio(0.5)


def test_approx_ratio_is_optimal_brute_force():
    """For every exponent d in [1, 31] the best numerator is floor or ceil of
    r*2^d (|r - c/2^d| is convex in c); compare exactly with rationals."""
    rng = _rng(50)
    rs = list(rng.uniform(1, 4, 200)) + list(np.exp(rng.uniform(0, 20, 200)))
    for r in rs:
        c, d = ref.approx_ratio(float(r))
        fr = Fraction(float(r))
        best = abs(fr - Fraction(c, 1 << d))
        assert 0 < c < (1 << 31) and 1 <= d <= 31
        for dd in range(1, 32):
            t = fr * (1 << dd)
            for cc in (math.floor(t), math.ceil(t)):
                if 0 <= cc < (1 << 31):
                    e = abs(fr - Fraction(cc, 1 << dd))
                    assert best < e or (best == e and d <= dd)


# -------------------------------------------- requant multiplier, BN fold
def test_normalize_multiplier():
    rng = _rng(60)
    for r in list(np.exp(rng.uniform(-20, 20, 500))) + [2.0 ** -9, 1.0, 0.75]:
        m, sh = ref.normalize_multiplier(float(r))
        assert (1 << 30) <= m < (1 << 31) and -31 <= sh <= 31
        err = abs(Fraction(float(r)) - Fraction(m, 1 << (31 + sh)) if sh >= -31 else 0)
        assert err <= Fraction(1, 1 << (32 + sh))
    assert ref.normalize_multiplier(2.0 ** -9) == (1 << 30, 8)
    assert ref.normalize_multiplier(1.0) == (1 << 30, -1)
    assert ref.normalize_multiplier(-0.5) == (-(1 << 30), 0)


def test_bn_fold_error_bound():
    """z from Eq. 5's first line vs the folded integer form (Eq. 6):
    |z_bar - z| <= alpha_z / 2."""
    rng = _rng(61)
    c = 64
    gamma, beta = rng.uniform(0.5, 1.5, c), rng.uniform(-1, 1, c)
    mean, var = rng.normal(0, 3, c), rng.uniform(0.1, 9, c)
    alpha_conv = 0.013
    bias, alpha_z = ref.fold_bn(gamma, beta, mean, var, 1e-5, alpha_conv)
    acc = rng.integers(-5000, 5000, size=(1000, c))
    z = (acc * alpha_conv - mean) / np.sqrt(var + 1e-5) * gamma + beta
    zbar = (acc + bias) * alpha_z
    assert np.all(np.abs(zbar - z) <= alpha_z / 2 * (1 + 1e-9) + 1e-12)


def test_bn_stats_from_sums():
    rng = _rng(62)
    acc = rng.integers(-30000, 30000, size=(5, 17, 13, 24))
    s1, s2, n = ref.channel_sums(acc)
    assert n == 5 * 17 * 13
    mean, var = ref.bn_stats_from_sums(s1, s2, n, 0.25)
    flat = acc.reshape(-1, 24).astype(np.float64)
    assert np.allclose(mean, 0.25 * flat.mean(0), rtol=1e-12, atol=1e-9)
    assert np.allclose(var, 0.0625 * flat.var(0), rtol=1e-9)


# ---- max-pooling (Sec. 3.2.4) -------------------------------------------------
@pytest.mark.parametrize("k,stride,pad", [(3, 2, 1), (2, 2, 0), (3, 1, 1), (5, 3, 2), (1, 1, 0)])
def test_maxpool_equals_torch_max_pool2d(k, stride, pad):
    """The library routine (float64 on the CPU, padding ignored as -inf) on
    integer codes is exact."""
    rng = np.random.default_rng(k * 100 + stride * 10 + pad)
    x = rng.integers(0, 256, size=(2, 13, 11, 6))
    want = torch.nn.functional.max_pool2d(torch.from_numpy(x).permute(0, 3, 1, 2).double(), k,
                                          stride, pad).permute(0, 2, 3, 1).numpy().astype(np.int64)
    assert np.array_equal(ref.maxpool(x, k, stride, pad), want)


def test_maxpool_brute_force_tiny_and_identity():
    rng = np.random.default_rng(7)
    x = rng.integers(0, 16, size=(1, 5, 4, 3))
    got = ref.maxpool(x, 3, 2, 1)
    ho, wo = (5 + 2 - 3) // 2 + 1, (4 + 2 - 3) // 2 + 1
    assert got.shape == (1, ho, wo, 3)
    for i in range(ho):
        for j in range(wo):
            for c in range(3):
                vals = [x[0, i * 2 - 1 + dy, j * 2 - 1 + dx, c] for dy in range(3) for dx in range(3)
                        if 0 <= i * 2 - 1 + dy < 5 and 0 <= j * 2 - 1 + dx < 4]
                assert got[0, i, j, c] == max(vals)
    assert np.array_equal(ref.maxpool(x, 1, 1, 0), x)


# ------------------------------------- Eq. 7 side/scale rule, requant scale
# These pin the oracle's host derivation of the skip alignment (side, c, d,
# the sum's scale) and of the requantisation multiplier to what Eq. 7-8 and
# Eq. 2 mean: the integer result must track the real-valued sum of the two
# dequantized operands, quantized to the output step. A derivation with the
# wrong side, the larger scale or an inverted ratio fails these checks (each
# such mistake is planted below and must be caught).

def _frac(x):
    return Fraction(float(x))


def test_skip_params_hand_worked_channels():
    az = np.array([0.25, 0.75, 0.5, 0.125, -0.25, -0.75, 0.375])
    ak = np.array([0.75, 0.25, 0.5, 0.3125, 0.75, 0.25, -0.375])
    c, d, side, scale = ref.skip_params(az, ak)
    # 3 = 6/2^1, 1 = 2/2^1, 2.5 = 5/2^1 (dyadic ratios are exact, smallest d)
    assert c.tolist() == [6, 6, 2, 5, -6, -6, -2]
    assert d.tolist() == [1, 1, 1, 1, 1, 1, 1]
    assert side.tolist() == [0, 1, 0, 0, 0, 1, 0]
    assert scale.tolist() == [0.25, 0.25, 0.5, 0.125, -0.25, 0.25, 0.375]


def test_skip_params_rule_with_exact_rationals():
    rng = _rng(71)
    m = 600
    az = np.exp(rng.uniform(np.log(1e-3), np.log(10.0), m)) * rng.choice([-1.0, 1.0], m, p=[0.2, 0.8])
    ak = np.exp(rng.uniform(np.log(1e-3), np.log(10.0), m))
    ak[:50] = np.abs(az[:50])                       # equal magnitudes: side 0, ratio 1
    c, d, side, scale = ref.skip_params(az, ak)
    for i in range(m):
        Z, K = _frac(az[i]), _frac(ak[i])
        big, small = (K, Z) if abs(K) >= abs(Z) else (Z, K)
        assert side[i] == (0 if abs(K) >= abs(Z) else 1)
        assert _frac(scale[i]) == small                       # the smaller scale, signed
        assert abs(_frac(scale[i])) == min(abs(Z), abs(K))
        R = big / small                                       # exact ratio (signed)
        assert (c[i] < 0) == (R < 0)
        assert 1 <= d[i] <= 31 and abs(int(c[i])) < (1 << 31)
        # as good as the largest exponent Eq. 8 allows for this ratio (the
        # ratio itself was rounded once to a double: relative 2^-52)
        dmax = max(e for e in range(1, 32) if abs(R) * (1 << e) + Fraction(1, 2) < (1 << 31))
        err = abs(Fraction(int(c[i]), 1 << int(d[i])) - R)
        assert err <= Fraction(1, 1 << (dmax + 1)) + abs(R) * Fraction(1, 1 << 52)
        if i < 50:
            assert side[i] == 0 and Fraction(int(c[i]), 1 << int(d[i])) == (1 if az[i] > 0 else -1)


def test_requant_params_dyadic_bound():
    rng = _rng(72)
    m = 600
    scale = np.exp(rng.uniform(np.log(1e-6), np.log(50.0), m)) * rng.choice([-1.0, 1.0], m)
    alpha_out = np.exp(rng.uniform(np.log(1e-2), np.log(2.0), m))
    for i in range(m):
        M, sh = ref.requant_params(np.array([scale[i]]), float(alpha_out[i]))
        M, sh = int(M[0]), int(sh[0])
        r = _frac(scale[i]) / _frac(alpha_out[i])
        assert (1 << 30) <= abs(M) < (1 << 31) and -31 <= sh <= 31
        assert (M < 0) == (r < 0)
        err = abs(Fraction(M, 1 << (31 + sh)) - r)
        assert err <= Fraction(1, 1 << (32 + sh)) + abs(r) * Fraction(1, 1 << 52)


_skip_params = ref.skip_params   # the oracle's own, for the planted mistakes below


def _mut_swapped_side(alpha_z, alpha_k):
    c, d, side, scale = _skip_params(alpha_z, alpha_k)
    return c, d, 1 - side, scale


def _mut_max_scale(alpha_z, alpha_k):
    c, d, side, scale = _skip_params(alpha_z, alpha_k)
    az = np.asarray(alpha_z, np.float64)
    ak = np.broadcast_to(np.asarray(alpha_k, np.float64), az.shape)
    return c, d, side, np.where(side == 0, ak, az)


def _mut_inverted_ratio(alpha_z, alpha_k):
    c, d, side, scale = _skip_params(alpha_z, alpha_k)
    inv = [int(round(2.0 ** 30 * (1 << int(di)) / ci)) for ci, di in zip(c, d)]
    return np.array(inv, np.int64), np.full(c.shape, 30, np.int64), side, scale


def _skip_add_violations(derive, rng, m=4000):
    """Integer skip add + requantisation (the oracle's qadd) against the real
    sum of the dequantized operands; returns the number of outputs outside
    the error bound of Eq. 7-8 and Eq. 2."""
    qm = 15
    az = np.exp(rng.uniform(np.log(0.02), np.log(0.2), m))
    ratio = np.exp(rng.uniform(np.log(1.5), np.log(8.0), m))
    flip = rng.random(m) < 0.5
    ak = np.where(flip, az * ratio, az / ratio)                    # both sides
    az = az * np.where(rng.random(m) < 0.25, -1.0, 1.0)           # gamma < 0 channels
    alpha_out = 0.2
    v = rng.integers(-200, 201, m)
    k = rng.integers(0, 16, m)
    c, d, side, scale = derive(az, ak)
    mult, shift = ref.requant_params(scale, alpha_out)
    # one channel per element
    out = ref.qadd(v.reshape(1, 1, 1, m), k.reshape(1, 1, 1, m), False, c, d, side, mult, shift,
                   4).reshape(m)
    real = (az * v + ak * k) / alpha_out
    small = np.minimum(np.abs(az), np.abs(ak))
    # alignment rounding (1/2 of the smaller scale) + dyadic approximations
    # (below 1e-6 here) + the final rounding
    bound = 0.5 * small / alpha_out + 1e-6 + 0.5
    return int(np.sum(np.abs(out - np.clip(real, 0, qm)) > bound))


def test_skip_add_requant_tracks_the_real_sum():
    assert _skip_add_violations(ref.skip_params, _rng(73)) == 0


@pytest.mark.parametrize("mutant", [_mut_swapped_side, _mut_max_scale, _mut_inverted_ratio])
def test_skip_add_real_sum_check_catches_planted_mistakes(mutant):
    assert _skip_add_violations(mutant, _rng(73)) > 400


def _tiny_residual_net():
    """Identity code skip, int32 projection skip and an upsampled code skip,
    every conv calibrated (odd weight grid, 4-bit codes)."""
    from paper_2007_06919_amd import workloads as wl
    net = wl.NetSpec(wenc=wl.WENC_PAPER_ODD)
    net.add_tensor("x", 1, 8, 9, 64, 4)
    net.add_tensor("u", 1, 4, 5, 64, 4)
    net.inputs += ["x", "u"]
    net.conv("c1", "x", "a", 64, 3, 1, 4, 4)
    net.conv("c2", "a", "b", 64, 3, 1, 4, 4, skip="x")
    net.conv("dn", "x", "ds", 64, 1, 1, 4, 32)
    net.conv("c3", "b", "o", 64, 1, 1, 4, 4, skip="ds")
    net.conv("lat", "o", "p", 64, 1, 1, 4, 4, skip="u", skip_up2=True)
    net.outputs.append("p")
    params = wl.make_params(net, 74, "calibrated")
    rng = _rng(75)
    for segs in params.segs.values():       # a quarter of the channels with gamma < 0
        for sp in segs:
            sp["gamma"] = sp["gamma"] * np.where(rng.random(sp["gamma"].size) < 0.25, -1.0, 1.0)
    return net, params


def _float_layer_violations(net, params, vals):
    """Each layer in float64 from the oracle's integer inputs to it:
    dequantize (Eq. 1), convolve, batch-normalise with the calibration
    image's statistics, add the dequantized skip, quantize to the output
    step (Eq. 2). Returns the number of outputs outside the error bound of
    the integer path (folded-bias rounding, Eq. 6; alignment rounding, Eq. 7;
    final rounding)."""
    bad = 0
    real, az_of = {}, {}
    for conv in net.convs:
        x, skip, y = conv.segs[0]
        ax = params.alpha[x]
        aw = 1.0 / 15.0
        wv = 2.0 * params.weights[conv.name].astype(np.float64) - 15.0       # Eq. 3 grid
        xr = torch.from_numpy(ax * vals[x].astype(np.float64)).permute(0, 3, 1, 2)
        wr = torch.from_numpy(aw * wv).permute(0, 3, 1, 2)
        z = torch.nn.functional.conv2d(xr, wr, padding=conv.pad, stride=conv.stride)
        z = z.permute(0, 2, 3, 1).numpy()
        zz = z.reshape(-1, conv.cout)
        mu = zz.mean(axis=0)
        var = (zz * zz).mean(axis=0) - mu * mu
        sp = params.segs[conv.name][0]
        sd = np.sqrt(var + params.bn_eps)
        bn = sp["gamma"] * (z - mu) / sd + sp["beta"]
        az = (ax * aw) * sp["gamma"] / sd
        if net.tensors[y].bits == 32:
            # v = acc + round(s) carries the scale alpha_z (Eq. 6): within alpha_z / 2
            assert np.all(np.abs(az * vals[y] - bn) <= np.abs(az) / 2 + 1e-9)
            real[y], az_of[y] = bn, az
            continue
        ay = params.alpha[y]
        extra = np.abs(az)                                   # this conv's bias rounding
        pre = bn
        if skip is not None:
            if net.tensors[skip].bits == 32:
                sk, ak = real[skip], az_of[skip]
                extra = extra + np.abs(ak)                   # the skip's own bias rounding
            else:
                ks = vals[skip]
                if conv.skip_up2:
                    ks = ks[:, np.arange(z.shape[1]) >> 1][:, :, np.arange(z.shape[2]) >> 1]
                ak = params.alpha[skip]
                sk = ak * ks
            pre = bn + sk
            extra = extra + np.minimum(np.abs(az), np.abs(ak))   # alignment rounding
        target = np.clip(pre / ay, 0, 15)
        bound = 0.5 + extra / (2 * ay) + 1e-6
        bad += int(np.sum(np.abs(vals[y] - target) > bound))
    return bad


def test_calibrated_residual_network_tracks_float64():
    from oracle import network
    net, params = _tiny_residual_net()
    vals, tables = network.run(net, params)
    assert any(int(c) < 0 for t in tables.values() for s in t for c in s.get("skip_c", []))
    assert any(int(m) < 0 for t in tables.values() for s in t for m in s.get("mult", []))
    interior = [np.mean((vals[t] > 0) & (vals[t] < 15)) for t in ("a", "b", "o", "p")]
    assert min(interior) > 0.2, interior
    assert _float_layer_violations(net, params, vals) == 0


@pytest.mark.parametrize("mutant", [_mut_swapped_side, _mut_max_scale, _mut_inverted_ratio])
def test_float64_network_check_catches_planted_mistakes(mutant, monkeypatch):
    from oracle import network
    net, params = _tiny_residual_net()
    monkeypatch.setattr(ref, "skip_params", mutant)
    vals, _ = network.run(net, params)
    assert _float_layer_violations(net, params, vals) > 100
