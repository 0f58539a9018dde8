"""CPU oracle for AQD's integer-only inference path (arXiv 2007.06919).

TEST INFRASTRUCTURE: only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import this module. It shares no code with
the GPU path (its packing, decoding, parameter derivation and arithmetic are
written here independently) and imports nothing from the product package.

Contents, each following the paper:
  * Eq. 2 / Eq. 3 float quantizers (host reference for the pins),
  * weight decoding for the two weight grids (Eq. 3/4, two's complement),
  * the integer convolution + epilogue and the standalone skip add, run by
    the C nested-loop code in ``qconv_oracle.c`` (Eq. 4, 6, 7, 8 and Eq. 2
    carried out on integers),
  * host parameter derivation: BN folding (Eq. 5-6), the power-of-two ratio
    approximation F (Eq. 8), the dyadic requantisation multiplier,
  * packing of b-bit codes along the channel axis (the storage format of a
    code tensor: channel c occupies bits (c*b) mod 8 .. of byte (c*b) div 8).

Rounding ``round(.)`` is round-half-up (floor(x + 1/2)) throughout; the paper
only says "nearest integer".
"""
from __future__ import annotations

import ctypes
import math
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")

WENC_TWOS = 0       # b-bit two's complement weight fields
WENC_PAPER_ODD = 1  # Eq. 3 fields eta_w, value 2*eta_w - (2^b - 1)

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"oracle library not built: {LIB_PATH} (run oracle/build.py)")
        L = ctypes.CDLL(LIB_PATH)
        p = ctypes.c_void_p
        i = ctypes.c_int
        L.oracle_qconv.argtypes = [i, i, i, i, p, i, i, i, i, i, p, p, i, p, p, i,
                                   p, i, i, i, p, p, p, i, i, p]
        L.oracle_qconv.restype = i
        L.oracle_qadd.argtypes = [i, i, i, i, p, i, i, i, p, p, p, p, p, p, i, p]
        L.oracle_qadd.restype = i
        L.oracle_rsm_array.argtypes = [ctypes.c_int64, p, p, p, p, p]
        L.oracle_rsm_array.restype = None
        L.oracle_num_threads.argtypes = []
        L.oracle_num_threads.restype = i
        _lib = L
    return _lib


def num_threads() -> int:
    return lib().oracle_num_threads()


def qmax(bits: int) -> int:
    return (1 << bits) - 1


def round_half_up(x):
    return np.floor(np.asarray(x, dtype=np.float64) + 0.5)


# ---------------------------------------------------------------- Eq. 2 / 3
def quantize_activation(x, nu, bits):
    """Eq. 2: eta = round(clip(x / nu, 0, 1) * (2^b - 1)); value = eta * nu / (2^b - 1)."""
    q = qmax(bits)
    eta = round_half_up(np.clip(np.asarray(x, np.float64) / nu, 0.0, 1.0) * q)
    return eta.astype(np.int64), eta * (nu / q)


def quantize_weight(w, nu, bits):
    """Eq. 3: eta = round((clip(w / nu, -1, 1) + 1) / 2 * (2^b - 1));
    value = (2 * eta / (2^b - 1) - 1) * nu."""
    q = qmax(bits)
    eta = round_half_up((np.clip(np.asarray(w, np.float64) / nu, -1.0, 1.0) + 1.0) / 2.0 * q)
    return eta.astype(np.int64), (eta * (1.0 / q) * 2.0 - 1.0) * nu


def decode_weights(fields, bits, wenc=WENC_TWOS):
    """Integer weight values from b-bit fields.

    Paper grid (Eq. 3-4): the factor multiplying eta_x is 2*eta_w - 2^b + 1.
    Two's complement: a field f >= 2^(b-1) stands for f - 2^b.
    """
    f = np.asarray(fields, dtype=np.int64)
    if wenc == WENC_PAPER_ODD:
        return 2 * f - qmax(bits)
    return np.where(f >= (1 << (bits - 1)), f - (1 << bits), f)


# ----------------------------------------------------------------- packing
def container_bits(bits):
    """Bits one code occupies in a tensor: 3-bit codes (the paper's 3-bit
    networks, Tables 2 and 4) sit in 4-bit containers, the others fill their
    width."""
    return 4 if bits == 3 else bits


def pack_codes(codes, bits):
    """Pack b-bit codes along the last (channel) axis, little-endian within a
    byte: channel j of a group of 8/s sits at bits j*s .. j*s+b-1, where s is
    the container width (s = b, or 4 for b = 3)."""
    codes = np.asarray(codes)
    if bits == 8:
        return codes.astype(np.uint8)
    s = container_bits(bits)
    per = 8 // s
    c = codes.shape[-1]
    assert c % per == 0, "channels * bits must be a multiple of 8"
    grp = codes.astype(np.uint32).reshape(codes.shape[:-1] + (c // per, per))
    out = np.zeros(grp.shape[:-1], dtype=np.uint32)
    for j in range(per):
        out |= (grp[..., j] & qmax(bits)) << (j * s)
    return out.astype(np.uint8)


def unpack_codes(packed, bits, c):
    """Inverse of ``pack_codes``: [..., c*s/8] bytes -> [..., c] codes."""
    packed = np.asarray(packed, dtype=np.uint8)
    if bits == 8:
        return packed.astype(np.int64)
    s = container_bits(bits)
    per = 8 // s
    b = packed.astype(np.int64)
    parts = [(b >> (j * s)) & qmax(bits) for j in range(per)]
    out = np.stack(parts, axis=-1)
    return out.reshape(packed.shape[:-1] + (c,))


# --------------------------------------------------------------- the conv
def _i32(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _i64(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.int64))


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


ORACLE_ERRORS = {1: "accumulator outside int32", 2: "acc + bias outside int32",
                 3: "skip-aligned sum outside int32", 4: "bad arguments"}


def qconv(x, w_fields, bits_w, stride, pad, bias, *, wenc=WENC_TWOS, out_int32=False,
          mult=None, shift=None, bits_out=4, skip=None, skip_up2=False,
          skip_c=None, skip_d=None, skip_side=None):
    """Integer conv + epilogue (Eq. 4, 6, 7-8, requantisation per Eq. 2).

    x: [n, h, w, cin] codes; w_fields: [cout, kh, kw, cin] b-bit fields;
    skip: [n, hs, ws, cout] integer values (codes or int32) or None.
    Returns int64 [n, ho, wo, cout]: codes in [0, 2^bits_out - 1], or v = acc + bias.
    """
    x = _i32(x)
    wv = _i32(decode_weights(w_fields, bits_w, wenc))
    n, h, w, cin = x.shape
    cout, kh, kw, cin2 = wv.shape
    assert cin == cin2
    ho = (h + 2 * pad - kh) // stride + 1
    wo = (w + 2 * pad - kw) // stride + 1
    out = np.zeros((n, ho, wo, cout), dtype=np.int64)
    bias = _i32(bias)
    if out_int32:
        mult = shift = None
        q = 0
    else:
        mult, shift, q = _i32(mult), _i32(shift), qmax(bits_out)
    if skip is not None:
        skip = _i64(skip)
        _, hs, ws, cs = skip.shape
        assert cs == cout
        sc, sd, ss = _i32(skip_c), _i32(skip_d), _i32(skip_side)
    else:
        hs = ws = 0
        sc = sd = ss = None
    rc = lib().oracle_qconv(n, h, w, cin, _ptr(x), cout, kh, kw, stride, pad, _ptr(wv),
                            _ptr(bias), int(out_int32), _ptr(mult), _ptr(shift), q,
                            _ptr(skip), int(skip_up2), hs, ws, _ptr(sc), _ptr(sd), _ptr(ss),
                            ho, wo, _ptr(out))
    if rc != 0:
        raise ValueError(f"oracle_qconv: {ORACLE_ERRORS.get(rc, rc)}")
    return out


def qadd(a, b, up2, skip_c, skip_d, skip_side, mult, shift, bits_out):
    """Standalone skip connection (Eq. 7) + requantisation; b optionally the
    coarser map of a nearest 2x upsample."""
    a, b = _i64(a), _i64(b)
    n, h, w, c = a.shape
    _, hb, wb, cb = b.shape
    assert cb == c
    out = np.zeros_like(a)
    rc = lib().oracle_qadd(n, h, w, c, _ptr(a), int(up2), hb, wb, _ptr(b),
                           _ptr(_i32(skip_c)), _ptr(_i32(skip_d)), _ptr(_i32(skip_side)),
                           _ptr(_i32(mult)), _ptr(_i32(shift)), qmax(bits_out), _ptr(out))
    if rc != 0:
        raise ValueError(f"oracle_qadd: {ORACLE_ERRORS.get(rc, rc)}")
    return out


def maxpool(x, k, stride, pad):
    """Max-pooling of codes (Sec. 3.2.4: the layer leaves the scale factor
    unchanged, so the codes are pooled as they are). x: [n, h, w, c] codes;
    y[n, i, j, c] = max of x over the k x k window whose top-left input
    position is (i * stride - pad, j * stride - pad); positions outside the
    input are skipped. Returns int64 [n, ho, wo, c]."""
    x = _i64(x)
    n, h, w, c = x.shape
    ho = (h + 2 * pad - k) // stride + 1
    wo = (w + 2 * pad - k) // stride + 1
    assert ho >= 1 and wo >= 1
    out = np.full((n, ho, wo, c), -1, dtype=np.int64)
    for dy in range(k):
        ih = np.arange(ho) * stride - pad + dy
        vi = (ih >= 0) & (ih < h)
        for dx in range(k):
            iw = np.arange(wo) * stride - pad + dx
            vj = (iw >= 0) & (iw < w)
            if not vi.any() or not vj.any():
                continue
            win = x[:, ih[vi]][:, :, iw[vj]]               # [n, |vi|, |vj|, c]
            sub = out[:, vi][:, :, vj]
            out[np.ix_(np.arange(n), np.nonzero(vi)[0], np.nonzero(vj)[0], np.arange(c))] = \
                np.maximum(sub, win)
    assert (out >= 0).all(), "every window holds at least one input position"
    return out


def rsm_array(a, c, d):
    """RSM over arrays via the C code; returns Python ints (exact)."""
    a, c = _i64(a).ravel(), _i64(c).ravel()
    d = _i32(d).ravel()
    hi = np.zeros(a.shape, np.int64)
    lo = np.zeros(a.shape, np.uint64)
    lib().oracle_rsm_array(a.size, _ptr(a), _ptr(c), _ptr(d), _ptr(hi), _ptr(lo))
    # a two's-complement 128-bit value is hi * 2^64 + lo with hi signed, lo unsigned
    return [int(h_) * (1 << 64) + int(l_) for h_, l_ in zip(hi, lo)]


# ------------------------------------------------- host parameter derivation
I32_MAX = (1 << 31) - 1


def approx_ratio(r):
    """Eq. 8: F = c / 2^d with c a natural number, d a positive integer,
    minimising |r - c/2^d|. Domain used here: d in [1, 31], c < 2^31; among
    equally good pairs the smallest d. Requires 1 <= r < 2^30 (Eq. 8 is used
    with m >= n)."""
    r = float(r)
    if not (math.isfinite(r) and 1.0 <= r < 2.0 ** 30):
        raise ValueError(f"approx_ratio: ratio {r} outside [1, 2^30)")
    best = None
    best_err = None
    for d in range(1, 32):
        x = math.ldexp(r, d)
        if x + 0.5 >= 2.0 ** 31:
            break
        c = math.floor(x + 0.5)
        err = abs(r - math.ldexp(c, -d))
        if best is None or err < best_err:
            best, best_err = (c, d), err
    return best


def normalize_multiplier(r):
    """Dyadic form M / 2^(31 + shift) of a real scale r != 0, with
    |M| in [2^30, 2^31) and shift in [-31, 31]; M = round(|r| * 2^(31+shift))."""
    r = float(r)
    if not math.isfinite(r) or r == 0.0:
        raise ValueError("normalize_multiplier: scale must be finite and non-zero")
    sign = -1 if r < 0 else 1
    a = abs(r)
    _, e = math.frexp(a)          # a = m * 2^e, m in [0.5, 1): floor(log2 a) = e - 1
    d = 31 - e                    # a * 2^d in [2^30, 2^31)
    c = math.floor(math.ldexp(a, d) + 0.5)
    if c == 1 << 31:
        c, d = 1 << 30, d - 1
    shift = d - 31
    if not -31 <= shift <= 31:
        raise ValueError(f"normalize_multiplier: scale {r} out of range")
    return sign * c, shift


def fold_bn(gamma, beta, mean, var, eps, alpha_conv):
    """Eq. 5-6: s = (beta * sqrt(var + eps) / gamma - mean) / alpha_conv,
    bias = round(s), alpha_z = alpha_conv * gamma / sqrt(var + eps)."""
    gamma, beta = np.asarray(gamma, np.float64), np.asarray(beta, np.float64)
    mean, var = np.asarray(mean, np.float64), np.asarray(var, np.float64)
    bias = np.zeros(gamma.shape, np.int64)
    alpha_z = np.zeros(gamma.shape, np.float64)
    for i in range(gamma.size):
        g, b_, m, v = float(gamma[i]), float(beta[i]), float(mean[i]), float(var[i])
        if g == 0.0 or not v + eps > 0.0:
            raise ValueError("fold_bn: gamma must be non-zero and var + eps positive")
        sd = math.sqrt(v + eps)
        s = (b_ * sd / g - m) / alpha_conv
        rb = math.floor(s + 0.5)
        if not -(1 << 31) < rb < (1 << 31):
            raise ValueError("fold_bn: bias outside int32")
        bias[i] = rb
        alpha_z[i] = alpha_conv * g / sd
    return bias, alpha_z


def channel_sums(acc):
    """Exact per-channel sums of an int accumulator tensor [..., c]:
    (sum acc, sum acc^2, count) as Python integers."""
    a = np.asarray(acc, dtype=np.int64).reshape(-1, np.asarray(acc).shape[-1])
    big = int(np.abs(a).max(initial=0))
    if big < (1 << 31) and a.shape[0] * big * big < (1 << 63):
        # no int64 overflow possible: exact in machine integers
        s1 = [int(v) for v in a.sum(axis=0)]
        s2 = [int(v) for v in (a * a).sum(axis=0)]
    else:
        s1 = [int(v) for v in a.sum(axis=0, dtype=object)]
        s2 = [int(v) for v in (a.astype(object) ** 2).sum(axis=0)]
    return s1, s2, a.shape[0]


def bn_stats_from_sums(s1, s2, count, alpha_conv):
    """Running statistics of BN from exact accumulator sums, in real units:
    mean = alpha_conv * (s1 / count), var = alpha_conv^2 * (s2 / count - m^2)."""
    mean = np.zeros(len(s1), np.float64)
    var = np.zeros(len(s1), np.float64)
    for i in range(len(s1)):
        m = float(s1[i]) / float(count)
        va = float(s2[i]) / float(count) - m * m
        mean[i] = alpha_conv * m
        var[i] = (alpha_conv * alpha_conv) * va
    return mean, var


def skip_params(alpha_z, alpha_k):
    """Per channel, Eq. 7-8: the operand whose scale is larger in magnitude is
    rescaled to the other one's scale, and the sum carries the smaller scale.

    side 0 (|alpha_k| >= |alpha_z|): the skip operand is multiplied by
        c / 2^d ~ alpha_k / alpha_z, the sum's scale is alpha_z;
    side 1 (|alpha_k| < |alpha_z|): the conv operand is multiplied by
        c / 2^d ~ alpha_z / alpha_k, the sum's scale is alpha_k.
    (c, d) = F of the magnitude of the ratio (Eq. 8, ratio >= 1), with c
    negated when the two scales have opposite signs (a normalisation with
    gamma < 0 gives a negative alpha_z; the paper's scales are positive, where
    this is exactly its rule). Returns c, d, side and the sum's scale."""
    alpha_z = np.asarray(alpha_z, np.float64)
    alpha_k = np.broadcast_to(np.asarray(alpha_k, np.float64), alpha_z.shape)
    c = np.zeros(alpha_z.shape, np.int64)
    d = np.zeros(alpha_z.shape, np.int64)
    side = np.zeros(alpha_z.shape, np.int64)
    scale = np.zeros(alpha_z.shape, np.float64)
    for i in range(alpha_z.size):
        az, ak = float(alpha_z[i]), float(alpha_k[i])
        if az == 0.0 or ak == 0.0:
            raise ValueError("skip_params: scales must be non-zero")
        sign = -1 if (az < 0) != (ak < 0) else 1
        if abs(ak) >= abs(az):
            ci, d[i] = approx_ratio(abs(ak / az))
            side[i], scale[i] = 0, az
        else:
            ci, d[i] = approx_ratio(abs(az / ak))
            side[i], scale[i] = 1, ak
        c[i] = sign * ci
    return c, d, side, scale


def requant_params(scale, alpha_out):
    """Multiplier/shift of the requantisation to codes of step alpha_out."""
    scale = np.asarray(scale, np.float64)
    mult = np.zeros(scale.shape, np.int64)
    shift = np.zeros(scale.shape, np.int64)
    for i in range(scale.size):
        mult[i], shift[i] = normalize_multiplier(float(scale[i]) / alpha_out)
    return mult, shift
