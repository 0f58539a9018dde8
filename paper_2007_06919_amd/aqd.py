"""ctypes binding of ``libaqd.so`` (declarations in include/aqd.h).

Argument marshalling only: every computation runs in the library. Tensor
arguments may be torch tensors (their data pointer is passed), plain integer
addresses, or None. Streams default to torch's current stream. The library
is loaded on first use; if it is missing this raises instead of falling back
to anything else.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_double, c_int, c_int32, c_int64, c_void_p

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libaqd.so")

AQD_OK, AQD_ERR_INVALID, AQD_ERR_UNSUPPORTED, AQD_ERR_NOMEM, AQD_ERR_DEVICE = range(5)
WENC_TWOS, WENC_PAPER_ODD = 0, 1
OUT_CODES, OUT_INT32 = 0, 1
MAX_SEGS = 16

STATUS_NAMES = {0: "AQD_OK", 1: "AQD_ERR_INVALID", 2: "AQD_ERR_UNSUPPORTED",
                3: "AQD_ERR_NOMEM", 4: "AQD_ERR_DEVICE"}


class AqdError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class QconvDesc(ctypes.Structure):
    _fields_ = [(n, c_int) for n in ("cin", "cout", "kh", "kw", "stride", "pad", "bits_in",
                                     "bits_w", "wenc", "out_mode", "bits_out", "skip_bits",
                                     "skip_up2", "num_levels")] + \
               [(n, c_double) for n in ("step_in", "step_w", "step_out")]


class QconvEpilogue(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("bias", "mult", "shift", "skip_c", "skip_d", "skip_side")]


class QconvSeg(ctypes.Structure):
    _fields_ = [("conv", c_void_p), ("level", c_int), ("n", c_int), ("h", c_int), ("w", c_int),
                ("x", c_void_p), ("skip", c_void_p), ("hs", c_int), ("ws", c_int),
                ("y", c_void_p)]


class QaddDesc(ctypes.Structure):
    _fields_ = [(n, c_int) for n in ("n", "h", "w", "c", "bits_a", "bits_b", "bits_out", "up2",
                                     "hb", "wb")]


class MaxpoolDesc(ctypes.Structure):
    _fields_ = [(n, c_int) for n in ("n", "h", "w", "c", "bits", "k", "stride", "pad")]


class QaddParams(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("skip_c", "skip_d", "skip_side", "mult", "shift")]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build() first")
        L = ctypes.CDLL(LIB_PATH)
        vp, i, st = c_void_p, c_int, c_int
        sig = {
            "qconv_create": ([POINTER(QconvDesc), vp, POINTER(QconvEpilogue), POINTER(c_void_p)], st),
            "qconv_out_shape": ([vp, i, i, POINTER(c_int), POINTER(c_int)], st),
            "qconv_scales": ([vp, POINTER(c_double), POINTER(c_double)], st),
            "qconv_run": ([vp, i, i, i, i, vp, vp, i, i, vp, vp], st),
            "qconv_run_group": ([i, POINTER(QconvSeg), vp], st),
            "qconv_group_workspace": ([i, POINTER(QconvSeg), POINTER(ctypes.c_size_t)], st),
            "qconv_run_group_ws": ([i, POINTER(QconvSeg), vp, ctypes.c_size_t, vp], st),
            "qconv_run_group_static": ([i, POINTER(QconvSeg), vp], st),
            "qconv_run_proj": ([vp, vp, i, i, i, i, vp, i, i, vp, vp, vp], st),
            "qconv_destroy": ([vp], None),
            "qconv_path": ([vp], ctypes.c_char_p),
            "qadd_run": ([POINTER(QaddDesc), vp, vp, vp, POINTER(QaddParams), vp], st),
            "aqd_channel_sums": ([vp, c_int64, i, vp, vp], st),
            "aqd_maxpool_run": ([POINTER(MaxpoolDesc), vp, vp, vp], st),
            "aqd_mfma_probe": ([i, i, vp, vp], st),
            "aqd_graph_begin": ([vp], st),
            "aqd_graph_end": ([vp, POINTER(c_void_p)], st),
            "aqd_graph_launch": ([vp, vp], st),
            "aqd_graph_destroy": ([vp], None),
            "aqd_last_error": ([], ctypes.c_char_p),
            "aqd_pack_codes": ([vp, c_int64, i, i, vp], st),
            "aqd_unpack_codes": ([vp, c_int64, i, i, vp], st),
            "aqd_approx_ratio": ([c_double, POINTER(c_int32), POINTER(c_int32)], st),
            "aqd_normalize_multiplier": ([c_double, POINTER(c_int32), POINTER(c_int32)], st),
            "aqd_bn_stats_from_sums": ([i, vp, vp, c_int64, c_double, vp, vp], st),
            "aqd_fold_bn": ([i, vp, vp, vp, vp, c_double, c_double, vp, vp], st),
            "aqd_skip_params": ([i, vp, vp, i, vp, vp, vp, vp], st),
            "aqd_requant_params": ([i, vp, c_double, vp, vp], st),
        }
        for name, (args, res) in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def exported_symbols():
    return ["qconv_create", "qconv_out_shape", "qconv_scales", "qconv_run", "qconv_run_group",
            "qconv_group_workspace", "qconv_run_group_ws", "qconv_run_group_static",
            "qconv_run_proj", "qconv_destroy", "qconv_path",
            "qadd_run", "aqd_maxpool_run", "aqd_mfma_probe", "aqd_channel_sums", "aqd_graph_begin", "aqd_graph_end",
            "aqd_graph_launch", "aqd_graph_destroy", "aqd_last_error", "aqd_pack_codes",
            "aqd_unpack_codes", "aqd_approx_ratio", "aqd_normalize_multiplier",
            "aqd_bn_stats_from_sums", "aqd_fold_bn", "aqd_skip_params", "aqd_requant_params"]


def last_error() -> str:
    return lib().aqd_last_error().decode()


def _check(status):
    if status != AQD_OK:
        raise AqdError(status, last_error())


def _addr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _host(a, dtype):
    return np.ascontiguousarray(np.asarray(a, dtype=dtype))


# ------------------------------------------------------------------ qconv
def qconv_create(cin, cout, k, stride, pad, bits_in, bits_w, w_packed, levels, *,
                 wenc=WENC_TWOS, out_mode=OUT_CODES, bits_out=4, skip_bits=0, skip_up2=0,
                 step_in=0.0, step_w=0.0, step_out=0.0):
    """levels: list of dicts with int32 arrays 'bias' and, as the mode needs,
    'mult', 'shift', 'skip_c', 'skip_d', 'skip_side'. step_*: the step sizes
    (0: not given). Returns the handle."""
    d = QconvDesc(cin, cout, k, k, stride, pad, bits_in, bits_w, wenc, out_mode, bits_out,
                  skip_bits, int(skip_up2), len(levels), float(step_in), float(step_w),
                  float(step_out))
    keep = []
    eps = (QconvEpilogue * len(levels))()
    for i, lv in enumerate(levels):
        for name in ("bias", "mult", "shift", "skip_c", "skip_d", "skip_side"):
            if lv.get(name) is not None:
                a = _host(lv[name], np.int32)
                keep.append(a)
                setattr(eps[i], name, a.ctypes.data)
    w = _host(w_packed, np.uint8)
    h = c_void_p()
    _check(lib().qconv_create(ctypes.byref(d), w.ctypes.data, eps, ctypes.byref(h)))
    return h.value


def qconv_out_shape(conv, h, w):
    ho, wo = c_int(), c_int()
    _check(lib().qconv_out_shape(conv, h, w, ctypes.byref(ho), ctypes.byref(wo)))
    return ho.value, wo.value


def qconv_scales(conv):
    """(alpha_conv, step_out) of a handle created with its step sizes."""
    a, o = c_double(), c_double()
    _check(lib().qconv_scales(conv, ctypes.byref(a), ctypes.byref(o)))
    return a.value, o.value


def qconv_run(conv, level, n, h, w, x, skip, hs, ws, y, stream=None):
    _check(lib().qconv_run(conv, level, n, h, w, _addr(x), _addr(skip), hs, ws, _addr(y),
                           _stream(stream)))


def _seg_array(segs):
    arr = (QconvSeg * len(segs))()
    for i, (conv, level, n, h, w, x, skip, hs, ws, y) in enumerate(segs):
        arr[i] = QconvSeg(conv, level, n, h, w, _addr(x), _addr(skip), hs, ws, _addr(y))
    return arr


def qconv_run_group(segs, stream=None):
    """segs: list of tuples (conv, level, n, h, w, x, skip, hs, ws, y)."""
    _check(lib().qconv_run_group(len(segs), _seg_array(segs), _stream(stream)))


def qconv_group_workspace(segs) -> int:
    """Workspace bytes with which qconv_run_group_ws splits the K reduction
    of this group (0: never split)."""
    b = ctypes.c_size_t(0)
    _check(lib().qconv_group_workspace(len(segs), _seg_array(segs), ctypes.byref(b)))
    return b.value


def qconv_run_group_ws(segs, workspace, ws_bytes, stream=None):
    _check(lib().qconv_run_group_ws(len(segs), _seg_array(segs), _addr(workspace), ws_bytes,
                                    _stream(stream)))


def qconv_run_group_static(segs, stream=None):
    """qconv_run_group_ws on the library's static scratch (allocates nothing)."""
    _check(lib().qconv_run_group_static(len(segs), _seg_array(segs), _stream(stream)))


def qconv_run_proj(conv, proj, level, n, h, w, x, hp, wp, xp, y, stream=None):
    """Residual tail with the projection shortcut fused (see aqd.h)."""
    _check(lib().qconv_run_proj(conv, proj, level, n, h, w, _addr(x), hp, wp, _addr(xp), _addr(y),
                                _stream(stream)))


def qconv_destroy(conv):
    if conv:
        lib().qconv_destroy(conv)


def qconv_path(conv) -> str:
    """'fp4-mfma', 'i8-mfma' or 'direct': the arithmetic of the handle's launches."""
    return lib().qconv_path(conv).decode()


# ------------------------------------------------------------------- qadd
def qadd_run(n, h, w, c, bits_a, bits_b, bits_out, up2, hb, wb, a, b, y, params, stream=None):
    """params: dict of device int32 tensors skip_c, skip_d, skip_side, mult, shift."""
    d = QaddDesc(n, h, w, c, bits_a, bits_b, bits_out, int(up2), hb, wb)
    p = QaddParams(*[_addr(params[k]) for k in ("skip_c", "skip_d", "skip_side", "mult", "shift")])
    _check(lib().qadd_run(ctypes.byref(d), _addr(a), _addr(b), _addr(y), ctypes.byref(p),
                          _stream(stream)))


def channel_sums(v, rows, c, sums, stream=None):
    _check(lib().aqd_channel_sums(_addr(v), rows, c, _addr(sums), _stream(stream)))


def maxpool_run(n, h, w, c, bits, k, stride, pad, x, y, stream=None):
    """Max-pooling of a code tensor (see aqd.h)."""
    d = MaxpoolDesc(n, h, w, c, bits, k, stride, pad)
    _check(lib().aqd_maxpool_run(ctypes.byref(d), _addr(x), _addr(y), _stream(stream)))


def mfma_probe(workgroups, iters, out, stream=None):
    """The matrix-core rate probe (see aqd.h); out: device int32 tensor of
    workgroups x 256 entries."""
    _check(lib().aqd_mfma_probe(workgroups, iters, _addr(out), _stream(stream)))


def graph_begin(stream):
    """Start recording the library calls on `stream` (not the null stream)."""
    _check(lib().aqd_graph_begin(_stream(stream)))


def graph_end(stream) -> int:
    """End the recording; returns the executable graph handle."""
    h = c_void_p()
    _check(lib().aqd_graph_end(_stream(stream), ctypes.byref(h)))
    return h.value


def graph_launch(graph, stream=None):
    _check(lib().aqd_graph_launch(graph, _stream(stream)))


def graph_destroy(graph):
    lib().aqd_graph_destroy(graph)


# ----------------------------------------------------------- host helpers
def stored_bits(bits):
    """Bits a code of width ``bits`` takes in a tensor (3-bit codes sit in
    4-bit containers; int32 tensors: 32)."""
    return 4 if bits == 3 else bits


def pack_codes(codes, bits):
    codes = _host(codes, np.uint8)
    c = codes.shape[-1]
    rows = codes.size // c
    out = np.empty(codes.shape[:-1] + (c * stored_bits(bits) // 8,), np.uint8)
    _check(lib().aqd_pack_codes(codes.ctypes.data, rows, c, bits, out.ctypes.data))
    return out


def unpack_codes(packed, bits, c):
    packed = _host(packed, np.uint8)
    rows = packed.size // (c * stored_bits(bits) // 8)
    out = np.empty(packed.shape[:-1] + (c,), np.uint8)
    _check(lib().aqd_unpack_codes(packed.ctypes.data, rows, c, bits, out.ctypes.data))
    return out


def approx_ratio(r):
    c, d = c_int32(), c_int32()
    _check(lib().aqd_approx_ratio(float(r), ctypes.byref(c), ctypes.byref(d)))
    return c.value, d.value


def normalize_multiplier(r):
    m, s = c_int32(), c_int32()
    _check(lib().aqd_normalize_multiplier(float(r), ctypes.byref(m), ctypes.byref(s)))
    return m.value, s.value


def bn_stats_from_sums(s1, s2, count, alpha_conv):
    s1, s2 = _host(s1, np.int64), _host(s2, np.int64)
    mean = np.empty(s1.size, np.float64)
    var = np.empty(s1.size, np.float64)
    _check(lib().aqd_bn_stats_from_sums(s1.size, s1.ctypes.data, s2.ctypes.data, int(count),
                                        float(alpha_conv), mean.ctypes.data, var.ctypes.data))
    return mean, var


def fold_bn(gamma, beta, mean, var, eps, alpha_conv):
    g, b, m, v = (_host(a, np.float64) for a in (gamma, beta, mean, var))
    bias = np.empty(g.size, np.int32)
    alpha_z = np.empty(g.size, np.float64)
    _check(lib().aqd_fold_bn(g.size, g.ctypes.data, b.ctypes.data, m.ctypes.data, v.ctypes.data,
                             float(eps), float(alpha_conv), bias.ctypes.data, alpha_z.ctypes.data))
    return bias, alpha_z


def skip_params(alpha_z, alpha_k):
    az = _host(alpha_z, np.float64)
    ak = _host(np.atleast_1d(alpha_k), np.float64)
    per_channel = int(ak.size == az.size and ak.size > 1)
    c = np.empty(az.size, np.int32)
    d = np.empty(az.size, np.int32)
    side = np.empty(az.size, np.int32)
    scale = np.empty(az.size, np.float64)
    _check(lib().aqd_skip_params(az.size, az.ctypes.data, ak.ctypes.data, per_channel,
                                 c.ctypes.data, d.ctypes.data, side.ctypes.data, scale.ctypes.data))
    return c, d, side, scale


def requant_params(scale, alpha_out):
    s = _host(scale, np.float64)
    m = np.empty(s.size, np.int32)
    sh = np.empty(s.size, np.int32)
    _check(lib().aqd_requant_params(s.size, s.ctypes.data, float(alpha_out), m.ctypes.data,
                                    sh.ctypes.data))
    return m, sh
