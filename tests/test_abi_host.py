"""Host side of the C ABI, no GPU needed: the library loads and exports every
symbol of include/aqd.h; descriptors are validated before any device call;
the host parameter helpers agree bit for bit with the oracle's own
derivation; the packers agree with the oracle's packers."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import ref
from paper_2007_06919_amd import aqd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    text = open(os.path.join(ROOT, "include", "aqd.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"^\s*#.*$", "", text, flags=re.M)          # preprocessor lines
    return sorted(set(re.findall(r"\b(\w+)\s*\([^;{]*\)\s*;", text)) - {"if", "for", "while"})


def test_library_exports_every_declared_function():
    L = aqd.lib()
    names = _header_functions()
    assert len(names) >= 16
    for name in names:
        assert hasattr(L, name), name
    assert sorted(names) == sorted(aqd.exported_symbols())


def _desc(**kw):
    d = dict(cin=64, cout=64, kh=3, kw=3, stride=1, pad=1, bits_in=4, bits_w=4, wenc=0,
             out_mode=0, bits_out=4, skip_bits=0, skip_up2=0, num_levels=1)
    d.update(kw)
    return aqd.QconvDesc(**d)


def _levels(cout, skip=False):
    lv = {"bias": np.zeros(cout, np.int32), "mult": np.full(cout, 1 << 30, np.int32),
          "shift": np.zeros(cout, np.int32)}
    if skip:
        lv.update(skip_c=np.full(cout, 2, np.int32), skip_d=np.ones(cout, np.int32),
                  skip_side=np.zeros(cout, np.int32))
    return lv


def _create(desc, levels, w=None):
    keep = []
    eps = (aqd.QconvEpilogue * len(levels))()
    for i, lv in enumerate(levels):
        for k, v in lv.items():
            a = np.ascontiguousarray(v, np.int32)
            keep.append(a)
            setattr(eps[i], k, a.ctypes.data)
    if w is None:
        w = np.zeros(desc.cout * desc.kh * desc.kw * desc.cin * desc.bits_w // 8, np.uint8)
    h = ctypes.c_void_p()
    st = aqd.lib().qconv_create(ctypes.byref(desc), w.ctypes.data, eps, ctypes.byref(h))
    return st, h.value


@pytest.mark.parametrize("bad", [
    dict(cin=0), dict(kh=9), dict(stride=0), dict(pad=3), dict(bits_in=5), dict(bits_w=1),
    dict(cin=3, bits_in=3), dict(bits_out=6),
    dict(wenc=5), dict(out_mode=2), dict(bits_out=16), dict(cin=3, bits_in=4),
    dict(cout=3, bits_out=2), dict(skip_bits=5), dict(skip_bits=4, out_mode=1, bits_out=0),
    dict(skip_up2=1), dict(num_levels=0), dict(num_levels=65),
    dict(step_in=-1.0), dict(step_w=float("nan")), dict(step_out=float("inf")),
])
def test_create_rejects_bad_descriptors(bad):
    d = _desc(**bad)
    st, h = _create(d, [_levels(max(d.cout, 1), skip=bool(d.skip_bits))] * max(d.num_levels, 1))
    assert st == aqd.AQD_ERR_INVALID and not h
    assert aqd.last_error()


def test_create_rejects_bad_epilogue_ranges():
    lv = _levels(64)
    lv["shift"][3] = 40
    assert _create(_desc(), [lv])[0] == aqd.AQD_ERR_INVALID
    lv = _levels(64, skip=True)
    lv["skip_d"][0] = 32
    assert _create(_desc(skip_bits=4), [lv])[0] == aqd.AQD_ERR_INVALID
    lv = _levels(64, skip=True)
    lv["skip_side"][0] = 2
    assert _create(_desc(skip_bits=4), [lv])[0] == aqd.AQD_ERR_INVALID


def test_create_rejects_accumulator_overflow():
    st, _ = _create(_desc(cin=8192, kh=7, kw=7, pad=3, bits_in=8, bits_w=8), [_levels(64)])
    assert st == aqd.AQD_ERR_UNSUPPORTED


def test_injected_allocation_failure(monkeypatch):
    monkeypatch.setenv("AQD_FAULT_INJECT", "alloc")
    st, h = _create(_desc(), [_levels(64)])
    assert st == aqd.AQD_ERR_NOMEM and not h
    assert "injected" in aqd.last_error()


def test_run_rejects_null_handle_without_device():
    st = aqd.lib().qconv_run(None, 0, 1, 8, 8, None, None, 0, 0, None, None)
    assert st == aqd.AQD_ERR_INVALID


def test_qadd_rejects_bad_descriptor():
    d = aqd.QaddDesc(1, 4, 4, 8, 3, 4, 4, 0, 4, 4)
    p = aqd.QaddParams()
    assert aqd.lib().qadd_run(ctypes.byref(d), None, None, None, ctypes.byref(p), None) == \
        aqd.AQD_ERR_INVALID


# ----------------------------------------------- packers and host helpers
@pytest.mark.parametrize("bits", [2, 3, 4, 8])
def test_packers_agree_with_oracle(bits):
    rng = np.random.Generator(np.random.PCG64(bits))
    codes = rng.integers(0, 1 << bits, size=(5, 7, 64)).astype(np.uint8)
    assert np.array_equal(aqd.pack_codes(codes, bits), ref.pack_codes(codes, bits))
    packed = ref.pack_codes(codes, bits)
    assert np.array_equal(aqd.unpack_codes(packed, bits, 64), codes)


def test_approx_ratio_agrees_with_oracle():
    rng = np.random.Generator(np.random.PCG64(1))
    rs = list(rng.uniform(1, 3, 2000)) + list(np.exp(rng.uniform(0, 20, 2000))) + \
        [1.0, 1.5, 3.0, np.pi, 4 / 3, 2.0 ** 29, 1.0000000001]
    for r in rs:
        assert aqd.approx_ratio(r) == ref.approx_ratio(r), r
    with pytest.raises(aqd.AqdError):
        aqd.approx_ratio(0.99)


def test_normalize_multiplier_agrees_with_oracle():
    rng = np.random.Generator(np.random.PCG64(2))
    rs = list(np.exp(rng.uniform(-21, 21, 4000))) + list(-np.exp(rng.uniform(-5, 5, 100)))
    rs += [1.0, 0.5, 2.0 ** -9, (2 ** 31 - 0.5) / 2 ** 31, 0.99999999999]
    for r in rs:
        assert aqd.normalize_multiplier(r) == ref.normalize_multiplier(r), r


def test_bn_fold_chain_agrees_with_oracle():
    rng = np.random.Generator(np.random.PCG64(3))
    for trial in range(20):
        c = 256
        acc = rng.integers(-50000, 50000, size=(300, c)) + rng.integers(-3000, 3000, size=c)
        s1, s2, cnt = ref.channel_sums(acc)
        alpha_conv = float(rng.uniform(0.001, 0.1))
        m1, v1 = ref.bn_stats_from_sums(s1, s2, cnt, alpha_conv)
        m2, v2 = aqd.bn_stats_from_sums(s1, s2, cnt, alpha_conv)
        assert np.array_equal(m1, m2) and np.array_equal(v1, v2)
        # gamma < 0 on some channels: alpha_z < 0 and the signed rule of Eq. 7
        g = rng.uniform(0.5, 1.5, c) * np.where(rng.random(c) < 0.3, -1.0, 1.0)
        b = rng.uniform(0, 1, c)
        b1, az1 = ref.fold_bn(g, b, m1, v1, 1e-5, alpha_conv)
        b2, az2 = aqd.fold_bn(g, b, m2, v2, 1e-5, alpha_conv)
        assert np.array_equal(b1, b2) and np.array_equal(az1, az2)
        ak = float(rng.uniform(0.05, 0.5)) if trial % 2 else rng.uniform(0.001, 0.2, c)
        r1 = ref.skip_params(az1, ak)
        r2 = aqd.skip_params(az2, ak)
        for x1, x2 in zip(r1, r2):
            assert np.array_equal(np.asarray(x1), np.asarray(x2))
        mm1, sh1 = ref.requant_params(r1[3], 0.2)
        mm2, sh2 = aqd.requant_params(r2[3], 0.2)
        assert np.array_equal(mm1, mm2) and np.array_equal(sh1, sh2)


def test_mfma_probe_rejects_bad_arguments():
    """Argument checks of the probe run before any launch (no GPU needed)."""
    L = aqd.lib()
    assert L.aqd_mfma_probe(0, 1, None, None) == aqd.AQD_ERR_INVALID
    assert L.aqd_mfma_probe(1, 0, None, None) == aqd.AQD_ERR_INVALID
    assert L.aqd_mfma_probe(1, 1, None, None) == aqd.AQD_ERR_INVALID
