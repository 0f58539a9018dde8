"""qconv_run_group_static (the group launch on the library's static scratch,
for callers that cannot allocate) against qconv_run_group_ws with a caller
workspace: the same bytes, bit for bit, on two calls in a row whose second
has a smaller input (the scratch keeps the first call's partial sums), and
both against the oracle."""
import numpy as np
import pytest

from gpu_helpers import assert_same, oracle_conv
from paper_2007_06919_amd import aqd, workloads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    return t


def _tensors(torch, case, h):
    dev = torch.device("cuda:0")
    ho, wo = aqd.qconv_out_shape(h, case.h, case.w)
    x = torch.from_numpy(aqd.pack_codes(case.x, case.bits_in)).to(dev)
    skip, hs, ws = None, 0, 0
    if case.skip_bits:
        hs, ws = case.skip.shape[1], case.skip.shape[2]
        skip = (torch.from_numpy(case.skip.astype(np.int32)).to(dev) if case.skip_bits == 32
                else torch.from_numpy(aqd.pack_codes(case.skip, case.skip_bits)).to(dev))
    if case.bits_out == 32:
        shape, dt = (case.n, ho, wo, case.cout), torch.int32
    else:
        shape, dt = (case.n, ho, wo, case.cout * case.bits_out // 8), torch.uint8
    y_static = torch.full(shape, 0x3C, dtype=dt, device=dev)
    y_ws = torch.full(shape, 0x3C, dtype=dt, device=dev)
    return x, skip, hs, ws, y_static, y_ws


# (n, h, w, cin, cout, k, stride, wenc, bits_out, skip_bits, up2): launches
# with few output tiles and a long K range, which split their reduction
CASES = [
    ((2, 27, 41, 512, 256, 3, 2, 1, 4, 4, False), (1, 13, 21, 512, 256, 3, 2, 1, 4, 4, False)),
    ((2, 11, 13, 256, 720, 3, 1, 1, 32, 0, False), (1, 7, 9, 256, 720, 3, 1, 1, 32, 0, False)),
    ((2, 9, 11, 1024, 256, 1, 1, 0, 4, 32, False), (1, 5, 6, 1024, 256, 1, 1, 0, 4, 32, False)),
]


@pytest.mark.parametrize("pair", CASES, ids=["p6_code_skip", "int32_out", "int32_skip"])
def test_static_scratch_matches_workspace(torch, pair):
    for call, (n, h, w, cin, cout, k, s, wenc, bo, sb, up2) in enumerate(pair):
        case = workloads.random_conv_case(seed=900 + 10 * call + cin % 7, n=n, h=h, w=w, cin=cin,
                                          cout=cout, k=k, stride=s, bits_in=4, bits_w=4, wenc=wenc,
                                          bits_out=bo, skip_bits=sb, skip_up2=up2)
        out_mode = aqd.OUT_INT32 if bo == 32 else aqd.OUT_CODES
        hd = aqd.qconv_create(cin, cout, k, s, k // 2, 4, 4, aqd.pack_codes(case.w_fields, 4),
                              case.levels, wenc=wenc, out_mode=out_mode,
                              bits_out=0 if bo == 32 else bo, skip_bits=sb, skip_up2=up2)
        try:
            x, skip, hs, ws, y_static, y_ws = _tensors(torch, case, hd)
            segs = [(hd, 0, n, h, w, x, skip, hs, ws, y_static)]
            nbytes = aqd.qconv_group_workspace(segs)
            assert 0 < nbytes <= 64 << 20
            wsbuf = torch.full((nbytes,), 0x77, dtype=torch.uint8, device=torch.device("cuda:0"))
            aqd.qconv_run_group_static(segs)
            aqd.qconv_run_group_ws([(hd, 0, n, h, w, x, skip, hs, ws, y_ws)], wsbuf, nbytes)
            torch.cuda.synchronize()
            got, ref_ws = y_static.cpu().numpy(), y_ws.cpu().numpy()
            assert_same(got, ref_ws, f"static vs workspace, call {call}")
            assert_same(got, oracle_conv(case), f"static vs oracle, call {call}")
        finally:
            aqd.qconv_destroy(hd)


def test_static_scratch_rejects_oversized_split(torch):
    """A split needing more than the static scratch is refused without a
    launch: a 1x1 conv with a very long K range (cin 16384) over 24576 pixels
    splits its reduction into parts of 24 MiB each."""
    cin, cout, n, h, w = 16384, 256, 1, 96, 256
    rng = np.random.Generator(np.random.PCG64(8))
    fields = rng.integers(0, 16, size=(cout, 1, 1, cin)).astype(np.uint8)
    lv = {"bias": np.zeros(cout, np.int32), "mult": np.full(cout, 1 << 30, np.int32),
          "shift": np.full(cout, 8, np.int32)}
    hd = aqd.qconv_create(cin, cout, 1, 1, 0, 4, 4, aqd.pack_codes(fields, 4), [lv], wenc=1)
    try:
        dev = torch.device("cuda:0")
        x = torch.zeros((n, h, w, cin // 2), dtype=torch.uint8, device=dev)
        y = torch.full((n, h, w, cout // 2), 0x5A, dtype=torch.uint8, device=dev)
        segs = [(hd, 0, n, h, w, x, None, 0, 0, y)]
        assert aqd.qconv_group_workspace(segs) > 64 << 20
        with pytest.raises(aqd.AqdError) as e:
            aqd.qconv_run_group_static(segs)
        assert e.value.status == aqd.AQD_ERR_UNSUPPORTED and "scratch" in str(e.value)
        torch.cuda.synchronize()
        assert bool((y == 0x5A).all())          # nothing was launched
    finally:
        aqd.qconv_destroy(hd)
