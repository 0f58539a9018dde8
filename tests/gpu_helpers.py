"""Shared pieces of the GPU parity tests: run one random conv case through the
C ABI and through the CPU oracle, compare bit for bit."""
import numpy as np

from oracle import ref
from paper_2007_06919_amd import aqd, workloads


def gpu_conv(case, torch, stream=None, split=False):
    """Run a ConvCase through qconv_create/qconv_run (split: through
    qconv_run_group_ws with the queried workspace, filled with junk first);
    returns the output bytes of every level."""
    dev = torch.device("cuda:0")
    skip_bits = case.skip_bits
    out_mode = aqd.OUT_INT32 if case.bits_out == 32 else aqd.OUT_CODES
    h = aqd.qconv_create(case.cin, case.cout, case.k, case.stride, case.pad, case.bits_in,
                         case.bits_w, aqd.pack_codes(case.w_fields, case.bits_w), case.levels,
                         wenc=case.wenc, out_mode=out_mode,
                         bits_out=0 if case.bits_out == 32 else case.bits_out,
                         skip_bits=skip_bits, skip_up2=case.skip_up2)
    try:
        ho, wo = aqd.qconv_out_shape(h, case.h, case.w)
        x = torch.from_numpy(aqd.pack_codes(case.x, case.bits_in)).to(dev)
        skip, hs, ws = None, 0, 0
        if skip_bits:
            hs, ws = case.skip.shape[1], case.skip.shape[2]
            if skip_bits == 32:
                skip = torch.from_numpy(case.skip.astype(np.int32)).to(dev)
            else:
                skip = torch.from_numpy(aqd.pack_codes(case.skip, skip_bits)).to(dev)
        if case.bits_out == 32:
            y = torch.full((case.n, ho, wo, case.cout), -7, dtype=torch.int32, device=dev)
        else:
            y = torch.full((case.n, ho, wo, case.cout * aqd.stored_bits(case.bits_out) // 8), 0xA5,
                           dtype=torch.uint8, device=dev)
        outs = []
        for level in range(len(case.levels)):
            if split:
                segs = [(h, level, case.n, case.h, case.w, x, skip, hs, ws, y)]
                nbytes = aqd.qconv_group_workspace(segs)
                assert nbytes > 0, "this case is expected to split"
                wsbuf = torch.full((nbytes,), 0x77, dtype=torch.uint8, device=dev)
                aqd.qconv_run_group_ws(segs, wsbuf, nbytes, stream)
            else:
                aqd.qconv_run(h, level, case.n, case.h, case.w, x, skip, hs, ws, y, stream)
            torch.cuda.synchronize()
            outs.append(y.cpu().numpy().copy())
        return outs
    finally:
        aqd.qconv_destroy(h)


def oracle_conv(case, level=0):
    lv = case.levels[level]
    out32 = case.bits_out == 32
    y = ref.qconv(case.x, case.w_fields, case.bits_w, case.stride, case.pad, lv["bias"],
                  wenc=case.wenc, out_int32=out32, mult=lv.get("mult"), shift=lv.get("shift"),
                  bits_out=0 if out32 else case.bits_out, skip=case.skip, skip_up2=case.skip_up2,
                  skip_c=lv.get("skip_c"), skip_d=lv.get("skip_d"), skip_side=lv.get("skip_side"))
    if out32:
        return y.astype(np.int32)
    return ref.pack_codes(y, case.bits_out)


def assert_same(got, want, what):
    assert got.shape == want.shape, (what, got.shape, want.shape)
    if not np.array_equal(got, want):
        bad = np.argwhere(got != want)
        raise AssertionError(f"{what}: {len(bad)} of {got.size} elements differ; first at "
                             f"{tuple(bad[0])}: got {got[tuple(bad[0])]}, want {want[tuple(bad[0])]}")


def check_case(torch, **kw):
    case = workloads.random_conv_case(**kw)
    outs = gpu_conv(case, torch)
    for level, got in enumerate(outs):
        assert_same(got, oracle_conv(case, level), f"{kw} level {level}")
    return case
