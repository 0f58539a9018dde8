"""GPU parity of single convolutions, grouped launches, the standalone add and
the channel sums: the C ABI on the MI355X against the CPU oracle, bit for bit.

Shapes span several 128 x 256 workgroup tiles with ragged pixel and channel
tails, every bitwidth and output mode, both weight grids, skip operands of
every width (with and without the nearest 2x upsample), strides 1 and 2, and
both kernels (the MFMA kernel and the direct kernel for shapes it does not
take).
"""
import numpy as np
import pytest

from gpu_helpers import assert_same, check_case, gpu_conv, oracle_conv
from oracle import ref
from paper_2007_06919_amd import aqd, workloads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    return t


MFMA_CASES = [
    # (n, h, w, cin, cout, k, stride, bits_in, bits_w, wenc, bits_out, skip_bits, up2)
    (1, 32, 32, 64, 64, 3, 1, 4, 4, 0, 4, 0, False),
    (2, 17, 23, 128, 144, 3, 1, 4, 4, 0, 4, 0, False),      # ragged pixels and channels
    (1, 19, 30, 64, 128, 3, 2, 2, 2, 0, 2, 0, False),       # stride 2, 2-bit
    (2, 13, 11, 192, 256, 1, 1, 4, 4, 1, 4, 0, False),      # 1x1, odd grid
    (1, 25, 21, 64, 256, 1, 2, 2, 2, 1, 2, 0, False),       # 1x1 stride 2
    (1, 21, 19, 128, 96, 3, 1, 4, 8, 0, 8, 0, False),       # 8-bit weights and output codes
    (2, 15, 17, 64, 64, 3, 1, 2, 4, 1, 4, 4, False),        # mixed widths, code skip
    (1, 20, 22, 64, 128, 3, 1, 4, 4, 0, 2, 2, False),       # 2-bit skip, 2-bit out
    (1, 16, 18, 128, 64, 1, 1, 4, 4, 0, 4, 4, True),        # FPN top-down: upsampled skip
    (1, 17, 19, 64, 64, 1, 1, 2, 2, 0, 2, 2, True),         # odd output size, upsampled skip
    (2, 9, 14, 64, 256, 1, 1, 4, 4, 1, 4, 32, False),       # int32 skip (normalised branch)
    (1, 12, 12, 64, 64, 3, 1, 4, 4, 0, 8, 8, False),        # 8-bit skip
    (1, 23, 29, 256, 720, 3, 1, 4, 4, 1, 32, 0, False),     # class prediction: int32 out
    (2, 11, 13, 256, 36, 3, 1, 4, 4, 1, 32, 0, False),      # box prediction: 36 channels
    (1, 7, 11, 64, 64, 3, 1, 4, 4, 0, 4, 0, False),         # one partial tile
    (3, 1, 1, 64, 32, 3, 1, 4, 4, 0, 4, 0, False),          # 1x1 image, all taps but one padded
    (1, 30, 31, 128, 256, 1, 1, 4, 4, 0, 4, 0, False),      # 2 K steps
    (1, 29, 33, 256, 128, 1, 1, 2, 2, 1, 2, 0, False),      # 4 K steps, 2-bit
    (1, 31, 17, 320, 64, 1, 1, 4, 4, 0, 4, 4, False),       # 5 K steps
    (2, 40, 37, 64, 512, 3, 2, 4, 4, 1, 4, 0, False),       # several 256x256 tiles, stride 2
]


def test_conv_mfma_general_requant_path(torch):
    """Levels with shift < 2 take the 64-bit requantisation path."""
    for seed, skip in ((11, 0), (12, 4)):
        case = workloads.random_conv_case(seed=seed, n=1, h=21, w=23, cin=64, cout=128, k=1,
                                          bits_in=2, bits_w=2, bits_out=4, skip_bits=skip)
        rng = np.random.Generator(np.random.PCG64(seed))
        for lv in case.levels:
            lv["shift"] = rng.integers(-2, 2, size=128).astype(np.int32)
            lv["mult"] = rng.integers(1 << 26, 1 << 28, size=128).astype(np.int32)
        for level, got in enumerate(gpu_conv(case, torch)):
            assert_same(got, oracle_conv(case, level), f"general path, skip {skip}")


@pytest.mark.parametrize("case", MFMA_CASES, ids=lambda c: "x".join(map(str, c)))
def test_conv_mfma_parity(torch, case):
    n, h, w, cin, cout, k, s, bi, bw, wenc, bo, sb, up2 = case
    check_case(torch, seed=hash(case) % 1000, n=n, h=h, w=w, cin=cin, cout=cout, k=k, stride=s,
               bits_in=bi, bits_w=bw, wenc=wenc, bits_out=bo, skip_bits=sb, skip_up2=up2)


SPLIT_CASES = [
    # few output tiles and a long K range: the K reduction is split over workgroups
    (1, 13, 21, 512, 256, 3, 2, 4, 4, 1, 4, 0, False),      # P6-like: 3x3 stride 2, 72 K steps
    (2, 9, 11, 1024, 256, 1, 1, 4, 4, 1, 4, 4, True),       # lateral 1x1 + upsampled code skip
    (1, 7, 9, 1024, 256, 1, 1, 4, 4, 0, 4, 32, False),      # int32 skip
    (1, 10, 12, 256, 720, 3, 1, 4, 4, 1, 32, 0, False),     # int32 out, 720 channels
    (1, 9, 9, 256, 128, 3, 1, 2, 2, 0, 2, 2, False),        # 2-bit, code skip
    (1, 6, 7, 448, 64, 3, 1, 4, 4, 0, 4, 0, False),         # 63 K steps: a shorter last part
]


@pytest.mark.parametrize("case", SPLIT_CASES, ids=lambda c: "x".join(map(str, c)))
def test_conv_split_k_parity(torch, case):
    """qconv_run_group_ws with a workspace: the split reduction and the
    combining epilogue give the oracle's outputs bit for bit, and the same
    bytes as the unsplit launch."""
    n, h, w, cin, cout, k, s, bi, bw, wenc, bo, sb, up2 = case
    c = workloads.random_conv_case(seed=hash(case) % 1000 + 3, n=n, h=h, w=w, cin=cin, cout=cout,
                                   k=k, stride=s, bits_in=bi, bits_w=bw, wenc=wenc, bits_out=bo,
                                   skip_bits=sb, skip_up2=up2)
    got = gpu_conv(c, torch, split=True)
    plain = gpu_conv(c, torch)
    for level, g in enumerate(got):
        assert_same(g, oracle_conv(c, level), f"split {case} level {level}")
        assert_same(g, plain[level], f"split vs unsplit {case}")


def test_split_k_not_used_for_full_launches(torch):
    """A launch that already fills the GPU asks for no workspace."""
    case = workloads.random_conv_case(seed=4, n=4, h=64, w=96, cin=256, cout=256, k=3,
                                      bits_in=4, bits_w=4, bits_out=4)
    h = aqd.qconv_create(256, 256, 3, 1, 1, 4, 4, aqd.pack_codes(case.w_fields, 4), case.levels)
    try:
        dev = torch.device("cuda:0")
        x = torch.zeros((4, 64, 96, 128), dtype=torch.uint8, device=dev)
        y = torch.zeros((4, 64, 96, 128), dtype=torch.uint8, device=dev)
        assert aqd.qconv_group_workspace([(h, 0, 4, 64, 96, x, None, 0, 0, y)]) == 0
    finally:
        aqd.qconv_destroy(h)


# 1x1 convolutions with cin <= 128, code outputs and cout a multiple of 256
# run on persistent 256 x 64 tiles (weights kept in LDS, the next tile's
# copies overlapping the current epilogue): ragged tails, several channel
# tiles, code skips with and without the upsample, stride 2, several tiles
# per workgroup.
STREAM_CASES = [
    # (n, h, w, cin, cout, k, stride, bits_in, bits_w, wenc, bits_out, skip_bits, up2)
    (2, 41, 52, 64, 256, 1, 1, 4, 4, 1, 4, 4, False),       # 1 K step, code skip
    (1, 33, 37, 128, 512, 1, 1, 4, 4, 0, 4, 4, False),      # 2 K steps, 2 channel tiles
    (2, 16, 18, 64, 256, 1, 1, 4, 4, 0, 4, 4, True),        # upsampled code skip
    (1, 25, 21, 128, 256, 1, 2, 4, 4, 1, 4, 0, False),      # stride 2, no skip
    (8, 120, 161, 64, 256, 1, 1, 4, 4, 1, 4, 4, False),     # ~4.7 tiles per workgroup
    (3, 70, 90, 128, 768, 1, 1, 4, 4, 0, 4, 4, False),      # 3 channel tiles, 2 tiles per workgroup
    # handles laid out for 128- and 64-channel tiles, up to 4 K steps, no skip
    (2, 41, 52, 256, 128, 1, 1, 4, 4, 0, 4, 0, False),      # 128 x 64 tiles, 4 K steps
    (4, 60, 90, 192, 128, 1, 1, 4, 4, 1, 4, 0, False),      # 3 K steps, several tiles per workgroup
    (1, 45, 41, 128, 128, 1, 2, 4, 4, 0, 4, 0, False),      # stride 2
    (2, 41, 52, 256, 64, 1, 1, 4, 4, 1, 4, 0, False),       # 64 x 128 tiles, 4 K steps
    (1, 33, 37, 64, 64, 1, 1, 4, 4, 0, 4, 0, False),        # 1 K step
    (8, 200, 168, 256, 64, 1, 1, 4, 4, 1, 4, 0, False),     # ~2.7 tiles per workgroup
    # handles laid out for 256-channel tiles with 3-4 K steps: 128 x 64 tiles
    # reading each 256-row weight tile as two halves, with or without a skip
    (2, 41, 52, 256, 512, 1, 1, 4, 4, 1, 4, 4, False),      # 4 K steps, code skip
    (1, 33, 37, 192, 256, 1, 1, 4, 4, 0, 4, 0, False),      # 3 K steps, no skip
    (2, 16, 18, 256, 256, 1, 1, 4, 4, 0, 4, 4, True),       # upsampled code skip
    (1, 25, 21, 256, 256, 1, 2, 4, 4, 1, 4, 4, False),      # stride 2
    (8, 50, 84, 256, 1024, 1, 1, 4, 4, 1, 4, 4, False),     # ResNet-50 res4 conv3 at batch 8
    # (the cin-256 cases above with cout a multiple of 256 run on the
    # weight-stationary tiles: 1x1, cin 256, one segment, persistent 256 x 64
    # tiles with the weights in registers)
    (3, 77, 91, 256, 768, 1, 1, 4, 4, 1, 4, 4, False),      # weight-stationary: three channel tiles, skip
    (1, 31, 29, 256, 512, 1, 2, 4, 4, 0, 4, 0, False),      # weight-stationary: stride 2, a ragged last tile
    (1, 5, 7, 256, 256, 1, 1, 4, 4, 1, 4, 4, False),        # weight-stationary: fewer tiles than slots
    (8, 100, 167, 256, 256, 1, 1, 4, 4, 0, 4, 4, True),     # weight-stationary: ~4 tiles per workgroup, upsampled skip
]


@pytest.mark.parametrize("case", STREAM_CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("variant", ["random_sides", "side0", "small_shifts"])
def test_conv_stream_parity(torch, case, variant):
    """Per-channel skip sides (64-bit-free alignment), all sides 0 (the skip
    table), and shifts < 2 (64-bit requantisation)."""
    n, h, w, cin, cout, k, s, bi, bw, wenc, bo, sb, up2 = case
    c = workloads.random_conv_case(seed=hash(case) % 1000 + 21, n=n, h=h, w=w, cin=cin, cout=cout,
                                   k=k, stride=s, bits_in=bi, bits_w=bw, wenc=wenc, bits_out=bo,
                                   skip_bits=sb, skip_up2=up2)
    rng = np.random.Generator(np.random.PCG64(17))
    for lv in c.levels:
        if variant == "side0" and sb:
            lv["skip_side"][:] = 0
        if variant == "small_shifts":
            lv["shift"] = rng.integers(-2, 2, size=cout).astype(np.int32)
            lv["mult"] = rng.integers(1 << 24, 1 << 27, size=cout).astype(np.int32)
    for level, got in enumerate(gpu_conv(c, torch)):
        assert_same(got, oracle_conv(c, level), f"stream {variant} {case} level {level}")


# cin a multiple of 256, code outputs and at least 200 tiles of 256 x 128:
# the register-fed kernel (weights read into registers, codes staged in LDS
# four K steps at a time), on 256 x 64 tiles for K ranges of at most 8
# steps, on 256 x 144 tiles (one round, one workgroup per CU) where 256 x 128
# tiles would be a little above one round, on 256 x 128 tiles otherwise. The head-tower shape, two and four stages per tap,
# stride 2, a partial channel tile, code skips with and without the
# upsample, 3-bit codes, ragged pixel tails.
WV_CASES = [
    # (n, h, w, cin, cout, k, stride, bits_in, bits_w, wenc, bits_out, skip_bits, up2)
    (2, 100, 167, 256, 256, 3, 1, 4, 4, 1, 4, 0, False),    # head-tower shape: 261 tiles (232 of 144 px)
    (1, 120, 230, 512, 256, 3, 1, 4, 4, 0, 4, 0, False),    # two stages per tap: 216 tiles
    (1, 150, 181, 1024, 256, 1, 1, 4, 4, 1, 4, 4, True),    # 1x1, four stages per tap, upsampled skip
    (2, 203, 131, 256, 288, 3, 2, 4, 4, 0, 4, 4, False),    # stride 2, a partial channel tile, skip
    (8, 50, 84, 256, 256, 3, 1, 3, 3, 1, 3, 3, False),      # 3-bit codes and skip: 263 tiles (234 of 144)
    (2, 150, 181, 1024, 256, 1, 1, 4, 4, 1, 4, 4, True),    # 425 tiles; upsampled skip
    (4, 100, 167, 256, 256, 3, 1, 4, 4, 1, 4, 0, False),    # head-tower shape: 522 tiles
    (5, 203, 131, 256, 288, 3, 2, 4, 4, 0, 4, 4, False),    # stride 2, a partial channel tile, skip
    (5, 75, 90, 256, 256, 3, 1, 4, 4, 0, 4, 4, False),      # 264 tiles (235 of 144 px), skip
    (4, 130, 130, 256, 288, 3, 2, 4, 4, 0, 4, 4, False),    # 266 tiles (236 of 144): stride 2, partial channel tile
    # more than one round of 256 x 128 tiles without a skip
    (3, 100, 167, 256, 288, 3, 1, 4, 4, 0, 4, 0, False),    # 784 tiles, a partial channel tile
    (16, 50, 84, 256, 256, 3, 1, 3, 3, 1, 3, 0, False),     # 3-bit codes: 528 tiles
    (1, 150, 181, 1024, 512, 1, 1, 4, 4, 1, 4, 0, False),   # 1x1, four stages per tile: 426 tiles
    # 256 x 64 tiles (8 K steps)
    (2, 100, 167, 512, 256, 1, 1, 4, 4, 1, 4, 4, True),     # 1x1 with an upsampled skip (FPN lateral shape)
    (1, 60, 100, 512, 2048, 1, 1, 4, 4, 0, 4, 4, False),    # 1x1 512 -> 2048 with a skip, eight channel tiles
    (3, 90, 100, 512, 288, 1, 1, 4, 4, 0, 4, 0, False),     # a partial channel tile
    # 8 K steps, no skip, more than one round
    (4, 100, 167, 512, 256, 1, 1, 4, 4, 0, 4, 0, False),    # res4.0 conv1 shape: 1044 tiles
    (3, 90, 110, 512, 288, 1, 1, 3, 3, 1, 3, 0, False),     # 3-bit codes, a partial channel tile: 930 tiles
    # fewer 256 x 128 tiles than CUs: 256 x 64 tiles, one round (long K ranges)
    (1, 50, 84, 512, 512, 3, 1, 4, 4, 0, 4, 4, False),      # res5 3x3 shape: 132 tiles, 72 K steps, skip
    (1, 101, 167, 512, 288, 3, 2, 4, 4, 1, 4, 0, False),    # stride 2, a partial channel tile: 134 tiles
    (8, 25, 42, 2048, 512, 1, 1, 4, 4, 0, 4, 0, False),     # 1x1 2048 -> 512: 132 tiles, 32 K steps
    (2, 50, 84, 1024, 256, 1, 1, 4, 4, 1, 4, 4, True),      # 1x1 with an upsampled skip: 132 tiles, 16 K steps
]


def _wv_tiles(case):
    n, h, w, cin, cout, k, s = case[:7]
    ho, wo = (h + 2 * (k // 2) - k) // s + 1, (w + 2 * (k // 2) - k) // s + 1
    return -(-n * ho * wo // 128) * -(-cout // 256)


@pytest.mark.parametrize("case", WV_CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("variant", ["random_sides", "side0", "small_shifts"])
def test_conv_register_fed_parity(torch, case, variant):
    """Per-channel skip sides, all sides 0 (the skip table), and shifts < 2
    (64-bit requantisation)."""
    assert _wv_tiles(case) >= 64 and case[3] % 256 == 0
    n, h, w, cin, cout, k, s, bi, bw, wenc, bo, sb, up2 = case
    c = workloads.random_conv_case(seed=hash(case) % 1000 + 81, n=n, h=h, w=w, cin=cin, cout=cout,
                                   k=k, stride=s, bits_in=bi, bits_w=bw, wenc=wenc, bits_out=bo,
                                   skip_bits=sb, skip_up2=up2)
    rng = np.random.Generator(np.random.PCG64(31))
    for lv in c.levels:
        if variant == "side0" and sb:
            lv["skip_side"][:] = 0
        if variant == "small_shifts":
            lv["shift"] = rng.integers(-2, 2, size=cout).astype(np.int32)
            lv["mult"] = rng.integers(1 << 24, 1 << 27, size=cout).astype(np.int32)
    for level, got in enumerate(gpu_conv(c, torch)):
        assert_same(got, oracle_conv(c, level), f"register-fed {variant} {case} level {level}")


WV_INT32_CASES = [
    # int32 outputs v = acc + bias through the register-fed kernel
    (1, 100, 167, 256, 720, 3, 1, 4, 4, 1, 32, 0, False),   # class predictor: 720 = 2 x 256 + 208
    (5, 60, 100, 512, 256, 1, 1, 4, 4, 0, 32, 0, False),    # 1x1, two stages per tap
    (8, 201, 163, 256, 256, 3, 2, 4, 4, 1, 32, 0, False),   # stride 2, ragged pixel tail
]


@pytest.mark.parametrize("case", WV_INT32_CASES, ids=lambda c: "x".join(map(str, c)))
def test_conv_register_fed_int32_parity(torch, case):
    assert _wv_tiles(case) >= 200 and case[3] % 256 == 0
    n, h, w, cin, cout, k, s, bi, bw, wenc, bo, sb, up2 = case
    c = workloads.random_conv_case(seed=hash(case) % 1000 + 85, n=n, h=h, w=w, cin=cin, cout=cout,
                                   k=k, stride=s, bits_in=bi, bits_w=bw, wenc=wenc, bits_out=bo)
    for level, got in enumerate(gpu_conv(c, torch)):
        assert_same(got, oracle_conv(c, level), f"register-fed int32 {case} level {level}")


def test_register_fed_grouped_levels_and_guard_bytes(torch):
    """The head towers' launch shape on the register-fed kernel: two handles
    (class and box towers), five pyramid levels each with its own table, one
    launch; every output sits between guard bytes that must stay untouched."""
    dev = torch.device("cuda:0")
    n, sizes = 3, [(50, 75), (25, 38), (13, 19), (7, 10), (4, 5)]
    cases = [workloads.random_conv_case(seed=90 + t, n=1, h=8, w=8, cin=256, cout=256, k=3,
                                        bits_in=4, bits_w=4, wenc=1, bits_out=4, num_levels=5)
             for t in range(2)]
    handles = [aqd.qconv_create(256, 256, 3, 1, 1, 4, 4, aqd.pack_codes(c.w_fields, 4), c.levels,
                                wenc=1, bits_out=4) for c in cases]
    rng = np.random.Generator(np.random.PCG64(19))
    try:
        segs, expect, outs = [], [], []
        for t, c in enumerate(cases):
            for lv, (h, w) in enumerate(sizes):
                x = rng.integers(0, 16, size=(n, h, w, 256))
                xd = torch.from_numpy(aqd.pack_codes(x, 4)).to(dev)
                nbytes = n * h * w * 128
                buf = torch.full((nbytes + 4096,), 0x5A, dtype=torch.uint8, device=dev)
                yd = buf[2048:2048 + nbytes]
                segs.append((handles[t], lv, n, h, w, xd, None, 0, 0, yd))
                outs.append((buf, nbytes))
                L = c.levels[lv]
                want = ref.qconv(x, c.w_fields, 4, 1, 1, L["bias"], wenc=1, mult=L["mult"],
                                 shift=L["shift"], bits_out=4)
                expect.append(ref.pack_codes(want, 4).reshape(-1))
        tiles = sum(-(-s[2] * s[3] * s[4] // 128) for s in segs)
        assert tiles >= 200
        aqd.qconv_run_group(segs)
        torch.cuda.synchronize()
        for i, ((buf, nbytes), want) in enumerate(zip(outs, expect)):
            host = buf.cpu().numpy()
            assert np.all(host[:2048] == 0x5A) and np.all(host[2048 + nbytes:] == 0x5A), i
            assert_same(host[2048:2048 + nbytes], want, f"segment {i}")
    finally:
        for h in handles:
            aqd.qconv_destroy(h)


# Launches of more than one round of 128 x 256 or 64 x 512 tiles without a
# skip run on tiles half as wide, three workgroups to a CU: 1x1 and 3x3,
# stride 2, int32 and code outputs, ragged pixel tails.
OCC3_CASES = [
    # (n, h, w, cin, cout, k, stride, bits_out)
    (1, 363, 363, 64, 64, 1, 1, 32),        # 64 x 256 tiles, 258 handle tiles
    (1, 257, 257, 64, 128, 1, 1, 32),       # 128 x 128 tiles, 259 handle tiles
    (4, 182, 182, 64, 64, 3, 1, 4),         # 3x3 codes, 64-channel handle
    (2, 182, 182, 64, 128, 3, 1, 4),        # 3x3 codes, 128-channel handle
    (2, 363, 363, 64, 128, 3, 2, 4),        # stride 2
    (4, 182, 182, 256, 36, 3, 1, 32),       # a box predictor: 36 of 64 channels
    (1, 300, 500, 320, 64, 1, 1, 4),        # 1x1 with 5 K steps (not streamed)
]


@pytest.mark.parametrize("case", OCC3_CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("variant", ["plain", "small_shifts"])
def test_conv_three_per_cu_parity(torch, case, variant):
    """Shifts < 2 take the 64-bit requantisation."""
    n, h, w, cin, cout, k, s, bo = case
    c = workloads.random_conv_case(seed=hash(case) % 1000 + 41, n=n, h=h, w=w, cin=cin, cout=cout,
                                   k=k, stride=s, bits_in=4, bits_w=4, wenc=1, bits_out=bo)
    if variant == "small_shifts" and bo != 32:
        rng = np.random.Generator(np.random.PCG64(23))
        for lv in c.levels:
            lv["shift"] = rng.integers(-2, 2, size=cout).astype(np.int32)
            lv["mult"] = rng.integers(1 << 24, 1 << 27, size=cout).astype(np.int32)
    for level, got in enumerate(gpu_conv(c, torch)):
        assert_same(got, oracle_conv(c, level), f"three per CU {variant} {case} level {level}")


# 3-bit codes (stored in 4-bit containers, outputs clamped to 7) on every
# launch path: 256 x 128 tiles with a code skip, 128- and 64-channel handles,
# the streaming 1x1 kernel, the three-per-CU tiles, int32 predictions,
# split K, the direct kernel, and 3-bit inputs with 4-bit outputs.
THREE_BIT_CASES = [
    # (n, h, w, cin, cout, k, stride, bits_in, bits_w, wenc, bits_out, skip_bits, up2)
    (1, 19, 23, 128, 256, 3, 1, 3, 3, 1, 3, 3, False),      # 256 x 128, code skip
    (2, 17, 13, 64, 512, 1, 2, 3, 3, 1, 3, 3, True),        # upsampled skip, stride 2
    (1, 21, 18, 64, 128, 3, 1, 3, 3, 1, 3, 0, False),       # 128-channel handle
    (1, 15, 22, 128, 64, 3, 2, 3, 3, 0, 3, 0, False),       # 64-channel handle
    (2, 41, 52, 64, 256, 1, 1, 3, 3, 1, 3, 3, False),       # streaming 1x1 with skip
    (2, 41, 52, 256, 128, 1, 1, 3, 3, 1, 3, 0, False),      # streaming 128 x 64
    (1, 363, 363, 64, 64, 1, 1, 3, 3, 1, 3, 0, False),      # three per CU, 64 x 256
    (2, 41, 52, 256, 512, 1, 1, 3, 3, 1, 3, 3, False),      # streaming halves of 256-row tiles
    (1, 19, 23, 256, 720, 3, 1, 3, 3, 1, 32, 0, False),     # int32 class predictor
    (1, 16, 18, 64, 256, 3, 1, 3, 3, 0, 3, 32, False),      # int32 skip
    (1, 21, 19, 48, 96, 3, 1, 3, 3, 1, 3, 3, False),        # direct kernel (cin 48)
    (1, 19, 23, 128, 256, 3, 1, 3, 3, 1, 4, 4, False),      # 3-bit in, 4-bit out
]


@pytest.mark.parametrize("case", THREE_BIT_CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("variant", ["random_sides", "side0", "small_shifts"])
def test_three_bit_parity(torch, case, variant):
    n, h, w, cin, cout, k, s, bi, bw, wenc, bo, sb, up2 = case
    c = workloads.random_conv_case(seed=hash(case) % 1000 + 61, n=n, h=h, w=w, cin=cin, cout=cout,
                                   k=k, stride=s, bits_in=bi, bits_w=bw, wenc=wenc, bits_out=bo,
                                   skip_bits=sb, skip_up2=up2)
    rng = np.random.Generator(np.random.PCG64(29))
    for lv in c.levels:
        if variant == "side0" and sb and sb != 32:
            lv["skip_side"][:] = 0
        if variant == "small_shifts" and bo != 32:
            lv["shift"] = rng.integers(-2, 2, size=cout).astype(np.int32)
            lv["mult"] = rng.integers(1 << 24, 1 << 27, size=cout).astype(np.int32)
    for level, got in enumerate(gpu_conv(c, torch)):
        want = oracle_conv(c, level)
        assert_same(got, want, f"3-bit {variant} {case} level {level}")
        if bo == 3 and variant != "small_shifts":  # the clamp at 7 is reached
            codes = ref.unpack_codes(got, 4, cout)
            assert codes.max() == 7


def test_three_bit_split_k(torch):
    """Split K with 3-bit codes: the combining epilogue clamps at 7."""
    c = workloads.random_conv_case(seed=71, n=1, h=6, w=7, cin=448, cout=64, k=3, bits_in=3,
                                   bits_w=3, wenc=1, bits_out=3, skip_bits=3)
    got = gpu_conv(c, torch, split=True)
    assert_same(got[0], oracle_conv(c, 0), "3-bit split K")


def test_stream_grouped_segments(torch):
    """One launch over segments of two handles (weights and tables reloaded at
    each segment change) and two levels, with code skips."""
    dev = torch.device("cuda:0")
    sizes = [(40, 57), (20, 29), (10, 15)]
    cases = [workloads.random_conv_case(seed=60 + t, n=2, h=40, w=57, cin=64, cout=256, k=1,
                                        bits_in=4, bits_w=4, wenc=1, bits_out=4, skip_bits=4,
                                        num_levels=2)
             for t in range(2)]
    handles = [aqd.qconv_create(64, 256, 1, 1, 0, 4, 4, aqd.pack_codes(c.w_fields, 4), c.levels,
                                wenc=1, bits_out=4, skip_bits=4) for c in cases]
    rng = np.random.Generator(np.random.PCG64(19))
    try:
        segs, expect, outs = [], [], []
        for t, c in enumerate(cases):
            for i, (h, w) in enumerate(sizes):
                lv = i % 2
                x = rng.integers(0, 16, size=(2, h, w, 64))
                sk = rng.integers(0, 16, size=(2, h, w, 256))
                xd = torch.from_numpy(aqd.pack_codes(x, 4)).to(dev)
                sd = torch.from_numpy(aqd.pack_codes(sk, 4)).to(dev)
                yd = torch.zeros((2, h, w, 128), dtype=torch.uint8, device=dev)
                segs.append((handles[t], lv, 2, h, w, xd, sd, h, w, yd))
                outs.append(yd)
                L = c.levels[lv]
                want = ref.qconv(x, c.w_fields, 4, 1, 0, L["bias"], wenc=1, mult=L["mult"],
                                 shift=L["shift"], bits_out=4, skip=sk, skip_c=L["skip_c"],
                                 skip_d=L["skip_d"], skip_side=L["skip_side"])
                expect.append(ref.pack_codes(want, 4))
        aqd.qconv_run_group(segs)
        torch.cuda.synchronize()
        for i, (yd, want) in enumerate(zip(outs, expect)):
            assert_same(yd.cpu().numpy(), want, f"segment {i}")
    finally:
        for h in handles:
            aqd.qconv_destroy(h)


@pytest.mark.parametrize("bits,k,stride,pad,shape", [
    (4, 3, 2, 1, (2, 37, 41, 64)),      # ResNet stem pooling on 4-bit codes
    (8, 3, 2, 1, (1, 25, 30, 16)),
    (2, 2, 2, 0, (3, 17, 19, 32)),
    (4, 5, 1, 2, (1, 9, 8, 6)),         # 6 channels: three bytes per pixel
    (8, 7, 3, 3, (1, 20, 22, 3)),       # 3-channel 8-bit input
    (3, 3, 2, 1, (2, 21, 17, 32)),      # 3-bit codes in 4-bit containers
])
def test_maxpool_parity(torch, bits, k, stride, pad, shape):
    dev = torch.device("cuda:0")
    rng = np.random.Generator(np.random.PCG64(bits * 1000 + k * 10 + stride))
    n, h, w, c = shape
    x = rng.integers(0, 1 << bits, size=shape)
    want = ref.pack_codes(ref.maxpool(x, k, stride, pad), bits)
    xd = torch.from_numpy(aqd.pack_codes(x, bits)).to(dev)
    yd = torch.full(want.shape, 0xA5, dtype=torch.uint8, device=dev)
    aqd.maxpool_run(n, h, w, c, bits, k, stride, pad, xd, yd)
    torch.cuda.synchronize()
    assert_same(yd.cpu().numpy(), want, f"maxpool {bits} {k} {stride} {pad} {shape}")


def test_stem_8bit_conv_then_pool(torch):
    """The 8-bit input layer of a fully quantized ResNet: 7x7 stride 2 conv of a
    3-channel 8-bit image (direct kernel) to 4-bit codes, then 3x3 stride 2
    max-pooling, against the oracle's conv and pooling."""
    dev = torch.device("cuda:0")
    case = workloads.random_conv_case(seed=31, n=1, h=67, w=81, cin=3, cout=64, k=7, stride=2,
                                      bits_in=8, bits_w=8, bits_out=4)
    conv = gpu_conv(case, torch)[0]
    assert_same(conv, oracle_conv(case, 0), "stem conv")
    ho, wo = case.out_hw
    want = ref.pack_codes(ref.maxpool(ref.unpack_codes(oracle_conv(case, 0), 4, 64).reshape(
        1, ho, wo, 64), 3, 2, 1), 4)
    yd = torch.full(want.shape, 0xA5, dtype=torch.uint8, device=dev)
    aqd.maxpool_run(1, ho, wo, 64, 4, 3, 2, 1, torch.from_numpy(conv).to(dev), yd)
    torch.cuda.synchronize()
    assert_same(yd.cpu().numpy(), want, "stem pooling")


DIRECT_CASES = [
    (1, 9, 10, 32, 16, 3, 1, 4, 4, 0, 4, 0, False),         # cin not a multiple of 64
    (2, 8, 7, 16, 12, 3, 2, 8, 4, 0, 8, 0, False),          # 8-bit activations
    (1, 6, 9, 24, 20, 1, 1, 2, 2, 1, 2, 2, False),          # 20 channels (not 16k)
    (1, 7, 8, 64, 24, 3, 1, 4, 8, 1, 4, 4, True),           # 8-bit odd-grid weights
    (1, 5, 6, 8, 10, 3, 1, 8, 8, 0, 32, 0, False),          # int32 out, 10 channels
    (1, 11, 9, 40, 8, 5, 2, 4, 2, 0, 4, 32, False),         # 5x5, int32 skip
]


@pytest.mark.parametrize("case", DIRECT_CASES, ids=lambda c: "x".join(map(str, c)))
def test_conv_direct_parity(torch, case):
    n, h, w, cin, cout, k, s, bi, bw, wenc, bo, sb, up2 = case
    check_case(torch, seed=hash(case) % 1000 + 7, n=n, h=h, w=w, cin=cin, cout=cout, k=k,
               stride=s, bits_in=bi, bits_w=bw, wenc=wenc, bits_out=bo, skip_bits=sb,
               skip_up2=up2)


def test_multi_level_tables(torch):
    """One handle, three epilogue tables (multi-level BN): each level's output
    uses its own table."""
    check_case(torch, seed=5, n=1, h=20, w=26, cin=128, cout=128, k=3, bits_in=4, bits_w=4,
               wenc=1, bits_out=4, num_levels=3)


def test_grouped_launch_matches_separate_runs(torch):
    """Two handles (class and box towers), five pyramid levels each, one launch."""
    dev = torch.device("cuda:0")
    sizes = [(20, 33), (10, 17), (5, 9), (3, 5), (2, 3)]
    cases = [workloads.random_conv_case(seed=40 + t, n=2, h=20, w=33, cin=128, cout=128, k=3,
                                        bits_in=4, bits_w=4, wenc=1, bits_out=4, num_levels=5)
             for t in range(2)]
    handles = [aqd.qconv_create(128, 128, 3, 1, 1, 4, 4, aqd.pack_codes(c.w_fields, 4), c.levels,
                                wenc=1, bits_out=4) for c in cases]
    rng = np.random.Generator(np.random.PCG64(9))
    try:
        segs, expect, outs = [], [], []
        for t, c in enumerate(cases):
            for lv, (h, w) in enumerate(sizes):
                x = rng.integers(0, 16, size=(2, h, w, 128))
                xd = torch.from_numpy(aqd.pack_codes(x, 4)).to(dev)
                yd = torch.zeros((2, h, w, 64), dtype=torch.uint8, device=dev)
                segs.append((handles[t], lv, 2, h, w, xd, None, 0, 0, yd))
                outs.append(yd)
                L = c.levels[lv]
                want = ref.qconv(x, c.w_fields, 4, 1, 1, L["bias"], wenc=1, mult=L["mult"],
                                 shift=L["shift"], bits_out=4)
                expect.append(ref.pack_codes(want, 4))
        aqd.qconv_run_group(segs)
        torch.cuda.synchronize()
        for i, (yd, want) in enumerate(zip(outs, expect)):
            assert_same(yd.cpu().numpy(), want, f"segment {i}")
    finally:
        for h in handles:
            aqd.qconv_destroy(h)


def test_run_is_deterministic_and_leaves_guard_bytes(torch):
    case = workloads.random_conv_case(seed=77, n=1, h=30, w=31, cin=64, cout=128, k=3,
                                      bits_in=4, bits_w=4, bits_out=4)
    a = gpu_conv(case, torch)[0]
    b = gpu_conv(case, torch)[0]
    assert np.array_equal(a, b)
    dev = torch.device("cuda:0")
    h = aqd.qconv_create(64, 128, 3, 1, 1, 4, 4, aqd.pack_codes(case.w_fields, 4), case.levels)
    try:
        x = torch.from_numpy(aqd.pack_codes(case.x, 4)).to(dev)
        nbytes = 30 * 31 * 64
        buf = torch.full((nbytes + 4096,), 0x5A, dtype=torch.uint8, device=dev)
        y = buf[2048:2048 + nbytes]
        aqd.qconv_run(h, 0, 1, 30, 31, x, None, 0, 0, y)
        torch.cuda.synchronize()
        host = buf.cpu().numpy()
        assert np.all(host[:2048] == 0x5A) and np.all(host[2048 + nbytes:] == 0x5A)
        assert np.array_equal(host[2048:2048 + nbytes].reshape(a.shape), a)
    finally:
        aqd.qconv_destroy(h)


@pytest.mark.parametrize("bits_a,bits_b,bits_out,up2", [(4, 4, 4, True), (2, 2, 2, False),
                                                        (32, 4, 4, False), (4, 32, 8, True),
                                                        (8, 2, 4, True), (3, 3, 3, True),
                                                        (32, 3, 3, False)])
def test_qadd_parity(torch, bits_a, bits_b, bits_out, up2):
    dev = torch.device("cuda:0")
    rng = np.random.Generator(np.random.PCG64(bits_a * 100 + bits_b))
    n, h, w, c = 2, 21, 34, 64
    hb, wb = ((h + 1) // 2, (w + 1) // 2) if up2 else (h, w)

    def draw(bits, shape):
        if bits == 32:
            return rng.integers(-5000, 5000, size=shape)
        return rng.integers(0, 1 << bits, size=shape)

    a, b = draw(bits_a, (n, h, w, c)), draw(bits_b, (n, hb, wb, c))
    p = {"skip_c": rng.integers(1, 1 << 12, c), "skip_d": rng.integers(9, 14, c),
         "skip_side": rng.integers(0, 2, c), "mult": rng.integers(1 << 30, 1 << 31, c),
         "shift": rng.integers(-3, 6, c)}
    want = ref.pack_codes(ref.qadd(a, b, up2, p["skip_c"], p["skip_d"], p["skip_side"], p["mult"],
                                   p["shift"], bits_out), bits_out)

    def dev_t(v, bits):
        if bits == 32:
            return torch.from_numpy(v.astype(np.int32)).to(dev)
        return torch.from_numpy(aqd.pack_codes(v, bits)).to(dev)

    pd = {k: torch.from_numpy(v.astype(np.int32)).to(dev) for k, v in p.items()}
    y = torch.zeros((n, h, w, c * aqd.stored_bits(bits_out) // 8), dtype=torch.uint8, device=dev)
    aqd.qadd_run(n, h, w, c, bits_a, bits_b, bits_out, up2, hb, wb, dev_t(a, bits_a),
                 dev_t(b, bits_b), y, pd)
    torch.cuda.synchronize()
    assert_same(y.cpu().numpy(), want, "qadd")


def test_channel_sums(torch):
    dev = torch.device("cuda:0")
    rng = np.random.Generator(np.random.PCG64(3))
    v = rng.integers(-40000, 40000, size=(3001, 300)).astype(np.int32)
    sums = torch.zeros(600, dtype=torch.int64, device=dev)
    aqd.channel_sums(torch.from_numpy(v).to(dev), 3001, 300, sums)
    torch.cuda.synchronize()
    s = sums.cpu().numpy()
    s1, s2, cnt = ref.channel_sums(v)
    assert cnt == 3001
    assert s[:300].tolist() == s1 and s[300:].tolist() == s2


PROJ_CASES = [
    # (n, h, w, cin, hp, wp, cin_p, stride_p, cout, k, wenc)
    (1, 20, 23, 64, 20, 23, 64, 1, 256, 1, 1),       # first bottleneck block: stride 1 shortcut
    (2, 13, 17, 128, 26, 33, 256, 2, 512, 1, 1),     # later stages: stride 2 shortcut, 2 channel tiles
    (1, 9, 11, 256, 17, 21, 512, 2, 1024, 1, 0),     # ragged pixels, two's-complement weights
    (1, 12, 10, 64, 12, 10, 128, 1, 256, 3, 1),      # 3x3 main convolution
    # one K step each (cin 64): persistent streaming tiles
    (8, 120, 100, 64, 120, 100, 64, 1, 256, 1, 1),   # ~3 tiles per workgroup
    (2, 13, 17, 64, 26, 33, 64, 2, 512, 1, 0),       # stride 2 shortcut, 2 channel tiles
    (1, 9, 11, 64, 9, 11, 64, 1, 768, 1, 1),         # 3 channel tiles, ragged pixels
    # both inputs in 256-channel chunks: register-fed 256 x 64 tiles
    (2, 25, 21, 512, 50, 42, 1024, 2, 2048, 1, 1),   # res5.0 shape: 8 channel tiles
    (4, 21, 27, 256, 21, 27, 256, 1, 512, 1, 0),     # stride 1 shortcut, one stage each
    (8, 30, 41, 256, 60, 81, 512, 2, 1024, 1, 1),    # res4.0 shape: 616 tiles, ragged pixels
    (4, 50, 84, 128, 100, 167, 256, 2, 512, 1, 0),   # res3.0 shape (main cin 128: a padded stage)
]


def _proj_case(case, seed, general=False):
    n, h, w, cin, hp, wp, cin_p, sp, cout, k, wenc = case
    main = workloads.random_conv_case(seed=seed, n=n, h=h, w=w, cin=cin, cout=cout, k=k, bits_in=4,
                                      bits_w=4, wenc=wenc, bits_out=4, skip_bits=32)
    proj = workloads.random_conv_case(seed=seed + 1, n=n, h=hp, w=wp, cin=cin_p, cout=cout, k=1,
                                      stride=sp, bits_in=4, bits_w=4, wenc=wenc, bits_out=32)
    # the skip operand of the main convolution is the projection's int32 output
    t = oracle_conv(proj)
    assert t.shape == (n, main.skip.shape[1], main.skip.shape[2], cout)
    main.skip = t
    if general:
        rng = np.random.Generator(np.random.PCG64(seed))
        main.levels[0]["shift"] = rng.integers(-2, 2, size=cout).astype(np.int32)
        main.levels[0]["mult"] = rng.integers(1 << 24, 1 << 26, size=cout).astype(np.int32)
    return main, proj


def _run_proj(torch, main, proj, fused=True):
    dev = torch.device("cuda:0")
    L = main.levels
    hm = aqd.qconv_create(main.cin, main.cout, main.k, 1, main.pad, 4, 4,
                          aqd.pack_codes(main.w_fields, 4), L, wenc=main.wenc, bits_out=4,
                          skip_bits=32)
    hp_ = aqd.qconv_create(proj.cin, proj.cout, 1, proj.stride, 0, 4, 4,
                           aqd.pack_codes(proj.w_fields, 4), proj.levels, wenc=proj.wenc,
                           out_mode=aqd.OUT_INT32, bits_out=0)
    try:
        ho, wo = aqd.qconv_out_shape(hm, main.h, main.w)
        x = torch.from_numpy(aqd.pack_codes(main.x, 4)).to(dev)
        xp = torch.from_numpy(aqd.pack_codes(proj.x, 4)).to(dev)
        y = torch.full((main.n, ho, wo, main.cout // 2), 0xA5, dtype=torch.uint8, device=dev)
        if fused:
            aqd.qconv_run_proj(hm, hp_, 0, main.n, main.h, main.w, x, proj.h, proj.w, xp, y)
        else:
            t = torch.empty((main.n, ho, wo, main.cout), dtype=torch.int32, device=dev)
            aqd.qconv_run(hp_, 0, proj.n, proj.h, proj.w, xp, None, 0, 0, t)
            aqd.qconv_run(hm, 0, main.n, main.h, main.w, x, t, ho, wo, y)
        torch.cuda.synchronize()
        return y.cpu().numpy()
    finally:
        aqd.qconv_destroy(hm)
        aqd.qconv_destroy(hp_)


@pytest.mark.parametrize("case", PROJ_CASES, ids=lambda c: "x".join(map(str, c)))
def test_fused_projection_parity(torch, case):
    """qconv_run_proj: bit-exact against the oracle's two convolutions, and
    the same bytes as the two separate launches."""
    main, proj = _proj_case(case, seed=hash(case) % 1000 + 11)
    got = _run_proj(torch, main, proj)
    assert_same(got, oracle_conv(main), f"fused projection {case}")
    assert_same(got, _run_proj(torch, main, proj, fused=False), f"fused vs separate {case}")


@pytest.mark.parametrize("which", [1, 2, 4, 7, 10])
def test_fused_projection_general_requant(torch, which):
    """Levels with shift < 2 take the 64-bit requantisation in the fused launch
    (tiled kernel, register-fed kernel and streaming kernel)."""
    main, proj = _proj_case(PROJ_CASES[which], seed=23, general=True)
    assert_same(_run_proj(torch, main, proj), oracle_conv(main), "fused projection, shift < 2")


def test_fused_projection_unsupported_pairs(torch):
    """A pair the fused kernel does not cover is refused without a launch."""
    case = workloads.random_conv_case(seed=2, n=1, h=8, w=8, cin=64, cout=128, k=1, bits_in=2,
                                      bits_w=2, bits_out=2, skip_bits=32)
    hm = aqd.qconv_create(64, 128, 1, 1, 0, 2, 2, aqd.pack_codes(case.w_fields, 2), case.levels,
                          bits_out=2, skip_bits=32)
    hp_ = aqd.qconv_create(64, 128, 1, 1, 0, 2, 2, aqd.pack_codes(case.w_fields, 2), case.levels,
                           out_mode=aqd.OUT_INT32, bits_out=0)
    try:
        dev = torch.device("cuda:0")
        x = torch.zeros((1, 8, 8, 16), dtype=torch.uint8, device=dev)
        y = torch.zeros((1, 8, 8, 32), dtype=torch.uint8, device=dev)
        with pytest.raises(aqd.AqdError) as e:
            aqd.qconv_run_proj(hm, hp_, 0, 1, 8, 8, x, 8, 8, x, y)
        assert e.value.status == aqd.AQD_ERR_UNSUPPORTED
    finally:
        aqd.qconv_destroy(hm)
        aqd.qconv_destroy(hp_)


def test_mfma_probe_is_deterministic(torch):
    """The matrix-core rate probe (a diagnostic the benchmark times) runs and
    writes the same checksums twice."""
    out = torch.zeros(4 * 256, dtype=torch.int32, device="cuda:0")
    aqd.mfma_probe(4, 3, out)
    torch.cuda.synchronize()
    first = out.cpu().numpy().copy()
    out.zero_()
    aqd.mfma_probe(4, 3, out)
    torch.cuda.synchronize()
    assert np.array_equal(first, out.cpu().numpy()) and np.any(first != 0)
