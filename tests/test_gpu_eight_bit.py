"""GPU parity of the 8-bit input and output layers of the paper's fully
quantized networks (Sec. 4): 8-bit codes on the int8 MFMA (re-centred by
-128, the bias carrying 128 * sum(w)), the 7x7 stride-2 stem on a 3-channel
8-bit image, 8-bit code outputs of the register-fed kernel, and the whole
network (stem, max-pooling, ResNet-50, FPN, heads with 8-bit prediction
convolutions) against the oracle."""
import numpy as np
import pytest

from gpu_helpers import assert_same, gpu_conv, oracle_conv
from paper_2007_06919_amd import aqd, workloads

pytestmark = pytest.mark.gpu

TWOS = workloads.WENC_TWOS


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available()
    return t


def _case(seed, n, h, w, cin, cout, k, stride, bits_in, bits_w, wenc, bits_out, skip_bits=0, up2=False):
    return workloads.random_conv_case(seed=seed, n=n, h=h, w=w, cin=cin, cout=cout, k=k, stride=stride,
                                      bits_in=bits_in, bits_w=bits_w, wenc=wenc, bits_out=bits_out,
                                      skip_bits=skip_bits, skip_up2=up2)


def _path(c):
    h = aqd.qconv_create(c.cin, c.cout, c.k, c.stride, c.pad, c.bits_in, c.bits_w,
                         aqd.pack_codes(c.w_fields, c.bits_w), c.levels, wenc=c.wenc,
                         out_mode=aqd.OUT_INT32 if c.bits_out == 32 else aqd.OUT_CODES,
                         bits_out=0 if c.bits_out == 32 else c.bits_out, skip_bits=c.skip_bits,
                         skip_up2=c.skip_up2)
    try:
        return aqd.qconv_path(h)
    finally:
        aqd.qconv_destroy(h)


B8_CASES = [
    # (n, h, w, cin, cout, k, stride): 8-bit codes, 8-bit weights, int32 outputs
    (1, 30, 50, 256, 720, 3, 1),     # class predictor: a partial channel tile
    (2, 20, 33, 128, 36, 3, 1),      # box predictor shape, 128 input channels
    (1, 25, 40, 384, 256, 1, 1),     # 1x1, three stages per tap
    (3, 17, 13, 256, 512, 3, 2),     # stride 2, ragged pixel tail
]


@pytest.mark.parametrize("case", B8_CASES, ids=lambda c: "x".join(map(str, c)))
def test_eight_bit_codes_on_mfma(torch, case):
    n, h, w, cin, cout, k, s = case
    c = _case(hash(case) % 1000 + 3, n, h, w, cin, cout, k, s, 8, 8, TWOS, 32)
    assert _path(c) == "i8-mfma"
    assert_same(gpu_conv(c, torch)[0], oracle_conv(c), f"8-bit {case}")


def test_eight_bit_split_k(torch):
    c = _case(5, 1, 9, 13, 1024, 256, 3, 1, 8, 8, TWOS, 32)
    assert_same(gpu_conv(c, torch, split=True)[0], oracle_conv(c), "8-bit split K")


def test_eight_bit_extremes(torch):
    """Codes 0 and 255 and weights -128 and 127 (the re-centring's worst
    cases: every product of the shifted codes at its largest magnitude),
    padding taps included."""
    c = _case(9, 1, 11, 14, 256, 256, 3, 1, 8, 8, TWOS, 32)
    rng = np.random.Generator(np.random.PCG64(9))
    c.x[:] = np.where(rng.random(c.x.shape) < 0.5, 0, 255)
    c.w_fields[:] = np.where(rng.random(c.w_fields.shape) < 0.5, 0x80, 0x7F)   # -128 / 127
    c.w_fields[:8] = 0x7F
    c.x[0, :, :, :] = 255
    assert_same(gpu_conv(c, torch)[0], oracle_conv(c), "8-bit extremes")


WV8_CASES = [
    # 4-bit codes in, 8-bit codes out (the last tower layer before 8-bit predictions)
    (2, 50, 84, 256, 256, 3, 1),     # head-tower shape
    (8, 50, 84, 256, 256, 3, 1),     # 263 tiles of 256 x 128: 256 x 144 tiles
    (1, 7, 9, 256, 256, 3, 1),       # one partial tile (a launch far below one round)
    (1, 20, 30, 512, 288, 1, 1),     # 1x1, two stages per tap, a partial channel tile
    (1, 20, 30, 256, 256, 1, 1),     # 1x1, one stage in all (the first is the last)
    (8, 50, 84, 256, 256, 1, 1),     # one stage on 256 x 144 tiles
]


@pytest.mark.parametrize("case", WV8_CASES, ids=lambda c: "x".join(map(str, c)))
@pytest.mark.parametrize("variant", ["plain", "small_shifts"])
def test_eight_bit_code_outputs(torch, case, variant):
    n, h, w, cin, cout, k, s = case
    c = _case(hash(case) % 1000 + 19, n, h, w, cin, cout, k, s, 4, 4, workloads.WENC_PAPER_ODD, 8)
    if variant == "small_shifts":
        rng = np.random.Generator(np.random.PCG64(21))
        for lv in c.levels:
            lv["shift"] = rng.integers(-2, 2, size=cout).astype(np.int32)
            lv["mult"] = rng.integers(1 << 20, 1 << 24, size=cout).astype(np.int32)
    assert _path(c) == "i8-mfma"
    for level, got in enumerate(gpu_conv(c, torch)):
        assert_same(got, oracle_conv(c, level), f"8-bit outputs {variant} {case} level {level}")


STEM_CASES = [
    # (n, h, w, bits_out, variant): 7x7 stride 2 pad 3, 3 -> 64 channels, 8-bit
    # image and weights; small_shifts: the 64-bit requantisation
    (2, 64, 96, 4, "plain"),
    (2, 64, 96, 4, "small_shifts"),
    (1, 33, 47, 4, "plain"),         # odd sizes; the image's byte count is not a multiple of 4
    (1, 33, 47, 32, "plain"),        # int32 outputs (the calibration pass)
    (3, 21, 18, 4, "plain"),         # several images, ragged pixel tail
    (3, 21, 18, 4, "small_shifts"),
]


@pytest.mark.parametrize("case", STEM_CASES, ids=lambda c: "x".join(map(str, c)))
def test_stem_on_mfma(torch, case):
    n, h, w, bo, variant = case
    c = _case(hash(case) % 1000 + 23, n, h, w, 3, 64, 7, 2, 8, 8, TWOS, bo)
    if variant == "small_shifts":
        rng = np.random.Generator(np.random.PCG64(25))
        for lv in c.levels:
            lv["shift"] = rng.integers(-2, 2, size=64).astype(np.int32)
            lv["mult"] = rng.integers(1 << 18, 1 << 22, size=64).astype(np.int32)
    assert _path(c) == "i8-mfma"
    for level, got in enumerate(gpu_conv(c, torch)):
        assert_same(got, oracle_conv(c, level), f"stem {variant} {case} level {level}")


def test_aqd_full_retinanet_scaled(torch):
    """The fully quantized RetinaNet-R50 (8-bit image, stem and prediction
    convolutions, max-pooling, 4-bit elsewhere), calibrated: every tensor and
    every epilogue table against the oracle."""
    from test_gpu_network import compare_network
    net, params = workloads.retinanet_config(2, 192, 256, 4, io_bits=8)
    compare_network(torch, net, params)


def test_aqd_full_retinanet_full_size(torch):
    """The same network on two 800x1333 images."""
    from test_gpu_network import compare_network
    net, params = workloads.retinanet_config(2, 800, 1333, 4, io_bits=8)
    compare_network(torch, net, params)
