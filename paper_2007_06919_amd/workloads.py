"""Seeded synthetic inputs for the integer low-bit detector path.

This module describes layer shapes and wiring and draws random codes and
parameters from a seed. It performs none of the method's integer arithmetic
(no convolution, rounding, requantisation or skip alignment): both the GPU
path and the CPU oracle consume what it produces, each with its own code.

Tensors are NHWC. Activation tensors hold b-bit unsigned codes (the integer
part of the representation of Sec. 3.1.1, Eq. 1); a tensor with ``bits=32``
holds raw int32 values (the output of a convolution whose normalisation is
applied but which is not requantised, as the skip operand of Eq. 7 allows).

Weights are handed over as their b-bit fields, the form a packed weight
tensor stores, in one of two grids: two's complement (field ``w & (2^b - 1)``
of a signed value w drawn uniformly from [-2^(b-1), 2^(b-1) - 1]), or the
paper's odd grid of Eq. 3 (field eta_w uniform in [0, 2^b - 1], weight value
2*eta_w - (2^b - 1)). The network workloads use the odd grid (zero mean, as
trained weights are); the single-layer workloads state two's-complement ranges.

Two parameter modes:

* ``literal``: integer epilogue parameters drawn directly (bias, multiplier,
  shift, skip numerator/exponent/side), as the single-layer workloads state.
* ``calibrated``: per-channel affine normalisation parameters (gamma, beta)
  are drawn; the running mean and variance are the exact statistics of each
  layer's integer accumulator on the calibration images, so every layer's
  output codes stay spread over [0, 2^b - 1] however deep the network is.
  Each side computes those statistics with its own convolution and turns them
  into integers with its own implementation of Eq. 5-8.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

# Clip range nu of every synthetic activation quantizer (Eq. 2): the step of a
# b-bit code tensor is NU / (2^b - 1).
NU = 3.0
# BN epsilon used by every synthetic normalisation layer.
BN_EPS = 1e-5


def out_size(size: int, k: int, stride: int, pad: int) -> int:
    return (size + 2 * pad - k) // stride + 1


def qmax(bits: int) -> int:
    return (1 << bits) - 1


WENC_TWOS = 0       # two's-complement weight fields
WENC_PAPER_ODD = 1  # Eq. 3 fields: value 2*eta_w - (2^b - 1)


# --------------------------------------------------------------------------
# network description
# --------------------------------------------------------------------------
@dataclass
class TensorSpec:
    name: str
    n: int
    h: int
    w: int
    c: int
    bits: int  # 2/4/8: unsigned codes; 32: raw int32 values

    @property
    def shape(self) -> Tuple[int, int, int, int]:
        return (self.n, self.h, self.w, self.c)


@dataclass
class ConvSpec:
    """One set of conv weights applied to one or more (x, skip, y) segments.

    Segments share the weights and each has its own epilogue table; the
    detection heads use one segment per pyramid level (multi-level BN,
    Sec. 3.2.2, Fig. 3).
    """
    name: str
    cin: int
    cout: int
    k: int
    stride: int
    bits_w: int
    segs: List[Tuple[str, Optional[str], str]]
    skip_up2: bool = False
    wenc: int = WENC_TWOS
    op: str = "conv"     # "conv", or "maxpool" (k x k, stride, pad k // 2; no weights)

    @property
    def pad(self) -> int:
        return self.k // 2


@dataclass
class NetSpec:
    tensors: Dict[str, TensorSpec] = field(default_factory=dict)
    convs: List[ConvSpec] = field(default_factory=list)
    inputs: List[str] = field(default_factory=list)
    outputs: List[str] = field(default_factory=list)
    wenc: int = WENC_TWOS  # weight grid of every conv added afterwards

    def add_tensor(self, name, n, h, w, c, bits) -> TensorSpec:
        assert name not in self.tensors, name
        t = TensorSpec(name, n, h, w, c, bits)
        self.tensors[name] = t
        return t

    def conv(self, name, x, y, cout, k, stride, bits_w, bits_out, skip=None,
             skip_up2=False) -> ConvSpec:
        """Single-segment conv; creates the output tensor."""
        tx = self.tensors[x]
        ho = out_size(tx.h, k, stride, k // 2)
        wo = out_size(tx.w, k, stride, k // 2)
        self.add_tensor(y, tx.n, ho, wo, cout, bits_out)
        c = ConvSpec(name, tx.c, cout, k, stride, bits_w, [(x, skip, y)], skip_up2, self.wenc)
        self.convs.append(c)
        return c

    def maxpool(self, name, x, y, k, stride) -> ConvSpec:
        """k x k max-pooling of codes (pad k // 2); the output has the input's
        width and step (Sec. 3.2.4)."""
        tx = self.tensors[x]
        ho, wo = out_size(tx.h, k, stride, k // 2), out_size(tx.w, k, stride, k // 2)
        self.add_tensor(y, tx.n, ho, wo, tx.c, tx.bits)
        c = ConvSpec(name, tx.c, tx.c, k, stride, 0, [(x, None, y)], False, self.wenc, op="maxpool")
        self.convs.append(c)
        return c

    def conv_levels(self, name, xs, ys, cout, k, bits_w, bits_out) -> ConvSpec:
        """Stride-1 conv with shared weights over several levels."""
        segs = []
        for x, y in zip(xs, ys):
            tx = self.tensors[x]
            self.add_tensor(y, tx.n, tx.h, tx.w, cout, bits_out)
            segs.append((x, None, y))
        c = ConvSpec(name, self.tensors[xs[0]].c, cout, k, 1, bits_w, segs, False, self.wenc)
        self.convs.append(c)
        return c

    def macs(self, conv: ConvSpec) -> int:
        if conv.op != "conv":
            return 0
        total = 0
        for _, _, y in conv.segs:
            t = self.tensors[y]
            total += t.n * t.h * t.w * conv.cout * conv.k * conv.k * conv.cin
        return total

    def total_macs(self) -> int:
        return sum(self.macs(c) for c in self.convs)


# --------------------------------------------------------------------------
# networks of the five workloads
# --------------------------------------------------------------------------
def single_conv_net(n, h, w, cin, cout, k, stride, bits_in, bits_w, bits_out,
                    skip_bits=None, skip_up2=False) -> NetSpec:
    net = NetSpec()
    net.add_tensor("x", n, h, w, cin, bits_in)
    net.inputs.append("x")
    skip = None
    if skip_bits is not None:
        ho, wo = out_size(h, k, stride, k // 2), out_size(w, k, stride, k // 2)
        hs, ws = ((ho + 1) // 2, (wo + 1) // 2) if skip_up2 else (ho, wo)
        net.add_tensor("skip", n, hs, ws, cout, skip_bits)
        net.inputs.append("skip")
        skip = "skip"
    net.conv("conv", "x", "y", cout, k, stride, bits_w, bits_out, skip, skip_up2)
    net.outputs.append("y")
    return net


def basic_block_net(n, h, w, c, bits) -> NetSpec:
    """ResNet-18 basic block: 3x3 conv, BN, ReLU; 3x3 conv, BN, + identity, ReLU."""
    net = NetSpec()
    net.add_tensor("x", n, h, w, c, bits)
    net.inputs.append("x")
    net.conv("conv1", "x", "h", c, 3, 1, bits, bits)
    net.conv("conv2", "h", "y", c, 3, 1, bits, bits, skip="x")
    net.outputs.append("y")
    return net


LEVELS = ("p3", "p4", "p5", "p6", "p7")
NUM_ANCHORS = 9
NUM_CLASSES = 80


def pyramid_sizes(h: int, w: int) -> List[Tuple[int, int]]:
    """Spatial sizes of P3..P7 for an h x w image (ResNet strides 8..128)."""
    sizes = []
    ch, cw = out_size(out_size(h, 7, 2, 3), 3, 2, 1), out_size(out_size(w, 7, 2, 3), 3, 2, 1)
    for _ in range(3):  # C3, C4, C5 (3x3 stride-2 convs, pad 1)
        ch, cw = out_size(ch, 3, 2, 1), out_size(cw, 3, 2, 1)
        sizes.append((ch, cw))
    for _ in range(2):  # P6, P7
        ch, cw = out_size(ch, 3, 2, 1), out_size(cw, 3, 2, 1)
        sizes.append((ch, cw))
    return sizes


def add_retina_heads(net: NetSpec, levels, bits, towers=("cls", "box"), io_bits=None):
    """RetinaNet heads shared over the pyramid levels, with a private epilogue
    table per level (multi-level BN). io_bits: the prediction convolutions as
    output layers of that width (their input codes, from the last tower
    layer, and their two's-complement weights; Sec. 4, the fully quantized
    networks), else at ``bits``."""
    for tower in towers:
        xs = list(levels)
        for i in range(1, 5):
            ys = [f"{tower}{i}.{lv}" for lv in levels]
            net.conv_levels(f"{tower}.t{i}", xs, ys, 256, 3, bits, io_bits if (io_bits and i == 4) else bits)
            xs = ys
        cout = NUM_ANCHORS * NUM_CLASSES if tower == "cls" else NUM_ANCHORS * 4
        ys = [f"{tower}_out.{lv}" for lv in levels]
        wenc = net.wenc
        if io_bits:
            net.wenc = WENC_TWOS
        net.conv_levels(f"{tower}.pred", xs, ys, cout, 3, io_bits or bits, 32)
        net.wenc = wenc
        net.outputs.extend(ys)


def add_fcos_heads(net: NetSpec, levels, bits):
    """FCOS heads (the paper's second detector, Table 4), shared over the
    pyramid levels with a private epilogue table per level: a class tower and
    a box tower of four 3x3 256->256 convs each; predictions (int32) of the
    per-location class scores (NUM_CLASSES), box distances (4) and
    centerness (1, from the box tower)."""
    tops = {}
    for tower in ("cls", "box"):
        xs = list(levels)
        for i in range(1, 5):
            ys = [f"{tower}{i}.{lv}" for lv in levels]
            net.conv_levels(f"{tower}.t{i}", xs, ys, 256, 3, bits, bits)
            xs = ys
        tops[tower] = xs
    for name, tower, cout in (("cls.pred", "cls", NUM_CLASSES), ("box.pred", "box", 4),
                              ("ctr.pred", "box", 1)):
        ys = [f"{name.split('.')[0]}_out.{lv}" for lv in levels]
        net.conv_levels(name, tops[tower], ys, cout, 3, bits, 32)
        net.outputs.extend(ys)


def fcos_r50_net(n, h, w, bits, wenc=WENC_PAPER_ODD) -> NetSpec:
    """ResNet-50 + FPN (as retinanet_r50_net) with the FCOS heads."""
    net = retinanet_r50_net(n, h, w, bits, heads=False, wenc=wenc)
    net.outputs.clear()
    add_fcos_heads(net, LEVELS, bits)
    return net


def fcos_config(n, h, w, bits=4, seed=5):
    """(NetSpec, NetParams) of the FCOS network, calibrated recipe."""
    net = fcos_r50_net(n, h, w, bits)
    return net, make_params(net, seed, "calibrated")


def head_tower_net(n, h, w, bits, wenc=WENC_PAPER_ODD) -> NetSpec:
    """Class tower of the RetinaNet head on the five pyramid levels of an
    h x w image: four 3x3 256->256 convs and the 3x3 256->720 prediction."""
    net = NetSpec(wenc=wenc)
    for lv, (lh, lw) in zip(LEVELS, pyramid_sizes(h, w)):
        net.add_tensor(lv, n, lh, lw, 256, bits)
        net.inputs.append(lv)
    add_retina_heads(net, LEVELS, bits, towers=("cls",))
    return net


def retinanet_r50_net(n, h, w, bits, heads=True, wenc=WENC_PAPER_ODD, io_bits=None) -> NetSpec:
    """ResNet-50 (bottleneck, stride on the 3x3), FPN with fused top-down
    adds, P6/P7, and optionally the RetinaNet heads. Without io_bits the
    network starts after the stem (input: the max-pooled stem output); with
    io_bits (8: the paper's fully quantized networks, Sec. 4) it starts at
    the image (3 channels of io_bits codes) with the 7x7 stride-2 stem
    (io_bits two's-complement weights, ``bits`` output codes) and the 3x3
    stride-2 max-pooling, and the heads' prediction convolutions are io_bits
    layers."""
    net = NetSpec(wenc=wenc)
    if io_bits:
        net.add_tensor("img", n, h, w, 3, io_bits)
        net.inputs.append("img")
        net.wenc = WENC_TWOS
        net.conv("stem", "img", "c1", 64, 7, 2, io_bits, bits)
        net.wenc = wenc
        net.maxpool("pool", "c1", "c2in", 3, 2)
    else:
        h2 = out_size(out_size(h, 7, 2, 3), 3, 2, 1)
        w2 = out_size(out_size(w, 7, 2, 3), 3, 2, 1)
        net.add_tensor("c2in", n, h2, w2, 64, bits)
        net.inputs.append("c2in")
    x = "c2in"
    cin = 64
    stage_out = {}
    for si, (width, blocks, stride) in enumerate(((64, 3, 1), (128, 4, 2), (256, 6, 2), (512, 3, 2))):
        st = si + 2
        for bi in range(blocks):
            s = stride if bi == 0 else 1
            p = f"res{st}.{bi}"
            net.conv(f"{p}.conv1", x, f"{p}.a", width, 1, 1, bits, bits)
            net.conv(f"{p}.conv2", f"{p}.a", f"{p}.b", width, 3, s, bits, bits)
            if bi == 0:
                net.conv(f"{p}.down", x, f"{p}.ds", 4 * width, 1, s, bits, 32)
                skip = f"{p}.ds"
            else:
                skip = x
            net.conv(f"{p}.conv3", f"{p}.b", f"{p}.out", 4 * width, 1, 1, bits, bits, skip=skip)
            x = f"{p}.out"
            cin = 4 * width
        stage_out[st] = x
    c3, c4, c5 = stage_out[3], stage_out[4], stage_out[5]
    net.conv("fpn.lat5", c5, "p5in", 256, 1, 1, bits, bits)
    net.conv("fpn.lat4", c4, "p4in", 256, 1, 1, bits, bits, skip="p5in", skip_up2=True)
    net.conv("fpn.lat3", c3, "p3in", 256, 1, 1, bits, bits, skip="p4in", skip_up2=True)
    net.conv("fpn.out3", "p3in", "p3", 256, 3, 1, bits, bits)
    net.conv("fpn.out4", "p4in", "p4", 256, 3, 1, bits, bits)
    net.conv("fpn.out5", "p5in", "p5", 256, 3, 1, bits, bits)
    net.conv("fpn.p6", c5, "p6", 256, 3, 2, bits, bits)
    net.conv("fpn.p7", "p6", "p7", 256, 3, 2, bits, bits)
    if heads:
        add_retina_heads(net, LEVELS, bits, io_bits=io_bits)
    else:
        net.outputs.extend(LEVELS)
    return net


# --------------------------------------------------------------------------
# random draws
# --------------------------------------------------------------------------
def draw_codes(rng, shape, bits) -> np.ndarray:
    return rng.integers(0, qmax(bits), size=shape, endpoint=True).astype(np.uint8)


def draw_weights(rng, cout, k, cin, bits, wenc):
    """(fields, values) of a [cout][k][k][cin] weight tensor."""
    shape = (cout, k, k, cin)
    if wenc == WENC_PAPER_ODD:
        fields = rng.integers(0, qmax(bits), size=shape, endpoint=True)
        values = 2 * fields - qmax(bits)
    else:
        lo, hi = -(1 << (bits - 1)), (1 << (bits - 1)) - 1
        values = rng.integers(lo, hi, size=shape, endpoint=True)
        fields = values & qmax(bits)
    return fields.astype(np.uint8), values.astype(np.int32)


def draw_literal_epilogue(rng, cout, with_skip):
    """Integer epilogue parameters as the single-layer workloads state them:
    bias U[-2^12, 2^12], multiplier U[2^30, 2^31), right shift U[8, 16];
    skip numerator U[2^30, 2^31), exponent U[22, 30], side U{0, 1}."""
    p = {
        "bias": rng.integers(-(1 << 12), 1 << 12, size=cout, endpoint=True).astype(np.int32),
        "mult": rng.integers(1 << 30, 1 << 31, size=cout).astype(np.int32),
        "shift": rng.integers(8, 16, size=cout, endpoint=True).astype(np.int32),
    }
    if with_skip:
        p["skip_c"] = rng.integers(1 << 30, 1 << 31, size=cout).astype(np.int32)
        p["skip_d"] = rng.integers(22, 30, size=cout, endpoint=True).astype(np.int32)
        p["skip_side"] = rng.integers(0, 1, size=cout, endpoint=True).astype(np.int32)
    return p


@dataclass
class NetParams:
    mode: str
    inputs: Dict[str, np.ndarray]
    alpha: Dict[str, float]            # step of each code tensor
    weights: Dict[str, np.ndarray]     # b-bit fields [cout][k][k][cin]
    alpha_w: Dict[str, float]
    segs: Dict[str, List[dict]]        # per conv, per segment
    bn_eps: float = BN_EPS
    calib_images: Tuple[int, ...] = (0,)


def make_params(net: NetSpec, seed: int, mode: str) -> NetParams:
    """Draw every input and parameter of ``net`` from PCG64(seed).

    Draw order: each input tensor (in ``net.inputs`` order), then per conv:
    weights, then per segment the epilogue draws (literal: bias, multiplier,
    shift, then skip numerator, exponent, side; calibrated: gamma U[0.5, 1.5],
    beta U[0, 1]).

    In calibrated mode the running mean and variance of each normalisation are
    not drawn: they are the statistics of that layer's integer accumulator
    over the images ``calib_images`` of the batch, which each side computes
    with its own convolution.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    inputs = {name: draw_codes(rng, net.tensors[name].shape, net.tensors[name].bits)
              for name in net.inputs}
    alpha = {name: NU / qmax(t.bits) for name, t in net.tensors.items() if t.bits != 32}
    weights, alpha_w, segs = {}, {}, {}
    for conv in net.convs:
        if conv.op != "conv":
            continue
        weights[conv.name], _ = draw_weights(rng, conv.cout, conv.k, conv.cin, conv.bits_w,
                                             conv.wenc)
        alpha_w[conv.name] = 1.0 / qmax(conv.bits_w)
        seg_params = []
        for (x, skip, y) in conv.segs:
            if mode == "literal":
                seg_params.append(draw_literal_epilogue(rng, conv.cout, skip is not None))
            else:
                gamma = rng.uniform(0.5, 1.5, size=conv.cout)
                beta = rng.uniform(0.0, 1.0, size=conv.cout)
                seg_params.append({"gamma": gamma, "beta": beta})
        segs[conv.name] = seg_params
    return NetParams(mode, inputs, alpha, weights, alpha_w, segs)


# --------------------------------------------------------------------------
# the five workloads
# --------------------------------------------------------------------------
CONFIG_NAMES = (
    "conv3x3_64x64_32x32_4bit",
    "r18_basic_block_stage2_n2_100x168_2bit",
    "retina_cls_tower_p3p7_800x1333_4bit",
    "r50_fpn_n1_800x1333_2bit",
    "retinanet_r50_fpn_n8_800x1333_4bit",
)


def config(idx: int):
    """(NetSpec, NetParams) of workload ``idx`` with seed = idx."""
    if idx == 0:
        net = single_conv_net(1, 32, 32, 64, 64, 3, 1, 4, 4, 4)
        return net, make_params(net, 0, "literal")
    if idx == 1:
        net = basic_block_net(2, 100, 168, 128, 2)
        return net, make_params(net, 1, "literal")
    if idx == 2:
        net = head_tower_net(1, 800, 1333, 4)
        return net, make_params(net, 2, "calibrated")
    if idx == 3:
        net = retinanet_r50_net(1, 800, 1333, 2, heads=False)
        return net, make_params(net, 3, "calibrated")
    if idx == 4:
        net = retinanet_r50_net(8, 800, 1333, 4, heads=True)
        return net, make_params(net, 4, "calibrated")
    raise ValueError(idx)


def scaled_config(idx: int, n: int, h: int, w: int, seed: Optional[int] = None):
    """Workloads 2-4 at a reduced image size / batch (same wiring and recipe)."""
    seed = idx if seed is None else seed
    if idx == 2:
        net = head_tower_net(n, h, w, 4)
    elif idx == 3:
        net = retinanet_r50_net(n, h, w, 2, heads=False)
    elif idx == 4:
        net = retinanet_r50_net(n, h, w, 4, heads=True)
    else:
        raise ValueError(idx)
    return net, make_params(net, seed, "calibrated")


def retinanet_config(n: int, h: int, w: int, bits: int, seed: int = 6, io_bits=None):
    """ResNet-50 + FPN + RetinaNet heads at any code width (3: the paper's
    3-bit networks, Tables 2 and 4), calibrated, same recipe as workload 4;
    io_bits=8: the fully quantized network (8-bit image, stem and
    prediction convolutions, max-pooling)."""
    net = retinanet_r50_net(n, h, w, bits, heads=True, io_bits=io_bits)
    return net, make_params(net, seed, "calibrated")


# --------------------------------------------------------------------------
# random single-conv cases (parity fuzzing)
# --------------------------------------------------------------------------
@dataclass
class ConvCase:
    n: int
    h: int
    w: int
    cin: int
    cout: int
    k: int
    stride: int
    pad: int
    bits_in: int
    bits_w: int
    wenc: int
    bits_out: int        # 32: int32 output
    skip_bits: int       # 0: none
    skip_up2: bool
    x: np.ndarray        # [n][h][w][cin] codes
    w_fields: np.ndarray  # [cout][k][k][cin]
    skip: Optional[np.ndarray]   # [n][hs][ws][cout] codes or int32 values
    levels: List[dict]   # integer epilogue tables

    @property
    def out_hw(self):
        return (out_size(self.h, self.k, self.stride, self.pad),
                out_size(self.w, self.k, self.stride, self.pad))


def random_conv_case(seed, n, h, w, cin, cout, k=3, stride=1, bits_in=4, bits_w=4,
                     wenc=WENC_TWOS, bits_out=4, skip_bits=0, skip_up2=False, num_levels=1):
    """Random codes and an integer epilogue whose scale keeps the output codes
    spread over their range (multiplier U[2^30, 2^31), exponent chosen from
    the accumulator's standard deviation under the drawn distributions)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    pad = k // 2
    x = draw_codes(rng, (n, h, w, cin), bits_in)
    w_fields, wv = draw_weights(rng, cout, k, cin, bits_w, wenc)
    ho, wo = out_size(h, k, stride, pad), out_size(w, k, stride, pad)
    qx = qmax(bits_in)
    ex2 = (qx * (2 * qx + 1)) / 6.0                 # E[x^2], x uniform on 0..qx
    ew2 = float(np.mean(wv.astype(np.float64) ** 2)) + 1e-9
    acc_sd = np.sqrt(k * k * cin * ex2 * ew2)
    # expected accumulator per channel (interior pixels): E[x] * sum of the channel's weights
    acc_mean = (qx / 2.0) * wv.reshape(cout, -1).sum(axis=1).astype(np.float64)
    skip = None
    if skip_bits:
        hs, ws = ((ho + 1) // 2, (wo + 1) // 2) if skip_up2 else (ho, wo)
        if skip_bits == 32:
            lim = int(4 * acc_sd) + 1
            skip = rng.integers(-lim, lim, size=(n, hs, ws, cout)).astype(np.int32)
        else:
            skip = draw_codes(rng, (n, hs, ws, cout), skip_bits)
    levels = []
    for _ in range(num_levels):
        noise = rng.integers(-int(acc_sd / 2), int(acc_sd / 2) + 1, size=cout)
        lv = {"bias": (np.round(-acc_mean) + noise).astype(np.int32)}
        if bits_out != 32:
            target = qmax(bits_out) / (2.0 * acc_sd)   # scale mapping ~2 sd onto the code range
            lv["mult"] = rng.integers(1 << 30, 1 << 31, size=cout).astype(np.int32)
            base = int(np.floor(-np.log2(target)))     # M / 2^(31 + shift) ~ target
            lv["shift"] = (base + rng.integers(-1, 2, size=cout)).clip(-31, 31).astype(np.int32)
        if skip_bits:
            lv["skip_c"] = rng.integers(1, 1 << 12, size=cout).astype(np.int32)
            lv["skip_d"] = rng.integers(9, 14, size=cout).astype(np.int32)
            lv["skip_side"] = rng.integers(0, 2, size=cout).astype(np.int32)
        levels.append(lv)
    return ConvCase(n, h, w, cin, cout, k, stride, pad, bits_in, bits_w, wenc, bits_out,
                    skip_bits, skip_up2, x, w_fields, skip, levels)
