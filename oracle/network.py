"""Oracle evaluation of a whole quantized network, layer by layer.

TEST INFRASTRUCTURE (see ``oracle/ref.py``). Takes a network description
(tensors with shapes and bitwidths, convolutions with their (x, skip, y)
segments, max-pooling layers) and its seeded parameters as plain objects, derives each layer's
integer epilogue with the oracle's own host derivation, and evaluates the
layers in order with the oracle convolution. Images of a batch are
independent, so ``images`` may select a subset of the batch; the calibration
images must be part of it.
"""
from __future__ import annotations

import numpy as np

from . import ref


def _segment_table(net, params, conv, seg, p, vals, alpha_t, pos):
    """Integer epilogue of one segment.

    literal mode: the drawn integers as they are.
    calibrated mode:
      acc statistics on the calibration images -> running mean/var
      alpha_conv = alpha_x * alpha_w                              (Eq. 4)
      bias, alpha_z = BN fold                                     (Eq. 5-6)
      int32 output: alpha_z per channel becomes that tensor's scale
      code output: with a skip, c, d, side and the sum's scale   (Eq. 7-8);
                   multiplier/shift of (scale / alpha_y)          (Eq. 2)
    """
    x, skip, y = seg
    if params.mode == "literal":
        return {k: np.asarray(v, np.int64) for k, v in p.items()}
    ty = net.tensors[y]
    sel = [pos[i] for i in params.calib_images]
    acc = ref.qconv(vals[x][sel], params.weights[conv.name], conv.bits_w, conv.stride,
                    conv.pad, np.zeros(conv.cout, np.int64), wenc=conv.wenc, out_int32=True)
    s1, s2, count = ref.channel_sums(acc)
    alpha_conv = params.alpha[x] * params.alpha_w[conv.name]
    mean, var = ref.bn_stats_from_sums(s1, s2, count, alpha_conv)
    bias, alpha_z = ref.fold_bn(p["gamma"], p["beta"], mean, var, params.bn_eps, alpha_conv)
    t = {"bias": bias}
    if ty.bits == 32:
        alpha_t[y] = alpha_z
    else:
        scale = alpha_z
        if skip is not None:
            ak = alpha_t[skip] if net.tensors[skip].bits == 32 else params.alpha[skip]
            c, d, side, scale = ref.skip_params(alpha_z, ak)
            t.update(skip_c=c, skip_d=d, skip_side=side)
        t["mult"], t["shift"] = ref.requant_params(scale, params.alpha[y])
    return t


def run(net, params, images=None, keep=None):
    """Evaluate the network; returns ({tensor name: int64 NHWC array}, tables).

    images: optional list of batch indices to evaluate (must include the
            calibration images in calibrated mode).
    keep:   optional set of tensor names to keep; other intermediate tensors
            are dropped once no later layer reads them.
    """
    n = net.tensors[net.inputs[0]].n
    images = list(range(n)) if images is None else list(images)
    pos = {img: i for i, img in enumerate(images)}
    if params.mode != "literal":
        missing = [i for i in params.calib_images if i not in pos]
        assert not missing, f"calibration images {missing} not evaluated"
    vals = {name: params.inputs[name].astype(np.int64)[images] for name in net.inputs}
    last_use = {}
    for i, conv in enumerate(net.convs):
        for x, skip, _ in conv.segs:
            last_use[x] = i
            if skip is not None:
                last_use[skip] = i
    tables = {}
    alpha_t = {}
    for i, conv in enumerate(net.convs):
        if conv.op == "maxpool":
            # codes pooled as they are, the scale unchanged (Sec. 3.2.4)
            x, _, y = conv.segs[0]
            vals[y] = ref.maxpool(vals[x], conv.k, conv.stride, conv.pad)
            tables[conv.name] = []
            continue
        segs = []
        for si, seg in enumerate(conv.segs):
            x, skip, y = seg
            t = _segment_table(net, params, conv, seg, params.segs[conv.name][si], vals,
                               alpha_t, pos)
            segs.append(t)
            ty = net.tensors[y]
            out32 = ty.bits == 32
            vals[y] = ref.qconv(
                vals[x], params.weights[conv.name], conv.bits_w, conv.stride, conv.pad,
                t["bias"], wenc=conv.wenc, out_int32=out32, mult=t.get("mult"),
                shift=t.get("shift"), bits_out=0 if out32 else ty.bits,
                skip=vals[skip] if skip is not None else None, skip_up2=conv.skip_up2,
                skip_c=t.get("skip_c"), skip_d=t.get("skip_d"), skip_side=t.get("skip_side"))
        tables[conv.name] = segs
        if keep is not None:
            for name in list(vals):
                if name not in keep and name not in net.inputs and last_use.get(name, -1) <= i:
                    del vals[name]
    return vals, tables
