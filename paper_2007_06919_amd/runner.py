"""Stream-ordered whole-network runner on the C ABI.

A network description (``workloads.NetSpec``) becomes a list of grouped
``qconv_run_group`` launches on one HIP stream:

* every tensor gets one device buffer (packed codes, or int32), so a forward
  pass allocates nothing and can be captured in a HIP graph;
* convolutions are ordered by dependency depth, and convolutions of the same
  depth and configuration (same shapes, bitwidths and modes) share a launch:
  the pyramid levels of a head layer (one epilogue table per level,
  multi-level BN, Sec. 3.2.2) and the class and box towers at equal depth;
* a residual block's projection shortcut (1x1 conv with int32 output read
  only by the block's last conv) runs fused into that conv
  (``qconv_run_proj``): its int32 tensor is not written during a forward
  pass (it is written once, at set-up, by the calibration pass);
* ``capture()`` records one forward pass into a HIP graph (``aqd_graph_*``)
  and ``replay()`` enqueues the whole network as one graph launch;
* launches that do not continue the main chain of dependencies (the FPN's
  P6/P7 branch and P4/P5 output convolutions, the box prediction) run on two
  side streams, joined by events (``plan_streams``);
* one workspace, sized for the largest group's split-K need
  (``qconv_group_workspace``), lets small launches split their K reduction
  over more workgroups (``qconv_run_group_ws``);
* in calibrated mode the integer epilogue of every layer is derived here,
  from the exact accumulator sums of the calibration images computed on the
  GPU (int32 conv output + ``aqd_channel_sums``) and the library's host
  helpers for Eq. 5-8; layers are calibrated in network order.

PyTorch provides device memory and the stream; all arithmetic is in
``libaqd.so``.
"""
from __future__ import annotations

from typing import Dict, List, Tuple

import numpy as np

from . import aqd
from .workloads import NetParams, NetSpec


def _conv_key(net: NetSpec, conv) -> tuple:
    x, skip, y = conv.segs[0]
    ty = net.tensors[y]
    if conv.op != "conv":
        return (conv.op, conv.name)   # launched alone
    return (conv.cin, conv.cout, conv.k, conv.stride, net.tensors[x].bits, conv.bits_w, conv.wenc,
            ty.bits, net.tensors[skip].bits if skip else 0, conv.skip_up2)


def group_inputs(group, fused, fused_away):
    """Tensors a launch of this group reads (codes, skips, fused shortcut inputs)."""
    ins = []
    for conv, si in group:
        if conv.name in fused_away:
            continue
        x, skip, _ = conv.segs[si]
        ins.append(x)
        if conv.name in fused:
            ins.append(fused[conv.name].segs[0][0])  # the shortcut's input
        elif skip is not None:
            ins.append(skip)
    return ins


def plan_streams(schedule, fused, fused_away, nstreams):
    """Stream plan of a pass: per group, the groups it depends on (producers
    of the tensors it reads) and its stream (0 = the main stream; None for
    groups that launch nothing, the fused-away shortcuts); and the set of
    groups after which an event is recorded (those another stream waits for,
    and each side stream's last group, which the main stream joins at the end
    of a pass). A group continues the stream whose last group it depends on
    (latest first); otherwise it opens on the side stream least recently used."""
    producer = {}
    for gi, group in enumerate(schedule):
        for conv, si in group:
            if conv.name not in fused_away:
                producer[conv.segs[si][2]] = gi
    deps, lane, last = [], [], [None] * nstreams
    used = [0] * nstreams
    for gi, group in enumerate(schedule):
        ins = group_inputs(group, fused, fused_away)
        d = sorted({producer[t] for t in ins if t in producer} - {gi})
        deps.append(d)
        if not ins:
            lane.append(None)
            continue
        pick = None
        for dep in sorted(d, reverse=True):
            if lane[dep] is not None and last[lane[dep]] == dep:
                pick = lane[dep]
                break
        if pick is None:
            if gi == 0 or not d or nstreams == 1:
                pick = 0
            else:
                pick = min(range(1, nstreams), key=lambda k: used[k])
        lane.append(pick)
        last[pick] = gi
        used[pick] = gi + 1
    signal = {d for gi, ds in enumerate(deps) for d in ds
              if lane[gi] is not None and lane[d] is not None and lane[d] != lane[gi]}
    for k in range(1, nstreams):
        mine = [gi for gi, l in enumerate(lane) if l == k]
        if mine:
            signal.add(mine[-1])
    return deps, lane, signal


class Net:
    def __init__(self, net: NetSpec, params: NetParams, device="cuda:0", stream=None,
                 split_k: bool = True, fuse_proj: bool = True, side_streams: int = 2):
        import torch

        self.torch = torch
        self.net, self.params = net, params
        self.device = torch.device(device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self.bufs: Dict[str, "torch.Tensor"] = {}
        for name, t in net.tensors.items():
            if t.bits == 32:
                self.bufs[name] = torch.empty(t.shape, dtype=torch.int32, device=self.device)
            else:
                self.bufs[name] = torch.empty((t.n, t.h, t.w, t.c * aqd.stored_bits(t.bits) // 8), dtype=torch.uint8,
                                              device=self.device)
        for name in net.inputs:
            t = net.tensors[name]
            packed = aqd.pack_codes(params.inputs[name], t.bits)
            self.bufs[name].copy_(torch.from_numpy(packed))
        self.handles: Dict[str, int] = {}
        self._pool_descs = []
        self.tables: Dict[str, List[dict]] = {}
        self._alpha_t: Dict[str, np.ndarray] = {}
        self.schedule = self._make_schedule()
        self.fused = self._fusable() if fuse_proj else {}
        self._fused_away = {d.name for d in self.fused.values()}
        self._build()
        self.ws_bytes = 0
        if split_k:
            self.ws_bytes = max([aqd.qconv_group_workspace([self._seg_args(c, si) for c, si in g])
                                 for g in self.schedule if g[0][0].op == "conv"], default=0)
        self.ws = (torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)
                   if self.ws_bytes else None)
        # independent launches (FPN side branches, the box prediction next to
        # the class prediction) run on side streams; each stream has its own
        # split-K workspace
        self.side = [torch.cuda.Stream(device=self.device) for _ in range(side_streams)]
        self.side_ws = [torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)
                        if self.ws_bytes else None for _ in self.side]
        self.deps, self.lane, self.signal = plan_streams(self.schedule, self.fused,
                                                         self._fused_away, len(self.side) + 1)
        self._calls = self._marshal()
        self.graph = None
        self.graph_stream = None

    # ---------------------------------------------------------------- setup
    def _fusable(self) -> dict:
        """conv name -> projection conv, for the pairs qconv_run_proj covers."""
        net = self.net
        producer, consumers = {}, {}
        for conv in net.convs:
            for x, skip, y in conv.segs:
                producer[y] = conv
                for src in (x, skip):
                    if src is not None:
                        consumers[src] = consumers.get(src, 0) + 1
        out = {}
        for conv in net.convs:
            if len(conv.segs) != 1:
                continue
            x, skip, y = conv.segs[0]
            if skip is None or net.tensors[skip].bits != 32 or conv.skip_up2:
                continue
            d = producer.get(skip)
            if d is None or len(d.segs) != 1 or d.k != 1 or consumers.get(skip) != 1:
                continue
            sb = aqd.stored_bits
            if (sb(net.tensors[x].bits) != 4 or sb(net.tensors[y].bits) != 4 or conv.cout % 256 or
                    sb(net.tensors[d.segs[0][0]].bits) != 4 or d.cin % 64 or conv.cin % 64):
                continue
            out[conv.name] = d
        return out

    def _marshal(self):
        """Per group, the C-ABI calls of one pass with their arguments
        converted once (the tensors never move): a forward pass then costs
        one foreign call per launch."""
        L = aqd.lib()
        wss = [self.ws] + self.side_ws
        calls = []
        for gi, group in enumerate(self.schedule):
            k = self.lane[gi]
            cs = []
            if k is not None and group[0][0].op == "maxpool":
                cs.append(self._pool_call(group[0][0]))
            elif k is not None:
                plain = [(c, si) for c, si in group
                         if c.name not in self._fused_away and c.name not in self.fused]
                if plain:
                    arr = aqd._seg_array([self._seg_args(conv, si) for conv, si in plain])
                    if wss[k] is not None:
                        cs.append((L.qconv_run_group_ws,
                                   (len(plain), arr, wss[k].data_ptr(), self.ws_bytes)))
                    else:
                        cs.append((L.qconv_run_group, (len(plain), arr)))
                for conv, si in group:
                    if conv.name in self.fused:
                        proj = self.fused[conv.name]
                        x, _, y = conv.segs[0]
                        xp = proj.segs[0][0]
                        tx, tp = self.net.tensors[x], self.net.tensors[xp]
                        cs.append((L.qconv_run_proj,
                                   (self.handles[conv.name], self.handles[proj.name], 0, tx.n, tx.h,
                                    tx.w, self.bufs[x].data_ptr(), tp.h, tp.w,
                                    self.bufs[xp].data_ptr(), self.bufs[y].data_ptr())))
            calls.append(cs)
        return calls

    def _pool_call(self, conv):
        """(function, arguments) of a max-pooling layer's launch; the
        descriptor is kept alive on the runner."""
        x, _, y = conv.segs[0]
        tx = self.net.tensors[x]
        d = aqd.MaxpoolDesc(tx.n, tx.h, tx.w, tx.c, tx.bits, conv.k, conv.stride, conv.pad)
        self._pool_descs.append(d)
        return (aqd.lib().aqd_maxpool_run, (aqd.ctypes.byref(d), self.bufs[x].data_ptr(),
                                            self.bufs[y].data_ptr()))

    def launches_per_forward(self) -> int:
        n = 0
        for group in self.schedule:
            plain = [c for c, _ in group if c.name not in self._fused_away and c.name not in self.fused]
            n += (1 if plain else 0) + sum(1 for c, _ in group if c.name in self.fused)
        return n

    def _make_schedule(self) -> List[List[Tuple[object, int]]]:
        producer = {}
        for conv in self.net.convs:
            for si, (_, _, y) in enumerate(conv.segs):
                producer[y] = conv.name
        depth = {}
        for conv in self.net.convs:
            d = 0
            for x, skip, _ in conv.segs:
                for src in (x, skip):
                    if src is not None and src in producer:
                        d = max(d, depth[producer[src]] + 1)
            depth[conv.name] = d
        groups: Dict[tuple, List[Tuple[object, int]]] = {}
        order = []
        for conv in self.net.convs:
            key = (depth[conv.name], _conv_key(self.net, conv))
            if key not in groups:
                groups[key] = []
                order.append(key)
            groups[key].extend((conv, si) for si in range(len(conv.segs)))
        sched = []
        for key in sorted(order, key=lambda k: (k[0], order.index(k))):
            segs = groups[key]
            for i in range(0, len(segs), aqd.MAX_SEGS):
                sched.append(segs[i:i + aqd.MAX_SEGS])
        return sched

    def _create(self, conv, levels, out_mode, bits_out, skip_bits, skip_up2):
        x, _, y = conv.segs[0]
        p = self.params
        return aqd.qconv_create(conv.cin, conv.cout, conv.k, conv.stride, conv.pad,
                                self.net.tensors[x].bits, conv.bits_w,
                                self._packed_weights(conv), levels, wenc=conv.wenc,
                                out_mode=out_mode, bits_out=bits_out, skip_bits=skip_bits,
                                skip_up2=skip_up2, step_in=p.alpha[x],
                                step_w=p.alpha_w[conv.name],
                                step_out=p.alpha[y] if out_mode == aqd.OUT_CODES else 0.0)

    def _packed_weights(self, conv):
        return aqd.pack_codes(self.params.weights[conv.name], conv.bits_w)

    def _seg_args(self, conv, si, level=None, images=None):
        x, skip, y = conv.segs[si]
        tx, ty = self.net.tensors[x], self.net.tensors[y]
        xb, yb = self.bufs[x], self.bufs[y]
        sb, hs, ws = None, 0, 0
        if skip is not None:
            ts = self.net.tensors[skip]
            sb, hs, ws = self.bufs[skip], ts.h, ts.w
        return (self.handles[conv.name], si if level is None else level, tx.n, tx.h, tx.w, xb, sb,
                hs, ws, yb)

    def _calibrate(self, conv, si, stats_handle) -> dict:
        """Integer epilogue of one segment from the statistics of its
        accumulator on the calibration images."""
        torch = self.torch
        p = self.params
        x, skip, y = conv.segs[si]
        tx, ty = self.net.tensors[x], self.net.tensors[y]
        ho, wo = ty.h, ty.w
        imgs = list(p.calib_images)
        assert imgs == list(range(imgs[0], imgs[0] + len(imgs))), "calibration images must be contiguous"
        img_bytes = self.bufs[x][0].numel() * self.bufs[x].element_size()
        xptr = self.bufs[x].data_ptr() + imgs[0] * img_bytes
        acc = torch.empty((len(imgs), ho, wo, conv.cout), dtype=torch.int32, device=self.device)
        sums = torch.zeros(2 * conv.cout, dtype=torch.int64, device=self.device)
        aqd.qconv_run(stats_handle, 0, len(imgs), tx.h, tx.w, xptr, None, 0, 0, acc,
                      self.stream)
        aqd.channel_sums(acc, len(imgs) * ho * wo, conv.cout, sums, self.stream)
        self.stream.synchronize()
        s = sums.cpu().numpy()
        alpha_conv, _ = aqd.qconv_scales(stats_handle)   # Eq. 4, from the handle's steps
        mean, var = aqd.bn_stats_from_sums(s[:conv.cout], s[conv.cout:], len(imgs) * ho * wo,
                                           alpha_conv)
        sp = p.segs[conv.name][si]
        bias, alpha_z = aqd.fold_bn(sp["gamma"], sp["beta"], mean, var, p.bn_eps, alpha_conv)
        t = {"bias": bias}
        if ty.bits == 32:
            self._alpha_t[y] = alpha_z
            return t
        scale = alpha_z
        if skip is not None:
            ak = self._alpha_t[skip] if self.net.tensors[skip].bits == 32 else p.alpha[skip]
            c, d, side, scale = aqd.skip_params(alpha_z, ak)
            t.update(skip_c=c, skip_d=d, skip_side=side)
        t["mult"], t["shift"] = aqd.requant_params(scale, p.alpha[y])
        return t

    def _build(self):
        """Derive every epilogue, create the handles, and run each layer once
        (later layers calibrate on the outputs of earlier ones)."""
        for conv in self.net.convs:
            x, skip, y = conv.segs[0]
            if conv.op == "maxpool":
                tx = self.net.tensors[x]
                self.tables[conv.name] = []
                aqd.maxpool_run(tx.n, tx.h, tx.w, tx.c, tx.bits, conv.k, conv.stride, conv.pad,
                                self.bufs[x], self.bufs[y], self.stream)
                continue
            ty = self.net.tensors[y]
            out_mode = aqd.OUT_INT32 if ty.bits == 32 else aqd.OUT_CODES
            bits_out = 0 if ty.bits == 32 else ty.bits
            skip_bits = self.net.tensors[skip].bits if skip else 0
            if self.params.mode == "literal":
                levels = [dict(s) for s in self.params.segs[conv.name]]
            else:
                zero = {"bias": np.zeros(conv.cout, np.int32)}
                stats = self._create(conv, [zero], aqd.OUT_INT32, 0, 0, 0)
                try:
                    levels = [self._calibrate(conv, si, stats) for si in range(len(conv.segs))]
                finally:
                    aqd.qconv_destroy(stats)
            self.tables[conv.name] = levels
            self.handles[conv.name] = self._create(conv, levels, out_mode, bits_out, skip_bits,
                                                   conv.skip_up2)
            aqd.qconv_run_group([self._seg_args(conv, si) for si in range(len(conv.segs))],
                                self.stream)
        self.stream.synchronize()

    # -------------------------------------------------------------- running
    def forward(self, stream=None, launch_hook=None, serial=False):
        """Enqueue the whole network on the stream. launch_hook(group_index,
        'before'|'after', stream) is called around each grouped launch (for
        timing). serial: every launch on the one stream, in schedule order
        (a topological order), so that no two launches overlap."""
        torch = self.torch
        main = self.stream if stream is None else stream
        streams = [main] + self.side
        done = {}          # group -> event recorded after its launch
        tail = {}          # side stream -> event after its last launch
        # side streams start after the work already enqueued on the main stream
        start = None
        if len(self.side) and not serial:
            start = torch.cuda.Event()
            start.record(main)
        started = set()
        for gi, group in enumerate(self.schedule):
            k = self.lane[gi]
            if k is None:
                continue
            if serial:
                k = 0
            s = streams[k]
            if k and k not in started:
                s.wait_event(start)
                started.add(k)
            for d in self.deps[gi] if not serial else ():
                if self.lane[d] is not None and self.lane[d] != k:
                    s.wait_event(done[d])
            if launch_hook:
                launch_hook(gi, "before", s)
            sh = s.cuda_stream
            for fn, args in self._calls[gi]:
                st = fn(*args, sh)
                if st != aqd.AQD_OK:
                    raise aqd.AqdError(st, aqd.last_error())
            if launch_hook:
                launch_hook(gi, "after", s)
            if gi in self.signal and not serial:
                ev = torch.cuda.Event()
                ev.record(s)
                done[gi] = ev
                if k:
                    tail[k] = ev
        # the pass ends on the main stream once every side stream is done
        for k in sorted(tail):
            main.wait_event(tail[k])

    def launch_group(self, gi, stream=None):
        """Enqueue grouped launch gi alone on the stream, on the tensors the
        last pass left (it rewrites its outputs with the same values): for
        timing one launch back to back."""
        s = self.stream if stream is None else stream
        for fn, args in self._calls[gi]:
            st = fn(*args, s.cuda_stream)
            if st != aqd.AQD_OK:
                raise aqd.AqdError(st, aqd.last_error())

    def capture(self, stream=None):
        """Record one forward pass on the (non-null) stream into a HIP graph;
        replay() then enqueues the whole network as one launch. The recorded
        pointers are this runner's buffers and workspace."""
        s = self.stream if stream is None else stream
        if self.graph is not None:
            aqd.graph_destroy(self.graph)
            self.graph = None
        aqd.graph_begin(s)
        try:
            self.forward(s)
        except Exception:
            try:
                aqd.graph_destroy(aqd.graph_end(s))
            except aqd.AqdError:
                pass
            raise
        self.graph = aqd.graph_end(s)
        self.graph_stream = s

    def replay(self, stream=None):
        assert self.graph is not None, "capture() first"
        aqd.graph_launch(self.graph, self.graph_stream if stream is None else stream)

    def group_macs(self, group) -> int:
        tot = 0
        for conv, si in group:
            if conv.op != "conv":
                continue
            t = self.net.tensors[conv.segs[si][2]]
            tot += t.n * t.h * t.w * conv.cout * conv.k * conv.k * conv.cin
        return tot

    def raw(self, name) -> np.ndarray:
        """Host copy of a tensor's device bytes (packed codes or int32)."""
        return self.bufs[name].cpu().numpy()

    def close(self):
        if getattr(self, "graph", None) is not None:
            self.torch.cuda.synchronize(self.device)   # no replay may be pending
            aqd.graph_destroy(self.graph)
            self.graph = None
        for h in self.handles.values():
            aqd.qconv_destroy(h)
        self.handles = {}

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
