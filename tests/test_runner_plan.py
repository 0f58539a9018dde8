"""Host logic of the runner's stream plan (no GPU): dependencies come from
the tensors each launch reads; every cross-stream dependency and every side
stream's last launch records an event; the plan keeps the backbone chain on
the main stream and moves independent FPN branches and the box prediction to
side streams."""
import types

from paper_2007_06919_amd import runner, workloads


def _plan(cfg, nstreams, scaled=None):
    net, _ = workloads.scaled_config(*scaled) if scaled else workloads.config(cfg)
    o = types.SimpleNamespace(net=net)
    sched = runner.Net._make_schedule(o)
    fused = runner.Net._fusable(o)
    away = {d.name for d in fused.values()}
    return net, sched, fused, away, runner.plan_streams(sched, fused, away, nstreams)


def test_plan_invariants():
    net, sched, fused, away, (deps, lane, signal) = _plan(4, 3)
    names = [g[0][0].name for g in sched]
    for gi, ds in enumerate(deps):
        assert all(d < gi for d in ds), names[gi]
        if lane[gi] is None:
            assert all(c.name in away for c, _ in sched[gi])
            continue
        for d in ds:
            assert lane[d] is not None, (names[gi], names[d])
            if lane[d] != lane[gi]:
                assert d in signal, (names[gi], names[d])
    for k in (1, 2):
        mine = [gi for gi, l in enumerate(lane) if l == k]
        assert mine and mine[-1] in signal
    # every tensor a launch reads is produced earlier in the pass or is an input
    produced = {c.segs[si][2] for g in sched for c, si in g if c.name not in away}
    for gi, g in enumerate(sched):
        for t in runner.group_inputs(g, fused, away):
            assert t in produced or t in net.inputs, (names[gi], t)


def test_plan_places_independent_branches_on_side_streams():
    _, sched, _, _, (deps, lane, _) = _plan(4, 3)
    by = {g[0][0].name: gi for gi, g in enumerate(sched)}
    main_chain = ["res2.0.conv1", "res3.1.conv2", "res5.2.conv3", "fpn.lat5", "fpn.lat4",
                  "fpn.lat3", "fpn.out3", "cls.t1", "cls.t4", "cls.pred"]
    assert all(lane[by[n]] == 0 for n in main_chain)
    assert all(lane[by[n]] != 0 for n in ("fpn.p6", "fpn.p7", "fpn.out4", "fpn.out5", "box.pred"))
    assert lane[by["fpn.p7"]] == lane[by["fpn.p6"]]          # continues its producer's stream
    assert by["cls.t4"] in deps[by["box.pred"]]


def test_plan_single_stream():
    _, sched, _, _, (deps, lane, signal) = _plan(4, 1)
    assert all(l in (0, None) for l in lane) and not signal


def test_plan_scaled_and_small_networks():
    for scaled in ((2, 1, 320, 448), (3, 1, 256, 384), (4, 2, 192, 256)):
        _, sched, _, _, (deps, lane, signal) = _plan(None, 3, scaled)
        assert lane[0] == 0
    _, sched, _, _, (deps, lane, signal) = _plan(1, 3)
    assert all(l == 0 for l in lane if l is not None)
