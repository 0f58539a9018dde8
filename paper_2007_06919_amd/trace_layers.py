"""Per-launch durations from a rocprofv3 kernel trace of bench.py.

The runner issues its launches in a fixed order (grouped convolutions, fused
projection shortcuts, split-K convolutions followed by their combining
kernel); this rebuilds that order for the workload, maps the trace's last
forward passes onto it and prints, per launch, the median duration over
those passes, its share and its integer TOPS (the fused launches count the
shortcut's MACs too).

usage: python -m paper_2007_06919_amd.trace_layers <kernel_trace.csv> [workload] [top] [passes]
workload: a workload number, or io8 for the fully quantized RetinaNet-R50
(batch 8, 800x1333, 8-bit image, stem, pooling and predictions).
"""
import csv
import sys
import types

from . import runner, workloads


def launch_list(net):
    """[(name, convs, macs)] in the runner's launch order."""
    o = types.SimpleNamespace(net=net)
    sched = runner.Net._make_schedule(o)
    fused = runner.Net._fusable(o)
    away = {d.name for d in fused.values()}

    def macs(c, si):
        if c.op != "conv":
            return 0
        t = net.tensors[c.segs[si][2]]
        return t.n * t.h * t.w * c.cout * c.k * c.k * c.cin

    out = []
    for g in sched:
        plain = [(c, si) for c, si in g if c.name not in away and c.name not in fused]
        if plain:
            c = plain[0][0]
            out.append((c.name + (f"+{len(plain) - 1}seg" if len(plain) > 1 else ""), c,
                        sum(macs(cc, si) for cc, si in plain)))
        for c, si in g:
            if c.name in fused:
                d = fused[c.name]
                out.append((c.name + "+" + d.name.split(".")[-1], c, macs(c, si) + macs(d, 0)))
    return out


def layer_table(trace_csv, workload=4, top=30, passes=5):
    if workload == "io8":
        net = workloads.retinanet_r50_net(8, 800, 1333, 4, io_bits=8)
    else:
        net, _ = workloads.config(int(workload))
    launches = launch_list(net)
    rows = sorted((r for r in csv.DictReader(open(trace_csv))
                   if any(k in r["Kernel_Name"] for k in ("qconv_", "splitk_", "maxpool"))),
                  key=lambda r: int(r["Dispatch_Id"]))  # enqueue order (launches on several streams overlap)
    # one entry per launch; a combining kernel belongs to the launch before it
    seq = []
    for r in rows:
        us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        if "splitk" in r["Kernel_Name"] and seq:
            seq[-1][0] += us
            seq[-1][2] = True
        else:
            seq.append([us, int(r["Grid_Size_X"]) // int(r["Workgroup_Size_X"]), False])
    n = len(launches)
    passes = min(passes, len(seq) // n)
    seq = seq[len(seq) - passes * n:]
    out, tot = [], 0.0
    for k, (name, c, macs) in enumerate(launches):
        ts = sorted(seq[p * n + k][0] for p in range(passes))
        us = ts[len(ts) // 2]
        wg, split = seq[k][1], seq[k][2]
        out.append((us, name + (" (split K)" if split else ""),
                    f"{c.k}x{c.k}s{c.stride} {c.cin}->{c.cout}", wg, 2 * macs / (us * 1e-6) / 1e12))
        tot += us
    lines = [f"total {tot / 1e3:.3f} ms over {n} launches (median of {passes} passes)"]
    for us, name, shape, wg, tops in sorted(out, reverse=True)[:top]:
        lines.append(f"{us:8.1f} us {100 * us / tot:5.1f}%  {name:30s} {shape:18s} wg={wg:6d} "
                     f"{tops:7.1f} TOPS")
    return "\n".join(lines)


if __name__ == "__main__":
    print(layer_table(sys.argv[1], sys.argv[2] if len(sys.argv) > 2 else 4,
                      int(sys.argv[3]) if len(sys.argv) > 3 else 30,
                      int(sys.argv[4]) if len(sys.argv) > 4 else 5))
