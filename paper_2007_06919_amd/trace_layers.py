"""Per-layer durations from a rocprofv3 kernel trace of bench.py.

The runner issues its grouped launches in schedule order, so the last
len(schedule) convolution dispatches of a trace are one forward pass; this
maps them to layer names and prints duration, share and integer TOPS.

usage: python -m paper_2007_06919_amd.trace_layers <kernel_trace.csv> [workload] [top]
"""
import csv
import sys
import types

from . import runner, workloads


def layer_table(trace_csv, workload=4, top=30):
    net, _ = workloads.config(workload)
    sched = runner.Net._make_schedule(types.SimpleNamespace(net=net))
    rows = [r for r in csv.DictReader(open(trace_csv))
            if "qconv_mfma" in r["Kernel_Name"] or "qconv_direct" in r["Kernel_Name"]]
    last = rows[-len(sched):]
    out, tot = [], 0.0
    for g, r in zip(sched, last):
        us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        macs = sum(net.tensors[c.segs[si][2]].n * net.tensors[c.segs[si][2]].h *
                   net.tensors[c.segs[si][2]].w * c.cout * c.k * c.k * c.cin for c, si in g)
        c = g[0][0]
        name = c.name + (f"+{len(g) - 1}seg" if len(g) > 1 else "")
        out.append((us, name, f"{c.k}x{c.k}s{c.stride} {c.cin}->{c.cout}",
                    int(r["Grid_Size_X"]) // int(r["Workgroup_Size_X"]), 2 * macs / (us * 1e-6) / 1e12))
        tot += us
    lines = [f"total {tot / 1e3:.3f} ms over {len(sched)} launches"]
    for us, name, shape, wg, tops in sorted(out, reverse=True)[:top]:
        lines.append(f"{us:8.1f} us {100 * us / tot:5.1f}%  {name:22s} {shape:18s} wg={wg:6d} "
                     f"{tops:7.1f} TOPS")
    return "\n".join(lines)


if __name__ == "__main__":
    print(layer_table(sys.argv[1], int(sys.argv[2]) if len(sys.argv) > 2 else 4,
                      int(sys.argv[3]) if len(sys.argv) > 3 else 30))
