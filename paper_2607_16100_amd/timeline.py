"""Phase timeline of the one-shot and two-shot AllReduce with one wave per peer.

Run with the diagnostic build of the library, whose wave kernels record phase
times (``python -m paper_2607_16100_amd.build --phases``):

    LLCOLL_LIBRARY=paper_2607_16100_amd/libllcoll_phases.so \\
        python -m paper_2607_16100_amd.timeline [--twoshot] [--calls 300] [--json out.jsonl]

For each case, `calls` back-to-back calls are queued behind a spin kernel and
each records, from the 100 MHz constant clock, every workgroup's start and end
and, for lane 0 of every wave, its phase times.  One-shot (8 ranks, bfloat16,
128 bytes and 16 KiB per rank, every packet format): its packet store issued,
its peer's packets all seen, past the workgroup barrier.  Two-shot
(``--twoshot``: 8 ranks, bfloat16, 1 MiB per rank, every packet format; the
first tile of each workgroup): its ReduceScatter packets issued, its peer's
ReduceScatter packets seen, past the barrier, its peer's AllGather packets
seen.  The table gives microseconds from the call's first workgroup start, as
the median over calls of the median over waves (max over the grid in
brackets), plus the median call-to-call interval.  The stamps themselves add
about 0.1 us.
"""
from __future__ import annotations

import argparse
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

TICK_US = 0.01
PHASES = ("store issued", "peer's packets seen", "past the barrier")
PHASES_TWOSHOT = ("RS packets issued", "peer's RS packets seen", "past the barrier", "peer's AG packets seen")


def run_case(p: int, n: int, dtype: str, algo: str, calls: int, phases=PHASES):
    import torch

    from paper_2607_16100_amd import llcoll as ll
    from paper_2607_16100_amd import workloads as wl
    from paper_2607_16100_amd.region import SymRegion

    x = wl.normal(p, n, dtype, seed=0)
    reg = SymRegion(p, n, dtype)
    reg.init()
    reg.write_inputs(x)
    s = reg.stream_handle()
    shape = ll.Options(report=True)
    for _ in range(50):
        ll.check(reg.allreduce(n, algo, opt=shape))
    torch.cuda.synchronize()
    grid, threads = shape.grid, shape.threads
    waves = grid * (threads // 64)
    st = torch.zeros(calls, 2 * grid, dtype=torch.int64, device="cuda")
    ph = torch.zeros(calls, 4 * waves, dtype=torch.int64, device="cuda")
    opts = [ll.Options(stamps=st[c].data_ptr(), phases=ph[c].data_ptr()) for c in range(calls)]
    ll.check(ll.ll_probe_spin(3_000_000, s))
    for c in range(calls):
        ll.check(reg.allreduce(n, algo, opt=opts[c]))
    torch.cuda.synchronize()
    ll.check(ll.ll_check(s))
    st = st.cpu().numpy()
    ph = ph.cpu().numpy().reshape(calls, waves, 4)
    t0 = st[:, :grid].min(axis=1)
    ends = st[:, grid:].max(axis=1)

    def med_max(a):  # a: [calls, k] times relative to t0, in us
        return round(float(np.median(np.median(a, axis=1))), 3), round(float(np.median(np.max(a, axis=1))), 3)

    rel = lambda a: (a - t0[:, None]) * TICK_US  # noqa: E731
    row = {"ranks": p, "bytes_per_rank": n * (2 if dtype == "bf16" else 4), "dtype": dtype, "algo": algo,
           "grid": grid, "threads": threads, "interval_p50_us": round(float(np.median(np.diff(ends))) * TICK_US, 3),
           "span_p50_us": round(float(np.median(ends - t0)) * TICK_US, 3), "workgroup_start": med_max(rel(st[:, :grid]))}
    for k, name in enumerate(phases):
        a = ph[:, :, k]
        ok = a[0] != 0
        if ok.any():
            row[name] = med_max(rel(a[:, ok]))
    row["workgroup_end"] = med_max(rel(st[:, grid:]))
    return row


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--calls", type=int, default=300)
    ap.add_argument("--json", default="")
    ap.add_argument("--twoshot", action="store_true")
    args = ap.parse_args()
    import torch

    torch.cuda.set_device(0)
    rows = []
    if args.twoshot:
        phases = PHASES_TWOSHOT
        cases = [(64 * 8192, a) for a in ("twoshot_line_waves", "twoshot_sentinel_waves", "twoshot_waves")]
    else:
        phases = PHASES
        cases = [(n, a) for n in (64, 8192) for a in ("oneshot_waves", "oneshot_line_waves", "oneshot_sentinel_waves")]
    for n, algo in cases:
        rows.append(run_case(8, n, "bf16", algo, args.calls, phases))
        print(json.dumps(rows[-1]), file=sys.stderr, flush=True)
    if args.json:
        with open(args.json, "w") as f:
            for r in rows:
                f.write(json.dumps(r) + "\n")
    keys = ["workgroup_start", *phases, "workgroup_end"]
    print("| phase (us from the first workgroup start) | " +
          " | ".join(f"{r['algo']} {r['bytes_per_rank']} B" for r in rows) + " |")
    print("|---|" + "---:|" * len(rows))
    print("| workgroups | " + " | ".join(str(r["grid"]) for r in rows) + " |")
    for k in keys:
        print(f"| {k.replace('_', ' ')} | " +
              " | ".join(f"{r[k][0]:.2f} ({r[k][1]:.2f})" if k in r else "-" for r in rows) + " |")
    print("| call-to-call interval, p50 | " + " | ".join(f"{r['interval_p50_us']:.2f}" for r in rows) + " |")


if __name__ == "__main__":
    main()
