"""Phase times of the fused step's kernels from the instrumented build.

libewsjf_stamps.so (python -m paper_2601_21758_amd.build --stamps) records,
in thread 0 of each streaming workgroup and each merge workgroup, the
device's 100 MHz constant clock at numbered points of the kernel.  This
script runs the step on one of the pools (`--config`: 0 the 4,096-request
pool, 1 the 262,144-request pool, 2 (default) the large mixed pool of
4,194,304 requests with the 256-queue partition of its 1,048,576-length
window and B = 1,024), rotating over independent draws of it, in bursts of back-to-back steps (the stamps are the last step's),
and prints, per kernel and point, the median over steps of the median and
the maximum over workgroups, in microseconds after the kernel's first
workgroup started ("median_us", "max_us") and after the workgroup's own
start ("own_median_us", "own_max_us"), and the median start of each XCD's
workgroups (block index mod 8).

Points:
  local_candidates  0 start, 1 table staged (first barrier), 2 wave 0 done
                    with the pool, 3 every wave done with the pool, 4 list
                    filtered, 5 list published; 6 is not a time but the
                    length of the filtered list (entries at or above the
                    workgroup's bound), reported as "list_length"
  merge_rank        0 start, 1 slots and bounds in (first barrier), 2 own
                    slots counted, 3 merge found safe, 4 outputs written, 7
                    took the exact merge
  merge_exact       0 start, 1 cut and order done, 2 published
"""
from __future__ import annotations

import argparse
import ctypes as C
import json
import os
import sys

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
KERNELS = ("local_candidates", "merge_rank", "merge_exact", "local_candidates_multi")
BLOCKS, PHASES = 256, 8
TICK_US = 0.01  # 100 MHz


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--config", type=int, default=2, choices=(0, 1, 2))
    ap.add_argument("--rotate", type=int, default=10)
    ap.add_argument("--lib", default=os.path.join(PKG, "libewsjf_stamps.so"),
                    help="an instrumented build of the library (default: the package's)")
    ap.add_argument("--burst", type=int, default=8,
                    help="steps run back to back per sample; the stamps are the last step's")
    args = ap.parse_args()
    sys.path.insert(0, ROOT)
    from paper_2601_21758_amd import _lib as L
    path = os.path.abspath(args.lib)
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built (python -m paper_2601_21758_amd.build --stamps)")
    L.LIB_PATH = path
    import torch

    from paper_2601_21758_amd import ewsjf as E
    from paper_2601_21758_amd import workloads as W
    lib = L.lib()
    lib.ewsjf_debug_stamps.argtypes = [C.c_void_p, C.c_size_t]
    lib.ewsjf_debug_stamps_clear.argtypes = []
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    pools = [W.config(args.config, draw=r) for r in range(args.rotate)]
    pool = pools[0]
    lens = [torch.from_numpy(p.length).to(dev) for p in pools]
    arrs = [torch.from_numpy(p.arrival).to(dev) for p in pools]
    nows = [float(p.now) for p in pools]
    theta = torch.from_numpy(pool.theta).to(dev)
    table = E.partition(torch.from_numpy(pool.window).to(dev),
                        E.params(init_queues=pool.init_queues, max_queues=pool.max_queues))
    ws = E.Workspace(dev)
    out = E._outs(1, pool.B, dev, None)
    for i in range(5):
        r = i % args.rotate
        E.step(lens[r], arrs[r], nows[r], table, theta, pool.B, pool.cost, out=out, ws=ws)
    torch.cuda.synchronize()
    host = np.zeros(len(KERNELS) * BLOCKS * PHASES, np.uint64)
    per = {k: [] for k in KERNELS}
    for i in range(args.steps):
        assert lib.ewsjf_debug_stamps_clear() == 0
        torch.cuda.synchronize()
        torch.cuda._sleep(int(2.4e9 * 1e-3))  # hold the stream while the burst is enqueued
        for j in range(args.burst):
            r = (i * args.burst + j) % args.rotate
            E.step(lens[r], arrs[r], nows[r], table, theta, pool.B, pool.cost, out=out, ws=ws)
        torch.cuda.synchronize()
        assert lib.ewsjf_debug_stamps(host.ctypes.data, host.size) == 0
        st = host.reshape(len(KERNELS), BLOCKS, PHASES).astype(np.int64)
        for ki, k in enumerate(KERNELS):
            s = st[ki]
            used = s[:, 0] != 0
            if not used.any():
                continue
            t0 = s[used, 0].min()
            row = {}
            if k == "local_candidates":
                row["list_length"] = s[used, 6].copy()
            for ph in [q for q in range(PHASES) if not (k == "local_candidates" and q == 6)]:
                sel = s[:, ph] != 0
                if sel.any():
                    # after the first workgroup's start, and after the workgroup's own start
                    own = sel & used
                    row[ph] = ((s[sel, ph] - t0) * TICK_US, int(sel.sum()), (s[own, ph] - s[own, 0]) * TICK_US)
            # start of each XCD's workgroups (block index mod 8) after the first start
            xcd = {str(x): float(np.median((s[x::8, 0][s[x::8, 0] != 0] - t0) * TICK_US)) for x in range(8)
                   if (s[x::8, 0] != 0).any()}
            row["xcd_start"] = xcd
            per[k].append(row)
    report = {}
    for k, rows in per.items():
        if not rows:
            continue
        phases = sorted({ph for r in rows for ph in r if ph not in ("xcd_start", "list_length")})
        rep = {}
        for ph in phases:
            med = [float(np.median(r[ph][0])) for r in rows if ph in r]
            mx = [float(np.max(r[ph][0])) for r in rows if ph in r]
            own = [float(np.median(r[ph][2])) for r in rows if ph in r and r[ph][2].size]
            own_mx = [float(np.max(r[ph][2])) for r in rows if ph in r and r[ph][2].size]
            cnt = [r[ph][1] for r in rows if ph in r]
            rep[str(ph)] = {"median_us": round(float(np.median(med)), 3), "max_us": round(float(np.median(mx)), 3),
                            "own_median_us": round(float(np.median(own)), 3) if own else None,
                            "own_max_us": round(float(np.median(own_mx)), 3) if own_mx else None,
                            "workgroups": int(np.median(cnt)), "steps": len(med)}
        xs = sorted({x for r in rows for x in r["xcd_start"]})
        rep["xcd_start_us"] = {x: round(float(np.median([r["xcd_start"][x] for r in rows if x in r["xcd_start"]])), 3)
                               for x in xs}
        if k == "local_candidates":
            ll = np.concatenate([r["list_length"] for r in rows])
            rep["list_length"] = {"p10": float(np.percentile(ll, 10)), "p50": float(np.median(ll)),
                                  "p90": float(np.percentile(ll, 90)), "max": float(ll.max())}
        report[k] = rep
    print(json.dumps({"workload": f"{pool.name} step, B={pool.B}, {args.rotate} pool draws", "steps": args.steps, "phases": report}, indent=1),
          flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
