"""End-to-end configuration sweep for the fused GEMM + tile-reduce call.

The paper picks the GEMM block shape, the reducer grid size x and its thread
count b by the lowest end-to-end latency under concurrent execution, with an
offline profiler (Section 3.2 "End-to-end optimization", Section 4.3).  This
module does the same on the device it runs on: for one workload it times the
fused call over a grid of (block shape, x, b, block walk) and records the
winner in ``tuned.json`` (read back by :func:`tuning.tuned_config`).  The
"layer" scope times the call with the residual addition and RMSNorm
(Section 5.2, layer-level performance), which runs as one launch only.

Timing follows the benchmark: synthetic seeded inputs resident on the device,
``warmup`` untimed calls, then ``steps`` calls whose wall time (host clock
around a synchronised batch) gives ms per call; the destination chunk cycles
through 0 .. P-1 in rank scope.  The engine clock drifts with power and
temperature, so the whole grid is timed ``passes`` times and each
configuration keeps its best pass.

    python -m paper_2609_11562_amd.tune --workload llama70b_attn_out_tp8 --write
"""
from __future__ import annotations

import argparse
import itertools
import json
import os
import statistics
import sys
import time

from . import entwine as E
from .inputs import bits_to_torch
from .tuning import _TABLE
from .workloads import WORKLOADS

DEFAULT_XS = (8, 12, 16, 24, 32, 48, 64)
DEFAULT_BS = (512, 1024)
DEFAULT_CFGS = (E.GEMM_256x256, E.GEMM_256x128, E.GEMM_128x256, E.GEMM_128x128)
DEFAULT_GROUP_M = (1, 4)


def _time_config(ctx, A, B, peers, partial, outs, P, scope, cfg, steps, warmup, gs, rs, layer=None):
    import torch

    def call(i):
        d = E.DEST_ALL if scope == "all" else i % P
        if scope == "layer":
            R, gamma, h, y = layer
            ctx.gemm_rs_rmsnorm(A, B, peers, d, R, gamma, 1e-5, h_out=h, y_out=y, partial=partial, cfg=cfg, stream=gs)
        else:
            ctx.gemm_rs(A, B, peers, d, out=outs[d], partial=partial, cfg=cfg, gemm_stream=gs, reduce_stream=rs)

    for i in range(warmup):
        call(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        call(i)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    st = ctx.query_status()
    if st[0] != E.OK:
        raise RuntimeError(f"reducer reported status {st}")
    e2e = statistics.median(ctx.last_timing(b)[2] for b in range(min(steps, 255)))
    return wall, e2e


def sweep(workload: str, scope: str = "rank", xs=DEFAULT_XS, bs=DEFAULT_BS, cfgs=DEFAULT_CFGS,
          group_ms=DEFAULT_GROUP_M, steps: int = 30, warmup: int = 10, launch: int = 0, release_blocks=(1,),
          passes: int = 2, log=None):
    """Time every valid configuration; returns (best, rows) where rows are
    dicts with the configuration, wall ms per call and median event time.
    With launch 0 (one kernel, reducers of 256 threads) b has no effect and
    is recorded as 256."""
    import torch

    if scope == "layer" and launch != 0:
        raise ValueError("the layer epilogue runs as one launch (launch 0)")
    w = WORKLOADS[workload]
    M, N, K, P = w.M, w.N, w.K, w.P
    prob = w.problem()
    A = bits_to_torch(prob.A).cuda()
    B = bits_to_torch(prob.B).cuda()
    peers = [bits_to_torch(p).cuda() for p in prob.peers]
    rows = {}
    with E.Context(M, N, K, P) as ctx:
        partial = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
        dests = [E.DEST_ALL] if scope == "all" else list(range(P))
        outs = {d: torch.empty(ctx.out_rows(d), N, dtype=torch.bfloat16, device="cuda") for d in dests}
        layer = None
        if scope == "layer":
            R, gamma = w.layer_inputs()
            layer = (bits_to_torch(R).cuda(), bits_to_torch(gamma).cuda(),
                     torch.empty(M // P, N, dtype=torch.bfloat16, device="cuda"),
                     torch.empty(M // P, N, dtype=torch.bfloat16, device="cuda"))
        gs = torch.cuda.current_stream()
        rs = torch.cuda.Stream()
        # the single launch's reducers are its own 256-thread workgroups
        grid = list(itertools.product(cfgs, xs, (256,) if launch == 0 else bs, group_ms, release_blocks))
        for _ in range(passes):
            for gc, x, b, gm, g in grid:
                kw = dict(gemm_cfg=gc, reduce_wgs=x, reduce_threads=b, group_m=gm, launch=launch, release_blocks=g,
                          record_timing=1)
                cfg = E.Config.make(**kw)
                if E.validate(M, N, K, P, E.DEST_ALL if scope == "all" else 0, cfg) != E.OK:
                    continue   # e.g. a block that does not divide the chunk, or x = -1 with two streams
                wall, e2e = _time_config(ctx, A, B, peers, partial, outs, P, scope, cfg, steps, warmup, gs, rs, layer)
                row = {k: v for k, v in kw.items() if k != "record_timing"}
                row.update(order=E.ORDER_INTERLEAVED, wall_ms=round(wall, 5), event_ms=round(e2e, 5),
                           tflops=round(2.0 * M * N * K / (wall * 1e-3) / 1e12, 1))
                key = (gc, x, b, gm, g)
                if key not in rows or row["wall_ms"] < rows[key]["wall_ms"]:
                    rows[key] = row
                if log:
                    log(json.dumps(row))
    best = min(rows.values(), key=lambda r: r["wall_ms"])
    return best, list(rows.values())


def write_entry(workload: str, scope: str, best: dict, path: str = _TABLE) -> None:
    table = {}
    if os.path.exists(path):
        with open(path) as f:
            table = json.load(f)
    keep = ("order", "gemm_cfg", "reduce_wgs", "reduce_threads", "group_m", "launch", "release_blocks")
    table.setdefault(workload, {})[scope] = {k: best[k] for k in keep}
    table[workload][scope]["measured_ms"] = best["wall_ms"]
    with open(path, "w") as f:
        json.dump(table, f, indent=1, sort_keys=True)
        f.write("\n")


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workload", action="append", required=True)
    ap.add_argument("--scope", default="rank", choices=["rank", "all", "layer"],
                    help="rank = one chunk, all = every chunk, layer = one chunk + residual addition + RMSNorm")
    ap.add_argument("--xs", default=",".join(map(str, DEFAULT_XS)))
    ap.add_argument("--bs", default=",".join(map(str, DEFAULT_BS)))
    ap.add_argument("--cfgs", default=",".join(map(str, DEFAULT_CFGS)))
    ap.add_argument("--group-m", default=",".join(map(str, DEFAULT_GROUP_M)))
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--launch", type=int, default=0, help="0 = one kernel launch, 1 = two streams, 2 = shared pool")
    ap.add_argument("--release-blocks", default="1", help="release granularities g to try (-1 = once per workgroup)")
    ap.add_argument("--passes", type=int, default=2, help="times the grid is timed; each configuration keeps its best")
    ap.add_argument("--write", action="store_true", help="record the winners in the table")
    ap.add_argument("--table", default=_TABLE, help="JSON table to update (default: the package's tuned.json)")
    a = ap.parse_args(argv)
    ints = lambda s: tuple(int(v) for v in s.split(","))
    for wl in a.workload:
        best, _ = sweep(wl, a.scope, ints(a.xs), ints(a.bs), ints(a.cfgs), ints(a.group_m), a.steps, a.warmup,
                        a.launch, ints(a.release_blocks), a.passes, log=lambda s: print(s, flush=True))
        print(json.dumps({"workload": wl, "scope": a.scope, "best": best}), flush=True)
        if a.write:
            write_entry(wl, a.scope, best, a.table)


if __name__ == "__main__":
    sys.exit(main())
