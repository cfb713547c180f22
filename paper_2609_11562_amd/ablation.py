"""Mechanism ablations of the fused GEMM + tile-reduce call on one device.

Each study changes one policy and keeps the workload, block shape, data path
and consumer task order fixed; where a policy has a communication budget (the
reducer workgroup count x), every budget in the list is timed and the
policy's lowest end-to-end latency is reported, as the paper does for its
ablations (Section 5.3):

* ``order``   computation order (Section 5.3.1, Figure 6a): Equation 1's
              interleaved order against the M-major traversal and the
              partition-contiguous row-major order, K in {512, 2048}.
* ``pool``    resource sharing (Section 5.3.2, Figure 6b): reducers on a
              static share of the CUs (two kernels on two streams, each
              reducer resident until the GEMM ends) against the shared pool
              (reducers beside the producer on every CU) and the single
              launch (producers become reducers when their blocks are done).
* ``release`` release granularity (Section 5.3.2, Figure 6c): one-tile
              reduction tasks (128 x 128 blocks, the two-stream form) with
              tiles published after every g blocks of a workgroup, once per
              workgroup, per row partition or for the whole output; K in
              {2048, 4096, 8192}.
* ``budget``  the communication-budget sweep (Appendix B): GEMM window, tail
              and end-to-end latency against x for eight values of K.
* ``range``   the operating range (Section 5.4.1): both workload suites of
              Table 1, each with its GEMM wave count (256 x 256 producer
              blocks per CU), the single launch at its best budget and the
              non-overlapped baseline.
* ``clock``   what bounds the producer on this device: the single launch on
              the three LLM shapes with the seeded operands, with A = 0 and
              with A = B = 1 (the same instructions, cycles and bytes; only
              the switching activity of the matrix cores differs), each with
              the engine clock the producers ran at.

M = N = 8192 and P = 8 throughout, except in ``range``.  Every row reports the wall-clock latency
per call (median over rounds of ``steps`` calls), the producer's window and
the tail from the call's own event / device timestamps, and the speedup over
the non-overlapped baseline (GEMM, then reduction with the whole device, on
one stream).

    python -m paper_2609_11562_amd.ablation release --out results.jsonl
"""
from __future__ import annotations

import argparse
import json
import statistics
import sys
import time

from . import entwine as E
from .inputs import bits_to_torch
from .workloads import SUITES, WORKLOADS, _llm

M_ABL, N_ABL, P_ABL = 8192, 8192, 8
BUDGETS = (4, 8, 16, 24, 32, 48, 64)
SEQ_BUDGETS = (64, 128, 255)


def workload(K: int):
    name = f"sweep_8192x{K}x8192_p8"
    return WORKLOADS.get(name) or _llm(name, M_ABL, K, N_ABL, P_ABL, "ablation shape")


class Bench:
    """Inputs of one workload resident on the device, and a timer."""

    def __init__(self, w, steps: int, warmup: int, rounds: int):
        import torch
        self.w, self.steps, self.warmup, self.rounds = w, steps, warmup, rounds
        prob = w.problem()
        self.A = bits_to_torch(prob.A).cuda()
        self.B = bits_to_torch(prob.B).cuda()
        self.peers = [bits_to_torch(p).cuda() for p in prob.peers]
        self.ctx = E.Context(w.M, w.N, w.K, w.P)
        self.partial = torch.empty(w.M, w.N, dtype=torch.bfloat16, device="cuda")
        self.out = torch.empty(w.M // w.P, w.N, dtype=torch.bfloat16, device="cuda")
        self.gs = torch.cuda.current_stream()
        self.rs = torch.cuda.Stream()

    def close(self):
        import torch
        self.ctx.close()
        del self.A, self.B, self.peers, self.partial, self.out
        torch.cuda.empty_cache()

    def time(self, sequential: bool = False, **kw) -> dict | None:
        """Median wall ms per call over the rounds, and the median producer
        window and end-to-end time of the calls' own timing; None if the
        configuration is not valid for the shape."""
        import torch
        cfg = E.Config.make(record_timing=1, **kw)
        w = self.w
        if E.validate(w.M, w.N, w.K, w.P, 0, cfg) != E.OK:
            return None
        rs = self.gs if sequential else self.rs

        def call(i):
            self.ctx.gemm_rs(self.A, self.B, self.peers, i % w.P, out=self.out, partial=self.partial, cfg=cfg,
                             gemm_stream=self.gs, reduce_stream=rs)

        walls, gemm, e2e, clk = [], [], [], []
        for _ in range(self.rounds):
            for i in range(self.warmup):
                call(i)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for i in range(self.steps):
                call(i)
            torch.cuda.synchronize()
            walls.append((time.perf_counter() - t0) * 1e3 / self.steps)
            st = self.ctx.query_status()
            if st[0] != E.OK:
                raise RuntimeError(f"status {st} for {kw}")
            for b in range(min(self.steps, 255)):
                g, _, e = self.ctx.last_timing(b)
                gemm.append(g)
                e2e.append(e)
                if cfg.launch == 0:
                    clk.append(self.ctx.last_clock(b))
        T = statistics.median(walls)
        G, Ee = statistics.median(gemm), statistics.median(e2e)
        out = {"ms": round(T, 5), "gemm_window_ms": round(G, 5), "e2e_event_ms": round(Ee, 5),
               "tail_ms": round(max(0.0, Ee - G), 5), "tflops": round(w.flops / (T * 1e-3) / 1e12, 1)}
        if clk:
            out["clock_ghz"] = round(statistics.median(clk), 3)
        return out


def best_over_budgets(bench: Bench, budgets, **kw):
    rows = []
    for x in budgets:
        r = bench.time(reduce_wgs=x, **kw)
        if r:
            rows.append(dict(r, reduce_wgs=x))
    return min(rows, key=lambda r: r["ms"]) if rows else None, rows


def baseline(bench: Bench, **kw) -> dict:
    """The non-overlapped baseline: the same kernels, GEMM then reduction on
    one stream (the two-stream form's kernels), the reduction given the
    budget that makes it fastest once it has the device to itself."""
    rows = [bench.time(sequential=True, launch=1, reduce_wgs=x, **kw) for x in SEQ_BUDGETS]
    return min((r for r in rows if r), key=lambda r: r["ms"])


def study_order(ks, budgets, emit, **tk):
    for K in ks:
        b = Bench(workload(K), **tk)
        base = baseline(b)
        for name, order in (("interleaved", E.ORDER_INTERLEAVED), ("m_major", E.ORDER_M_MAJOR),
                            ("row_major", E.ORDER_ROW_MAJOR)):
            for launch in (1, 0):
                best, _ = best_over_budgets(b, budgets, order=order, launch=launch, group_m=1)
                emit({"study": "order", "K": K, "order": name, "launch": launch, "group_m": 1, **best,
                      "baseline_ms": base["ms"], "speedup": round(base["ms"] / best["ms"], 3)})
        b.close()


def study_pool(ks, budgets, emit, **tk):
    for K in ks:
        b = Bench(workload(K), **tk)
        base = baseline(b)
        for name, launch, xs in (("static_partition", 1, budgets), ("shared_pool", 2, budgets + (256,)),
                                 ("single_launch", 0, budgets + (-1,))):
            best, _ = best_over_budgets(b, xs, launch=launch)
            emit({"study": "pool", "K": K, "policy": name, "launch": launch, **best,
                  "baseline_ms": base["ms"], "speedup": round(base["ms"] / best["ms"], 3)})
        b.close()


def study_release(ks, budgets, emit, **tk):
    groups = ((1, "1 block (1 tile)"), (2, "2 blocks"), (4, "4 blocks"), (8, "8 blocks"), (16, "16 blocks"),
              (E.RELEASE_AT_END, "once per workgroup"), (E.RELEASE_PARTITION, "row partition"),
              (E.RELEASE_OUTPUT, "whole output"))
    for K in ks:
        b = Bench(workload(K), **tk)
        base = baseline(b, gemm_cfg=E.GEMM_128x128)
        for g, name in groups:
            best, _ = best_over_budgets(b, budgets, launch=1, gemm_cfg=E.GEMM_128x128, release_blocks=g,
                                        reduce_threads=512)
            emit({"study": "release", "K": K, "release_blocks": g, "group": name, "launch": 1, "gemm_cfg": 3,
                  **best, "baseline_ms": base["ms"], "speedup": round(base["ms"] / best["ms"], 3)})
        b.close()


def study_budget(ks, budgets, emit, **tk):
    for K in ks:
        b = Bench(workload(K), **tk)
        base = baseline(b)
        for launch, xs in ((1, budgets), (0, (-1,) + budgets)):
            for x in xs:
                r = b.time(launch=launch, reduce_wgs=x)
                if r:
                    emit({"study": "budget", "K": K, "launch": launch, "reduce_wgs": x, **r,
                          "baseline_ms": base["ms"], "speedup": round(base["ms"] / r["ms"], 3)})
        b.close()


def study_range(ks, budgets, emit, **tk):
    """ks: unused (the suites fix K)."""
    del ks
    for suite in ("models", "main"):
        for name in SUITES[suite]:
            w = WORKLOADS[name]
            b = Bench(w, **tk)
            base = baseline(b)
            best, _ = best_over_budgets(b, (-1,) + tuple(x for x in budgets if x in (16, 32)), release_blocks=2)
            waves = (w.M // 256) * (w.N // 256) / 256.0
            emit({"study": "range", "suite": suite, "workload": name, "M": w.M, "N": w.N, "K": w.K, "waves": waves,
                  **best, "baseline_gemm_ms": base["gemm_window_ms"], "baseline_ms": base["ms"],
                  "speedup": round(base["ms"] / best["ms"], 3)})
            b.close()


def study_clock(ks, budgets, emit, **tk):
    """ks, budgets: unused (the LLM shapes and the default single launch)."""
    del ks, budgets
    for name in ("llama7b_mlp_down_tp8", "llama70b_attn_out_tp8", "llama70b_mlp_down_tp8"):
        b = Bench(WORKLOADS[name], **tk)
        A0, B0 = b.A.clone(), b.B.clone()
        for data in ("seeded", "a_zero", "ones", "seeded"):
            b.A.copy_(A0)
            b.B.copy_(B0)
            if data == "a_zero":
                b.A.zero_()
            elif data == "ones":
                b.A.fill_(1.0)
                b.B.fill_(1.0)
            r = b.time(launch=0)
            emit({"study": "clock", "workload": name, "data": data, **r})
        del A0, B0
        b.close()


STUDIES = {"clock": (study_clock, ()), "order": (study_order, (512, 2048)), "pool": (study_pool, (512, 2048)), "range": (study_range, ()),
           "release": (study_release, (2048, 4096, 8192)),
           "budget": (study_budget, (256, 512, 768, 1024, 1536, 2048, 3072, 4096))}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("study", choices=sorted(STUDIES) + ["all"])
    ap.add_argument("--ks", default=None, help="comma-separated K values (default: the study's own)")
    ap.add_argument("--budgets", default=",".join(map(str, BUDGETS)), help="reducer workgroup counts x")
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--rounds", type=int, default=3)
    ap.add_argument("--out", default=None, help="also append the JSON rows to this file")
    a = ap.parse_args(argv)
    budgets = tuple(int(v) for v in a.budgets.split(","))
    sink = open(a.out, "a") if a.out else None

    def emit(row):
        s = json.dumps(row)
        print(s, flush=True)
        if sink:
            sink.write(s + "\n")
            sink.flush()

    for name in (sorted(STUDIES) if a.study == "all" else [a.study]):
        fn, ks = STUDIES[name]
        if a.ks:
            ks = tuple(int(v) for v in a.ks.split(","))
        fn(ks, budgets, emit, steps=a.steps, warmup=a.warmup, rounds=a.rounds)
    if sink:
        sink.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
