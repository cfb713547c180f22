"""Named workloads: one tensor-parallel rank's share of a row-parallel
GEMM-ReduceScatter, with the shapes of the paper's LLM projections.

Each rank holds A (M x K_local) and B (K_local x N) and emits an M x N partial;
the output is split into P equal row chunks.  The synthetic peer partials
stand in for the other P-1 ranks and are drawn with the variance a real
partial of the same shape would have: with A, B ~ N(0, s^2) a K-term dot
product has standard deviation s*s*sqrt(K).
"""
from __future__ import annotations

import dataclasses
import math

from .inputs import BASE_SEED, Dist, Problem, make_layer_inputs, make_problem


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    M: int
    N: int
    K: int
    P: int
    ab: Dist
    peer: Dist
    note: str = ""
    layer: bool = False   # the call adds the residual and applies RMSNorm

    @property
    def flops(self) -> float:
        return 2.0 * self.M * self.N * self.K

    def problem(self, seed: int = BASE_SEED) -> Problem:
        return make_problem(self.M, self.N, self.K, self.P, self.ab, self.peer, seed)

    def layer_inputs(self, seed: int = BASE_SEED):
        """(R, gamma) of the layer epilogue for one rank's chunk of M/P rows."""
        return make_layer_inputs(self.M // self.P, self.N, seed)


def _llm(name, M, K, N, P, note, layer=False):
    s = 0.02
    return Workload(name, M, N, K, P, Dist("normal", s), Dist("normal", s * s * math.sqrt(K)), note, layer)


WORKLOADS = {
    w.name: w
    for w in [
        # U[-1,1] entries: a 256-term dot product has std sqrt(256/9).
        Workload("tiny_512x256x1024_p2", 512, 1024, 256, 2,
                 Dist("uniform", 1.0), Dist("normal", math.sqrt(256 / 9)),
                 "small parity case, two row chunks of 256 x 1024"),
        _llm("llama7b_mlp_down_tp8", 4096, 1376, 4096, 8,
             "Llama-7B MLP down projection (K = 11008 / 8), 4096 tokens"),
        _llm("llama70b_attn_out_tp8", 8192, 1024, 8192, 8,
             "Llama-3-70B attention output projection, 8192 tokens"),
        _llm("llama70b_mlp_down_tp8", 16384, 3584, 8192, 8,
             "Llama-3-70B MLP down projection, 16384 tokens"),
    ]
}

# Schedule / CU-split sweep: M = N = 8192, K_local in {512, 2048}, P in {2, 4, 8}.
for _K in (512, 2048):
    for _P in (2, 4, 8):
        _w = _llm(f"sweep_8192x{_K}x8192_p{_P}", 8192, _K, 8192, _P,
                  "budget / tile-order sweep window (the paper's two K windows)")
        WORKLOADS[_w.name] = _w

# Layer level: the Llama-3-70B attention output projection followed by the
# residual addition and RMSNorm, at global sequence lengths 4K, 8K and 16K
# (the GEMM's M; model width and K_local fixed).
for _S in (4, 8, 16):
    _w = _llm(f"llama70b_attn_out_layer_seq{_S}k_tp8", _S * 1024, 1024, 8192, 8,
              f"attention output + residual addition + RMSNorm, {_S}K tokens", layer=True)
    WORKLOADS[_w.name] = _w

# The paper's two evaluation suites (Table 1), one rank's share at P = 8.
# Main operator suite: N = 8192 (Llama-3-70B width) with M in {8192, 16384,
# 32768, 49152} and N = 16384 (Llama-3.1-405B width) with M = 16384, each at
# K_local in {2048, 4096, 8192}: 15 workloads.
SUITES = {"main": [], "models": []}
for _N, _Ms in ((8192, (8192, 16384, 32768, 49152)), (16384, (16384,))):
    for _M in _Ms:
        for _K in (2048, 4096, 8192):
            _w = _llm(f"main_{_M}x{_K}x{_N}_p8", _M, _K, _N, 8, "main operator suite")
            WORKLOADS[_w.name] = _w
            SUITES["main"].append(_w.name)
# Model-derived suite at TP = 8: five projections (N, K_local) at logical M in
# {512, ..., 8192}; M = 512 runs padded to 1024 rows, as the paper's methods
# do: 25 workloads.
for _p, _N, _K in (("llama3_8b_attn_out", 4096, 512), ("llama3_8b_mlp_down", 4096, 1792),
                   ("llama3_70b_attn_out", 8192, 1024), ("llama3_70b_mlp_down", 8192, 3584),
                   ("qwen25_72b_mlp_down", 8192, 3696)):
    for _M in (512, 1024, 2048, 4096, 8192):
        _w = _llm(f"{_p}_m{_M}_tp8", max(_M, 1024), _K, _N, 8,
                  f"model-derived suite, logical M = {_M}" + (" (padded to 1024 rows)" if _M < 1024 else ""))
        WORKLOADS[_w.name] = _w
        SUITES["models"].append(_w.name)

BENCH_WORKLOAD = "llama7b_mlp_down_tp8"
SMALL_WORKLOAD = "tiny_512x256x1024_p2"

__all__ = ["Workload", "WORKLOADS", "SUITES", "BENCH_WORKLOAD", "SMALL_WORKLOAD", "BASE_SEED"]
