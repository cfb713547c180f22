"""Per-workload launch configuration chosen by end-to-end latency.

The paper selects the GEMM block shape, the reducer grid size x and its
thread count b together, by the lowest end-to-end latency under concurrent
execution (Section 3.2 "End-to-end optimization", Section 4.3).  The table
in ``tuned.json`` holds the winners of that sweep, keyed by workload name and
scope ("rank" = one chunk, "all" = every chunk, "layer" = one chunk followed
by the residual addition and RMSNorm); anything missing falls back to the
library defaults.
"""
from __future__ import annotations

import json
import os

_TABLE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tuned.json")
_FIELDS = ("order", "gemm_cfg", "reduce_wgs", "reduce_threads", "group_m", "launch", "release_blocks", "store_mode")


def load_table() -> dict:
    if not os.path.exists(_TABLE):
        return {}
    with open(_TABLE) as f:
        return json.load(f)


def tuned_config(workload: str, scope: str = "rank") -> dict:
    entry = load_table().get(workload, {}).get(scope, {})
    return {k: int(entry[k]) for k in _FIELDS if k in entry}
