"""Host-only checks of the configuration table (paper Section 4.3: the
offline profiler's choice of block shape, x and b is looked up per
workload)."""
import json

from paper_2609_11562_amd import entwine as E
from paper_2609_11562_amd import tune, tuning
from paper_2609_11562_amd.workloads import WORKLOADS


def test_table_entries_are_valid_configs():
    table = tuning.load_table()
    for name, scopes in table.items():
        assert name in WORKLOADS, name
        w = WORKLOADS[name]
        for scope, entry in scopes.items():
            assert scope in ("rank", "all", "layer")
            assert (scope == "layer") == w.layer, (name, scope)
            kw = tuning.tuned_config(name, scope)
            assert set(kw) <= set(tuning._FIELDS) and kw
            dest = E.DEST_ALL if scope == "all" else 0
            assert E.validate(w.M, w.N, w.K, w.P, dest, E.Config.make(**kw)) == E.OK


def test_missing_workload_falls_back_to_defaults():
    assert tuning.tuned_config("no_such_workload") == {}


def test_write_entry_round_trip(tmp_path):
    path = tmp_path / "t.json"
    best = dict(order=0, gemm_cfg=1, reduce_wgs=24, reduce_threads=512, group_m=4, launch=0, release_blocks=1, wall_ms=0.5,
                event_ms=0.4)
    tune.write_entry("llama7b_mlp_down_tp8", "rank", best, str(path))
    tune.write_entry("llama7b_mlp_down_tp8", "all", dict(best, reduce_wgs=32), str(path))
    t = json.loads(path.read_text())
    assert t["llama7b_mlp_down_tp8"]["rank"]["reduce_wgs"] == 24
    assert t["llama7b_mlp_down_tp8"]["all"]["reduce_wgs"] == 32
    assert t["llama7b_mlp_down_tp8"]["rank"]["measured_ms"] == 0.5


def test_ablation_studies_and_shapes():
    from paper_2609_11562_amd import ablation
    assert set(ablation.STUDIES) == {"order", "pool", "release", "budget", "range", "clock"}
    assert len(ablation.STUDIES["budget"][1]) == 8
    for K in (512, 768, 4096):
        w = ablation.workload(K)
        assert (w.M, w.N, w.K, w.P) == (8192, 8192, K, 8)
        cfg = E.Config.make(launch=1, gemm_cfg=E.GEMM_128x128, release_blocks=E.RELEASE_PARTITION, reduce_wgs=16)
        assert E.validate(w.M, w.N, w.K, w.P, 0, cfg) == E.OK


def test_paper_suites_have_table_1_shapes():
    from paper_2609_11562_amd.workloads import SUITES
    main = [WORKLOADS[n] for n in SUITES["main"]]
    assert len(main) == 15 and {w.K for w in main} == {2048, 4096, 8192}
    assert {(w.M, w.N) for w in main} == {(8192, 8192), (16384, 8192), (32768, 8192), (49152, 8192), (16384, 16384)}
    models = [WORKLOADS[n] for n in SUITES["models"]]
    assert len(models) == 25 and min(w.M for w in models) == 1024
    assert {(w.N, w.K) for w in models} == {(4096, 512), (4096, 1792), (8192, 1024), (8192, 3584), (8192, 3696)}
    for w in main + models:
        assert E.validate(w.M, w.N, w.K, w.P, 0, E.Config.make()) == E.OK, w.name
