"""Pins for the oracle's schedule: the paper's two worked examples (golden
fixtures with citations) and the structural properties of Equation 1."""
import json
import os

import pytest

from oracle import schedule as S

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_fig3_worked_example():
    g = _load("fig3_interleaved_example.json")
    P, M, N, BM, BN = g["P"], g["M"], g["N"], g["BM"], g["BN"]
    sched = S.full_schedule(S.INTERLEAVED, M, N, P, BM, BN)
    assert [sched[p][0] for p in range(4)] == g["first_positions_partitions"]
    visits = [p for p, s in enumerate(sched) if s[0] == g["dest"]]
    assert visits == g["visits_to_dest"]
    for p, tiles in g["tiles_of_position"].items():
        assert [t for t, _, _ in sched[int(p)][4]] == tiles
    Q = S.tiles_per_partition(M, N, P)
    assert Q == 6
    for j, tasks in g["consumer_tasks"].items():
        assert S.consumer_tasks(int(j), g["x"], Q) == tasks


def _local_runs(dests, r):
    runs, cur = [], 0
    for d in dests:
        if d == r:
            cur += 1
        elif cur:
            runs.append(cur)
            cur = 0
    if cur:
        runs.append(cur)
    return runs


def test_fig1_local_runs():
    g = _load("fig1_local_runs.json")
    P, M, N, BM, BN = g["P"], g["M"], g["N"], g["BM"], g["BN"]
    for name, order in (("row_major", S.ROW_MAJOR), ("interleaved", S.INTERLEAVED)):
        dests = [s[0] for s in S.full_schedule(order, M, N, P, BM, BN)]
        for r in range(P):
            assert _local_runs(dests, r) == g["local_run_lengths"][name]


SHAPES = [(512, 1024, 2, 256, 256), (4096, 4096, 8, 256, 256), (1024, 768, 4, 128, 256),
          (2048, 512, 8, 128, 128), (1536, 512, 3, 256, 128)]


@pytest.mark.parametrize("M,N,P,BM,BN", SHAPES)
@pytest.mark.parametrize("order", [S.INTERLEAVED, S.ROW_MAJOR, S.M_MAJOR])
def test_schedule_is_a_bijection_onto_blocks_and_tiles(M, N, P, BM, BN, order):
    sched = S.full_schedule(order, M, N, P, BM, BN)
    nb = (M // BM) * (N // BN)
    assert len({(s[2], s[3]) for s in sched}) == nb
    Q = S.tiles_per_partition(M, N, P)
    per_part = {d: [] for d in range(P)}
    for d, l, mb, nb_, tiles in sched:
        # the block lies inside its partition's rows
        assert d * (M // P) <= mb * BM and (mb + 1) * BM <= (d + 1) * (M // P)
        per_part[d].extend(t for t, _, _ in tiles)
        for t, tr, tc in tiles:
            assert mb * BM <= tr * 128 < (mb + 1) * BM and nb_ * BN <= tc * 128 < (nb_ + 1) * BN
    for d in range(P):
        assert sorted(per_part[d]) == list(range(Q))


@pytest.mark.parametrize("M,N,P,BM,BN", SHAPES)
def test_interleaved_local_blocks_are_p_apart(M, N, P, BM, BN):
    sched = S.full_schedule(S.INTERLEAVED, M, N, P, BM, BN)
    for r in range(P):
        pos = [p for p, s in enumerate(sched) if s[0] == r]
        assert pos[0] == r and all(b - a == P for a, b in zip(pos, pos[1:]))
        # within a partition, production follows the consumer's N-major order
        assert [sched[p][1] for p in pos] == list(range(len(pos)))


@pytest.mark.parametrize("M,N,P,BM,BN", SHAPES)
def test_row_major_is_partition_contiguous(M, N, P, BM, BN):
    sched = S.full_schedule(S.ROW_MAJOR, M, N, P, BM, BN)
    nb = len(sched)
    for p, s in enumerate(sched):
        assert s[0] == p // (nb // P)


def test_m_major_walks_m_fastest():
    sched = S.full_schedule(S.M_MAJOR, 1024, 512, 4, 128, 128)
    assert [(s[2], s[3]) for s in sched[:9]] == [(i, 0) for i in range(8)] + [(0, 1)]


@pytest.mark.parametrize("Q,x", [(6, 2), (128, 16), (7, 3), (5, 5), (512, 32)])
def test_consumer_tasks_cover_each_tile_once_in_order(Q, x):
    seen = []
    for j in range(x):
        tasks = S.consumer_tasks(j, x, Q)
        assert tasks == sorted(tasks)
        seen.extend(tasks)
    assert sorted(seen) == list(range(Q))


def test_all_chunk_assignment_splits_budget_evenly():
    P, Q, x = 4, 10, 8
    cover = {d: [] for d in range(P)}
    for j in range(x):
        d, tasks = S.all_chunk_consumer_tasks(j, x, P, Q)
        cover[d].extend(tasks)
    assert all(sorted(v) == list(range(Q)) for v in cover.values())
    with pytest.raises(ValueError):
        S.all_chunk_consumer_tasks(0, 6, 4, Q)
