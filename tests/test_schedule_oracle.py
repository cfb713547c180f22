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
@pytest.mark.parametrize("group_m", [1, 4])
def test_schedule_is_a_bijection_onto_blocks_and_tiles(M, N, P, BM, BN, order, group_m):
    sched = S.full_schedule(order, M, N, P, BM, BN, group_m)
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
@pytest.mark.parametrize("group_m", [1, 4])
def test_interleaved_local_blocks_are_p_apart(M, N, P, BM, BN, group_m):
    sched = S.full_schedule(S.INTERLEAVED, M, N, P, BM, BN, group_m)
    for r in range(P):
        pos = [p for p, s in enumerate(sched) if s[0] == r]
        assert pos[0] == r and all(b - a == P for a, b in zip(pos, pos[1:]))
        # within a partition, production follows the partition walk (the consumer's order)
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


def test_grouped_walk_keeps_xcd_patches_compact():
    """With P = 8 every partition runs on one XCD; 32 consecutive blocks of
    the grouped walk (group_m = 4) touch 4 block rows and 8 block columns,
    against 1 row and 32 columns for the N-major walk."""
    RB, NB = 4, 32
    for gm, rows, cols in ((4, 4, 8), (1, 1, 32)):
        walk = S.partition_walk(RB, NB, 8, gm)
        assert sorted(walk) == [(r, c) for r in range(RB) for c in range(NB)]
        first = walk[:32]
        assert len({r for r, _ in first}) == rows and len({c for _, c in first}) == cols


def test_grouped_walk_stripes_follow_xcds():
    """P = 2: blocks of partition d at positions p = 2 l + d run on XCD
    p mod 8, i.e. stripe l mod 4; each stripe is a fixed quarter of the columns."""
    RB, NB, P = 4, 16, 2
    walk = S.partition_walk(RB, NB, P, 4)
    for l, (r, c) in enumerate(walk):
        assert c // 4 == l % 4
