"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Floating-point results must pass both the paper's gate
(|err| <= 0.1 + 0.05 |ref|) and the elementwise rounding bound of a
bf16-in / fp32-accumulate / bf16-partial / fp32-reduce / bf16-out path.
Integer-valued inputs small enough to be exact at every step must match
bit for bit.  Full-size workloads are checked on sampled rows (every column
of each sampled row, so every column tile is covered)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_11562_amd import entwine as E
from paper_2609_11562_amd.inputs import Dist, bits_to_torch, make_problem
from paper_2609_11562_amd.tuning import tuned_config
from paper_2609_11562_amd.workloads import WORKLOADS

pytestmark = pytest.mark.gpu


def dev(bits):
    return bits_to_torch(bits).cuda()


def host_bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def upload(prob):
    return dev(prob.A), dev(prob.B), [dev(p) for p in prob.peers]


def out_global_rows(M, P, dest):
    return np.arange(M) if dest == E.DEST_ALL else np.arange(dest * (M // P), (dest + 1) * (M // P))


def check_rows(prob, got_bits, grow, local_rows=None):
    """got_bits: GPU output rows (bf16 bits) for global rows `grow`."""
    ref = oracle.output_rows(prob.A, prob.B, prob.peers, grow)
    bound = oracle.error_bound_rows(prob.A, prob.B, prob.peers, grow)
    got = oracle.bf16_to_f64(got_bits)
    assert not np.isnan(got).any(), "NaN in output"
    gate = oracle.paper_gate(got, ref)
    err = np.abs(got - ref)
    assert gate.all(), f"paper gate fails at {np.argwhere(~gate)[:5].tolist()}"
    bad = err > bound
    assert not bad.any(), (f"rounding bound exceeded at {np.argwhere(bad)[:5].tolist()}, "
                           f"max err {err.max():.3g}")


def run(ctx, A, B, peers, dest, cfg=None, fused=True, out=None, partial=None):
    rs = torch.cuda.Stream() if fused else None
    o = ctx.gemm_rs(A, B, peers, dest, out=out, partial=partial, cfg=cfg, reduce_stream=rs)
    st, tile, src = ctx.query_status()
    assert st == E.OK, f"status {st} tile {tile} src {src}"
    return o


# --------------------------------------------------------------- small case
@pytest.fixture(scope="module")
def tiny():
    w = WORKLOADS["tiny_512x256x1024_p2"]
    prob = w.problem()
    ctx = E.Context(w.M, w.N, w.K, w.P)
    yield w, prob, ctx, upload(prob)
    ctx.close()


@pytest.mark.parametrize("dest", [0, 1, E.DEST_ALL])
@pytest.mark.parametrize("order", [E.ORDER_INTERLEAVED, E.ORDER_ROW_MAJOR, E.ORDER_M_MAJOR])
def test_tiny_matches_oracle(tiny, dest, order):
    w, prob, ctx, (A, B, peers) = tiny
    print(f"[tiny] dest={dest} order={order}", flush=True)
    o = run(ctx, A, B, peers, dest, E.Config.make(order=order))
    torch.cuda.synchronize()
    check_rows(prob, host_bits(o), out_global_rows(w.M, w.P, dest))


@pytest.mark.parametrize("gemm_cfg", [0, 1, 2, 3])
def test_tiny_every_block_shape(tiny, gemm_cfg):
    w, prob, ctx, (A, B, peers) = tiny
    print(f"[tiny] gemm_cfg={gemm_cfg}", flush=True)
    o = run(ctx, A, B, peers, E.DEST_ALL, E.Config.make(gemm_cfg=gemm_cfg, reduce_wgs=4))
    torch.cuda.synchronize()
    check_rows(prob, host_bits(o), np.arange(w.M))


# --------------------------------------------------------------- exact integer cases
@pytest.mark.parametrize("M,N,K,P,a,pk", [(512, 256, 96, 4, 1, 16), (1024, 384, 128, 8, 1, 16),
                                          (256, 128, 16, 2, 2, 16), (2048, 512, 40, 8, 1, 8),
                                          (128, 128, 8, 1, 1, 0)])
def test_integer_inputs_bit_exact(M, N, K, P, a, pk):
    print(f"[int] M={M} N={N} K={K} P={P}", flush=True)
    prob = make_problem(M, N, K, P, Dist("int", a), Dist("int", max(pk, 1)), seed=M + K)
    A, B, peers = upload(prob)
    ref = oracle.gemm_reduce_scatter(prob.A, prob.B, prob.peers, P, E.DEST_ALL)
    with E.Context(M, N, K, P) as ctx:
        for cfg in (0, 3):
            if (M // P) % E.GEMM_SHAPES[cfg][0] or N % E.GEMM_SHAPES[cfg][1]:
                continue
            o = run(ctx, A, B, peers, E.DEST_ALL, E.Config.make(gemm_cfg=cfg))
            torch.cuda.synchronize()
            got = oracle.bf16_to_f64(host_bits(o))
            assert np.array_equal(got, ref), f"max diff {np.abs(got - ref).max()}"


# --------------------------------------------------------------- K tails, odd shapes
@pytest.mark.parametrize("M,N,K,P", [(256, 128, 8, 2), (512, 256, 40, 4), (1024, 512, 1376, 8),
                                     (768, 384, 200, 3), (1280, 640, 72, 5)])
def test_k_tail_and_odd_p(M, N, K, P):
    print(f"[tail] M={M} N={N} K={K} P={P}", flush=True)
    prob = make_problem(M, N, K, P, Dist("normal", 0.02), Dist("normal", 4e-4 * K ** 0.5), seed=K)
    A, B, peers = upload(prob)
    with E.Context(M, N, K, P) as ctx:
        for dest in (0, P - 1, E.DEST_ALL):
            o = run(ctx, A, B, peers, dest, E.Config.make(gemm_cfg=E.GEMM_128x128))
            torch.cuda.synchronize()
            check_rows(prob, host_bits(o), out_global_rows(M, P, dest))


# --------------------------------------------------------------- invariants (bitwise)
def test_results_independent_of_order_budget_threads_and_mode():
    M, N, K, P = 2048, 1024, 520, 4
    print("[invariants]", flush=True)
    prob = make_problem(M, N, K, P, Dist("normal", 0.02), Dist("normal", 4e-4 * K ** 0.5), seed=99)
    A, B, peers = upload(prob)
    with E.Context(M, N, K, P) as ctx:
        base = host_bits(run(ctx, A, B, peers, E.DEST_ALL))
        torch.cuda.synchronize()
        check_rows(prob, base[::37], np.arange(M)[::37])
        variants = [dict(order=o) for o in (1, 2)] + [dict(gemm_cfg=c) for c in (1, 2, 3)] + \
                   [dict(group_m=g) for g in (1, 2, 8)] + [dict(order=2, group_m=1)] + \
                   [dict(gemm_wgs=8), dict(gemm_cfg=1, gemm_wgs=24), dict(gemm_cfg=2, gemm_wgs=16),
                    dict(gemm_cfg=3, gemm_wgs=40)] + \
                   [dict(reduce_wgs=x) for x in (4, 8, 32, 64)] + \
                   [dict(reduce_threads=b) for b in (128, 512)] + \
                   [dict(launch=1), dict(launch=1, reduce_threads=512, reduce_wgs=8),
                    dict(launch=1, gemm_cfg=3, reduce_threads=1024)] + \
                   [dict(launch=2), dict(launch=2, reduce_wgs=5), dict(launch=2, gemm_cfg=1, reduce_wgs=40)] + \
                   [dict(reduce_wgs=-1), dict(reduce_wgs=-1, gemm_cfg=3)] + \
                   [dict(release_blocks=g, launch=l, gemm_cfg=c)
                    for g in (2, E.RELEASE_AT_END, E.RELEASE_PARTITION, E.RELEASE_OUTPUT)
                    for l, c in ((0, 0), (1, 3), (2, 1))] + \
                   [dict(release_blocks=E.RELEASE_PARTITION, reduce_wgs=-1, gemm_cfg=2)] + \
                   [dict(store_mode=m, release_blocks=g, reduce_wgs=x, launch=l)
                    for m in (1, 2) for g, x, l in ((2, -1, 0), (E.RELEASE_AT_END, 16, 0), (1, 8, 1))]
        for kw in variants:
            o = host_bits(run(ctx, A, B, peers, E.DEST_ALL, E.Config.make(**kw)))
            assert np.array_equal(o, base), kw
        seq = host_bits(run(ctx, A, B, peers, E.DEST_ALL, fused=False))
        assert np.array_equal(seq, base), "sequential differs from fused"
        # x = -1 (no dedicated reducers) is a fused-launch setting; the
        # standalone reducer of the sequential form falls back to its default.
        seq = host_bits(run(ctx, A, B, peers, E.DEST_ALL, E.Config.make(reduce_wgs=-1), fused=False))
        assert np.array_equal(seq, base), "sequential with reduce_wgs=-1 differs"
        parts = [host_bits(run(ctx, A, B, peers, d, E.Config.make(reduce_wgs=x)))
                 for d, x in zip(range(P), (1, 3, 16, 64))]
        assert np.array_equal(np.concatenate(parts, axis=0), base), "chunks differ from all-chunk output"
        # release groups on single chunks, each call leaving its counters at a multiple
        for d, g in zip(range(P), (E.RELEASE_PARTITION, E.RELEASE_OUTPUT, E.RELEASE_PARTITION, 1)):
            o = host_bits(run(ctx, A, B, peers, d, E.Config.make(release_blocks=g, gemm_cfg=d % 4)))
            assert np.array_equal(o, base[d * (M // P):(d + 1) * (M // P)]), (d, g)


def test_zero_peers_give_the_partial_itself():
    """With every peer zero the reduced chunk is the bf16 partial, bit for bit
    (adding +0 in fp32 and rounding back changes nothing)."""
    M, N, K, P = 1024, 512, 200, 4
    print("[zero peers]", flush=True)
    prob = make_problem(M, N, K, P, Dist("normal", 0.02), Dist("const", 0.0), seed=77)
    A, B, peers = upload(prob)
    with E.Context(M, N, K, P) as ctx:
        part = ctx.gemm_only(A, B)
        torch.cuda.synchronize()
        pb = host_bits(part)
        for dest, kw in ((E.DEST_ALL, {}), (2, dict(reduce_wgs=-1)), (1, dict(launch=1)), (3, dict(launch=2))):
            o = run(ctx, A, B, peers, dest, E.Config.make(**kw))
            torch.cuda.synchronize()
            assert np.array_equal(host_bits(o), pb[out_global_rows(M, P, dest)]), (dest, kw)


def test_every_budget_up_to_the_cap_completes_and_agrees():
    """No budget x from 1 to past the cap hangs or changes a bit, in any fused
    form (the library clamps x to min(tiles per chunk, CUs - 1))."""
    M, N, K, P = 4096, 2048, 64, 4
    print("[budgets]", flush=True)
    prob = make_problem(M, N, K, P, Dist("normal", 0.02), Dist("normal", 0.01), seed=88)
    A, B, peers = upload(prob)
    with E.Context(M, N, K, P) as ctx:
        base = host_bits(run(ctx, A, B, peers, 1))
        torch.cuda.synchronize()
        check_rows(prob, base[::61], out_global_rows(M, P, 1)[::61])
        for launch in (0, 1, 2):
            for x in (1, 2, 3, 7, 31, 64, 127, 128, 200, 255):
                o = host_bits(run(ctx, A, B, peers, 1, E.Config.make(launch=launch, reduce_wgs=x, timeout_us=500000)))
                assert np.array_equal(o, base), (launch, x)


def test_reducer_is_exact_on_given_partial():
    """reduce_only on a known partial equals the fp32 rank-order sum rounded
    to bf16, bit for bit; gemm_only's partial stays within the GEMM bound."""
    M, N, K, P = 1024, 512, 256, 8
    print("[reduce_only]", flush=True)
    prob = make_problem(M, N, K, P, Dist("normal", 0.02), Dist("normal", 0.01), seed=5)
    A, B, peers = upload(prob)
    with E.Context(M, N, K, P) as ctx:
        partial = ctx.gemm_only(A, B)
        torch.cuda.synchronize()
        pbits = host_bits(partial)
        C = oracle.local_partial(prob.A, prob.B)
        absab = np.abs(oracle.bf16_to_f64(prob.A)) @ np.abs(oracle.bf16_to_f64(prob.B))
        err = np.abs(oracle.bf16_to_f64(pbits) - C)
        assert np.all(err <= 2 * 2.0 ** -8 * np.abs(C) + 2 * 2.0 ** -24 * K * absab)
        for dest, cfg in ((3, None), (E.DEST_ALL, None), (2, E.Config.make(reduce_wgs=-1))):
            o = ctx.reduce_only(partial, peers, dest, cfg=cfg)
            assert ctx.query_status()[0] == E.OK
            rows = out_global_rows(M, P, dest)
            want = oracle.reduce_scatter.reduce_tile_f32(pbits[rows], [p[rows] for p in prob.peers])
            assert np.array_equal(host_bits(o), want)


# --------------------------------------------------------------- protocol
def test_withheld_peer_times_out_then_recovers(tiny):
    w, prob, ctx, (A, B, peers) = tiny
    print("[timeout]", flush=True)
    for launch in (0, 1, 2):
        cfg = E.Config.make(withhold_peer=0, timeout_us=20000, reduce_wgs=2, launch=launch)
        ctx.gemm_rs(A, B, peers, 1, cfg=cfg, reduce_stream=torch.cuda.Stream())
        st, tile, src = ctx.query_status()
        assert st == E.ETIMEOUT and src == 0 and 0 <= tile < (w.M // 128) * (w.N // 128), launch
        o = run(ctx, A, B, peers, 1)
        torch.cuda.synchronize()
        check_rows(prob, host_bits(o), out_global_rows(w.M, w.P, 1))


def test_poisoned_buffers_never_leak_across_repeated_calls():
    """Partial and output are NaN-poisoned before every call and two input
    sets alternate, so a read before publication, a stale cache line from an
    earlier call or a missed tile shows up as NaN or as the other set's value."""
    M, N, K, P = 2048, 2048, 256, 8
    print("[poison]", flush=True)
    probs = [make_problem(M, N, K, P, Dist("normal", 0.02), Dist("normal", 0.01), seed=s) for s in (1, 2)]
    ups = [upload(p) for p in probs]
    want = []
    nan = torch.tensor(0x7FC0, dtype=torch.int16).view(torch.bfloat16)
    partial = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    out = torch.empty(M // P, N, dtype=torch.bfloat16, device="cuda")
    rs = torch.cuda.Stream()
    with E.Context(M, N, K, P) as ctx:
        for i in range(24):
            A, B, peers = ups[i % 2]
            partial.fill_(nan)
            out.fill_(nan)
            release = (1, 2, E.RELEASE_AT_END, E.RELEASE_PARTITION, E.RELEASE_OUTPUT)[i % 5]
            ctx.gemm_rs(A, B, peers, 5, out=out, partial=partial, reduce_stream=rs,
                        cfg=E.Config.make(reduce_wgs=8 + i, launch=(i // 2) % 3, release_blocks=release,
                                          store_mode=(i // 6) % 3))
            got = host_bits(out)
            if i < 2:
                check_rows(probs[i], got, out_global_rows(M, P, 5))
                want.append(got)
            else:
                assert np.array_equal(got, want[i % 2]), f"call {i}"
        assert ctx.query_status()[0] == E.OK


def test_bad_arguments_are_rejected(tiny):
    w, prob, ctx, (A, B, peers) = tiny
    with pytest.raises(E.EntwineError) as ei:
        ctx.gemm_rs(A, B, peers, 5)
    assert ei.value.status == E.EINVAL
    with pytest.raises(ValueError):
        ctx.gemm_rs(A[:, :128], B, peers, 0)
    with pytest.raises(ValueError):
        ctx.gemm_rs(A, B, peers[:0], 0)


# --------------------------------------------------------------- full sizes
def sample_rows(M, P, dest, n=24, seed=0):
    rows = out_global_rows(M, P, dest)
    rng = np.random.default_rng(seed)
    pick = set(rng.choice(rows, size=min(n, len(rows)), replace=False).tolist())
    pick |= {int(rows[0]), int(rows[-1]), int(rows[len(rows) // 2]), int(rows[127 % len(rows)])}
    return np.array(sorted(pick))


@pytest.mark.parametrize("name", ["llama7b_mlp_down_tp8", "llama70b_attn_out_tp8", "llama70b_mlp_down_tp8",
                                  "sweep_8192x512x8192_p2", "sweep_8192x2048x8192_p4",
                                  "qwen25_72b_mlp_down_m512_tp8", "llama3_8b_attn_out_m2048_tp8"])
def test_full_size_workloads_on_sampled_rows(name):
    w = WORKLOADS[name]
    print(f"[full] {name}", flush=True)
    prob = w.problem()
    A, B, peers = upload(prob)
    with E.Context(w.M, w.N, w.K, w.P) as ctx:
        for dest in (0, w.P - 1, E.DEST_ALL):
            scope = "all" if dest == E.DEST_ALL else "rank"
            # the launch configuration the benchmark times, then a fixed budget
            for kw in (tuned_config(name, scope), dict(reduce_wgs=16)):
                o = run(ctx, A, B, peers, dest, E.Config.make(**kw))
                torch.cuda.synchronize()
                grow = sample_rows(w.M, w.P, dest, seed=dest + 1)
                local = grow - (0 if dest == E.DEST_ALL else dest * (w.M // w.P))
                check_rows(prob, host_bits(o[torch.as_tensor(local, device="cuda")]), grow)
    del A, B, peers
    torch.cuda.empty_cache()


def test_sweep_orders_and_budgets_full_size():
    """The schedule / CU-split sweep at full size (M = N = 8192, K = 2048,
    P = 8): row-major against chunk-interleaved order, reducer budgets 4 and
    32, single launch and two streams, on sampled rows of one chunk and of
    every chunk."""
    w = WORKLOADS["sweep_8192x2048x8192_p8"]
    print("[full sweep]", flush=True)
    prob = w.problem()
    A, B, peers = upload(prob)
    with E.Context(w.M, w.N, w.K, w.P) as ctx:
        for order in (E.ORDER_INTERLEAVED, E.ORDER_ROW_MAJOR):
            for x in (4, 32):
                for launch in (0, 1):
                    for dest in (3, E.DEST_ALL):
                        o = run(ctx, A, B, peers, dest, E.Config.make(order=order, reduce_wgs=x, launch=launch))
                        torch.cuda.synchronize()
                        grow = sample_rows(w.M, w.P, dest, n=12, seed=x + launch)
                        local = grow - (0 if dest == E.DEST_ALL else dest * (w.M // w.P))
                        check_rows(prob, host_bits(o[torch.as_tensor(local, device="cuda")]), grow)
    del A, B, peers
    torch.cuda.empty_cache()


def test_workgroup_timeline_is_consistent(tiny):
    w, prob, ctx, (A, B, peers) = tiny
    print("[stamps]", flush=True)
    run(ctx, A, B, peers, 1, E.Config.make(record_timing=1, reduce_wgs=4))
    us, G = ctx.last_stamps()
    assert us.shape[1] == 4 and 0 < G < us.shape[0]
    assert np.all(us[:, 0] >= 0) and np.all(us[:, 1] >= us[:, 0]) and np.all(us[:, 3] >= us[:, 1])
    ready = ~np.isnan(us[:, 2])
    assert ready.any() and np.all(us[ready, 2] >= us[ready, 1]) and np.all(us[ready, 2] <= us[ready, 3])
    assert np.all(us[G:, 1] == us[G:, 0])   # dedicated reducers have no producer role
    # the engine clock the producers ran at: above 0.1 GHz, at most the
    # 2.4 GHz maximum (with a margin for counter granularity on a tiny call)
    ghz = ctx.last_clock()
    assert 0.1 < ghz < 2.6, ghz
    run(ctx, A, B, peers, 1, E.Config.make(record_timing=1, launch=1))
    for query in (ctx.last_stamps, ctx.last_clock):
        with pytest.raises(E.EntwineError) as ei:
            query()
        assert ei.value.status == E.EUNSUPPORTED
