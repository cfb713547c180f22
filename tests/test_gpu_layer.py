"""GPU parity of the layer epilogue (residual addition + RMSNorm after the
reduce-scatter; paper Section 5.2, layer-level performance) through the C ABI
against the float64 oracle.

h (the new residual stream) must match the reducer's own fp32 arithmetic bit
for bit on the partial of the same call, and both h and y must pass the
paper's gate and the elementwise rounding bounds of the fused path.  Both are
reproducible bit for bit across configurations (one workgroup per row)."""
import numpy as np
import pytest
import torch

import oracle
from oracle import layer as L
from paper_2609_11562_amd import entwine as E
from paper_2609_11562_amd.inputs import Dist, bits_to_torch, make_layer_inputs, make_problem
from paper_2609_11562_amd.tuning import tuned_config
from paper_2609_11562_amd.workloads import WORKLOADS

pytestmark = pytest.mark.gpu

EPS = 1e-5


def dev(bits):
    return bits_to_torch(bits).cuda()


def host_bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def out_rows(M, P, dest):
    return np.arange(M) if dest == E.DEST_ALL else np.arange(dest * (M // P), (dest + 1) * (M // P))


def layer_inputs(M, N, P, dest, seed):
    return make_layer_inputs(len(out_rows(M, P, dest)), N, seed)


def check_layer(prob, R_bits, gamma, h_bits, y_bits, grow, lrow):
    """grow: global rows of the reduced output; lrow: their rows in h/y/R."""
    O = oracle.output_rows(prob.A, prob.B, prob.peers, grow)
    h_ref, y_ref = L.layer(O, R_bits[lrow], gamma, EPS)
    sb = oracle.error_bound_rows(prob.A, prob.B, prob.peers, grow, final_rounding=False)
    hb = L.h_bound(sb, h_ref, R_bits[lrow])
    yb = L.y_bound(h_ref, hb, gamma, EPS)
    h = oracle.bf16_to_f64(h_bits[lrow])
    y = oracle.bf16_to_f64(y_bits[lrow])
    assert not np.isnan(h).any() and not np.isnan(y).any(), "NaN in output"
    for name, got, ref, bound in (("h", h, h_ref, hb), ("y", y, y_ref, yb)):
        assert oracle.paper_gate(got, ref).all(), f"{name}: paper gate fails"
        bad = np.abs(got - ref) > bound
        assert not bad.any(), f"{name}: bound exceeded at {np.argwhere(bad)[:5].tolist()}"


@pytest.mark.parametrize("dest,N", [(1, 1024), (E.DEST_ALL, 1024), (2, 3200), (0, 16384), (3, 12416)])
def test_layer_matches_oracle_and_reducer_arithmetic(dest, N):
    """N = 3200 leaves a ragged last step of columns (a row is walked 2048
    columns at a time); N above 8192 takes a second batch of loads per row
    (16384 the largest row, 12416 with a ragged last step)."""
    M, K, P = 1024, 256, 4
    print(f"[layer small dest={dest} N={N}]", flush=True)
    prob = make_problem(M, N, K, P, Dist("normal", 0.02), Dist("normal", 0.02), seed=31)
    A, B, peers = dev(prob.A), dev(prob.B), [dev(p) for p in prob.peers]
    R, gamma = layer_inputs(M, N, P, dest, 40)
    partial = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    with E.Context(M, N, K, P) as ctx:
        h, y = ctx.gemm_rs_rmsnorm(A, B, peers, dest, dev(R), dev(gamma), EPS, partial=partial)
        assert ctx.query_status()[0] == E.OK
        hb, yb, pb = host_bits(h), host_bits(y), host_bits(partial)
    grow = out_rows(M, P, dest)
    # h is the reducer's fp32 chain on this call's partial, bit for bit
    want = L.residual_add_f32(pb[grow], [p[grow] for p in prob.peers], R)
    assert np.array_equal(hb, want)
    check_layer(prob, R, gamma, hb, yb, grow, np.arange(len(grow)))


def test_layer_invariant_across_configs_and_repeated_calls():
    """h and y are bitwise stable across block shapes, walks, budgets and
    repeated calls (with plain fused calls in between), and within their
    bounds.  Outputs are NaN-poisoned before each call."""
    M, N, K, P = 1024, 2048, 392, 8
    dest = 5
    print("[layer invariants]", flush=True)
    prob = make_problem(M, N, K, P, Dist("normal", 0.02), Dist("normal", 0.01), seed=32)
    A, B, peers = dev(prob.A), dev(prob.B), [dev(p) for p in prob.peers]
    R, gamma = layer_inputs(M, N, P, dest, 50)
    Rd, gd = dev(R), dev(gamma)
    nan = torch.tensor(0x7FC0, dtype=torch.int16).view(torch.bfloat16)
    grow = out_rows(M, P, dest)
    rows = len(grow)
    h = torch.empty(rows, N, dtype=torch.bfloat16, device="cuda")
    y = torch.empty(rows, N, dtype=torch.bfloat16, device="cuda")
    rs = torch.cuda.Stream()
    cfgs = [None, dict(group_m=1), dict(gemm_cfg=3), dict(reduce_wgs=16), dict(reduce_wgs=-1, release_blocks=-1),
            dict(gemm_cfg=2, release_blocks=2), dict(release_blocks=E.RELEASE_PARTITION, reduce_wgs=8),
            dict(release_blocks=E.RELEASE_OUTPUT, store_mode=2), dict(store_mode=1, order=E.ORDER_M_MAJOR), None]
    with E.Context(M, N, K, P) as ctx:
        base = None
        for i, kw in enumerate(cfgs):
            h.fill_(nan)
            y.fill_(nan)
            cfg = E.Config.make(**kw) if kw else None
            ctx.gemm_rs_rmsnorm(A, B, peers, dest, Rd, gd, EPS, h_out=h, y_out=y, cfg=cfg)
            assert ctx.query_status()[0] == E.OK
            hb, yb = host_bits(h), host_bits(y)
            if base is None:
                base = hb, yb
                check_layer(prob, R, gamma, hb, yb, grow, np.arange(rows))
            else:
                assert np.array_equal(hb, base[0]) and np.array_equal(yb, base[1]), kw
            if i % 2 == 0:   # a plain fused call between layer calls
                ctx.gemm_rs(A, B, peers, i % P, reduce_stream=rs)
                assert ctx.query_status()[0] == E.OK


@pytest.mark.parametrize("name", ["llama70b_attn_out_layer_seq4k_tp8", "llama70b_attn_out_layer_seq8k_tp8",
                                  "llama70b_attn_out_layer_seq16k_tp8"])
def test_layer_full_size_sampled_rows(name):
    """Every layer workload at full size, in the launch configuration the
    benchmark times (its tuned entry) and with a fixed reducer budget, on
    sampled rows of the first and last chunks."""
    w = WORKLOADS[name]
    prob = w.problem()
    A, B, peers = dev(prob.A), dev(prob.B), [dev(p) for p in prob.peers]
    R, gamma = w.layer_inputs()
    Rd, gd = dev(R), dev(gamma)
    rows = w.M // w.P
    lrow = np.unique(np.array([0, 1, 63, 64, 127, 128, rows // 2, rows - 65, rows - 1]))
    with E.Context(w.M, w.N, w.K, w.P) as ctx:
        for dest in (0, w.P - 1):
            for kw in (tuned_config(name, "layer"), dict(reduce_wgs=16)):
                print(f"[layer full {name} dest={dest} cfg={kw}]", flush=True)
                h, y = ctx.gemm_rs_rmsnorm(A, B, peers, dest, Rd, gd, EPS, cfg=E.Config.make(**kw))
                assert ctx.query_status()[0] == E.OK
                sel = torch.as_tensor(lrow, device="cuda")
                hb, yb = host_bits(h[sel]), host_bits(y[sel])
                grow = out_rows(w.M, w.P, dest)[lrow]
                check_layer(prob, R[lrow], gamma, hb, yb, grow, np.arange(len(lrow)))
    del A, B, peers
    torch.cuda.empty_cache()


def test_layer_full_size_every_chunk_sampled_rows():
    """All chunks at once (M row tasks) at the 4K-token layer shape."""
    w = WORKLOADS["llama70b_attn_out_layer_seq4k_tp8"]
    print(f"[layer full all-chunks {w.name}]", flush=True)
    prob = w.problem()
    A, B, peers = dev(prob.A), dev(prob.B), [dev(p) for p in prob.peers]
    R, gamma = make_layer_inputs(w.M, w.N, 61)
    with E.Context(w.M, w.N, w.K, w.P) as ctx:
        h, y = ctx.gemm_rs_rmsnorm(A, B, peers, E.DEST_ALL, dev(R), dev(gamma), EPS)
        assert ctx.query_status()[0] == E.OK
        lrow = np.array([0, 127, 511, 512, 1500, 2047, 2048, 3333, 4095])
        sel = torch.as_tensor(lrow, device="cuda")
        check_layer(prob, R[lrow], gamma, host_bits(h[sel]), host_bits(y[sel]), lrow, np.arange(len(lrow)))
    del A, B, peers
    torch.cuda.empty_cache()


def test_layer_in_place_residual_update():
    """h_out may be the residual buffer itself."""
    M, N, K, P = 1024, 2048, 128, 4
    dest = 3
    print("[layer in place]", flush=True)
    prob = make_problem(M, N, K, P, Dist("normal", 0.02), Dist("normal", 0.02), seed=34)
    A, B, peers = dev(prob.A), dev(prob.B), [dev(p) for p in prob.peers]
    R, gamma = layer_inputs(M, N, P, dest, 80)
    with E.Context(M, N, K, P) as ctx:
        h, y = ctx.gemm_rs_rmsnorm(A, B, peers, dest, dev(R), dev(gamma), EPS)
        Rd = dev(R)
        h2, y2 = ctx.gemm_rs_rmsnorm(A, B, peers, dest, Rd, dev(gamma), EPS, h_out=Rd)
        assert ctx.query_status()[0] == E.OK and h2.data_ptr() == Rd.data_ptr()
        assert torch.equal(h.view(torch.int16), h2.view(torch.int16))
        assert torch.equal(y.view(torch.int16), y2.view(torch.int16))


def test_layer_withheld_peer_times_out_then_recovers():
    M, N, K, P = 1024, 1024, 128, 4
    dest = 0
    print("[layer timeout]", flush=True)
    prob = make_problem(M, N, K, P, Dist("normal", 0.02), Dist("normal", 0.02), seed=35)
    A, B, peers = dev(prob.A), dev(prob.B), [dev(p) for p in prob.peers]
    R, gamma = layer_inputs(M, N, P, dest, 90)
    Rd, gd = dev(R), dev(gamma)
    with E.Context(M, N, K, P) as ctx:
        ctx.gemm_rs_rmsnorm(A, B, peers, dest, Rd, gd, EPS, cfg=E.Config.make(withhold_peer=1, timeout_us=20000))
        st, tile, src = ctx.query_status()
        assert st == E.ETIMEOUT and src == 1 and 0 <= tile < (M // 128) * (N // 128)
        h, y = ctx.gemm_rs_rmsnorm(A, B, peers, dest, Rd, gd, EPS)
        assert ctx.query_status()[0] == E.OK
        grow = out_rows(M, P, dest)
        check_layer(prob, R, gamma, host_bits(h), host_bits(y), grow, np.arange(len(grow)))


def test_layer_rejects_bad_arguments():
    M, N, K, P = 512, 256, 64, 2
    prob = make_problem(M, N, K, P, Dist("normal", 0.02), Dist("normal", 0.02), seed=33)
    A, B, peers = dev(prob.A), dev(prob.B), [dev(p) for p in prob.peers]
    R, gamma = layer_inputs(M, N, P, 0, 70)
    with E.Context(M, N, K, P) as ctx:
        with pytest.raises(E.EntwineError) as ei:
            ctx.gemm_rs_rmsnorm(A, B, peers, 0, dev(R), dev(gamma), 0.0)
        assert ei.value.status == E.EINVAL
        with pytest.raises(E.EntwineError) as ei:
            ctx.gemm_rs_rmsnorm(A, B, peers, 0, dev(R), dev(gamma), EPS, cfg=E.Config.make(launch=1))
        assert ei.value.status == E.EUNSUPPORTED
    # a row wider than the registers that hold it
    M, N, K, P = 256, 16384 + 128, 64, 2
    A = torch.zeros(M, K, dtype=torch.bfloat16, device="cuda")
    B = torch.zeros(K, N, dtype=torch.bfloat16, device="cuda")
    peer = torch.zeros(M, N, dtype=torch.bfloat16, device="cuda")
    R = torch.zeros(M // P, N, dtype=torch.bfloat16, device="cuda")
    gamma = torch.ones(N, dtype=torch.bfloat16, device="cuda")
    with E.Context(M, N, K, P) as ctx:
        with pytest.raises(E.EntwineError) as ei:
            ctx.gemm_rs_rmsnorm(A, B, [peer], 0, R, gamma, EPS)
        assert ei.value.status == E.EUNSUPPORTED
