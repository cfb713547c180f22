"""Pins for the CPU oracle's arithmetic: each test checks the oracle against
something other than itself (bit patterns fixed by the bfloat16 format, exact
rational brute force, closed forms, invariants, and the rounding bound of an
emulated bf16/fp32 pipeline), so that a dropped term, a wrong sign, a wrong
row chunk or a transposed operand fails at least one of them."""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from oracle import reduce_scatter as rs
from paper_2609_11562_amd.inputs import Dist, draw_bf16, make_problem, to_bf16_bits
from paper_2609_11562_amd.workloads import WORKLOADS


# ---------------------------------------------------------------- decoding
def test_bf16_decode_fixed_patterns():
    # Values fixed by the bfloat16 format (sign, 8-bit exponent bias 127, 7-bit fraction).
    pats = {0x3F80: 1.0, 0xC000: -2.0, 0x0000: 0.0, 0x3F81: 1.0 + 2.0 ** -7,
            0x4049: 3.140625, 0x0001: 2.0 ** -133, 0x7F7F: (2 - 2.0 ** -7) * 2.0 ** 127,
            0x3C00: 2.0 ** -7}
    got = rs.bf16_to_f64(np.array(list(pats), dtype=np.uint16))
    assert got.tolist() == list(pats.values())
    neg0 = rs.bf16_to_f64(np.array([0x8000], dtype=np.uint16))[0]
    assert neg0 == 0.0 and np.signbit(neg0)
    assert np.isinf(rs.bf16_to_f64(np.array([0xFF80], dtype=np.uint16))[0])
    assert np.isnan(rs.bf16_to_f64(np.array([0x7FC0], dtype=np.uint16))[0])


def test_bf16_decode_matches_torch():
    bits = np.random.default_rng(1).integers(0, 2 ** 16, size=4096, dtype=np.uint16)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    got = rs.bf16_to_f64(bits)
    finite = np.isfinite(ref)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    assert np.array_equal(got[finite], ref[finite])


# ---------------------------------------------------------- brute force
def _exact_reference(A, B, peers, P, dest):
    """Exact rational triple loop, written without numpy arithmetic."""
    a = [[Fraction(float(v)) for v in row] for row in rs.bf16_to_f64(A)]
    b = [[Fraction(float(v)) for v in row] for row in rs.bf16_to_f64(B)]
    pk = [[[Fraction(float(v)) for v in row] for row in rs.bf16_to_f64(pq)] for pq in peers]
    M, K, N = len(a), len(b), len(b[0])
    h = M // P
    dests = range(P) if dest == -1 else [dest]
    out = []
    for d in dests:
        for i in range(d * h, (d + 1) * h):
            row = []
            for j in range(N):
                acc = Fraction(0)
                for k in range(K):
                    acc += a[i][k] * b[k][j]
                for q in range(P - 1):
                    acc += pk[q][i][j]
                row.append(acc)
            out.append(row)
    return out


@pytest.mark.parametrize("M,N,K,P", [(8, 6, 5, 2), (12, 4, 7, 3), (16, 3, 9, 4), (6, 5, 3, 1)])
@pytest.mark.parametrize("dest_kind", ["first", "last", "all"])
def test_oracle_matches_exact_brute_force(M, N, K, P, dest_kind):
    dest = {"first": 0, "last": P - 1, "all": -1}[dest_kind]
    prob = make_problem(M, N, K, P, Dist("normal", 1.0), Dist("normal", 3.0), seed=77 + M)
    got = oracle.gemm_reduce_scatter(prob.A, prob.B, prob.peers, P, dest)
    exact = _exact_reference(prob.A, prob.B, prob.peers, P, dest)
    assert got.shape == (len(exact), N)
    for i, row in enumerate(exact):
        for j, v in enumerate(row):
            # float64 sum of K + P exactly representable terms.
            assert abs(got[i, j] - float(v)) <= (K + P) * 2.0 ** -52 * (abs(float(v)) + 64)


def test_integer_inputs_are_exact():
    M, N, K, P = 32, 24, 96, 4
    prob = make_problem(M, N, K, P, Dist("int", 1), Dist("int", 16), seed=5)
    got = oracle.gemm_reduce_scatter(prob.A, prob.B, prob.peers, P, -1)
    a = rs.bf16_to_f64(prob.A).astype(np.int64)
    b = rs.bf16_to_f64(prob.B).astype(np.int64)
    exact = [[sum(int(a[i, k]) * int(b[k, j]) for k in range(K)) + sum(
        int(rs.bf16_to_f64(pq)[i, j]) for pq in prob.peers) for j in range(N)] for i in range(M)]
    assert np.array_equal(got, np.array(exact, dtype=np.float64))
    assert np.abs(got).max() <= 96 + 3 * 16


# ---------------------------------------------------------- closed forms
def test_closed_form_ones():
    M, N, K, P = 16, 8, 12, 4
    A = to_bf16_bits(np.ones((M, K), np.float32))
    B = to_bf16_bits(np.ones((K, N), np.float32))
    peers = [to_bf16_bits(np.full((M, N), c, np.float32)) for c in (0.5, -3.0, 8.0)]
    out = oracle.gemm_reduce_scatter(A, B, peers, P, -1)
    assert np.all(out == K + 0.5 - 3.0 + 8.0)


def test_closed_form_row_selection():
    """A picks row (i mod K) of B, and every peer holds its own row index,
    so chunk d must contain B[i mod K] + (P-1) * i for exactly its rows i."""
    M, N, K, P = 24, 10, 6, 3
    A = np.zeros((M, K), np.float32)
    A[np.arange(M), np.arange(M) % K] = 1.0
    Bv = np.arange(K * N, dtype=np.float32).reshape(K, N) - 20
    rowidx = np.repeat(np.arange(M, dtype=np.float32)[:, None], N, axis=1)
    peers = [to_bf16_bits(rowidx) for _ in range(P - 1)]
    for d in range(P):
        got = oracle.gemm_reduce_scatter(to_bf16_bits(A), to_bf16_bits(Bv), peers, P, d)
        rows = np.arange(d * M // P, (d + 1) * M // P)
        want = Bv[rows % K] + (P - 1) * rows[:, None]
        assert np.array_equal(got, want)


def test_transpose_identity_nonsquare():
    """(A B)^T = B^T A^T with P = 1 on a non-square shape: a transposed or
    swapped operand inside the oracle breaks it."""
    prob = make_problem(8, 5, 3, 1, Dist("uniform", 1.0), Dist("normal", 1.0), seed=3)
    ab = oracle.gemm_reduce_scatter(prob.A, prob.B, [], 1, 0)
    ba = oracle.gemm_reduce_scatter(prob.B.T.copy(), prob.A.T.copy(), [], 1, 0)
    assert ab.shape == (8, 5)
    assert np.allclose(ab.T, ba, rtol=0, atol=1e-12)


# ---------------------------------------------------------- invariants
def test_chunks_concatenate_to_all():
    w = WORKLOADS["tiny_512x256x1024_p2"]
    prob = w.problem(seed=11)
    full = oracle.gemm_reduce_scatter(prob.A, prob.B, prob.peers, w.P, -1)
    parts = [oracle.gemm_reduce_scatter(prob.A, prob.B, prob.peers, w.P, d) for d in range(w.P)]
    assert np.array_equal(np.concatenate(parts, axis=0), full)


def test_single_chunk_is_plain_product():
    prob = make_problem(64, 32, 40, 1, Dist("normal", 1.0), Dist("normal", 1.0), seed=4)
    got = oracle.gemm_reduce_scatter(prob.A, prob.B, [], 1, 0)
    ref = (torch.from_numpy(rs.bf16_to_f64(prob.A)) @ torch.from_numpy(rs.bf16_to_f64(prob.B))).numpy()
    assert np.allclose(got, ref, rtol=1e-13, atol=1e-12)


def test_linearity_in_peers_and_sampled_rows():
    M, N, K, P = 32, 16, 8, 4
    prob = make_problem(M, N, K, P, Dist("normal", 1.0), Dist("normal", 1.0), seed=9)
    base = oracle.gemm_reduce_scatter(prob.A, prob.B, prob.peers, P, -1)
    zero = [to_bf16_bits(np.zeros((M, N), np.float32))] * (P - 1)
    gemm_only = oracle.gemm_reduce_scatter(prob.A, prob.B, zero, P, -1)
    peer_sum = sum(rs.bf16_to_f64(p) for p in prob.peers)
    assert np.allclose(base, gemm_only + peer_sum, rtol=1e-14, atol=1e-13)
    rows = [0, 7, 8, 31]
    assert np.array_equal(oracle.output_rows(prob.A, prob.B, prob.peers, rows), base[rows])


# ---------------------------------------------------------- error bound
def _emulated_path(A, B, peers, P):
    """bf16 x bf16 -> fp32 GEMM, bf16 partial, fp32 sum in rank order, bf16 out."""
    a = torch.from_numpy(rs.bf16_to_f64(A)).float()
    b = torch.from_numpy(rs.bf16_to_f64(B)).float()
    c = (a @ b).to(torch.bfloat16).float()
    acc = c.clone()
    for pq in peers:
        acc += torch.from_numpy(rs.bf16_to_f64(pq)).float()
    return acc.to(torch.bfloat16).to(torch.float64).numpy()


@pytest.mark.parametrize("name", ["tiny_512x256x1024_p2"])
def test_emulated_pipeline_within_bound_and_gate(name):
    w = WORKLOADS[name]
    prob = w.problem()
    ref = oracle.gemm_reduce_scatter(prob.A, prob.B, prob.peers, w.P, -1)
    got = _emulated_path(prob.A, prob.B, prob.peers, w.P)
    rows = np.arange(w.M)
    bound = oracle.error_bound_rows(prob.A, prob.B, prob.peers, rows)
    assert np.all(np.abs(got - ref) <= bound)
    assert np.all(oracle.paper_gate(got, ref))


def test_bound_rejects_plausible_mistakes():
    M, N, K, P = 64, 32, 256, 4
    prob = make_problem(M, N, K, P, Dist("normal", 0.02), Dist("normal", 0.02 * 0.02 * 16), seed=21)
    rows = np.arange(M)
    ref = oracle.gemm_reduce_scatter(prob.A, prob.B, prob.peers, P, -1)
    bound = oracle.error_bound_rows(prob.A, prob.B, prob.peers, rows)
    good = _emulated_path(prob.A, prob.B, prob.peers, P)
    assert np.all(np.abs(good - ref) <= bound)
    dropped = _emulated_path(prob.A, prob.B, prob.peers[:-1] + [to_bf16_bits(np.zeros((M, N), np.float32))], P)
    assert np.any(np.abs(dropped - ref) > bound)
    flipped = _emulated_path(prob.A, prob.B, prob.peers[:-1] + [prob.peers[-1] ^ np.uint16(0x8000)], P)
    assert np.any(np.abs(flipped - ref) > bound)
    shifted = np.roll(good, M // P, axis=0)          # wrong row chunk
    assert np.any(np.abs(shifted - ref) > bound)
    bt = _emulated_path(prob.A, to_bf16_bits(np.ascontiguousarray(
        rs.bf16_to_f64(prob.B)[::-1]).astype(np.float32)), prob.peers, P)  # wrong K index
    assert np.any(np.abs(bt - ref) > bound)


def test_paper_gate_edges():
    ref = np.array([0.0, 1.0, -10.0])
    tol = 0.1 + 0.05 * np.abs(ref)
    assert np.all(oracle.paper_gate(ref + tol * 0.999, ref))
    assert not np.any(oracle.paper_gate(ref + tol * 1.001, ref))


def test_input_generator_is_seeded_and_rounded():
    a1 = draw_bf16(123, (64, 64), Dist("normal", 0.02))
    a2 = draw_bf16(123, (64, 64), Dist("normal", 0.02))
    assert a1.dtype == np.uint16 and np.array_equal(a1, a2)
    v = rs.bf16_to_f64(a1)
    assert 0.015 < v.std() < 0.025


# ---------------------------------------------------------- reducer arithmetic
def test_rne_encoder_fixed_cases():
    cases = {1.0: 0x3F80, -2.0: 0xC000, 1.0 + 2.0 ** -8: 0x3F80,            # tie -> even (down)
             1.0 + 3 * 2.0 ** -8: 0x3F82,                                      # tie -> even (up)
             1.0 + 2.0 ** -8 + 2.0 ** -20: 0x3F81, float("inf"): 0x7F80, 0.0: 0x0000,
             (2 - 2.0 ** -7) * 2.0 ** 127: 0x7F7F,                             # largest finite
             (2 - 2.0 ** -8) * 2.0 ** 127: 0x7F80}                             # tie above it -> inf
    got = rs.f32_to_bf16_rne_bits(np.array(list(cases), dtype=np.float32))
    assert got.tolist() == list(cases.values())
    assert np.isnan(rs.bf16_to_f64(rs.f32_to_bf16_rne_bits(np.array([np.nan], np.float32))))[0]


def test_rne_encoder_matches_torch():
    x = np.random.default_rng(2).standard_normal(1 << 16).astype(np.float32) * 1e3
    x[::7] = np.float32(1.0) + np.float32(2.0 ** -8) * np.arange(len(x[::7]), dtype=np.float32) % 4
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(rs.f32_to_bf16_rne_bits(x), ref)


def test_reduce_tile_order_matters_and_is_rank_order():
    # fp32 addition is not associative: 2^24 + 1 - 2^24 depends on the order.
    big, one = to_bf16_bits(np.array([2.0 ** 24], np.float32)), to_bf16_bits(np.array([1.0], np.float32))
    nbig = to_bf16_bits(np.array([-(2.0 ** 24)], np.float32))
    got = rs.reduce_tile_f32(big, [one, nbig])          # (2^24 + 1) - 2^24 = 0 in fp32
    assert rs.bf16_to_f64(got).tolist() == [0.0]
    got = rs.reduce_tile_f32(big, [nbig, one])          # (2^24 - 2^24) + 1 = 1
    assert rs.bf16_to_f64(got).tolist() == [1.0]


def test_reduce_tile_matches_emulation_and_oracle_bound():
    M, N, P = 32, 64, 8
    prob = make_problem(M, N, 8, P, Dist("normal", 1.0), Dist("normal", 0.5), seed=31)
    part = to_bf16_bits(np.random.default_rng(3).standard_normal((M, N)).astype(np.float32))
    acc = torch.from_numpy(rs.bf16_to_f64(part)).float()
    for pq in prob.peers:
        acc = acc + torch.from_numpy(rs.bf16_to_f64(pq)).float()
    ref = acc.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(rs.reduce_tile_f32(part, prob.peers), ref)
