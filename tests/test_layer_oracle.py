"""Pins for the layer-epilogue oracle (residual addition + RMSNorm after the
reduce-scatter; paper Section 5.2, layer-level performance): a library
routine, closed forms, an invariance, bit-exactness of the fp32 emulation
and the bounds' power to reject plausible mistakes."""
import numpy as np
import pytest
import torch

from oracle import layer as L
from oracle import reduce_scatter as R
from paper_2609_11562_amd.inputs import Dist, draw_bf16, to_bf16_bits


def _bits(x):
    return to_bf16_bits(np.asarray(x, dtype=np.float32))


def test_rmsnorm_matches_torch_rms_norm():
    rng = np.random.default_rng(3)
    h = rng.standard_normal((16, 256))
    gamma = _bits(rng.uniform(0.5, 1.5, 256))
    eps = 1e-5
    want = torch.nn.functional.rms_norm(torch.from_numpy(h), (256,), torch.from_numpy(R.bf16_to_f64(gamma)), eps)
    assert np.allclose(L.rmsnorm(h, gamma, eps), want.numpy(), rtol=1e-13, atol=0)


def test_closed_forms():
    N = 64
    gamma = _bits(np.linspace(0.5, 2.0, N))
    g = R.bf16_to_f64(gamma)
    # constant row c: mean square c^2, so y = gamma c / sqrt(c^2 + eps)
    c, eps = -3.0, 0.25
    y = L.rmsnorm(np.full((1, N), c), gamma, eps)
    assert np.allclose(y[0], g * c / np.sqrt(c * c + eps), rtol=1e-15)
    # a single nonzero a: mean square a^2 / N; with eps = 0, y_0 = gamma_0 sign(a) sqrt(N)
    h = np.zeros((1, N))
    h[0, 5] = 7.0
    y = L.rmsnorm(h, gamma, 0.0)
    assert y[0, 5] == pytest.approx(g[5] * np.sqrt(N), rel=1e-15)
    assert np.count_nonzero(y) == 1


def test_scale_invariance_without_eps():
    rng = np.random.default_rng(4)
    h = rng.standard_normal((4, 128))
    gamma = _bits(np.ones(128))
    assert np.allclose(L.rmsnorm(3.5 * h, gamma, 0.0), L.rmsnorm(h, gamma, 0.0), rtol=1e-14)


def test_residual_add_is_exact_sum():
    rng = np.random.default_rng(5)
    O = rng.standard_normal((8, 32))
    Rb = _bits(rng.standard_normal((8, 32)))
    assert np.array_equal(L.residual_add(O, Rb), O + R.bf16_to_f64(Rb))


def test_residual_add_f32_matches_torch_float32_chain():
    rng = np.random.default_rng(6)
    part, peers, res = [_bits(rng.standard_normal((16, 128))) for _ in range(3)]
    peers = [peers, _bits(rng.standard_normal((16, 128)))]
    t = lambda b: torch.from_numpy(R.bf16_to_f64(b)).to(torch.float32)
    acc = t(part)
    for p in peers:
        acc = acc + t(p)
    acc = acc + t(res)
    want = acc.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(L.residual_add_f32(part, peers, res), want)


def _emulate_device(A, B, peers, Rb, gamma, eps, rows, mistake=None):
    """Float32 emulation of the fused path on the given rows, with an
    optional planted mistake; returns (h_bf16_as_f64, y_as_f64)."""
    a = torch.from_numpy(R.bf16_to_f64(A[rows])).float()
    b = torch.from_numpy(R.bf16_to_f64(B)).float()
    acc = (a @ b).to(torch.bfloat16).float()
    for q, p in enumerate(peers):
        if mistake == "drop_peer" and q == 0:
            continue
        acc = acc + torch.from_numpy(R.bf16_to_f64(p[rows])).float()
    if mistake != "drop_residual":
        acc = acc + torch.from_numpy(R.bf16_to_f64(Rb)).float()
    h = acc.to(torch.bfloat16).float()
    N = h.shape[1]
    ms = (h * h).sum(dim=1, keepdim=True) / (N - 1 if mistake == "n_minus_1" else N)
    r = torch.rsqrt(ms) + eps if mistake == "eps_outside" else torch.rsqrt(ms + eps)
    g = torch.from_numpy(R.bf16_to_f64(gamma)).float()
    y = h * r * (1.0 if mistake == "no_gamma" else g)
    return h.double().numpy(), y.to(torch.bfloat16).double().numpy()


@pytest.mark.parametrize("mistake", [None, "drop_peer", "drop_residual", "n_minus_1", "eps_outside", "no_gamma"])
def test_bounds_accept_the_path_and_reject_mistakes(mistake):
    # Short rows and a large eps, so that adding eps outside the root moves y
    # by more than bf16 resolution; rows of 8 for the N - 1 divisor (a 14%
    # change of the mean), with a small eps.
    M, N, K, P = 64, (8 if mistake == "n_minus_1" else 32), 96, 4
    A = draw_bf16(11, (M, K), Dist("normal", 0.05))
    B = draw_bf16(12, (K, N), Dist("normal", 0.05))
    peers = [draw_bf16(13 + q, (M, N), Dist("normal", 0.02)) for q in range(P - 1)]
    rows = np.arange(16, 32)
    Rb = draw_bf16(20, (len(rows), N), Dist("normal", 0.5))
    gamma = to_bf16_bits(np.random.default_rng(21).uniform(0.5, 1.5, N).astype(np.float32))
    eps = 1e-5 if mistake == "n_minus_1" else 0.25
    O = R.output_rows(A, B, peers, rows)
    h, y = L.layer(O, Rb, gamma, eps)
    hb = L.h_bound(R.error_bound_rows(A, B, peers, rows, final_rounding=False), h, Rb)
    yb = L.y_bound(h, hb, gamma, eps)
    h_dev, y_dev = _emulate_device(A, B, peers, Rb, gamma, eps, rows, mistake)
    ok = np.all(np.abs(h_dev - h) <= hb) and np.all(np.abs(y_dev - y) <= yb)
    assert ok == (mistake is None)
