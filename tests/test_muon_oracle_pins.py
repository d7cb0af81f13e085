"""Pins of the optimizer-side oracle (Newton-Schulz, Muon update, spectrum).

Each test checks the oracle against another route to the same value: the
scalar recurrence the iteration applies to every singular value of a matrix
built from chosen singular vectors and values; the orthogonal polar factor
from NumPy's SVD, which the cubic iteration converges to; equivariance under
transposition and invariance under positive scaling; closed forms of the
update for a zero gradient and of the momentum recurrence; and spectra of
matrices with constructed singular values.  Everything runs on the CPU.
"""
import numpy as np
import pytest

from oracle import muon_oracle as MU


def orthonormal(rng, rows, cols):
    """rows x cols with orthonormal columns (rows >= cols)."""
    q, r = np.linalg.qr(rng.standard_normal((rows, cols)))
    return q * np.sign(np.diag(r))


def built_uv(rng, L, s, sigma):
    """L x s matrix U diag(sigma) V^T with random orthonormal U (L x s) and V (s x s), and U, V."""
    U, V = orthonormal(rng, L, s), orthonormal(rng, s, s)
    return U @ np.diag(sigma) @ V.T, U, V


def scalar_ns(x, steps, coeffs):
    """The odd polynomial the iteration applies to each normalised singular value."""
    a, b, c = coeffs
    x = np.array(x, dtype=np.float64)
    for _ in range(steps):
        x = a * x + b * x ** 3 + c * x ** 5
    return x


SHAPES = [(64, 8), (40, 40), (200, 3), (17, 1)]


@pytest.mark.parametrize("L,s", SHAPES)
@pytest.mark.parametrize("wide", [False, True])
@pytest.mark.parametrize("coeffs,steps", [(MU.NS_QUINTIC, 5), (MU.NS_CUBIC, 7), ((2.0, -1.5, 0.5), 3)])
def test_newton_schulz_acts_on_singular_values(L, s, wide, coeffs, steps):
    """NS(U S V^T) = U f(S / ||S||) V^T with f the scalar recurrence (singular vectors kept)."""
    rng = np.random.default_rng(L * 31 + s)
    sigma = np.sort(rng.uniform(0.05, 3.0, s))[::-1]
    G, U, V = built_uv(rng, L, s, sigma)
    nrm = np.sqrt(np.sum(sigma ** 2))
    f = scalar_ns(sigma / (nrm + MU.NS_EPS), steps, coeffs)
    expect = U @ np.diag(f) @ V.T
    got = MU.newton_schulz(G.T if wide else G, steps, coeffs)
    np.testing.assert_allclose(got.T if wide else got, expect, rtol=0, atol=1e-12 * max(1.0, np.abs(f).max()))


@pytest.mark.parametrize("L,s", [(96, 12), (50, 50), (300, 7)])
def test_cubic_iteration_reaches_polar_factor(L, s):
    """(1.5, -0.5, 0) converges to the orthogonal polar factor U V^T of U S V^T."""
    rng = np.random.default_rng(7 + s)
    G = rng.standard_normal((L, s))
    u, _, vt = np.linalg.svd(G, full_matrices=False)
    got = MU.newton_schulz(G, 80, MU.NS_CUBIC)
    np.testing.assert_allclose(got, u @ vt, rtol=0, atol=1e-11)
    np.testing.assert_allclose(got.T @ got, np.eye(s), rtol=0, atol=1e-11)


def test_newton_schulz_transpose_and_scale():
    rng = np.random.default_rng(3)
    G = rng.standard_normal((120, 10))
    O1 = MU.newton_schulz(G, 5, MU.NS_QUINTIC, eps=0.0)
    np.testing.assert_allclose(MU.newton_schulz(G.T, 5, MU.NS_QUINTIC, eps=0.0), O1.T, rtol=0, atol=1e-13)
    np.testing.assert_allclose(MU.newton_schulz(37.5 * G, 5, MU.NS_QUINTIC, eps=0.0), O1, rtol=0, atol=1e-13)


def test_newton_schulz_of_zero_is_zero():
    assert not np.any(MU.newton_schulz(np.zeros((9, 4))))


def test_quintic_singular_values_land_near_one():
    """The quintic's purpose: 5 steps take every normalised singular value in [2e-3, 1] into [0.68, 1.21]."""
    x = np.logspace(np.log10(2e-3), 0, 4000)
    f = scalar_ns(x, 5, MU.NS_QUINTIC)
    assert f.min() > 0.68 and f.max() < 1.21
    rng = np.random.default_rng(5)
    sigma = np.logspace(0, -2, 16)
    G, _, _ = built_uv(rng, 200, 16, sigma)
    sv = np.linalg.svd(MU.newton_schulz(G), compute_uv=False)
    assert sv.min() > 0.68 and sv.max() < 1.21


def test_muon_update_zero_gradient_is_pure_decay():
    rng = np.random.default_rng(11)
    W = MU.to_f32(rng.standard_normal((64, 8)))
    Z = np.zeros_like(W)
    W1, M1, O = MU.muon_update(W, Z, Z, lr=0.01, momentum=0.95, weight_decay=0.1)
    assert not np.any(O) and not np.any(M1)
    np.testing.assert_array_equal(W1, MU.to_f32(W - 0.01 * 0.1 * W))


def test_muon_update_momentum_recurrence_and_direction():
    """Two steps: M_2 = f32(mu f32(G_1) + G_2); W moves along -lr scale NS(M) (or NS(G + mu M))."""
    rng = np.random.default_rng(12)
    p, q, lr, mu = 32, 96, 0.02, 0.9
    W = MU.to_f32(rng.standard_normal((p, q)) * 0.1)
    G1 = MU.to_f32(rng.standard_normal((p, q)))
    G2 = MU.to_f32(rng.standard_normal((p, q)))
    M0 = np.zeros((p, q))
    for nesterov in (False, True):
        W1, M1, _ = MU.muon_update(W, G1, M0, lr, mu, nesterov=nesterov)
        np.testing.assert_array_equal(M1, G1)
        W2, M2, O2 = MU.muon_update(W1, G2, M1, lr, mu, nesterov=nesterov)
        np.testing.assert_array_equal(M2, MU.to_f32(mu * G1 + G2))
        U = G2 + mu * M2 if nesterov else M2
        # the applied direction has U's singular vectors (checked through NS's spectral action)
        u, sv, vt = np.linalg.svd(U, full_matrices=False)
        f = scalar_ns(sv / (np.sqrt(np.sum(sv ** 2)) + MU.NS_EPS), 5, MU.NS_QUINTIC)
        np.testing.assert_allclose(O2, u @ np.diag(f) @ vt, rtol=0, atol=1e-12)
        scale = 0.2 * np.sqrt(q)
        np.testing.assert_allclose(W2, W1 - lr * scale * O2, rtol=0, atol=4e-7 * np.abs(W1).max())


@pytest.mark.parametrize("L,s", [(128, 32), (32, 128), (90, 9), (5, 5)])
def test_spectrum_of_built_matrices(L, s):
    rng = np.random.default_rng(L + s)
    k = min(L, s)
    sigma = np.sort(rng.uniform(0.1, 4.0, k))[::-1]
    if L >= s:
        W, _, _ = built_uv(rng, L, s, sigma)
    else:
        W, _, _ = built_uv(rng, s, L, sigma)
        W = W.T
    sv, r_eff = MU.spectrum(W)
    np.testing.assert_allclose(sv, sigma, rtol=1e-12)
    assert abs(r_eff - np.sum(sigma ** 2) / sigma[0] ** 2) < 1e-12 * k


def test_spectrum_extremes():
    rng = np.random.default_rng(21)
    Q = orthonormal(rng, 64, 16)
    assert abs(MU.spectrum(Q)[1] - 16.0) < 1e-12            # all singular values equal: r_eff = b
    u, v = rng.standard_normal(64), rng.standard_normal(16)
    assert abs(MU.spectrum(np.outer(u, v))[1] - 1.0) < 1e-12  # one direction: r_eff = 1
    assert MU.spectrum(np.zeros((8, 4)))[1] == 0.0
