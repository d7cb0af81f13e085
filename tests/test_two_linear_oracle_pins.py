"""Pins of the two-linears-per-side oracle (Sec. 3.2).

Each test reaches the same values by another route: float64 torch autograd of
the forward graph; central finite differences of the loss; the one-linear
oracle (itself pinned) when phi is the identity (the two layers collapse to
their product) or when the encoder's second layer is the r x r identity (the
encoder is then the one-linear encoder with W_e = W1).  Everything runs on
the CPU.
"""
import numpy as np
import pytest
import torch

from oracle import resbm_oracle as R
from oracle import two_linear_oracle as TL

ACTS = [R.ACT_IDENTITY, R.ACT_SILU]
GRAD_NAMES = ["x_attn", "z", "W1", "W2", "W3", "W4"]


def inputs(rng, T, n, m, r):
    s = lambda *shape, sc=1.0: rng.standard_normal(shape) * sc  # noqa: E731
    return {"x_attn": s(T, n), "z": s(T, n), "W1": s(n, m, sc=n ** -0.5), "W2": s(m, r, sc=m ** -0.5),
            "W3": s(r, m, sc=r ** -0.5), "W4": s(m, n, sc=m ** -0.5), "g_zt": s(T, n, sc=0.1),
            "g_id": s(T, n, sc=0.1)}


def loss(d, act):
    return TL.loss_and_grads(d["x_attn"], d["z"], d["W1"], d["W2"], d["W3"], d["W4"], d["g_zt"], d["g_id"], act)


@pytest.mark.parametrize("act", ACTS)
def test_gradients_torch_autograd(act):
    rng = np.random.default_rng(31 + act)
    T, n, m, r = 9, 24, 16, 8
    d = inputs(rng, T, n, m, r)
    t = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in d.items()}
    f = torch.nn.functional.silu if act == R.ACT_SILU else (lambda x: x)
    u = t["z"] @ t["W1"]
    b = t["x_attn"][:, :r] + f(u) @ t["W2"]
    zt = f(b @ t["W3"]) @ t["W4"]
    L = (t["g_zt"] * zt).sum() + (t["g_id"] * torch.nn.functional.pad(b, (0, n - r))).sum()
    tg = torch.autograd.grad(L, [t[k] for k in GRAD_NAMES])
    L_o, og = loss(d, act)
    assert abs(L_o - float(L.detach())) <= 1e-12 * max(1.0, abs(L_o))
    for k, g in zip(GRAD_NAMES, tg):
        np.testing.assert_allclose(og[k], g.numpy(), rtol=1e-11, atol=1e-13, err_msg=k)
    b_o, u_o = TL.encode2_fwd(d["x_attn"], d["z"], d["W1"], d["W2"], act)
    np.testing.assert_allclose(b_o, b.detach().numpy(), rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(u_o, u.detach().numpy(), rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("act", ACTS)
def test_gradients_finite_differences(act):
    """<grad L, D> against (L(x + hD) - L(x - hD)) / 2h for a random direction D of every input."""
    rng = np.random.default_rng(41 + act)
    d = inputs(rng, 5, 16, 8, 8)
    _, g = loss(d, act)
    h = 1e-5
    for k in GRAD_NAMES:
        D = rng.standard_normal(d[k].shape)
        up, dn = dict(d), dict(d)
        up[k], dn[k] = d[k] + h * D, d[k] - h * D
        fd = (loss(up, act)[0] - loss(dn, act)[0]) / (2 * h)
        an = float(np.sum(g[k] * D))
        assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), (k, fd, an)


def test_identity_phi_collapses_to_one_linear():
    """phi = identity: E(z) = z (W1 W2), D(b) = b (W3 W4), and the gradients follow the product."""
    rng = np.random.default_rng(5)
    T, n, m, r = 13, 32, 24, 8
    d = inputs(rng, T, n, m, r)
    We, Wd = d["W1"] @ d["W2"], d["W3"] @ d["W4"]
    b2, u = TL.encode2_fwd(d["x_attn"], d["z"], d["W1"], d["W2"], R.ACT_IDENTITY)
    b1, a = R.encode_fwd(d["x_attn"], d["z"], We, R.ACT_IDENTITY)
    np.testing.assert_allclose(b2, b1, rtol=1e-12, atol=1e-12)
    zt2, v = TL.decode2_fwd(b2, d["W3"], d["W4"], R.ACT_IDENTITY)
    np.testing.assert_allclose(zt2, R.decode_fwd(b1, Wd, False), rtol=1e-12, atol=1e-12)
    g_b2, dW3, dW4 = TL.decode2_bwd(b2, v, d["g_zt"], d["g_id"], d["W3"], d["W4"], R.ACT_IDENTITY)
    g_b1, dWd = R.decode_bwd(b1, Wd, d["g_zt"], d["g_id"])
    np.testing.assert_allclose(g_b2, g_b1, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dW3, dWd @ d["W4"].T, rtol=1e-12, atol=1e-12)   # dL/dW3 = dL/dW_d W4^T
    np.testing.assert_allclose(dW4, d["W3"].T @ dWd, rtol=1e-12, atol=1e-12)   # dL/dW4 = W3^T dL/dW_d
    g_z2, dW1, dW2 = TL.encode2_bwd(d["z"], u, g_b1, d["W1"], d["W2"], R.ACT_IDENTITY)
    g_z1, dWe = R.encode_bwd(d["z"], We, a, g_b1, R.ACT_IDENTITY)
    np.testing.assert_allclose(g_z2, g_z1, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dW1, dWe @ d["W2"].T, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dW2, d["W1"].T @ dWe, rtol=1e-12, atol=1e-12)


def test_unit_second_layer_is_one_linear_encoder():
    """W2 = I_r (m = r): b = x_attn P^id + phi(z W1), the one-linear encoder with W_e = W1 (SiLU)."""
    rng = np.random.default_rng(6)
    T, n, r = 17, 40, 8
    d = inputs(rng, T, n, r, r)
    I_r = np.eye(r)
    b2, u = TL.encode2_fwd(d["x_attn"], d["z"], d["W1"], I_r, R.ACT_SILU)
    b1, a = R.encode_fwd(d["x_attn"], d["z"], d["W1"], R.ACT_SILU)
    np.testing.assert_allclose(b2, b1, rtol=1e-13, atol=1e-13)
    g_b = rng.standard_normal((T, r))
    g_z2, dW1, dW2 = TL.encode2_bwd(d["z"], u, g_b, d["W1"], I_r, R.ACT_SILU)
    g_z1, dWe = R.encode_bwd(d["z"], d["W1"], a, g_b, R.ACT_SILU)
    np.testing.assert_allclose(g_z2, g_z1, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dW1, dWe, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dW2, R.phi(a, R.ACT_SILU).T @ g_b, rtol=1e-12, atol=1e-13)


def test_zero_branch_leaves_identity_path():
    """All-zero weights: b is the first r columns of x_attn, z~ = 0, and only g_id reaches g_b."""
    rng = np.random.default_rng(7)
    T, n, m, r = 6, 16, 8, 8
    d = inputs(rng, T, n, m, r)
    Z = {k: np.zeros_like(d[k]) for k in ("W1", "W2", "W3", "W4")}
    b, u = TL.encode2_fwd(d["x_attn"], d["z"], Z["W1"], Z["W2"], R.ACT_SILU)
    np.testing.assert_array_equal(b, d["x_attn"][:, :r])
    zt, v = TL.decode2_fwd(b, Z["W3"], Z["W4"], R.ACT_SILU)
    assert not np.any(zt)
    g_b, dW3, dW4 = TL.decode2_bwd(b, v, d["g_zt"], d["g_id"], Z["W3"], Z["W4"], R.ACT_SILU)
    np.testing.assert_array_equal(g_b, d["g_id"][:, :r])
    assert not np.any(dW3) and not np.any(dW4)      # phi(0) = 0 and g_v = 0
