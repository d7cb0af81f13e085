"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: the
elementwise definition of Eq. 4 used through Eq. 5, the composition law of
Eq. 6, the degenerate cases of Sec. 3.3 (full rank h = H; a zero branch
leaves only the identity path), linearity of the linear maps, central finite
differences, torch autograd in float64, scalar brute force, torch's own
float -> bf16 rounding and the byte counts printed in App. A.3.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
ACTS = [O.ACT_IDENTITY, O.ACT_SILU]


def rand(rng, *shape, scale=1.0):
    return scale * rng.standard_normal(shape)


def module_inputs(rng, T, n, r):
    return dict(x_attn=rand(rng, T, n), z=rand(rng, T, n),
                W_e=rand(rng, n, r, scale=n ** -0.5), W_d=rand(rng, r, n, scale=r ** -0.5),
                g_zt=rand(rng, T, n, scale=0.1), g_id=rand(rng, T, n, scale=0.1))


# ---------------------------------------------------------------- Eq. 4 / 5 / 6
@pytest.mark.parametrize("c,C", [(3, 7), (7, 3), (5, 5), (1, 4), (4, 1)])
def test_p_id_matches_rectangular_identity_product(c, C):
    """Eq. 5: the three stated cases equal x times the Eq. 4 matrix built elementwise."""
    rng = np.random.default_rng(1)
    x = rand(rng, 6, c)
    I = np.array([[1.0 if i == j else 0.0 for j in range(C)] for i in range(c)])
    np.testing.assert_array_equal(O.rect_identity(c, C), I)
    np.testing.assert_array_equal(O.p_id(x, C), x @ I)


def test_p_id_cases_worked_example():
    """Eq. 5 cases: pad appends zero columns, truncation drops the LAST columns."""
    x = np.array([[1.0, 2.0, 3.0], [4.0, 5.0, 6.0]])
    np.testing.assert_array_equal(O.p_id(x, 5), [[1, 2, 3, 0, 0], [4, 5, 6, 0, 0]])
    np.testing.assert_array_equal(O.p_id(x, 2), [[1, 2], [4, 5]])
    np.testing.assert_array_equal(O.p_id(x, 3), x)
    g = np.array([[7.0, 8.0, 9.0, 10.0]])
    np.testing.assert_array_equal(O.p_id_adjoint(g, 2), [[7, 8]])


@pytest.mark.parametrize("dims", [[8, 3, 8], [8, 3, 8, 5, 8], [4, 6, 2, 9], [5, 5, 5], [2, 7, 7, 3]])
def test_eq6_chain_of_identities(dims):
    """Eq. 6 (rank reading): the product of I_{c_i x c_{i+1}} is the c_0 x c_D matrix
    with ones at (i, i) for i < min over all c_i."""
    prod = np.eye(dims[0])
    for c, C in zip(dims[:-1], dims[1:]):
        prod = prod @ O.rect_identity(c, C)
    k = min(dims)
    expect = np.zeros((dims[0], dims[-1]))
    expect[np.arange(k), np.arange(k)] = 1.0
    np.testing.assert_array_equal(prod, expect)
    assert np.linalg.matrix_rank(prod) == k


def test_eq6_through_the_module_reading_a():
    """Two zero-weight boundaries n->r1->n->r2->n (reading A) pass x_attn's first
    min(r1, r2) columns and zero the rest."""
    rng = np.random.default_rng(2)
    T, n, r1, r2 = 5, 16, 6, 4
    x = rand(rng, T, n)
    for act in ACTS:
        h = x
        for r in (r1, r2):
            b, _ = O.encode_fwd(h, rand(rng, T, n), np.zeros((n, r)), act)
            h = O.decode_fwd(b, np.zeros((r, n)), add_identity=True)
        expect = x.copy()
        expect[:, min(r1, r2):] = 0.0
        np.testing.assert_array_equal(h, expect)


# ---------------------------------------------------------------- degenerate cases
@pytest.mark.parametrize("act", ACTS)
def test_zero_bottleneck_closed_form(act):
    """A zero encoder/decoder branch leaves only the identity path (Eq. 2 with F = 0)."""
    rng = np.random.default_rng(3)
    T, n, r = 7, 12, 4
    d = module_inputs(rng, T, n, r)
    W_e, W_d = np.zeros((n, r)), np.zeros((r, n))
    b, a = O.encode_fwd(d["x_attn"], d["z"], W_e, act)
    np.testing.assert_array_equal(a, 0.0)
    np.testing.assert_array_equal(b, d["x_attn"][:, :r])
    np.testing.assert_array_equal(O.decode_fwd(b, W_d, False), 0.0)
    zt_a = O.decode_fwd(b, W_d, True)
    np.testing.assert_array_equal(zt_a[:, :r], b)
    np.testing.assert_array_equal(zt_a[:, r:], 0.0)
    g_b, dW_d = O.decode_bwd(b, W_d, d["g_zt"], d["g_id"])
    np.testing.assert_array_equal(g_b, d["g_id"][:, :r])
    # dW_d is the outer-product sum over tokens, written as a scalar loop
    loop = np.zeros((r, n))
    for t in range(T):
        loop += np.outer(b[t], d["g_zt"][t])
    np.testing.assert_allclose(dW_d, loop, rtol=1e-13, atol=1e-15)
    g_z, dW_e = O.encode_bwd(d["z"], W_e, a, g_b, act)
    np.testing.assert_array_equal(g_z, 0.0)
    slope = 0.5 if act == O.ACT_SILU else 1.0      # SiLU'(0) = 1/2
    loop = np.zeros((n, r))
    for t in range(T):
        loop += slope * np.outer(d["z"][t], g_b[t])
    np.testing.assert_allclose(dW_e, loop, rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("act", ACTS)
def test_full_rank_reduces_to_standard_residual(act):
    """h = H (Sec. 3.3): P^id is I_H and Eq. 2 becomes Eq. 1, x + F(x)."""
    rng = np.random.default_rng(4)
    T, n = 6, 8
    x, z, W = rand(rng, T, n), rand(rng, T, n), rand(rng, n, n)
    b, a = O.encode_fwd(x, z, W, act)
    F = a / (1 + np.exp(-a)) if act == O.ACT_SILU else a
    np.testing.assert_allclose(b, x + F, rtol=1e-15, atol=1e-15)
    b0, _ = O.encode_fwd(x, z, np.zeros((n, n)), act)
    np.testing.assert_array_equal(b0, x)
    # vanilla residual through both halves with zero branches, reading A
    np.testing.assert_array_equal(O.decode_fwd(b0, np.zeros((n, n)), True), x)


def test_silu_values():
    """SiLU closed forms: phi(0) = 0, phi'(0) = 1/2, phi(a) -> a and phi'(a) -> 1 for
    large a, phi(a) -> 0 for very negative a."""
    a = np.array([0.0, 40.0, -40.0, 1.0])
    p = O.phi(a, O.ACT_SILU)
    dp = O.dphi(a, O.ACT_SILU)
    assert p[0] == 0.0 and dp[0] == 0.5
    assert abs(p[1] - 40.0) < 1e-15 * 40 and abs(dp[1] - 1.0) < 1e-15
    assert abs(p[2]) < 1e-15
    np.testing.assert_allclose(p[3], 1.0 / (1.0 + np.exp(-1.0)), rtol=1e-15)


# ---------------------------------------------------------------- linearity
def test_linearity():
    rng = np.random.default_rng(5)
    T, n, r = 9, 16, 4
    d, e = module_inputs(rng, T, n, r), module_inputs(rng, T, n, r)
    al, be = 0.7, -1.3
    tol = dict(rtol=1e-12, atol=1e-12)
    # decode_fwd is linear in b (both readings)
    b1, b2 = rand(rng, T, r), rand(rng, T, r)
    for add in (False, True):
        np.testing.assert_allclose(
            O.decode_fwd(al * b1 + be * b2, d["W_d"], add),
            al * O.decode_fwd(b1, d["W_d"], add) + be * O.decode_fwd(b2, d["W_d"], add), **tol)
    # decode_bwd is linear in (g_zt, g_id)
    gA = O.decode_bwd(b1, d["W_d"], d["g_zt"], d["g_id"])
    gB = O.decode_bwd(b1, d["W_d"], e["g_zt"], e["g_id"])
    gC = O.decode_bwd(b1, d["W_d"], al * d["g_zt"] + be * e["g_zt"], al * d["g_id"] + be * e["g_id"])
    for x, y, w in zip(gA, gB, gC):
        np.testing.assert_allclose(w, al * x + be * y, **tol)
    # encode_bwd is linear in g_b for fixed a
    for act in ACTS:
        _, a = O.encode_fwd(d["x_attn"], d["z"], d["W_e"], act)
        hA = O.encode_bwd(d["z"], d["W_e"], a, b1, act)
        hB = O.encode_bwd(d["z"], d["W_e"], a, b2, act)
        hC = O.encode_bwd(d["z"], d["W_e"], a, al * b1 + be * b2, act)
        for x, y, w in zip(hA, hB, hC):
            np.testing.assert_allclose(w, al * x + be * y, **tol)
        # the skip enters additively: b(x + delta) = b(x) + delta[:, :r]
        delta = rand(rng, T, n)
        bx, _ = O.encode_fwd(d["x_attn"], d["z"], d["W_e"], act)
        bxd, _ = O.encode_fwd(d["x_attn"] + delta, d["z"], d["W_e"], act)
        np.testing.assert_allclose(bxd, bx + delta[:, :r], **tol)
    # with phi = identity, encode_fwd is linear in (x_attn, z) and in W_e
    I = O.ACT_IDENTITY
    bA, _ = O.encode_fwd(d["x_attn"], d["z"], d["W_e"], I)
    bB, _ = O.encode_fwd(e["x_attn"], e["z"], d["W_e"], I)
    bC, _ = O.encode_fwd(al * d["x_attn"] + be * e["x_attn"], al * d["z"] + be * e["z"], d["W_e"], I)
    np.testing.assert_allclose(bC, al * bA + be * bB, **tol)
    zero = np.zeros_like(d["x_attn"])
    wA, _ = O.encode_fwd(zero, d["z"], d["W_e"], I)
    wB, _ = O.encode_fwd(zero, d["z"], e["W_e"], I)
    wC, _ = O.encode_fwd(zero, d["z"], al * d["W_e"] + be * e["W_e"], I)
    np.testing.assert_allclose(wC, al * wA + be * wB, **tol)


# ---------------------------------------------------------------- brute force
def brute_forward(x_attn, z, W_e, W_d, act, add_identity):
    """Scalar loops; the identity path uses Eq. 4's entries directly."""
    T, n = z.shape
    r = W_e.shape[1]
    a = np.zeros((T, r))
    b = np.zeros((T, r))
    zt = np.zeros((T, n))
    for t in range(T):
        for j in range(r):
            s = 0.0
            for k in range(n):
                s += z[t, k] * W_e[k, j]
            a[t, j] = s
            skip = 0.0
            for i in range(n):
                skip += x_attn[t, i] * (1.0 if i == j else 0.0)
            f = s / (1.0 + np.exp(-s)) if act == O.ACT_SILU else s
            b[t, j] = skip + f
        for c in range(n):
            s = 0.0
            for j in range(r):
                s += b[t, j] * W_d[j, c]
            if add_identity:
                for j in range(r):
                    s += b[t, j] * (1.0 if j == c else 0.0)
            zt[t, c] = s
    return a, b, zt


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("add_identity", [False, True])
@pytest.mark.parametrize("T,n,r", [(3, 8, 2), (4, 6, 6), (2, 10, 4)])
def test_forward_brute_force(act, add_identity, T, n, r):
    rng = np.random.default_rng(6)
    d = module_inputs(rng, T, n, r)
    a0, b0, zt0 = brute_forward(d["x_attn"], d["z"], d["W_e"], d["W_d"], act, add_identity)
    b, a = O.encode_fwd(d["x_attn"], d["z"], d["W_e"], act)
    zt = O.decode_fwd(b, d["W_d"], add_identity)
    np.testing.assert_allclose(a, a0, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(b, b0, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(zt, zt0, rtol=1e-13, atol=1e-14)


# ---------------------------------------------------------------- gradients
def module_loss(x_attn, z, W_e, W_d, G_zt, G_id, act, add_identity):
    """Scalar whose gradient the backward ops return.

    Reading B: the caller's output is P^id_{r->n}(b) + (something of z~), so
    L = <G_zt, z~> + <G_id, P^id(b)>.  Reading A: L = <G_zt, z~> with the pad in z~.
    """
    b, _ = O.encode_fwd(x_attn, z, W_e, act)
    zt = O.decode_fwd(b, W_d, add_identity)
    L = np.sum(G_zt * zt)
    if not add_identity:
        L += np.sum(G_id * O.p_id(b, z.shape[1]))
    return L


def oracle_grads(d, act, add_identity):
    g_id = d["g_zt"] if add_identity else d["g_id"]
    out = O.boundary_fwd_bwd(d["x_attn"], d["z"], d["W_e"], d["W_d"], d["g_zt"], g_id,
                             act, add_identity, wire_round=False)
    g_x = O.skip_grad(np.zeros_like(d["x_attn"]), out["g_b"])
    return {"x_attn": g_x, "z": out["g_z"], "W_e": out["dW_e"], "W_d": out["dW_d"]}


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("add_identity", [False, True])
@pytest.mark.parametrize("T,n,r", [(3, 8, 2), (5, 16, 4)])
def test_gradients_finite_differences(act, add_identity, T, n, r):
    rng = np.random.default_rng(7)
    d = module_inputs(rng, T, n, r)
    grads = oracle_grads(d, act, add_identity)
    h = 1e-6
    for name in ("x_attn", "z", "W_e", "W_d"):
        fd = np.zeros_like(d[name])
        for idx in np.ndindex(d[name].shape):
            p = {k: v.copy() for k, v in d.items()}
            m = {k: v.copy() for k, v in d.items()}
            p[name][idx] += h
            m[name][idx] -= h
            lp = module_loss(p["x_attn"], p["z"], p["W_e"], p["W_d"], d["g_zt"], d["g_id"], act, add_identity)
            lm = module_loss(m["x_attn"], m["z"], m["W_e"], m["W_d"], d["g_zt"], d["g_id"], act, add_identity)
            fd[idx] = (lp - lm) / (2 * h)
        err = np.linalg.norm(fd - grads[name]) / np.linalg.norm(grads[name])
        assert err < 1e-7, (name, err)


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("add_identity", [False, True])
def test_gradients_torch_autograd(act, add_identity):
    """Float64 torch autograd of the forward graph (slicing/padding for P^id)."""
    rng = np.random.default_rng(8)
    T, n, r = 11, 24, 8
    d = module_inputs(rng, T, n, r)
    tt = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in d.items()}
    a = tt["z"] @ tt["W_e"]
    f = torch.nn.functional.silu(a) if act == O.ACT_SILU else a
    b = tt["x_attn"][:, :r] + f
    zt = b @ tt["W_d"]
    pad_b = torch.nn.functional.pad(b, (0, n - r))
    if add_identity:
        zt = zt + pad_b
        L = (tt["g_zt"] * zt).sum()
    else:
        L = (tt["g_zt"] * zt).sum() + (tt["g_id"] * pad_b).sum()
    names = ["x_attn", "z", "W_e", "W_d"]
    tg = torch.autograd.grad(L, [tt[k] for k in names])
    og = oracle_grads(d, act, add_identity)
    for k, g in zip(names, tg):
        np.testing.assert_allclose(og[k], g.numpy(), rtol=1e-12, atol=1e-13)
    # forward values agree too
    b_o, a_o = O.encode_fwd(d["x_attn"], d["z"], d["W_e"], act)
    np.testing.assert_allclose(b_o, b.detach().numpy(), rtol=1e-13, atol=1e-14)


class _Wire(torch.autograd.Function):
    """The link of App. A.3 as a graph node: the payload crosses as bf16 on the
    way forward and its gradient crosses as bf16 on the way back (torch's own
    float -> bfloat16 conversion, via float32)."""

    @staticmethod
    def forward(ctx, x):
        return x.to(torch.float32).to(torch.bfloat16).to(torch.float64)

    @staticmethod
    def backward(ctx, g):
        return g.to(torch.float32).to(torch.bfloat16).to(torch.float64)


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("add_identity", [False, True])
def test_wire_rounded_chain_torch_autograd(act, add_identity):
    """The oracle's chain mode (wire_round=True) against float64 torch autograd
    of the forward graph with the link as a node that rounds to bf16 both ways:
    b is rounded before the decoder and its weight gradient, the wire gradient
    is rounded before the encoder backward, and a keeps its unrounded value."""
    rng = np.random.default_rng(12)
    T, n, r = 13, 40, 8
    d = module_inputs(rng, T, n, r)
    tt = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in d.items()}
    a = tt["z"] @ tt["W_e"]
    f = torch.nn.functional.silu(a) if act == O.ACT_SILU else a
    b = tt["x_attn"][:, :r] + f
    bw = _Wire.apply(b)
    bw.retain_grad()
    zt = bw @ tt["W_d"]
    pad_b = torch.nn.functional.pad(bw, (0, n - r))
    if add_identity:
        zt = zt + pad_b
        L = (tt["g_zt"] * zt).sum()
    else:
        L = (tt["g_zt"] * zt).sum() + (tt["g_id"] * pad_b).sum()
    names = ["x_attn", "z", "W_e", "W_d"]
    tg = dict(zip(names, torch.autograd.grad(L, [tt[k] for k in names] + [bw], retain_graph=False)[:4]))
    g_id = d["g_zt"] if add_identity else d["g_id"]
    out = O.boundary_fwd_bwd(d["x_attn"], d["z"], d["W_e"], d["W_d"], d["g_zt"], g_id, act, add_identity,
                             wire_round=True)
    np.testing.assert_array_equal(out["b_wire"], bw.detach().numpy())
    np.testing.assert_allclose(out["z_tilde"], zt.detach().numpy(), rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(out["dW_d"], tg["W_d"].numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(out["dW_e"], tg["W_e"].numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(out["g_z"], tg["z"].numpy(), rtol=1e-12, atol=1e-13)
    # the residual gradient on the encoder side is the rounded wire gradient on columns [0, r)
    np.testing.assert_allclose(O.skip_grad(np.zeros((T, n)), out["g_b_wire"]), tg["x_attn"].numpy(),
                               rtol=1e-12, atol=1e-13)
    # the rounding is not vacuous here: the unrounded chain differs
    plain = O.boundary_fwd_bwd(d["x_attn"], d["z"], d["W_e"], d["W_d"], d["g_zt"], g_id, act, add_identity,
                               wire_round=False)
    assert not np.array_equal(plain["b"], out["b_wire"])
    assert np.max(np.abs(plain["dW_e"] - out["dW_e"])) > 1e-6 * np.max(np.abs(plain["dW_e"]))


def test_skip_grad_is_adjoint_of_p_id():
    """<P^id(b), G> = <b, P^id^T(G)> for the encoder-side identity path."""
    rng = np.random.default_rng(9)
    b, G = rand(rng, 4, 3), rand(rng, 4, 10)
    lhs = np.sum(O.p_id(b, 10) * G)
    rhs = np.sum(b * O.p_id_adjoint(G, 3))
    assert abs(lhs - rhs) < 1e-13
    gx = rand(rng, 4, 10)
    out = O.skip_grad(gx, b)
    np.testing.assert_array_equal(out[:, 3:], gx[:, 3:])
    np.testing.assert_array_equal(out[:, :3], gx[:, :3] + b)


# ---------------------------------------------------------------- bf16 wire rounding
def _bf16_edge_values():
    f32 = np.float32
    vals = [0.0, -0.0, 1.0, -1.0, 1.00390625, 1.005859375, 1.0078125 + 2 ** -9,
            3.0e38, 3.3895314e38, 3.4e38, np.finfo(f32).max, 1e-40, 2 ** -133, 2 ** -134,
            3 * 2 ** -135, 2 ** -126, 2 ** -127 + 2 ** -134, np.inf, -np.inf]
    return np.array(vals, dtype=f32)


def test_rne_bf16_matches_torch_on_float32_inputs():
    """For float32 inputs, torch's float -> bfloat16 conversion is round-to-nearest-even."""
    rng = np.random.default_rng(10)
    bits = rng.integers(0, 2 ** 32, size=200000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = np.concatenate([x[np.isfinite(x)], _bf16_edge_values()])
    # ties: exactly half-way between bf16 neighbours, both parities
    ties = ((rng.integers(0, 2 ** 16, 5000).astype(np.uint32) << 16) | np.uint32(0x8000)).view(np.float32)
    x = np.concatenate([x, ties[np.isfinite(ties)]]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = O.rne_bf16(x.astype(np.float64))
    np.testing.assert_array_equal(got, ref)
    assert np.all(np.signbit(got) == np.signbit(ref))
    nan = O.rne_bf16(np.array([np.nan]))
    assert np.isnan(nan[0])


def test_rne_bf16_brute_force_nearest():
    """Float64 inputs: the result is the nearest of all finite bf16 values, ties to an
    even last bit, beyond the largest finite value plus half a step -> inf."""
    grid_bits = np.arange(0, 0x7F80, dtype=np.uint32)       # all finite non-negative bf16
    grid = (grid_bits << 16).view(np.float32).astype(np.float64)
    rng = np.random.default_rng(11)
    x = np.concatenate([
        np.exp(rng.uniform(np.log(1e-41), np.log(3e38), 3000)),
        (grid[1:200] + grid[:199]) / 2,                     # exact midpoints (subnormal)
        (grid[16000:16200] + grid[15999:16199]) / 2,        # exact midpoints (normal)
        grid[rng.integers(0, grid.size, 500)] * (1 + 1e-12),
    ])
    got = O.rne_bf16(x)
    for xi, gi in zip(x, got):
        dist = np.abs(grid - xi)
        best = np.flatnonzero(dist == dist.min())
        if best.size == 2:
            pick = best[(grid_bits[best] & 1) == 0][0]
        else:
            pick = best[0]
        assert gi == grid[pick], (xi, gi, grid[pick])
    top = grid[-1]
    half_step = (top - grid[-2]) / 2
    assert O.rne_bf16(np.array([top + half_step * 0.999]))[0] == top
    assert np.isinf(O.rne_bf16(np.array([top + half_step]))[0])
    assert O.rne_bf16(np.array([-(top + 2 * half_step)]))[0] == -np.inf


# ---------------------------------------------------------------- App. A.3 byte counts
def test_payload_bytes_match_paper():
    with open(os.path.join(GOLDEN, "payload_bytes.json")) as f:
        g = json.load(f)
    rng = np.random.default_rng(12)
    T = g["micro_batch"] * g["seq_len"]
    b = rand(rng, T, g["bottleneck"])
    full = rand(rng, T, g["hidden"])
    assert len(O.wire_payload(b)) == g["bytes_per_boundary_compressed"]
    assert len(O.wire_payload(full)) == g["bytes_per_boundary_uncompressed"]
    per_step = g["boundaries"] * g["directions"]
    assert per_step * len(O.wire_payload(b)) == g["bytes_per_step_compressed"]
    assert per_step * len(O.wire_payload(full)) == g["bytes_per_step_uncompressed"]
    assert g["bytes_per_step_compressed"] == 896 * 1024
    assert g["bytes_per_step_uncompressed"] == 112 * 1024 * 1024


def test_payload_layout():
    """Row-major [T][r], little-endian bf16, no header: 1.0 = 0x3F80, -2.0 = 0xC000."""
    b = np.array([[1.0, -2.0], [0.5, 3.0]])
    assert O.wire_payload(b) == bytes([0x80, 0x3F, 0x00, 0xC0, 0x00, 0x3F, 0x40, 0x40])


def test_compression_ratios():
    with open(os.path.join(GOLDEN, "compression.json")) as f:
        g = json.load(f)
    for case in g["cases"]:
        assert g["hidden"] / case["bottleneck"] == case["ratio"]
