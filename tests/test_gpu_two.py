"""Two-linears-per-side ops (resbm2_*) against the float64 oracle.

Inputs are seeded bf16 tensors; the oracle computes in float64 on the same
values.  Bound (as for the one-linear ops): max error <= 2e-2 RMS(ref), after
a half-ulp discount for bf16 outputs, with no further allowance.  Error
budget: the GPU rounds phi(u), phi(v) (formed from the float32 accumulator),
g_u and g_v to bf16 once before the next product (relative 2^-9 per element,
averaging out over the contraction) and accumulates in float32.  Beside the
exact oracle every output is also compared with a float64 reference that takes
exactly those roundings (``spec_*`` below), to the same bound.
Small shapes are checked everywhere, a fixed-seed sweep of 24 random small
shapes stresses short contractions, and the full 16384-token shape is checked
on sampled rows (row-local outputs) and sampled columns (token sums).
"""
import numpy as np
import pytest
import torch

from oracle import resbm_oracle as R
from oracle import two_linear_oracle as TL
from gpu_helpers import check, errors, f64, guarded, lib, say, strided
from paper_2604_11947_amd import inputs as I

pytestmark = pytest.mark.gpu

SHAPES = [(333, 520, 136, 40), (1000, 256, 1024, 32), (64, 64, 8, 8), (1, 128, 64, 16), (513, 384, 520, 128)]
IDS = [f"T{T}_n{n}_m{m}_r{r}" for T, n, m, r in SHAPES]
ACTS = [R.ACT_IDENTITY, R.ACT_SILU]


def data(T, n, m, r, seed=0):
    d = I.make_activations(T, n, "normal", seed)
    d.update(I.make_two_weights(n, m, r, seed))
    d["b"] = I.make_bf16(T, r, seed + 11)
    d["u"] = I.make_bf16(T, m, seed + 12)
    d["v"] = I.make_bf16(T, m, seed + 13)
    d["g_b"] = I.make_bf16(T, r, seed + 14, std=0.1)
    return d


def np64(d, k):
    return d[k].to(torch.float64).numpy()


# Float64 references that round the op-formed intermediates to bf16 where the
# kernels are specified to (include/resbm.h): phi(u), phi(v), g_u, g_v.  They
# use the oracle's bf16 rounding and its phi / phi'; the exact oracle itself
# stays unrounded.
def rb(x):
    return R.rne_bf16(x)


def spec_encode2_fwd(x, z, W1, W2, act):
    u = z @ W1
    return R.p_id(x, W2.shape[1]) + rb(R.phi(u, act)) @ W2


def spec_decode2_fwd(b, W3, W4, act):
    return rb(R.phi(b @ W3, act)) @ W4


def spec_decode2_bwd(b, v, g_zt, g_id, W3, W4, act):
    g_v = rb((g_zt @ W4.T) * R.dphi(v, act))
    g_b = g_v @ W3.T
    if g_id is not None:
        g_b = g_b + R.p_id(g_id, W3.shape[0])
    return g_b, b.T @ g_v, rb(R.phi(v, act)).T @ g_zt


def spec_encode2_bwd(z, u, g_b, W1, W2, act):
    g_u = rb((g_b @ W2.T) * R.dphi(u, act))
    return g_u @ W1.T, z.T @ g_u, rb(R.phi(u, act)).T @ g_b


# A weight gradient dW = A^T B (a sum over T tokens) in which one factor is an
# op-formed bf16 intermediate (phi(u), phi(v), g_u, g_v) inherits that factor's
# rounding, up to 2^-9 of |A_t||B_t| per term.  Over many tokens it averages
# out; over a handful it does not (at T = 1 the gradient is one outer product
# and its elementwise relative error is the rounding itself), so below
# FEW_TOKENS the exact-oracle check of a weight gradient discounts exactly that
# worst case, 2^-9 sum_t |A_t||B_t| (the weight-gradient counterpart of the
# half-ulp discount of bf16 outputs), and the specified-rounding check, which
# could differ by one flipped rounding of a factor, only reports.  Row
# products (b, z~, g_b, g_z) and every output at T >= FEW_TOKENS get no
# allowance.
FEW_TOKENS = 16


def token_sum_rounding(A, B):
    return 2.0 ** -9 * (np.abs(A).T @ np.abs(B))


def both(name, gpu, ref, spec, bf16_output, factors=None):
    """The exact oracle and the specified-rounding reference, each to the plain
    bound; `factors` (A, B) marks a weight gradient A^T B (see FEW_TOKENS)."""
    few = factors is not None and factors[0].shape[0] < FEW_TOKENS
    check(name, gpu, ref, bf16_output, allow=token_sum_rounding(*factors) if few else None)
    if few:
        e = errors(f64(gpu), spec, bf16_output)
        say(f"    {name + ' spec':10s} raw={e['raw']:.2e} (reported only: {factors[0].shape[0]} tokens)")
    else:
        check(name + " spec", gpu, spec, bf16_output)


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("T,n,m,r", SHAPES, ids=IDS)
def test_encode2_fwd(T, n, m, r, act):
    L = lib()
    say(f"encode2_fwd T={T} n={n} m={m} r={r} act={act}")
    d = data(T, n, m, r)
    x, z = strided(d["x_attn"].cuda(), 8), strided(d["z"].cuda(), 24)
    b, _, chk_b = guarded((T, r), torch.bfloat16, "cuda")
    u, _, chk_u = guarded((T, m), torch.bfloat16, "cuda")
    L.encode2_fwd(x, z, d["W1"].cuda(), d["W2"].cuda(), b, u, act=act)
    torch.cuda.synchronize()
    chk_b()
    chk_u()
    rb_, ru = TL.encode2_fwd(np64(d, "x_attn"), np64(d, "z"), np64(d, "W1"), np64(d, "W2"), act)
    check("u", u, ru, True)
    both("b", b, rb_, spec_encode2_fwd(np64(d, "x_attn"), np64(d, "z"), np64(d, "W1"), np64(d, "W2"), act), True)


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("T,n,m,r", SHAPES, ids=IDS)
def test_decode2_fwd(T, n, m, r, act):
    L = lib()
    say(f"decode2_fwd T={T} n={n} m={m} r={r} act={act}")
    d = data(T, n, m, r)
    zt_buf = torch.full((T, n + 16), float("nan"), dtype=torch.bfloat16, device="cuda")
    zt = zt_buf[:, :n]
    v, _, chk_v = guarded((T, m), torch.bfloat16, "cuda")
    L.decode2_fwd(d["b"].cuda(), d["W3"].cuda(), d["W4"].cuda(), zt, v, act=act)
    torch.cuda.synchronize()
    chk_v()
    assert bool(torch.isnan(zt_buf[:, n:].float()).all()), "row padding of z~ overwritten"
    rzt, rv = TL.decode2_fwd(np64(d, "b"), np64(d, "W3"), np64(d, "W4"), act)
    check("v", v, rv, True)
    both("z~", zt, rzt, spec_decode2_fwd(np64(d, "b"), np64(d, "W3"), np64(d, "W4"), act), True)


@pytest.mark.parametrize("with_gid", [True, False])
@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("T,n,m,r", SHAPES, ids=IDS)
def test_decode2_bwd(T, n, m, r, act, with_gid):
    L = lib()
    say(f"decode2_bwd T={T} n={n} m={m} r={r} act={act} g_id={with_gid}")
    d = data(T, n, m, r)
    g_zt = strided(d["g_zt"].cuda(), 8)
    g_id = strided(d["g_id"].cuda(), 40) if with_gid else None
    g_b, _, chk = guarded((T, r), torch.bfloat16, "cuda")
    dW3 = torch.full((r, m), float("nan"), device="cuda")
    dW4 = torch.full((m, n), float("nan"), device="cuda")
    L.decode2_bwd(d["b"].cuda(), d["v"].cuda(), g_zt, g_id, d["W3"].cuda(), d["W4"].cuda(), g_b, dW3, dW4, act=act)
    torch.cuda.synchronize()
    chk()
    rg_b, rdW3, rdW4 = TL.decode2_bwd(np64(d, "b"), np64(d, "v"), np64(d, "g_zt"),
                                      np64(d, "g_id") if with_gid else None, np64(d, "W3"), np64(d, "W4"), act)
    sg_b, sdW3, sdW4 = spec_decode2_bwd(np64(d, "b"), np64(d, "v"), np64(d, "g_zt"),
                                        np64(d, "g_id") if with_gid else None, np64(d, "W3"), np64(d, "W4"), act)
    b, v, g_zt = np64(d, "b"), np64(d, "v"), np64(d, "g_zt")
    g_v = (g_zt @ np64(d, "W4").T) * R.dphi(v, act)
    both("g_b", g_b, rg_b, sg_b, True)
    both("dW3", dW3, rdW3, sdW3, False, factors=(b, g_v))
    both("dW4", dW4, rdW4, sdW4, False, factors=(R.phi(v, act), g_zt))


@pytest.mark.parametrize("gx_mode", ["separate", "fused", "none"])
@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("T,n,m,r", SHAPES, ids=IDS)
def test_encode2_bwd(T, n, m, r, act, gx_mode):
    L = lib()
    say(f"encode2_bwd T={T} n={n} m={m} r={r} act={act} g_x={gx_mode}")
    d = data(T, n, m, r)
    z = strided(d["z"].cuda(), 16)
    gz_buf = torch.full((T, n + 8), float("nan"), dtype=torch.bfloat16, device="cuda")
    g_z = gz_buf[:, :n]
    g_x = None
    gx0 = I.make_bf16(T, n, 21, std=0.1)
    if gx_mode == "separate":
        g_x = strided(gx0.cuda(), 8)
    elif gx_mode == "fused":
        g_x = g_z
    dW1 = torch.full((n, m), float("nan"), device="cuda")
    dW2 = torch.full((m, r), float("nan"), device="cuda")
    L.encode2_bwd(z, d["u"].cuda(), d["g_b"].cuda(), d["W1"].cuda(), d["W2"].cuda(), g_z, dW1, dW2, g_x=g_x,
                  act=act)
    torch.cuda.synchronize()
    assert bool(torch.isnan(gz_buf[:, n:].float()).all()), "row padding of g_z overwritten"
    rg_z, rdW1, rdW2 = TL.encode2_bwd(np64(d, "z"), np64(d, "u"), np64(d, "g_b"), np64(d, "W1"), np64(d, "W2"), act)
    if gx_mode == "fused":
        rg_z = R.skip_grad(rg_z, np64(d, "g_b"))
    sg_z, sdW1, sdW2 = spec_encode2_bwd(np64(d, "z"), np64(d, "u"), np64(d, "g_b"), np64(d, "W1"), np64(d, "W2"), act)
    if gx_mode == "fused":
        sg_z = R.skip_grad(sg_z, np64(d, "g_b"))
    u, gb = np64(d, "u"), np64(d, "g_b")
    g_u = (gb @ np64(d, "W2").T) * R.dphi(u, act)
    both("g_z", g_z, rg_z, sg_z, True)
    both("dW1", dW1, rdW1, sdW1, False, factors=(np64(d, "z"), g_u))
    both("dW2", dW2, rdW2, sdW2, False, factors=(R.phi(u, act), gb))
    if gx_mode == "separate":
        gx_ref = R.skip_grad(gx0.to(torch.float64).numpy(), np64(d, "g_b"))
        got = f64(g_x)
        assert np.array_equal(got[:, r:], gx_ref[:, r:]), "g_x columns >= r changed"
        check("g_x", g_x, gx_ref, True)


def sweep_shapes(count=24, seed=2404):
    """Fixed-seed random small shapes: short contractions (m, r, T down to 8, 8, 1)."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        n = 8 * int(rng.integers(1, 65))
        m = 8 * int(rng.integers(1, 41))
        r = 8 * int(rng.integers(1, min(n // 8, 16) + 1))
        T = int(rng.choice([1, 2, 7, int(rng.integers(1, 700))]))
        out.append((T, n, m, r))
    return out


SWEEP = sweep_shapes()


@pytest.mark.parametrize("T,n,m,r", SWEEP, ids=[f"T{T}_n{n}_m{m}_r{r}" for T, n, m, r in SWEEP])
def test_two_sweep(T, n, m, r):
    """All four ops with SiLU on a seeded sweep of small shapes, to the plain bound."""
    L = lib()
    act = R.ACT_SILU
    say(f"two-linear sweep T={T} n={n} m={m} r={r}")
    d = data(T, n, m, r, seed=T + n + m + r)
    W1, W2, W3, W4 = (np64(d, k) for k in ("W1", "W2", "W3", "W4"))
    dv = {k: v.cuda() for k, v in d.items() if isinstance(v, torch.Tensor)}
    bf = torch.bfloat16
    b, u = torch.empty(T, r, dtype=bf, device="cuda"), torch.empty(T, m, dtype=bf, device="cuda")
    zt, v = torch.empty(T, n, dtype=bf, device="cuda"), torch.empty(T, m, dtype=bf, device="cuda")
    g_b, g_z = torch.empty(T, r, dtype=bf, device="cuda"), torch.empty(T, n, dtype=bf, device="cuda")
    dW1, dW2 = torch.empty(n, m, device="cuda"), torch.empty(m, r, device="cuda")
    dW3, dW4 = torch.empty(r, m, device="cuda"), torch.empty(m, n, device="cuda")
    L.encode2_fwd(dv["x_attn"], dv["z"], dv["W1"], dv["W2"], b, u, act=act)
    L.decode2_fwd(dv["b"], dv["W3"], dv["W4"], zt, v, act=act)
    L.decode2_bwd(dv["b"], dv["v"], dv["g_zt"], dv["g_id"], dv["W3"], dv["W4"], g_b, dW3, dW4, act=act)
    L.encode2_bwd(dv["z"], dv["u"], dv["g_b"], dv["W1"], dv["W2"], g_z, dW1, dW2, g_x=g_z, act=act)
    torch.cuda.synchronize()
    x, z = np64(d, "x_attn"), np64(d, "z")
    rb_, ru = TL.encode2_fwd(x, z, W1, W2, act)
    check("u", u, ru, True)
    both("b", b, rb_, spec_encode2_fwd(x, z, W1, W2, act), True)
    rzt, rv = TL.decode2_fwd(np64(d, "b"), W3, W4, act)
    check("v", v, rv, True)
    both("z~", zt, rzt, spec_decode2_fwd(np64(d, "b"), W3, W4, act), True)
    bb, vv, gzt, gb = np64(d, "b"), np64(d, "v"), np64(d, "g_zt"), np64(d, "g_b")
    g_v = (gzt @ W4.T) * R.dphi(vv, act)
    args = (bb, vv, gzt, np64(d, "g_id"), W3, W4, act)
    factors = (None, (bb, g_v), (R.phi(vv, act), gzt))
    for nm, got, ref, spec, fa in zip(("g_b", "dW3", "dW4"), (g_b, dW3, dW4), TL.decode2_bwd(*args),
                                      spec_decode2_bwd(*args), factors):
        both(nm, got, ref, spec, nm == "g_b", factors=fa)
    uu = np64(d, "u")
    g_u = (gb @ W2.T) * R.dphi(uu, act)
    args = (z, uu, gb, W1, W2, act)
    ref = list(TL.encode2_bwd(*args))
    spec = list(spec_encode2_bwd(*args))
    ref[0] = R.skip_grad(ref[0], gb)
    spec[0] = R.skip_grad(spec[0], gb)
    factors = (None, (z, g_u), (R.phi(uu, act), gb))
    for nm, got, rr, ss, fa in zip(("g_z", "dW1", "dW2"), (g_z, dW1, dW2), ref, spec, factors):
        both(nm, got, rr, ss, nm == "g_z", factors=fa)


def test_two_empty_batch_is_noop():
    L = lib()
    n, m, r = 64, 32, 8
    w = {k: v.cuda() for k, v in I.make_two_weights(n, m, r).items()}
    e = torch.empty((0, n), dtype=torch.bfloat16, device="cuda")
    L.encode2_fwd(e, e, w["W1"], w["W2"], torch.empty((0, r), dtype=torch.bfloat16, device="cuda"),
                  torch.empty((0, m), dtype=torch.bfloat16, device="cuda"))
    torch.cuda.synchronize()


def test_two_deterministic():
    L = lib()
    T, n, m, r = 4096, 512, 256, 32
    d = data(T, n, m, r, seed=3)
    outs = []
    for _ in range(2):
        g_z = torch.empty((T, n), dtype=torch.bfloat16, device="cuda")
        dW1, dW2 = torch.empty((n, m), device="cuda"), torch.empty((m, r), device="cuda")
        L.encode2_bwd(d["z"].cuda(), d["u"].cuda(), d["g_b"].cuda(), d["W1"].cuda(), d["W2"].cuda(), g_z, dW1, dW2)
        torch.cuda.synchronize()
        outs.append((g_z.view(torch.int16).clone(), dW1.view(torch.int32).clone(), dW2.view(torch.int32).clone()))
    for a, b in zip(*outs):
        assert torch.equal(a, b)


# ---------------------------------------------------------------- full size, sampled
FULL = (16384, 4096, 1024, 32)


@pytest.fixture(scope="module")
def full():
    T, n, m, r = FULL
    say(f"drawing full-size inputs T={T} n={n} m={m} r={r}")
    d = data(T, n, m, r, seed=5)
    dev = {k: v.cuda() for k, v in d.items() if isinstance(v, torch.Tensor)}
    rng = np.random.default_rng(17)
    rows = np.unique(np.concatenate([[0, T - 1], rng.choice(T, 61, replace=False)]))
    cols_m = np.unique(np.concatenate([[0, m - 1], rng.choice(m, 14, replace=False)]))
    cols_n = np.unique(np.concatenate([[0, n - 1], rng.choice(n, 14, replace=False)]))
    return d, dev, rows, cols_m, cols_n


def test_full_forward_sampled(full):
    L = lib()
    d, dv, rows, _, _ = full
    T, n, m, r = FULL
    act = R.ACT_SILU
    b = torch.empty((T, r), dtype=torch.bfloat16, device="cuda")
    u = torch.empty((T, m), dtype=torch.bfloat16, device="cuda")
    L.encode2_fwd(dv["x_attn"], dv["z"], dv["W1"], dv["W2"], b, u, act=act)
    zt = torch.empty((T, n), dtype=torch.bfloat16, device="cuda")
    v = torch.empty((T, m), dtype=torch.bfloat16, device="cuda")
    L.decode2_fwd(dv["b"], dv["W3"], dv["W4"], zt, v, act=act)
    torch.cuda.synchronize()
    sel = lambda k: d[k][rows].to(torch.float64).numpy()  # noqa: E731
    rb, ru = TL.encode2_fwd(sel("x_attn"), sel("z"), np64(d, "W1"), np64(d, "W2"), act)
    check("u", u[rows].cpu(), ru, True)
    check("b", b[rows].cpu(), rb, True)
    rzt, rv = TL.decode2_fwd(sel("b"), np64(d, "W3"), np64(d, "W4"), act)
    check("v", v[rows].cpu(), rv, True)
    check("z~", zt[rows].cpu(), rzt, True)


def test_full_backward_sampled(full):
    L = lib()
    d, dv, rows, cols_m, cols_n = full
    T, n, m, r = FULL
    act = R.ACT_SILU
    g_b = torch.empty((T, r), dtype=torch.bfloat16, device="cuda")
    dW3, dW4 = torch.empty((r, m), device="cuda"), torch.empty((m, n), device="cuda")
    L.decode2_bwd(dv["b"], dv["v"], dv["g_zt"], dv["g_id"], dv["W3"], dv["W4"], g_b, dW3, dW4, act=act)
    g_z = torch.empty((T, n), dtype=torch.bfloat16, device="cuda")
    dW1, dW2 = torch.empty((n, m), device="cuda"), torch.empty((m, r), device="cuda")
    L.encode2_bwd(dv["z"], dv["u"], dv["g_b"], dv["W1"], dv["W2"], g_z, dW1, dW2, g_x=g_z, act=act)
    torch.cuda.synchronize()
    W1, W2, W3, W4 = (np64(d, k) for k in ("W1", "W2", "W3", "W4"))
    b, v, u, gb_in = np64(d, "b"), np64(d, "v"), np64(d, "u"), np64(d, "g_b")
    g_zt, g_id, z = np64(d, "g_zt"), np64(d, "g_id"), np64(d, "z")
    # row-local outputs on sampled rows
    rg_b, _, _ = TL.decode2_bwd(b[rows], v[rows], g_zt[rows], g_id[rows], W3, W4, act)
    check("g_b", g_b[rows].cpu(), rg_b, True)
    rg_z, _, _ = TL.encode2_bwd(z[rows], u[rows], gb_in[rows], W1, W2, act)
    check("g_z", g_z[rows].cpu(), R.skip_grad(rg_z, gb_in[rows]), True)
    # token sums on sampled columns: dW4[:, j] = phi(v)^T g_zt[:, j]; dW3[:, j] = b^T g_v[:, j];
    # dW1[:, j] = z^T g_u[:, j]; dW2 whole
    p = R.phi(v, act)
    check("dW4[:, s]", dW4[:, cols_n].cpu(), p.T @ g_zt[:, cols_n], False)
    g_v = (g_zt @ W4[cols_m].T) * R.dphi(v[:, cols_m], act)
    check("dW3[:, s]", dW3[:, cols_m].cpu(), b.T @ g_v, False)
    g_u = (gb_in @ W2[cols_m].T) * R.dphi(u[:, cols_m], act)
    check("dW1[:, s]", dW1[:, cols_m].cpu(), z.T @ g_u, False)
    check("dW2", dW2, R.phi(u, act).T @ gb_in, False)


def test_two_graph_replay_matches_eager():
    """The four two-linear ops and the fused FFN-projection encoder captured in one
    HIP graph replay bit for bit like eager calls, with the workspaces and outputs
    scribbled over and unrelated eager work between the replays."""
    L = lib()
    T, n, m, r, d_ff = 700, 512, 264, 40, 328
    say(f"graph replay T={T} n={n} m={m} r={r} d_ff={d_ff}")
    d = {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in data(T, n, m, r, seed=7).items()}
    h = I.make_bf16(T, d_ff, 51).cuda()
    W_down = I.make_bf16(d_ff, n, 52, std=d_ff ** -0.5).cuda()
    W_e = I.make_weights(n, r, 7)["W_e"].cuda()
    bf = torch.bfloat16
    outs = {"b": torch.empty(T, r, dtype=bf, device="cuda"), "u": torch.empty(T, m, dtype=bf, device="cuda"),
            "zt": torch.empty(T, n, dtype=bf, device="cuda"), "v": torch.empty(T, m, dtype=bf, device="cuda"),
            "g_b": torch.empty(T, r, dtype=bf, device="cuda"), "g_z": torch.empty(T, n, dtype=bf, device="cuda"),
            "dW1": torch.empty(n, m, device="cuda"), "dW2": torch.empty(m, r, device="cuda"),
            "dW3": torch.empty(r, m, device="cuda"), "dW4": torch.empty(m, n, device="cuda"),
            "z": torch.empty(T, n, dtype=bf, device="cuda"), "b2": torch.empty(T, r, dtype=bf, device="cuda"),
            "a": torch.empty(T, r, device="cuda")}
    ws = L.two_workspace(T, n, m, r, "cuda")
    nb = int(L.cdll.resbm_ffn_encode_workspace_bytes(T, n, r))
    ws2 = torch.empty(nb, dtype=torch.uint8, device="cuda")
    o = outs

    def step():
        L.encode2_fwd(d["x_attn"], d["z"], d["W1"], d["W2"], o["b"], o["u"], ws=ws)
        L.decode2_fwd(o["b"], d["W3"], d["W4"], o["zt"], o["v"], ws=ws)
        L.decode2_bwd(o["b"], o["v"], d["g_zt"], d["g_id"], d["W3"], d["W4"], o["g_b"], o["dW3"], o["dW4"], ws=ws)
        L.encode2_bwd(d["z"], o["u"], o["g_b"], d["W1"], d["W2"], o["g_z"], o["dW1"], o["dW2"], g_x=o["g_z"], ws=ws)
        L.ffn_encode_fwd(h, W_down, d["x_attn"], W_e, o["z"], o["b2"], a_save=o["a"], ws=ws2)

    step()
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in o.items()}
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(3):
        for v in o.values():
            v.view(torch.uint8).fill_(0x5A)
        ws.fill_(0xA5)
        ws2.fill_(0x3C)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in o.items():
            assert torch.equal(v.view(torch.uint8), ref[k].view(torch.uint8)), f"replay {rep}: {k} differs"
