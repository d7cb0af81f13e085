"""Optimizer-side ops (Newton-Schulz, Muon update, spectrum) vs the CPU oracle.

Inputs are float32 matrices from the seeded generator; the oracle computes in
float64 on the same values.  Tolerances follow from the arithmetic: the GPU
runs float64 inside and rounds each float32 output once, so
  - O and W: max |gpu - ref| <= MAT_BOUND max |ref| (one float32 rounding is
    <= 2^-24 = 6e-8 of an element; the float64 paths differ by ~1e-14);
  - the momentum buffer M: bit-exact (same float64 operations, one rounding);
  - singular values: |gpu - ref| <= SIG_BOUND sigma_max (they come from the
    Gram's eigenvalues, whose float64 error ~1e-16 lambda_max becomes ~1e-8
    sigma_max on the smallest); r_eff: relative 1e-9.
"""
import numpy as np
import pytest
import torch

from oracle import muon_oracle as MU
from gpu_helpers import f64, guarded, lib, say
from paper_2604_11947_amd import inputs as I

pytestmark = pytest.mark.gpu

MAT_BOUND = 1.5e-7
SIG_BOUND = 1e-7
REFF_BOUND = 1e-9

NS_SHAPES = [(4096, 32), (32, 4096), (8192, 64), (64, 8192), (333, 40), (40, 333), (4096, 256), (256, 520),
             (64, 64), (7, 3), (3, 7), (1000, 1), (1, 1000), (1, 1), (100, 5)]
NS_IDS = [f"{p}x{q}" for p, q in NS_SHAPES]


def dev(t):
    return t.to("cuda")


def max_rel(gpu: np.ndarray, ref: np.ndarray) -> float:
    m = float(np.abs(ref).max()) if ref.size else 0.0
    d = float(np.abs(gpu - ref).max()) if ref.size else 0.0
    return d / m if m > 0 else d


def run_ns(L, G, steps, coeffs):
    p, q = G.shape
    O, _, chk = guarded((p, q), torch.float32, "cuda")
    L.newton_schulz(dev(G), O, steps=steps, coeffs=coeffs)
    torch.cuda.synchronize()
    chk()
    return O


@pytest.mark.parametrize("p,q", NS_SHAPES, ids=NS_IDS)
@pytest.mark.parametrize("kind", ["gaussian", "powerlaw"])
@pytest.mark.parametrize("coeffs,steps", [(MU.NS_QUINTIC, 5), (MU.NS_CUBIC, 12), (MU.NS_QUINTIC, 0)],
                         ids=["quintic5", "cubic12", "steps0"])
def test_newton_schulz_parity(p, q, kind, coeffs, steps):
    L = lib()
    say(f"newton_schulz {p}x{q} {kind} steps={steps}")
    G = I.make_matrix(p, q, kind, seed=1)
    O = run_ns(L, G, steps, coeffs)
    ref = MU.newton_schulz(G.double().numpy(), steps, coeffs)
    e = max_rel(f64(O), ref)
    say(f"    max err / max|ref| = {e:.2e}")
    assert np.all(np.isfinite(f64(O)))
    assert e <= MAT_BOUND


@pytest.mark.parametrize("p,q,kind", [(4096, 32, "gaussian"), (333, 40, "powerlaw"), (7, 3, "rank1"), (64, 64, "powerlaw")],
                         ids=["4096x32-gaussian", "333x40-powerlaw", "7x3-rank1", "64x64-powerlaw"])
@pytest.mark.parametrize("steps", [8, 9, 30])
def test_newton_schulz_long_runs(p, q, kind, steps):
    """Step counts on both sides of the switch between the short-side
    recurrence (quintic: up to 8 steps) and the row-by-row iteration, and a
    long run of a rank-deficient matrix, whose rounding-level Gram directions
    the recurrence would amplify."""
    L = lib()
    say(f"newton_schulz {p}x{q} {kind} steps={steps}")
    G = I.make_matrix(p, q, kind, seed=3)
    O = run_ns(L, G, steps, MU.NS_QUINTIC)
    ref = MU.newton_schulz(G.double().numpy(), steps, MU.NS_QUINTIC)
    e = max_rel(f64(O), ref)
    say(f"    max err / max|ref| = {e:.2e}")
    assert np.all(np.isfinite(f64(O)))
    assert e <= MAT_BOUND


def test_newton_schulz_deterministic_and_zero():
    L = lib()
    G = I.make_matrix(4096, 32, "gaussian", seed=2)
    a, b = run_ns(L, G, 5, MU.NS_QUINTIC), run_ns(L, G, 5, MU.NS_QUINTIC)
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    Z = run_ns(L, I.make_matrix(32, 4096, "zero"), 5, MU.NS_QUINTIC)
    assert not bool(Z.any())


@pytest.mark.parametrize("p,q", [(4096, 32), (32, 4096), (8192, 64), (333, 40), (7, 3), (1, 64)],
                         ids=["4096x32", "32x4096", "8192x64", "333x40", "7x3", "1x64"])
@pytest.mark.parametrize("nesterov", [False, True])
def test_muon_update_two_steps(p, q, nesterov):
    L = lib()
    say(f"muon_update {p}x{q} nesterov={nesterov}")
    lr, mu, wd = 0.02, 0.95, 0.1
    W0 = I.make_matrix(p, q, "gaussian", seed=3, scale=(1.0 / min(p, q)) ** 0.5)
    G1 = I.make_matrix(p, q, "gaussian", seed=4, scale=0.01)
    G2 = I.make_matrix(p, q, "powerlaw", seed=5, scale=0.01)
    W = dev(W0.clone())
    M = dev(torch.zeros(p, q))
    Wr, Mr = W0.double().numpy(), np.zeros((p, q))
    for G in (G1, G2):
        L.muon_update(W, dev(G), M, lr, momentum=mu, weight_decay=wd, nesterov=nesterov)
        torch.cuda.synchronize()
        Wr, Mr, _ = MU.muon_update(Wr, G.double().numpy(), Mr, lr, mu, wd, nesterov=nesterov)
        assert np.array_equal(f64(M), Mr), "momentum buffer differs"
        e = max_rel(f64(W) - W0.double().numpy(), Wr - W0.double().numpy())
        d = float(np.abs(f64(W) - Wr).max())
        say(f"    W max err {d:.2e} (update-relative {e:.2e})")
        assert d <= MAT_BOUND * float(np.abs(Wr).max())


def test_muon_update_without_momentum_buffer():
    L = lib()
    p, q = 32, 4096
    W0 = I.make_matrix(p, q, "gaussian", seed=6, scale=0.1)
    G = I.make_matrix(p, q, "gaussian", seed=7, scale=0.01)
    W = dev(W0.clone())
    L.muon_update(W, dev(G), None, 0.05, momentum=0.9, weight_decay=0.0, steps=5)
    torch.cuda.synchronize()
    Wr, _, _ = MU.muon_update(W0.double().numpy(), G.double().numpy(), np.zeros((p, q)), 0.05, 0.0)
    assert float(np.abs(f64(W) - Wr).max()) <= MAT_BOUND * float(np.abs(Wr).max())


@pytest.mark.parametrize("scale", [0.7, 0.0], ids=["explicit", "zero"])
def test_muon_update_explicit_scale(scale):
    """An explicit scale is used as given (a negative one selects the default,
    0.2 sqrt(max(p, q)), which the other Muon tests exercise)."""
    L = lib()
    p, q = 333, 40
    W0 = I.make_matrix(p, q, "gaussian", seed=12, scale=0.1)
    G = I.make_matrix(p, q, "gaussian", seed=13, scale=0.01)
    W, M = dev(W0.clone()), dev(torch.zeros(p, q))
    L.muon_update(W, dev(G), M, 0.05, momentum=0.9, weight_decay=0.01, scale=scale)
    torch.cuda.synchronize()
    Wr, _, _ = MU.muon_update(W0.double().numpy(), G.double().numpy(), np.zeros((p, q)), 0.05, 0.9, 0.01,
                              scale=scale)
    assert float(np.abs(f64(W) - Wr).max()) <= MAT_BOUND * float(np.abs(Wr).max())


SPEC_CASES = [(4096, 32, "gaussian"), (32, 4096, "gaussian"), (8192, 64, "powerlaw"), (333, 40, "powerlaw"),
              (128, 4096, "powerlaw"), (64, 64, "gaussian"), (4096, 32, "orthonormal"), (32, 4096, "rank1"),
              (40, 333, "zero"), (7, 3, "gaussian"), (1, 5, "gaussian"), (5, 1, "gaussian"), (1, 1, "gaussian"),
              # hard cases for bisection: two tight clusters, six decades of singular values (s = 32, 128)
              (4096, 32, "clustered"), (32, 4096, "graded"), (128, 4096, "graded"),
              # 64 < s < 128: the LDS path on 1024 threads (ragged s4)
              (100, 3000, "powerlaw"), (4096, 65, "gaussian"),
              # s > 128: the reduction in place on the workspace Gram (s = 129, 200, 256; ragged s4)
              (129, 1000, "gaussian"), (4096, 200, "powerlaw"), (4096, 256, "gaussian"), (256, 8192, "graded"),
              (4096, 256, "clustered"), (256, 300, "rank1"), (2000, 130, "orthonormal")]


@pytest.mark.parametrize("p,q,kind", SPEC_CASES, ids=[f"{p}x{q}_{k}" for p, q, k in SPEC_CASES])
def test_spectrum_parity(p, q, kind):
    L = lib()
    say(f"spectrum {p}x{q} {kind}")
    W = I.make_matrix(p, q, kind, seed=8)
    s = min(p, q)
    sig = torch.full((s + 8,), float("nan"), dtype=torch.float64, device="cuda")
    reff = torch.full((2,), float("nan"), dtype=torch.float64, device="cuda")
    L.spectrum(dev(W), sig[:s], reff[:1])
    torch.cuda.synchronize()
    g_sig, g_reff = f64(sig), f64(reff)
    assert np.all(np.isnan(g_sig[s:])) and np.isnan(g_reff[1]), "wrote past the outputs"
    ref_sig, ref_reff = MU.spectrum(W.double().numpy())
    top = float(ref_sig[0]) if ref_sig.size else 0.0
    err = float(np.abs(g_sig[:s] - ref_sig).max())
    say(f"    sigma err {err:.2e} (top {top:.3e}), r_eff {g_reff[0]:.6f} vs {ref_reff:.6f}")
    assert err <= SIG_BOUND * max(top, 1e-300)
    assert np.all(np.diff(g_sig[:s]) <= 0)
    assert abs(g_reff[0] - ref_reff) <= REFF_BOUND * max(ref_reff, 1.0)
    if kind == "orthonormal":  # float32 rounding leaves sigma^2 within ~1e-7 of 1
        assert abs(g_reff[0] - s) < 1e-5 * s
    if kind == "rank1":
        assert abs(g_reff[0] - 1.0) < 1e-9


@pytest.mark.parametrize("bad", ["nan", "inf", "-inf"])
@pytest.mark.parametrize("p,q", [(4096, 32), (32, 4096), (7, 3), (1, 1), (200, 128), (300, 256)],
                         ids=["4096x32", "32x4096", "7x3", "1x1", "200x128", "300x256"])
def test_spectrum_non_finite(p, q, bad):
    """A NaN or an infinity anywhere in W makes every sigma_i and r_eff NaN (the
    Gram's eigenvalues are undefined); the outputs stop at s, and a finite
    matrix on the same workspace right after gets its own spectrum."""
    L = lib()
    say(f"spectrum non-finite {p}x{q} {bad}")
    W = I.make_matrix(p, q, "gaussian", seed=9)
    W[p // 2, q - 1] = float(bad)
    s = min(p, q)
    ws = torch.empty(L.matrix_workspace_bytes(p, q), dtype=torch.uint8, device="cuda")
    sig = torch.full((s + 8,), -7.0, dtype=torch.float64, device="cuda")
    reff = torch.full((2,), -7.0, dtype=torch.float64, device="cuda")
    L.spectrum(dev(W), sig[:s], reff[:1], ws=ws)
    torch.cuda.synchronize()
    g_sig, g_reff = f64(sig), f64(reff)
    assert np.all(np.isnan(g_sig[:s])) and np.isnan(g_reff[0])
    assert np.all(g_sig[s:] == -7.0) and g_reff[1] == -7.0, "wrote past the outputs"
    W2 = I.make_matrix(p, q, "gaussian", seed=10)
    L.spectrum(dev(W2), sig[:s], reff[:1], ws=ws)
    torch.cuda.synchronize()
    ref_sig, ref_reff = MU.spectrum(W2.double().numpy())
    assert float(np.abs(f64(sig)[:s] - ref_sig).max()) <= SIG_BOUND * float(ref_sig[0])
    assert abs(f64(reff)[0] - ref_reff) <= REFF_BOUND * max(ref_reff, 1.0)


@pytest.mark.parametrize("p,q", [(4096, 32), (40, 333), (256, 520)], ids=["4096x32", "40x333", "256x520"])
def test_graph_replay_matches_eager(p, q):
    """A Muon update, a Newton-Schulz call and the spectrum captured in one HIP
    graph replay exactly like eager launches (fixed-order sums), with unrelated
    eager work and a scribbled workspace between the replays."""
    L = lib()
    say(f"matrix graph replay {p}x{q}")
    W0 = dev(I.make_matrix(p, q, "gaussian", seed=9, scale=0.1))
    G = dev(I.make_matrix(p, q, "powerlaw", seed=10, scale=0.01))
    M0 = dev(I.make_matrix(p, q, "gaussian", seed=11, scale=0.001))
    W, M, O = W0.clone(), M0.clone(), torch.empty(p, q, device="cuda")
    ws = L.matrix_workspace(p, q, "cuda")
    spec = True
    sig = torch.empty(min(p, q), dtype=torch.float64, device="cuda")
    reff = torch.empty(1, dtype=torch.float64, device="cuda")

    def step():
        L.muon_update(W, G, M, 0.02, momentum=0.9, weight_decay=0.01, nesterov=True, ws=ws)
        L.newton_schulz(G, O, steps=5, ws=ws)
        if spec:
            L.spectrum(W, sig, reff, ws=ws)

    step()
    torch.cuda.synchronize()
    ref = {"W": W.clone(), "M": M.clone(), "O": O.clone(), "sig": sig.clone(), "reff": reff.clone()}
    graph = torch.cuda.CUDAGraph()
    W.copy_(W0)
    M.copy_(M0)
    with torch.cuda.graph(graph):
        step()
    for rep in range(3):
        W.copy_(W0)
        M.copy_(M0)
        O.fill_(float("nan"))
        sig.fill_(float("nan"))
        reff.fill_(float("nan"))
        ws.fill_(0x5A)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in (("W", W), ("M", M), ("O", O)):
            assert torch.equal(v.view(torch.int32), ref[k].view(torch.int32)), f"replay {rep}: {k} differs"
        if spec:
            for k, v in (("sig", sig), ("reff", reff)):
                assert torch.equal(v.view(torch.int64), ref[k].view(torch.int64)), f"replay {rep}: {k} differs"
