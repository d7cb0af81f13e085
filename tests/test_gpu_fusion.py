"""Encoder fused into the FFN output projection (resbm_ffn_encode_fwd) against
the float64 oracle: z = h W_down, then the encoder on the stored (bf16) z.

Bounds as for the one-linear encoder: max error <= 2e-2 RMS(ref) after a
half-ulp discount for the bf16 outputs z and b; a_save (float32) raw.
"""
import numpy as np
import pytest
import torch

from oracle import fusion_oracle as F
from oracle import resbm_oracle as R
from gpu_helpers import check, guarded, lib, say, strided
from paper_2604_11947_amd import inputs as I

pytestmark = pytest.mark.gpu

SHAPES = [(333, 200, 520, 40), (1000, 1024, 256, 32), (64, 64, 64, 8), (1, 256, 512, 16), (513, 768, 384, 128),
          (300, 512, 1024, 256)]
IDS = [f"T{T}_dff{f}_n{n}_r{r}" for T, f, n, r in SHAPES]


def data(T, d_ff, n, r, seed=0):
    d = I.make_activations(T, n, "normal", seed, grads=False)
    d["h"] = I.make_bf16(T, d_ff, seed + 31)
    d["W_down"] = I.make_bf16(d_ff, n, seed + 32, std=d_ff ** -0.5)
    d["W_e"] = I.make_weights(n, r, seed)["W_e"]
    return d


def f64(t):
    return t.detach().cpu().to(torch.float64).numpy()


@pytest.mark.parametrize("act", [R.ACT_IDENTITY, R.ACT_SILU])
@pytest.mark.parametrize("T,d_ff,n,r", SHAPES, ids=IDS)
def test_ffn_encode_fwd(T, d_ff, n, r, act):
    L = lib()
    say(f"ffn_encode_fwd T={T} d_ff={d_ff} n={n} r={r} act={act}")
    d = data(T, d_ff, n, r)
    h, x = strided(d["h"].cuda(), 8), strided(d["x_attn"].cuda(), 16)
    zbuf = torch.full((T, n + 8), float("nan"), dtype=torch.bfloat16, device="cuda")
    z = zbuf[:, :n]
    b, _, chk = guarded((T, r), torch.bfloat16, "cuda")
    a = torch.full((T, r), float("nan"), device="cuda")
    L.ffn_encode_fwd(h, d["W_down"].cuda(), x, d["W_e"].cuda(), z, b, a_save=a, act=act)
    torch.cuda.synchronize()
    chk()
    assert bool(torch.isnan(zbuf[:, n:].float()).all()), "row padding of z overwritten"
    rz, rb, ra = F.ffn_encode_fwd(f64(d["h"]), f64(d["W_down"]), f64(d["x_attn"]), d["W_e"].double().numpy(), act)
    check("z", z, rz, True)
    check("a", a, ra, False)
    check("b", b, rb, True)


def test_ffn_encode_deterministic():
    L = lib()
    T, d_ff, n, r = 2048, 1024, 1024, 32
    d = data(T, d_ff, n, r, seed=2)
    outs = []
    for _ in range(2):
        z = torch.empty((T, n), dtype=torch.bfloat16, device="cuda")
        b = torch.empty((T, r), dtype=torch.bfloat16, device="cuda")
        a = torch.empty((T, r), device="cuda")
        L.ffn_encode_fwd(d["h"].cuda(), d["W_down"].cuda(), d["x_attn"].cuda(), d["W_e"].cuda(), z, b, a_save=a)
        torch.cuda.synchronize()
        outs.append((z.view(torch.int16).clone(), b.view(torch.int16).clone(), a.view(torch.int32).clone()))
    for u, v in zip(*outs):
        assert torch.equal(u, v)


def test_ffn_encode_full_size_sampled():
    """T = 16384 tokens, d_ff = 14336, n = 4096, r = 32 on sampled rows."""
    L = lib()
    T, d_ff, n, r = 16384, 14336, 4096, 32
    say(f"ffn_encode_fwd full size T={T} d_ff={d_ff} n={n} r={r}")
    d = data(T, d_ff, n, r, seed=4)
    z = torch.empty((T, n), dtype=torch.bfloat16, device="cuda")
    b = torch.empty((T, r), dtype=torch.bfloat16, device="cuda")
    a = torch.empty((T, r), device="cuda")
    L.ffn_encode_fwd(d["h"].cuda(), d["W_down"].cuda(), d["x_attn"].cuda(), d["W_e"].cuda(), z, b, a_save=a)
    torch.cuda.synchronize()
    rng = np.random.default_rng(9)
    rows = np.unique(np.concatenate([[0, T - 1], rng.choice(T, 30, replace=False)]))
    rz, rb, ra = F.ffn_encode_fwd(f64(d["h"][rows]), f64(d["W_down"]), f64(d["x_attn"][rows]),
                                  d["W_e"].double().numpy(), R.ACT_SILU)
    check("z", z[rows], rz, True)
    check("a", a[rows], ra, False)
    check("b", b[rows], rb, True)
