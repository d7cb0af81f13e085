"""Boundary ops fused into their neighbours, against the float64 oracle:
- the encoder fused into the FFN output projection (resbm_ffn_encode_fwd):
  z = h W_down, then the encoder on the stored (bf16) z;
- the decoder fused into the next block's RMS normalisation and QKV projection
  (resbm_decode_qkv_fwd): out = RMSNorm(b W_d) W_qkv.

Bounds as for the one-linear ops: max error <= 2e-2 RMS(ref) after a half-ulp
discount for bf16 outputs; a_save (float32) raw.  The fused decoder rounds
z~ gamma to bf16 before the projection (relative 2^-9 per element, averaging
out over the n-deep contraction).
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


# ---- decoder into RMSNorm + QKV
DQ_SHAPES = [(333, 256, 32, 384), (1000, 1024, 32, 520), (64, 64, 8, 64), (1, 256, 16, 256), (513, 512, 64, 264),
             (300, 4096, 32, 1032)]
DQ_IDS = [f"T{T}_n{n}_r{r}_N{N}" for T, n, r, N in DQ_SHAPES]
EPS = 1e-5


def dq_data(T, n, r, N, seed=0):
    return {"b": I.make_bf16(T, r, seed + 41), "W_d": I.make_weights(n, r, seed)["W_d"],
            "gamma": I.make_gain(n, seed + 42), "W_qkv": I.make_bf16(n, N, seed + 43, std=n ** -0.5)}


def dq_ref(d, rows=None):
    b = d["b"] if rows is None else d["b"][rows]
    return F.decode_qkv_fwd(f64(b), d["W_d"].double().numpy(), d["gamma"].double().numpy(), f64(d["W_qkv"]), EPS)[2]


@pytest.mark.parametrize("T,n,r,N", DQ_SHAPES, ids=DQ_IDS)
def test_decode_qkv_fwd(T, n, r, N):
    L = lib()
    say(f"decode_qkv_fwd T={T} n={n} r={r} N={N}")
    d = dq_data(T, n, r, N)
    obuf = torch.full((T, N + 8), float("nan"), dtype=torch.bfloat16, device="cuda")
    out = obuf[:, :N]
    L.decode_qkv_fwd(d["b"].cuda(), d["W_d"].cuda(), d["gamma"].cuda(), d["W_qkv"].cuda(), out, eps=EPS)
    torch.cuda.synchronize()
    assert bool(torch.isnan(obuf[:, N:].float()).all()), "row padding of out overwritten"
    check("out", out, dq_ref(d), True)


def test_decode_qkv_zero_payload_and_determinism():
    """A zero payload gives a zero output (the eps keeps the scale finite);
    repeated calls are bit-identical."""
    L = lib()
    T, n, r, N = 700, 512, 32, 512
    d = dq_data(T, n, r, N, seed=5)
    d["b"][100:200] = 0
    outs = []
    for _ in range(2):
        out = torch.empty((T, N), dtype=torch.bfloat16, device="cuda")
        L.decode_qkv_fwd(d["b"].cuda(), d["W_d"].cuda(), d["gamma"].cuda(), d["W_qkv"].cuda(), out, eps=EPS)
        torch.cuda.synchronize()
        outs.append(out.view(torch.int16).clone())
    assert torch.equal(outs[0], outs[1])
    assert not bool(outs[0][100:200].any())


def test_decode_qkv_full_size_sampled():
    """T = 16384, n = 4096, r = 32, N = 6144 (Q 4096 + K 1024 + V 1024 of an
    8B-class block with grouped KV heads) on sampled rows."""
    L = lib()
    T, n, r, N = 16384, 4096, 32, 6144
    say(f"decode_qkv_fwd full size T={T} n={n} r={r} N={N}")
    d = dq_data(T, n, r, N, seed=6)
    out = torch.empty((T, N), dtype=torch.bfloat16, device="cuda")
    L.decode_qkv_fwd(d["b"].cuda(), d["W_d"].cuda(), d["gamma"].cuda(), d["W_qkv"].cuda(), out, eps=EPS)
    torch.cuda.synchronize()
    rng = np.random.default_rng(10)
    rows = np.unique(np.concatenate([[0, 255, 256, T - 1], rng.choice(T, 24, replace=False)]))
    check("out", out[rows], dq_ref(d, rows), True)
