"""Parity at the full sizes of every named workload, in the configuration bench.py
times (SiLU, decoder reading B, one shared workspace), on sampled outputs.

The four ops run over the whole workload; the oracle recomputes a sample of every
output from the inputs the GPU op saw (its own b, a_save and g_b downstream):
token rows for the row-local outputs (b, a_save, g_b), token rows x columns for
z~ and g_z, and whole columns (sums over all T tokens) for dW_d and dW_e.  The
sample always holds the first and last token and the columns around r and at the
edges, so ragged tails and the identity path are covered.
"""
import functools

import numpy as np
import pytest
import torch

import oracle as O
from gpu_helpers import check, f64, lib, say
from paper_2604_11947_amd import inputs as I

pytestmark = pytest.mark.gpu

SILU = O.ACT_SILU


@functools.lru_cache(maxsize=1)
def activations(T, n, dist, seed):
    return I.make_activations(T, n, dist, seed)


def pick(rng, size, must, k):
    extra = rng.choice(size, size=min(size, k), replace=False)
    return np.unique(np.concatenate([np.asarray([m for m in must if 0 <= m < size], dtype=np.int64), extra]))


@pytest.mark.timeout(600)  # drawing the n = 8192 inputs on the host takes about two minutes
@pytest.mark.parametrize("name", list(I.WORKLOADS))
def test_fullsize_sampled(name):
    w = I.WORKLOADS[name]
    T, n, r = w.tokens, w.n, w.r
    say(f"full size {name}: T={T} n={n} r={r} dist={w.dist}")
    L = lib()
    d = dict(activations(T, n, w.dist, w.seed))
    d.update(I.make_weights(n, r, w.seed))
    g = {k: d[k].cuda() for k in ("x_attn", "z", "W_e", "W_d", "g_zt", "g_id")}
    io = L.io_dtype
    b = torch.empty(T, r, dtype=io, device="cuda")
    a = torch.empty(T, r, dtype=torch.float32, device="cuda")
    zt = torch.empty(T, n, dtype=io, device="cuda")
    gb = torch.empty(T, r, dtype=io, device="cuda")
    dWd = torch.empty(r, n, dtype=torch.float32, device="cuda")
    gz = torch.empty(T, n, dtype=io, device="cuda")
    dWe = torch.empty(n, r, dtype=torch.float32, device="cuda")
    ws = L.workspace(T, n, r, "cuda")
    L.encode_fwd(g["x_attn"], g["z"], g["W_e"], b, a, act=SILU, ws=ws)
    L.decode_fwd(b, g["W_d"], zt, ws=ws)
    L.decode_bwd(b, g["W_d"], g["g_zt"], g["g_id"], gb, dWd, ws=ws)
    L.encode_bwd(g["z"], g["W_e"], a, gb, gz, dWe, act=SILU, ws=ws)
    torch.cuda.synchronize()
    del g

    rng = np.random.default_rng(11)
    rows = pick(rng, T, [0, 1, T // 2, T - 2, T - 1], 48)
    cols = pick(rng, n, [0, r - 1, r, n // 2, n - 1], 48)
    rows_t, cols_t = torch.from_numpy(rows), torch.from_numpy(cols)
    rows_d, cols_d = rows_t.cuda(), cols_t.cuda()
    x = I.bf16_to_f64(d["x_attn"][rows_t])
    z_rows = I.bf16_to_f64(d["z"][rows_t])
    W_e, W_d = I.bf16_to_f64(d["W_e"]), I.bf16_to_f64(d["W_d"])
    b_all, a_all, gb_all = f64(b), f64(a), f64(gb)

    ref_b, ref_a = O.encode_fwd(x, z_rows, W_e, SILU)
    check("b", b_all[rows], ref_b, True)
    check("a_save", a_all[rows], ref_a, False)
    ref_zt = O.decode_fwd(b_all[rows], W_d[:, cols], False)
    check("z_tilde", f64(zt[rows_d][:, cols_d]), ref_zt, True)
    g_zt_rows = I.bf16_to_f64(d["g_zt"][rows_t])
    ref_gb = O.decode_input_grad(g_zt_rows, W_d, I.bf16_to_f64(d["g_id"][rows_t]))
    check("g_b", gb_all[rows], ref_gb, True)
    g_zt_cols = I.bf16_to_f64(d["g_zt"][:, cols_t])
    check("dW_d", f64(dWd)[:, cols], O.decode_weight_grad(b_all, g_zt_cols), False)
    g_h = O.encode_local_grad(gb_all, a_all, SILU)
    ref_gz = O.encode_input_grad(g_h[rows], W_e[cols])
    check("g_z", f64(gz[rows_d][:, cols_d]), ref_gz, True)
    z_cols = I.bf16_to_f64(d["z"][:, cols_t])
    check("dW_e", f64(dWe)[cols], O.encode_weight_grad(z_cols, g_h), False)
