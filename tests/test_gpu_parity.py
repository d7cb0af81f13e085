"""HIP path vs the CPU oracle, through the C ABI.

Per-op parity feeds the oracle the same inputs the GPU op saw (including the
GPU's own bf16 payload / wire gradient / a_save for downstream ops); chain
parity runs the four ops back to back against the oracle's forward+backward
with bf16 rounding at the two wire crossings.  Tolerances: bf16 outputs
max(|gpu - ref| - ulp/2) <= 2e-2 RMS(ref); float32 outputs max|gpu - ref| <=
2e-2 RMS(ref); the fp32 validation build <= 1e-5 RMS(ref).
"""
import numpy as np
import pytest
import torch

import oracle as O
from gpu_helpers import (BF16_BOUND, F32_BOUND, check, f64, guarded, lib, say, strided, to_dev)
from paper_2604_11947_amd import inputs as I

pytestmark = pytest.mark.gpu

ID, SILU = O.ACT_IDENTITY, O.ACT_SILU

# (T, n, r): several tiles in every direction, ragged token tails, r not a
# multiple of 16 (4, 12, 40, 100, 136), full rank (r = n), the largest r, and
# the wide-rank kernels (r > 64) at odd tile counts.
SHAPES = [(1000, 512, 32), (777, 256, 4), (333, 320, 40), (517, 1024, 64), (45, 192, 12),
          (130, 128, 128), (96, 256, 256), (64, 64, 64), (1, 64, 4),
          # wide rank (r > 64): r % 8 == 4, r a multiple of 16, 48, 64, odd tile counts, n % 128 == 64, T = 1
          (333, 768, 100), (700, 576, 136), (1000, 1024, 192), (64, 256, 80), (1, 128, 128),
          # row contraction with r split over two blocks: one token, one group plus one token
          (1, 256, 200), (129, 512, 256),
          # token contraction in 64-token steps: 96-token groups (a step and a half) and a
          # ragged last group (28 and 24 tokens), with and without the split operand at its LDS limit
          (700, 4096, 136), (600, 4096, 256),
          # the remaining rank tilings (16-column tiles of r: 6, 10, 11, 14, 15), two with a ragged last tile
          (257, 512, 92), (130, 640, 160), (65, 384, 176), (200, 1024, 224), (97, 768, 236),
          # the maximum width n = 65536, narrow and widest rank
          (70, 65536, 32), (33, 65536, 256)]
IDS = [f"T{T}_n{n}_r{r}" for T, n, r in SHAPES]


def host(T, n, r, dist="normal", seed=0):
    d = I.make_inputs(T, n, r, dist, seed)
    return d, {k: I.bf16_to_f64(v) for k, v in d.items() if k != "meta"}


def run_encode_fwd(L, g, act, pad=0, save=True):
    T, n = g["z"].shape
    r = g["W_e"].shape[1]
    x = strided(g["x_attn"], pad)
    z = strided(g["z"], pad)
    b, _, chk_b = guarded((T, r), L.io_dtype, "cuda")
    a, _, chk_a = guarded((T, r), torch.float32, "cuda")
    L.encode_fwd(x, z, g["W_e"], b, a if save else None, act=act)
    torch.cuda.synchronize()
    chk_b()
    if save:
        chk_a()
    return b, a


@pytest.mark.parametrize("act", [ID, SILU])
@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_encode_fwd(shape, act):
    T, n, r = shape
    say(f"encode_fwd T={T} n={n} r={r} act={act}")
    L = lib()
    d, f = host(T, n, r)
    b, a = run_encode_fwd(L, to_dev(d), act, pad=8 if n > 64 else 0)
    ref_b, ref_a = O.encode_fwd(f["x_attn"], f["z"], f["W_e"], act)
    check("b", b, ref_b, bf16_output=True)
    check("a_save", a, ref_a, bf16_output=False)


@pytest.mark.parametrize("add_identity", [False, True])
@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_decode_fwd(shape, add_identity):
    T, n, r = shape
    say(f"decode_fwd T={T} n={n} r={r} add_identity={add_identity}")
    L = lib()
    d, f = host(T, n, r, seed=1)
    g = to_dev(d)
    b, _ = run_encode_fwd(L, g, SILU)
    pad = 24 if n > 64 else 0
    zt, _, chk = guarded((T, n), L.io_dtype, "cuda", pad=pad)
    L.decode_fwd(b, g["W_d"], zt, add_identity=add_identity)
    torch.cuda.synchronize()
    chk()
    ref = O.decode_fwd(f64(b), f["W_d"], add_identity)
    check("z_tilde", zt, ref, bf16_output=True)


@pytest.mark.parametrize("mode", ["separate", "alias", "none", "accumulate"])
@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_decode_bwd(shape, mode):
    T, n, r = shape
    say(f"decode_bwd T={T} n={n} r={r} mode={mode}")
    L = lib()
    d, f = host(T, n, r, seed=2)
    g = to_dev(d)
    b, _ = run_encode_fwd(L, g, SILU)
    g_zt = strided(g["g_zt"], 8 if n > 64 else 0)
    g_id = {"separate": g["g_id"], "alias": g_zt, "none": None, "accumulate": g["g_id"]}[mode]
    gb, _, chk = guarded((T, r), L.io_dtype, "cuda")
    prev = torch.randn(r, n, dtype=torch.float32, device="cuda") if mode == "accumulate" else None
    dW = prev.clone() if prev is not None else torch.full((r, n), float("nan"), device="cuda")
    L.decode_bwd(b, g["W_d"], g_zt, g_id, gb, dW, accumulate=(mode == "accumulate"))
    torch.cuda.synchronize()
    chk()
    f_id = {"separate": f["g_id"], "alias": f["g_zt"], "none": None, "accumulate": f["g_id"]}[mode]
    ref_gb, ref_dw = O.decode_bwd(f64(b), f["W_d"], f["g_zt"], f_id)
    if prev is not None:
        ref_dw = ref_dw + f64(prev)
    check("g_b", gb, ref_gb, bf16_output=True)
    check("dW_d", dW, ref_dw, bf16_output=False)


@pytest.mark.parametrize("gx", ["none", "separate", "fused"])
@pytest.mark.parametrize("act", [ID, SILU])
@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_encode_bwd(shape, act, gx):
    T, n, r = shape
    say(f"encode_bwd T={T} n={n} r={r} act={act} g_x={gx}")
    L = lib()
    d, f = host(T, n, r, seed=3)
    g = to_dev(d)
    b, a = run_encode_fwd(L, g, act)
    gb = torch.empty(T, r, dtype=L.io_dtype, device="cuda")
    dWd = torch.empty(r, n, dtype=torch.float32, device="cuda")
    L.decode_bwd(b, g["W_d"], g["g_zt"], g["g_id"], gb, dWd)
    pad = 16 if n > 64 else 0
    z = strided(g["z"], pad)
    gz, _, chk = guarded((T, n), L.io_dtype, "cuda", pad=pad)
    g_x = None
    if gx == "separate":
        g_x = strided(g["g_id"], 8 if n > 64 else 0)  # any residual gradient
        gx0 = f64(g_x)
    elif gx == "fused":
        g_x = gz
    accumulate = act == SILU and gx == "none"
    dWe = torch.randn(n, r, device="cuda") if accumulate else torch.full((n, r), float("nan"), device="cuda")
    prev = f64(dWe)
    L.encode_bwd(z, g["W_e"], a if act == SILU else None, gb, gz, dWe, g_x=g_x, act=act, accumulate=accumulate)
    torch.cuda.synchronize()
    chk()
    ref_gz, ref_dw = O.encode_bwd(f["z"], f["W_e"], f64(a), f64(gb), act)
    if accumulate:
        ref_dw = ref_dw + prev
    if gx == "fused":
        ref_gz = O.skip_grad(ref_gz, f64(gb))
    check("g_z", gz, ref_gz, bf16_output=True)
    check("dW_e", dWe, ref_dw, bf16_output=False)
    if gx == "separate":
        check("g_x", g_x, O.skip_grad(gx0, f64(gb)), bf16_output=True)
        np.testing.assert_array_equal(f64(g_x)[:, r:], gx0[:, r:])


@pytest.mark.parametrize("add_identity", [False, True])
@pytest.mark.parametrize("shape", [(1000, 512, 32), (333, 320, 40), (517, 1024, 64), (96, 256, 256)],
                         ids=["T1000_n512_r32", "T333_n320_r40", "T517_n1024_r64", "T96_n256_r256"])
def test_chain(shape, add_identity):
    """encode -> decode -> decode_bwd -> encode_bwd against the oracle's chain with
    bf16 rounding where the payload and its gradient cross the boundary."""
    T, n, r = shape
    say(f"chain T={T} n={n} r={r} add_identity={add_identity}")
    L = lib()
    d, f = host(T, n, r, dist="student_t3", seed=4)
    g = to_dev(d)
    b, a = run_encode_fwd(L, g, SILU)
    zt = torch.empty(T, n, dtype=L.io_dtype, device="cuda")
    L.decode_fwd(b, g["W_d"], zt, add_identity=add_identity)
    g_id = g["g_zt"] if add_identity else g["g_id"]
    gb = torch.empty(T, r, dtype=L.io_dtype, device="cuda")
    dWd = torch.empty(r, n, dtype=torch.float32, device="cuda")
    L.decode_bwd(b, g["W_d"], g["g_zt"], g_id, gb, dWd)
    gz = torch.empty(T, n, dtype=L.io_dtype, device="cuda")
    dWe = torch.empty(n, r, dtype=torch.float32, device="cuda")
    L.encode_bwd(g["z"], g["W_e"], a, gb, gz, dWe, act=SILU)
    torch.cuda.synchronize()
    ref = O.boundary_fwd_bwd(f["x_attn"], f["z"], f["W_e"], f["W_d"], f["g_zt"],
                             f["g_zt"] if add_identity else f["g_id"], SILU, add_identity)
    check("b", b, ref["b"], True)
    check("z_tilde", zt, ref["z_tilde"], True)
    check("g_b", gb, ref["g_b"], True)
    check("dW_d", dWd, ref["dW_d"], False)
    check("g_z", gz, ref["g_z"], True)
    check("dW_e", dWe, ref["dW_e"], False)


@pytest.mark.parametrize("act", [ID, SILU])
def test_zero_branch_is_exact_identity(act):
    """Zero weights leave only the identity path (Eq. 2 with F = 0, Eq. 5): exact."""
    L = lib()
    T, n, r = 300, 256, 32
    say(f"zero-branch T={T} n={n} r={r} act={act}")
    d, f = host(T, n, r, seed=5)
    g = to_dev(d)
    g["W_e"].zero_()
    g["W_d"].zero_()
    b, a = run_encode_fwd(L, g, act)
    assert torch.equal(b.view(torch.int16).cpu(), g["x_attn"][:, :r].contiguous().view(torch.int16).cpu())
    for add in (False, True):
        zt = torch.empty(T, n, dtype=L.io_dtype, device="cuda")
        L.decode_fwd(b, g["W_d"], zt, add_identity=add)
        torch.cuda.synchronize()
        expect = torch.zeros(T, n, dtype=L.io_dtype, device="cuda")
        if add:
            expect[:, :r] = b
        assert torch.equal(zt, expect)
    gb = torch.empty(T, r, dtype=L.io_dtype, device="cuda")
    dWd = torch.empty(r, n, dtype=torch.float32, device="cuda")
    L.decode_bwd(b, g["W_d"], g["g_zt"], g["g_id"], gb, dWd)
    torch.cuda.synchronize()
    assert torch.equal(gb, g["g_id"][:, :r].contiguous())
    gz = torch.empty(T, n, dtype=L.io_dtype, device="cuda")
    dWe = torch.empty(n, r, dtype=torch.float32, device="cuda")
    L.encode_bwd(g["z"], g["W_e"], a, gb, gz, dWe, act=act)
    torch.cuda.synchronize()
    assert not bool(gz.float().abs().max() > 0)
    ref = O.encode_weight_grad(f["z"], O.encode_local_grad(f64(gb), np.zeros((T, r)), act))
    check("dW_e", dWe, ref, bf16_output=False)


@pytest.mark.parametrize("n", [64, 128, 256])
def test_full_rank_reduces_to_residual(n):
    """r = n (Sec. 3.3): with a zero encoder branch b equals x_attn bit for bit."""
    L = lib()
    T = 200
    say(f"full-rank T={T} n={n}")
    d, f = host(T, n, n, seed=6)
    g = to_dev(d)
    g["W_e"].zero_()
    b, _ = run_encode_fwd(L, g, SILU)
    assert torch.equal(b.view(torch.int16), g["x_attn"].view(torch.int16))
    d2, f2 = host(T, n, n, seed=7)
    g2 = to_dev(d2)
    b2, a2 = run_encode_fwd(L, g2, SILU)
    check("b", b2, O.encode_fwd(f2["x_attn"], f2["z"], f2["W_e"], SILU)[0], True)


@pytest.mark.parametrize("shape", [(1000, 512, 32), (517, 1024, 64)], ids=["r32", "r64"])
def test_bitwise_deterministic(shape):
    T, n, r = shape
    say(f"determinism T={T} n={n} r={r}")
    L = lib()
    d, _ = host(T, n, r, seed=8)
    g = to_dev(d)

    def once():
        b, a = run_encode_fwd(L, g, SILU)
        zt = torch.empty(T, n, dtype=L.io_dtype, device="cuda")
        L.decode_fwd(b, g["W_d"], zt)
        gb = torch.empty(T, r, dtype=L.io_dtype, device="cuda")
        dWd = torch.empty(r, n, device="cuda")
        L.decode_bwd(b, g["W_d"], g["g_zt"], g["g_id"], gb, dWd)
        gz = torch.empty(T, n, dtype=L.io_dtype, device="cuda")
        dWe = torch.empty(n, r, device="cuda")
        L.encode_bwd(g["z"], g["W_e"], a, gb, gz, dWe, act=SILU)
        torch.cuda.synchronize()
        return [t.cpu().view(torch.uint8) for t in (b, a, zt, gb, dWd, gz, dWe)]

    for x, y in zip(once(), once()):
        assert torch.equal(x, y)


def test_empty_tokens_is_noop():
    from paper_2604_11947_amd import resbm as R
    L = lib()
    say("T=0")
    n, r = 256, 32
    W_e = torch.randn(n, r, device="cuda")
    W_d = torch.randn(r, n, device="cuda")
    e = torch.empty(0, n, dtype=L.io_dtype, device="cuda")
    p = torch.empty(0, r, dtype=L.io_dtype, device="cuda")
    a = torch.empty(0, r, dtype=torch.float32, device="cuda")
    dWd = torch.full((r, n), 3.0, device="cuda")
    dWe = torch.full((n, r), 3.0, device="cuda")
    L.encode_fwd(e, e, W_e, p, a)
    L.decode_fwd(p, W_d, e)
    L.decode_bwd(p, W_d, e, e, p, dWd)
    L.encode_bwd(e, W_e, a, p, e, dWe)
    torch.cuda.synchronize()
    assert bool((dWd == 3.0).all()) and bool((dWe == 3.0).all())
    assert R.OK == 0


def test_error_paths_with_real_buffers():
    from paper_2604_11947_amd import resbm as R
    L = lib()
    say("error paths")
    T, n, r = 128, 256, 32
    d, _ = host(T, n, r)
    g = to_dev(d)
    b = torch.empty(T, r, dtype=L.io_dtype, device="cuda")
    a = torch.empty(T, r, dtype=torch.float32, device="cuda")
    ws = L.workspace(T, n, r, "cuda")
    c = L.cdll
    s = None
    base = (T, n, r, 1, g["x_attn"].data_ptr(), n, g["z"].data_ptr(), n, g["W_e"].data_ptr(), b.data_ptr(),
            a.data_ptr(), ws.data_ptr(), ws.numel(), s)

    def call(**over):
        args = list(base)
        names = ["T", "n", "r", "act", "x", "ldx", "z", "ldz", "We", "b", "a", "ws", "wsb", "s"]
        for k, v in over.items():
            args[names.index(k)] = v
        return c.resbm_encode_fwd(*args)

    assert call(z=g["z"].data_ptr() + 2) == R.E_ALIGN
    assert call(wsb=256) == R.E_WORKSPACE
    assert call(act=7) == R.E_ACT
    assert call(ldz=n - 8) == R.E_SHAPE
    assert call(r=6) == R.E_SHAPE
    assert call(b=g["z"].data_ptr()) == R.E_ALIAS
    assert call(ws=None) == R.E_NULL
    gz = torch.empty(T, n, dtype=L.io_dtype, device="cuda")
    dWe = torch.empty(n, r, device="cuda")
    with pytest.raises(R.ResbmError) as ei:
        L.encode_bwd(g["z"], g["W_e"], None, b, gz, dWe, act=R.ACT_SILU)
    assert ei.value.status == R.E_ACT
    with pytest.raises(R.ResbmError) as ei:
        L.encode_bwd(g["z"], g["W_e"], a, b, gz, dWe, g_x=g["z"], act=R.ACT_SILU)
    assert ei.value.status == R.E_ALIAS
    torch.cuda.synchronize()
