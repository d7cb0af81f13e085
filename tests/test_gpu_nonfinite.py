"""Non-finite inputs propagate as IEEE arithmetic says (GPU against the oracle).

The kernels carry float32 weights as hi + lo bf16 pairs.  An infinite weight
gets an infinite hi part and a zero lo part, so each of its products is an
infinity of the right sign, never inf - inf = NaN; a NaN activation or
gradient makes every output it reaches NaN.  The GPU's NaNs and infinities
must sit exactly where the float64 oracle's are (infinities with the same
sign), and the finite entries keep the parity tests' bound.  One exception:
encode_bwd's g_z multiplies the split g_h by the split W_e (three products),
so an infinite weight also meets g_h's lo part (inf * 0, or an opposite sign)
and those entries come out NaN where the oracle has +-inf; there only the set
of non-finite entries must match.  Shapes cover the
in-kernel weight split (r = 16), the prepared fragments (r = 32) and the
wide-rank kernels (r = 128).
"""
import numpy as np
import pytest
import torch

import oracle as O
from gpu_helpers import check, f64, lib, say, to_dev
from paper_2604_11947_amd import inputs as I

pytestmark = pytest.mark.gpu

ID, SILU = O.ACT_IDENTITY, O.ACT_SILU
SHAPES = [(300, 256, 16), (300, 256, 32), (200, 512, 128)]
IDS = [f"T{T}_n{n}_r{r}" for T, n, r in SHAPES]


def same_nonfinite(name: str, gpu, ref: np.ndarray, bf16_output: bool, exact: bool = True) -> None:
    g = f64(gpu)
    fin = np.isfinite(ref)
    assert np.array_equal(np.isfinite(g), fin), \
        f"{name}: finiteness differs at {np.argwhere(np.isfinite(g) != fin)[:4].tolist()}"
    if exact:
        nan_g, nan_r = np.isnan(g), np.isnan(ref)
        assert np.array_equal(nan_g, nan_r), f"{name}: NaN at {np.argwhere(nan_g != nan_r)[:4].tolist()}"
        assert np.array_equal(np.isposinf(g), np.isposinf(ref)), f"{name}: +inf pattern differs"
        assert np.array_equal(np.isneginf(g), np.isneginf(ref)), f"{name}: -inf pattern differs"
    assert (~fin).any(), f"{name}: the case planted no non-finite output"
    say(f"    {name:10s} {int(np.isnan(ref).sum())} NaN, {int(np.isinf(ref).sum())} inf of {ref.size}")
    check(name, np.where(fin, g, 0.0), np.where(fin, ref, 0.0), bf16_output=bf16_output)


def inputs(T, n, r, seed):
    d = I.make_inputs(T, n, r, "normal", seed)
    g = to_dev(d)
    return g, {k: I.bf16_to_f64(v) for k, v in d.items() if k != "meta"}


@pytest.mark.parametrize("act", [ID, SILU])
@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_encode_fwd_inf_weight_nan_token(shape, act):
    """W_e[5][3] = +inf: column 3 of a is +-inf for every token (SiLU of -inf
    is NaN); z[7][11] = NaN: token 7's a and b are NaN."""
    T, n, r = shape
    say(f"encode_fwd non-finite T={T} n={n} r={r} act={act}")
    L = lib()
    g, f = inputs(T, n, r, seed=21)
    g["W_e"][5, 3] = float("inf")
    g["z"][7, 11] = float("nan")
    f["W_e"] = f64(g["W_e"])
    f["z"] = f64(g["z"])
    b = torch.empty(T, r, dtype=L.io_dtype, device="cuda")
    a = torch.empty(T, r, dtype=torch.float32, device="cuda")
    L.encode_fwd(g["x_attn"], g["z"], g["W_e"], b, a, act=act)
    torch.cuda.synchronize()
    with np.errstate(all="ignore"):
        ref_b, ref_a = O.encode_fwd(f["x_attn"], f["z"], f["W_e"], act)
    same_nonfinite("a_save", a, ref_a, bf16_output=False)
    same_nonfinite("b", b, ref_b, bf16_output=True)


@pytest.mark.parametrize("add_identity", [False, True])
@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_decode_fwd_inf_weight(shape, add_identity):
    """W_d[2][17] = -inf: column 17 of z~ is -+inf for every token."""
    T, n, r = shape
    say(f"decode_fwd non-finite T={T} n={n} r={r} add_identity={add_identity}")
    L = lib()
    g, f = inputs(T, n, r, seed=22)
    b = torch.empty(T, r, dtype=L.io_dtype, device="cuda")
    L.encode_fwd(g["x_attn"], g["z"], g["W_e"], b, None, act=SILU)
    g["W_d"][2, 17] = float("-inf")
    zt = torch.empty(T, n, dtype=L.io_dtype, device="cuda")
    L.decode_fwd(b, g["W_d"], zt, add_identity=add_identity)
    torch.cuda.synchronize()
    with np.errstate(all="ignore"):
        ref = O.decode_fwd(f64(b), f64(g["W_d"]), add_identity)
    same_nonfinite("z_tilde", zt, ref, bf16_output=True)


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_decode_bwd_inf_weight_nan_gradient(shape):
    """W_d[2][17] = -inf: column 2 of g_b is +-inf for every token; g_z~[9][40]
    = NaN: token 9's g_b and column 40 of dW_d are NaN."""
    T, n, r = shape
    say(f"decode_bwd non-finite T={T} n={n} r={r}")
    L = lib()
    g, f = inputs(T, n, r, seed=23)
    b = torch.empty(T, r, dtype=L.io_dtype, device="cuda")
    L.encode_fwd(g["x_attn"], g["z"], g["W_e"], b, None, act=SILU)
    g["W_d"][2, 17] = float("-inf")
    g["g_zt"][9, 40] = float("nan")
    gb = torch.empty(T, r, dtype=L.io_dtype, device="cuda")
    dW = torch.empty(r, n, dtype=torch.float32, device="cuda")
    L.decode_bwd(b, g["W_d"], g["g_zt"], g["g_id"], gb, dW)
    torch.cuda.synchronize()
    with np.errstate(all="ignore"):
        ref_gb, ref_dw = O.decode_bwd(f64(b), f64(g["W_d"]), f64(g["g_zt"]), f["g_id"])
    same_nonfinite("g_b", gb, ref_gb, bf16_output=True)
    same_nonfinite("dW_d", dW, ref_dw, bf16_output=False)


@pytest.mark.parametrize("act", [ID, SILU])
@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_encode_bwd_nan_gradient_inf_weight(shape, act):
    """g_b[4][1] = NaN: token 4's g_z and column 1 of dW_e are NaN; W_e[6][0] =
    +inf: column 6 of g_z is non-finite wherever g_h[:, 0] is non-zero (the
    oracle's +-inf; NaN or +-inf on the GPU)."""
    T, n, r = shape
    say(f"encode_bwd non-finite T={T} n={n} r={r} act={act}")
    L = lib()
    g, f = inputs(T, n, r, seed=24)
    b = torch.empty(T, r, dtype=L.io_dtype, device="cuda")
    a = torch.empty(T, r, dtype=torch.float32, device="cuda")
    L.encode_fwd(g["x_attn"], g["z"], g["W_e"], b, a, act=act)
    gb = torch.empty(T, r, dtype=L.io_dtype, device="cuda")
    L.decode_bwd(b, g["W_d"], g["g_zt"], g["g_id"], gb, torch.empty(r, n, dtype=torch.float32, device="cuda"))
    gb[4, 1] = float("nan")
    g["W_e"][6, 0] = float("inf")
    gz = torch.empty(T, n, dtype=L.io_dtype, device="cuda")
    dWe = torch.empty(n, r, dtype=torch.float32, device="cuda")
    L.encode_bwd(g["z"], g["W_e"], a if act == SILU else None, gb, gz, dWe, act=act)
    torch.cuda.synchronize()
    with np.errstate(all="ignore"):
        ref_gz, ref_dw = O.encode_bwd(f["z"], f64(g["W_e"]), f64(a), f64(gb), act)
    same_nonfinite("g_z", gz, ref_gz, bf16_output=True, exact=False)
    same_nonfinite("dW_e", dWe, ref_dw, bf16_output=False)
