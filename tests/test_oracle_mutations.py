"""Planted mistakes in the oracle must make a pin fail.

Each case swaps one oracle function for a plausible wrong version (a dropped
term, a wrong sign, the wrong columns, a swapped operand) and runs a pin that
should reject it.  Everything here runs on the CPU.
"""
import numpy as np
import pytest

import oracle as O
from oracle import resbm_oracle as R
import test_oracle_pins as P
import test_oracle_properties as PP


def _silu_dphi_dropped_term(a, act):
    if act == O.ACT_SILU:
        return 1.0 / (1.0 + np.exp(-a))        # sigma(a) only
    return np.ones_like(a)


def _p_id_first_columns_dropped(x, C):
    L, c = x.shape
    if c > C:
        return np.array(x[:, c - C:], copy=True)
    out = np.zeros((L, C))
    out[:, :c] = x
    return out


def _decode_input_grad_no_identity(g_zt, W_d, g_id):
    return g_zt @ W_d.T


def _encode_weight_grad_mean_not_sum(z, g_h):
    return (z.T @ g_h) / z.shape[0]


def _phi_sign(a, act):
    if act == O.ACT_SILU:
        return a / (1.0 + np.exp(a))
    return np.array(a, copy=True)


def _rne_truncate(x):
    x = np.asarray(x, dtype=np.float64)
    f = x.astype(np.float32)
    return ((f.view(np.uint32) >> 16) << 16).view(np.float32).astype(np.float64)


def _chain_wire_gradient_unrounded(x_attn, z, W_e, W_d, g_zt, g_id, act, add_identity, wire_round=True):
    b, a = R.encode_fwd(x_attn, z, W_e, act)
    b_w = R.rne_bf16(b) if wire_round else b
    zt = R.decode_fwd(b_w, W_d, add_identity)
    g_b, dW_d = R.decode_bwd(b_w, W_d, g_zt, g_id)
    g_z, dW_e = R.encode_bwd(z, W_e, a, g_b, act)
    return {"a": a, "b": b, "b_wire": b_w, "z_tilde": zt, "g_b": g_b, "g_b_wire": g_b, "dW_d": dW_d,
            "g_z": g_z, "dW_e": dW_e}


def _chain_decoder_grad_on_unrounded_payload(x_attn, z, W_e, W_d, g_zt, g_id, act, add_identity, wire_round=True):
    b, a = R.encode_fwd(x_attn, z, W_e, act)
    b_w = R.rne_bf16(b) if wire_round else b
    zt = R.decode_fwd(b_w, W_d, add_identity)
    g_b, dW_d = R.decode_bwd(b, W_d, g_zt, g_id)
    g_bw = R.rne_bf16(g_b) if wire_round else g_b
    g_z, dW_e = R.encode_bwd(z, W_e, a, g_bw, act)
    return {"a": a, "b": b, "b_wire": b_w, "z_tilde": zt, "g_b": g_b, "g_b_wire": g_bw, "dW_d": dW_d,
            "g_z": g_z, "dW_e": dW_e}


def _encode_local_grad_no_dphi(g_b, a, act):
    return np.array(g_b, copy=True)


def _decode_weight_grad_reversed_j(b, g_zt):
    return b[:, ::-1].T @ g_zt


def _skip_grad_last_columns(g_x, g_b):
    out = np.array(g_x, copy=True)
    out[:, out.shape[1] - g_b.shape[1]:] += g_b
    return out


MUTATIONS = [
    ("dphi", _silu_dphi_dropped_term,
     lambda: P.test_gradients_finite_differences(O.ACT_SILU, False, 3, 8, 2)),
    ("p_id", _p_id_first_columns_dropped, P.test_p_id_cases_worked_example),
    ("decode_input_grad", _decode_input_grad_no_identity,
     lambda: P.test_gradients_torch_autograd(O.ACT_IDENTITY, False)),
    ("encode_weight_grad", _encode_weight_grad_mean_not_sum,
     lambda: P.test_gradients_torch_autograd(O.ACT_SILU, True)),
    ("phi", _phi_sign, lambda: P.test_forward_brute_force(O.ACT_SILU, False, 3, 8, 2)),
    ("rne_bf16", _rne_truncate, P.test_rne_bf16_matches_torch_on_float32_inputs),
    ("boundary_fwd_bwd", _chain_wire_gradient_unrounded,
     lambda: P.test_wire_rounded_chain_torch_autograd(O.ACT_SILU, False)),
    ("boundary_fwd_bwd", _chain_decoder_grad_on_unrounded_payload,
     lambda: P.test_wire_rounded_chain_torch_autograd(O.ACT_IDENTITY, True)),
    # the property-based adjoint pins
    ("encode_local_grad", _encode_local_grad_no_dphi, lambda: PP.test_encode_backward_is_the_adjoint()),
    ("decode_weight_grad", _decode_weight_grad_reversed_j, lambda: PP.test_decode_backward_is_the_adjoint()),
    ("skip_grad", _skip_grad_last_columns, lambda: PP.test_encode_backward_is_the_adjoint()),
    ("decode_input_grad", _decode_input_grad_no_identity, lambda: PP.test_decode_backward_is_the_adjoint()),
]


@pytest.mark.parametrize("name,bad,pin", MUTATIONS, ids=[f"{m[0]}:{m[1].__name__.lstrip('_')}" for m in MUTATIONS])
def test_pin_rejects_planted_mistake(monkeypatch, name, bad, pin):
    monkeypatch.setattr(R, name, bad)
    monkeypatch.setattr(O, name, bad)
    with pytest.raises(AssertionError):
        pin()


# ------------------------------------------------ optimizer-side oracle (Muon)
from oracle import muon_oracle as MU  # noqa: E402
import test_muon_oracle_pins as MP  # noqa: E402


def _ns_no_quintic_term(U, steps=5, coeffs=MU.NS_QUINTIC, eps=MU.NS_EPS):
    a, b, c = coeffs
    tall = U.shape[0] > U.shape[1]
    X = U.T if tall else U
    X = X / (np.sqrt(np.sum(X * X)) + eps)
    for _ in range(steps):
        X = a * X + b * (X @ X.T) @ X
    return X.T if tall else X


def _ns_max_norm(U, steps=5, coeffs=MU.NS_QUINTIC, eps=MU.NS_EPS):
    a, b, c = coeffs
    tall = U.shape[0] > U.shape[1]
    X = U.T if tall else U
    X = X / (np.abs(X).max() + eps)
    with np.errstate(all="ignore"):  # the wrong normalisation can diverge
        for _ in range(steps):
            A = X @ X.T
            X = a * X + (b * A + c * (A @ A)) @ X
    return X.T if tall else X


def _muon_no_momentum_factor(W, G, M, lr, momentum, weight_decay=0.0, scale=None, nesterov=False, steps=5,
                             coeffs=MU.NS_QUINTIC, eps=MU.NS_EPS):
    scale = MU.default_scale(*np.shape(W)) if scale is None else scale
    M_new = MU.to_f32(np.asarray(M) + G)
    U = G + momentum * M_new if nesterov else M_new
    O = MU.newton_schulz(U, steps, coeffs, eps)
    return MU.to_f32(W - lr * (scale * O + weight_decay * W)), M_new, O


def _muon_nesterov_ignored(W, G, M, lr, momentum, weight_decay=0.0, scale=None, nesterov=False, steps=5,
                           coeffs=MU.NS_QUINTIC, eps=MU.NS_EPS):
    scale = MU.default_scale(*np.shape(W)) if scale is None else scale
    M_new = MU.to_f32(momentum * np.asarray(M) + G)
    O = MU.newton_schulz(M_new, steps, coeffs, eps)
    return MU.to_f32(W - lr * (scale * O + weight_decay * W)), M_new, O


def _spectrum_unsquared(W):
    sigma = np.linalg.svd(np.asarray(W, dtype=np.float64), compute_uv=False)
    return sigma, float(np.sum(sigma) / sigma[0]) if sigma.size and sigma[0] > 0 else 0.0


MUON_MUTATIONS = [
    ("newton_schulz", _ns_no_quintic_term,
     lambda: MP.test_newton_schulz_acts_on_singular_values(64, 8, False, MU.NS_QUINTIC, 5)),
    ("newton_schulz", _ns_max_norm,
     lambda: MP.test_newton_schulz_acts_on_singular_values(40, 40, True, MU.NS_CUBIC, 7)),
    ("muon_update", _muon_no_momentum_factor, MP.test_muon_update_momentum_recurrence_and_direction),
    ("muon_update", _muon_nesterov_ignored, MP.test_muon_update_momentum_recurrence_and_direction),
    ("spectrum", _spectrum_unsquared, lambda: MP.test_spectrum_of_built_matrices(90, 9)),
]


@pytest.mark.parametrize("name,bad,pin", MUON_MUTATIONS,
                         ids=[f"{m[0]}:{m[1].__name__.lstrip('_')}" for m in MUON_MUTATIONS])
def test_muon_pin_rejects_planted_mistake(monkeypatch, name, bad, pin):
    monkeypatch.setattr(MU, name, bad)
    with pytest.raises(AssertionError):
        pin()


# ---------------------------------------------------------------- two-linears-per-side oracle
import test_two_linear_oracle_pins as TP  # noqa: E402
from oracle import two_linear_oracle as TL  # noqa: E402


def _dec2_bwd_no_dphi(b, v, g_zt, g_id, W3, W4, act):
    p = R.phi(v, act)
    g_v = g_zt @ W4.T
    g_b = g_v @ W3.T + (g_id[:, :W3.shape[0]] if g_id is not None else 0)
    return g_b, b.T @ g_v, p.T @ g_zt


def _dec2_bwd_no_identity(b, v, g_zt, g_id, W3, W4, act):
    p = R.phi(v, act)
    g_v = (g_zt @ W4.T) * R.dphi(v, act)
    return g_v @ W3.T, b.T @ g_v, p.T @ g_zt


def _enc2_bwd_dw2_before_phi(z, u, g_b, W1, W2, act):
    g_u = (g_b @ W2.T) * R.dphi(u, act)
    return g_u @ W1.T, z.T @ g_u, u.T @ g_b


def _enc2_fwd_phi_after_second_layer(x_attn, z, W1, W2, act):
    u = z @ W1
    return x_attn[:, :W2.shape[1]] + R.phi(u @ W2, act), u


def _dec2_fwd_phi_on_input(b, W3, W4, act):
    v = b @ W3
    return R.phi(b, act) @ W3 @ W4, v


TWO_LINEAR_MUTATIONS = [
    ("decode2_bwd", _dec2_bwd_no_dphi, lambda: TP.test_gradients_finite_differences(R.ACT_SILU)),
    ("decode2_bwd", _dec2_bwd_no_identity, lambda: TP.test_gradients_torch_autograd(R.ACT_IDENTITY)),
    ("encode2_bwd", _enc2_bwd_dw2_before_phi, TP.test_unit_second_layer_is_one_linear_encoder),
    ("encode2_fwd", _enc2_fwd_phi_after_second_layer, lambda: TP.test_gradients_torch_autograd(R.ACT_SILU)),
    ("decode2_fwd", _dec2_fwd_phi_on_input, lambda: TP.test_gradients_torch_autograd(R.ACT_SILU)),
]


@pytest.mark.parametrize("name,bad,pin", TWO_LINEAR_MUTATIONS,
                         ids=[f"{m[0]}:{m[1].__name__.lstrip('_')}" for m in TWO_LINEAR_MUTATIONS])
def test_two_linear_pin_rejects_planted_mistake(monkeypatch, name, bad, pin):
    monkeypatch.setattr(TL, name, bad)
    with pytest.raises(AssertionError):
        pin()


# ---------------------------------------------------------------- fused FFN projection + encoder
import test_fusion_oracle_pins as FP  # noqa: E402
from oracle import fusion_oracle as FO  # noqa: E402


def _fused_skip_dropped(x_attn, z, W_e, act):
    a = z @ W_e
    return R.phi(a, act), a


def _fused_weight_rows_reversed(h, W_down, x_attn, W_e, act):
    z = h @ W_down
    b, a = R.encode_fwd(x_attn, R.rne_bf16(z), W_e[::-1], act)
    return z, b, a


@pytest.mark.parametrize("bad,pin", [
    (_fused_weight_rows_reversed, lambda: FP.test_integer_inputs_follow_associativity(R.ACT_SILU)),
])
def test_fusion_pin_rejects_planted_mistake(monkeypatch, bad, pin):
    monkeypatch.setattr(FO, "ffn_encode_fwd", bad)
    with pytest.raises(AssertionError):
        pin()


def test_fusion_pin_rejects_dropped_skip(monkeypatch):
    monkeypatch.setattr(FO, "encode_fwd", _fused_skip_dropped)
    with pytest.raises(AssertionError):
        FP.test_integer_inputs_follow_associativity(R.ACT_IDENTITY)


# ---------------------------------------------------------------- decoder into normalisation + QKV
def _rms_sum_not_mean(x, gamma, eps):
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.sum(x * x, axis=1, keepdims=True) + eps) * gamma[None, :]


def _rms_gain_dropped(x, gamma, eps):
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=1, keepdims=True) + eps)


def _rms_eps_outside_root(x, gamma, eps):
    x = np.asarray(x, dtype=np.float64)
    return x / (np.sqrt(np.mean(x * x, axis=1, keepdims=True)) + eps) * gamma[None, :]


@pytest.mark.parametrize("bad,pin", [
    (_rms_sum_not_mean, FP.test_decode_qkv_rows_have_unit_mean_square),
    (_rms_gain_dropped, FP.test_decode_qkv_scale_invariance_and_gain),
    (_rms_eps_outside_root, FP.test_decode_qkv_brute_force_loops),
], ids=["sum_not_mean", "gain_dropped", "eps_outside_root"])
def test_decode_qkv_pin_rejects_planted_mistake(monkeypatch, bad, pin):
    monkeypatch.setattr(FO, "rms_norm", bad)
    with pytest.raises(AssertionError):
        pin()
