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
]


@pytest.mark.parametrize("name,bad,pin", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_pin_rejects_planted_mistake(monkeypatch, name, bad, pin):
    monkeypatch.setattr(R, name, bad)
    monkeypatch.setattr(O, name, bad)
    with pytest.raises(AssertionError):
        pin()
