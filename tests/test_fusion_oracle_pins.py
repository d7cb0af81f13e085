"""Pins of the fused FFN-projection + encoder oracle.

With small-integer h and W_down every element of z is exact in bf16, so the
fused result must equal the encoder applied to h (W_down W_e) by
associativity; with W_down the identity it must equal the (pinned) encoder on
h itself.  Everything runs on the CPU.
"""
import numpy as np
import pytest

from oracle import fusion_oracle as F
from oracle import resbm_oracle as R


@pytest.mark.parametrize("act", [R.ACT_IDENTITY, R.ACT_SILU])
def test_integer_inputs_follow_associativity(act):
    rng = np.random.default_rng(3)
    T, d_ff, n, r = 7, 8, 24, 8
    h = rng.integers(-2, 3, (T, d_ff)).astype(np.float64)
    Wd = rng.integers(-2, 3, (d_ff, n)).astype(np.float64)
    x = rng.standard_normal((T, n))
    We = rng.standard_normal((n, r)) / np.sqrt(n)
    z, b, a = F.ffn_encode_fwd(h, Wd, x, We, act)
    assert np.all(np.abs(z) <= 32) and np.array_equal(R.rne_bf16(z), z)
    np.testing.assert_allclose(a, h @ (Wd @ We), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(b, x[:, :r] + R.phi(h @ (Wd @ We), act), rtol=1e-12, atol=1e-12)


def test_identity_projection_is_the_encoder():
    rng = np.random.default_rng(4)
    T, n, r = 9, 32, 8
    h = R.rne_bf16(rng.standard_normal((T, n)))
    x = rng.standard_normal((T, n))
    We = rng.standard_normal((n, r))
    z, b, a = F.ffn_encode_fwd(h, np.eye(n), x, We, R.ACT_SILU)
    np.testing.assert_array_equal(z, h)
    b1, a1 = R.encode_fwd(x, h, We, R.ACT_SILU)
    np.testing.assert_array_equal(b, b1)
    np.testing.assert_array_equal(a, a1)
