"""Pins of the fusion oracles (encoder into the FFN projection, decoder into
the next block's normalisation and QKV projection).

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


# ---- decoder into the normalisation and QKV projection

def _dq_inputs(seed, T=6, n=32, r=8, N=24):
    rng = np.random.default_rng(seed)
    b = rng.standard_normal((T, r))
    Wd = rng.standard_normal((r, n)) / np.sqrt(r)
    g = 1.0 + 0.1 * rng.standard_normal(n)
    W = rng.standard_normal((n, N)) / np.sqrt(n)
    return b, Wd, g, W


def test_decode_qkv_rows_have_unit_mean_square():
    """gamma = 1, W_qkv = I, eps = 0: every output row has mean square exactly 1
    and is parallel to the decoder output."""
    b, Wd, _, _ = _dq_inputs(5)
    n = Wd.shape[1]
    zt, y, out = F.decode_qkv_fwd(b, Wd, np.ones(n), np.eye(n), 0.0)
    np.testing.assert_allclose(np.mean(out * out, axis=1), 1.0, rtol=1e-13)
    np.testing.assert_allclose(out * np.sqrt(np.mean(zt * zt, axis=1, keepdims=True)), zt, rtol=1e-12, atol=1e-14)
    np.testing.assert_array_equal(zt, R.decode_fwd(b, Wd, False))


def test_decode_qkv_scale_invariance_and_gain():
    """eps = 0: scaling b leaves the output unchanged; the output is linear in
    gamma and in W_qkv."""
    b, Wd, g, W = _dq_inputs(6)
    _, _, o1 = F.decode_qkv_fwd(b, Wd, g, W, 0.0)
    _, _, o2 = F.decode_qkv_fwd(7.5 * b, Wd, g, W, 0.0)
    np.testing.assert_allclose(o2, o1, rtol=1e-12, atol=1e-13)
    g2 = np.linspace(0.5, 1.5, g.size)
    _, _, oa = F.decode_qkv_fwd(b, Wd, g + g2, W, 1e-5)
    _, _, ob = F.decode_qkv_fwd(b, Wd, g, W, 1e-5)
    _, _, oc = F.decode_qkv_fwd(b, Wd, g2, W, 1e-5)
    np.testing.assert_allclose(oa, ob + oc, rtol=1e-12, atol=1e-13)
    _, _, od = F.decode_qkv_fwd(b, Wd, g, 2.0 * W, 1e-5)
    np.testing.assert_allclose(od, 2.0 * ob, rtol=1e-13)


def test_decode_qkv_brute_force_loops():
    """Scalar loops at a tiny shape, eps > 0, and a zero payload row (output 0)."""
    b, Wd, g, W = _dq_inputs(7, T=3, n=8, r=2, N=5)
    b[1] = 0.0
    eps = 1e-3
    _, _, out = F.decode_qkv_fwd(b, Wd, g, W, eps)
    T, r = b.shape
    n, N = W.shape
    for t in range(T):
        zt = [sum(b[t][j] * Wd[j][c] for j in range(r)) for c in range(n)]
        ms = sum(v * v for v in zt) / n
        y = [zt[c] / (ms + eps) ** 0.5 * g[c] for c in range(n)]
        for k in range(N):
            ref = sum(y[c] * W[c][k] for c in range(n))
            assert abs(out[t][k] - ref) <= 1e-12 * (1 + abs(ref))
    assert np.all(out[1] == 0.0)
