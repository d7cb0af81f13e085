"""Property-based pins of the oracle: its backward ops are the adjoints of its
forward ops, on random shapes.

For a map f with upstream gradient g and any direction d, the vector-Jacobian
product the backward op returns must satisfy <J^T g, d> = <g, J d>, with J d
taken by central finite differences of the forward op (exact for the linear
maps, O(eps^2) for SiLU).  Shapes are drawn over 1 <= r <= n (r = n, the
full-rank case, included), single tokens and odd widths, both activations and
both decoder readings, so a transposed operand, a dropped term or a wrong index
anywhere in the backward formulas fails for some draw.  Forward (Sec. 3.2 with
Eq. 2 and Eq. 5) and backward (their exact adjoints) as in the oracle.
"""
import numpy as np
from hypothesis import given, settings, strategies as st

import oracle as O

EPS = 1e-6
SETTINGS = settings(max_examples=60, deadline=None, derandomize=True)


@st.composite
def boundary(draw):
    T = draw(st.integers(1, 6))
    n = draw(st.integers(1, 12))
    r = draw(st.integers(1, n))
    seed = draw(st.integers(0, 2**31 - 1))
    return T, n, r, np.random.default_rng(seed)


def dot(a, b) -> float:
    return float(np.sum(a * b))


def close(lhs: float, rhs: float, scale: float, tol: float) -> None:
    assert abs(lhs - rhs) <= tol * max(scale, 1e-300), (lhs, rhs, scale)


@SETTINGS
@given(boundary(), st.sampled_from([O.ACT_IDENTITY, O.ACT_SILU]))
def test_encode_backward_is_the_adjoint(case, act):
    T, n, r, rng = case
    x, z = rng.standard_normal((T, n)), rng.standard_normal((T, n))
    W = rng.standard_normal((n, r)) / np.sqrt(n)
    g_b = rng.standard_normal((T, r))
    dz, dW, dx = rng.standard_normal((T, n)), rng.standard_normal((n, r)), rng.standard_normal((T, n))
    _, a = O.encode_fwd(x, z, W, act)
    g_z, g_W = O.encode_bwd(z, W, a, g_b, act)

    def b_of(x_, z_, W_):
        return O.encode_fwd(x_, z_, W_, act)[0]

    jz = (b_of(x, z + EPS * dz, W) - b_of(x, z - EPS * dz, W)) / (2 * EPS)
    jW = (b_of(x, z, W + EPS * dW) - b_of(x, z, W - EPS * dW)) / (2 * EPS)
    jx = (b_of(x + EPS * dx, z, W) - b_of(x - EPS * dx, z, W)) / (2 * EPS)
    scale = np.linalg.norm(g_b) * (np.linalg.norm(jz) + np.linalg.norm(jW) + np.linalg.norm(jx) + 1.0)
    close(dot(g_b, jz), dot(g_z, dz), scale, 1e-7)
    close(dot(g_b, jW), dot(g_W, dW), scale, 1e-7)
    # the identity path's adjoint: g_x[:, :r] += g_b, columns >= r untouched
    g_x = O.skip_grad(np.zeros((T, n)), g_b)
    close(dot(g_b, jx), dot(g_x, dx), scale, 1e-7)
    assert not np.any(g_x[:, r:])


@SETTINGS
@given(boundary(), st.booleans())
def test_decode_backward_is_the_adjoint(case, add_identity):
    T, n, r, rng = case
    b = rng.standard_normal((T, r))
    W = rng.standard_normal((r, n)) / np.sqrt(r)
    g_zt = rng.standard_normal((T, n))
    db, dW = rng.standard_normal((T, r)), rng.standard_normal((r, n))
    # reading A (add_identity): the skip's gradient is g_z~ itself
    g_b, g_W = O.decode_bwd(b, W, g_zt, g_zt if add_identity else None)

    def zt_of(b_, W_):
        return O.decode_fwd(b_, W_, add_identity)

    jb = (zt_of(b + EPS * db, W) - zt_of(b - EPS * db, W)) / (2 * EPS)
    jW = (zt_of(b, W + EPS * dW) - zt_of(b, W - EPS * dW)) / (2 * EPS)
    scale = np.linalg.norm(g_zt) * (np.linalg.norm(jb) + np.linalg.norm(jW) + 1.0)
    close(dot(g_zt, jb), dot(g_b, db), scale, 1e-8)
    close(dot(g_zt, jW), dot(g_W, dW), scale, 1e-8)


@SETTINGS
@given(boundary())
def test_decode_inverts_encode_at_full_rank_zero_branch(case):
    """Zero weights, r = n: the encoder passes the skip through and reading A's
    decoder returns it (Eq. 5 at c = C; Sec. 3.3)."""
    T, n, _, rng = case
    x, z = rng.standard_normal((T, n)), rng.standard_normal((T, n))
    b, _ = O.encode_fwd(x, z, np.zeros((n, n)), O.ACT_SILU)
    np.testing.assert_array_equal(b, x)
    np.testing.assert_array_equal(O.decode_fwd(b, np.zeros((n, n)), True), x)
