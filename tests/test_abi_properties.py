"""Property-based checks of the C ABI's shape rules (host only: workspace
queries and calls that validation rejects before any HIP call).

For random (T, n, r) the workspace query is non-zero exactly when the header's
shape rules hold, is a multiple of 256 and grows with T; every op returns
RESBM_E_SHAPE for shapes outside the rules (with otherwise valid arguments) and
succeeds as a no-op at T = 0 inside them.  The two-linear and optimizer-side
queries follow their own rules the same way.
"""
import os

import pytest
import torch
from hypothesis import HealthCheck, given, settings, strategies as st

from paper_2604_11947_amd import build as B
from paper_2604_11947_amd import resbm as R

SETTINGS = settings(max_examples=300, deadline=None, derandomize=True,
                    suppress_health_check=[HealthCheck.function_scoped_fixture])
needs_no_gpu = pytest.mark.skipif(torch.cuda.is_available(),
                                  reason="fake device addresses; host validation is covered on CPU hosts")


@pytest.fixture(scope="module", params=["bf16", "f32"])
def lib(request):
    if not os.path.exists(B.lib_path(request.param)):
        B.build_all()
    return R.Library(request.param)


def rules(T: int, n: int, r: int) -> bool:
    """The one-linear ops' shape rules as the header states them."""
    return T >= 0 and 64 <= n <= 65536 and n % 64 == 0 and 4 <= r <= min(n, 256) and r % 4 == 0


widths = st.integers(-64, 70000) | st.sampled_from([64, 128, 4096, 65536, 65600, 8192 + 32])
ranks = st.integers(-4, 300) | st.sampled_from([4, 16, 32, 64, 256])


@SETTINGS
@given(T=st.integers(-3, 1 << 22), n=widths, r=ranks)
def test_workspace_query_follows_the_rules(lib, T, n, r):
    w = lib.workspace_bytes(T, n, r)
    assert (w > 0) == rules(T, n, r), (T, n, r, w)
    if w:
        assert w % 256 == 0
        assert lib.workspace_bytes(T + 4096, n, r) >= w


A = 0x10000000   # fake, 256-byte aligned device addresses far apart


@needs_no_gpu
@SETTINGS
@given(T=st.integers(-3, 4096), n=widths, r=ranks)
def test_ops_reject_out_of_rule_shapes(lib, T, n, r):
    ok = rules(T, n, r)
    if ok and T > 0:
        return  # a valid call would launch kernels; not a host-only case
    want = R.OK if ok else R.E_SHAPE
    c, ld, wsb = lib.cdll, max(n, 64), 1 << 40
    assert c.resbm_encode_fwd(T, n, r, 1, A, ld, 2 * A, ld, 3 * A, 4 * A, 5 * A, 6 * A, wsb, None) == want
    assert c.resbm_decode_fwd(T, n, r, 0, A, 2 * A, 3 * A, ld, 4 * A, wsb, None) == want
    assert c.resbm_decode_bwd(T, n, r, A, 2 * A, 3 * A, ld, 4 * A, ld, 5 * A, 6 * A, 0, 7 * A, wsb,
                              None) == want
    assert c.resbm_encode_bwd(T, n, r, 1, A, ld, 2 * A, 3 * A, 4 * A, 5 * A, ld, 0, 0, 6 * A, 0, 7 * A,
                              wsb, None) == want


@SETTINGS
@given(T=st.integers(-3, 1 << 20), n=st.integers(-8, 70000), m=st.integers(-8, 70000), r=st.integers(-8, 300))
def test_two_linear_workspace_query_follows_its_rules(lib, T, n, m, r):
    ok = (0 < T <= 1 << 31 and 8 <= n <= 65536 and n % 8 == 0 and 8 <= m <= 65536 and m % 8 == 0
          and 8 <= r <= n and r % 8 == 0)
    w = lib.two_workspace_bytes(T, n, m, r)
    assert (w > 0) == ok, (T, n, m, r, w)


@SETTINGS
@given(p=st.integers(-2, (1 << 20) + 8), q=st.integers(-2, 300))
def test_matrix_workspace_query_follows_its_rules(lib, p, q):
    for a, b in ((p, q), (q, p)):
        s, L = min(a, b), max(a, b)
        w = lib.matrix_workspace_bytes(a, b)
        assert (w > 0) == (1 <= s <= 256 and L <= 1 << 20), (a, b, w)
