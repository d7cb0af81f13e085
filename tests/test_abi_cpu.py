"""Host-side checks of the C ABI: exports, workspace sizing, validation.

Every call here is rejected by host validation before any HIP call (or is a
pure host query), so these run without a GPU.  They use fake device addresses
and are therefore skipped where a GPU is visible.
"""
import ctypes
import os
import re
import subprocess

import pytest
import torch

from paper_2604_11947_amd import build as B
from paper_2604_11947_amd import resbm as R

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "resbm.h")


@pytest.fixture(scope="module", params=["bf16", "f32"])
def lib(request):
    if not os.path.exists(B.lib_path(request.param)):
        B.build_all()
    return R.Library(request.param)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(resbm2?_\w+)\s*\(", text)))


def test_header_declares_the_ops_and_helpers():
    names = declared_functions()
    for op in ("resbm_encode_fwd", "resbm_decode_fwd", "resbm_decode_bwd", "resbm_encode_bwd",
               "resbm_newton_schulz", "resbm_muon_update", "resbm_spectrum", "resbm_matrix_workspace_bytes",
               "resbm_workspace_bytes", "resbm_io_dtype", "resbm_strerror", "resbm2_encode_fwd", "resbm2_decode_fwd",
               "resbm2_decode_bwd", "resbm2_encode_bwd", "resbm2_workspace_bytes", "resbm_ffn_encode_fwd",
               "resbm_ffn_encode_workspace_bytes", "resbm_decode_qkv_fwd", "resbm_decode_qkv_workspace_bytes"):
        assert op in names
    assert sorted(n for n, _, _ in R.SIGNATURES) == names


def test_every_declared_symbol_is_exported(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", lib.path], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (resbm2?_\w+)$", out, flags=re.M))
    for name in declared_functions():
        assert name in exported, name
        assert getattr(lib.cdll, name)


def test_io_dtype(lib):
    want = R.IO_BF16 if lib.path.endswith("libresbm.so") else R.IO_F32
    assert lib.io_code == want


def test_strerror(lib):
    for st in (0, -1, -2, -3, -4, -5, -6, -7):
        assert lib.strerror(st) and lib.strerror(st) != "unknown status"
    assert lib.strerror(-99) == "unknown status"


def test_workspace_bytes(lib):
    assert lib.workspace_bytes(1024, 100, 32) == 0          # n % 64
    assert lib.workspace_bytes(1024, 512, 6) == 0           # r % 4
    assert lib.workspace_bytes(1024, 512, 260) == 0         # r > 256
    assert lib.workspace_bytes(1024, 64, 128) == 0          # r > n
    assert lib.workspace_bytes(-1, 512, 32) == 0
    prev = 0
    for T in (1, 31, 32, 1000, 16384, 65536, 1 << 20):
        w = lib.workspace_bytes(T, 4096, 32)
        assert w % 256 == 0 and w >= prev
        prev = w
    # headline shape: bounded by a modest fraction of its 4 x 128 MiB streams
    assert lib.workspace_bytes(16384, 4096, 32) <= 64 << 20


def test_library_missing_raises(monkeypatch, tmp_path):
    monkeypatch.setattr(B, "lib_path", lambda variant="bf16": str(tmp_path / "nope.so"))
    with pytest.raises(R.LibraryNotBuilt):
        R.Library("bf16")


def test_product_never_imports_the_oracle():
    pkg = os.path.join(ROOT, "paper_2604_11947_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".hpp", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(import|from)\s+oracle\b", text, flags=re.M), f
                assert "resbm_oracle" not in text, f


# ---------------------------------------------------------------- validation
needs_no_gpu = pytest.mark.skipif(torch.cuda.is_available(),
                                  reason="fake device addresses; host validation is covered on CPU hosts")

A = 0x10000000   # fake, 256-byte aligned addresses far apart
T, N, RR = 64, 256, 32


def enc_fwd_args(**over):
    names = ["T", "n", "r", "act", "x", "ldx", "z", "ldz", "We", "b", "a", "ws", "wsb", "s"]
    vals = [T, N, RR, 1, A, N, 2 * A, N, 3 * A, 4 * A, 5 * A, 6 * A, 1 << 30, None]
    for k, v in over.items():
        vals[names.index(k)] = v
    return vals


@needs_no_gpu
@pytest.mark.parametrize("over,status", [
    (dict(T=-1), R.E_SHAPE), (dict(n=100), R.E_SHAPE), (dict(n=0), R.E_SHAPE), (dict(r=0), R.E_SHAPE),
    (dict(r=6), R.E_SHAPE), (dict(r=260), R.E_SHAPE), (dict(n=64, r=128, ldx=64, ldz=64), R.E_SHAPE),
    (dict(act=2), R.E_ACT), (dict(x=None), R.E_NULL), (dict(z=None), R.E_NULL), (dict(We=None), R.E_NULL),
    (dict(b=None), R.E_NULL), (dict(ws=None), R.E_NULL), (dict(ldx=N - 8), R.E_SHAPE),
    (dict(ldz=N + 4), R.E_SHAPE), (dict(x=A + 8), R.E_ALIGN), (dict(z=2 * A + 2), R.E_ALIGN),
    (dict(a=5 * A + 4), R.E_ALIGN), (dict(ws=6 * A + 128), R.E_ALIGN), (dict(wsb=1024), R.E_WORKSPACE),
    (dict(b=2 * A + 64), R.E_ALIAS), (dict(a=A), R.E_ALIAS), (dict(ws=2 * A), R.E_ALIAS),
])
def test_encode_fwd_validation(lib, over, status):
    assert lib.cdll.resbm_encode_fwd(*enc_fwd_args(**over)) == status


@needs_no_gpu
def test_zero_tokens_needs_no_pointers(lib):
    c = lib.cdll
    assert c.resbm_encode_fwd(0, N, RR, 1, None, 0, None, 0, None, None, None, None, 0, None) == R.OK
    assert c.resbm_decode_fwd(0, N, RR, 0, None, None, None, 0, None, 0, None) == R.OK
    assert c.resbm_decode_bwd(0, N, RR, None, None, None, 0, None, 0, None, None, 0, None, 0, None) == R.OK
    assert c.resbm_encode_bwd(0, N, RR, 1, None, 0, None, None, None, None, 0, None, 0, None, 0, None, 0,
                              None) == R.OK
    # shape rules still apply at T = 0
    assert c.resbm_decode_fwd(0, 100, RR, 0, None, None, None, 0, None, 0, None) == R.E_SHAPE


@needs_no_gpu
def test_decode_fwd_validation(lib):
    c = lib.cdll
    ok = [T, N, RR, 0, A, 2 * A, 3 * A, N, None, 0, None]

    def call(i, v):
        a = list(ok)
        a[i] = v
        return c.resbm_decode_fwd(*a)

    assert call(4, None) == R.E_NULL
    assert call(5, None) == R.E_NULL
    assert call(6, None) == R.E_NULL
    assert call(7, N - 8) == R.E_SHAPE
    assert call(4, A + 2) == R.E_ALIGN
    assert call(6, A) == R.E_ALIAS          # z_tilde over b
    assert call(1, 96) == R.E_SHAPE


@needs_no_gpu
def test_decode_bwd_validation(lib):
    c = lib.cdll
    ws = lib.workspace_bytes(T, N, RR)
    ok = [T, N, RR, A, 2 * A, 3 * A, N, 4 * A, N, 5 * A, 6 * A, 0, 7 * A, ws, None]

    def call(i, v):
        a = list(ok)
        a[i] = v
        return c.resbm_decode_bwd(*a)

    assert call(3, None) == R.E_NULL
    assert call(5, None) == R.E_NULL
    assert call(9, None) == R.E_NULL
    assert call(10, None) == R.E_NULL
    assert call(12, None) == R.E_NULL
    assert call(13, 256) == R.E_WORKSPACE
    assert call(8, N - 8) == R.E_SHAPE       # g_id leading dimension
    assert call(7, 4 * A + 8) == R.E_ALIGN
    assert call(9, 3 * A) == R.E_ALIAS       # g_b over g_zt
    assert call(10, 2 * A) == R.E_ALIAS      # dW_d over W_d
    assert call(12, 3 * A + 256) == R.E_ALIAS


@needs_no_gpu
def test_encode_bwd_validation(lib):
    c = lib.cdll
    ws = lib.workspace_bytes(T, N, RR)
    ok = [T, N, RR, 1, A, N, 2 * A, 3 * A, 4 * A, 5 * A, N, 6 * A, N, 7 * A, 0, 8 * A, ws, None]

    def call(**kw):
        names = ["T", "n", "r", "act", "z", "ldz", "We", "a", "gb", "gz", "ldgz", "gx", "ldgx", "dWe", "acc",
                 "ws", "wsb", "s"]
        a = list(ok)
        for k, v in kw.items():
            a[names.index(k)] = v
        return c.resbm_encode_bwd(*a)

    assert call(a=None) == R.E_ACT            # SiLU needs a_save
    assert call(act=5) == R.E_ACT
    assert call(z=None) == R.E_NULL
    assert call(gz=None) == R.E_NULL
    assert call(dWe=None) == R.E_NULL
    assert call(gx=5 * A, ldgx=N + 8) == R.E_ALIAS   # fused g_x needs the same ld
    assert call(gz=A) == R.E_ALIAS
    assert call(gx=A) == R.E_ALIAS
    assert call(ldgx=N - 8) == R.E_SHAPE
    assert call(wsb=256) == R.E_WORKSPACE
    assert call(gb=4 * A + 4) == R.E_ALIGN


@needs_no_gpu
def test_descriptor_window_limit(lib):
    """A block's rows of a streamed matrix are addressed through one buffer
    descriptor with 32-bit byte offsets: a row stride so large that the rows one
    block (or one token group of the expand kernel) covers exceed that range is
    rejected, never wrapped."""
    c = lib.cdll
    n, r, t = 64, 4, 64
    big = 1 << 27            # 16 rows of 2^27 elements: 4 GiB of bf16, 8 GiB of fp32
    ws = lib.workspace_bytes(t, n, r)
    assert c.resbm_decode_fwd(t, n, r, 0, A, 2 * A, 3 * A, big, None, 0, None) == R.E_SHAPE
    assert c.resbm_encode_fwd(t, n, r, 1, A, n, 2 * A, big, 3 * A, 4 * A, 5 * A, 6 * A, ws, None) == R.E_SHAPE
    assert c.resbm_decode_bwd(t, n, r, A, 2 * A, 3 * A, big, None, 0, 5 * A, 6 * A, 0, 7 * A, ws,
                              None) == R.E_SHAPE
    assert c.resbm_encode_bwd(t, n, r, 1, A, big, 2 * A, 3 * A, 4 * A, 5 * A, n, None, 0, 7 * A, 0, 8 * A, ws,
                              None) == R.E_SHAPE
    assert c.resbm_encode_bwd(t, n, r, 1, A, n, 2 * A, 3 * A, 4 * A, 5 * A, big, None, 0, 7 * A, 0, 8 * A, ws,
                              None) == R.E_SHAPE
    # wide rank: the row contraction's token group (128 rows at r = 256) is the
    # window; 2^24-element rows fit 16 or 32 rows in range but not 128
    n, r, t, ld = 256, 256, 256, 1 << 24
    ws = lib.workspace_bytes(t, n, r)
    assert c.resbm_encode_fwd(t, n, r, 1, A, n, 2 * A, ld, 3 * A, 4 * A, 5 * A, 6 * A, ws, None) == R.E_SHAPE
    assert c.resbm_decode_bwd(t, n, r, A, 2 * A, 3 * A, ld, None, 0, 5 * A, 6 * A, 0, 7 * A, ws,
                              None) == R.E_SHAPE


@needs_no_gpu
def test_encode_bwd_noalloc_validation(lib):
    """The allocation-free encode_bwd validates like encode_bwd and rejects a call
    whose scratch would exceed the fixed array, all before any HIP call."""
    c = lib.cdll
    ok = [T, N, RR, 1, A, N, 2 * A, 3 * A, 4 * A, 5 * A, N, 6 * A, N, 7 * A, 0, None]

    def call(**kw):
        names = ["T", "n", "r", "act", "z", "ldz", "We", "a", "gb", "gz", "ldgz", "gx", "ldgx", "dWe", "acc", "s"]
        a = list(ok)
        for k, v in kw.items():
            a[names.index(k)] = v
        return c.resbm_encode_bwd_noalloc(*a)

    assert call(T=0, z=None, We=None, a=None, gb=None, gz=None, gx=None, dWe=None) == R.OK
    assert call(a=None) == R.E_ACT
    assert call(z=None) == R.E_NULL
    assert call(n=100) == R.E_SHAPE
    assert call(gz=A) == R.E_ALIAS
    assert call(gb=4 * A + 4) == R.E_ALIGN
    assert call(T=16384, n=65536, r=256, ldz=65536, ldgz=65536, gx=None) == R.E_WORKSPACE


# ---------------------------------------------------------------- optimizer-side ops
def test_matrix_workspace_bytes(lib):
    assert lib.matrix_workspace_bytes(0, 32) == 0
    assert lib.matrix_workspace_bytes(4096, 257) == 0        # short side > 256
    assert lib.matrix_workspace_bytes(257, 4096) == 0
    assert lib.matrix_workspace_bytes((1 << 20) + 1, 8) == 0  # long side > 2^20
    for p, q in ((4096, 32), (32, 4096), (8192, 64), (4096, 256), (1, 1), (7, 3)):
        w = lib.matrix_workspace_bytes(p, q)
        assert w % 256 == 0 and w >= max(p, q) * ((min(p, q) + 3) // 4 * 4) * 8
    assert lib.matrix_workspace_bytes(4096, 32) == lib.matrix_workspace_bytes(32, 4096)


@needs_no_gpu
def test_newton_schulz_validation(lib):
    c = lib.cdll
    p, q = 512, 32
    ws = lib.matrix_workspace_bytes(p, q)
    ok = [p, q, A, 2 * A, 5, 3.4445, -4.775, 2.0315, 3 * A, ws, None]

    def call(i, v):
        a = list(ok)
        a[i] = v
        return c.resbm_newton_schulz(*a)

    assert call(0, 0) == R.E_SHAPE
    assert call(1, 300) == R.E_SHAPE
    assert call(4, -1) == R.E_SHAPE
    assert call(4, 101) == R.E_SHAPE
    assert call(2, None) == R.E_NULL
    assert call(3, None) == R.E_NULL
    assert call(8, None) == R.E_NULL
    assert call(9, ws - 256) == R.E_WORKSPACE
    assert call(8, 3 * A + 64) == R.E_ALIGN
    assert call(2, A + 2) == R.E_ALIGN
    assert call(3, A + 4096) == R.E_ALIAS      # O over G
    assert call(8, 2 * A) == R.E_ALIAS         # ws over O


@needs_no_gpu
def test_muon_update_validation(lib):
    c = lib.cdll
    p, q = 32, 4096
    ws = lib.matrix_workspace_bytes(p, q)
    ok = [p, q, A, 2 * A, 3 * A, 0.02, 0.95, 0.0, 1.0, 0, 5, 3.4445, -4.775, 2.0315, 4 * A, ws, None]

    def call(i, v):
        a = list(ok)
        a[i] = v
        return c.resbm_muon_update(*a)

    assert call(1, 0) == R.E_SHAPE
    assert call(2, None) == R.E_NULL           # W
    assert call(3, None) == R.E_NULL           # G
    assert call(15, 0) == R.E_WORKSPACE
    assert call(4, 3 * A + 1) == R.E_ALIGN     # M
    assert call(4, 2 * A + 512) == R.E_ALIAS   # M over G
    assert call(3, A) == R.E_ALIAS             # G over W
    assert call(14, 3 * A) == R.E_ALIAS        # ws over M


@needs_no_gpu
def test_spectrum_validation(lib):
    c = lib.cdll
    p, q = 64, 4096
    ws = lib.matrix_workspace_bytes(p, q)
    ok = [p, q, A, 2 * A, 3 * A, 4 * A, ws, None]

    def call(i, v):
        a = list(ok)
        a[i] = v
        return c.resbm_spectrum(*a)

    assert call(0, 257) == R.E_SHAPE           # short side > 256
    assert call(0, 0) == R.E_SHAPE
    assert call(2, None) == R.E_NULL
    assert call(3, None) == R.E_NULL
    assert call(4, None) == R.E_NULL
    assert call(3, 2 * A + 4) == R.E_ALIGN
    assert call(4, 2 * A + 8) == R.E_ALIAS     # r_eff inside sigma
    assert call(6, 1024) == R.E_WORKSPACE


# ---------------------------------------------------------------- two-linears-per-side ops
M2 = 128


def test_two_workspace_bytes(lib):
    c = lib.cdll
    assert c.resbm2_workspace_bytes(0, N, M2, RR) == 0
    assert c.resbm2_workspace_bytes(T, N, M2, 12) == 0          # r % 8
    assert c.resbm2_workspace_bytes(T, N, 100, RR) == 0         # m % 8
    assert c.resbm2_workspace_bytes(T, 64, M2, 72) == 0         # r > n
    w = c.resbm2_workspace_bytes(T, N, M2, RR)
    assert w >= T * M2 * 2 and w % 256 == 0


@needs_no_gpu
def test_two_encode_fwd_validation(lib):
    c = lib.cdll
    ws = c.resbm2_workspace_bytes(T, N, M2, RR)
    ok = [T, N, M2, RR, 1, A, N, 2 * A, N, 3 * A, 4 * A, 5 * A, 6 * A, 7 * A, ws, None]

    def call(i, v):
        a = list(ok)
        a[i] = v
        return c.resbm2_encode_fwd(*a)

    assert call(4, 7) == R.E_ACT
    assert call(3, 12) == R.E_SHAPE
    assert call(2, 4) == R.E_SHAPE
    assert call(6, N - 8) == R.E_SHAPE
    assert call(0, 0) == R.OK                 # T = 0: nothing read
    for i in (5, 7, 9, 10, 11, 12, 13):       # with SiLU phi(u) needs the workspace
        assert call(i, None) == R.E_NULL, i
    assert call(14, T * M2 * 2 - 256) == R.E_WORKSPACE
    assert call(11, 5 * A + 8) == R.E_ALIGN
    assert call(13, 7 * A + 128) == R.E_ALIGN
    assert call(11, 2 * A) == R.E_ALIAS       # b over z
    assert call(12, 3 * A) == R.E_ALIAS       # u over W1
    assert call(13, 6 * A) == R.E_ALIAS       # ws over u


@needs_no_gpu
def test_two_decode_bwd_validation(lib):
    c = lib.cdll
    ws = c.resbm2_workspace_bytes(T, N, M2, RR)
    ok = [T, N, M2, RR, 1, A, 2 * A, 3 * A, N, 4 * A, N, 5 * A, 6 * A, 7 * A, 8 * A, 9 * A, 10 * A, ws, None]

    def call(i, v):
        a = list(ok)
        a[i] = v
        return c.resbm2_decode_bwd(*a)

    assert call(16, None) == R.E_NULL
    assert call(17, ws - 256) == R.E_WORKSPACE
    assert call(16, 10 * A + 64) == R.E_ALIGN
    assert call(10, N - 8) == R.E_SHAPE
    assert call(13, 3 * A) == R.E_ALIAS       # g_b over g_zt
    assert call(15, 8 * A) == R.E_ALIAS       # dW4 over dW3... distinct outputs may not overlap
    assert call(16, 2 * A) == R.E_ALIAS       # workspace over v


@needs_no_gpu
def test_two_encode_bwd_validation(lib):
    c = lib.cdll
    ws = c.resbm2_workspace_bytes(T, N, M2, RR)
    ok = [T, N, M2, RR, 1, A, N, 2 * A, 3 * A, 4 * A, 5 * A, 6 * A, N, 7 * A, N, 8 * A, 9 * A, 10 * A, ws, None]

    def call(i, v):
        a = list(ok)
        a[i] = v
        return c.resbm2_encode_bwd(*a)

    assert call(4, 2) == R.E_ACT
    assert call(17, None) == R.E_NULL
    assert call(18, 0) == R.E_WORKSPACE
    assert call(12, N + 4) == R.E_SHAPE
    fused = list(ok)
    fused[13], fused[14] = 6 * A, N + 8
    assert c.resbm2_encode_bwd(*fused) == R.E_ALIAS   # g_x == g_z needs equal leading dimensions
    assert call(11, A) == R.E_ALIAS           # g_z over z
    assert call(15, 9 * A) == R.E_ALIAS       # dW1 over dW2


@needs_no_gpu
def test_ffn_encode_validation(lib):
    c = lib.cdll
    DFF = 512
    ws = c.resbm_ffn_encode_workspace_bytes(T, N, RR)
    assert ws >= T * RR * 4 and ws % 256 == 0
    assert c.resbm_ffn_encode_workspace_bytes(T, N, 12) == 0
    ok = [T, DFF, N, RR, 1, A, DFF, 2 * A, 3 * A, N, 4 * A, 5 * A, N, 6 * A, 7 * A, 8 * A, ws, None]

    def call(i, v):
        a = list(ok)
        a[i] = v
        return c.resbm_ffn_encode_fwd(*a)

    assert call(4, 3) == R.E_ACT
    assert call(1, 100) == R.E_SHAPE          # d_ff % 8
    assert call(3, 2 * N) == R.E_SHAPE        # r > n
    assert call(0, 0) == R.OK
    assert call(6, DFF - 8) == R.E_SHAPE      # ld_h < d_ff
    for i in (5, 7, 8, 10, 11, 13):
        assert call(i, None) == R.E_NULL, i
    assert call(16, ws - 256) == R.E_WORKSPACE
    assert call(13, 6 * A + 8) == R.E_ALIGN
    assert call(11, 2 * A) == R.E_ALIAS       # z over W_down
    assert call(13, A) == R.E_ALIAS           # b over h


def test_decode_qkv_validation(lib):
    """Host-side checks of the decoder fused into RMSNorm + QKV (no GPU needed:
    every rejected call returns before any HIP call)."""
    import ctypes
    c = lib.cdll
    n, r, NQ, TT = 256, 32, 384, 300
    ws = c.resbm_decode_qkv_workspace_bytes(n, r)
    assert ws >= (n // 16) * 2048 and ws % 256 == 0
    assert c.resbm_decode_qkv_workspace_bytes(n, 12) == 0      # r % 8
    assert c.resbm_decode_qkv_workspace_bytes(n, 72) == 0      # r > 64
    assert c.resbm_decode_qkv_workspace_bytes(200, r) == 0     # n % 64
    ok = [TT, n, r, NQ, A, 2 * A, 3 * A, 4 * A, ctypes.c_float(1e-5), 5 * A, NQ, 6 * A, ws, None]

    def call(i, v):
        a = list(ok)
        a[i] = v
        return c.resbm_decode_qkv_fwd(*a)

    assert call(0, 0) == R.OK
    assert call(1, 200) == R.E_SHAPE        # n % 64
    assert call(2, 12) == R.E_SHAPE         # r % 8
    assert call(2, 128) == R.E_SHAPE        # r > 64
    assert call(3, 100) == R.E_SHAPE        # N % 8
    assert call(8, ctypes.c_float(-1.0)) == R.E_SHAPE
    assert call(8, ctypes.c_float(float("nan"))) == R.E_SHAPE
    assert call(10, NQ - 8) == R.E_SHAPE    # ld_out < N
    for i in (4, 5, 6, 7, 9):
        assert call(i, None) == R.E_NULL, i
    assert call(11, None) == R.E_NULL
    assert call(12, ws - 256) == R.E_WORKSPACE
    assert call(11, 6 * A + 64) == R.E_ALIGN
    assert call(9, 5 * A + 8) == R.E_ALIGN
    assert call(9, 4 * A) == R.E_ALIAS      # out over W_qkv
    assert call(11, A) == R.E_ALIAS         # workspace over b
