"""ctypes binding of ``libresbm`` -- the C ABI declared in ``include/resbm.h``.

Argument marshalling only: torch tensors supply device pointers, row strides
and the current HIP stream; every step of the module runs in the library's
kernels.  A missing library raises ``LibraryNotBuilt``; nothing falls back to
another implementation.
"""
from __future__ import annotations

import ctypes
import os

import torch

from . import build as _build

ACT_IDENTITY = 0
ACT_SILU = 1
IO_BF16 = 0
IO_F32 = 1

OK = 0
E_NULL = -1
E_SHAPE = -2
E_ALIGN = -3
E_WORKSPACE = -4
E_ACT = -5
E_HIP = -6
E_ALIAS = -7

# Newton-Schulz coefficients of the Muon method the paper cites (Sec. 3.4)
NS_QUINTIC = (3.4445, -4.7750, 2.0315)
NS_CUBIC = (1.5, -0.5, 0.0)

# (name, restype, argtypes) of every exported symbol
_i64, _i32, _p, _sz, _d = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_double
SIGNATURES = [
    ("resbm_encode_fwd", _i32, [_i64, _i32, _i32, _i32, _p, _i64, _p, _i64, _p, _p, _p, _p, _sz, _p]),
    ("resbm_decode_fwd", _i32, [_i64, _i32, _i32, _i32, _p, _p, _p, _i64, _p, _sz, _p]),
    ("resbm_decode_bwd", _i32, [_i64, _i32, _i32, _p, _p, _p, _i64, _p, _i64, _p, _p, _i32, _p, _sz, _p]),
    ("resbm_encode_bwd", _i32, [_i64, _i32, _i32, _i32, _p, _i64, _p, _p, _p, _p, _i64, _p, _i64, _p, _i32,
                                _p, _sz, _p]),
    ("resbm_encode_bwd_noalloc", _i32, [_i64, _i32, _i32, _i32, _p, _i64, _p, _p, _p, _p, _i64, _p, _i64, _p,
                                        _i32, _p]),
    ("resbm_newton_schulz", _i32, [_i32, _i32, _p, _p, _i32, _d, _d, _d, _p, _sz, _p]),
    ("resbm_muon_update", _i32, [_i32, _i32, _p, _p, _p, _d, _d, _d, _d, _i32, _i32, _d, _d, _d, _p, _sz, _p]),
    ("resbm_spectrum", _i32, [_i32, _i32, _p, _p, _p, _p, _sz, _p]),
    ("resbm_matrix_workspace_bytes", _sz, [_i32, _i32]),
    ("resbm_workspace_bytes", _sz, [_i64, _i32, _i32]),
    ("resbm2_encode_fwd", _i32, [_i64, _i32, _i32, _i32, _i32, _p, _i64, _p, _i64, _p, _p, _p, _p, _p, _sz, _p]),
    ("resbm2_decode_fwd", _i32, [_i64, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _i64, _p, _p, _sz, _p]),
    ("resbm2_decode_bwd", _i32, [_i64, _i32, _i32, _i32, _i32, _p, _p, _p, _i64, _p, _i64, _p, _p, _p, _p, _p,
                                 _p, _sz, _p]),
    ("resbm2_encode_bwd", _i32, [_i64, _i32, _i32, _i32, _i32, _p, _i64, _p, _p, _p, _p, _p, _i64, _p, _i64,
                                 _p, _p, _p, _sz, _p]),
    ("resbm2_workspace_bytes", _sz, [_i64, _i32, _i32, _i32]),
    ("resbm_ffn_encode_fwd", _i32, [_i64, _i32, _i32, _i32, _i32, _p, _i64, _p, _p, _i64, _p, _p, _i64, _p, _p, _p,
                                    _sz, _p]),
    ("resbm_ffn_encode_workspace_bytes", _sz, [_i64, _i32, _i32]),
    ("resbm_decode_qkv_fwd", _i32, [_i64, _i32, _i32, _i32, _p, _p, _p, _p, ctypes.c_float, _p, _i64, _p, _sz, _p]),
    ("resbm_decode_qkv_workspace_bytes", _sz, [_i32, _i32]),
    ("resbm_io_dtype", _i32, []),
    ("resbm_strerror", ctypes.c_char_p, [_i32]),
]


class LibraryNotBuilt(RuntimeError):
    pass


class ResbmError(RuntimeError):
    def __init__(self, op: str, status: int, message: str):
        super().__init__(f"{op}: status {status}: {message}")
        self.status = status


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _ld(t: torch.Tensor, rows: int, cols: int, name: str) -> int:
    if t.dim() != 2 or t.shape[0] != rows or t.shape[1] != cols:
        raise ValueError(f"{name}: expected shape ({rows}, {cols}), got {tuple(t.shape)}")
    if rows > 1 and cols > 0 and t.stride(1) != 1:
        raise ValueError(f"{name}: rows must be contiguous")
    return t.stride(0) if rows > 1 else max(t.stride(0), cols)


def _packed(t: torch.Tensor, rows: int, cols: int, name: str) -> None:
    if t.dim() != 2 or t.shape[0] != rows or t.shape[1] != cols or not t.is_contiguous():
        raise ValueError(f"{name}: expected a contiguous ({rows}, {cols}) tensor, got {tuple(t.shape)}")


def _dtype(t, dtype, name):
    if t is not None and t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")


def _stream(stream, ref: torch.Tensor):
    if stream is None:
        stream = torch.cuda.current_stream(ref.device)
    return ctypes.c_void_p(getattr(stream, "cuda_stream", stream))


class Library:
    """One loaded variant of the library ("bf16" or "f32")."""

    def __init__(self, variant: str = "bf16"):
        path = _build.lib_path(variant)
        if not os.path.exists(path):
            raise LibraryNotBuilt(f"{path} is missing; run `python -m paper_2604_11947_amd.build`")
        self.path = path
        self.cdll = ctypes.CDLL(path)
        for name, res, args in SIGNATURES:
            fn = getattr(self.cdll, name)
            fn.restype = res
            fn.argtypes = args
        self.io_code = int(self.cdll.resbm_io_dtype())
        self.io_dtype = torch.bfloat16 if self.io_code == IO_BF16 else torch.float32

    # ------------------------------------------------------------ helpers
    def workspace_bytes(self, T: int, n: int, r: int) -> int:
        return int(self.cdll.resbm_workspace_bytes(T, n, r))

    def strerror(self, status: int) -> str:
        return self.cdll.resbm_strerror(status).decode()

    def workspace(self, T: int, n: int, r: int, device) -> torch.Tensor:
        nbytes = self.workspace_bytes(T, n, r)
        buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        off = (-buf.data_ptr()) % 256
        return buf[off:off + nbytes]

    def matrix_workspace_bytes(self, p: int, q: int) -> int:
        return int(self.cdll.resbm_matrix_workspace_bytes(p, q))

    def matrix_workspace(self, p: int, q: int, device) -> torch.Tensor:
        nbytes = self.matrix_workspace_bytes(p, q)
        buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        off = (-buf.data_ptr()) % 256
        return buf[off:off + nbytes]

    def _check(self, op: str, status: int) -> None:
        if status != OK:
            raise ResbmError(op, status, self.strerror(status))

    # ------------------------------------------------------------ ops
    def encode_fwd(self, x_attn, z, W_e, b, a_save=None, act=ACT_SILU, ws=None, stream=None):
        T = z.shape[0]
        n, r = W_e.shape
        io = self.io_dtype
        for t, nm in ((x_attn, "x_attn"), (z, "z"), (b, "b")):
            _dtype(t, io, nm)
        _dtype(W_e, torch.float32, "W_e")
        _dtype(a_save, torch.float32, "a_save")
        ld_x, ld_z = _ld(x_attn, T, n, "x_attn"), _ld(z, T, n, "z")
        _packed(b, T, r, "b")
        _packed(W_e, n, r, "W_e")
        if a_save is not None:
            _packed(a_save, T, r, "a_save")
        if ws is None:
            ws = self.workspace(T, n, r, z.device)
        st = self.cdll.resbm_encode_fwd(T, n, r, act, _ptr(x_attn), ld_x, _ptr(z), ld_z, _ptr(W_e), _ptr(b),
                                        _ptr(a_save), _ptr(ws), ws.numel(), _stream(stream, z))
        self._check("resbm_encode_fwd", st)

    def decode_fwd(self, b, W_d, z_tilde, add_identity=False, ws=None, stream=None):
        T = b.shape[0]
        r, n = W_d.shape
        _dtype(b, self.io_dtype, "b")
        _dtype(z_tilde, self.io_dtype, "z_tilde")
        _dtype(W_d, torch.float32, "W_d")
        _packed(b, T, r, "b")
        _packed(W_d, r, n, "W_d")
        ld = _ld(z_tilde, T, n, "z_tilde")
        nbytes = 0 if ws is None else ws.numel()
        st = self.cdll.resbm_decode_fwd(T, n, r, int(bool(add_identity)), _ptr(b), _ptr(W_d), _ptr(z_tilde), ld,
                                        _ptr(ws), nbytes, _stream(stream, b))
        self._check("resbm_decode_fwd", st)

    def decode_bwd(self, b, W_d, g_zt, g_id, g_b, dW_d, accumulate=False, ws=None, stream=None):
        T = b.shape[0]
        r, n = W_d.shape
        io = self.io_dtype
        for t, nm in ((b, "b"), (g_zt, "g_zt"), (g_id, "g_id"), (g_b, "g_b")):
            _dtype(t, io, nm)
        _dtype(W_d, torch.float32, "W_d")
        _dtype(dW_d, torch.float32, "dW_d")
        _packed(b, T, r, "b")
        _packed(g_b, T, r, "g_b")
        _packed(W_d, r, n, "W_d")
        _packed(dW_d, r, n, "dW_d")
        ld_g = _ld(g_zt, T, n, "g_zt")
        ld_i = _ld(g_id, T, n, "g_id") if g_id is not None else 0
        if ws is None:
            ws = self.workspace(T, n, r, g_zt.device)
        st = self.cdll.resbm_decode_bwd(T, n, r, _ptr(b), _ptr(W_d), _ptr(g_zt), ld_g, _ptr(g_id), ld_i, _ptr(g_b),
                                        _ptr(dW_d), int(bool(accumulate)), _ptr(ws), ws.numel(),
                                        _stream(stream, g_zt))
        self._check("resbm_decode_bwd", st)

    def encode_bwd(self, z, W_e, a_save, g_b, g_z, dW_e, g_x=None, act=ACT_SILU, accumulate=False, ws=None,
                   stream=None):
        T = z.shape[0]
        n, r = W_e.shape
        io = self.io_dtype
        for t, nm in ((z, "z"), (g_b, "g_b"), (g_z, "g_z"), (g_x, "g_x")):
            _dtype(t, io, nm)
        _dtype(W_e, torch.float32, "W_e")
        _dtype(a_save, torch.float32, "a_save")
        _dtype(dW_e, torch.float32, "dW_e")
        ld_z = _ld(z, T, n, "z")
        ld_gz = _ld(g_z, T, n, "g_z")
        ld_gx = _ld(g_x, T, n, "g_x") if g_x is not None else 0
        _packed(W_e, n, r, "W_e")
        _packed(g_b, T, r, "g_b")
        _packed(dW_e, n, r, "dW_e")
        if a_save is not None:
            _packed(a_save, T, r, "a_save")
        if ws is None:
            ws = self.workspace(T, n, r, z.device)
        st = self.cdll.resbm_encode_bwd(T, n, r, act, _ptr(z), ld_z, _ptr(W_e), _ptr(a_save), _ptr(g_b), _ptr(g_z),
                                        ld_gz, _ptr(g_x), ld_gx, _ptr(dW_e), int(bool(accumulate)), _ptr(ws),
                                        ws.numel(), _stream(stream, z))
        self._check("resbm_encode_bwd", st)


    def encode_bwd_noalloc(self, z, W_e, a_save, g_b, g_z, dW_e, g_x=None, act=ACT_SILU, accumulate=False,
                           stream=None):
        """resbm_encode_bwd_noalloc: encode_bwd on the library's fixed device-resident
        scratch (no workspace argument, nothing allocated)."""
        T = z.shape[0]
        n, r = W_e.shape
        io = self.io_dtype
        for t, nm in ((z, "z"), (g_b, "g_b"), (g_z, "g_z"), (g_x, "g_x")):
            _dtype(t, io, nm)
        _dtype(W_e, torch.float32, "W_e")
        _dtype(a_save, torch.float32, "a_save")
        _dtype(dW_e, torch.float32, "dW_e")
        ld_z = _ld(z, T, n, "z")
        ld_gz = _ld(g_z, T, n, "g_z")
        ld_gx = _ld(g_x, T, n, "g_x") if g_x is not None else 0
        _packed(W_e, n, r, "W_e")
        _packed(g_b, T, r, "g_b")
        _packed(dW_e, n, r, "dW_e")
        if a_save is not None:
            _packed(a_save, T, r, "a_save")
        st = self.cdll.resbm_encode_bwd_noalloc(T, n, r, act, _ptr(z), ld_z, _ptr(W_e), _ptr(a_save), _ptr(g_b),
                                                _ptr(g_z), ld_gz, _ptr(g_x), ld_gx, _ptr(dW_e),
                                                int(bool(accumulate)), _stream(stream, z))
        self._check("resbm_encode_bwd_noalloc", st)

    # ------------------------------------------------------------ two-linears-per-side ops
    # Weights W1 (n x m), W2 (m x r), W3 (r x m), W4 (m x n) and every activation
    # are bf16; the weight gradients float32.
    def two_workspace_bytes(self, T: int, n: int, m: int, r: int) -> int:
        return int(self.cdll.resbm2_workspace_bytes(T, n, m, r))

    def two_workspace(self, T: int, n: int, m: int, r: int, device) -> torch.Tensor:
        nbytes = self.two_workspace_bytes(T, n, m, r)
        buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        off = (-buf.data_ptr()) % 256
        return buf[off:off + nbytes]

    @staticmethod
    def _two_weights(W1, W2, W3=None, W4=None):
        n, m = W1.shape
        r = W2.shape[1]
        for t, nm, shape in ((W1, "W1", (n, m)), (W2, "W2", (m, r)), (W3, "W3", (r, m)), (W4, "W4", (m, n))):
            if t is not None:
                _dtype(t, torch.bfloat16, nm)
                _packed(t, *shape, nm)
        return n, m, r

    def encode2_fwd(self, x_attn, z, W1, W2, b, u, act=ACT_SILU, ws=None, stream=None):
        T = z.shape[0]
        n, m, r = self._two_weights(W1, W2)
        for t, nm in ((x_attn, "x_attn"), (z, "z"), (b, "b"), (u, "u")):
            _dtype(t, torch.bfloat16, nm)
        ld_x, ld_z = _ld(x_attn, T, n, "x_attn"), _ld(z, T, n, "z")
        _packed(b, T, r, "b")
        _packed(u, T, m, "u")
        if ws is None and act != ACT_IDENTITY:
            ws = self.two_workspace(T, n, m, r, z.device)
        st = self.cdll.resbm2_encode_fwd(T, n, m, r, act, _ptr(x_attn), ld_x, _ptr(z), ld_z, _ptr(W1), _ptr(W2),
                                         _ptr(b), _ptr(u), _ptr(ws), 0 if ws is None else ws.numel(),
                                         _stream(stream, z))
        self._check("resbm2_encode_fwd", st)

    def decode2_fwd(self, b, W3, W4, z_tilde, v, act=ACT_SILU, ws=None, stream=None):
        T = b.shape[0]
        m, n = W4.shape
        r = W3.shape[0]
        for t, nm, shape in ((W3, "W3", (r, m)), (W4, "W4", (m, n))):
            _dtype(t, torch.bfloat16, nm)
            _packed(t, *shape, nm)
        for t, nm in ((b, "b"), (z_tilde, "z_tilde"), (v, "v")):
            _dtype(t, torch.bfloat16, nm)
        _packed(b, T, r, "b")
        _packed(v, T, m, "v")
        ld_zt = _ld(z_tilde, T, n, "z_tilde")
        if ws is None:
            ws = self.two_workspace(T, n, m, r, b.device)
        st = self.cdll.resbm2_decode_fwd(T, n, m, r, act, _ptr(b), _ptr(W3), _ptr(W4), _ptr(z_tilde), ld_zt, _ptr(v),
                                         _ptr(ws), ws.numel(), _stream(stream, b))
        self._check("resbm2_decode_fwd", st)

    def decode2_bwd(self, b, v, g_zt, g_id, W3, W4, g_b, dW3, dW4, act=ACT_SILU, ws=None, stream=None):
        T = b.shape[0]
        m, n = W4.shape
        r = W3.shape[0]
        for t, nm, shape in ((W3, "W3", (r, m)), (W4, "W4", (m, n))):
            _dtype(t, torch.bfloat16, nm)
            _packed(t, *shape, nm)
        for t, nm in ((b, "b"), (v, "v"), (g_zt, "g_zt"), (g_id, "g_id"), (g_b, "g_b")):
            _dtype(t, torch.bfloat16, nm)
        _dtype(dW3, torch.float32, "dW3")
        _dtype(dW4, torch.float32, "dW4")
        _packed(b, T, r, "b")
        _packed(v, T, m, "v")
        _packed(g_b, T, r, "g_b")
        _packed(dW3, r, m, "dW3")
        _packed(dW4, m, n, "dW4")
        ld_gzt = _ld(g_zt, T, n, "g_zt")
        ld_gid = _ld(g_id, T, n, "g_id") if g_id is not None else 0
        if ws is None:
            ws = self.two_workspace(T, n, m, r, b.device)
        st = self.cdll.resbm2_decode_bwd(T, n, m, r, act, _ptr(b), _ptr(v), _ptr(g_zt), ld_gzt, _ptr(g_id), ld_gid,
                                         _ptr(W3), _ptr(W4), _ptr(g_b), _ptr(dW3), _ptr(dW4), _ptr(ws), ws.numel(),
                                         _stream(stream, b))
        self._check("resbm2_decode_bwd", st)

    def encode2_bwd(self, z, u, g_b, W1, W2, g_z, dW1, dW2, g_x=None, act=ACT_SILU, ws=None, stream=None):
        T = z.shape[0]
        n, m, r = self._two_weights(W1, W2)
        for t, nm in ((z, "z"), (u, "u"), (g_b, "g_b"), (g_z, "g_z"), (g_x, "g_x")):
            _dtype(t, torch.bfloat16, nm)
        _dtype(dW1, torch.float32, "dW1")
        _dtype(dW2, torch.float32, "dW2")
        _packed(u, T, m, "u")
        _packed(g_b, T, r, "g_b")
        _packed(dW1, n, m, "dW1")
        _packed(dW2, m, r, "dW2")
        ld_z, ld_gz = _ld(z, T, n, "z"), _ld(g_z, T, n, "g_z")
        ld_gx = _ld(g_x, T, n, "g_x") if g_x is not None else 0
        if ws is None:
            ws = self.two_workspace(T, n, m, r, z.device)
        st = self.cdll.resbm2_encode_bwd(T, n, m, r, act, _ptr(z), ld_z, _ptr(u), _ptr(g_b), _ptr(W1), _ptr(W2),
                                         _ptr(g_z), ld_gz, _ptr(g_x), ld_gx, _ptr(dW1), _ptr(dW2), _ptr(ws),
                                         ws.numel(), _stream(stream, z))
        self._check("resbm2_encode_bwd", st)

    # ------------------------------------------------------------ encoder fused into the FFN output projection
    def ffn_encode_fwd(self, h, W_down, x_attn, W_e, z, b, a_save=None, act=ACT_SILU, ws=None, stream=None):
        T, d_ff = h.shape
        n, r = W_e.shape
        for t, nm in ((h, "h"), (W_down, "W_down"), (x_attn, "x_attn"), (z, "z"), (b, "b")):
            _dtype(t, torch.bfloat16, nm)
        _dtype(W_e, torch.float32, "W_e")
        _dtype(a_save, torch.float32, "a_save")
        _packed(W_down, d_ff, n, "W_down")
        _packed(W_e, n, r, "W_e")
        _packed(b, T, r, "b")
        if a_save is not None:
            _packed(a_save, T, r, "a_save")
        ld_h, ld_x, ld_z = _ld(h, T, d_ff, "h"), _ld(x_attn, T, n, "x_attn"), _ld(z, T, n, "z")
        if ws is None:
            nbytes = int(self.cdll.resbm_ffn_encode_workspace_bytes(T, n, r))
            buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=h.device)
            ws = buf[(-buf.data_ptr()) % 256:][:nbytes]
        st = self.cdll.resbm_ffn_encode_fwd(T, d_ff, n, r, act, _ptr(h), ld_h, _ptr(W_down), _ptr(x_attn), ld_x,
                                            _ptr(W_e), _ptr(z), ld_z, _ptr(b), _ptr(a_save), _ptr(ws), ws.numel(),
                                            _stream(stream, h))
        self._check("resbm_ffn_encode_fwd", st)

    def decode_qkv_fwd(self, b, W_d, gamma, W_qkv, out, eps=1e-5, ws=None, stream=None):
        T, r = b.shape
        n, N = W_qkv.shape
        for t, nm in ((b, "b"), (W_qkv, "W_qkv"), (out, "out")):
            _dtype(t, torch.bfloat16, nm)
        _dtype(W_d, torch.float32, "W_d")
        _dtype(gamma, torch.float32, "gamma")
        _packed(b, T, r, "b")
        _packed(W_d, r, n, "W_d")
        _packed(W_qkv, n, N, "W_qkv")
        if gamma.dim() != 1 or gamma.numel() != n or not gamma.is_contiguous():
            raise ValueError("gamma: expected a contiguous vector of n elements")
        ld_out = _ld(out, T, N, "out")
        if ws is None:
            nbytes = int(self.cdll.resbm_decode_qkv_workspace_bytes(n, r))
            buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=b.device)
            ws = buf[(-buf.data_ptr()) % 256:][:nbytes]
        st = self.cdll.resbm_decode_qkv_fwd(T, n, r, N, _ptr(b), _ptr(W_d), _ptr(gamma), _ptr(W_qkv), eps, _ptr(out),
                                            ld_out, _ptr(ws), ws.numel(), _stream(stream, b))
        self._check("resbm_decode_qkv_fwd", st)

    # ------------------------------------------------------------ optimizer-side ops
    def newton_schulz(self, G, O, steps=5, coeffs=NS_QUINTIC, ws=None, stream=None):
        p, q = G.shape
        _dtype(G, torch.float32, "G")
        _dtype(O, torch.float32, "O")
        _packed(G, p, q, "G")
        _packed(O, p, q, "O")
        if ws is None:
            ws = self.matrix_workspace(p, q, G.device)
        a, b, c = coeffs
        st = self.cdll.resbm_newton_schulz(p, q, _ptr(G), _ptr(O), steps, a, b, c, _ptr(ws), ws.numel(),
                                           _stream(stream, G))
        self._check("resbm_newton_schulz", st)

    def muon_update(self, W, G, M, lr, momentum=0.95, weight_decay=0.0, scale=None, nesterov=False, steps=5,
                    coeffs=NS_QUINTIC, ws=None, stream=None):
        p, q = W.shape
        for t, nm in ((W, "W"), (G, "G"), (M, "M")):
            _dtype(t, torch.float32, nm)
            if t is not None:
                _packed(t, p, q, nm)
        if scale is None:
            scale = -1.0  # the library's default (negative selects it)
        if ws is None:
            ws = self.matrix_workspace(p, q, W.device)
        a, b, c = coeffs
        st = self.cdll.resbm_muon_update(p, q, _ptr(W), _ptr(G), _ptr(M), lr, momentum, weight_decay, scale,
                                         int(bool(nesterov)), steps, a, b, c, _ptr(ws), ws.numel(),
                                         _stream(stream, W))
        self._check("resbm_muon_update", st)

    def spectrum(self, W, sigma, r_eff, ws=None, stream=None):
        p, q = W.shape
        _dtype(W, torch.float32, "W")
        _packed(W, p, q, "W")
        _dtype(sigma, torch.float64, "sigma")
        _dtype(r_eff, torch.float64, "r_eff")
        if sigma.numel() < min(p, q) or r_eff.numel() < 1 or not sigma.is_contiguous():
            raise ValueError("sigma needs min(p, q) contiguous float64 elements, r_eff one")
        if ws is None:
            ws = self.matrix_workspace(p, q, W.device)
        st = self.cdll.resbm_spectrum(p, q, _ptr(W), _ptr(sigma), _ptr(r_eff), _ptr(ws), ws.numel(),
                                      _stream(stream, W))
        self._check("resbm_spectrum", st)


_LOADED: dict[str, Library] = {}


def library(variant: str = "bf16") -> Library:
    """The loaded library variant ("bf16" = libresbm.so, "f32" = libresbm_f32.so)."""
    if variant not in _LOADED:
        _LOADED[variant] = Library(variant)
    return _LOADED[variant]
