"""Plain float64 CPU oracle of the boundary fused into its neighbouring layers:
the encoder into the FFN output projection, the decoder into the next block's
normalisation and QKV projection.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the test suite, the smoke
check and the benchmark's CPU-baseline leg may import or call this module.  It
shares no code with the HIP path; a NumPy matmul is its only library primitive.

Sec. 3.2 places the encoder directly after the feed-forward layer: its input z
is the output of the FFN's down projection, z = h W_down.  Fusing changes where
the encoder's contraction runs, not what it computes: z is still produced (and
stored, in bf16, for the backward step), and the encoder reads that stored z,
    (b, a) = encode_fwd(x_attn, rne_bf16(z), W_e)
exactly as the unfused pair (projection, then the encoder op) would.

Sec. 3.2 places the decoder at the start of stage l + 1, and under the main
reading (decoder identity path added by the caller) the decoder output z~ is
the input of that stage's first block, whose attention starts with an RMS
normalisation and the QKV projection.  Fused there, the decoder computes
    out = RMSNorm(z~) W_qkv,  z~ = b W_d,
    RMSNorm(x)[t][c] = x[t][c] / sqrt(mean_c' x[t][c']^2 + eps) * gamma[c],
the normalisation of the Llama-style block the paper trains (Sec. 4.1).
"""
from __future__ import annotations

import numpy as np

from .resbm_oracle import decode_fwd, encode_fwd, rne_bf16


def ffn_encode_fwd(h: np.ndarray, W_down: np.ndarray, x_attn: np.ndarray, W_e: np.ndarray, act: int):
    """Returns (z, b, a): z = h W_down unrounded, and the encoder on rne_bf16(z)."""
    z = h @ W_down
    b, a = encode_fwd(x_attn, rne_bf16(z), W_e, act)
    return z, b, a


def rms_norm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """Row-wise RMS normalisation with gain gamma."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gamma, dtype=np.float64)[None, :]


def decode_qkv_fwd(b: np.ndarray, W_d: np.ndarray, gamma: np.ndarray, W_qkv: np.ndarray, eps: float):
    """Returns (z~, y, out): the decoder output (reading B), its normalisation and
    the QKV projection, all unrounded."""
    zt = decode_fwd(b, W_d, False)
    y = rms_norm(zt, gamma, eps)
    return zt, y, y @ np.asarray(W_qkv, dtype=np.float64)
