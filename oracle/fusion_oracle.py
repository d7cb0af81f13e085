"""Plain float64 CPU oracle of the encoder fused into the FFN output projection.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the test suite, the smoke
check and the benchmark's CPU-baseline leg may import or call this module.  It
shares no code with the HIP path; a NumPy matmul is its only library primitive.

Sec. 3.2 places the encoder directly after the feed-forward layer: its input z
is the output of the FFN's down projection, z = h W_down.  Fusing changes where
the encoder's contraction runs, not what it computes: z is still produced (and
stored, in bf16, for the backward step), and the encoder reads that stored z,
    (b, a) = encode_fwd(x_attn, rne_bf16(z), W_e)
exactly as the unfused pair (projection, then the encoder op) would.
"""
from __future__ import annotations

import numpy as np

from .resbm_oracle import encode_fwd, rne_bf16


def ffn_encode_fwd(h: np.ndarray, W_down: np.ndarray, x_attn: np.ndarray, W_e: np.ndarray, act: int):
    """Returns (z, b, a): z = h W_down unrounded, and the encoder on rne_bf16(z)."""
    z = h @ W_down
    b, a = encode_fwd(x_attn, rne_bf16(z), W_e, act)
    return z, b, a
