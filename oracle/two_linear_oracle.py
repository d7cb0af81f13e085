"""Plain float64 CPU oracle of the two-linears-per-side bottleneck (Sec. 3.2).

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the test suite, the smoke
check and the benchmark's CPU-baseline leg may import or call this module.  It
shares no code with the HIP path; NumPy matmuls are its only library
primitive, and nothing here is blocked, fused or reordered beyond the
definitions below.

Sec. 3.2 describes the encoder and the decoder each as two linear layers with
a non-linearity between them, the encoder mapping the feed-forward output down
to the bottleneck width and the decoder mapping it back.  With the readings of
the one-linear module (no biases; phi identity or SiLU; the encoder's skip is
the attention output through P^id_{n->r}, Eq. 2 and Eq. 5; decoder identity
reading B, added by the caller) and an intermediate width m:

    encoder   u = z W1                       (T x m;  W1 is n x m)
              b = x_attn P^id_{n->r} + phi(u) W2   (T x r;  W2 is m x r)
    decoder   v = b W3                       (T x m;  W3 is r x m)
              z~ = phi(v) W4                 (T x n;  W4 is m x n)

The backward steps are the exact adjoints (chain rule through both layers);
the forward's pre-activations u and v are the saved tensors the backward
steps take.  Inputs are float64 arrays (bf16 values widen exactly);
row-independent steps may be called on any subset of tokens, and the weight
gradients on any subset of output columns.
"""
from __future__ import annotations

import numpy as np

from .resbm_oracle import dphi, p_id, p_id_adjoint, phi


def encode2_fwd(x_attn: np.ndarray, z: np.ndarray, W1: np.ndarray, W2: np.ndarray, act: int):
    """Encoder E(z) = phi(z W1) W2 plus the skip.  Returns (b, u) with u = z W1."""
    r = W2.shape[1]
    u = z @ W1
    b = p_id(x_attn, r) + phi(u, act) @ W2
    return b, u


def decode2_fwd(b: np.ndarray, W3: np.ndarray, W4: np.ndarray, act: int):
    """Decoder D(b) = phi(b W3) W4.  Returns (z~, v) with v = b W3."""
    v = b @ W3
    return phi(v, act) @ W4, v


def decode2_bwd(b, v, g_zt, g_id, W3, W4, act: int):
    """Adjoint of decode2_fwd at (b, v = b W3).  Returns (g_b, dW3, dW4).

    p = phi(v);  dW4 = p^T g_z~;  g_p = g_z~ W4^T;  g_v = g_p * phi'(v);
    dW3 = b^T g_v;  g_b = g_v W3^T + g_id P^id_{n->r} (g_id None: no identity term).
    """
    r = W3.shape[0]
    p = phi(v, act)
    dW4 = p.T @ g_zt
    g_v = (g_zt @ W4.T) * dphi(v, act)
    dW3 = b.T @ g_v
    g_b = g_v @ W3.T
    if g_id is not None:
        g_b = g_b + p_id_adjoint(g_id, r)
    return g_b, dW3, dW4


def encode2_bwd(z, u, g_b, W1, W2, act: int):
    """Adjoint of the encoder branch at (z, u = z W1).  Returns (g_z, dW1, dW2).

    h = phi(u);  dW2 = h^T g_b;  g_u = (g_b W2^T) * phi'(u);
    dW1 = z^T g_u;  g_z = g_u W1^T.  The skip's gradient g_b P^id_{r->n} is
    added to the caller's residual gradient (resbm_oracle.skip_grad).
    """
    h = phi(u, act)
    dW2 = h.T @ g_b
    g_u = (g_b @ W2.T) * dphi(u, act)
    dW1 = z.T @ g_u
    g_z = g_u @ W1.T
    return g_z, dW1, dW2


def loss_and_grads(x_attn, z, W1, W2, W3, W4, g_zt, g_id, act: int):
    """Encoder then decoder on one batch, with the reading-B identity added
    after the decoder: y = z~ + P^id_{r->n}(b), L = <g_zt, z~> + <g_id, P^id(b)>.
    Returns the forward values and every gradient of L (used to check the
    adjoints against finite differences)."""
    n = W1.shape[0]
    b, u = encode2_fwd(x_attn, z, W1, W2, act)
    zt, v = decode2_fwd(b, W3, W4, act)
    L = float(np.sum(g_zt * zt) + np.sum(g_id * p_id(b, n)))
    g_b, dW3, dW4 = decode2_bwd(b, v, g_zt, g_id, W3, W4, act)
    g_z, dW1, dW2 = encode2_bwd(z, u, g_b, W1, W2, act)
    g_x = p_id(g_b, n)
    return L, {"z": g_z, "x_attn": g_x, "W1": dW1, "W2": dW2, "W3": dW3, "W4": dW4}
