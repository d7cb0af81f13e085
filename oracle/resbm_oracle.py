"""Plain float64 CPU oracle of the ResBM residual bottleneck boundary module.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the test suite, the smoke
check and the benchmark's CPU-baseline leg may import or call this module.  It
shares no code with the HIP path: it is written from the paper's definitions
(Sec. 3.1-3.3) with NumPy matmuls as the only library primitive, and nothing
here is blocked, fused or reordered beyond what those definitions state.

What the module computes (paper notation: x^Attn, z_l, b_l, E_l, D_l, P^id):

* Sec. 3.1, Eq. 2 -- generalised residual update  x_{l+1} = x_l P^id_l + F(x_l, W_l).
* Sec. 3.3, Eq. 4 -- rectangular identity  [I_{c x C}]_{ij} = 1 if i = j else 0.
* Sec. 3.3, Eq. 5 -- identity projection  P^id(x) = x I_{c x C}: zero-pads when
  c < C, drops the last c - C columns when c > C, identity when c = C.
* Sec. 3.2 -- encoder after the feed-forward layer, b_l = E_l(z_l) in R^{L x h};
  its skip is the attention output x^Attn projected by P^id_l; decoder
  z~_l = D_l(b_l) in R^{L x H} on the far side of the pipeline boundary.
* App. A.3 -- b_l crosses the boundary as bf16, T*r*2 bytes per direction.

Readings taken where the paper is open (each is listed in the design notes):

* The encoder branch is one n->r linear map followed by the non-linearity phi,
  the decoder one r->n linear map; no biases.  phi is identity or SiLU, applied
  inside the encoder branch before the skip sum:
      b = P^id_{n->r}(x_attn) + phi(z W_e).
* Decoder identity: reading B (default) returns z~ = b W_d and the caller adds
  P^id_{r->n}(b) after its attention branch, sending back that path's gradient
  g_id; reading A (add_identity) returns z~ = b W_d + P^id_{r->n}(b) and the
  caller passes g_id = g_z~.
* The backward formulas are the exact adjoints of the forward maps (the paper
  trains end-to-end but prints no gradient); the adjoint of P^id_{c->C} is
  P^id_{C->c}.
* Wire rounding (chain mode) is float -> bf16 round-to-nearest-even with
  NaN/Inf preserved and no flush-to-zero.

Inputs are float64 arrays (bf16/fp32 values widen exactly).  Row-independent
steps may be called on any subset of tokens; the weight-gradient steps may be
called on any subset of hidden channels.
"""
from __future__ import annotations

import numpy as np

ACT_IDENTITY = 0
ACT_SILU = 1


# --------------------------------------------------------------------------
# Sec. 3.3: the identity path
# --------------------------------------------------------------------------
def rect_identity(c: int, C: int) -> np.ndarray:
    """Eq. 4: the c x C matrix with ones where the row equals the column."""
    m = np.zeros((c, C))
    for i in range(min(c, C)):
        m[i, i] = 1.0
    return m


def p_id(x: np.ndarray, C: int) -> np.ndarray:
    """Eq. 5 with its three cases: x in R^{L x c} mapped to R^{L x C}.

    c < C appends C - c zero columns, c > C truncates the last c - C columns,
    c = C returns x unchanged (as a copy).
    """
    L, c = x.shape
    if c >= C:
        return np.array(x[:, :C], dtype=np.float64, copy=True)
    out = np.zeros((L, C))
    out[:, :c] = x
    return out


def p_id_adjoint(g: np.ndarray, c: int) -> np.ndarray:
    """Adjoint of P^id_{c->C} applied to a gradient g in R^{L x C}: g I_{c x C}^T = g I_{C x c}."""
    return p_id(g, c)


# --------------------------------------------------------------------------
# Non-linearity inside the encoder branch (Sec. 3.2; unnamed there)
# --------------------------------------------------------------------------
def phi(a: np.ndarray, act: int) -> np.ndarray:
    if act == ACT_IDENTITY:
        return np.array(a, dtype=np.float64, copy=True)
    if act == ACT_SILU:
        return a / (1.0 + np.exp(-a))
    raise ValueError(f"unknown activation {act}")


def dphi(a: np.ndarray, act: int) -> np.ndarray:
    """d phi / d a."""
    if act == ACT_IDENTITY:
        return np.ones_like(a, dtype=np.float64)
    if act == ACT_SILU:
        s = 1.0 / (1.0 + np.exp(-a))
        return s * (1.0 + a * (1.0 - s))
    raise ValueError(f"unknown activation {act}")


# --------------------------------------------------------------------------
# Forward (Sec. 3.2 with Eq. 2 and Eq. 5)
# --------------------------------------------------------------------------
def encode_fwd(x_attn: np.ndarray, z: np.ndarray, W_e: np.ndarray, act: int):
    """Encoder side of the boundary at the end of stage l.

    a = z W_e (the encoder's linear map), then Eq. 2 with P^id_l from n to r:
    b = x_attn P^id_{n->r} + phi(a).  Returns (b, a).
    """
    r = W_e.shape[1]
    a = z @ W_e
    b = p_id(x_attn, r) + phi(a, act)
    return b, a


def decode_fwd(b: np.ndarray, W_d: np.ndarray, add_identity: bool) -> np.ndarray:
    """Decoder D_{l+1} at the start of stage l+1: z~ = b W_d (+ P^id_{r->n}(b), reading A)."""
    n = W_d.shape[1]
    zt = b @ W_d
    if add_identity:
        zt = zt + p_id(b, n)
    return zt


# --------------------------------------------------------------------------
# Backward: adjoints of the forward maps
# --------------------------------------------------------------------------
def decode_input_grad(g_zt: np.ndarray, W_d: np.ndarray, g_id) -> np.ndarray:
    """g_b = g_z~ W_d^T + g_id P^id_{n->r}  (g_id is None: no identity gradient)."""
    r = W_d.shape[0]
    g_b = g_zt @ W_d.T
    if g_id is not None:
        g_b = g_b + p_id_adjoint(g_id, r)
    return g_b


def decode_weight_grad(b: np.ndarray, g_zt: np.ndarray) -> np.ndarray:
    """dL/dW_d = b^T g_z~ (sum over tokens)."""
    return b.T @ g_zt


def decode_bwd(b, W_d, g_zt, g_id):
    """Returns (g_b, dW_d)."""
    return decode_input_grad(g_zt, W_d, g_id), decode_weight_grad(b, g_zt)


def encode_local_grad(g_b: np.ndarray, a: np.ndarray, act: int) -> np.ndarray:
    """g_h = g_b * phi'(a): gradient at the encoder's linear output."""
    return g_b * dphi(a, act)


def encode_input_grad(g_h: np.ndarray, W_e: np.ndarray) -> np.ndarray:
    """dL/dz = g_h W_e^T."""
    return g_h @ W_e.T


def encode_weight_grad(z: np.ndarray, g_h: np.ndarray) -> np.ndarray:
    """dL/dW_e = z^T g_h (sum over tokens)."""
    return z.T @ g_h


def encode_bwd(z, W_e, a, g_b, act):
    """Returns (g_z, dW_e)."""
    g_h = encode_local_grad(g_b, a, act)
    return encode_input_grad(g_h, W_e), encode_weight_grad(z, g_h)


def skip_grad(g_x: np.ndarray, g_b: np.ndarray) -> np.ndarray:
    """Residual gradient through the encoder-side identity path:
    g_x + g_b P^id_{r->n}, i.e. columns [0, r) gain g_b, the rest are unchanged."""
    return g_x + p_id(g_b, g_x.shape[1])


# --------------------------------------------------------------------------
# Wire format (App. A.3): bf16, row-major [T][r], no header
# --------------------------------------------------------------------------
def rne_bf16(x) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (ties to even).

    bfloat16: 8 exponent bits (bias 127), 7 stored fraction bits, subnormals
    down to 2^-133, overflow to +-inf, NaN and Inf unchanged, no flush-to-zero.
    Returns the rounded values as float64.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.array(x, copy=True)
    fin = np.isfinite(x)
    ax = np.abs(x[fin])
    _, E = np.frexp(ax)                        # ax = m 2^E, 0.5 <= m < 1
    quantum_exp = np.maximum(E - 1, -126) - 7  # spacing of bf16 values near ax
    q = np.ldexp(1.0, quantum_exp)
    y = np.round(ax / q) * q                   # exact scaling; np.round is half-to-even
    y[y >= 2.0 ** 128] = np.inf
    out[fin] = np.copysign(y, x[fin])
    return out


def bf16_bits(x) -> np.ndarray:
    """uint16 bit patterns of values that are exactly representable in bf16."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    return (f.view(np.uint32) >> 16).astype(np.uint16)


def wire_payload(b) -> bytes:
    """The bytes that cross the boundary: RNE bf16, little-endian, [T][r] packed."""
    return bf16_bits(rne_bf16(b)).astype("<u2").tobytes()


# --------------------------------------------------------------------------
# One boundary, forward and backward, with the wire rounded as on the link
# --------------------------------------------------------------------------
def boundary_fwd_bwd(x_attn, z, W_e, W_d, g_zt, g_id, act: int,
                     add_identity: bool, wire_round: bool = True) -> dict:
    """encode -> wire -> decode -> decode backward -> wire -> encode backward.

    With ``wire_round`` the payload b and the wire gradient g_b are rounded to
    bf16 where they cross the boundary, as on the link; every other quantity
    stays float64.  Reading A passes g_id = g_zt and add_identity = True.
    """
    b, a = encode_fwd(x_attn, z, W_e, act)
    b_w = rne_bf16(b) if wire_round else b
    zt = decode_fwd(b_w, W_d, add_identity)
    g_b, dW_d = decode_bwd(b_w, W_d, g_zt, g_id)
    g_bw = rne_bf16(g_b) if wire_round else g_b
    g_z, dW_e = encode_bwd(z, W_e, a, g_bw, act)
    return {"a": a, "b": b, "b_wire": b_w, "z_tilde": zt, "g_b": g_b,
            "g_b_wire": g_bw, "dW_d": dW_d, "g_z": g_z, "dW_e": dW_e}
