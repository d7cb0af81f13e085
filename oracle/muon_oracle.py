"""Plain float64 CPU oracle of the optimizer-side steps on the bottleneck weights.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the test suite, the smoke
check and the benchmark's CPU-baseline leg may import or call this module.  It
shares no code with the HIP path; NumPy matmuls and NumPy's SVD are its only
library primitives, and nothing here is blocked, fused or reordered beyond the
definitions below.

What the paper states:

* Sec. 3.4 -- the bottleneck (subspace projection) weights are trained end to
  end with Muon, which updates a weight matrix with its gradient momentum
  orthogonalised by a Newton-Schulz iteration; Sec. 4.1 -- every bottleneck
  model uses Muon.
* App. B.1 -- the effective rank of a bottleneck projection is
  r_eff = sum_i sigma_i^2 / max_i sigma_i^2 over its singular values: 1 when
  one singular value dominates, the short side when all are equal.

The paper prints neither the iteration nor its constants; these readings
follow the Muon method it cites (each is listed in the design notes):

* M1 momentum: M <- mu M + G; the matrix orthogonalised is M, or G + mu M
  with Nesterov momentum.
* M2 Newton-Schulz: X_0 = U / (||U||_F + eps), then `steps` times
  A = X X^T, X <- a X + (b A + c A^2) X, with X taken in its wide orientation
  (rows <= columns; a tall U is transposed in and out).  Defaults: the quintic
  (a, b, c) = (3.4445, -4.7750, 2.0315), 5 steps, eps = 1e-7.  With
  (1.5, -0.5, 0) the same loop is the cubic iteration whose limit is the
  orthogonal polar factor U V^T of U = U S V^T.
* M3 update: W <- W - lr (scale O + weight_decay W), O the orthogonalised
  matrix; scale defaults to 0.2 sqrt(max(p, q)) (update RMS matched to AdamW).
* M4 storage: W, G and M are float32; the arithmetic is float64 and every
  stored float32 is rounded once, to nearest even.
* M5 r_eff of the zero matrix is 0 (no energy in any direction).
"""
from __future__ import annotations

import numpy as np

NS_QUINTIC = (3.4445, -4.7750, 2.0315)
NS_CUBIC = (1.5, -0.5, 0.0)
NS_EPS = 1e-7


def to_f32(x: np.ndarray) -> np.ndarray:
    """M4: round float64 values to float32 (nearest even), returned as float64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def newton_schulz(U: np.ndarray, steps: int = 5, coeffs=NS_QUINTIC, eps: float = NS_EPS) -> np.ndarray:
    """M2: the Newton-Schulz orthogonalisation of a p x q matrix (Sec. 3.4)."""
    a, b, c = coeffs
    U = np.asarray(U, dtype=np.float64)
    tall = U.shape[0] > U.shape[1]
    X = U.T if tall else U
    X = X / (np.sqrt(np.sum(X * X)) + eps)
    for _ in range(steps):
        A = X @ X.T
        B = b * A + c * (A @ A)
        X = a * X + B @ X
    return X.T if tall else X


def default_scale(p: int, q: int) -> float:
    """M3: 0.2 sqrt(max(p, q))."""
    return 0.2 * float(np.sqrt(max(p, q)))


def muon_update(W, G, M, lr, momentum, weight_decay=0.0, scale=None, nesterov=False, steps=5,
                coeffs=NS_QUINTIC, eps: float = NS_EPS):
    """M1-M4: one Muon step of a float32 p x q weight.  Returns (W_new, M_new, O).

    W, G, M hold float32 values (as any float array); W_new and M_new are those
    of the float32 results, O the float64 orthogonalised matrix.
    """
    W = np.asarray(W, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    M = np.asarray(M, dtype=np.float64)
    if scale is None:
        scale = default_scale(*W.shape)
    M_new = to_f32(momentum * M + G)
    U = G + momentum * M_new if nesterov else M_new
    O = newton_schulz(U, steps, coeffs, eps)
    W_new = to_f32(W - lr * (scale * O + weight_decay * W))
    return W_new, M_new, O


def spectrum(W: np.ndarray):
    """App. B.1: singular values (descending) and r_eff = sum sigma^2 / max sigma^2."""
    W = np.asarray(W, dtype=np.float64)
    sigma = np.linalg.svd(W, compute_uv=False)
    top = sigma[0] ** 2 if sigma.size else 0.0
    r_eff = float(np.sum(sigma ** 2) / top) if top > 0 else 0.0
    return sigma, r_eff
