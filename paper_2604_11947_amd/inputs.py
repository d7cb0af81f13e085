"""Seeded synthetic inputs for the ResBM boundary module.

This module only draws random numbers and stores them; it holds none of the
module's arithmetic.  Both the HIP path (tests, bench) and the CPU oracle
tests take their inputs from here and from nowhere else.

Shapes follow the boundary module of Sec. 3.2: token-major activations
``[T][n]`` (T = batch x sequence), an encoder weight ``W_e[n][r]`` and a
decoder weight ``W_d[r][n]`` (right-multiplied, as in Eq. 2 and Eq. 5).
The paper trains on C4 text through a Llama-3 style model (Sec. 4.1); no
data or checkpoint is available here, so every workload stands in for those
activations with a seeded distribution of the same shape.

Draw order (NumPy PCG64, ``SeedSequence(seed).spawn(7)``):
``x_attn, z, W_e, W_d, g_zt, g_id, structure``.  Activations and upstream
gradients are drawn in float64 and stored as bfloat16 (torch's conversion);
weights are drawn in float64 and stored as float32 masters.  Variance
conventions: ``N(0, v)`` means variance v.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import torch

# Rows drawn per chunk when filling large activation tensors (keeps the float64
# staging buffer near 256 MiB at n = 8192).
_CHUNK_ROWS = 4096


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic boundary workload.

    ``dist`` names the activation distribution:
      * ``normal``      i.i.d. N(0, 1)
      * ``outliers``    N(0, 1) with floor(0.01 n) channels scaled by 20; the same
                        channel indices in x_attn and z
      * ``student_t3``  Student-t with 3 degrees of freedom, each tensor divided by
                        its own empirical RMS
      * ``token_lognormal`` N(0, 1) times a per-token factor exp(N(0, 0.5^2)); the
                        same factor for x_attn and z (they describe the same token)
    Upstream gradients are N(0, 1e-2) for every workload.
    """

    name: str
    n: int
    r: int
    batch: int
    seq: int
    dist: str = "normal"
    seed: int = 0

    @property
    def tokens(self) -> int:
        return self.batch * self.seq


def _sweep(r: int) -> Workload:
    return Workload(f"sweep_n4096_r{r}", 4096, r, 4, 4096, "normal")


# Shapes mirror the paper's hidden widths (4096 in Table 1, 2048 in the
# boundary schematic of App. C) at the 128x compression of Sec. 4.1.
WORKLOADS: dict[str, Workload] = {
    w.name: w
    for w in [
        Workload("tiny_n512_r4", 512, 4, 2, 128, "normal"),
        Workload("n2048_r16_outliers", 2048, 16, 8, 1024, "outliers"),
        # the same boundary at the 16,384 tokens its description also states
        Workload("n2048_r16_outliers_t16k", 2048, 16, 8, 2048, "outliers"),
        Workload("n4096_r32_t3", 4096, 32, 4, 4096, "student_t3"),
        Workload("n8192_r64_lognormal", 8192, 64, 4, 8192, "token_lognormal"),
    ]
    + [_sweep(r) for r in (256, 128, 64, 32, 16)]
}

# The workload the throughput figure is quoted on.
HEADLINE = "n4096_r32_t3"

GRAD_STD = 0.1  # N(0, 1e-2)


def _to_bf16(x: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x)).to(torch.bfloat16)


def _activation(rng: np.random.Generator, T: int, n: int, dist: str,
                struct: dict) -> torch.Tensor:
    out = torch.empty((T, n), dtype=torch.bfloat16)
    if dist == "student_t3":
        x = rng.standard_t(3, size=(T, n))
        rms = np.sqrt(np.mean(np.square(x))) if x.size else 1.0
        x /= rms
        out.copy_(_to_bf16(x))
        return out
    for r0 in range(0, T, _CHUNK_ROWS):
        r1 = min(T, r0 + _CHUNK_ROWS)
        x = rng.standard_normal((r1 - r0, n))
        if dist == "outliers":
            x[:, struct["channels"]] *= 20.0
        elif dist == "token_lognormal":
            x *= struct["token_scale"][r0:r1, None]
        elif dist != "normal":
            raise ValueError(f"unknown distribution {dist!r}")
        out[r0:r1].copy_(_to_bf16(x))
    return out


def _grad(rng: np.random.Generator, T: int, n: int) -> torch.Tensor:
    out = torch.empty((T, n), dtype=torch.bfloat16)
    for r0 in range(0, T, _CHUNK_ROWS):
        r1 = min(T, r0 + _CHUNK_ROWS)
        out[r0:r1].copy_(_to_bf16(GRAD_STD * rng.standard_normal((r1 - r0, n))))
    return out


def _streams(seed: int) -> list[np.random.Generator]:
    ss = np.random.SeedSequence(seed).spawn(7)
    return [np.random.Generator(np.random.PCG64(s)) for s in ss]


def make_weights(n: int, r: int, seed: int = 0) -> dict[str, torch.Tensor]:
    """The weights make_inputs would draw for (n, r, seed): W_e ~ N(0, 1/n) fp32
    ``[n][r]`` and W_d ~ N(0, 1/r) fp32 ``[r][n]``."""
    rngs = _streams(seed)
    return {
        "W_e": torch.from_numpy((rngs[2].standard_normal((n, r)) / np.sqrt(n)).astype(np.float32)),
        "W_d": torch.from_numpy((rngs[3].standard_normal((r, n)) / np.sqrt(r)).astype(np.float32)),
    }


def make_activations(T: int, n: int, dist: str = "normal", seed: int = 0,
                     grads: bool = True) -> dict:
    """The activations and upstream gradients make_inputs would draw (they do
    not depend on r): ``x_attn, z, g_zt, g_id`` bf16 ``[T][n]`` plus ``meta``."""
    if T < 0 or n <= 0:
        raise ValueError("T must be >= 0 and n positive")
    rngs = _streams(seed)
    struct_rng = rngs[6]
    struct: dict = {}
    if dist == "outliers":
        k = int(np.floor(0.01 * n))
        struct["channels"] = np.sort(struct_rng.choice(n, size=k, replace=False))
    elif dist == "token_lognormal":
        struct["token_scale"] = np.exp(0.5 * struct_rng.standard_normal(T))
    out: dict = {
        "x_attn": _activation(rngs[0], T, n, dist, struct),
        "z": _activation(rngs[1], T, n, dist, struct),
    }
    if grads:
        out["g_zt"] = _grad(rngs[4], T, n)
        out["g_id"] = _grad(rngs[5], T, n)
    meta = {"dist": dist, "seed": seed}
    if "channels" in struct:
        meta["outlier_channels"] = struct["channels"].tolist()
    out["meta"] = meta
    return out


def make_inputs(T: int, n: int, r: int, dist: str = "normal", seed: int = 0,
                grads: bool = True) -> dict:
    """Draw one boundary's inputs on the host.

    Returns CPU tensors ``x_attn, z, g_zt, g_id`` (bf16, ``[T][n]``), ``W_e``
    (fp32 ``[n][r]``, N(0, 1/n)) and ``W_d`` (fp32 ``[r][n]``, N(0, 1/r)), plus
    ``meta`` describing structural draws (outlier channels).
    """
    if r <= 0:
        raise ValueError("r must be positive")
    out = make_activations(T, n, dist, seed, grads)
    out.update(make_weights(n, r, seed))
    if "outlier_channels" in out["meta"]:
        out["meta"]["outliers_in_skip"] = int(sum(c < r for c in out["meta"]["outlier_channels"]))
    return out


def workload_inputs(name: str, tokens: int | None = None, seed: int | None = None,
                    grads: bool = True) -> dict[str, torch.Tensor]:
    """Inputs of a named workload; ``tokens`` overrides T (a prefix-sized draw)."""
    w = WORKLOADS[name]
    T = w.tokens if tokens is None else tokens
    return make_inputs(T, w.n, w.r, w.dist, w.seed if seed is None else seed, grads)


def upstream_grad(T: int, n: int, seed: int) -> torch.Tensor:
    """An extra N(0, 1e-2) bf16 gradient tensor from its own seed."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    return _grad(rng, T, n)


def bf16_to_f64(t: torch.Tensor) -> np.ndarray:
    """Exact widening of a bf16/fp32 CPU tensor to a float64 NumPy array."""
    return t.to(torch.float64).numpy()


# ---------------------------------------------------------------- bottleneck-weight matrices
MATRIX_KINDS = ("gaussian", "powerlaw", "orthonormal", "rank1", "zero", "clustered", "graded")


def make_matrix(p: int, q: int, kind: str = "gaussian", seed: int = 0, scale: float = 1.0) -> torch.Tensor:
    """A seeded float32 p x q matrix for the optimizer-side ops.

    gaussian     N(0, scale^2) entries (a gradient or momentum draw);
    powerlaw     U diag(sigma) V^T with random orthonormal U, V and
                 sigma_i = scale (i + 1)^-1.5 (i < min(p, q)): a decaying
                 spectrum down to ~1e-3 of the top at s = 128;
    orthonormal  scale times orthonormal columns (rows if p < q): all singular
                 values equal;
    rank1        scale u v^T with Gaussian u, v;
    zero         all zeros;
    clustered    U diag(sigma) V^T with two tight clusters: sigma_i = scale
                 (1 + 1e-6 i) for the first half, half that for the rest;
    graded       U diag(sigma) V^T with sigma_i = scale 10^(-6 i / (s - 1)): six
                 decades from the top to the smallest.
    """
    if p <= 0 or q <= 0:
        raise ValueError("p and q must be positive")
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, p, q, MATRIX_KINDS.index(kind)])))
    s, L = min(p, q), max(p, q)

    def orth(rows, cols):
        qm, rm = np.linalg.qr(rng.standard_normal((rows, cols)))
        return qm * np.sign(np.diag(rm))

    if kind == "gaussian":
        m = scale * rng.standard_normal((p, q))
    elif kind == "powerlaw":
        sig = scale * (np.arange(s) + 1.0) ** -1.5
        tall = orth(L, s) @ np.diag(sig) @ orth(s, s).T
        m = tall if p >= q else tall.T
    elif kind == "orthonormal":
        tall = scale * orth(L, s)
        m = tall if p >= q else tall.T
    elif kind == "rank1":
        m = scale * np.outer(rng.standard_normal(p), rng.standard_normal(q))
    elif kind == "zero":
        m = np.zeros((p, q))
    elif kind in ("clustered", "graded"):
        i = np.arange(s, dtype=float)
        if kind == "clustered":
            sig = scale * (1.0 + 1e-6 * i) * np.where(i < s // 2, 1.0, 0.5)
        else:
            sig = scale * 10.0 ** (-6.0 * i / max(s - 1, 1))
        tall = orth(L, s) @ np.diag(sig) @ orth(s, s).T
        m = tall if p >= q else tall.T
    else:
        raise ValueError(f"unknown matrix kind {kind!r}")
    return torch.from_numpy(np.ascontiguousarray(m).astype(np.float32))


# ---------------------------------------------------------------- two-linears-per-side variant
def make_two_weights(n: int, m: int, r: int, seed: int = 0) -> dict[str, torch.Tensor]:
    """bf16 weights of the two-linears-per-side bottleneck: W1 [n][m] ~ N(0, 1/n),
    W2 [m][r] ~ N(0, 1/m), W3 [r][m] ~ N(0, 1/r), W4 [m][n] ~ N(0, 1/m)."""
    ss = np.random.SeedSequence([seed, n, m, r, 2]).spawn(4)
    g = [np.random.Generator(np.random.PCG64(s)) for s in ss]
    return {
        "W1": _to_bf16(g[0].standard_normal((n, m)) / np.sqrt(n)),
        "W2": _to_bf16(g[1].standard_normal((m, r)) / np.sqrt(m)),
        "W3": _to_bf16(g[2].standard_normal((r, m)) / np.sqrt(r)),
        "W4": _to_bf16(g[3].standard_normal((m, n)) / np.sqrt(m)),
    }


def make_gain(n: int, seed: int) -> torch.Tensor:
    """A normalisation gain: n float32 values 1 + 0.1 N(0, 1) from their own seed."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, n, 5])))
    return torch.from_numpy((1.0 + 0.1 * rng.standard_normal(n)).astype(np.float32))


def make_bf16(rows: int, cols: int, seed: int, std: float = 1.0) -> torch.Tensor:
    """rows x cols bf16 N(0, std^2) from its own seed (payloads, saved
    pre-activations, wire gradients of the two-linears-per-side ops)."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, rows, cols, 3])))
    out = torch.empty((rows, cols), dtype=torch.bfloat16)
    for r0 in range(0, rows, _CHUNK_ROWS):
        r1 = min(rows, r0 + _CHUNK_ROWS)
        out[r0:r1].copy_(_to_bf16(std * rng.standard_normal((r1 - r0, cols))))
    return out
