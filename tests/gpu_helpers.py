"""Shared helpers of the GPU parity tests (not collected by pytest itself)."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

from paper_2604_11947_amd import inputs as I

BF16_BOUND = 2e-2   # max err <= 2e-2 RMS(ref) for bf16 I/O (ulp-discounted for bf16 outputs)
F32_BOUND = 1e-5    # max |err| <= 1e-5 RMS(ref) for the fp32 validation build


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


def lib(variant: str = "bf16"):
    """The built library; with a GPU present a missing build is an error, never a skip."""
    require_gpu()
    from paper_2604_11947_amd import resbm as R
    return R.library(variant)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu").to(torch.float64).numpy()


def half_ulp_bf16(ref: np.ndarray) -> np.ndarray:
    """Half the spacing of bf16 values around |ref| (2^(floor(log2|x|) - 8), subnormal floor 2^-134)."""
    a = np.abs(ref)
    _, E = np.frexp(a)
    e = np.maximum(E - 1, -126)
    h = np.ldexp(1.0, e - 8)
    h[a == 0] = 2.0 ** -134
    return h


def errors(gpu: np.ndarray, ref: np.ndarray, bf16_output: bool, allow=None) -> dict:
    """Raw and discounted max error, relative to RMS(ref).  The discount is half
    a bf16 ulp of ref for bf16 outputs, plus the elementwise allowance `allow`
    (the rounding of a bf16 intermediate the op is specified to take)."""
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    rms = float(np.sqrt(np.mean(ref ** 2))) if ref.size else 0.0
    d = np.abs(gpu - ref)
    raw = float(d.max()) if d.size else 0.0
    slack = (half_ulp_bf16(ref) if bf16_output else 0.0) + (0.0 if allow is None else allow)
    disc = float(np.maximum(0.0, d - slack).max()) if (d.size and (bf16_output or allow is not None)) else raw
    scale = rms if rms > 0 else 1.0
    return {"rms": rms, "raw": raw / scale, "disc": disc / scale, "finite": bool(np.all(np.isfinite(gpu)))}


def check(name: str, gpu, ref: np.ndarray, bf16_output: bool, bound: float = BF16_BOUND,
          scale: float | None = None, allow=None) -> dict:
    """Assert max error <= bound x RMS(ref) (x ``scale`` instead of RMS(ref) when given)."""
    g = f64(gpu) if isinstance(gpu, torch.Tensor) else gpu
    e = errors(g, ref, bf16_output, allow)
    if scale is not None and e["rms"] > 0:
        k = e["rms"] / scale
        e["raw"] *= k
        e["disc"] *= k
    say(f"    {name:10s} rms={e['rms']:.3e} raw={e['raw']:.2e} disc={e['disc']:.2e}"
        + (f" (vs abs-sum rms {scale:.3e})" if scale is not None else ""))
    assert e["finite"], f"{name}: non-finite values"
    assert e["disc"] <= bound, f"{name}: max err {e['disc']:.3e} RMS > {bound}"
    return e


def to_dev(d: dict, dev="cuda") -> dict:
    return {k: (v.to(dev) if isinstance(v, torch.Tensor) else v) for k, v in d.items()}


def strided(t: torch.Tensor, pad: int) -> torch.Tensor:
    """A copy of t whose rows sit in a wider buffer (leading dimension n + pad)."""
    if pad == 0:
        return t.clone()
    T, n = t.shape
    buf = torch.full((T, n + pad), float("nan"), dtype=t.dtype, device=t.device)
    buf[:, :n] = t
    return buf[:, :n]


SENTINEL = {torch.bfloat16: 0x7FC1, torch.float32: 0x7FC00001}


def guarded(shape, dtype, dev, guard: int = 4096, pad: int = 0):
    """An output view surrounded by sentinel NaN guard bands (and row padding).

    Returns (view, buffer, check) where check() asserts the guards and padding are
    untouched and the view holds no sentinel (every element was written)."""
    rows, cols = shape
    ld = cols + pad
    total = guard + rows * ld + guard
    ity = torch.int16 if dtype == torch.bfloat16 else torch.int32
    s = SENTINEL[dtype]
    if dtype == torch.bfloat16:
        s = s - 0x10000 if s >= 0x8000 else s
    bits = torch.full((total,), s, dtype=ity, device=dev)
    buf = bits.view(dtype)
    view = buf[guard:guard + rows * ld].view(rows, ld)[:, :cols] if rows else buf[guard:guard].view(0, cols)

    def check_guards():
        b = bits.cpu()
        assert bool((b[:guard] == s).all()), "leading guard band overwritten"
        assert bool((b[guard + rows * ld:] == s).all()), "trailing guard band overwritten"
        body = b[guard:guard + rows * ld].view(rows, ld) if rows else b[guard:guard].view(0, ld)
        if pad:
            assert bool((body[:, cols:] == s).all()), "row padding overwritten"
        assert not bool((body[:, :cols] == s).any()), "some outputs were not written"

    return view, buf, check_guards
