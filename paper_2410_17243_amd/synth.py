"""Seeded synthetic CLIP-shaped embedding pairs.

This module only draws inputs; it holds none of the loss arithmetic, and both
the GPU path's callers (tests, benchmark) and the CPU checks use it.

Recipe (the paper trains on image/text features of LAION-400M, which are not
available; these synthetic pairs stand in for them):

  g, n ~ N(0, 1)^{b x d}  (float32, per 65,536-row chunk c drawn from
                           numpy.random.default_rng([seed, c]))
  img = g / ||g||
  txt = (g + sigma * n) / ||g + sigma * n||          mode "clip"
  txt = L2norm(img + sigma * n)                       mode "weak" (noise added to
                                                      the unit vector itself)

Normalisation is done in float32; the bf16 and f16 variants round the float32
values to bfloat16 or IEEE half with round-to-nearest-even.  The positive cosine is about
1/sqrt(1 + sigma^2) in mode "clip" and about 1/sqrt(1 + sigma^2 d) in "weak".
"""

from __future__ import annotations

import numpy as np

CHUNK_ROWS = 65536


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round-to-nearest-even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _l2norm_rows(a: np.ndarray) -> np.ndarray:
    nrm = np.sqrt(np.sum(a * a, axis=1, dtype=np.float32), dtype=np.float32)
    return a / nrm[:, None]


def clip_pairs(b: int, d: int, sigma: float, seed: int = 0, dtype: str = "bf16", mode: str = "clip"):
    """Return (img, txt) as numpy arrays of shape [b, d].

    dtype "bf16" returns uint16 bfloat16 bit patterns, "f16" uint16 IEEE half
    bit patterns; "f32" returns float32.
    """
    if dtype not in ("bf16", "f16", "f32"):
        raise ValueError(f"dtype must be 'bf16', 'f16' or 'f32', got {dtype!r}")
    if mode not in ("clip", "weak"):
        raise ValueError(f"mode must be 'clip' or 'weak', got {mode!r}")
    out_dt = np.float32 if dtype == "f32" else np.uint16
    img = np.empty((b, d), dtype=out_dt)
    txt = np.empty((b, d), dtype=out_dt)
    sig = np.float32(sigma)
    for c, r0 in enumerate(range(0, b, CHUNK_ROWS)):
        r1 = min(b, r0 + CHUNK_ROWS)
        rng = np.random.default_rng([seed, c])
        g = rng.standard_normal((r1 - r0, d), dtype=np.float32)
        n = rng.standard_normal((r1 - r0, d), dtype=np.float32)
        im = _l2norm_rows(g)
        if mode == "clip":
            tx = _l2norm_rows(g + sig * n)
        else:
            tx = _l2norm_rows(im + sig * n)
        if dtype == "bf16":
            img[r0:r1] = f32_to_bf16_bits(im)
            txt[r0:r1] = f32_to_bf16_bits(tx)
        elif dtype == "f16":
            img[r0:r1] = im.astype(np.float16).view(np.uint16)  # round to nearest even
            txt[r0:r1] = tx.astype(np.float16).view(np.uint16)
        else:
            img[r0:r1] = im
            txt[r0:r1] = tx
    return img, txt


def as_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 view of generator output (bf16 or f16 bits, or float32)."""
    if dtype == "bf16":
        return bf16_bits_to_f32(a).astype(np.float64)
    if dtype == "f16":
        return np.asarray(a, dtype=np.uint16).view(np.float16).astype(np.float64)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


# The five workloads: shapes, noise and scale of the benchmark configurations.
WORKLOADS = {
    1: dict(b=1024, d=512, dtype="f32", sigma=1.0, scale=1.0 / 0.07),
    2: dict(b=32768, d=512, dtype="bf16", sigma=1.0, scale=14.29),
    3: dict(b=131072, d=768, dtype="bf16", sigma=0.5, scale=100.0),
    4: dict(b=1048576, d=1024, dtype="bf16", sigma=1.0, scale=50.0),
    5: dict(b=4194304, d=768, dtype="bf16", sigma=1.0, scale=14.29),
}
