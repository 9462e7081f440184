"""Rotary position re-encoding of cached keys after compaction (oracle, float64).

Test infrastructure: used only by tests, the smoke check and the CPU baseline.

Paper passage followed (section 5.2, Applying the retention plan): after a deletion a kept
token's logical position is lower by the deleted tokens before it, so its cached key, rotated
for the old position, is turned by that shift to read as rotated for the new one.

Readings where the paper is silent (its model's attention uses standard rotary embeddings):
  * A key stored after rotation at position p is moved to position p + shift by rotating each
    dimension pair (x, y) by shift * theta_j: (x cos - y sin, x sin + y cos), the same rotation
    that the position difference applies to an unrotated key.
  * Frequencies theta_j = base ** (-2 j / R) for the first R (rotary) dimensions of each head,
    j = 0 .. R/2 - 1; dimensions >= R are not rotated.
  * Pairing "half": dims (j, j + R/2) (the split-halves layout of common decoder
    implementations); "interleaved": dims (2j, 2j + 1) (the layout of the original RoPE paper).
  * Values are re-encoded exactly (float64); storage rounding is the caller's business.
"""
from __future__ import annotations

import numpy as np

STYLES = ("half", "interleaved")


def rope_thetas(base: float, rot_dims: int) -> np.ndarray:
    """theta_j = base^(-2j/R), j < R/2, float64."""
    if rot_dims < 2 or rot_dims % 2:
        raise ValueError("rotary dims must be a positive even number")
    j = np.arange(rot_dims // 2, dtype=np.float64)
    return float(base) ** (-2.0 * j / rot_dims)


def pair_dims(rot_dims: int, style: str):
    """Index arrays (a, b): dimension pair j is (a[j], b[j])."""
    j = np.arange(rot_dims // 2)
    if style == "half":
        return j, j + rot_dims // 2
    if style == "interleaved":
        return 2 * j, 2 * j + 1
    raise ValueError(f"unknown rotary layout {style!r}")


def shift_keys(k, shift, base: float, rot_dims: int, style: str) -> np.ndarray:
    """Rotate keys k [n, H, d] (any real dtype) by their position shifts [n]; float64 result."""
    k = np.asarray(k, np.float64)
    if rot_dims > k.shape[-1]:
        raise ValueError("rotary dims exceed the head dimension")
    a, b = pair_dims(rot_dims, style)
    phi = np.asarray(shift, np.float64)[:, None] * rope_thetas(base, rot_dims)[None, :]
    c = np.cos(phi)[:, None, :]
    s = np.sin(phi)[:, None, :]
    x, y = k[..., a], k[..., b]
    out = k.copy()
    out[..., a] = x * c - y * s
    out[..., b] = x * s + y * c
    return out
