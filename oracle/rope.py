"""Rotary position encoding (RoPE), float64.

The paper does not define positional encoding; it only requires that fork and
merge keep position semantics (correctness-constraints section) and that
restricted merge must not blend states in a way that breaks RoPE (branching
optimisation section).  Reading used here (Llama family convention):

* frequencies theta_i = base^(-2 i / dh), i in [0, dh/2);
* the rotated pairs are (u_i, u_{i + dh/2}) ("half split");
* at position p:  u'_i        = u_i cos(p theta_i) - u_{i+dh/2} sin(p theta_i)
                  u'_{i+dh/2} = u_i sin(p theta_i) + u_{i+dh/2} cos(p theta_i)

Re-rotation by a shift Delta (used when composition moves a segment to new
positions) is the same rotation with p replaced by Delta, applied to keys that
already carry the encoding of their old position.
"""
import numpy as np


def inv_freq(dh: int, base: float) -> np.ndarray:
    """theta_i = base^(-2i/dh) for i in [0, dh/2), float64."""
    i = np.arange(dh // 2, dtype=np.float64)
    return np.power(float(base), -2.0 * i / dh)


def rope_angles(positions, dh: int, base: float) -> np.ndarray:
    """Angles p * theta_i, shape [n, dh/2]."""
    p = np.asarray(positions, dtype=np.float64).reshape(-1, 1)
    return p * inv_freq(dh, base)[None, :]


def apply_rope(u: np.ndarray, positions, base: float) -> np.ndarray:
    """Rotate the last axis of ``u`` (shape [..., n, dh]) by the angles of
    ``positions`` (length n)."""
    u = np.asarray(u, dtype=np.float64)
    dh = u.shape[-1]
    half = dh // 2
    ang = rope_angles(positions, dh, base)          # [n, half]
    c, s = np.cos(ang), np.sin(ang)
    a, b = u[..., :half], u[..., half:]
    out = np.empty_like(u)
    out[..., :half] = a * c - b * s
    out[..., half:] = a * s + b * c
    return out


def rerotate(u: np.ndarray, delta: int, base: float) -> np.ndarray:
    """Rotate already-encoded keys (shape [..., n, dh]) by a constant shift."""
    n = u.shape[-2]
    return apply_rope(u, np.full(n, delta, dtype=np.int64), base)
