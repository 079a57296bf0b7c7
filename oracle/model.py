"""Per-layer QKV projection, float64.

Reading used here (the paper runs real models inside its backends; the hot
path only needs the K/V each layer writes): one hidden-state matrix X [T, d]
feeds every layer, and layer l projects it with its own weight
W_l [(Hq + 2 Hkv) dh, d] (rows: the Hq query heads, then the Hkv key heads,
then the Hkv value heads, dh rows each), i.e. QKV = X W_l^T.  There is no
output projection, MLP or normalisation and no chaining between layers, so the
K/V of a token depend only on its own row of X and its position.
"""
import numpy as np


def split_w(w, hq: int, hkv: int, dh: int):
    """Split W_l into (Wq [Hq*dh, d], Wk [Hkv*dh, d], Wv [Hkv*dh, d])."""
    w = np.asarray(w, dtype=np.float64)
    a, b = hq * dh, (hq + hkv) * dh
    return w[:a], w[a:b], w[b:]


def project_qkv(x, w, hq: int, hkv: int, dh: int):
    """x [T, d], W_l -> q [Hq, T, dh], k [Hkv, T, dh], v [Hkv, T, dh] (no RoPE)."""
    x = np.asarray(x, dtype=np.float64)
    wq, wk, wv = split_w(w, hq, hkv, dh)
    t = x.shape[0]
    q = (x @ wq.T).reshape(t, hq, dh).transpose(1, 0, 2)
    k = (x @ wk.T).reshape(t, hkv, dh).transpose(1, 0, 2)
    v = (x @ wv.T).reshape(t, hkv, dh).transpose(1, 0, 2)
    return q, k, v


def project_kv(x, w, hq: int, hkv: int, dh: int):
    """Keys and values only: x [T, d] -> k, v [Hkv, T, dh] (no RoPE)."""
    x = np.asarray(x, dtype=np.float64)
    _, wk, wv = split_w(w, hq, hkv, dh)
    t = x.shape[0]
    k = (x @ wk.T).reshape(t, hkv, dh).transpose(1, 0, 2)
    v = (x @ wv.T).reshape(t, hkv, dh).transpose(1, 0, 2)
    return k, v


def project_q(x_rows, w, hq: int, hkv: int, dh: int):
    """Queries of selected token rows: x_rows [R, d] -> q [R, Hq, dh] (no RoPE)."""
    x_rows = np.asarray(x_rows, dtype=np.float64)
    wq, _, _ = split_w(w, hq, hkv, dh)
    return (x_rows @ wq.T).reshape(x_rows.shape[0], hq, dh)
