"""Causal grouped-query attention, float64.

Not defined by the paper (its backends run the model).  Reading used here:
scaled dot product with scale 1/sqrt(dh); query head h reads KV head
floor(h / G) with G = Hq / Hkv (consecutive grouping); key s is visible to
query t iff position(s) <= position(t); the softmax subtracts the row maximum.
"""
import numpy as np


def causal_gqa_attention(q, k, v, q_pos, k_pos):
    """q [Hq, Tq, dh], k/v [Hkv, Tk, dh], positions -> o [Hq, Tq, dh]."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    hq, tq, dh = q.shape
    hkv = k.shape[0]
    if hq % hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    g = hq // hkv
    q_pos = np.asarray(q_pos).reshape(-1)
    k_pos = np.asarray(k_pos).reshape(-1)
    visible = k_pos[None, :] <= q_pos[:, None]             # [Tq, Tk]
    out = np.empty_like(q)
    scale = 1.0 / np.sqrt(dh)
    for h in range(hq):
        kv = h // g
        s = (q[h] @ k[kv].T) * scale                        # [Tq, Tk]
        s = np.where(visible, s, -np.inf)
        m = s.max(axis=1, keepdims=True)
        p = np.exp(s - m)
        p /= p.sum(axis=1, keepdims=True)
        out[h] = p @ v[kv]
    return out


def attention_rows(q_rows, k, v, q_pos, k_pos, heads):
    """Attention for selected (row, head) pairs.

    q_rows [R, dh] are query vectors of heads ``heads`` [R] at positions
    ``q_pos`` [R]; k/v [Hkv, Tk, dh]; returns o [R, dh].  Used for sampled
    checks at full workload size.
    """
    q_rows = np.asarray(q_rows, dtype=np.float64)
    hkv = k.shape[0]
    heads = np.asarray(heads).reshape(-1)
    out = np.empty_like(q_rows)
    dh = q_rows.shape[-1]
    k_pos = np.asarray(k_pos).reshape(-1)
    return _rows(q_rows, k, v, q_pos, k_pos, heads, hkv, dh, out)


def _rows(q_rows, k, v, q_pos, k_pos, heads, hkv, dh, out):
    scale = 1.0 / np.sqrt(dh)
    for r in range(q_rows.shape[0]):
        kvh = int(heads[r])
        vis = k_pos <= q_pos[r]
        s = (k[kvh][vis] @ q_rows[r]) * scale
        p = np.exp(s - s.max())
        out[r] = (p / p.sum()) @ v[kvh][vis]
    return out
