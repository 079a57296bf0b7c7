"""Transfer-vs-recompute decision (oracle, float64; test infrastructure).

The paper's state-aware scheduling rule chooses, for a state S, transfer
when its estimated transfer time is below the time to recompute it by
prefill, and recompute otherwise; the KV-Transfer algorithm opens with the
same comparison, estimating the transfer as the KV size over the link
bandwidth plus a fixed latency.  The paper leaves both estimates to the
runtime.  Readings used here (the device library implements the same):

* the KV size is what a transfer moves: the whole blocks covering the state
  (ceil(n / B) blocks of L * 2 * Hkv * B * dh elements);
* on a GPU the transfer also pays packing the blocks into a contiguous buffer
  and unpacking them at the destination, at measured rates (omitted when a
  rate is not given);
* the prefill time is the algorithmic work of recomputing the state (the QKV
  projections of n tokens in every layer and causal attention over the
  visible (query, key) pairs) over a measured prefill rate.
"""
from __future__ import annotations

import math


def kv_bytes(L: int, Hkv: int, dh: int, B: int, elt_bytes: int, n: int) -> float:
    """Bytes of the blocks that hold an n-token state."""
    blocks = math.ceil(n / B)
    return float(blocks) * (2.0 * L * Hkv * B * dh * elt_bytes)


def prefill_flops(L: int, d: int, Hq: int, Hkv: int, dh: int, n: int) -> float:
    """Projection flops (2 per multiply-add, every layer, Q, K and V) plus
    causal attention flops (scores and weighted values: 4 dh per visible
    (query, key) pair per query head)."""
    proj = 2.0 * n * d * (Hq + 2 * Hkv) * dh
    pairs = n * (n + 1) / 2.0
    attn = 4.0 * Hq * dh * pairs
    return L * (proj + attn)


def plan_transfer(L, d, Hq, Hkv, dh, B, elt_bytes, n, link_bytes_per_s, link_latency_s,
                  pack_bytes_per_s, unpack_bytes_per_s, prefill_flops_per_s) -> dict:
    """Both estimates and the decision (transfer iff t_transfer < t_prefill)."""
    kb = kv_bytes(L, Hkv, dh, B, elt_bytes, n)
    t_transfer = kb / link_bytes_per_s + link_latency_s
    if pack_bytes_per_s > 0:
        t_transfer += kb / pack_bytes_per_s
    if unpack_bytes_per_s > 0:
        t_transfer += kb / unpack_bytes_per_s
    fl = prefill_flops(L, d, Hq, Hkv, dh, n)
    t_prefill = fl / prefill_flops_per_s
    return {"kv_bytes": kb, "t_transfer": t_transfer, "t_prefill": t_prefill,
            "prefill_flops": fl, "transfer": t_transfer < t_prefill}
