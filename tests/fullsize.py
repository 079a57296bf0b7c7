"""Helpers for parity checks at the benchmark's full workload sizes.

At these sizes the oracle cannot run the whole workload, so:

* block tables, refcounts, the ring and state metadata are compared in full
  against the oracle pool in metadata-only mode (exact integers);
* numbers are compared for sampled layers (first and last), all KV heads, and
  sampled token rows: the oracle projects the keys/values of every token of a
  sampled layer in float64 and evaluates attention row by row.
"""
from __future__ import annotations

import numpy as np
import torch

import synth
from oracle import OraclePool, apply_rope, attention_rows, project_kv, project_q
from oracle.pool import PoolShape
from paper_2607_10987_amd import kvstate as kv
from twin import close, close_rerotated


class MetaTwin:
    """Device pool with all layers' weights + a metadata-only oracle pool."""

    def __init__(self, wl: synth.Workload, n_blocks: int, max_pos: int, max_states: int = 64,
                 scratch_tokens: int = 8192, batch: int = 16, order=None, seed: int = 0):
        s = wl.shape
        self.wl, self.s, self.seed = wl, s, seed
        L, cols, d = s.n_layers, s.qkv_cols, s.d_model
        self.w = torch.empty((L, cols, d), dtype=torch.bfloat16, device="cuda")
        for layer in range(L):
            self.w[layer] = synth.normal_torch(synth.w_key(seed, wl.name, layer), (cols, d),
                                               s.w_std, s.dtype, "cuda")
        self.cfg = kv.make_cfg(L, d, s.n_q_heads, s.n_kv_heads, s.head_dim, s.block_size,
                               s.dtype, max_pos, max_states, s.rope_base, 1)
        scratch = kv.kv_scratch_bytes(self.cfg, scratch_tokens, batch, max_pos)
        self.pool = kv.Pool(self.cfg, n_blocks, scratch, init_free_order=order)
        self.pool.set_weights(self.w, cols * d)
        self.orc = OraclePool(PoolShape(L, d, s.n_q_heads, s.n_kv_heads, s.head_dim,
                                        s.block_size, s.dtype, s.rope_base, max_pos, max_states,
                                        1), n_blocks, init_free_order=order, store_kv=False)
        self.sid = {}
        self._w64 = {}

    @property
    def h(self):
        return self.pool.h

    # ------------------------------------------------------------ inputs
    def x(self, key, shape):
        return synth.normal_torch(key, shape, 1.0, self.s.dtype, "cuda")

    def x64(self, key, shape):
        return synth.normal_f64(key, shape, 1.0, self.s.dtype, device="cuda")

    def w64(self, layer):
        if layer not in self._w64:
            s = self.s
            self._w64[layer] = synth.normal_f64(synth.w_key(self.seed, self.wl.name, layer),
                                                (s.qkv_cols, s.d_model), s.w_std, s.dtype,
                                                device="cuda")
        return self._w64[layer]

    # ------------------------------------------------------------ metadata
    def check_meta(self):
        torch.cuda.synchronize()
        kv.kv_sync(self.h)
        P = self.pool.n_blocks
        rc, ring, head, tail = kv.kv_read_allocator(self.h, P)
        orc_rc, orc_ring, oh, ot = self.orc.allocator()
        assert (head, tail) == (oh, ot)
        assert rc == orc_rc.tolist(), "refcounts differ"
        assert ring == orc_ring.tolist(), "free ring differs"
        for h, sid in self.sid.items():
            if self.orc.states[sid].status != "ACTIVE":
                continue
            info = kv.kv_state_info(self.h, h)
            assert (info["pos0"], info["n_tokens"], info["n_blocks"], info["lineage"]) == \
                self.orc.info(sid)
            assert kv.kv_read_block_table(self.h, h) == self.orc.table(sid), "block table"
            st = self.orc.states[sid]
            u = kv.kv_state_usage(self.h, h)
            assert (u["reuse"], u["last_access"], u["pinned"]) == \
                (st.reuse, st.last_access, st.pinned), ("eviction score terms", u)

    # ------------------------------------------------------------ device state
    def state_kv(self, h, layer):
        """Device K and V of a state at one layer: two [Hkv, n, dh] bf16 tensors."""
        table = kv.kv_read_block_table(self.h, h)
        n = kv.kv_state_info(self.h, h)["n_tokens"]
        blocks = self.pool.blocks_view()[table, layer]          # [nb, 2, Hkv, B, dh]
        nb, _, hkv, B, dh = blocks.shape
        x = blocks.permute(1, 2, 0, 3, 4).reshape(2, hkv, nb * B, dh)[:, :, :n]
        return x[0], x[1]


def ref_kv(mt: MetaTwin, layer: int, x64: np.ndarray, positions):
    """Oracle keys (rotated) and values of rows x64 at `positions`: [Hkv, n, dh]."""
    s = mt.s
    k, v = project_kv(x64, mt.w64(layer), s.n_q_heads, s.n_kv_heads, s.head_dim)
    return apply_rope(k, np.asarray(positions), s.rope_base), v


def ref_rows(mt: MetaTwin, layer: int, xq64: np.ndarray, q_pos, k, v, k_pos, nvis):
    """Oracle attention outputs [R, Hq * dh] for query rows xq64 [R, d] at q_pos,
    row r seeing the first nvis[r] keys of k / v ([Hkv, n, dh] at k_pos)."""
    s = mt.s
    q = project_q(xq64, mt.w64(layer), s.n_q_heads, s.n_kv_heads, s.head_dim)   # [R, Hq, dh]
    R = q.shape[0]
    G = s.n_q_heads // s.n_kv_heads
    out = np.empty((R, s.n_q_heads, s.head_dim))
    for r in range(R):
        qr = apply_rope(q[r][:, None, :], np.full(1, q_pos[r]), s.rope_base)[:, 0, :]
        n = int(nvis[r])
        heads = np.arange(s.n_q_heads) // G
        out[r] = attention_rows(qr, k[:, :n], v[:, :n], np.full(s.n_q_heads, q_pos[r]),
                                np.asarray(k_pos)[:n], heads)
    return out.reshape(R, -1)


def sample_rows(n: int, B: int, count: int, rng) -> np.ndarray:
    """First, last, block-boundary and random rows of [0, n)."""
    base = {0, 1, n - 1, n - 2}
    for b in (1, 2, n // B // 2, n // B - 1):
        if 0 < b * B < n:
            base |= {b * B - 1, b * B}
    extra = rng.choice(n, size=min(n, max(0, count - len(base))), replace=False)
    return np.array(sorted(base | set(int(e) for e in extra)))


def to64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to(torch.float64).cpu().numpy()


__all__ = ["MetaTwin", "ref_kv", "ref_rows", "sample_rows", "to64", "close", "close_rerotated"]
