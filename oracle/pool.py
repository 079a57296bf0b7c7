"""Paged KV block pool and the KV-state operators, float64 / exact integers.

What the paper fixes (stateful-operator section, KV-state-manager section,
metadata-catalog table, KV-operator algorithms appendix):

* a KV state is S_KV = (M, Theta, B, Pi, Lambda, Gamma): model id, model
  configuration, a set of fixed-size KV blocks, positional metadata, lineage
  and placement.  Here M = ``model_id``, Theta = the shape fields of the pool,
  B = the state's block table, Pi = (pos0, n), Lambda = a lineage word,
  Gamma = this (single) device;
* blocks are shared between states and carry a refcount equal to the number
  of logical states that reference them (metadata-catalog table);
* KV-Materialize runs prefill once, partitions K/V into blocks and registers
  them; KV-Fork checks the parent is valid and not evicted, then aliases its
  blocks into k children by raising refcounts, each child recording
  fork(j) in its lineage; forks share blocks until a branch needs its own
  continuation (copy-on-write);
* KV-Transfer selects the blocks a downstream range needs, ships metadata and
  raw block buffers, and registers the received blocks (here: pack / unpack);
* KV-Resume initialises the position from Pi, appends the suffix and decodes
  over the reused blocks, registering new continuation blocks (here: attend);
* Restricted-KV-Merge checks compatibility and only concatenates
  non-overlapping segments (here: compose);
* KV-Evict scores states with alpha*reuse - beta*size - gamma*age and releases
  the lowest-scored ones while allocated memory exceeds the budget; shared
  blocks survive as long as another state references them.

Readings taken where the paper is silent (each is listed in the design notes):

* free blocks sit in a FIFO ring initialised to ``init_free_order``
  (default 0..P-1); allocation pops from the head in order, frees append at
  the tail, so every operation has exactly one correct block table;
* materialize = an empty state at pos0 followed by an append of T tokens;
* attend processes the batch in order; for each state it first copies a
  shared partial tail block (copy-on-write, slots [0, n mod B)), then
  allocates the blocks the append needs, in logical order;
* compose: destination positions continue from the first token of segment 0;
  a destination block aliases a source block (refcount + 1) iff all of its
  slots come, at identical slot indices and with a zero position shift, from
  one source block (the final partial block qualifies only if it is the source
  state's own tail holding the same tokens); every other block is newly
  allocated in logical order and filled token by token, keys re-rotated by the
  segment's shift and values copied;
* pack writes the blocks [b0, b1) of a state in logical order, slots beyond
  the state's last token zero-filled;
* a logical clock advances once per state touched (inputs in argument order,
  then outputs); eviction orders unpinned active states by (score, state_id)
  with age = clock - last_access, size = blocks in the table, reuse = times
  the state was an operator input;
* KV-Evict's branch for a state whose blocks are shared (give up only the
  unshared continuation) is offered as ``evict_truncate``: the victim keeps
  the blocks in front of its first unshared one, whole blocks only;
* a checked transfer (header flag) is verified against the payload checksum
  of ``checksum.py`` after allocation; a mismatch returns the blocks to the
  ring and fails.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from enum import IntEnum

import numpy as np

from .attention import causal_gqa_attention
from .model import project_qkv
from .rope import apply_rope, rerotate
from .checksum import payload_checksum

PACK_MAGIC = 0x5453564B          # "KVST" read as a little-endian uint32
PACK_VERSION = 2
PACK_CHECKSUM = 1
NO_PARENT = 0xFFFFFFFF
MAX_SEGMENTS = 64
MAX_BATCH = 64


class Status(IntEnum):
    OK = 0
    ARG = -1
    OOM = -2
    INCOMPATIBLE = -3
    EVICTED = -4
    BAD_HEADER = -5
    BUFSIZE = -6
    CAPACITY = -7
    HIP = -8
    INTERNAL = -9
    CHECKSUM = -10
    IO = -11


class Lineage(IntEnum):
    MATERIALIZE = 1
    FORK = 2
    TRANSFER = 3
    MERGE = 4


def lineage_word(kind: int, parent: int = NO_PARENT, fork_index: int = 0) -> int:
    """kind in bits 56..63, fork index j in bits 32..55, parent state_id in 0..31."""
    return (int(kind) << 56) | ((int(fork_index) & 0xFFFFFF) << 32) | (int(parent) & 0xFFFFFFFF)


class OracleError(Exception):
    def __init__(self, status: Status, msg: str = ""):
        super().__init__(f"{status.name}: {msg}")
        self.status = status


@dataclass
class _State:
    sid: int
    pos0: int
    n: int
    table: list
    lineage: int
    status: str = "ACTIVE"        # ACTIVE, EVICTED, RELEASED
    pinned: bool = False
    last_access: int = 0
    reuse: int = 0


@dataclass
class PoolShape:
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    block_size: int
    dtype: str = "f32"
    rope_base: float = 10000.0
    max_pos: int = 4096
    max_states: int = 64
    model_id: int = 1

    def compat_key(self):
        return (self.n_layers, self.d_model, self.n_q_heads, self.n_kv_heads,
                self.head_dim, self.block_size, self.dtype, float(self.rope_base))

    @property
    def elt_bytes(self):
        return 4 if self.dtype == "f32" else 2

    @property
    def block_bytes(self):
        return (self.n_layers * 2 * self.n_kv_heads * self.block_size * self.head_dim
                * self.elt_bytes)


def _ceil_div(a, b):
    return -(-a // b)


class OraclePool:
    """Exact model of one pool of ``n_blocks`` KV blocks.

    ``weights`` is a list (one per layer) of float64 W_l [(Hq+2Hkv)dh, d].
    With ``store_kv=False`` only the integer metadata is modelled (block
    tables, refcounts, ring, catalog); numeric inputs may then be ``None``.
    """

    def __init__(self, shape: PoolShape, n_blocks: int, init_free_order=None,
                 weights=None, store_kv: bool = True):
        self.shape = shape
        self.P = int(n_blocks)
        if init_free_order is None:
            order = np.arange(self.P, dtype=np.int64)
        else:
            order = np.asarray(init_free_order, dtype=np.int64).reshape(-1)
            if order.size != self.P or not np.array_equal(np.sort(order), np.arange(self.P)):
                raise OracleError(Status.ARG, "init_free_order is not a permutation")
        self.ring = order.astype(np.int32).copy()
        self.head = 0
        self.tail = self.P
        self.refcount = np.zeros(self.P, dtype=np.int32)
        self.states: dict[int, _State] = {}
        self.next_sid = 0
        self.clock = 0
        self.weights = weights
        self.store_kv = store_kv
        s = shape
        if store_kv:
            self.kv = np.zeros((self.P, s.n_layers, 2, s.n_kv_heads, s.block_size,
                                s.head_dim), dtype=np.float64)
        else:
            self.kv = None

    # ------------------------------------------------------------ allocator

    def free_count(self) -> int:
        return self.tail - self.head

    def allocated(self) -> int:
        return self.P - self.free_count()

    def _alloc(self, n: int) -> list:
        if n > self.free_count():
            raise OracleError(Status.INTERNAL, "allocation beyond the free count")
        ids = [int(self.ring[(self.head + i) % self.P]) for i in range(n)]
        self.head += n
        for b in ids:
            self.refcount[b] = 1
        return ids

    def _free(self, b: int):
        self.ring[self.tail % self.P] = b
        self.tail += 1

    def _drop_refs(self, st: _State):
        for b in st.table:
            self.refcount[b] -= 1
            if self.refcount[b] == 0:
                self._free(b)
        st.table = []

    # ------------------------------------------------------------ catalog

    def _live(self) -> int:
        return sum(1 for st in self.states.values() if st.status == "ACTIVE")

    def _get(self, sid: int) -> _State:
        st = self.states.get(sid)
        if st is None or st.status != "ACTIVE":
            raise OracleError(Status.EVICTED, f"state {sid} is not active")
        return st

    def _new_state(self, pos0: int, lineage: int) -> _State:
        st = _State(sid=self.next_sid, pos0=pos0, n=0, table=[], lineage=lineage)
        self.next_sid += 1
        self.states[st.sid] = st
        return st

    def _touch(self, st: _State, as_input: bool):
        self.clock += 1
        st.last_access = self.clock
        if as_input:
            st.reuse += 1

    # ------------------------------------------------------------ numerics

    def _valid(self, st: _State, j: int) -> int:
        return min(self.shape.block_size, st.n - j * self.shape.block_size)

    def state_kv(self, sid: int, layer: int):
        """K and V of a state's tokens at one layer: two [Hkv, n, dh] arrays."""
        st = self.states[sid]
        s = self.shape
        k = np.empty((s.n_kv_heads, st.n, s.head_dim))
        v = np.empty_like(k)
        for j, b in enumerate(st.table):
            lo = j * s.block_size
            m = self._valid(st, j)
            k[:, lo:lo + m] = self.kv[b, layer, 0, :, :m]
            v[:, lo:lo + m] = self.kv[b, layer, 1, :, :m]
        return k, v

    def _store(self, st: _State, layer: int, t0: int, k, v):
        """Write K/V rows for logical tokens t0.. of a state."""
        B = self.shape.block_size
        for t in range(k.shape[1]):
            u = t0 + t
            b = st.table[u // B]
            self.kv[b, layer, 0, :, u % B] = k[:, t]
            self.kv[b, layer, 1, :, u % B] = v[:, t]

    def _append_compute(self, st: _State, x, n_before: int):
        """Project x [T, d], rotate, store, and attend causally; o [L, T, Hq*dh]."""
        s = self.shape
        T = x.shape[0]
        L, hq, hkv, dh = s.n_layers, s.n_q_heads, s.n_kv_heads, s.head_dim
        o = np.empty((L, T, hq * dh))
        qpos = st.pos0 + n_before + np.arange(T)
        for layer in range(L):
            q, k, v = project_qkv(x, self.weights[layer], hq, hkv, dh)
            q = apply_rope(q, qpos, s.rope_base)
            k = apply_rope(k, qpos, s.rope_base)
            self._store(st, layer, n_before, k, v)
            kall, vall = self.state_kv(st.sid, layer)
            kpos = st.pos0 + np.arange(st.n)
            out = causal_gqa_attention(q, kall, vall, qpos, kpos)
            o[layer] = out.transpose(1, 0, 2).reshape(T, hq * dh)
        return o

    # ------------------------------------------------------------ operators

    def materialize(self, x, T: int = None, pos0: int = 0):
        """KV-Materialize: returns (state_id, o [L, T, Hq*dh] or None)."""
        s = self.shape
        if x is not None:
            x = np.asarray(x, dtype=np.float64)
            T = x.shape[0]
        if T is None or T <= 0 or pos0 < 0:
            raise OracleError(Status.ARG, "empty context or negative position")
        if pos0 + T > s.max_pos:
            raise OracleError(Status.CAPACITY, "positions beyond max_pos")
        if self._live() >= s.max_states:
            raise OracleError(Status.CAPACITY, "catalog full")
        nb = _ceil_div(T, s.block_size)
        if nb > self.free_count():
            raise OracleError(Status.OOM, "not enough free blocks")
        st = self._new_state(pos0, lineage_word(Lineage.MATERIALIZE))
        st.table = self._alloc(nb)
        st.n = T
        o = None
        if self.store_kv and x is not None:
            o = self._append_compute(st, x, 0)
        self._touch(st, as_input=False)
        return st.sid, o

    def fork(self, sid: int, k: int):
        """KV-Fork: k children alias the parent's blocks."""
        if k < 1:
            raise OracleError(Status.ARG, "k < 1")
        parent = self._get(sid)
        if self._live() + k > self.shape.max_states:
            raise OracleError(Status.CAPACITY, "catalog full")
        children = []
        for j in range(1, k + 1):
            c = self._new_state(parent.pos0, lineage_word(Lineage.FORK, parent.sid, j))
            c.table = list(parent.table)
            c.n = parent.n
            children.append(c)
        for b in parent.table:
            self.refcount[b] += k
        self._touch(parent, as_input=True)
        for c in children:
            self._touch(c, as_input=False)
        return [c.sid for c in children]

    def attend_plan(self, sids, T: int):
        """Validate an append and return the number of blocks it allocates."""
        s = self.shape
        if len(sids) < 1 or len(sids) > MAX_BATCH or T <= 0:
            raise OracleError(Status.ARG, "bad batch or T")
        if len(set(sids)) != len(sids):
            raise OracleError(Status.ARG, "duplicate state in batch")
        sts = [self._get(x) for x in sids]
        for st in sts:
            if st.pos0 + st.n + T > s.max_pos:
                raise OracleError(Status.CAPACITY, "positions beyond max_pos")
        need = 0
        B = s.block_size
        for st in sts:
            if st.n % B and self.refcount[st.table[-1]] > 1:
                need += 1
            need += _ceil_div(st.n + T, B) - _ceil_div(st.n, B)
        return sts, need

    def attend(self, sids, x=None, T: int = None):
        """KV-Resume over a batch: append T tokens to each state and attend.

        x [batch, T, d]; returns o [L, batch, T, Hq*dh] (None without numerics).
        """
        if x is not None:
            x = np.asarray(x, dtype=np.float64)
            T = x.shape[1]
            if x.shape[0] != len(sids):
                raise OracleError(Status.ARG, "x batch mismatch")
        if T is None:
            raise OracleError(Status.ARG, "T missing")
        sts, need = self.attend_plan(sids, T)
        if need > self.free_count():
            raise OracleError(Status.OOM, "not enough free blocks")
        s = self.shape
        B = s.block_size
        for st in sts:
            if st.n % B and self.refcount[st.table[-1]] > 1:
                old = st.table[-1]
                new = self._alloc(1)[0]
                if self.store_kv:
                    m = st.n % B
                    self.kv[new, :, :, :, :m] = self.kv[old, :, :, :, :m]
                self.refcount[old] -= 1
                st.table[-1] = new
            st.table += self._alloc(_ceil_div(st.n + T, B) - _ceil_div(st.n, B))
        o = None
        if self.store_kv and x is not None:
            o = np.empty((s.n_layers, len(sts), T, s.n_q_heads * s.head_dim))
        for i, st in enumerate(sts):
            n0 = st.n
            st.n = n0 + T
            if o is not None:
                o[:, i] = self._append_compute(st, x[i], n0)
        for st in sts:
            self._touch(st, as_input=True)
        return o

    def compose_plan(self, segs):
        """Validate a composition; return (states, per-block plan, N, P0).

        plan[b] = ("alias", segment, source block index) or ("copy",).
        """
        s = self.shape
        B = s.block_size
        if len(segs) < 1 or len(segs) > MAX_SEGMENTS:
            raise OracleError(Status.ARG, "bad segment count")
        sts = []
        for sid, a, e in segs:
            st = self._get(sid)
            if not (0 <= a < e <= st.n):
                raise OracleError(Status.ARG, "bad segment range")
            sts.append(st)
        lens = [e - a for _, a, e in segs]
        N = sum(lens)
        P0 = sts[0].pos0 + segs[0][1]
        if P0 + N > s.max_pos:
            raise OracleError(Status.CAPACITY, "positions beyond max_pos")
        if self._live() >= s.max_states:
            raise OracleError(Status.CAPACITY, "catalog full")
        cum = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        plan = []
        for b in range(_ceil_div(N, B)):
            u0, u1 = b * B, min(b * B + B, N)
            i = int(np.searchsorted(cum, u0, side="right") - 1)
            st = sts[i]
            a, e = segs[i][1], segs[i][2]
            off = int(cum[i]) - a
            delta = P0 + off - st.pos0
            ok = (u1 <= cum[i + 1] and delta == 0 and off % B == 0)
            if ok and u1 - u0 < B:
                ok = (i == len(segs) - 1 and e == st.n and u1 == N)
            if ok:
                plan.append(("alias", i, (u0 - off) // B))
            else:
                plan.append(("copy",))
        return sts, plan, N, P0, cum

    def compose(self, segs):
        """Restricted merge by ordered concatenation of token-range segments.

        segs: list of (state_id, tok_begin, tok_end) with 0 <= begin < end <= n.
        """
        segs = [(int(a), int(b), int(c)) for a, b, c in segs]
        sts, plan, N, P0, cum = self.compose_plan(segs)
        ncopy = sum(1 for p in plan if p[0] == "copy")
        if ncopy > self.free_count():
            raise OracleError(Status.OOM, "not enough free blocks")
        s = self.shape
        B = s.block_size
        new = self._new_state(P0, lineage_word(Lineage.MERGE, sts[0].sid))
        fresh = iter(self._alloc(ncopy))
        table = []
        for p in plan:
            if p[0] == "alias":
                b = sts[p[1]].table[p[2]]
                self.refcount[b] += 1
                table.append(b)
            else:
                table.append(next(fresh))
        new.table = table
        new.n = N
        if self.store_kv:
            for b, p in enumerate(plan):
                if p[0] != "copy":
                    continue
                for u in range(b * B, min(b * B + B, N)):
                    i = int(np.searchsorted(cum, u, side="right") - 1)
                    st = sts[i]
                    off = int(cum[i]) - segs[i][1]
                    j = u - off
                    delta = P0 + off - st.pos0
                    src = st.table[j // B]
                    kk = self.kv[src, :, 0, :, j % B]          # [L, Hkv, dh]
                    self.kv[table[b], :, 0, :, u % B] = rerotate(
                        kk[:, :, None, :], delta, s.rope_base)[:, :, 0, :]
                    self.kv[table[b], :, 1, :, u % B] = self.kv[src, :, 1, :, j % B]
        for st in sts:
            self._touch(st, as_input=True)
        self._touch(new, as_input=False)
        return new.sid

    def pack(self, sid: int, b0: int, b1: int):
        """Transfer source side: header + blocks [b0, b1) in logical order."""
        st = self._get(sid)
        s = self.shape
        if not (0 <= b0 < b1 <= len(st.table)):
            raise OracleError(Status.ARG, "bad block range")
        nblk = b1 - b0
        hdr = dict(magic=PACK_MAGIC, version=PACK_VERSION, model_id=s.model_id,
                   compat=s.compat_key(), pos_begin=st.pos0 + b0 * s.block_size,
                   n_tokens=min(st.n, b1 * s.block_size) - b0 * s.block_size,
                   blk_begin=b0, n_blocks=nblk, block_bytes=s.block_bytes,
                   payload_bytes=nblk * s.block_bytes, lineage=st.lineage,
                   src_state_id=st.sid, flags=0, checksum=(0, 0))
        payload = None
        if self.store_kv:
            payload = np.zeros((nblk,) + self.kv.shape[1:])
            for i, j in enumerate(range(b0, b1)):
                m = self._valid(st, j)
                payload[i, :, :, :, :m] = self.kv[st.table[j], :, :, :, :m]
        self._touch(st, as_input=True)
        return hdr, payload

    def unpack(self, hdr: dict, payload=None, src_bytes: int = None, raw: bytes = None):
        """Transfer destination side: check the header, allocate, copy, register.

        A header flagged with a checksum is verified against ``raw``, the
        payload's bytes, after the blocks are allocated (the copy and the
        check are one pass on a device): on a mismatch the blocks go back to
        the ring tail in logical order, the drawn state id stays used, and
        the call fails with CHECKSUM.
        """
        s = self.shape
        if hdr.get("magic") != PACK_MAGIC or hdr.get("version") != PACK_VERSION:
            raise OracleError(Status.BAD_HEADER, "magic/version")
        if hdr.get("flags", 0) & ~PACK_CHECKSUM:
            raise OracleError(Status.BAD_HEADER, "unknown flags")
        if hdr["model_id"] != s.model_id or tuple(hdr["compat"]) != s.compat_key():
            raise OracleError(Status.INCOMPATIBLE, "model or configuration differs")
        nb, nt = hdr["n_blocks"], hdr["n_tokens"]
        B = s.block_size
        if (nb < 1 or not ((nb - 1) * B < nt <= nb * B) or hdr["block_bytes"] != s.block_bytes
                or hdr["payload_bytes"] != nb * s.block_bytes or hdr["pos_begin"] < 0):
            raise OracleError(Status.BAD_HEADER, "inconsistent sizes")
        if src_bytes is not None and src_bytes < hdr["payload_bytes"]:
            raise OracleError(Status.BUFSIZE, "source buffer too small")
        if hdr["pos_begin"] + nt > s.max_pos:
            raise OracleError(Status.CAPACITY, "positions beyond max_pos")
        if self._live() >= s.max_states:
            raise OracleError(Status.CAPACITY, "catalog full")
        if nb > self.free_count():
            raise OracleError(Status.OOM, "not enough free blocks")
        st = self._new_state(int(hdr["pos_begin"]),
                             lineage_word(Lineage.TRANSFER, hdr["src_state_id"]))
        st.table = self._alloc(nb)
        st.n = int(nt)
        if hdr.get("flags", 0) & PACK_CHECKSUM:
            if raw is None:
                raise OracleError(Status.ARG, "checked header without payload bytes")
            if payload_checksum(raw) != tuple(hdr["checksum"]):
                self._drop_refs(st)
                st.status = "RELEASED"
                raise OracleError(Status.CHECKSUM, "payload does not match its checksum")
        if self.store_kv and payload is not None:
            for i, b in enumerate(st.table):
                self.kv[b] = payload[i]
        self._touch(st, as_input=False)
        return st.sid

    def release(self, sid: int):
        st = self._get(sid)
        self._drop_refs(st)
        st.status = "RELEASED"

    def pin(self, sid: int, pinned: bool):
        self._get(sid).pinned = bool(pinned)

    def eviction_order(self, alpha=0.0, beta=0.0, gamma=1.0):
        c = [st for st in self.states.values() if st.status == "ACTIVE" and not st.pinned]

        def score(st):
            age = self.clock - st.last_access
            return (alpha * st.reuse - beta * len(st.table)) - gamma * age
        return sorted(c, key=lambda st: (score(st), st.sid))

    def evict(self, max_allocated: int, alpha=0.0, beta=0.0, gamma=1.0) -> int:
        """KV-Evict: release lowest-score states while allocated > budget."""
        if max_allocated < 0:
            raise OracleError(Status.ARG, "negative budget")
        n = 0
        for st in self.eviction_order(alpha, beta, gamma):
            if self.allocated() <= max_allocated:
                break
            self._drop_refs(st)
            st.status = "EVICTED"
            n += 1
        return n

    def evict_truncate(self, max_allocated: int, alpha=0.0, beta=0.0, gamma=1.0):
        """KV-Evict, the branch for a state that shares blocks (KV-Evict
        algorithm, the alternative to freeing the whole state): a victim keeps
        the prefix of its table in front of its first unshared block
        (refcount 1) and drops every block from there on, so only its
        continuation is given up; its token count becomes that prefix's
        (whole blocks).  A victim with no shared leading block is evicted
        whole; one with no unshared block frees nothing and is left as it is.
        Victims in score order while allocated > budget.  Returns
        (states evicted, states truncated)."""
        if max_allocated < 0:
            raise OracleError(Status.ARG, "negative budget")
        n_ev = n_tr = 0
        B = self.shape.block_size
        for st in self.eviction_order(alpha, beta, gamma):
            if self.allocated() <= max_allocated:
                break
            j = next((i for i, b in enumerate(st.table) if self.refcount[b] == 1),
                     len(st.table))
            if j == len(st.table):
                continue
            if j == 0:
                self._drop_refs(st)
                st.status = "EVICTED"
                n_ev += 1
                continue
            for b in st.table[j:]:
                self.refcount[b] -= 1
                if self.refcount[b] == 0:
                    self._free(b)
            st.table = st.table[:j]
            st.n = j * B
            n_tr += 1
        return n_ev, n_tr

    # ------------------------------------------------------------ queries

    def info(self, sid: int):
        st = self._get(sid)
        return st.pos0, st.n, len(st.table), st.lineage

    def table(self, sid: int):
        return list(self._get(sid).table)

    def allocator(self):
        return self.refcount.copy(), self.ring.copy(), self.head, self.tail
