"""Pins for the oracle's pool model and operators, CPU only.

* a hand-derived trace of the allocator (FIFO ring, refcounts, copy-on-write,
  aliasing in compose, LRU eviction) on an 8-block pool;
* invariants over random operation sequences (refcount = number of live
  tables holding a block; free ring and referenced blocks partition the pool);
* the equivalences the operators imply in exact arithmetic: attention after
  fork / compose / decode equals attention after recomputing the concatenated
  context; pack then unpack is an exact round trip; a child's write never
  changes its parent;
* error codes for the failure cases the paper names (evicted state,
  incompatible state, memory exhaustion).
"""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import OracleError, OraclePool, Status, causal_gqa_attention
from oracle.pool import PoolShape, Lineage, lineage_word

RNG = np.random.default_rng(77)


def meta_pool(P=8, B=2, max_pos=64, max_states=16, order=None):
    shape = PoolShape(n_layers=1, d_model=4, n_q_heads=2, n_kv_heads=1, head_dim=4,
                      block_size=B, max_pos=max_pos, max_states=max_states)
    return OraclePool(shape, P, init_free_order=order, store_kv=False)


# ------------------------------------------------------------------ hand trace

def test_allocator_hand_trace():
    p = meta_pool()
    s0, _ = p.materialize(None, T=5)                 # ceil(5/2) = 3 blocks from the head
    assert p.table(s0) == [0, 1, 2]
    s1, s2 = p.fork(s0, 2)                           # children alias, refcount + 2
    assert p.table(s1) == p.table(s2) == [0, 1, 2]
    assert list(p.refcount[:3]) == [3, 3, 3]
    p.attend([s1], T=1)                              # tail (5 mod 2 = 1 slot) shared: COW -> 3
    assert p.table(s1) == [0, 1, 3] and p.refcount[2] == 2
    p.attend([s2, s0], T=2)                          # s2: COW -> 4, +1 block -> 5
    assert p.table(s2) == [0, 1, 4, 5]               # s0: tail now private, +1 block -> 6
    assert p.table(s0) == [0, 1, 2, 6]
    assert list(p.refcount) == [3, 3, 1, 1, 1, 1, 1, 0]
    p.release(s1)                                    # frees block 3 only (0, 1 still shared)
    rc, ring, head, tail = p.allocator()
    assert (head, tail) == (7, 9) and ring[0] == 3
    # compose [s2 tokens 0..4 | s0 tokens 4..6]: dest blocks 0, 1 alias s2's blocks
    # (shift 0, aligned); block 2 straddles the segments; block 3 takes s0's tokens
    # with shift +1 -> two fresh blocks in logical order: ring[7] = 7, ring[8 mod 8] = 3
    s3 = p.compose([(s2, 0, 5), (s0, 4, 7)])
    assert p.table(s3) == [0, 1, 7, 3]
    assert p.info(s3)[:3] == (0, 8, 4)
    assert list(p.refcount) == [3, 3, 1, 1, 1, 1, 1, 1]
    # clock: s0 1, fork 2..4, attend s1 5, attend s2 6 / s0 7, compose s2 8, s0 9, s3 10
    # LRU order: s2 (age 2), s0 (age 1), s3 (age 0); budget 5 of 8 allocated
    n = p.evict(5)
    assert n == 2                                    # s2 frees 4, 5; s0 frees 2, 6
    rc, ring, head, tail = p.allocator()
    assert list(rc) == [1, 1, 0, 1, 0, 0, 0, 1]
    assert (head, tail) == (9, 13)
    assert list(ring) == [3, 4, 5, 2, 6, 5, 6, 7]
    with pytest.raises(OracleError) as e:
        p.fork(s2, 1)
    assert e.value.status == Status.EVICTED
    assert p.table(s3) == [0, 1, 7, 3]


def test_compose_alias_rule_final_partial_block():
    p = meta_pool(P=16, B=4)
    a, _ = p.materialize(None, T=8)                  # [0, 1]
    b, = p.fork(a, 1)
    p.attend([b], T=3)                               # b: [0, 1, 2] with 11 tokens
    # [a 0..8 | b 8..11]: shift 0, aligned; final partial block is b's own tail
    c = p.compose([(a, 0, 8), (b, 8, 11)])
    assert p.table(c) == [0, 1, 2]
    assert p.refcount[2] == 2
    # the same but ending before b's last token: final block must be copied
    d = p.compose([(a, 0, 8), (b, 8, 10)])
    assert p.table(d) == [0, 1, 3]
    # a segment starting mid-block: nothing aligned after it can alias
    e = p.compose([(b, 2, 11)])
    assert p.info(e)[0] == 2 and p.table(e) == [4, 5, 6]
    # the composed tail is shared with b: b's next append copies it first
    p.attend([b], T=1)
    assert p.table(b) == [0, 1, 7] and p.refcount[2] == 1


def test_lineage_words():
    p = meta_pool()
    s0, _ = p.materialize(None, T=3)
    c1, c2 = p.fork(s0, 2)
    assert p.info(s0)[3] == lineage_word(Lineage.MATERIALIZE)
    assert p.info(c2)[3] == (Lineage.FORK << 56) | (2 << 32) | s0
    m = p.compose([(c1, 0, 3), (c2, 0, 3)])
    assert p.info(m)[3] >> 56 == Lineage.MERGE
    hdr, _ = p.pack(m, 0, 2)
    u = p.unpack(hdr)
    assert p.info(u)[3] == (Lineage.TRANSFER << 56) | m


def test_eviction_score_general_and_ties():
    p = meta_pool(P=32, B=2)
    a, _ = p.materialize(None, T=4)      # 2 blocks
    b, _ = p.materialize(None, T=8)      # 4 blocks
    c, _ = p.materialize(None, T=2)      # 1 block
    p.pack(a, 0, 1)                      # reuse(a) = 1
    # size-only score (beta = 1): largest first
    assert [s.sid for s in p.eviction_order(0, 1, 0)] == [b, a, c]
    # reuse-only score: least reused first, ties by state id
    assert [s.sid for s in p.eviction_order(1, 0, 0)] == [b, c, a]
    p.pin(b, True)
    assert p.evict(0) == 2 and p.allocated() == 4


def test_evict_truncate_hand_trace():
    p = meta_pool(P=16, B=2)
    s0, _ = p.materialize(None, T=4)                 # [0, 1], clock 1
    c1, c2 = p.fork(s0, 2)                           # clock 2 (s0), 3, 4
    p.attend([c1], T=3)                              # c1 [0, 1, 2, 3], 7 tokens, clock 5
    p.attend([c2], T=1)                              # c2 [0, 1, 4], 5 tokens, clock 6
    s3, _ = p.materialize(None, T=3)                 # [5, 6], clock 7
    assert p.allocated() == 7
    # LRU order s0, c1, c2, s3.  s0 holds only shared blocks: nothing to give
    # up, skipped.  c1 keeps [0, 1] (first unshared block at index 2) and frees
    # 2, 3; c2 frees 4; allocated is then 4 > 3, so s3 (no shared block) goes
    # whole: 5, 6.
    assert p.evict_truncate(3) == (1, 2)
    rc, ring, head, tail = p.allocator()
    assert list(rc[:8]) == [3, 3, 0, 0, 0, 0, 0, 0]
    assert (head, tail) == (7, 21) and list(ring[:5]) == [2, 3, 4, 5, 6]
    assert p.info(c1)[:3] == (0, 4, 2) and p.info(c2)[:3] == (0, 4, 2)
    assert p.info(s0)[:3] == (0, 4, 2)
    with pytest.raises(OracleError) as e:
        p.fork(s3, 1)
    assert e.value.status == Status.EVICTED
    # a truncated state resumes as usual: its tail is a whole block
    p.attend([c1], T=1)
    assert p.table(c1) == [0, 1, 7]
    # under budget: nothing happens
    assert p.evict_truncate(16) == (0, 0)


def test_evict_truncate_shared_partial_tail():
    p = meta_pool(P=16, B=2)
    s0, _ = p.materialize(None, T=5)                 # [0, 1, 2], block 2 holds 1 token
    c1, = p.fork(s0, 1)
    p.attend([c1], T=1)                              # COW: c1 [0, 1, 3]; block 2 now s0's alone
    assert p.refcount[2] == 1 and p.refcount[3] == 1
    # order s0 (older), c1: both keep the two shared leading blocks
    assert p.evict_truncate(2) == (0, 2)
    assert p.table(s0) == [0, 1] and p.table(c1) == [0, 1]
    assert p.info(s0)[1] == 4 and p.info(c1)[1] == 4
    rc, ring, head, tail = p.allocator()
    assert list(rc[:4]) == [2, 2, 0, 0] and list(ring[:2]) == [2, 3] and tail == 18
    # pinned states are not candidates
    p.pin(s0, True)
    p.pin(c1, True)
    assert p.evict_truncate(0) == (0, 0)


def test_exp4_block_counts_full_size():
    # memory claim of the paper's memory-efficiency experiment as exact counts:
    # a fork grows with the continuation, not with the prefix
    shape = PoolShape(32, 4096, 32, 8, 128, 16, "bf16", max_pos=40000, max_states=64)
    p = OraclePool(shape, 4096, store_kv=False)
    root, _ = p.materialize(None, T=32768)
    kids = p.fork(root, 16)
    p.attend(kids, T=1024)
    assert p.allocated() == 2048 + 16 * 64
    assert p.allocated() < 16 * (2048 + 64)


# ------------------------------------------------------------------ errors

def test_error_codes():
    p = meta_pool(P=4, B=2, max_pos=16, max_states=3)
    with pytest.raises(OracleError) as e:
        p.materialize(None, T=9)                     # 5 blocks > 4
    assert e.value.status == Status.OOM
    assert p.free_count() == 4                       # all-or-nothing
    s, _ = p.materialize(None, T=4)
    with pytest.raises(OracleError) as e:
        p.attend([s], T=13)
    assert e.value.status == Status.CAPACITY
    with pytest.raises(OracleError) as e:
        p.fork(s, 0)
    assert e.value.status == Status.ARG
    with pytest.raises(OracleError) as e:
        p.fork(s, 3)                                 # 4 live states > 3
    assert e.value.status == Status.CAPACITY
    with pytest.raises(OracleError) as e:
        p.attend([s, s], T=1)
    assert e.value.status == Status.ARG
    hdr, _ = p.pack(s, 0, 2)
    for field, val, code in (("magic", 1, Status.BAD_HEADER), ("model_id", 9, Status.INCOMPATIBLE),
                             ("n_tokens", 5, Status.BAD_HEADER)):
        h = dict(hdr)
        h[field] = val
        with pytest.raises(OracleError) as e:
            p.unpack(h)
        assert e.value.status == code
    h = dict(hdr)
    h["compat"] = (1, 4, 2, 1, 4, 4, "f32", 10000.0)      # block size differs
    with pytest.raises(OracleError) as e:
        p.unpack(h)
    assert e.value.status == Status.INCOMPATIBLE
    with pytest.raises(OracleError) as e:
        p.unpack(hdr, src_bytes=hdr["payload_bytes"] - 1)
    assert e.value.status == Status.BUFSIZE
    p.release(s)
    with pytest.raises(OracleError) as e:
        p.pack(s, 0, 1)
    assert e.value.status == Status.EVICTED


# ------------------------------------------------------------------ invariants

def check_invariants(p: OraclePool):
    live = [s for s in p.states.values() if s.status == "ACTIVE"]
    count = np.zeros(p.P, dtype=np.int64)
    for s in live:
        assert len(set(s.table)) == len(s.table)
        assert len(s.table) == -(-s.n // p.shape.block_size)
        for b in s.table:
            count[b] += 1
    assert np.array_equal(count, p.refcount)
    free = [int(p.ring[i % p.P]) for i in range(p.head, p.tail)]
    assert len(set(free)) == len(free)
    used = set(np.nonzero(count)[0].tolist())
    assert used.isdisjoint(free)
    assert used | set(free) == set(range(p.P))


ops = st.lists(st.tuples(st.integers(0, 7), st.integers(0, 1000), st.integers(0, 1000),
                         st.integers(1, 9)), min_size=1, max_size=25)


@settings(max_examples=300, deadline=None)
@given(ops)
def test_random_sequences_keep_invariants(seq):
    p = meta_pool(P=24, B=2, max_pos=40, max_states=8)
    for op, a, b, c in seq:
        live = [s.sid for s in p.states.values() if s.status == "ACTIVE"]
        try:
            if op == 0 or not live:
                p.materialize(None, T=c)
            elif op == 1:
                p.fork(live[a % len(live)], 1 + b % 3)
            elif op == 2:
                k = 1 + b % len(live)
                p.attend(live[a % len(live):][:k] or live[:1], T=c)
            elif op == 3:
                segs = []
                for j in range(1 + b % 3):
                    s = live[(a + j) % len(live)]
                    n = p.info(s)[1]
                    lo = (a * (j + 1)) % n
                    segs.append((s, lo, min(n, lo + 1 + c)))
                p.compose(segs)
            elif op == 4:
                s = live[a % len(live)]
                nb = p.info(s)[2]
                hdr, _ = p.pack(s, b % nb, nb)
                p.unpack(hdr)
            elif op == 5:
                p.evict(a % 25, 0.0, 0.0, 1.0)
            elif op == 6:
                p.evict_truncate(a % 25, 0.0, 0.0, 1.0)
            else:
                p.release(live[a % len(live)])
        except OracleError as e:
            assert e.status in (Status.OOM, Status.CAPACITY)
        check_invariants(p)


# ------------------------------------------------------------------ numerics

def num_pool(P=64, B=4, L=2, d=16, hq=4, hkv=2, dh=8, base=10000.0, order=None):
    shape = PoolShape(L, d, hq, hkv, dh, B, "f32", rope_base=base, max_pos=256, max_states=32)
    w = [RNG.standard_normal(((hq + 2 * hkv) * dh, d)) / np.sqrt(d) for _ in range(L)]
    return OraclePool(shape, P, init_free_order=order, weights=w), w


def reference_outputs(pool, x, pos0=0):
    """Recompute: materialize x in a fresh pool with the same weights."""
    q = OraclePool(pool.shape, 256, weights=pool.weights)
    _, o = q.materialize(x, pos0=pos0)
    return o


def test_fork_append_equals_recompute():
    p, _ = num_pool()
    ctx = RNG.standard_normal((13, 16))                 # 13 mod 4 != 0: partial tail
    suf = [RNG.standard_normal((6, 16)) for _ in range(3)]
    root, _ = p.materialize(ctx)
    kids = p.fork(root, 3)
    o = p.attend(kids, np.stack(suf))
    for i in range(3):
        ref = reference_outputs(p, np.concatenate([ctx, suf[i]]))
        np.testing.assert_allclose(o[:, i], ref[:, 13:], atol=1e-12)
    # the parent never sees a child's tokens
    x2 = RNG.standard_normal((2, 16))
    o2 = p.attend([root], x2[None])
    ref = reference_outputs(p, np.concatenate([ctx, x2]))
    np.testing.assert_allclose(o2[:, 0], ref[:, 13:], atol=1e-12)


def test_decode_steps_equal_one_append():
    p, _ = num_pool()
    ctx = RNG.standard_normal((9, 16))
    dec = RNG.standard_normal((7, 16))
    a, _ = p.materialize(ctx)
    b, = p.fork(a, 1)
    outs = [p.attend([a], dec[i:i + 1][None])[:, 0, 0] for i in range(7)]
    o_b = p.attend([b], dec[None])[:, 0]
    np.testing.assert_allclose(np.stack(outs, axis=1), o_b, atol=1e-12)


def test_compose_equals_recompute_of_concatenation():
    p, _ = num_pool(P=96)
    ctx = RNG.standard_normal((16, 16))
    suf = [RNG.standard_normal((5, 16)) for _ in range(2)]
    root, _ = p.materialize(ctx)
    k1, k2 = p.fork(root, 2)
    p.attend([k1, k2], np.stack(suf))
    # [root 0..16 | k1 16..21 | k2 16..21 moved to 21..26]
    c = p.compose([(root, 0, 16), (k1, 16, 21), (k2, 16, 21)])
    full = np.concatenate([ctx, suf[0], suf[1]])
    nxt = RNG.standard_normal((3, 16))
    o = p.attend([c], nxt[None])
    ref = reference_outputs(p, np.concatenate([full, nxt]))
    np.testing.assert_allclose(o[:, 0], ref[:, 26:], atol=1e-11)
    # segments taken out of order and from the middle of states
    d = p.compose([(k2, 16, 21), (root, 3, 11)])
    assert p.info(d)[:2] == (16, 13)          # starts at k2's token 16's position
    seg = np.concatenate([suf[1], ctx[3:11]])
    o = p.attend([d], nxt[None])
    q = OraclePool(p.shape, 256, weights=p.weights)
    s, _ = q.materialize(seg, pos0=16)
    ref = q.attend([s], nxt[None])
    np.testing.assert_allclose(o, ref, atol=1e-11)


def test_pack_unpack_round_trip_permuted():
    p, w = num_pool(P=40)
    order = RNG.permutation(40)
    q = OraclePool(p.shape, 40, init_free_order=order, weights=w)
    ctx = RNG.standard_normal((21, 16))
    s, _ = p.materialize(ctx)
    hdr, buf = p.pack(s, 0, 6)
    # invalid slots of the last block are zero
    assert np.all(buf[-1, :, :, :, 1:] == 0)
    u = q.unpack(hdr, buf)
    assert q.table(u) == [int(x) for x in order[:6]]
    hdr2, buf2 = q.pack(u, 0, 6)
    assert np.array_equal(buf2, buf)
    for layer in range(2):
        for a, b in zip(p.state_kv(s, layer), q.state_kv(u, layer)):
            assert np.array_equal(a, b)
    # partial range: blocks [2, 6)
    hdr3, buf3 = p.pack(s, 2, 6)
    assert hdr3["pos_begin"] == 8 and hdr3["n_tokens"] == 13
    assert np.array_equal(buf3, buf[2:])
    # attention after transfer equals attention on the source
    x = RNG.standard_normal((1, 2, 16))
    s2, = p.fork(s, 1)
    np.testing.assert_allclose(q.attend([u], x), p.attend([s2], x), atol=1e-12)


def test_cow_leaves_siblings_intact():
    p, _ = num_pool()
    ctx = RNG.standard_normal((10, 16))
    a, _ = p.materialize(ctx)
    before = [p.state_kv(a, layer) for layer in range(2)]
    b, c = p.fork(a, 2)
    p.attend([b], RNG.standard_normal((1, 3, 16)))
    p.attend([c], RNG.standard_normal((1, 1, 16)))
    for layer in range(2):
        k, v = p.state_kv(a, layer)
        assert np.array_equal(k, before[layer][0]) and np.array_equal(v, before[layer][1])


def test_materialize_attention_is_causal_gqa_on_projected_rows():
    p, w = num_pool(L=1)
    x = RNG.standard_normal((11, 16))
    s, o = p.materialize(x, pos0=5)
    from oracle import apply_rope, project_qkv
    q, k, v = project_qkv(x, w[0], 4, 2, 8)
    pos = 5 + np.arange(11)
    ref = causal_gqa_attention(apply_rope(q, pos, 1e4), apply_rope(k, pos, 1e4), v, pos, pos)
    np.testing.assert_allclose(o[0], ref.transpose(1, 0, 2).reshape(11, 32), atol=1e-13)
    kk, vv = p.state_kv(s, 0)
    np.testing.assert_allclose(kk, apply_rope(k, pos, 1e4), atol=1e-14)
    np.testing.assert_array_equal(vv, v)
