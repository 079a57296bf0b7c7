"""GPU parity of the paths the workload-shaped twin runs do not reach.

Each test mirrors its calls on the float64 oracle through ``Twin`` (tables,
refcounts, ring, eviction score terms exact after every call; outputs and K/V
within the stated tolerances; re-rotated keys within one rounding of the
oracle's re-rotation of the stored source keys):

* KV-Evict's general score alpha*reuse - beta*size - gamma*age, with ties;
* layer groups: a scratch area smaller than a call needs for all layers, so
  that the call runs layer group by layer group (prefill, append, batched
  decode with its work plan reused across groups);
* decode batches beyond 64 query vectors per KV head (four wavefronts per
  unit, query slices) and contexts of more than 256 key chunks;
* a Llama-scale RoPE base (5e5) at positions near 35k and compositions that
  shift segments by about +-30k positions;
* the projection kernels for d_model values and row counts the 8B / 70B
  shapes never produce, and the bf16 compose copy for a head dimension that
  is not a power of two.
"""
import numpy as np
import pytest

import synth
from paper_2607_10987_amd import kvstate as kv
from twin import Twin

pytestmark = pytest.mark.gpu


def shape8b(L=2, d=None, hq=None, hkv=None, dh=None, B=None, rope_base=10000.0, name="8b"):
    b = synth.LLAMA8B_SHAPE
    return synth.ModelShape(name, L, d or b.d_model, hq or b.n_q_heads, hkv or b.n_kv_heads,
                            dh or b.head_dim, B or b.block_size, "bf16", rope_base)


def align256(n):
    return -(-n // 256) * 256


def pin(tw, h, on=True):
    kv.kv_pin(tw.gpu.h, h, 1 if on else 0)
    tw.orc.pin(tw.sid[h], on)


@pytest.mark.parametrize("abg", [(1.0, 0.0, 0.0), (0.0, 1.0, 0.0), (0.5, 0.25, 1.0)])
def test_eviction_scores_on_device(gpu_available, abg):
    """States with different reuse counts, sizes and ages; two states tie on
    reuse and size (broken by state id) and one is pinned.  The device must
    release the same states in the same order (the free ring's tail order
    shows it), then truncate with the same score, then evict the rest."""
    a, b, g = abg
    shape = synth.ModelShape("evs", 1, 32, 2, 1, 16, 2, "f32")
    tw = Twin(shape, n_blocks=64, max_pos=64, max_states=16, wl="evs", check_kv=False)
    r = tw.materialize(6)                   # 3 blocks
    kids = tw.fork(r, 3)                    # the root's reuse count becomes 1
    tw.attend([kids[0]], 3)                 # 9 tokens, 5 blocks
    tw.attend([kids[1], kids[2]], 1)        # 7 tokens, 4 blocks each
    tw.attend([kids[1]], 2)                 # reuse 2
    m = tw.materialize(4)
    tw.pack(m, 0, 2)                        # a pack source counts as an input
    m2 = tw.materialize(3)
    m3 = tw.materialize(3)                  # ties with m2 on reuse and size
    pin(tw, kids[2])
    tw.attend([m2], 1)                      # m2 is touched again: ages differ
    alloc = tw.orc.allocated()
    tw.evict(alloc - 5, a, b, g)
    tw.evict_truncate(max(tw.orc.allocated() - 3, 0), a, b, g)
    tw.evict(0, a, b, g)
    live = [h for h, s in tw.sid.items() if tw.orc.states[s].status == "ACTIVE"]
    assert live == [kids[2]], "only the pinned state survives"
    tw.close()


@pytest.mark.parametrize("per_group", [1, 3])
def test_layer_groups_prefill_and_append(gpu_available, per_group):
    """The scratch area holds the query rows of `per_group` of the 4 layers of
    a 48-row call: materialize, appends and a compose + append run layer
    group by layer group (groups that start past layer 0; a ragged last group
    of one layer for 3), checked against the oracle.  The projection and
    attention launch counts show the grouping."""
    shape = shape8b(L=4)
    M = 48
    q_layer = align256(M * shape.n_q_heads * shape.head_dim * 2)
    scratch = per_group * q_layer + q_layer // 2
    tw = Twin(shape, n_blocks=48, max_pos=256, max_states=10, wl="lgroups",
              scratch_bytes=scratch)
    h = tw.gpu.h
    groups = -(-shape.n_layers // per_group)
    kv.kv_profile_enable(h, True)
    root = tw.materialize(M)
    prof = kv.kv_profile_read(h)
    assert prof["qkv"][0] == groups and prof["attn"][0] == groups, prof
    kids = tw.fork(root, 3)
    tw.attend(kids, 16)                     # 3 x 16 rows
    prof = kv.kv_profile_read(h)
    assert prof["qkv"][0] == groups and prof["attn"][0] == groups, prof
    tw.attend(kids[:2], 24)                 # 2 x 24 rows over 64 cached keys
    c = tw.compose([(root, 0, 48), (kids[0], 48, 88), (kids[1], 48, 70)])
    tw.attend([c], 40)
    tw.attend([c, kids[2]], 1)              # decode: all layers fit at once
    tw.close()


@pytest.mark.parametrize("per_group", [1, 3])
def test_layer_groups_batched_decode(gpu_available, per_group):
    """A 2100-token context (a seeded payload unpacked into the pool) forked
    to 16 agents; batch-16 decode steps with a scratch area that holds the
    query rows and split-key partials of only `per_group` of the 4 layers
    (plus the work plan), so the plan computed for the first group is reused
    by the others."""
    shape = shape8b(L=4)
    A, n_ctx = 16, 2100
    chunks = -(-(n_ctx + 3) // 1024)          # keys per decode call <= n_ctx + 3
    q_layer = align256(A * shape.n_q_heads * shape.head_dim * 2)
    part_layer = align256(A * shape.n_q_heads * chunks * (shape.head_dim + 4) * 4)
    plan = align256(chunks * A * (16 + 64 * 4)) + align256(chunks * 4)   # unit records, counts
    scratch = plan + per_group * (q_layer + part_layer) + q_layer // 2
    tw = Twin(shape, n_blocks=200, max_pos=2304, max_states=A + 4, wl="lgdec",
              scratch_bytes=scratch)
    nb = -(-n_ctx // shape.block_size)
    hdr, ohdr, buf, pay = tw.synthetic_transfer(nb, n_ctx, 0, tag=1)
    root = tw.unpack(hdr, ohdr, buf, pay)
    kids = tw.fork(root, A)
    h = tw.gpu.h
    groups = -(-shape.n_layers // per_group)
    kv.kv_profile_enable(h, True)
    for _ in range(3):
        tw.attend(kids, 1)                  # the first step copies the shared tail
        prof = kv.kv_profile_read(h)
        assert prof["qkv_decode"][0] == groups and prof["merge"][0] == groups, prof
    tw.attend(kids[4:9], 1)
    tw.close()


def test_decode_query_slices(gpu_available):
    """Decode batches with more than 64 query vectors per KV head stay on the
    MFMA decode path (the merge kernel runs): 32 agents x 4 query heads at
    the 8B head shape (128 vectors: four wavefronts of 32 share a unit's
    stages), 64 agents x 4 query heads and 17 agents x 8 query heads at the
    70B head shape (more than 128: query slices of 64 vectors)."""
    shape = shape8b(L=2)
    tw = Twin(shape, n_blocks=260, max_pos=1200, max_states=70, wl="slices", check_kv=False)
    hdr, ohdr, buf, pay = tw.synthetic_transfer(66, 1050, 0, tag=2)   # 1050 keys: 2 chunks
    root = tw.unpack(hdr, ohdr, buf, pay)
    kids = tw.fork(root, 32)
    h = tw.gpu.h
    kv.kv_profile_enable(h, True)
    tw.attend(kids, 1)                      # copies the shared partial tail
    tw.attend(kids, 1)
    assert kv.kv_profile_read(h)["merge"][0] == 2
    more = tw.fork(root, 32)
    tw.attend(kids + more, 1)               # 64 agents: 256 query vectors
    tw.attend(kids[::3] + more[1::2], 1)    # mixed histories
    assert kv.kv_profile_read(h)["merge"][0] == 2
    tw.close()

    base = synth.LLAMA70B_SHAPE
    shape = synth.ModelShape("70b-l2", 2, base.d_model, base.n_q_heads, base.n_kv_heads,
                             base.head_dim, base.block_size, "bf16")
    tw = Twin(shape, n_blocks=80, max_pos=512, max_states=20, wl="slices70", check_kv=False)
    root = tw.materialize(300)
    kids = tw.fork(root, 17)
    kv.kv_profile_enable(tw.gpu.h, True)
    tw.attend(kids, 1)
    tw.attend(kids, 1)
    assert kv.kv_profile_read(tw.gpu.h)["merge"][0] == 2
    tw.close()


def test_rope_base_5e5_far_positions(gpu_available):
    """RoPE base 5e5 (the Llama-3 value) with positions up to ~35k: a context
    placed at 34600 through pos0 with appends and decode steps, and
    compositions that shift a segment by +30200 and by -29960 positions
    (re-rotated keys within one rounding of the oracle's re-rotation of the
    stored keys), followed by decode over the composed states."""
    shape = shape8b(L=2, rope_base=500000.0, name="8b-5e5")
    tw = Twin(shape, n_blocks=150, max_pos=35072, max_states=12, wl="rope5e5")
    far = tw.materialize(300, pos0=34600)        # positions 34600 .. 34899
    kids = tw.fork(far, 2)
    tw.attend(kids, 40)
    for _ in range(2):
        tw.attend(kids, 1)                       # positions up to 34941
    seg = tw.materialize(200, pos0=30000)        # 30000 .. 30199
    near = tw.materialize(100)                   # 0 .. 99
    c1 = tw.compose([(seg, 0, 200), (near, 0, 100)])     # near moves by +30200
    tw.attend([c1], 1)
    c2 = tw.compose([(near, 10, 90), (seg, 50, 150)])    # seg moves by 90 - 30050 = -29960
    tw.attend([c2], 1)
    c3 = tw.compose([(near, 0, 100), (kids[0], 0, 342)])  # a far context moves by -34500
    tw.attend([c3, c1], 2)
    tw.close()


@pytest.mark.parametrize("d,rows", [(2560, 16), (10752, 16), (2304, 24), (2112, 16)])
def test_projection_variants(gpu_available, d, rows):
    """Decode-size projections the 8B / 70B shapes do not produce (8 query / 2
    KV heads of 128, 2 layers): d_model 2560 with 16 token rows (token rows
    staged in LDS, weights loaded into registers), 10752 with 16 rows (token
    rows read from global memory), 2304 with 24 rows and 2112 (not a multiple
    of 256) with 16 rows (the 128-channel x 32-token MFMA tile).  Also a
    prefill (k_qkv_dl) and decode steps at each d_model."""
    shape = shape8b(L=2, d=d, hq=8, hkv=2, name=f"d{d}")
    tw = Twin(shape, n_blocks=48, max_pos=256, max_states=8, wl=f"proj{d}", scratch_tokens=64)
    root = tw.materialize(40)
    kids = tw.fork(root, rows // 8)
    tw.attend(kids, 8)                           # `rows` token rows
    tw.attend(kids, 1)
    tw.attend([root], 2)
    tw.close()


def test_compose_bf16_head_dim_96(gpu_available):
    """bf16 with head_dim 96 (not a power of two): the general compose copy
    (keys re-rotated by shifts of -60 and +32 positions), portable
    projection and attention kernels, pack / unpack of the result."""
    shape = synth.ModelShape("dh96", 2, 256, 4, 2, 96, 16, "bf16")
    tw = Twin(shape, n_blocks=64, max_pos=512, wl="dh96")
    a = tw.materialize(40)
    b = tw.materialize(30, pos0=100)
    kids = tw.fork(a, 2)
    tw.attend(kids, 5)
    c = tw.compose([(a, 0, 40), (b, 0, 30), (kids[1], 38, 45)])
    tw.attend([c], 1)
    nb = kv.kv_state_info(tw.gpu.h, c)["n_blocks"]
    hdr, ohdr, buf, pay = tw.pack(c, 0, nb)
    tw.unpack(hdr, ohdr, buf, pay, rerotated_from=c)
    tw.close()


def test_decode_many_chunks(gpu_available):
    """Decode over a 139990-token context (a seeded payload unpacked into the
    pool; one KV head of 128 channels, so the oracle stays small): a batch of
    one cuts it into 274 chunks of 512 keys, more than the persistent kernel
    indexes, so the per-unit stream kernel runs; batches of 2 and 3 forked
    agents cut it into 137 chunks of 1024 keys, which the persistent kernel
    finds through its unit counts in three registers per lane."""
    shape = synth.ModelShape("long", 2, 256, 4, 1, 128, 16, "bf16")
    n_ctx = 139990
    nb = -(-n_ctx // shape.block_size)
    tw = Twin(shape, n_blocks=nb + 64, max_pos=n_ctx + 64, max_states=8, wl="long",
              check_kv=False)
    hdr, ohdr, buf, pay = tw.synthetic_transfer(nb, n_ctx, 0, tag=3)
    root = tw.unpack(hdr, ohdr, buf, pay)
    tw.attend([root], 1)                    # 139991 keys, batch 1: 274 chunks
    kids = tw.fork(root, 3)
    tw.attend(kids[:2], 1)                  # batch 2: 137 chunks
    tw.attend(kids, 1)                      # mixed histories, batch 3
    tw.close()
