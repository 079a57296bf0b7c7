"""kv_attend_noalloc: the allocation-free variant of kv_attend (its work area
is a fixed device array) against kv_attend itself, through the C ABI.

Two forks of one context receive the same appends, one through each entry
point: outputs and the K/V each call writes must be identical bit for bit
(same kernels, same arithmetic), on consecutive calls whose second is
smaller than the first (the array keeps the first call's contents), on a call
that runs in two layer groups in the array, and on batched decode.  A call of
which not even one layer fits is refused and changes nothing, and a pool
with no scratch area of its own still attends through the fixed array.
"""
import pytest
import torch

import synth
from paper_2607_10987_amd import kvstate as kv

pytestmark = pytest.mark.gpu


def _state_kv(pool, h):
    table = kv.kv_read_block_table(pool.h, h)
    n = kv.kv_state_info(pool.h, h)["n_tokens"]
    blocks = pool.blocks_view()[table]                  # [nb, L, 2, Hkv, B, dh]
    nb, L, _, hkv, B, dh = blocks.shape
    return blocks.permute(1, 2, 3, 0, 4, 5).reshape(L, 2, hkv, nb * B, dh)[:, :, :, :n]


def test_noalloc_attend_matches_attend(gpu_available):
    base = synth.LLAMA8B_SHAPE
    L, d, hq, hkv, dh, B = 2, base.d_model, base.n_q_heads, base.n_kv_heads, base.head_dim, 16
    cols = (hq + 2 * hkv) * dh
    cfg = kv.make_cfg(L, d, hq, hkv, dh, B, "bf16", 16384, 16)
    w = torch.empty((L, cols, d), dtype=torch.bfloat16, device="cuda")
    for layer in range(L):
        w[layer] = synth.normal_torch(synth.w_key(0, "noalloc", layer), (cols, d),
                                      1.0 / d ** 0.5, "bf16", "cuda")
    big = 4200   # query rows of one layer: 4200 x 4096 x 2 bytes > half of the 64 MiB array
    pool = kv.Pool(cfg, 1800, kv.kv_scratch_bytes(cfg, 2 * big, 4, 16384))
    pool.set_weights(w, cols * d)
    h = pool.h

    def x(rows, tag):
        return synth.normal_torch(synth.x_key(0, "noalloc", tag), (rows, d), 1.0, "bf16", "cuda")

    ctx = 77                                                   # a partial tail: copy-on-write
    o = torch.empty((L, ctx, hq * dh), dtype=torch.bfloat16, device="cuda")
    root = kv.kv_materialize(h, x(ctx, 0), ctx, 0, o)
    a, b = kv.kv_fork(h, root, 2)

    def both(sa, sb, T, tag):
        n = len(sa)
        xi = x(n * T, tag)
        oa = torch.empty((L, n, T, hq * dh), dtype=torch.bfloat16, device="cuda")
        ob = torch.full_like(oa, float("nan"))
        kv.kv_attend(h, sa, xi, T, oa)
        kv.kv_attend_noalloc(h, sb, xi, T, ob)
        torch.cuda.synchronize()
        kv.kv_sync(h)
        assert torch.equal(oa, ob), f"outputs differ (T={T}, batch {n})"
        for p, q in zip(sa, sb):
            assert torch.equal(_state_kv(pool, p), _state_kv(pool, q)), "K/V differ"
            ip, iq = kv.kv_state_info(h, p), kv.kv_state_info(h, q)
            assert (ip["n_tokens"], ip["n_blocks"]) == (iq["n_tokens"], iq["n_blocks"])

    both([a], [b], 300, 1)          # 300 rows: both layers in one group
    both([a], [b], 1, 2)            # a smaller call after it: decode over 378 keys
    both([a], [b], big, 3)          # two layer groups in the fixed array
    both([a], [b], 1, 4)
    c1, c2, c3 = kv.kv_fork(h, a, 3)
    d1, d2, d3 = kv.kv_fork(h, b, 3)
    both([c1, c2, c3, a], [d1, d2, d3, b], 1, 5)   # batched decode over 4579 keys
    both([c2], [d2], 1, 6)

    # one layer of this call does not fit in the array: refused, nothing changed
    huge = 8200                                    # 8200 x 4096 x 2 bytes > 64 MiB
    before = kv.kv_pool_counts(h)
    info = kv.kv_state_info(h, b)
    with pytest.raises(kv.KVError) as e:
        kv.kv_attend_noalloc(h, [b], x(huge, 7),
                             huge, torch.empty((L, 1, huge, hq * dh), dtype=torch.bfloat16,
                                               device="cuda"))
    assert e.value.status == kv.KV_ERR_BUFSIZE
    assert kv.kv_pool_counts(h) == before and kv.kv_state_info(h, b) == info
    pool.close()

    # a pool without a scratch area of its own
    bare = kv.Pool(cfg, 64, 0)
    bare.set_weights(w, cols * d)
    o = torch.empty((L, 40, hq * dh), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(kv.KVError) as e:
        kv.kv_materialize(bare.h, x(40, 8), 40, 0, o)
    assert e.value.status == kv.KV_ERR_BUFSIZE
    pool2 = kv.Pool(cfg, 64, kv.kv_scratch_bytes(cfg, 40, 2, 256))
    pool2.set_weights(w, cols * d)
    r2 = kv.kv_materialize(pool2.h, x(40, 8), 40, 0, o)
    pack = torch.empty(3 * pool2.pool_t.numel() // 64, dtype=torch.uint8, device="cuda")
    hdr = kv.kv_pack(pool2.h, r2, 0, 3, pack)
    r = kv.kv_unpack(bare.h, hdr, pack)
    ob = torch.empty((L, 1, 1, hq * dh), dtype=torch.bfloat16, device="cuda")
    oa = torch.empty_like(ob)
    with pytest.raises(kv.KVError) as e:
        kv.kv_attend(bare.h, [r], x(1, 9), 1, ob)
    assert e.value.status == kv.KV_ERR_BUFSIZE
    kv.kv_attend_noalloc(bare.h, [r], x(1, 9), 1, ob)
    kv.kv_attend(pool2.h, [r2], x(1, 9), 1, oa)
    torch.cuda.synchronize()
    assert torch.equal(oa, ob)
    bare.close()
    pool2.close()
