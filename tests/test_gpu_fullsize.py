"""Parity at the benchmark's full workload sizes, in the launch configuration
the benchmark times (all layers, the workload's batch and lengths).

Tables, refcounts and the ring are compared exactly against the oracle's
metadata model after every phase; values are compared for the first and last
layer, every KV head and sampled token rows (first, last, block boundaries,
random), each evaluated by the float64 oracle; byte-level properties (pack =
gather of the pool, composed values = source values, unpack = copy) are
checked on the whole state.
"""
import numpy as np
import pytest
import torch

import synth
from fullsize import MetaTwin, close, close_rerotated, ref_kv, ref_rows, sample_rows, to64
from oracle import rerotate
from paper_2607_10987_amd import kvstate as kv
from twin import close_one_rounding

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def test_fork4_8b_full_size(gpu_available):
    wl = synth.WORKLOADS["fork4-8b"]
    s = wl.shape
    ctx, A, suf, ndec = wl.context, wl.agents, wl.suffix, 3
    B, L, d = s.block_size, s.n_layers, s.d_model
    HD = s.n_q_heads * s.head_dim
    cont = suf + ndec
    n_comp = ctx + A * cont
    max_pos = n_comp + 64
    n_blocks = ctx // B + 1 + A * (cont // B + 2) + 2 * (n_comp // B + 2) + 64
    mt = MetaTwin(wl, n_blocks, max_pos, scratch_tokens=max(ctx, A * suf), batch=A)
    kx, ks, kd = (synth.x_key(0, wl.name, i) for i in range(3))

    x_ctx = mt.x(kx, (ctx, d))
    o_ctx = torch.empty((L, ctx, HD), dtype=torch.bfloat16, device="cuda")
    root = kv.kv_materialize(mt.h, x_ctx, ctx, 0, o_ctx)
    mt.sid[root] = mt.orc.materialize(None, T=ctx)[0]
    mt.check_meta()
    kids = kv.kv_fork(mt.h, root, A)
    for a, b in zip(kids, mt.orc.fork(mt.sid[root], A)):
        mt.sid[a] = b
    x_suf = mt.x(ks, (A, suf, d))
    o_suf = torch.empty((L, A, suf, HD), dtype=torch.bfloat16, device="cuda")
    kv.kv_attend(mt.h, kids, x_suf, suf, o_suf)
    mt.orc.attend([mt.sid[k] for k in kids], T=suf)
    x_dec = mt.x(kd, (ndec, A, 1, d))
    o_dec = torch.empty((ndec, L, A, 1, HD), dtype=torch.bfloat16, device="cuda")
    for i in range(ndec):
        kv.kv_attend(mt.h, kids, x_dec[i], 1, o_dec[i])
        mt.orc.attend([mt.sid[k] for k in kids], T=1)
    mt.check_meta()
    segs = [(root, 0, ctx)] + [(k, ctx, ctx + cont) for k in kids]
    c = kv.kv_compose(mt.h, segs)
    mt.sid[c] = mt.orc.compose([(mt.sid[a], b, e) for a, b, e in segs])
    nb = kv.kv_state_info(mt.h, c)["n_blocks"]
    buf = torch.empty(nb * s.block_bytes, dtype=torch.uint8, device="cuda")
    hdr = kv.kv_pack(mt.h, c, 0, nb, buf)
    u = kv.kv_unpack(mt.h, hdr, buf)
    ohdr, _ = mt.orc.pack(mt.sid[c], 0, nb)
    mt.sid[u] = mt.orc.unpack(ohdr)
    mt.check_meta()

    # pack = gather of the pool in logical order, slots after the last token zeroed
    table = kv.kv_read_block_table(mt.h, c)
    expect = mt.pool.blocks_view()[table].clone()
    expect[-1, :, :, :, n_comp - (nb - 1) * B:] = 0
    assert torch.equal(buf.view(torch.bfloat16).view(expect.shape), expect)

    xc64 = mt.x64(kx, (ctx, d))
    xs64 = mt.x64(ks, (A, suf, d))
    xd64 = mt.x64(kd, (ndec, A, 1, d))
    rng = np.random.default_rng(0)
    for layer in (0, L - 1):
        k_ctx, v_ctx = ref_kv(mt, layer, xc64, np.arange(ctx))
        kr, vr = mt.state_kv(root, layer)
        close(to64(kr), k_ctx, "bf16", f"root K layer {layer}")
        close(to64(vr), v_ctx, "bf16", f"root V layer {layer}")
        rows = sample_rows(ctx, B, 64, rng)
        ref = ref_rows(mt, layer, xc64[rows], rows, k_ctx, v_ctx, np.arange(ctx), rows + 1)
        close(to64(o_ctx[layer, rows]), ref, "bf16", f"materialize output layer {layer}")
        comp_k, comp_v = [k_ctx], [v_ctx]
        for j, kid in enumerate(kids):
            xa = np.concatenate([xs64[j], xd64[:, j, 0]])
            k_a, v_a = ref_kv(mt, layer, xa, ctx + np.arange(cont))
            kk = np.concatenate([k_ctx, k_a], axis=1)
            vv = np.concatenate([v_ctx, v_a], axis=1)
            kg, vg = mt.state_kv(kid, layer)
            close(to64(kg), kk, "bf16", f"agent {j} K")
            close(to64(vg), vv, "bf16", f"agent {j} V")
            r = sample_rows(suf, B, 16, rng)
            ref = ref_rows(mt, layer, xs64[j][r], ctx + r, kk, vv, np.arange(ctx + cont),
                           ctx + r + 1)
            close(to64(o_suf[layer, j, r]), ref, "bf16", f"append output agent {j}")
            tq = ctx + suf + np.arange(ndec)
            ref = ref_rows(mt, layer, xd64[:, j, 0], tq, kk, vv, np.arange(ctx + cont), tq + 1)
            close(to64(o_dec[:, layer, j, 0]), ref, "bf16", f"decode output agent {j}")
            kn, vn = ref_kv(mt, layer, xa, ctx + j * cont + np.arange(cont))
            comp_k.append(kn)
            comp_v.append(vn)
            kc_j, vc_j = (t[:, ctx + j * cont:ctx + (j + 1) * cont] for t in mt.state_kv(c, layer))
            assert torch.equal(vc_j, vg[:, ctx:]), "composed values must be the source bytes"
            # keys: the oracle's re-rotation of the agent's stored keys (one rounding)
            if j == 0:
                assert torch.equal(kc_j, kg[:, ctx:]), "unshifted keys must be copied"
            else:
                close_one_rounding(to64(kc_j), rerotate(to64(kg[:, ctx:]), j * cont, s.rope_base),
                                   "bf16", f"re-rotated keys of agent {j}")
        kc, vc = mt.state_kv(c, layer)
        assert torch.equal(kc[:, :ctx], kr) and torch.equal(vc[:, :ctx], vr), \
            "the context's blocks are aliased"
        close_rerotated(to64(kc), np.concatenate(comp_k, axis=1), "bf16", "composed K")
        close(to64(vc), np.concatenate(comp_v, axis=1), "bf16", "composed V")
        ku, vu = mt.state_kv(u, layer)
        assert torch.equal(ku, kc) and torch.equal(vu, vc), "unpack must restore the bytes"

    assert kv.kv_evict(mt.h, 0) == mt.orc.evict(0)
    mt.check_meta()
    mt.pool.close()


def _sync_ids(mt, gpu_handles, oracle_ids):
    for a, b in zip(gpu_handles, oracle_ids):
        mt.sid[a] = b


def test_fanout16_8b_full_size(gpu_available):
    """32768-token context, 16 agents x 1024-token suffixes, batch-16 decode over
    the shared blocks, then 10 rounds of LRU churn freeing 25% of the blocks."""
    wl = synth.WORKLOADS["fanout16-8b"]
    s = wl.shape
    ctx, A, suf, ndec = wl.context, wl.agents, wl.suffix, 2
    B, L, d = s.block_size, s.n_layers, s.d_model
    HD = s.n_q_heads * s.head_dim
    max_pos = ctx + suf + ndec + 64
    n_blocks = ctx // B + A * (suf // B + 2) + 64
    mt = MetaTwin(wl, n_blocks, max_pos, max_states=40, scratch_tokens=max(ctx, A * suf),
                  batch=A)
    kx, ks, kd = (synth.x_key(0, wl.name, i) for i in range(3))
    o_ctx = torch.empty((L, ctx, HD), dtype=torch.bfloat16, device="cuda")
    root = kv.kv_materialize(mt.h, mt.x(kx, (ctx, d)), ctx, 0, o_ctx)
    mt.sid[root] = mt.orc.materialize(None, T=ctx)[0]
    del o_ctx
    kids = kv.kv_fork(mt.h, root, A)
    _sync_ids(mt, kids, mt.orc.fork(mt.sid[root], A))
    o_suf = torch.empty((L, A, suf, HD), dtype=torch.bfloat16, device="cuda")
    kv.kv_attend(mt.h, kids, mt.x(ks, (A, suf, d)), suf, o_suf)
    mt.orc.attend([mt.sid[k] for k in kids], T=suf)
    x_dec = mt.x(kd, (ndec, A, 1, d))
    o_dec = torch.empty((ndec, L, A, 1, HD), dtype=torch.bfloat16, device="cuda")
    for i in range(ndec):
        kv.kv_attend(mt.h, kids, x_dec[i], 1, o_dec[i])
        mt.orc.attend([mt.sid[k] for k in kids], T=1)
    mt.check_meta()
    # exact memory claim: the fork grows with the continuations, not the prefix
    assert mt.orc.allocated() == ctx // B + A * ((suf + ndec + B - 1) // B)

    xc64 = mt.x64(kx, (ctx, d))
    xs64 = mt.x64(ks, (A, suf, d))
    xd64 = mt.x64(kd, (ndec, A, 1, d))
    rng = np.random.default_rng(1)
    for layer in (0, L - 1):
        k_ctx, v_ctx = ref_kv(mt, layer, xc64, np.arange(ctx))
        kr, vr = mt.state_kv(root, layer)
        tok = sample_rows(ctx, B, 512, rng)
        close(to64(kr[:, tok]), k_ctx[:, tok], "bf16", "root K (sampled tokens)")
        close(to64(vr[:, tok]), v_ctx[:, tok], "bf16", "root V (sampled tokens)")
        for j in range(A):
            xa = np.concatenate([xs64[j], xd64[:, j, 0]])
            k_a, v_a = ref_kv(mt, layer, xa, ctx + np.arange(suf + ndec))
            kk = np.concatenate([k_ctx, k_a], axis=1)
            vv = np.concatenate([v_ctx, v_a], axis=1)
            tq = ctx + suf + np.arange(ndec)
            ref = ref_rows(mt, layer, xd64[:, j, 0], tq, kk, vv, np.arange(ctx + suf + ndec),
                           tq + 1)
            close(to64(o_dec[:, layer, j, 0]), ref, "bf16", f"batched decode agent {j}")
            if j < 2:
                r = sample_rows(suf, B, 8, rng)
                ref = ref_rows(mt, layer, xs64[j][r], ctx + r, kk, vv,
                               np.arange(ctx + suf + ndec), ctx + r + 1)
                close(to64(o_suf[layer, j, r]), ref, "bf16", f"append output agent {j}")

    # LRU churn: the root is pinned; each round frees 25% of the allocated
    # blocks (the 12 least recently used agents), then 12 new agents refill
    kv.kv_pin(mt.h, root, 1)
    mt.orc.pin(mt.sid[root], True)
    x_ref = mt.x(ks, (12, suf, d))
    o_ref = torch.empty((L, 12, suf, HD), dtype=torch.bfloat16, device="cuda")
    for rnd in range(wl.extra["evict_rounds"]):
        alloc = mt.orc.allocated()
        budget = int(alloc * (1 - wl.extra["evict_frac"]))
        n = kv.kv_evict(mt.h, budget, 0.0, 0.0, 1.0)
        assert n == mt.orc.evict(budget, 0.0, 0.0, 1.0) == 12
        assert mt.orc.allocated() <= budget
        mt.check_meta()
        new = kv.kv_fork(mt.h, root, 12)
        _sync_ids(mt, new, mt.orc.fork(mt.sid[root], 12))
        kv.kv_attend(mt.h, new, x_ref, suf, o_ref)
        mt.orc.attend([mt.sid[k] for k in new], T=suf)
        mt.check_meta()
    mt.pool.close()


def test_compose8_8b_full_size(gpu_available):
    """8 agents hold 4096-token segments at positions 0..4095; compose them into
    one 32768-token cache (keys re-rotated by 4096 k), append 2048, decode."""
    wl = synth.WORKLOADS["compose8-8b"]
    s = wl.shape
    seg, A, suf, ndec = wl.context, wl.agents, wl.suffix, 2
    B, L, d = s.block_size, s.n_layers, s.d_model
    HD = s.n_q_heads * s.head_dim
    N = seg * A
    max_pos = N + suf + ndec + 64
    n_blocks = 2 * N // B + (suf + ndec) // B + 64
    mt = MetaTwin(wl, n_blocks, max_pos, scratch_tokens=max(seg, suf), batch=1)
    keys = [synth.x_key(0, wl.name, 10 + j) for j in range(A)]
    o_seg = torch.empty((L, seg, HD), dtype=torch.bfloat16, device="cuda")
    agents = []
    for j in range(A):
        h = kv.kv_materialize(mt.h, mt.x(keys[j], (seg, d)), seg, 0, o_seg)
        mt.sid[h] = mt.orc.materialize(None, T=seg)[0]
        agents.append(h)
    del o_seg
    segs = [(h, 0, seg) for h in agents]
    c = kv.kv_compose(mt.h, segs)
    mt.sid[c] = mt.orc.compose([(mt.sid[a], b, e) for a, b, e in segs])
    mt.check_meta()
    # segment 0 is aliased (zero shift), the other seven are copied
    assert mt.orc.allocated() == A * seg // B + (A - 1) * seg // B
    ka, kd = synth.x_key(0, wl.name, 1), synth.x_key(0, wl.name, 2)
    o_app = torch.empty((L, 1, suf, HD), dtype=torch.bfloat16, device="cuda")
    kv.kv_attend(mt.h, [c], mt.x(ka, (1, suf, d)), suf, o_app)
    mt.orc.attend([mt.sid[c]], T=suf)
    x_dec = mt.x(kd, (ndec, 1, 1, d))
    o_dec = torch.empty((ndec, L, 1, 1, HD), dtype=torch.bfloat16, device="cuda")
    for i in range(ndec):
        kv.kv_attend(mt.h, [c], x_dec[i], 1, o_dec[i])
        mt.orc.attend([mt.sid[c]], T=1)
    mt.check_meta()

    xs = [mt.x64(keys[j], (seg, d)) for j in range(A)]
    xa64 = mt.x64(ka, (1, suf, d))[0]
    xd64 = mt.x64(kd, (ndec, 1, 1, d))[:, 0, 0]
    rng = np.random.default_rng(2)
    for layer in (0, L - 1):
        parts = [ref_kv(mt, layer, xs[j], j * seg + np.arange(seg)) for j in range(A)]
        k_c = np.concatenate([p[0] for p in parts], axis=1)
        v_c = np.concatenate([p[1] for p in parts], axis=1)
        kg, vg = mt.state_kv(c, layer)
        tok = sample_rows(N, B, 1024, rng)
        close_rerotated(to64(kg[:, tok]), k_c[:, tok], "bf16", "composed K (sampled)")
        close(to64(vg[:, tok]), v_c[:, tok], "bf16", "composed V (sampled)")
        # against the agents' own stored keys and values: values bit for bit
        # (every token), keys one rounding from the oracle's re-rotation of
        # the stored source keys (sampled tokens of every segment)
        for j in range(A):
            ks_j, vs_j = mt.state_kv(agents[j], layer)
            kc_j, vc_j = kg[:, j * seg:(j + 1) * seg], vg[:, j * seg:(j + 1) * seg]
            assert torch.equal(vc_j, vs_j), f"composed values of segment {j} must be the source bytes"
            if j == 0:
                assert torch.equal(kc_j, ks_j), "segment 0 is aliased"
                continue
            t = sample_rows(seg, B, 256, rng)
            close_one_rounding(to64(kc_j[:, t]), rerotate(to64(ks_j[:, t]), j * seg, s.rope_base),
                               "bf16", f"re-rotated keys of segment {j}, layer {layer}")
        k_t, v_t = ref_kv(mt, layer, np.concatenate([xa64, xd64]), N + np.arange(suf + ndec))
        kk = np.concatenate([k_c, k_t], axis=1)
        vv = np.concatenate([v_c, v_t], axis=1)
        kpos = np.arange(N + suf + ndec)
        r = sample_rows(suf, B, 32, rng)
        ref = ref_rows(mt, layer, xa64[r], N + r, kk, vv, kpos, N + r + 1)
        close(to64(o_app[layer, 0, r]), ref, "bf16", "append over the composed cache")
        tq = N + suf + np.arange(ndec)
        ref = ref_rows(mt, layer, xd64, tq, kk, vv, kpos, tq + 1)
        close(to64(o_dec[:, layer, 0, 0]), ref, "bf16", "decode over the composed cache")
    mt.pool.close()


def test_pack70b_full_size(gpu_available):
    """70B-shaped 16384-token context (80 layers, B = 32, ~5.4 GB of K/V): pack
    all blocks, unpack into a fresh pool whose free order is a seeded
    permutation, then fork 4 and decode over the restored blocks."""
    wl = synth.WORKLOADS["pack70b"]
    s = wl.shape
    ctx, A, ndec = wl.context, wl.agents, 2
    B, L, d = s.block_size, s.n_layers, s.d_model
    HD = s.n_q_heads * s.head_dim
    max_pos = ctx + ndec + 64
    nb = ctx // B
    P = nb + A * 2 + 16
    src = MetaTwin(wl, P, max_pos, max_states=8, scratch_tokens=ctx, batch=A)
    kx, kd = synth.x_key(0, wl.name, 0), synth.x_key(0, wl.name, 2)
    o_ctx = torch.empty((L, ctx, HD), dtype=torch.bfloat16, device="cuda")
    root = kv.kv_materialize(src.h, src.x(kx, (ctx, d)), ctx, 0, o_ctx)
    src.sid[root] = src.orc.materialize(None, T=ctx)[0]
    rows = sample_rows(ctx, B, 24, np.random.default_rng(3))
    o_rows = o_ctx[[0, L - 1]][:, rows].clone()
    del o_ctx
    buf = torch.empty(nb * s.block_bytes, dtype=torch.uint8, device="cuda")
    hdr = kv.kv_pack(src.h, root, 0, nb, buf)
    ohdr, _ = src.orc.pack(src.sid[root], 0, nb)
    src.check_meta()
    table = kv.kv_read_block_table(src.h, root)
    assert torch.equal(buf.view(torch.bfloat16).view(src.pool.blocks_view()[table].shape),
                       src.pool.blocks_view()[table])

    # destination: a second pool with the same weights and a permuted free ring
    order = synth.permutation(0, wl.name, P)
    dst = MetaTwin.__new__(MetaTwin)
    dst.__dict__.update({k: v for k, v in src.__dict__.items() if k in ("wl", "s", "seed", "w",
                                                                         "cfg", "_w64")})
    dst.pool = kv.Pool(src.cfg, P, kv.kv_scratch_bytes(src.cfg, A, A, max_pos),
                       init_free_order=order)
    dst.pool.set_weights(src.w, s.qkv_cols * d)
    from oracle import OraclePool
    from oracle.pool import PoolShape
    dst.orc = OraclePool(PoolShape(L, d, s.n_q_heads, s.n_kv_heads, s.head_dim, B, s.dtype,
                                   s.rope_base, max_pos, 8, 1), P, init_free_order=order,
                         store_kv=False)
    dst.sid = {}
    u = kv.kv_unpack(dst.h, hdr, buf)
    dst.sid[u] = dst.orc.unpack(ohdr)
    dst.check_meta()
    assert kv.kv_read_block_table(dst.h, u) == [int(v) for v in order[:nb]]
    for layer in (0, L - 1):
        a, b = src.state_kv(root, layer), dst.state_kv(u, layer)
        assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1]), "unpack must restore bytes"
    kids = kv.kv_fork(dst.h, u, A)
    _sync_ids(dst, kids, dst.orc.fork(dst.sid[u], A))
    x_dec = dst.x(kd, (ndec, A, 1, d))
    o_dec = torch.empty((ndec, L, A, 1, HD), dtype=torch.bfloat16, device="cuda")
    for i in range(ndec):
        kv.kv_attend(dst.h, kids, x_dec[i], 1, o_dec[i])
        dst.orc.attend([dst.sid[k] for k in kids], T=1)
    dst.check_meta()

    xc64 = src.x64(kx, (ctx, d))
    xd64 = src.x64(kd, (ndec, A, 1, d))
    for li, layer in enumerate((0, L - 1)):
        k_ctx, v_ctx = ref_kv(src, layer, xc64, np.arange(ctx))
        ref = ref_rows(src, layer, xc64[rows], rows, k_ctx, v_ctx, np.arange(ctx), rows + 1)
        close(to64(o_rows[li]), ref, "bf16", "70B materialize output")
        for j in range(A):
            k_d, v_d = ref_kv(src, layer, xd64[:, j, 0], ctx + np.arange(ndec))
            kk = np.concatenate([k_ctx, k_d], axis=1)
            vv = np.concatenate([v_ctx, v_d], axis=1)
            tq = ctx + np.arange(ndec)
            ref = ref_rows(src, layer, xd64[:, j, 0], tq, kk, vv, np.arange(ctx + ndec), tq + 1)
            close(to64(o_dec[:, layer, j, 0]), ref, "bf16", f"70B decode agent {j}")
    dst.pool.close()
    src.pool.close()
