#!/usr/bin/env python3
"""Throughput of the KV-state hot path on one MI355X.

One step is one pass of every operator over the 8B-shaped fork workload
(32 layers, d_model 4096, 32 query / 8 KV heads, head_dim 128, bf16, block 16):

  1. materialize an 8192-token shared context;
  2. fork it to 4 agents;
  3. append a 512-token prompt to each agent (batched append-prefill);
  4. 128 batched decode steps (batch 4);
  5. compose [context | agent 1 .. 4 continuations] into one state (agent 1's
     blocks are aliased, agents 2-4 are re-rotated by their position shift);
  6. pack the composed state into a transfer buffer and unpack it again;
  7. evict every state (LRU, budget 0), which returns the pool to empty.

All inputs are synthetic (seeded, see synth/) and resident in HBM before the
timed region.  ``value`` is the materialize + attend throughput in TFLOP/s
(algorithmic flops of the projections and the causal attention of steps 1, 3
and 4, divided by the wall time of whole steps).  Per-operator figures,
the roofline of the dominant kernel (timed live with HIP events on the launch
stream) and the float64 oracle's throughput on a bounded sample of the same
workload are reported alongside.

Usage: python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
MFMA_BF16_PEAK_TF = 2500.0   # MI355X dense bf16 MFMA


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="fork4-8b")
    ap.add_argument("--decode", type=int, default=None, help="override decode steps")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle baseline")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run one 1 GiB device copy first (reference for HBM byte counters)")
    ap.add_argument("--transfer-sweep", action="store_true",
                    help="instead of the step: measured materialize vs pack + unpack per context "
                         "length, and the transfer-vs-recompute decision at several link rates")
    ap.add_argument("--checkpoint-sweep", action="store_true",
                    help="instead of the step: plain vs checksummed pack / unpack and file "
                         "checkpoint save / load per context length")
    return ap.parse_args()


# ------------------------------------------------------------------ algorithmic work

def proj_flops(s, tokens):
    return 2.0 * tokens * s.d_model * s.qkv_cols * s.n_layers


def attn_flops(s, n_before, T):
    """Causal attention of T new queries over n_before cached + T new keys."""
    pairs = T * n_before + T * (T + 1) / 2.0
    return 4.0 * s.n_q_heads * s.head_dim * pairs * s.n_layers


def kv_bytes_per_token(s):
    return 2 * s.n_layers * s.n_kv_heads * s.head_dim * s.elt_bytes


# ------------------------------------------------------------------ cpu baseline

def measured_traffic(workload, kind):
    """HBM bytes per launch of a kernel kind, from the committed rocprofv3 PMC
    summary (FETCH_SIZE and WRITE_SIZE scaled by a plain copy's reading), or
    None when there is none or the kernel's source changed since."""
    path = os.path.join(ROOT, "profiles", f"pmc_traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    start = text.find("```json")
    if start < 0:
        return None
    end = text.find("```", start + 7)
    try:
        entry = json.loads(text[start + 7:end])["kinds"].get(kind)
    except (ValueError, KeyError):
        return None
    if not entry:
        return None
    with open(os.path.join(ROOT, entry["source"]), "rb") as f:
        if hashlib.sha256(f.read()).hexdigest() != entry["source_sha256"]:
            return None
    return entry["hbm_bytes_per_dispatch"]


def cpu_baseline(wl, seed):
    """The float64 oracle on a bounded sample: one layer of the workload's shape,
    materialize of the whole context, fork, then 16 batched decode steps."""
    import numpy as np
    import synth
    from oracle import OraclePool
    from oracle.pool import PoolShape
    s = wl.shape
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    T, b, steps = wl.context, wl.agents, 16
    cols, d = s.qkv_cols, s.d_model
    w = [synth.to_f64(synth.normal_np(synth.w_key(seed, wl.name, 0), (cols, d), s.w_std, s.dtype),
                      s.dtype)]
    shape = PoolShape(1, d, s.n_q_heads, s.n_kv_heads, s.head_dim, s.block_size, s.dtype,
                      s.rope_base, T + steps + 16, 16, 1)
    orc = OraclePool(shape, 4 * (T // s.block_size + 8), weights=w)
    x = synth.to_f64(synth.normal_np(synth.x_key(seed, wl.name, 0), (T, d), 1.0, s.dtype), s.dtype)
    xd = synth.to_f64(synth.normal_np(synth.x_key(seed, wl.name, 9), (steps, b, 1, d), 1.0,
                                      s.dtype), s.dtype)
    t0 = time.perf_counter()
    root, _ = orc.materialize(x)
    kids = orc.fork(root, b)
    for i in range(steps):
        orc.attend(kids, xd[i])
    dt = time.perf_counter() - t0
    flops = proj_flops(_Shape1(s), T) + attn_flops(_Shape1(s), 0, T)
    for i in range(steps):
        flops += b * (proj_flops(_Shape1(s), 1) + attn_flops(_Shape1(s), T + i, 1))
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"one layer of the {wl.shape.name} shape: materialize {T} tokens, fork "
                      f"{b}, {steps} batched decode steps; float64 NumPy, {dt:.1f} s"}


class _Shape1:
    """The workload shape restricted to one layer (for the sample's flop count)."""

    def __init__(self, s):
        self.__dict__.update({k: getattr(s, k) for k in ("d_model", "n_q_heads", "n_kv_heads",
                                                          "head_dim", "qkv_cols")})
        self.n_layers = 1



# ------------------------------------------------------------------ transfer sweep

LINKS = [("10 Gb/s", 1.25e9, 20e-6), ("25 Gb/s", 3.125e9, 20e-6), ("100 Gb/s", 12.5e9, 10e-6),
         ("400 Gb/s", 50e9, 5e-6), ("xGMI link 153 GB/s", 153e9, 2e-6)]


def transfer_sweep(args, kv, torch, synth):
    """Single-GPU counterpart of the paper's transfer-vs-recomputation
    experiment on the 8B shape: for each context length, materialize (the
    recompute cost) and pack + unpack (the device side of a transfer) are
    timed with the library's per-kernel events; the decision of
    kv_plan_transfer is then reported for several link rates."""
    wl = synth.WORKLOADS["fork4-8b"]
    s = wl.shape
    dev = "cuda"
    tdt = torch.bfloat16
    L, d, cols, B = s.n_layers, s.d_model, s.qkv_cols, s.block_size
    lengths = [1024, 2048, 4096, 8192, 16384, 32768]
    nmax = lengths[-1]
    cfg = kv.make_cfg(L, d, s.n_q_heads, s.n_kv_heads, s.head_dim, B, s.dtype, nmax + 64, 8,
                      s.rope_base, 1)
    n_blocks = 2 * (nmax // B) + 64
    pool = kv.Pool(cfg, n_blocks, kv.kv_scratch_bytes(cfg, nmax, 1, nmax + 64))
    w = torch.empty((L, cols, d), dtype=tdt, device=dev)
    for layer in range(L):
        w[layer] = synth.normal_torch(synth.w_key(args.seed, wl.name, layer), (cols, d), s.w_std,
                                      s.dtype, dev)
    pool.set_weights(w, cols * d)
    x = synth.normal_torch(synth.x_key(args.seed, wl.name, 0), (nmax, d), 1.0, s.dtype, dev)
    o = torch.empty((L, nmax, s.n_q_heads * s.head_dim), dtype=tdt, device=dev)
    buf = torch.empty((nmax // B) * s.block_bytes, dtype=torch.uint8, device=dev)
    host = torch.empty((nmax // B) * s.block_bytes, dtype=torch.uint8, pin_memory=True)
    rows = []
    for n in lengths:
        times = {"mat": [], "pack": [], "unpack": [], "pack_host": [], "unpack_host": []}
        for rep in range(3):
            kv.kv_profile_enable(pool.h, True)
            kv.kv_profile_read(pool.h)
            st = kv.kv_materialize(pool.h, x[:n], n, 0, o[:, :n])
            nb = kv.kv_state_info(pool.h, st)["n_blocks"]
            hdr = kv.kv_pack(pool.h, st, 0, nb, buf)
            u = kv.kv_unpack(pool.h, hdr, buf)
            prof = kv.kv_profile_read(pool.h)
            kv.kv_release(pool.h, u)
            # the host tier: pack into pinned host memory, unpack from it
            hdr_h = kv.kv_pack(pool.h, st, 0, nb, host)
            u = kv.kv_unpack(pool.h, hdr_h, host)
            prof_h = kv.kv_profile_read(pool.h)
            kv.kv_profile_enable(pool.h, False)
            kv.kv_release(pool.h, st)
            kv.kv_release(pool.h, u)
            if rep == 0:
                continue  # warm-up
            times["mat"].append(sum(prof[k][1] for k in ("alloc", "qkv", "attn")))
            times["pack"].append(prof["pack"][1])
            times["unpack"].append(prof["unpack"][1])
            times["pack_host"].append(prof_h["pack"][1])
            times["unpack_host"].append(prof_h["unpack"][1])
        t_mat = min(times["mat"]) / 1e3
        t_pack = min(times["pack"]) / 1e3
        t_unpack = min(times["unpack"]) / 1e3
        kvb = (-(-n // B)) * s.block_bytes
        fl = kv.kv_plan_transfer(cfg, n, 1.0, 0.0, 0.0, 0.0, 1.0)["prefill_flops"]
        rate = fl / t_mat
        t_ph = min(times["pack_host"]) / 1e3
        t_uh = min(times["unpack_host"]) / 1e3
        row = {"tokens": n, "kv_bytes": kvb, "materialize_ms": round(t_mat * 1e3, 3),
               "prefill_TFLOPs": round(rate / 1e12, 1), "pack_ms": round(t_pack * 1e3, 4),
               "unpack_ms": round(t_unpack * 1e3, 4),
               "host_tier": {"pack_ms": round(t_ph * 1e3, 3), "unpack_ms": round(t_uh * 1e3, 3),
                             "pack_GBs": round(kvb / t_ph / 1e9, 1),
                             "unpack_GBs": round(kvb / t_uh / 1e9, 1),
                             "reload_vs_recompute": round(t_mat / t_uh, 1)},
               "links": {}}
        for name, bw, lat in LINKS:
            plan = kv.kv_plan_transfer(cfg, n, bw, lat, kvb / t_pack, kvb / t_unpack, rate)
            row["links"][name] = {"transfer_ms": round(plan["t_transfer"] * 1e3, 3),
                                  "decision": "transfer" if plan["transfer"] else "recompute",
                                  "speedup": round(plan["t_prefill"] / plan["t_transfer"], 2)}
        rows.append(row)
        print(f"[bench] sweep {n} tokens done", file=sys.stderr, flush=True)
    pool.close()
    print(json.dumps({"experiment": "transfer vs recompute (8B shape, one MI355X)",
                      "data": "synthetic", "rows": rows}), flush=True)

def checkpoint_sweep(args, kv, torch, synth):
    """Cost of integrity and persistence on the 8B shape: the pack / unpack
    kernels with and without the fused payload checksum (kernel time from the
    library's events, and the whole call including the checksum read-back),
    and file checkpoints (save / load through pinned staging, wall time)."""
    import tempfile
    wl = synth.WORKLOADS["fork4-8b"]
    s = wl.shape
    dev = "cuda"
    tdt = torch.bfloat16
    L, d, cols, B = s.n_layers, s.d_model, s.qkv_cols, s.block_size
    lengths = [1024, 4096, 16384]
    nmax = lengths[-1]
    cfg = kv.make_cfg(L, d, s.n_q_heads, s.n_kv_heads, s.head_dim, B, s.dtype, nmax + 64, 8,
                      s.rope_base, 1)
    n_blocks = 2 * (nmax // B) + 64
    pool = kv.Pool(cfg, n_blocks, kv.kv_scratch_bytes(cfg, nmax, 1, nmax + 64))
    w = torch.empty((L, cols, d), dtype=tdt, device=dev)
    for layer in range(L):
        w[layer] = synth.normal_torch(synth.w_key(args.seed, wl.name, layer), (cols, d), s.w_std,
                                      s.dtype, dev)
    pool.set_weights(w, cols * d)
    x = synth.normal_torch(synth.x_key(args.seed, wl.name, 0), (nmax, d), 1.0, s.dtype, dev)
    o = torch.empty((L, nmax, s.n_q_heads * s.head_dim), dtype=tdt, device=dev)
    buf = torch.empty((nmax // B) * s.block_bytes, dtype=torch.uint8, device=dev)
    tmpdir = tempfile.mkdtemp(prefix="kvck")
    path = os.path.join(tmpdir, "state.kvck")
    rows = []

    def wall(fn):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        r = fn()
        torch.cuda.synchronize()
        return r, time.perf_counter() - t0

    for n in lengths:
        st = kv.kv_materialize(pool.h, x[:n], n, 0, o[:, :n])
        nb = kv.kv_state_info(pool.h, st)["n_blocks"]
        kvb = nb * s.block_bytes
        t = {k: [] for k in ("pack_k", "packc_k", "unpack_k", "unpackc_k", "packc_w",
                             "unpackc_w", "save_w", "load_w")}
        for rep in range(4):
            kv.kv_profile_enable(pool.h, True)
            kv.kv_profile_read(pool.h)
            hdr = kv.kv_pack(pool.h, st, 0, nb, buf)
            u = kv.kv_unpack(pool.h, hdr, buf)
            p0 = kv.kv_profile_read(pool.h)
            kv.kv_release(pool.h, u)
            kv.kv_profile_read(pool.h)
            hc, tw = wall(lambda: kv.kv_pack_checked(pool.h, st, 0, nb, buf))
            uc, tu = wall(lambda: kv.kv_unpack(pool.h, hc, buf))
            p1 = kv.kv_profile_read(pool.h)
            kv.kv_profile_enable(pool.h, False)
            kv.kv_release(pool.h, uc)
            _, ts = wall(lambda: kv.kv_checkpoint_save(pool.h, st, path))
            v, tl = wall(lambda: kv.kv_checkpoint_load(pool.h, path))
            kv.kv_release(pool.h, v)
            os.remove(path)
            if rep == 0:
                continue  # warm-up
            t["pack_k"].append(p0["pack"][1])
            t["unpack_k"].append(p0["unpack"][1])
            t["packc_k"].append(p1["pack"][1])
            t["unpackc_k"].append(p1["unpack"][1])
            t["packc_w"].append(tw * 1e3)
            t["unpackc_w"].append(tu * 1e3)
            t["save_w"].append(ts * 1e3)
            t["load_w"].append(tl * 1e3)
        kv.kv_release(pool.h, st)
        m = {k: min(v) for k, v in t.items()}

        def gbs(ms):
            return round(2 * kvb / (ms * 1e-3) / 1e9, 1)  # read + write bytes

        rows.append({
            "tokens": n, "kv_bytes": kvb,
            "pack": {"ms": round(m["pack_k"], 4), "GBs": gbs(m["pack_k"])},
            "pack_checked": {"kernel_ms": round(m["packc_k"], 4), "GBs": gbs(m["packc_k"]),
                             "call_ms": round(m["packc_w"], 4)},
            "unpack": {"ms": round(m["unpack_k"], 4), "GBs": gbs(m["unpack_k"])},
            "unpack_checked": {"kernel_ms": round(m["unpackc_k"], 4), "GBs": gbs(m["unpackc_k"]),
                               "call_ms": round(m["unpackc_w"], 4)},
            "checkpoint": {"save_ms": round(m["save_w"], 2), "load_ms": round(m["load_w"], 2),
                           "save_GBs": round(kvb / (m["save_w"] * 1e-3) / 1e9, 2),
                           "load_GBs": round(kvb / (m["load_w"] * 1e-3) / 1e9, 2)}})
        print(f"[bench] checkpoint sweep {n} tokens done", file=sys.stderr, flush=True)
    os.rmdir(tmpdir)
    pool.close()
    print(json.dumps({"experiment": "checksum and checkpoint cost (8B shape, one MI355X)",
                      "rate_bytes": "pack / unpack GB/s count read + write bytes; checkpoint "
                                    "GB/s count the payload once",
                      "data": "synthetic", "rows": rows}), flush=True)

# ------------------------------------------------------------------ main

def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark measures one GPU; --gpus must be 1"}))
        sys.exit(2)
    import torch
    import synth
    from paper_2607_10987_amd import kvstate as kv

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU"}))
        sys.exit(2)
    if args.transfer_sweep:
        transfer_sweep(args, kv, torch, synth)
        return
    if args.checkpoint_sweep:
        checkpoint_sweep(args, kv, torch, synth)
        return
    wl = synth.WORKLOADS[args.workload]
    s = wl.shape
    ndec = wl.decode if args.decode is None else args.decode
    dev = "cuda"
    tdt = torch.bfloat16 if s.dtype == "bf16" else torch.float32
    L, d, cols = s.n_layers, s.d_model, s.qkv_cols
    ctx, A, suf, B = wl.context, wl.agents, wl.suffix, s.block_size
    cont = suf + ndec                                   # tokens each agent adds
    n_comp = ctx + A * cont                             # composed state length
    max_pos = n_comp + 64
    blocks_needed = (ctx // B + 1) + A * (cont // B + 2) + 2 * (n_comp // B + 2)
    n_blocks = blocks_needed + 64
    t_setup = time.perf_counter()
    print(f"[bench] setup {wl.name}: {n_blocks} blocks of {s.block_bytes / 2**20:.1f} MiB",
          file=sys.stderr, flush=True)

    # inputs, resident in HBM before timing
    w = torch.empty((L, cols, d), dtype=tdt, device=dev)
    for layer in range(L):
        w[layer] = synth.normal_torch(synth.w_key(args.seed, wl.name, layer), (cols, d), s.w_std,
                                      s.dtype, dev)
    x_ctx = synth.normal_torch(synth.x_key(args.seed, wl.name, 0), (ctx, d), 1.0, s.dtype, dev)
    x_suf = synth.normal_torch(synth.x_key(args.seed, wl.name, 1), (A, suf, d), 1.0, s.dtype, dev)
    x_dec = synth.normal_torch(synth.x_key(args.seed, wl.name, 2), (ndec, A, 1, d), 1.0, s.dtype,
                               dev)
    o_ctx = torch.empty((L, ctx, s.n_q_heads * s.head_dim), dtype=tdt, device=dev)
    o_suf = torch.empty((L, A, suf, s.n_q_heads * s.head_dim), dtype=tdt, device=dev)
    o_dec = torch.empty((L, A, 1, s.n_q_heads * s.head_dim), dtype=tdt, device=dev)
    cfg = kv.make_cfg(L, d, s.n_q_heads, s.n_kv_heads, s.head_dim, B, s.dtype, max_pos, 64,
                      s.rope_base, 1)
    scratch = kv.kv_scratch_bytes(cfg, max(ctx, A * suf), A, max_pos)
    pool = kv.Pool(cfg, n_blocks, scratch)
    pool.set_weights(w, cols * d)
    nb_comp = -(-n_comp // B)
    pack_buf = torch.empty(nb_comp * s.block_bytes, dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    print(f"[bench] setup done in {time.perf_counter() - t_setup:.1f} s", file=sys.stderr,
          flush=True)

    # plain device copy of 1 GiB: reference rate for the HBM-bound operators
    # (and, with --copy-calibration, the reference for HBM byte counters)
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    copy_ms = []
    for _ in range(1 if args.copy_calibration else 4):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        copy_ms.append(e0.elapsed_time(e1))
    copy_gbs = 2.0 * (1 << 30) / (min(copy_ms[1:] or copy_ms) / 1e3) / 1e9
    del src, dst

    info = {}

    def step():
        root = kv.kv_materialize(pool.h, x_ctx, ctx, 0, o_ctx)
        kids = kv.kv_fork(pool.h, root, A)
        if suf:
            kv.kv_attend(pool.h, kids, x_suf, suf, o_suf)
        for i in range(ndec):
            kv.kv_attend(pool.h, kids, x_dec[i], 1, o_dec)
        segs = [(root, 0, ctx)] + [(k, ctx, ctx + cont) for k in kids]
        c = kv.kv_compose(pool.h, segs)
        nb = kv.kv_state_info(pool.h, c)["n_blocks"]
        hdr = kv.kv_pack(pool.h, c, 0, nb, pack_buf)
        u = kv.kv_unpack(pool.h, hdr, pack_buf)
        info["nb_comp"] = nb
        info["u"] = u
        n_ev = kv.kv_evict(pool.h, 0, 0.0, 0.0, 1.0)
        info["evicted"] = n_ev

    for i in range(args.warmup):
        step()
        print(f"[bench] warmup step {i + 1}/{args.warmup} done", file=sys.stderr, flush=True)
    kv.kv_sync(pool.h)
    kv.kv_profile_enable(pool.h, True)
    kv.kv_profile_read(pool.h)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step()
        print(f"[bench] step {i + 1}/{args.steps} done", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    prof = kv.kv_profile_read(pool.h)
    kv.kv_profile_enable(pool.h, False)
    kv.kv_sync(pool.h)
    ms_step = (t1 - t0) * 1000.0 / args.steps
    K = args.steps

    # ---- algorithmic work of one step
    f_mat = proj_flops(s, ctx) + attn_flops(s, 0, ctx)
    f_app = A * (proj_flops(s, suf) + attn_flops(s, ctx, suf))
    f_dec = sum(A * (proj_flops(s, 1) + attn_flops(s, ctx + suf + i, 1)) for i in range(ndec))
    flops = f_mat + f_app + f_dec
    kvb = kv_bytes_per_token(s)
    w_bytes = L * cols * d * s.elt_bytes
    # decode: weights once + unique KV (shared context once, private per agent) + x/o
    dec_kv_bytes = sum(kvb * (ctx + A * (suf + i + 1)) for i in range(ndec))
    dec_io = ndec * A * (d + L * s.n_q_heads * s.head_dim) * s.elt_bytes
    b_qkv_dec = ndec * (w_bytes + A * d * s.elt_bytes + A * L * cols * s.elt_bytes)
    b_attn_dec = dec_kv_bytes + ndec * A * L * s.n_q_heads * s.head_dim * s.elt_bytes * 2
    copied = A - 1                                        # agent 1's blocks are aliased
    b_compose = 2 * copied * (cont // B) * s.block_bytes
    b_pack = 2 * info["nb_comp"] * s.block_bytes
    b_unpack = b_pack

    def ms(kind):
        return prof[kind][1] / K

    ops = {}

    def put(name, kinds, work, unit, peak):
        t = sum(ms(k) for k in kinds)
        rate = (work / (t / 1e3) / (1e12 if unit == "TFLOP/s" else 1e9)) if t > 0 else None
        ops[name] = {"ms": round(t, 4), "rate": None if rate is None else round(rate, 2),
                     "unit": unit, "frac": None if rate is None else round(rate / peak, 4)}

    put("materialize+append qkv", ["qkv"], proj_flops(s, ctx) + A * proj_flops(s, suf),
        "TFLOP/s", MFMA_BF16_PEAK_TF)
    put("materialize+append attention", ["attn"], attn_flops(s, 0, ctx) +
        A * attn_flops(s, ctx, suf), "TFLOP/s", MFMA_BF16_PEAK_TF)
    put("decode qkv", ["qkv_decode"], b_qkv_dec, "GB/s", HBM_PEAK_GBS)
    put("decode attention", ["attn_decode", "merge"], b_attn_dec, "GB/s", HBM_PEAK_GBS)
    put("compose", ["compose_copy"], b_compose, "GB/s", HBM_PEAK_GBS)
    put("pack", ["pack"], b_pack, "GB/s", HBM_PEAK_GBS)
    put("unpack", ["unpack"], b_unpack, "GB/s", HBM_PEAK_GBS)
    for k in ("decode qkv", "decode attention", "compose", "pack", "unpack"):
        if ops[k]["rate"] is not None:
            ops[k]["frac_of_copy"] = round(ops[k]["rate"] / copy_gbs, 4)
    ops["fork"] = {"us": round(ms("fork") * 1e3, 2)}
    ops["evict"] = {"us": round(ms("release") * 1e3, 2)}

    # ---- roofline of the dominant kernel kind (largest summed duration)
    work_of = {
        "qkv": (proj_flops(s, ctx) + A * proj_flops(s, suf), "mfma"),
        "attn": (attn_flops(s, 0, ctx) + A * attn_flops(s, ctx, suf), "mfma"),
        "qkv_decode": (b_qkv_dec, "hbm"),
        "attn_decode": (b_attn_dec, "hbm"),
        "compose_copy": (b_compose, "hbm"),
        "pack": (b_pack, "hbm"),
        "unpack": (b_unpack, "hbm"),
    }
    dom = max(work_of, key=lambda k: prof[k][1])
    work, bound = work_of[dom]
    t_dom = prof[dom][1] / 1e3
    if bound == "mfma":
        achieved, peak, unit = work * K / t_dom / 1e12, MFMA_BF16_PEAK_TF, "TFLOP/s"
    else:
        achieved, peak, unit = work * K / t_dom / 1e9, HBM_PEAK_GBS, "GB/s"
    roofline = {"bound": bound, "kernel": dom, "achieved": round(achieved, 2), "peak": peak,
                "unit": unit, "frac": round(achieved / peak, 4),
                "traffic": measured_traffic(wl.name, dom),
                "algorithmic_bytes_per_launch": int(work / max(prof[dom][0] // K, 1))
                if bound == "hbm" else None,
                "launches_per_step": prof[dom][0] // K,
                "avg_launch_ms": round(prof[dom][1] / max(prof[dom][0], 1), 4)}

    value = flops / (ms_step / 1e3) / 1e12
    out = {
        "metric": "compose/pack GB/s (% HBM peak); materialize+attend TFLOP/s (% MFMA peak)",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": s.dtype,
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: {s.n_layers} layers, d_model {d}, "
                               f"{s.n_q_heads}/{s.n_kv_heads} heads, head_dim {s.head_dim}, "
                               f"block {B}; context {ctx}, fork {A}, append {suf}, "
                               f"decode {ndec}, compose {n_comp} tokens, pack/unpack "
                               f"{info['nb_comp']} blocks, evict all",
                   "global_batch": A, "seq_len": n_comp},
        "ops": ops,
        "roofline": roofline,
        "kernel_ms_per_step": {k: round(v[1] / K, 4) for k, v in prof.items() if v[0]},
        "copy_reference": {"GB/s": round(copy_gbs, 1), "what": "torch device-to-device copy "
                           "of 1 GiB (read + write bytes), same run"},
    }
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(wl, args.seed)
    pool.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
