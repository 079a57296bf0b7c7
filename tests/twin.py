"""Run the same operator sequence on the device library and on the oracle.

``Twin`` mirrors every call (materialize, fork, attend, compose, pack, unpack,
evict, release) on a GPU pool (through the C ABI) and on an ``OraclePool``
fed the same seeded inputs, and compares after each call:

* block tables, refcounts, the free ring and its counters, state metadata:
  bit-exact;
* attention outputs and pool K/V contents: max-abs and relative-L2 bounds
  (bf16: 2e-2 / 5e-3; float32: 1e-4 / 1e-5);
* the eviction score terms of every live state (reuse count, last access,
  pinned flag): exact;
* keys that a composition re-rotated: against the oracle's re-rotation of the
  device's own stored source keys, within half a unit in the last place of
  the storage type plus float32 arithmetic noise (one rounding), and values
  bit-exactly against the device's source values; later checks of such a
  state compare those tokens bit-exactly with what the composition wrote.
"""
from __future__ import annotations

import numpy as np
import torch

import synth
from oracle import OraclePool, rerotate
from oracle.pool import PoolShape
from paper_2607_10987_amd import kvstate as kv

TOL = {"bf16": (2e-2, 5e-3), "f32": (1e-4, 1e-5)}


def close(got, want, dtype, what=""):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    if got.size == 0:
        return 0.0, 0.0
    atol, rtol = TOL[dtype]
    err = np.abs(got - want)
    mx = float(err.max())
    rel = float(np.linalg.norm(got - want) / max(np.linalg.norm(want), 1e-30))
    assert np.all(np.isfinite(got)), f"{what}: non-finite values"
    assert mx <= atol and rel <= rtol, f"{what}: max-abs {mx:.3e} rel-L2 {rel:.3e}"
    return mx, rel


def close_rerotated(got, want, dtype, what=""):
    """Keys that were rounded to bf16, re-rotated in fp32 and rounded again.

    Each rounding moves an element by at most 2^-8 of its magnitude and a
    rotation preserves the norm of a pair (x_i, x_{i+dh/2}), so the error of
    an element is at most 2^-7 (1 + 2^-8) times its pair's norm (plus fp32
    arithmetic noise); the relative L2 bound stays the bf16 one.
    """
    if dtype != "bf16":
        return close(got, want, dtype, what)
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    half = want.shape[-1] // 2
    pn = np.sqrt(want[..., :half] ** 2 + want[..., half:] ** 2)
    bound = 2.0 ** -7 * (1 + 2.0 ** -8) * np.concatenate([pn, pn], axis=-1) + 1e-5
    err = np.abs(got - want)
    assert np.all(err <= bound), f"{what}: {int(np.sum(err > bound))} elements over the bound"
    rel = float(np.linalg.norm(got - want) / max(np.linalg.norm(want), 1e-30))
    assert rel <= TOL[dtype][1], f"{what}: rel-L2 {rel:.3e}"
    return float(err.max()), rel


def half_ulp(x, dtype):
    """Half a unit in the last place of |x| in the storage type."""
    mant = 8 if dtype == "bf16" else 24          # significand bits incl. the implicit one
    e = np.floor(np.log2(np.maximum(np.abs(x), 2.0 ** -100)))
    return np.ldexp(1.0, (e - mant).astype(np.int64))


def close_one_rounding(got, want, dtype, what=""):
    """got = the storage rounding of a float32 evaluation of want: each element
    within half an ulp (taken at |want| + noise) plus the float32 noise of a
    rotation, 2^-21 times the norm of the element's rotation pair."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    half = want.shape[-1] // 2
    pn = np.sqrt(want[..., :half] ** 2 + want[..., half:] ** 2)
    noise = 2.0 ** -21 * np.concatenate([pn, pn], axis=-1)
    bound = half_ulp(np.abs(want) + noise, dtype) + noise
    err = np.abs(got - want)
    bad = err > bound
    assert not bad.any(), (f"{what}: {int(bad.sum())} of {bad.size} elements beyond one "
                           f"rounding, worst excess {float((err - bound).max()):.3e}")
    return float(err.max())


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


class Twin:
    def __init__(self, shape: synth.ModelShape, n_blocks: int, max_pos: int, max_states: int = 32,
                 seed: int = 0, wl: str = "twin", order=None, scratch_tokens: int = 4096,
                 check_kv: bool = True, model_id: int = 7, scratch_bytes: int = None):
        self.s = shape
        self.seed = seed
        self.wl = wl
        self.dt = shape.dtype
        self.tdt = torch.bfloat16 if self.dt == "bf16" else torch.float32
        self.check_kv_each = check_kv
        L, cols, d = shape.n_layers, shape.qkv_cols, shape.d_model
        self.w_dev = torch.empty((L, cols, d), dtype=self.tdt, device="cuda")
        w64 = []
        for layer in range(L):
            key = synth.w_key(seed, wl, layer)
            self.w_dev[layer] = synth.normal_torch(key, (cols, d), shape.w_std, self.dt, "cuda")
            w64.append(synth.to_f64(synth.normal_np(key, (cols, d), shape.w_std, self.dt), self.dt))
        self.cfg = kv.make_cfg(L, d, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                               shape.block_size, self.dt, max_pos, max_states,
                               shape.rope_base, model_id)
        scratch = kv.kv_scratch_bytes(self.cfg, scratch_tokens, 8, max_pos) \
            if scratch_bytes is None else scratch_bytes
        self.gpu = kv.Pool(self.cfg, n_blocks, scratch, init_free_order=order)
        self.gpu.set_weights(self.w_dev, cols * d)
        pshape = PoolShape(L, d, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                           shape.block_size, self.dt, shape.rope_base, max_pos, max_states,
                           model_id)
        self.orc = OraclePool(pshape, n_blocks, init_free_order=order, weights=w64)
        self.sid = {}        # gpu handle -> oracle state id
        self.rerot = {}      # handle -> device K [L][Hkv, n, dh] a composition wrote
        self.calls = 0

    # -------------------------------------------------------------- inputs

    def x(self, rows: int, tag: int):
        key = synth.x_key(self.seed, self.wl, tag)
        d = self.s.d_model
        xd = synth.normal_torch(key, (rows, d), 1.0, self.dt, "cuda")
        x64 = synth.to_f64(synth.normal_np(key, (rows, d), 1.0, self.dt), self.dt)
        return xd, x64

    # -------------------------------------------------------------- checks

    def check_meta(self):
        torch.cuda.synchronize()
        kv.kv_sync(self.gpu.h)
        P = self.gpu.n_blocks
        rc, ring, head, tail = kv.kv_read_allocator(self.gpu.h, P)
        orc_rc, orc_ring, oh, ot = self.orc.allocator()
        assert (head, tail) == (oh, ot), ("ring counters", head, tail, oh, ot)
        assert rc == [int(v) for v in orc_rc], "refcounts differ"
        assert ring == [int(v) for v in orc_ring], "free ring differs"
        for h, sid in self.sid.items():
            st = self.orc.states[sid]
            if st.status != "ACTIVE":
                continue
            info = kv.kv_state_info(self.gpu.h, h)
            assert info["state_id"] == sid
            assert (info["pos0"], info["n_tokens"], info["n_blocks"], info["lineage"]) == \
                self.orc.info(sid), ("state info", info, self.orc.info(sid))
            assert kv.kv_read_block_table(self.gpu.h, h) == self.orc.table(sid), "block table"
            u = kv.kv_state_usage(self.gpu.h, h)
            assert (u["reuse"], u["last_access"], u["pinned"]) == \
                (st.reuse, st.last_access, st.pinned), ("eviction score terms", u)
        c = kv.kv_pool_counts(self.gpu.h)
        assert c["free_blocks"] == self.orc.free_count()
        assert c["clock"] == self.orc.clock

    def gpu_state_kv_raw(self, h, layer):
        """Device K and V of a state's valid tokens: two [Hkv, n, dh] tensors
        of the storage type."""
        table = kv.kv_read_block_table(self.gpu.h, h)
        n = kv.kv_state_info(self.gpu.h, h)["n_tokens"]
        blocks = self.gpu.blocks_view()[table, layer]         # [nb, 2, Hkv, B, dh]
        nb, _, hkv, B, dh = blocks.shape
        # valid slots only: the slots past the last token are unspecified and
        # may hold any bit pattern (signalling NaNs included)
        x = blocks.permute(1, 2, 0, 3, 4).reshape(2, hkv, nb * B, dh)[:, :, :n]
        return x[0], x[1]

    def gpu_state_kv(self, h, layer):
        k, v = self.gpu_state_kv_raw(h, layer)
        return to_np(k), to_np(v)

    def check_state_kv(self, h):
        sid = self.sid[h]
        for layer in range(self.s.n_layers):
            k, v = self.gpu_state_kv(h, layer)
            ko, vo = self.orc.state_kv(sid, layer)
            if h in self.rerot:
                m = min(self.rerot[h][layer].shape[1], k.shape[1])
                kr, _ = self.gpu_state_kv_raw(h, layer)
                assert torch.equal(kr[:, :m], self.rerot[h][layer][:, :m]), \
                    f"composed keys changed, layer {layer}"
                close(k[:, m:], ko[:, m:], self.dt, f"K after the composition, layer {layer}")
                close_rerotated(k[:, :m], ko[:, :m], self.dt, f"re-rotated K layer {layer}")
            else:
                close(k, ko, self.dt, f"K layer {layer}")
            close(v, vo, self.dt, f"V layer {layer}")

    def check_compose_kv(self, h, segs):
        """A composition against the device's own source state: per segment,
        keys = the oracle's re-rotation of the stored source keys by the
        segment's shift (one rounding), values = the source values bit for
        bit.  Records the composed keys for later checks of the state."""
        info = {a: kv.kv_state_info(self.gpu.h, a) for a, _, _ in segs}
        p_dst = info[segs[0][0]]["pos0"] + segs[0][1]
        snap = []
        for layer in range(self.s.n_layers):
            kd, vd = self.gpu_state_kv_raw(h, layer)
            cum = 0
            for a, b, e in segs:
                ks, vs = self.gpu_state_kv_raw(a, layer)
                delta = p_dst + cum - (info[a]["pos0"] + b)
                n = e - b
                assert torch.equal(vd[:, cum:cum + n], vs[:, b:e]), \
                    f"composed V differs from its source, layer {layer}"
                if delta == 0:
                    assert torch.equal(kd[:, cum:cum + n], ks[:, b:e]), \
                        f"unshifted composed K differs from its source, layer {layer}"
                else:
                    want = rerotate(to_np(ks[:, b:e]), delta, self.s.rope_base)
                    close_one_rounding(to_np(kd[:, cum:cum + n]), want, self.dt,
                                       f"re-rotated K (shift {delta}), layer {layer}")
                cum += n
            snap.append(kd.clone())
        self.rerot[h] = snap

    def _after(self, *handles):
        self.calls += 1
        self.check_meta()
        if self.check_kv_each:
            for h in handles:
                self.check_state_kv(h)

    # -------------------------------------------------------------- operators

    def materialize(self, T: int, pos0: int = 0, tag: int = None):
        xd, x64 = self.x(T, self.calls if tag is None else tag)
        s = self.s
        o = torch.empty((s.n_layers, T, s.n_q_heads * s.head_dim), dtype=self.tdt, device="cuda")
        h = kv.kv_materialize(self.gpu.h, xd, T, pos0, o)
        sid, o64 = self.orc.materialize(x64, pos0=pos0)
        self.sid[h] = sid
        torch.cuda.synchronize()
        close(to_np(o), o64, self.dt, "materialize output")
        self._after(h)
        return h

    def fork(self, h, k: int):
        kids = kv.kv_fork(self.gpu.h, h, k)
        okids = self.orc.fork(self.sid[h], k)
        for a, b in zip(kids, okids):
            self.sid[a] = b
            if h in self.rerot:
                self.rerot[a] = self.rerot[h]
        self._after()
        return kids

    def attend(self, hs, T: int, tag: int = None):
        b = len(hs)
        xd, x64 = self.x(b * T, self.calls if tag is None else tag)
        s = self.s
        o = torch.empty((s.n_layers, b, T, s.n_q_heads * s.head_dim), dtype=self.tdt,
                        device="cuda")
        kv.kv_attend(self.gpu.h, hs, xd, T, o)
        o64 = self.orc.attend([self.sid[h] for h in hs], x64.reshape(b, T, -1))
        torch.cuda.synchronize()
        close(to_np(o), o64, self.dt, "attend output")
        self._after(*hs)
        return o

    def compose(self, segs):
        h = kv.kv_compose(self.gpu.h, segs)
        sid = self.orc.compose([(self.sid[a], b, c) for a, b, c in segs])
        self.sid[h] = sid
        torch.cuda.synchronize()
        self.check_compose_kv(h, segs)   # shifted segments carry re-rotated keys
        self._after(h)
        return h

    def pack(self, h, b0: int, b1: int):
        nbytes = (b1 - b0) * self.s.block_bytes
        buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        hdr = kv.kv_pack(self.gpu.h, h, b0, b1, buf)
        ohdr, payload = self.orc.pack(self.sid[h], b0, b1)
        assert (hdr.pos_begin, hdr.n_tokens, hdr.blk_begin, hdr.n_blocks, hdr.block_bytes,
                hdr.payload_bytes, hdr.lineage, hdr.src_state_id) == \
            (ohdr["pos_begin"], ohdr["n_tokens"], ohdr["blk_begin"], ohdr["n_blocks"],
             ohdr["block_bytes"], ohdr["payload_bytes"], ohdr["lineage"], ohdr["src_state_id"])
        torch.cuda.synchronize()
        s = self.s
        got = to_np(buf.view(self.tdt).view(payload.shape))
        self.last_pack_raw = buf
        close(got, payload, self.dt, "packed payload")
        # invalid slots of the last block are zero on both sides, exactly
        last_valid = ohdr["n_tokens"] - (ohdr["n_blocks"] - 1) * s.block_size
        assert np.all(got[-1, :, :, :, last_valid:] == 0)
        self._after()
        return hdr, ohdr, buf, payload

    def unpack(self, hdr, ohdr, buf, payload64, rerotated_from=None):
        """Device unpacks its buffer, the oracle its own payload.
        rerotated_from: the composed state the buffer was packed from (its
        recorded keys then apply to the unpacked state)."""
        h = kv.kv_unpack(self.gpu.h, hdr, buf)
        sid = self.orc.unpack(ohdr, payload64)
        self.sid[h] = sid
        if rerotated_from is not None:
            lo = hdr.blk_begin * self.s.block_size
            self.rerot[h] = [k[:, lo:lo + hdr.n_tokens] for k in self.rerot[rerotated_from]]
        self._after(h)
        return h

    def synthetic_transfer(self, n_blocks: int, n_tokens: int, pos_begin: int, tag: int):
        """A seeded payload (same stored values on both sides) with its header."""
        s = self.s
        shp = (n_blocks, s.n_layers, 2, s.n_kv_heads, s.block_size, s.head_dim)
        key = synth.payload_key(self.seed, self.wl, tag)
        buf = synth.normal_torch(key, shp, 1.0, self.dt, "cuda").contiguous()
        pay = synth.to_f64(synth.normal_np(key, shp, 1.0, self.dt), self.dt)
        hdr = kv.kv_pack_header()
        hdr.magic, hdr.version, hdr.model_id = kv.KV_PACK_MAGIC, kv.KV_PACK_VERSION, \
            self.cfg.model_id
        hdr.cfg = self.cfg
        hdr.pos_begin, hdr.n_tokens, hdr.blk_begin, hdr.n_blocks = pos_begin, n_tokens, 0, n_blocks
        hdr.block_bytes = s.block_bytes
        hdr.payload_bytes = n_blocks * s.block_bytes
        hdr.lineage, hdr.src_state_id = 0, 1000 + tag
        ohdr = dict(magic=kv.KV_PACK_MAGIC, version=kv.KV_PACK_VERSION,
                    model_id=self.orc.shape.model_id, compat=self.orc.shape.compat_key(),
                    pos_begin=pos_begin, n_tokens=n_tokens, blk_begin=0, n_blocks=n_blocks,
                    block_bytes=s.block_bytes, payload_bytes=n_blocks * s.block_bytes,
                    lineage=0, src_state_id=1000 + tag)
        return hdr, ohdr, buf.view(torch.uint8).reshape(-1), pay

    def evict(self, max_alloc: int, a=0.0, b=0.0, g=1.0):
        n = kv.kv_evict(self.gpu.h, max_alloc, a, b, g)
        no = self.orc.evict(max_alloc, a, b, g)
        assert n == no
        self._after()
        return n

    def evict_truncate(self, max_alloc: int, a=0.0, b=0.0, g=1.0):
        r = kv.kv_evict_truncate(self.gpu.h, max_alloc, a, b, g)
        ro = self.orc.evict_truncate(max_alloc, a, b, g)
        assert r == ro
        self._after()
        return r

    def release(self, h):
        kv.kv_release(self.gpu.h, h)
        self.orc.release(self.sid[h])
        self._after()

    def close(self):
        self.gpu.close()
