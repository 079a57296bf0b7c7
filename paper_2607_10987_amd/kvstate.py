"""ctypes binding of the C ABI in include/kvstate.h (argument marshalling only).

Functions keep the C names.  Device buffers are passed as torch tensors (their
``data_ptr()``) or as integer addresses; streams default to torch's current
stream.  Every non-zero status raises :class:`KVError`.  The library must be
built (``__graft_entry__.build()``); nothing here computes anything itself.
"""
from __future__ import annotations

import ctypes
import os
import re

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkvstate.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "kvstate.h")

KV_OK = 0
KV_ERR_ARG = -1
KV_ERR_OOM = -2
KV_ERR_INCOMPATIBLE = -3
KV_ERR_EVICTED = -4
KV_ERR_BAD_HEADER = -5
KV_ERR_BUFSIZE = -6
KV_ERR_CAPACITY = -7
KV_ERR_HIP = -8
KV_ERR_INTERNAL = -9
KV_ERR_CHECKSUM = -10
KV_ERR_IO = -11
KV_DTYPE_F32 = 0
KV_DTYPE_BF16 = 1
KV_PACK_MAGIC = 0x5453564B
KV_PACK_VERSION = 2
KV_PACK_CHECKSUM = 1
KV_MAX_BATCH = 64
KV_MAX_SEGMENTS = 64
KV_MAX_FORK = 64
KV_NOALLOC_SCRATCH_MB = 64


class kv_model_cfg(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("max_pos", ctypes.c_int32),
                ("max_states", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("rope_base", ctypes.c_double), ("model_id", ctypes.c_uint64)]


class kv_segment(ctypes.Structure):
    _fields_ = [("state", ctypes.c_int64), ("tok_begin", ctypes.c_int64),
                ("tok_end", ctypes.c_int64)]


class kv_pack_header(ctypes.Structure):
    _fields_ = [("magic", ctypes.c_uint32), ("version", ctypes.c_uint32),
                ("model_id", ctypes.c_uint64), ("cfg", kv_model_cfg),
                ("pos_begin", ctypes.c_int64), ("n_tokens", ctypes.c_int64),
                ("blk_begin", ctypes.c_int64), ("n_blocks", ctypes.c_int64),
                ("block_bytes", ctypes.c_uint64), ("payload_bytes", ctypes.c_uint64),
                ("lineage", ctypes.c_uint64), ("src_state_id", ctypes.c_int64),
                ("flags", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
                ("checksum", ctypes.c_uint64 * 2)]


class KVError(RuntimeError):
    def __init__(self, status: int, where: str = ""):
        self.status = status
        super().__init__(f"{where}: {kv_strerror(status)} ({status})")


_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t
_PI64 = ctypes.POINTER(ctypes.c_int64)
_PI32 = ctypes.POINTER(ctypes.c_int32)
_PU64 = ctypes.POINTER(ctypes.c_uint64)
_PCFG = ctypes.POINTER(kv_model_cfg)
_PHDR = ctypes.POINTER(kv_pack_header)

_SIGS = {
    "kv_pool_bytes": (_I32, [_PCFG, _I64, ctypes.POINTER(_SZ), ctypes.POINTER(_SZ)]),
    "kv_scratch_bytes": (_SZ, [_PCFG, _I64, _I32, _I64]),
    "kv_pool_create": (_I32, [_PCFG, _I64, _P, _P, _P, _SZ, _PI32, _P, ctypes.POINTER(_P)]),
    "kv_pool_destroy": (_I32, [_P]),
    "kv_set_weights": (_I32, [_P, _P, _I64]),
    "kv_materialize": (_I32, [_P, _P, _I64, _I64, _P, _P, _PI64]),
    "kv_fork": (_I32, [_P, _I64, _I32, _PI64, _P]),
    "kv_compose": (_I32, [_P, ctypes.POINTER(kv_segment), _I32, _P, _PI64]),
    "kv_pack": (_I32, [_P, _I64, _I64, _I64, _P, _SZ, _PHDR, _P]),
    "kv_unpack": (_I32, [_P, _PHDR, _P, _SZ, _P, _PI64]),
    "kv_pack_checked": (_I32, [_P, _I64, _I64, _I64, _P, _SZ, _PHDR, _P]),
    "kv_checkpoint_save": (_I32, [_P, _I64, ctypes.c_char_p, _P]),
    "kv_checkpoint_load": (_I32, [_P, ctypes.c_char_p, _P, _PI64]),
    "kv_attend": (_I32, [_P, _PI64, _I32, _P, _I64, _P, _P]),
    "kv_attend_noalloc": (_I32, [_P, _PI64, _I32, _P, _I64, _P, _P]),
    "kv_evict": (_I32, [_P, _I64, ctypes.c_double, ctypes.c_double, ctypes.c_double, _P, _PI32]),
    "kv_evict_truncate": (_I32, [_P, _I64, ctypes.c_double, ctypes.c_double, ctypes.c_double, _P,
                                 _PI32, _PI32]),
    "kv_release": (_I32, [_P, _I64, _P]),
    "kv_pin": (_I32, [_P, _I64, _I32]),
    "kv_sync": (_I32, [_P, _P]),
    "kv_state_info": (_I32, [_P, _I64, _PI64, _PI64, _PI64, _PU64, _PI64]),
    "kv_pool_counts": (_I32, [_P, _PI64, _PI64, _PI64]),
    "kv_state_usage": (_I32, [_P, _I64, _PI64, _PI64, _PI32]),
    "kv_read_block_table": (_I32, [_P, _I64, _PI32, _I64, _P]),
    "kv_read_allocator": (_I32, [_P, _PI32, _PI32, _PI64, _PI64, _P]),
    "kv_strerror": (ctypes.c_char_p, [_I32]),
    "kv_plan_transfer": (_I32, [_P, _I64, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                ctypes.c_double, ctypes.c_double, _P]),
    "kv_profile_enable": (_I32, [_P, _I32]),
    "kv_profile_read": (_I32, [_P, ctypes.c_void_p]),
    "kv_profile_launches": (_I32, [_P, _I32, ctypes.POINTER(ctypes.c_float), _I64, _PI64]),
}

_lib = None


def lib():
    """Load libkvstate.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def header_functions():
    """Names of the functions declared in include/kvstate.h."""
    src = open(HEADER_PATH).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(kv_[a-z_]+)\s*\(", src)))


def _ptr(t) -> int:
    if t is None:
        return 0
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(st: int, where: str):
    if st != KV_OK:
        raise KVError(st, where)


# configuration of each live pool handle, for the tensor checks below
_CFGS: dict = {}


def _check_tensor(t, pool, min_elems: int, where: str):
    """A torch tensor handed to a kernel must be a contiguous CUDA tensor of
    the pool's dtype with at least ``min_elems`` elements; raise KVError
    before the call otherwise.  Raw integer addresses are left to the
    library's own checks."""
    if t is None or isinstance(t, int):
        return
    cfg = _CFGS.get(pool)
    if not getattr(t, "is_cuda", False) or not t.is_contiguous():
        raise KVError(KV_ERR_ARG, where)
    if cfg is not None:
        import torch
        want = torch.bfloat16 if cfg.dtype == KV_DTYPE_BF16 else torch.float32
        if t.dtype != want:
            raise KVError(KV_ERR_ARG, where)
    if t.numel() < min_elems:
        raise KVError(KV_ERR_BUFSIZE, where)


def kv_strerror(status: int) -> str:
    return lib().kv_strerror(status).decode()


def make_cfg(n_layers, d_model, n_q_heads, n_kv_heads, head_dim, block_size, dtype, max_pos,
             max_states, rope_base=10000.0, model_id=1) -> kv_model_cfg:
    dt = {"f32": KV_DTYPE_F32, "bf16": KV_DTYPE_BF16}.get(dtype, dtype)
    return kv_model_cfg(n_layers, d_model, n_q_heads, n_kv_heads, head_dim, block_size, dt,
                        max_pos, max_states, 0, float(rope_base), int(model_id))


def kv_pool_bytes(cfg: kv_model_cfg, n_blocks: int):
    a, b = _SZ(), _SZ()
    _check(lib().kv_pool_bytes(ctypes.byref(cfg), n_blocks, ctypes.byref(a), ctypes.byref(b)),
           "kv_pool_bytes")
    return a.value, b.value


def kv_scratch_bytes(cfg: kv_model_cfg, tokens: int, batch: int, max_keys: int) -> int:
    return lib().kv_scratch_bytes(ctypes.byref(cfg), tokens, batch, max_keys)


def kv_pool_create(cfg, n_blocks, pool, meta, scratch, scratch_bytes=None,
                   init_free_order=None, stream=None):
    order = None
    if init_free_order is not None:
        arr = (ctypes.c_int32 * n_blocks)(*[int(v) for v in init_free_order])
        order = ctypes.cast(arr, _PI32)
    if scratch_bytes is None:
        scratch_bytes = _nbytes(scratch) if scratch is not None else 0
    out = _P()
    _check(lib().kv_pool_create(ctypes.byref(cfg), n_blocks, _ptr(pool), _ptr(meta),
                                _ptr(scratch), scratch_bytes, order, _stream(stream),
                                ctypes.byref(out)), "kv_pool_create")
    _CFGS[out.value] = kv_model_cfg.from_buffer_copy(cfg)
    return out.value


def kv_pool_destroy(pool):
    _CFGS.pop(pool, None)
    _check(lib().kv_pool_destroy(pool), "kv_pool_destroy")


def _qkv_cols(c) -> int:
    return (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim


def kv_set_weights(pool, w, layer_stride_elems: int):
    c = _CFGS.get(pool)
    if c is not None:
        per = _qkv_cols(c) * c.d_model
        _check_tensor(w, pool, (c.n_layers - 1) * max(layer_stride_elems, 0) + per,
                      "kv_set_weights")
    _check(lib().kv_set_weights(pool, _ptr(w), layer_stride_elems), "kv_set_weights")


def kv_materialize(pool, x, T: int, pos0: int, o, stream=None) -> int:
    c = _CFGS.get(pool)
    if c is not None:
        _check_tensor(x, pool, T * c.d_model, "kv_materialize x")
        _check_tensor(o, pool, c.n_layers * T * c.n_q_heads * c.head_dim, "kv_materialize o")
    out = _I64()
    _check(lib().kv_materialize(pool, _ptr(x), T, pos0, _ptr(o), _stream(stream),
                                ctypes.byref(out)), "kv_materialize")
    return out.value


def kv_fork(pool, parent: int, k: int, stream=None):
    arr = (ctypes.c_int64 * max(k, 1))()
    _check(lib().kv_fork(pool, parent, k, arr, _stream(stream)), "kv_fork")
    return list(arr)[:k]


def kv_compose(pool, segs, stream=None) -> int:
    n = len(segs)
    arr = (kv_segment * max(n, 1))(*[kv_segment(int(s), int(a), int(e)) for s, a, e in segs])
    out = _I64()
    _check(lib().kv_compose(pool, arr, n, _stream(stream), ctypes.byref(out)), "kv_compose")
    return out.value


def kv_pack(pool, state: int, blk_begin: int, blk_end: int, dst, dst_bytes=None, stream=None):
    hdr = kv_pack_header()
    if dst_bytes is None:
        dst_bytes = _nbytes(dst)
    _check(lib().kv_pack(pool, state, blk_begin, blk_end, _ptr(dst), dst_bytes,
                         ctypes.byref(hdr), _stream(stream)), "kv_pack")
    return hdr


def kv_pack_checked(pool, state: int, blk_begin: int, blk_end: int, dst, dst_bytes=None,
                    stream=None):
    hdr = kv_pack_header()
    if dst_bytes is None:
        dst_bytes = _nbytes(dst)
    _check(lib().kv_pack_checked(pool, state, blk_begin, blk_end, _ptr(dst), dst_bytes,
                                 ctypes.byref(hdr), _stream(stream)), "kv_pack_checked")
    return hdr


def kv_checkpoint_save(pool, state: int, path: str, stream=None):
    _check(lib().kv_checkpoint_save(pool, state, os.fsencode(path), _stream(stream)),
           "kv_checkpoint_save")


def kv_checkpoint_load(pool, path: str, stream=None) -> int:
    out = _I64()
    _check(lib().kv_checkpoint_load(pool, os.fsencode(path), _stream(stream), ctypes.byref(out)),
           "kv_checkpoint_load")
    return out.value


def kv_unpack(pool, hdr: kv_pack_header, src, src_bytes=None, stream=None) -> int:
    if src_bytes is None:
        src_bytes = _nbytes(src)
    out = _I64()
    _check(lib().kv_unpack(pool, ctypes.byref(hdr), _ptr(src), src_bytes, _stream(stream),
                           ctypes.byref(out)), "kv_unpack")
    return out.value


def kv_attend(pool, states, x, T: int, o, stream=None):
    n = len(states)
    c = _CFGS.get(pool)
    if c is not None:
        _check_tensor(x, pool, n * T * c.d_model, "kv_attend x")
        _check_tensor(o, pool, c.n_layers * n * T * c.n_q_heads * c.head_dim, "kv_attend o")
    arr = (ctypes.c_int64 * max(n, 1))(*[int(s) for s in states])
    _check(lib().kv_attend(pool, arr, n, _ptr(x), T, _ptr(o), _stream(stream)), "kv_attend")


def kv_attend_noalloc(pool, states, x, T: int, o, stream=None):
    n = len(states)
    c = _CFGS.get(pool)
    if c is not None:
        _check_tensor(x, pool, n * T * c.d_model, "kv_attend_noalloc x")
        _check_tensor(o, pool, c.n_layers * n * T * c.n_q_heads * c.head_dim,
                      "kv_attend_noalloc o")
    arr = (ctypes.c_int64 * max(n, 1))(*[int(s) for s in states])
    _check(lib().kv_attend_noalloc(pool, arr, n, _ptr(x), T, _ptr(o), _stream(stream)),
           "kv_attend_noalloc")


def kv_evict(pool, max_allocated_blocks: int, alpha=0.0, beta=0.0, gamma=1.0, stream=None) -> int:
    n = _I32()
    _check(lib().kv_evict(pool, max_allocated_blocks, alpha, beta, gamma, _stream(stream),
                          ctypes.byref(n)), "kv_evict")
    return n.value


def kv_evict_truncate(pool, max_allocated_blocks: int, alpha=0.0, beta=0.0, gamma=1.0,
                      stream=None):
    """Returns (states evicted whole, states truncated to their shared prefix)."""
    ne, nt = _I32(), _I32()
    _check(lib().kv_evict_truncate(pool, max_allocated_blocks, alpha, beta, gamma,
                                   _stream(stream), ctypes.byref(ne), ctypes.byref(nt)),
           "kv_evict_truncate")
    return ne.value, nt.value


def kv_release(pool, state: int, stream=None):
    _check(lib().kv_release(pool, state, _stream(stream)), "kv_release")


def kv_pin(pool, state: int, pinned: bool):
    _check(lib().kv_pin(pool, state, 1 if pinned else 0), "kv_pin")


def kv_sync(pool, stream=None):
    _check(lib().kv_sync(pool, _stream(stream)), "kv_sync")


def kv_state_info(pool, state: int):
    a, b, c, e = _I64(), _I64(), _I64(), _I64()
    lin = ctypes.c_uint64()
    _check(lib().kv_state_info(pool, state, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c),
                               ctypes.byref(lin), ctypes.byref(e)), "kv_state_info")
    return dict(pos0=a.value, n_tokens=b.value, n_blocks=c.value, lineage=lin.value,
                state_id=e.value)


def kv_state_usage(pool, state: int):
    a, b = _I64(), _I64()
    c = _I32()
    _check(lib().kv_state_usage(pool, state, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)),
           "kv_state_usage")
    return dict(reuse=a.value, last_access=b.value, pinned=bool(c.value))


def kv_pool_counts(pool):
    a, b, c = _I64(), _I64(), _I64()
    _check(lib().kv_pool_counts(pool, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)),
           "kv_pool_counts")
    return dict(free_blocks=a.value, live_states=b.value, clock=c.value)


def kv_read_block_table(pool, state: int, stream=None):
    nb = kv_state_info(pool, state)["n_blocks"]
    arr = (ctypes.c_int32 * max(nb, 1))()
    _check(lib().kv_read_block_table(pool, state, arr, nb, _stream(stream)),
           "kv_read_block_table")
    return list(arr)[:nb]


def kv_read_allocator(pool, n_blocks: int, stream=None):
    rc = (ctypes.c_int32 * n_blocks)()
    ring = (ctypes.c_int32 * n_blocks)()
    h, t = _I64(), _I64()
    _check(lib().kv_read_allocator(pool, rc, ring, ctypes.byref(h), ctypes.byref(t),
                                   _stream(stream)), "kv_read_allocator")
    return list(rc), list(ring), h.value, t.value


KERNEL_KINDS = ["alloc", "fork", "release", "compose_meta", "compose_copy", "pack", "unpack",
                "cow", "qkv", "qkv_decode", "attn", "attn_decode", "merge"]


class kv_transfer_plan(ctypes.Structure):
    _fields_ = [("kv_bytes", ctypes.c_double), ("t_transfer", ctypes.c_double),
                ("t_prefill", ctypes.c_double), ("prefill_flops", ctypes.c_double),
                ("transfer", ctypes.c_int32), ("pad", ctypes.c_int32)]


def kv_plan_transfer(cfg: kv_model_cfg, n_tokens: int, link_bytes_per_s: float,
                     link_latency_s: float, pack_bytes_per_s: float, unpack_bytes_per_s: float,
                     prefill_flops_per_s: float) -> dict:
    """Transfer-vs-recompute decision (host only; see include/kvstate.h)."""
    out = kv_transfer_plan()
    _check(lib().kv_plan_transfer(ctypes.byref(cfg), n_tokens, link_bytes_per_s, link_latency_s,
                                  pack_bytes_per_s, unpack_bytes_per_s, prefill_flops_per_s,
                                  ctypes.byref(out)), "kv_plan_transfer")
    return {"kv_bytes": out.kv_bytes, "t_transfer": out.t_transfer, "t_prefill": out.t_prefill,
            "prefill_flops": out.prefill_flops, "transfer": bool(out.transfer)}


class kv_profile_entry(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_int64), ("total_ms", ctypes.c_double)]


def kv_profile_enable(pool, enabled: bool):
    _check(lib().kv_profile_enable(pool, 1 if enabled else 0), "kv_profile_enable")


def kv_profile_launches(pool, kind: str):
    """Durations (ms) of the individual launches of `kind` since the last
    kv_profile_read, in launch order."""
    k = KERNEL_KINDS.index(kind)
    n = _I64()
    _check(lib().kv_profile_launches(pool, k, None, 0, ctypes.byref(n)), "kv_profile_launches")
    arr = (ctypes.c_float * max(n.value, 1))()
    _check(lib().kv_profile_launches(pool, k, arr, n.value, ctypes.byref(n)),
           "kv_profile_launches")
    return list(arr)[:n.value]


def kv_profile_read(pool):
    """{kind: (launches, total_ms)} since the last read."""
    arr = (kv_profile_entry * len(KERNEL_KINDS))()
    _check(lib().kv_profile_read(pool, ctypes.cast(arr, ctypes.c_void_p)), "kv_profile_read")
    return {k: (arr[i].launches, arr[i].total_ms) for i, k in enumerate(KERNEL_KINDS)}


class Pool:
    """A pool plus the torch device buffers that back it (memory plumbing)."""

    def __init__(self, cfg: kv_model_cfg, n_blocks: int, scratch_bytes: int,
                 init_free_order=None, device="cuda", stream=None):
        import torch
        self.cfg = cfg
        self.n_blocks = n_blocks
        pb, mb = kv_pool_bytes(cfg, n_blocks)
        self.pool_t = torch.empty(pb, dtype=torch.uint8, device=device)
        self.meta_t = torch.empty(mb, dtype=torch.uint8, device=device)
        self.scratch_t = torch.empty(max(scratch_bytes, 256), dtype=torch.uint8, device=device)
        self.h = kv_pool_create(cfg, n_blocks, self.pool_t, self.meta_t, self.scratch_t,
                                init_free_order=init_free_order, stream=stream)
        self.w = None

    def set_weights(self, w, layer_stride_elems: int):
        self.w = w
        kv_set_weights(self.h, w, layer_stride_elems)

    def blocks_view(self):
        """The pool memory as [P, L, 2, Hkv, B, dh] of the storage dtype."""
        import torch
        c = self.cfg
        dt = torch.bfloat16 if c.dtype == KV_DTYPE_BF16 else torch.float32
        return self.pool_t.view(dt).view(self.n_blocks, c.n_layers, 2, c.n_kv_heads,
                                         c.block_size, c.head_dim)

    def close(self):
        if self.h:
            kv_pool_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
