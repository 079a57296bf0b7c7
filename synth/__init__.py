"""Seeded synthetic inputs for the KV-state operators.

This module is shared by the float64 oracle and by the device path's tests and
benchmark. It holds no arithmetic of the operators themselves: only workload
shapes, a counter-based integer hash and a quantile table of the normal
distribution.

Generator definition (the same bits on every device):

* A stream is named by a tuple of small integers ``key`` (seed, tensor kind,
  workload, layer, agent, step).  ``stream_id(key)`` folds it into 32 bits with
  the ``lowbias32`` integer finaliser (Wellons, "Prospecting for Hash
  Functions", 2018: xor-shift 16, multiply 0x7feb352d, xor-shift 15, multiply
  0x846ca68b, xor-shift 16).
* Element ``i`` of a stream draws ``h = mix(mix(i * 0x9E3779B9 + s) ^ s2)``
  (all mod 2**32), with ``s = stream_id(key)`` and ``s2 = mix(s ^ 0x9E3779B9)``.
* The top 16 bits of ``h`` index a table of 65536 normal quantiles
  ``std * Phi^-1((j + 0.5) / 65536)`` (float64, scipy's ``ndtri``), rounded
  to the storage type: float32 by round-to-nearest-even, bf16 by
  round-to-nearest-even from that float32.  The draw is N(0, std^2)
  discretised to 65536 equiprobable values and truncated at about 4.3 std.

The CPU (NumPy, uint32 arithmetic) and torch (int64 arithmetic reduced mod
2**32, any device) implementations produce identical bits; a CPU test pins
them against each other.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace
from functools import lru_cache

import numpy as np

MASK32 = 0xFFFFFFFF
GOLDEN = 0x9E3779B9
_C1 = 0x7FEB352D
_C2 = 0x846CA68B

# tensor kinds used in stream keys
KIND_X = 1          # hidden states fed to materialize / append
KIND_W = 2          # per-layer QKV weights
KIND_XDEC = 3       # per-step decode rows
KIND_PAYLOAD = 4    # synthetic transfer buffers (pack/unpack round trips)
KIND_PERM = 5       # block-id permutations


# ---------------------------------------------------------------- workloads

@dataclass(frozen=True)
class ModelShape:
    """Shape of the KV cache a workload runs on (a Llama-like attention stack)."""
    name: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    block_size: int
    dtype: str          # "f32" or "bf16"
    rope_base: float = 10000.0

    @property
    def qkv_cols(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def elt_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def block_bytes(self) -> int:
        return (self.n_layers * 2 * self.n_kv_heads * self.block_size
                * self.head_dim * self.elt_bytes)

    @property
    def w_std(self) -> float:
        return 1.0 / math.sqrt(self.d_model)


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: a shared context, agents, suffixes, decode steps."""
    name: str
    shape: ModelShape
    context: int            # tokens of the shared (materialized) context
    agents: int             # fork / compose fan-out
    suffix: int             # tokens each agent appends
    decode: int             # decode steps after the append
    extra: dict = field(default_factory=dict)

    def with_shape(self, **kw) -> "Workload":
        return replace(self, shape=replace(self.shape, **kw))


TINY_SHAPE = ModelShape("tiny", 1, 256, 4, 2, 64, 16, "f32")
LLAMA8B_SHAPE = ModelShape("llama3-8b", 32, 4096, 32, 8, 128, 16, "bf16")
LLAMA70B_SHAPE = ModelShape("llama3-70b", 80, 8192, 64, 8, 128, 32, "bf16")

WORKLOADS = {
    # 256-token context forked to 2 agents (+32 each), composed, 8 decode steps
    "tiny": Workload("tiny", TINY_SHAPE, context=256, agents=2, suffix=32, decode=8),
    # 8192-token context forked to 4 agents, 512-token prompts, 128 decode steps
    "fork4-8b": Workload("fork4-8b", LLAMA8B_SHAPE, context=8192, agents=4, suffix=512,
                         decode=128),
    # 32768-token context forked to 16 agents with 1024-token suffixes;
    # batched decode and LRU churn freeing 25% of blocks for 10 rounds
    "fanout16-8b": Workload("fanout16-8b", LLAMA8B_SHAPE, context=32768, agents=16,
                            suffix=1024, decode=64,
                            extra={"evict_rounds": 10, "evict_frac": 0.25}),
    # 8 agents x 4096-token segments composed into one 32768-token cache,
    # then a 2048-token append and 256 decode steps
    "compose8-8b": Workload("compose8-8b", LLAMA8B_SHAPE, context=4096, agents=8,
                            suffix=2048, decode=256),
    # 70B-shaped 16384-token context: pack, unpack into a permuted table,
    # 4-agent fork and decode
    "pack70b": Workload("pack70b", LLAMA70B_SHAPE, context=16384, agents=4, suffix=0,
                        decode=64),
}


# ---------------------------------------------------------------- hashing

def _mix32_int(x: int) -> int:
    x &= MASK32
    x ^= x >> 16
    x = (x * _C1) & MASK32
    x ^= x >> 15
    x = (x * _C2) & MASK32
    x ^= x >> 16
    return x


def stream_id(key) -> int:
    """Fold a tuple of non-negative integers into a 32-bit stream id."""
    s = 0x2545F491
    for k in key:
        k = int(k)
        if k < 0:
            raise ValueError("stream key entries must be non-negative")
        while True:
            s = _mix32_int(s ^ (k & MASK32))
            k >>= 32
            if k == 0:
                break
    return s


def _mix32_np(x: np.ndarray) -> np.ndarray:
    x = x ^ (x >> np.uint32(16))
    x = x * np.uint32(_C1)
    x = x ^ (x >> np.uint32(15))
    x = x * np.uint32(_C2)
    x = x ^ (x >> np.uint32(16))
    return x


def hash_np(key, start: int, n: int) -> np.ndarray:
    """32-bit draws for elements [start, start+n) of stream ``key`` (NumPy)."""
    s = stream_id(key)
    s2 = _mix32_int(s ^ GOLDEN)
    with np.errstate(over="ignore"):
        i = np.arange(start, start + n, dtype=np.uint64).astype(np.uint32)
        h = _mix32_np(i * np.uint32(GOLDEN) + np.uint32(s))
        h = _mix32_np(h ^ np.uint32(s2))
    return h


def _mulmod32_t(x, c: int):
    lo, hi = c & 0xFFFF, c >> 16
    return (x * lo + (((x * hi) & 0xFFFF) << 16)) & MASK32


def _mix32_t(x):
    x = x ^ (x >> 16)
    x = _mulmod32_t(x, _C1)
    x = x ^ (x >> 15)
    x = _mulmod32_t(x, _C2)
    x = x ^ (x >> 16)
    return x


def hash_torch(key, start: int, n: int, device):
    """Same draws as :func:`hash_np`, computed with torch int64 ops on ``device``."""
    import torch
    s = stream_id(key)
    s2 = _mix32_int(s ^ GOLDEN)
    i = torch.arange(start, start + n, dtype=torch.int64, device=device) & MASK32
    h = _mix32_t((_mulmod32_t(i, GOLDEN) + s) & MASK32)
    h = _mix32_t(h ^ s2)
    return h


# ---------------------------------------------------------------- quantile tables

def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); return uint16 bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact float64 values of bf16 bit patterns."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


@lru_cache(maxsize=32)
def _quantiles(std: float) -> np.ndarray:
    from scipy.special import ndtri
    j = np.arange(65536, dtype=np.float64)
    return std * ndtri((j + 0.5) / 65536.0)


@lru_cache(maxsize=32)
def normal_table(std: float, dtype: str) -> np.ndarray:
    """Storage values of the 65536 quantiles: float32 array or bf16 uint16 bits."""
    q = _quantiles(float(std)).astype(np.float32)
    if dtype == "f32":
        return q
    if dtype == "bf16":
        return f32_to_bf16_bits(q)
    raise ValueError(dtype)


def normal_np(key, shape, std: float, dtype: str) -> np.ndarray:
    """Seeded N(0, std^2) draws as storage values (float32, or bf16 uint16 bits)."""
    n = int(np.prod(shape))
    idx = (hash_np(key, 0, n) >> np.uint32(16)).astype(np.int64)
    return normal_table(float(std), dtype)[idx].reshape(shape)


def normal_rows_np(key, row_len: int, rows, std: float, dtype: str) -> np.ndarray:
    """Selected rows of a stream viewed as [*, row_len] (for sampled checks)."""
    rows = np.asarray(rows, dtype=np.int64).reshape(-1)
    out = []
    tab = normal_table(float(std), dtype)
    for r in rows:
        h = hash_np(key, int(r) * row_len, row_len)
        out.append(tab[(h >> np.uint32(16)).astype(np.int64)])
    return np.stack(out) if out else np.zeros((0, row_len), dtype=tab.dtype)


def to_f64(stored: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of stored inputs."""
    if dtype == "bf16":
        return bf16_bits_to_f64(stored)
    return np.asarray(stored, dtype=np.float32).astype(np.float64)


def normal_torch(key, shape, std: float, dtype: str, device, start: int = 0):
    """Same values as :func:`normal_np`, generated by torch on ``device``.

    Elements [start, start + prod(shape)) of the stream; returns a float32 or
    bfloat16 tensor.
    """
    import torch
    n = int(np.prod(shape))
    tab_np = normal_table(float(std), dtype)
    if dtype == "bf16":
        tab = torch.from_numpy(tab_np.view(np.int16).copy()).to(device)
    else:
        tab = torch.from_numpy(tab_np.copy()).to(device)
    out = torch.empty(n, dtype=tab.dtype, device=device)
    chunk = 1 << 26
    for s in range(0, n, chunk):
        m = min(chunk, n - s)
        idx = hash_torch(key, start + s, m, device) >> 16
        out[s:s + m] = tab[idx]
    if dtype == "bf16":
        out = out.view(torch.bfloat16)
    return out.reshape(shape)


# ---------------------------------------------------------------- keyed inputs

def x_key(seed: int, wl: str, call: int, agent: int = 0):
    return (seed, KIND_X, _wl_id(wl), call, agent)


def w_key(seed: int, wl: str, layer: int):
    return (seed, KIND_W, _wl_id(wl), layer)


def xdec_key(seed: int, wl: str, agent: int, step: int):
    return (seed, KIND_XDEC, _wl_id(wl), agent, step)


def payload_key(seed: int, wl: str, call: int):
    return (seed, KIND_PAYLOAD, _wl_id(wl), call)


def _wl_id(name: str) -> int:
    # a stable small integer per workload name
    return stream_id(tuple(name.encode()))


def permutation(seed: int, wl: str, n: int, tag: int = 0) -> np.ndarray:
    """Seeded permutation of 0..n-1 (host side, NumPy's PCG64)."""
    rng = np.random.default_rng(np.random.SeedSequence(
        [seed, KIND_PERM, _wl_id(wl), tag]))
    return rng.permutation(n).astype(np.int32)


def normal_f64(key, shape, std: float, dtype: str, start: int = 0, device="cpu"):
    """Float64 values of the stored inputs, generated with torch on ``device``
    and returned as a host array (the same bits as :func:`normal_np` on any
    device; faster for large tensors)."""
    import torch
    t = normal_torch(key, shape, std, dtype, device, start=start)
    return t.to(torch.float64).cpu().numpy()
