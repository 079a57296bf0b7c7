// Data-movement kernels over paged blocks: pack (gather a block range into a
// contiguous transfer buffer), unpack (scatter a buffer into freshly allocated
// blocks), copy-on-write of a shared partial tail block, and the token-granular
// gather of compose with RoPE re-rotation of keys.
//
// All of them are HBM-bound streams of 16-byte vector accesses; every byte is
// moved once.  Pack and unpack cut each (block, layer) slab of
// 2 * Hkv * B * dh elements (64 KiB for an 8B-shaped bf16 block with B = 16)
// into 4 KiB pieces, one per workgroup of 256 threads, one 16-byte load per
// thread: with the last-level cache flushed before each call, this measured
// 84% of HBM peak for both on the 70B shape, against 74% / 71% for 8 KiB
// pieces with two loads per thread (and less for 2 KiB, 16 KiB or more loads
// in flight per thread).  Compose moves one slab per workgroup.  Streaming
// loads and stores past the caches with non-temporal accesses measured 5-15%
// faster (unpack's scattered block writes included, since the 4 KiB pieces).
#include "kv_internal.h"

namespace kvs {

namespace {

constexpr int kMoveThreads = 256;  // compose, copy-on-write, checksum folding
constexpr int kPackThreads = 256;  // pack / unpack workgroups
constexpr int kUnroll = 1;         // 16-byte loads in flight per pack / unpack thread

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__device__ inline uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);  // quiet NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ inline void st_nt(uint4* p, const uint4& v) {
  __builtin_nontemporal_store((u32x4){v.x, v.y, v.z, v.w}, (u32x4*)p);
}

__device__ inline uint4 ld_nt(const uint4* p) {
  const u32x4 v = __builtin_nontemporal_load((const u32x4*)p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Bytes one workgroup moves: (block, layer) slabs are cut into pieces of
// this size (grid z), each thread keeping kUnroll 16-byte loads in flight.
constexpr int kPiece = kPackThreads * kUnroll * 16;

// Workgroup w of a (pieces x L x blocks) launch, piece fastest: consecutive
// workgroups walk a block's layers and pieces in address order.
struct PieceIdx {
  int piece, layer, block;
};
__device__ inline PieceIdx piece_idx(int pieces, int L) {
  const int w = blockIdx.x;
  return {w % pieces, (w / pieces) % L, w / (pieces * L)};
}

// Copy piece `piece` of a slab of n16 16-byte chunks; chunk c belongs to
// slot (c / row16) % B and is replaced by zeros when that slot is >= valid.
// Loads and stores are non-temporal.  With CSUM, the thread also adds the
// payload checksum terms of the chunks it copied (what it stores) to s1, s2;
// base16 is the payload chunk index of the slab's chunk 0.
template <bool CSUM>
__device__ inline void copy_piece(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                  int piece, int n16, int row16, int B, int valid,
                                  int64_t base16, uint64_t& s1, uint64_t& s2) {
  const int c0 = piece * (kPiece / 16) + threadIdx.x;
  uint4 v[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int c = c0 + u * kPackThreads;
    if (c < n16) {
      if (valid >= B || (c / row16) % B < valid) v[u] = ld_nt(src + c);
      else v[u] = make_uint4(0, 0, 0, 0);
    }
  }
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int c = c0 + u * kPackThreads;
    if (c < n16) {
      st_nt(dst + c, v[u]);
      if (CSUM) {
        // words 4C .. 4C+3 of the payload, weights 4C+1 .. 4C+4
        const uint64_t w = (uint64_t)v[u].x + v[u].y + v[u].z + v[u].w;
        const uint64_t C = (uint64_t)(base16 + c);
        s1 += w;
        s2 += (4 * C + 1) * w + v[u].y + 2ull * v[u].z + 3ull * v[u].w;
      }
    }
  }
}

// Workgroup sum of the checksum terms, added to one of kSumSlots slots
// (spread by workgroup id so that few workgroups meet on one address).
__device__ inline void csum_commit(uint64_t s1, uint64_t s2, unsigned long long* slots) {
  __shared__ uint64_t part[2][kPackThreads / 64];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    s1 += __shfl_xor((unsigned long long)s1, o);
    s2 += __shfl_xor((unsigned long long)s2, o);
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    part[0][wave] = s1;
    part[1][wave] = s2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t a = 0, b = 0;
    for (int i = 0; i < kPackThreads / 64; ++i) {
      a += part[0][i];
      b += part[1][i];
    }
    unsigned long long* slot = slots + 2 * (blockIdx.x % kSumSlots);
    atomicAdd(slot, (unsigned long long)a);
    atomicAdd(slot + 1, (unsigned long long)b);
  }
}

// grid pieces x L x nblk (flattened): buffer block i, layer l  <-  pool
// block trow[b0 + i], layer l
template <bool CSUM>
__global__ void __launch_bounds__(kPackThreads)
k_pack(PoolGeom g, int elt, int pieces, const int32_t* trow, int64_t b0, int32_t nblk,
       int32_t last_valid, char* dst, int64_t base16, unsigned long long* slots) {
  const PieceIdx pi = piece_idx(pieces, g.L);
  const int i = pi.block, l = pi.layer;
  const int64_t block_bytes = g.block_elems * elt;
  const int64_t layer_bytes = block_bytes / g.L;
  const int32_t id = trow[b0 + i];
  const char* s = (const char*)g.pool + id * block_bytes + l * layer_bytes;
  char* d = dst + i * block_bytes + l * layer_bytes;
  const int valid = (i == nblk - 1) ? last_valid : g.B;
  uint64_t s1 = 0, s2 = 0;
  copy_piece<CSUM>((const uint4*)s, (uint4*)d, pi.piece, (int)(layer_bytes / 16),
                   g.dh * elt / 16, g.B, valid,
                          base16 + (i * block_bytes + l * layer_bytes) / 16, s1, s2);
  if (CSUM) csum_commit(s1, s2, slots);
}

// grid pieces x L x nblk (flattened): pool block trow[i], layer l  <-  buffer
// block i, layer l
template <bool CSUM>
__global__ void __launch_bounds__(kPackThreads)
k_unpack(PoolGeom g, int elt, int pieces, const int32_t* trow, const char* src, int64_t base16,
         unsigned long long* slots) {
  const PieceIdx pi = piece_idx(pieces, g.L);
  const int i = pi.block, l = pi.layer;
  const int64_t block_bytes = g.block_elems * elt;
  const int64_t layer_bytes = block_bytes / g.L;
  const int32_t id = trow[i];
  const char* s = src + i * block_bytes + l * layer_bytes;
  char* d = (char*)g.pool + id * block_bytes + l * layer_bytes;
  uint64_t s1 = 0, s2 = 0;
  copy_piece<CSUM>((const uint4*)s, (uint4*)d, pi.piece, (int)(layer_bytes / 16),
                   g.dh * elt / 16, g.B, g.B,
                         base16 + (i * block_bytes + l * layer_bytes) / 16, s1, s2);
  if (CSUM) csum_commit(s1, s2, slots);
}

// One workgroup: out = sum of the slots (mod 2^64), slots cleared for the
// next checksummed copy.
__global__ void __launch_bounds__(kMoveThreads)
k_csum_final(unsigned long long* slots, unsigned long long* out) {
  __shared__ uint64_t part[2][kMoveThreads / 64];
  uint64_t s1 = 0, s2 = 0;
  for (int i = threadIdx.x; i < kSumSlots; i += kMoveThreads) {
    s1 += slots[2 * i];
    s2 += slots[2 * i + 1];
    slots[2 * i] = 0;
    slots[2 * i + 1] = 0;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    s1 += __shfl_xor((unsigned long long)s1, o);
    s2 += __shfl_xor((unsigned long long)s2, o);
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    part[0][wave] = s1;
    part[1][wave] = s2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t a = 0, b = 0;
    for (int i = 0; i < kMoveThreads / 64; ++i) {
      a += part[0][i];
      b += part[1][i];
    }
    out[0] = a;
    out[1] = b;
  }
}

// grid (n_req, L): for requests with cow > 0, copy slots [0, cow) of every
// (K|V, head) tile of layer l from the old tail block to its replacement.
__global__ void __launch_bounds__(kMoveThreads)
k_cow(PoolGeom g, int elt, const int2* pairs, AllocArgs a) {
  const int r = blockIdx.x, l = blockIdx.y;
  const int m = a.req[r].cow;
  if (m <= 0) return;
  const int2 p = pairs[r];
  const int64_t block_bytes = g.block_elems * elt;
  const int tile_bytes = g.B * g.dh * elt;
  const int run16 = m * g.dh * elt / 16;  // valid slots are a prefix of each tile
  const int ntiles = 2 * g.Hkv;
  const char* sb = (const char*)g.pool + p.x * block_bytes;
  char* db = (char*)g.pool + p.y * block_bytes;
  for (int t = 0; t < ntiles; ++t) {
    const int64_t off = tile_off(g, l, t / g.Hkv, t % g.Hkv, 0) * elt;
    const uint4* s = (const uint4*)(sb + off);
    uint4* d = (uint4*)(db + off);
    for (int c = threadIdx.x; c < run16; c += kMoveThreads) d[c] = s[c];
  }
  (void)tile_bytes;
}

template <typename T>
struct Vec;
template <>
struct Vec<uint16_t> {  // bf16 bits: 8 per 16 bytes
  static constexpr int N = 8;
  __device__ static float get(const uint4& v, int i) {
    const uint32_t w = (&v.x)[i >> 1];
    return bf16_to_f32((uint16_t)((i & 1) ? (w >> 16) : (w & 0xffffu)));
  }
  __device__ static void set(uint4& v, int i, float f) {
    uint32_t& w = (&v.x)[i >> 1];
    const uint32_t b = f32_to_bf16(f);
    w = (i & 1) ? ((w & 0xffffu) | (b << 16)) : ((w & 0xffff0000u) | b);
  }
};
template <>
struct Vec<float> {  // 4 per 16 bytes
  static constexpr int N = 4;
  __device__ static float get(const uint4& v, int i) { return __uint_as_float((&v.x)[i]); }
  __device__ static void set(uint4& v, int i, float f) { (&v.x)[i] = __float_as_uint(f); }
};

// Destination blocks that compose copies (those not aliased to a source
// block), as runs [b0[k], b0[k] + (cum[k + 1] - cum[k])) of consecutive ids.
struct CopyRuns {
  int32_t n;
  int32_t b0[KV_MAX_SEGMENTS + 1];
  int32_t cum[KV_MAX_SEGMENTS + 2];
};

// Per-row source of destination block b (rows r < B): source block id, slot
// and key shift; src = -1 past the end of the composed state.
__device__ inline void compose_rows(const PoolGeom& g, const ComposeArgs& a, int b, int32_t* s_src,
                                    int32_t* s_slot, int32_t* s_delta) {
  for (int r = threadIdx.x; r < g.B; r += kMoveThreads) {
    const int u = b * g.B + r;
    int32_t src = -1, slot = 0, delta = 0;
    if (u < a.n_tokens) {
      int i = 0;
      while (i + 1 < a.nseg && a.seg[i + 1].cum <= u) ++i;
      const int j = u - a.seg[i].off;
      src = g.tables[(int64_t)a.seg[i].slot * g.max_blocks + j / g.B];
      slot = j % g.B;
      delta = a.seg[i].delta;
    }
    s_src[r] = src;
    s_slot[r] = slot;
    s_delta[r] = delta;
  }
}

__device__ inline int copy_run_block(const CopyRuns& cr, int i) {
  int k = 0;
  while (k + 1 < cr.n && cr.cum[k + 1] <= i) ++k;
  return cr.b0[k] + (i - cr.cum[k]);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ inline void st_nt16(uint16_t* p, const uint4& v) { st_nt((uint4*)p, v); }
typedef float floatx2_t __attribute__((ext_vector_type(2)));

constexpr int kComposePieces = 2;

__device__ inline uint32_t cvt_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((floatx2_t){a, b}, bf16x2_t));
}

// bf16 compose copy.  grid kComposePieces x L x copied blocks (flattened,
// piece fastest): each (block, layer) slab is split over kComposePieces
// workgroups by KV head (two measured 3% faster than one, four and eight
// slower).  Work items are 16-byte chunks of key / value rows, a row's
// chunks on consecutive lanes (1 KiB per wavefront access).  Destination
// token u = b * B + r comes from segment i (source token u - off_i); keys of
// a shifted segment are rotated by its shift delta: for frequency index j the
// pair (x_j, x_{j + dh/2}) becomes (x cos - y sin, x sin + y cos) with
// cos / sin of |delta| * theta_j (sin negated for a negative shift).  The two
// halves of a row sit cpr / 2 lanes apart and are exchanged with a lane
// shuffle.  All loads of a thread are issued before its stores.
__global__ void __launch_bounds__(kMoveThreads)
k_compose_bf16(PoolGeom g, ComposeArgs a, CopyRuns runs) {
  constexpr int U = 4;  // items per thread per operand and pass
  __shared__ int32_t s_src[64], s_slot[64], s_delta[64];
  const int piece = blockIdx.x % kComposePieces, slab = blockIdx.x / kComposePieces;
  const int b = copy_run_block(runs, slab / g.L), l = slab % g.L;
  const int tid = threadIdx.x;
  compose_rows(g, a, b, s_src, s_slot, s_delta);
  const int32_t dst = g.tables[(int64_t)a.new_slot * g.max_blocks + b];
  __syncthreads();
  uint16_t* pool = (uint16_t*)g.pool;
  uint16_t* dblk = pool + (int64_t)dst * g.block_elems;
  const int cpr = g.dh / 8, hc = cpr / 2, half = g.dh / 2;  // chunks per row, per half row
  // this workgroup's items (16-byte chunks per operand), whole rows of
  // whole waves so that a row's chunks stay on consecutive lanes
  const int n_all = g.Hkv * g.B * cpr;
  const int per = ((n_all + kComposePieces - 1) / kComposePieces + kMoveThreads - 1) /
                  kMoveThreads * kMoveThreads;
  const int i0 = piece * per, n_items = min(n_all, i0 + per);
  for (int base = i0; base < n_items; base += kMoveThreads * U) {
    uint4 kx[U], vx[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int it = base + u * kMoveThreads + tid;
      const int c = it % cpr, r = (it / cpr) % g.B, h = it / (cpr * g.B);
      const int32_t src = it < n_items ? s_src[r] : -1;
      kx[u] = vx[u] = make_uint4(0, 0, 0, 0);
      if (src >= 0) {
        const uint16_t* sb = pool + (int64_t)src * g.block_elems + c * 8;
        kx[u] = ld_nt((const uint4*)(sb + tile_off(g, l, 0, h, s_slot[r])));
        vx[u] = ld_nt((const uint4*)(sb + tile_off(g, l, 1, h, s_slot[r])));
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int it = base + u * kMoveThreads + tid;
      const int c = it % cpr, r = (it / cpr) % g.B, h = it / (cpr * g.B);
      // partner half of the row (all lanes take part in the shuffle)
      uint4 px;
      px.x = __shfl_xor(kx[u].x, hc);
      px.y = __shfl_xor(kx[u].y, hc);
      px.z = __shfl_xor(kx[u].z, hc);
      px.w = __shfl_xor(kx[u].w, hc);
      if (it >= n_items || s_src[r] < 0) continue;
      const int delta = s_delta[r];
      uint4 ko = kx[u];
      if (delta != 0) {
        const int ad = delta < 0 ? -delta : delta;
        const bool lo = c < hc;
        const float sg = (delta < 0) == lo ? 1.f : -1.f;  // sign of sin on the partner
        const float* cp = g.rope_cos + (int64_t)ad * half + (c % hc) * 8;
        const float* sp = g.rope_sin + (int64_t)ad * half + (c % hc) * 8;
        const float4 c0 = *(const float4*)cp, c1 = *(const float4*)(cp + 4);
        const float4 s0 = *(const float4*)sp, s1 = *(const float4*)(sp + 4);
        const float cs[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
        const float sn[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
        const uint32_t ow[4] = {kx[u].x, kx[u].y, kx[u].z, kx[u].w};
        const uint32_t pw[4] = {px.x, px.y, px.z, px.w};
        uint32_t rw[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float o0 = __uint_as_float(ow[q] << 16), o1 = __uint_as_float(ow[q] & 0xffff0000u);
          const float p0 = __uint_as_float(pw[q] << 16), p1 = __uint_as_float(pw[q] & 0xffff0000u);
          rw[q] = cvt_bf16x2(fmaf(p0, sg * sn[2 * q], o0 * cs[2 * q]),
                             fmaf(p1, sg * sn[2 * q + 1], o1 * cs[2 * q + 1]));
        }
        ko = make_uint4(rw[0], rw[1], rw[2], rw[3]);
      }
      uint16_t* db = dblk + c * 8;
      st_nt16(db + tile_off(g, l, 0, h, r), ko);
      st_nt16(db + tile_off(g, l, 1, h, r), vx[u]);
    }
  }
}

// fp32 pools.  grid (copied blocks, L).  Destination block b of the new state takes token
// u = b*B + r from segment i (source token u - off_i).  Keys are rotated by
// the segment's shift delta: pair (x_i, x_{i+dh/2}) -> (x cos - y sin,
// x sin + y cos) with cos/sin of |delta| * theta_i from the float table
// (sin negated for a negative shift).  Values and unshifted keys are copied.
template <typename T>
__global__ void __launch_bounds__(kMoveThreads)
k_compose_copy(PoolGeom g, ComposeArgs a, CopyRuns runs) {
  constexpr int V = Vec<T>::N;
  __shared__ int32_t s_src[64], s_slot[64], s_delta[64];
  __shared__ int32_t s_dst;
  const int b = copy_run_block(runs, blockIdx.x), l = blockIdx.y;
  if (threadIdx.x < g.B) {
    const int r = threadIdx.x;
    const int u = b * g.B + r;
    int32_t src = -1, slot = 0, delta = 0;
    if (u < a.n_tokens) {
      int i = 0;
      while (i + 1 < a.nseg && a.seg[i + 1].cum <= u) ++i;
      const int j = u - a.seg[i].off;
      src = g.tables[(int64_t)a.seg[i].slot * g.max_blocks + j / g.B];
      slot = j % g.B;
      delta = a.seg[i].delta;
    }
    s_src[r] = src;
    s_slot[r] = slot;
    s_delta[r] = delta;
  }
  if (threadIdx.x == 0) s_dst = g.tables[(int64_t)a.new_slot * g.max_blocks + b];
  __syncthreads();
  T* pool = (T*)g.pool;
  T* dblk = pool + (int64_t)s_dst * g.block_elems;
  const int half = g.dh / 2;
  // keys: items (head, row, chunk) over the first half of each row
  const int kc = half / V;
  const int nk = g.Hkv * g.B * kc;
  for (int it = threadIdx.x; it < nk; it += kMoveThreads) {
    const int c = it % kc;
    const int r = (it / kc) % g.B;
    const int h = it / (kc * g.B);
    const int32_t src = s_src[r];
    if (src < 0) continue;
    const T* sp = pool + (int64_t)src * g.block_elems + tile_off(g, l, 0, h, s_slot[r]) + c * V;
    T* dp = dblk + tile_off(g, l, 0, h, r) + c * V;
    uint4 x = *(const uint4*)sp;
    uint4 y = *(const uint4*)(sp + half);
    const int delta = s_delta[r];
    if (delta != 0) {
      const int ad = delta < 0 ? -delta : delta;
      const float sg = delta < 0 ? -1.f : 1.f;
      const float* cr = g.rope_cos + (int64_t)ad * half + c * V;
      const float* sr = g.rope_sin + (int64_t)ad * half + c * V;
      uint4 xo = x, yo = y;
#pragma unroll
      for (int e = 0; e < V; ++e) {
        const float cs = cr[e], sn = sg * sr[e];
        const float xv = Vec<T>::get(x, e), yv = Vec<T>::get(y, e);
        Vec<T>::set(xo, e, xv * cs - yv * sn);
        Vec<T>::set(yo, e, xv * sn + yv * cs);
      }
      x = xo;
      y = yo;
    }
    st_nt((uint4*)dp, x);
    st_nt((uint4*)(dp + half), y);
  }
  // values: items (head, row, chunk) over the whole row
  const int vc = g.dh / V;
  const int nv = g.Hkv * g.B * vc;
  for (int it = threadIdx.x; it < nv; it += kMoveThreads) {
    const int c = it % vc;
    const int r = (it / vc) % g.B;
    const int h = it / (vc * g.B);
    const int32_t src = s_src[r];
    if (src < 0) continue;
    const T* sp = pool + (int64_t)src * g.block_elems + tile_off(g, l, 1, h, s_slot[r]) + c * V;
    T* dp = dblk + tile_off(g, l, 1, h, r) + c * V;
    st_nt((uint4*)dp, *(const uint4*)sp);
  }
}

}  // namespace

hipError_t launch_pack(const PoolGeom& g, int dtype, const int32_t* trow, int64_t b0,
                       int32_t nblk, int32_t last_valid, void* dst, unsigned long long* slots,
                       int64_t base16, hipStream_t s) {
  const int elt = dtype == KV_DTYPE_BF16 ? 2 : 4;
  const int64_t layer_bytes = g.block_elems * elt / g.L;
  const int pieces = (int)((layer_bytes + kPiece - 1) / kPiece);
  const int64_t n = (int64_t)pieces * g.L * nblk;
  if (n > 0x7fffffff) return hipErrorInvalidValue;
  if (slots)
    k_pack<true><<<(unsigned)n, kPackThreads, 0, s>>>(g, elt, pieces, trow, b0, nblk, last_valid,
                                                      (char*)dst, base16, slots);
  else
    k_pack<false><<<(unsigned)n, kPackThreads, 0, s>>>(g, elt, pieces, trow, b0, nblk,
                                                       last_valid, (char*)dst, 0, nullptr);
  return hipGetLastError();
}

hipError_t launch_unpack(const PoolGeom& g, int dtype, const int32_t* trow, int32_t nblk,
                         const void* src, unsigned long long* slots, int64_t base16,
                         hipStream_t s) {
  const int elt = dtype == KV_DTYPE_BF16 ? 2 : 4;
  const int64_t layer_bytes = g.block_elems * elt / g.L;
  const int pieces = (int)((layer_bytes + kPiece - 1) / kPiece);
  const int64_t n = (int64_t)pieces * g.L * nblk;
  if (n > 0x7fffffff) return hipErrorInvalidValue;
  if (slots)
    k_unpack<true><<<(unsigned)n, kPackThreads, 0, s>>>(g, elt, pieces, trow, (const char*)src,
                                                        base16, slots);
  else
    k_unpack<false><<<(unsigned)n, kPackThreads, 0, s>>>(g, elt, pieces, trow,
                                                         (const char*)src, 0, nullptr);
  return hipGetLastError();
}

hipError_t launch_csum_final(unsigned long long* slots, unsigned long long* out, hipStream_t s) {
  k_csum_final<<<1, kMoveThreads, 0, s>>>(slots, out);
  return hipGetLastError();
}

hipError_t launch_cow(const PoolGeom& g, int dtype, const int2* cow_pairs, const AllocArgs& a,
                      hipStream_t s) {
  const int elt = dtype == KV_DTYPE_BF16 ? 2 : 4;
  k_cow<<<dim3(a.n_req, g.L), kMoveThreads, 0, s>>>(g, elt, cow_pairs, a);
  return hipGetLastError();
}

hipError_t launch_compose_copy(const PoolGeom& g, int dtype, const ComposeArgs& a,
                               hipStream_t s) {
  // copied blocks: [0, n_dest_blocks) minus the (increasing, disjoint) alias ranges
  CopyRuns runs;
  runs.n = 0;
  int32_t next = 0, total = 0;
  auto add = [&](int32_t b0, int32_t b1) {
    if (b1 <= b0) return;
    runs.b0[runs.n] = b0;
    runs.cum[runs.n] = total;
    total += b1 - b0;
    ++runs.n;
  };
  for (int i = 0; i < a.nseg; ++i) {
    if (a.seg[i].alias_b1 <= a.seg[i].alias_b0) continue;
    add(next, a.seg[i].alias_b0);
    next = a.seg[i].alias_b1;
  }
  add(next, a.n_dest_blocks);
  runs.cum[runs.n] = total;
  if (total == 0) return hipSuccess;
  dim3 grid(total, g.L);
  if (dtype == KV_DTYPE_BF16 && g.dh >= 16 && (g.dh & (g.dh - 1)) == 0)
    k_compose_bf16<<<(unsigned)((int64_t)total * g.L * kComposePieces), kMoveThreads, 0, s>>>(
        g, a, runs);
  else if (dtype == KV_DTYPE_BF16)
    k_compose_copy<uint16_t><<<grid, kMoveThreads, 0, s>>>(g, a, runs);
  else
    k_compose_copy<float><<<grid, kMoveThreads, 0, s>>>(g, a, runs);
  return hipGetLastError();
}

}  // namespace kvs
