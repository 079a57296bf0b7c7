// Decode attention (one new token per sequence) over the paged cache on MFMA,
// split over key chunks, reading each shared block once for the whole batch.
//
// Forked agents share the blocks of their common context (same physical ids
// in their block tables).  The keys of a decode step are cut into chunks of
// ck positions (1024, or 512 for a batch of one, whose chunks are its only
// source of parallelism: +5-10% there).  k_decode_plan (one wavefront per chunk) groups the batch
// members whose key counts and block ids agree over the chunk; each group of
// a chunk is one work unit.  The grouping is the same for every layer and KV
// head, so it is computed once per call.
//
// The stream kernels run one wavefront per work item with no workgroup
// barriers: a wavefront streams the unit's K/V rows once, 32 keys at a time,
// through a ring of LDS stages filled by direct global->LDS copies, and scores
// all of the group's query vectors (members x the G query heads of the KV
// head) with MFMA in the transposed layout of the prefill kernel (query vector
// in the MFMA column, softmax state lane-local, V^T operands by transposed LDS
// reads).  Per (query vector, chunk) it writes a partial (running max m,
// running sum l, unnormalised output o); k_decode_merge combines the chunks of
// a query with the usual log-sum-exp rescaling.  A unit's record carries its
// block ids, so a wavefront can start copying after one read of it.
//
// k_decode_pers is persistent: one workgroup per resident slot walks a
// static list of (unit, layer, KV head) items, largest first, and keeps its
// stage ring running across items, so the copy latency is paid once per
// workgroup rather than once per item (a stream-only probe that read every
// unit twice without a restart took 1.9x, not 2x, the time of one pass); a
// switch between items still costs about one refill of the ring.  It takes
// units of 65 to 128 query vectors (four wavefronts sharing the ring) and
// units of at most 64 while each slot has few items.  k_decode_stream runs
// one wavefront per (unit, query slice of 64 vectors, KV head, layer) for
// the rest; the slices of a unit are launched on one XCD, so the later ones
// find the keys in its L2.
#include <algorithm>

#include "kv_dma.h"
#include "kv_fast.h"

namespace kvs {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef short v4s __attribute__((ext_vector_type(4)));
#define KV_LDS4(p) ((__attribute__((address_space(3))) v4s*)(p))

constexpr int kDh = 128;
constexpr int kCK = 1024;              // keys per chunk (at most; see decode_ck)
constexpr int kKT = 32;                // keys per pipeline stage
constexpr int kStage = 2 * kKT * kDh;  // elements per stage: K rows, then V rows
constexpr int kPart = kDh + 4;         // floats per partial: m, l, pad, pad, o[128]

constexpr int kUnitBlocks = 64;        // block ids per chunk, at most (ck / B)

// One work unit: the members in `mask` share block ids and key count `nk`
// over the chunk; `lead` is the first of them.  `blk` holds the chunk's
// block ids (0 past the unit's last key), so that a wavefront learns
// everything it needs to start copying from one load of the record.
struct DecodeUnit {
  int32_t lead, nk;
  uint32_t mask_lo, mask_hi;
  int32_t blk[kUnitBlocks];
};

// Reductions over lanes l and l ^ 32 (the two halves of a token's keys) with
// v_permlane32_swap, which leaves v[l % 32] and v[l % 32 + 32] in every lane.
__device__ inline float max_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float sum_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// LDS slot of chunk c of key row r: c ^ kswz(r) for K (read 16 rows at one
// chunk), c ^ vswz(r) for V (read transposed, 8 rows x 4 adjacent chunks);
// both spread each read over all bank groups.
__device__ inline int kswz(int r) { return r & 15; }
__device__ inline int vswz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }

__device__ inline uint32_t pack2(float a, float b) {
  const __bf16 x = (__bf16)a, y = (__bf16)b;
  return (uint32_t)__builtin_bit_cast(uint16_t, x) | ((uint32_t)__builtin_bit_cast(uint16_t, y) << 16);
}

// grid (n_chunks), block 64; dynamic LDS: batch * (ck / B) ints.
// Writes the units of chunk c to units[c * batch ...] and their number to
// n_units[c].
__global__ void __launch_bounds__(64)
k_decode_plan(PoolGeom g, AppendDesc a, DecodeUnit* __restrict__ units,
              int* __restrict__ n_units, int ck) {
  extern __shared__ int s_rows[];  // [batch][ck / B]: each member's block ids in the chunk
  const int lane = threadIdx.x, c = blockIdx.x, b = a.batch;
  const int c0 = c * ck;
  const int nbc = ck >> g.b_shift, nbs = __builtin_ctz(nbc);
  const int jb0 = c0 >> g.b_shift;
  for (int i = lane; i < b * nbc; i += 64) {
    const int m = i >> nbs, jb = jb0 + (i & (nbc - 1));
    const int n = a.seq[m].n_before + 1;
    s_rows[i] = (jb << g.b_shift) < n ? g.tables[(int64_t)a.seq[m].slot * g.max_blocks + jb] : -1;
  }
  const int nk_l = lane < b ? max(0, min(ck, a.seq[lane].n_before + 1 - c0)) : 0;
  __syncthreads();
  // lane q describes group q: leader, key count, first block id, members
  int n_groups = 0, g_lead = 0, g_nk = 0, g_first = 0;
  uint64_t g_mask = 0;
  for (int m = 0; m < b; ++m) {
    const int nk = __shfl(nk_l, m);
    if (nk == 0) continue;
    const int first = s_rows[m * nbc];
    const int nb = (nk + g.B - 1) >> g.b_shift;
    uint64_t cand = __ballot(lane < n_groups && g_nk == nk && g_first == first);
    int found = -1;
    while (cand) {
      const int q = __builtin_ctzll(cand);
      const int lead = __shfl(g_lead, q);
      const bool diff = lane < nb && s_rows[lead * nbc + lane] != s_rows[m * nbc + lane];
      if (__ballot(diff) == 0) {
        found = q;
        break;
      }
      cand &= cand - 1;
    }
    if (found < 0) {
      found = n_groups++;
      if (lane == found) {
        g_lead = m;
        g_nk = nk;
        g_first = first;
        g_mask = 0;
      }
    }
    if (lane == found) g_mask |= 1ull << m;
  }
  if (lane < n_groups) {
    DecodeUnit* up = units + c * b + lane;
    up->lead = g_lead;
    up->nk = g_nk;
    up->mask_lo = (uint32_t)g_mask;
    up->mask_hi = (uint32_t)(g_mask >> 32);
  }
  for (int q = 0; q < n_groups; ++q) {
    const int lead = __shfl(g_lead, q);
    units[c * b + q].blk[lane] = lane < nbc ? max(s_rows[lead * nbc + lane], 0) : 0;
  }
  if (lane == 0) n_units[c] = n_groups;
}

// Which chunk holds unit u of the concatenated per-chunk unit lists, and the
// unit's index within it.  Wave-uniform.
__device__ inline void locate_unit(const int* __restrict__ n_units, int n_chunks, int u,
                                   int* chunk, int* idx) {
  const int lane = threadIdx.x & 63;
  int run = 0;
  *chunk = -1;
  for (int cb = 0; cb < n_chunks; cb += 64) {
    const int v = cb + lane < n_chunks ? n_units[cb + lane] : 0;
    int inc = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int t = __shfl_up(inc, d);
      if (lane >= d) inc += t;
    }
    const uint64_t hit = __ballot(v > 0 && run + inc - v <= u && u < run + inc);
    if (hit) {
      const int q = __builtin_ctzll(hit);
      *chunk = cb + q;
      *idx = u - run - __shfl(inc - v, q);
      return;
    }
    run += __shfl(inc, 63);
  }
}

// Wait until this wavefront's copies of the stage about to be read have
// landed: a wavefront's copies complete in issue order and it issues
// 2 * (kKT / 4) / NW copies of each stage (NW wavefronts share the copies),
// so at most `ahead` newer stages may still be pending (ahead <= 2).  Memory
// operations issued after the stage only lengthen the wait.
template <int NW = 1>
__device__ inline void wait_stage(int ahead) {
  constexpr int per = 2 * (kKT / 4) / NW;
  if (ahead >= 2)
    wait_vmcnt<2 * per>();
  else if (ahead == 1)
    wait_vmcnt<per>();
  else
    wait_vmcnt<0>();
}

// Copies of one stage (keys [32 tile, 32 tile + 32) of a unit): 8 copies of
// 1 KiB (4 key rows, all in one block since B >= 16) per operand, block base
// in scalar registers, non-temporal (each byte is read once per call).
// pool_kv = the pool plus the offset of this (layer, KV head)'s K tile in a
// block; lane j of tb = block id of the unit's block j.  Rows past the
// unit's last key read slots of a real block; their scores are masked and
// their V rows zeroed in LDS before use.
// With NW > 1 wavefronts sharing the stage, wavefront w issues copies w, w +
// NW, ... of each operand.
template <int NW = 1>
__device__ inline void issue_stage(const PoolGeom& g, const char* pool_kv, int64_t kv_gap, int tb,
                                   int tile, uint32_t stage_lds, int lane, int w = 0) {
#pragma unroll
  for (int jj = 0; jj < kKT / 4 / NW; ++jj) {
    const int j = w + jj * NW;
    const int key0 = tile * kKT + j * 4;
    const int id = __builtin_amdgcn_readlane(tb, key0 >> g.b_shift);
    const char* kb = pool_kv + ((int64_t)id * g.block_elems + (key0 & (g.B - 1)) * kDh) * 2;
    const int r = j * 4 + (lane >> 4);
    const uint32_t ko = (lane >> 4) * (kDh * 2) + (((lane & 15) ^ kswz(r)) * 16);
    const uint32_t vo = (lane >> 4) * (kDh * 2) + (((lane & 15) ^ vswz(r)) * 16);
    lds_dma16_sv_nt(kb, ko, stage_lds + j * 1024);
    lds_dma16_sv_nt(kb + kv_gap, vo, stage_lds + kKT * kDh * 2 + j * 1024);
  }
}

// Q^T operands of query vectors q0 .. q0 + 32 RT - 1 of a unit whose members
// are the bits of `mask`: vector r = (member rank) * G + head.  qrow = the
// member's batch row (-1 past the unit's R vectors), qhead = its query head.
template <int RT>
__device__ __attribute__((always_inline)) inline void load_q(
    const PoolGeom& g, const uint16_t* __restrict__ qbuf, uint64_t mask, int R, int q0, int gk,
    int lc, int M, int lane, bf16x8 (&qf)[RT][8], int (&qrow)[RT], int (&qhead)[RT]) {
  const int G = g.Hq / g.Hkv, hl = lane >> 5, col = lane & 31;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = q0 + rt * 32 + col;
    const bool ok = r < R;
    const int mi = ok ? r / G : 0;
    uint64_t mm = mask;
    for (int i = 0; i < mi; ++i) mm &= mm - 1;
    qrow[rt] = ok ? __builtin_ctzll(mm) : -1;
    qhead[rt] = gk * G + (ok ? r - mi * G : 0);
    const uint16_t* qp = qbuf + (((int64_t)lc * M + (ok ? qrow[rt] : 0)) * g.Hq + qhead[rt]) * kDh;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
      qf[rt][ks] = ok ? *(const bf16x8*)(qp + ks * 16 + hl * 8) : bf16x8{};
  }
}

template <int RT>
__device__ __attribute__((always_inline)) inline void clear_state(floatx16 (&oacc)[RT][4],
                                                                  float (&m_run)[RT],
                                                                  float (&l_run)[RT]) {
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    m_run[rt] = -INFINITY;
    l_run[rt] = 0.f;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int e = 0; e < 16; ++e) oacc[rt][mt][e] = 0.f;
  }
}

// One stage, keys [k0, k0 + 32) of a unit with nk keys, K rows then V rows
// at Ks: S^T = K Q^T, the online softmax in base 2 (the running max moves
// only when it grows by more than 8), O^T += V^T P^T with V^T operands by
// transposed LDS reads.  `two`: the second query tile holds vectors.
template <int RT>
__device__ __attribute__((always_inline)) inline void attend_stage(
    uint16_t* Ks, int k0, int nk, bool two, const bf16x8 (&qf)[RT][8], floatx16 (&oacc)[RT][4],
    float (&m_run)[RT], float (&l_run)[RT], float qk_scale_log2, int lane) {
  const int hl = lane >> 5, col = lane & 31;
  uint16_t* Vs = Ks + kKT * kDh;
  const bool tail = k0 + kKT > nk;  // wave-uniform
  if (tail) {  // V rows of keys >= nk may hold anything: zero them
    for (int i = (nk - k0) * (kDh / 8) + lane; i < kKT * (kDh / 8); i += 64)
      *(uint4*)(Vs + i * 8) = make_uint4(0, 0, 0, 0);
  }

  floatx16 sacc[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int e = 0; e < 16; ++e) sacc[rt][e] = 0.f;
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) {
    const bf16x8 kf = *(const bf16x8*)(Ks + col * kDh + (((ks * 2 + hl) ^ kswz(col)) * 8));
    sacc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[0][ks], sacc[0], 0, 0, 0);
    if (two)
      sacc[RT - 1] =
          __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[RT - 1][ks], sacc[RT - 1], 0, 0, 0);
  }
  bf16x8 pf[RT][2];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    if (rt > 0 && !two) break;
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      float sv = sacc[rt][e];
      if (tail) {
        const int kk = k0 + (e >> 2) * 8 + hl * 4 + (e & 3);
        if (kk >= nk) sv = -INFINITY;
      }
      sacc[rt][e] = sv;
      mx = fmaxf(mx, sv);
    }
    mx = max_xor32(mx) * qk_scale_log2;
    const float m_new = mx > m_run[rt] + 8.f ? mx : m_run[rt];
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const bool moved =
        __builtin_amdgcn_readfirstlane((int)(__ballot(m_new != m_run[rt]) != 0)) != 0;
    float psum = 0.f;
#pragma unroll
    for (int hs = 0; hs < 2; ++hs) {
      float p[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        p[j] = __builtin_amdgcn_exp2f(fmaf(sacc[rt][hs * 8 + j], qk_scale_log2, -m_use));
        psum += p[j];
      }
      uint32_t wv[4] = {pack2(p[0], p[1]), pack2(p[2], p[3]), pack2(p[4], p[5]),
                        pack2(p[6], p[7])};
      pf[rt][hs] = __builtin_bit_cast(bf16x8, *(uint4*)wv);
    }
    if (moved) {
      const float alpha = __builtin_amdgcn_exp2f(m_run[rt] - m_use);
      l_run[rt] *= alpha;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[rt][mt][e] *= alpha;
    }
    l_run[rt] += psum;
    m_run[rt] = m_new;
  }
  const int g4 = lane >> 4, li = lane & 15;
#pragma unroll
  for (int s4 = 0; s4 < 2; ++s4) {
    const int key_a = s4 * 16 + (g4 >> 1) * 4 + (li >> 2), key_b = key_a + 8;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const int dc = mt * 32 + (g4 & 1) * 16 + (li & 3) * 4;
      const int ch = dc >> 3, hf = dc & 7;
      const v4s r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          KV_LDS4(Vs + key_a * kDh + ((ch ^ vswz(key_a)) * 8) + hf));
      const v4s r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          KV_LDS4(Vs + key_b * kDh + ((ch ^ vswz(key_b)) * 8) + hf));
      const v4s vv[2] = {r0, r1};
      const bf16x8 vf = __builtin_bit_cast(bf16x8, vv);
      oacc[0][mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[0][s4], oacc[0][mt], 0, 0, 0);
      if (two)
        oacc[RT - 1][mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[RT - 1][s4],
                                                                   oacc[RT - 1][mt], 0, 0, 0);
    }
  }
}

// Partials (m, l, o) of a unit's query vectors for chunk c, layer lc.
template <int RT>
__device__ __attribute__((always_inline)) inline void write_partials(
    float* __restrict__ part, const PoolGeom& g, int b, int lc, int c, int n_chunks,
    const int (&qrow)[RT], const int (&qhead)[RT], const floatx16 (&oacc)[RT][4],
    const float (&m_run)[RT], const float (&l_run)[RT], int lane) {
  const int hl = lane >> 5;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const float lt = sum_xor32(l_run[rt]);
    if (qrow[rt] < 0) continue;
    float* pp = part + ((((int64_t)lc * b + qrow[rt]) * g.Hq + qhead[rt]) * n_chunks + c) * kPart;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *(float4*)(pp + 4 + mt * 32 + q * 8 + hl * 4) =
            make_float4(oacc[rt][mt][q * 4], oacc[rt][mt][q * 4 + 1], oacc[rt][mt][q * 4 + 2],
                        oacc[rt][mt][q * 4 + 3]);
    if (hl == 0) {
      pp[0] = m_run[rt];
      pp[1] = lt;
    }
  }
}

// grid (slots x ns, Hkv, lc), block 64, ns = query slices per unit.  With
// ns = 1, workgroup x takes units x, x + slots, ...; with ns > 1 (slots a
// multiple of 8), x = (s / 8) * 8 ns + q * 8 + s % 8 takes slice q of units
// s, s + slots, ..., so all slices of a unit have the same x mod 8 (XCD).
// RT = query-vector tiles of 32 per slice (at most 32 RT vectors); S = LDS
// stages (S - 1 in flight while one is consumed).
template <int RT, int S>
__global__ void __launch_bounds__(64)
k_decode_stream(PoolGeom g, const uint16_t* __restrict__ qbuf, AppendDesc a,
                const DecodeUnit* __restrict__ units, const int* __restrict__ n_units,
                float* __restrict__ part, int n_chunks, int ck, int l0, float qk_scale_log2,
                int ns) {
  static_assert(S >= 2 && S <= 4, "stages");
  __shared__ __attribute__((aligned(16))) uint16_t smem[S * kStage];
  const int lane = threadIdx.x;
  const int gk = blockIdx.y, lc = blockIdx.z, layer = l0 + lc;
  const int G = g.Hq / g.Hkv, b = a.batch, M = b;  // T == 1
  const int64_t koff = tile_off(g, layer, 0, gk, 0), voff = tile_off(g, layer, 1, gk, 0);
  const char* pool_kv = (const char*)g.pool + koff * 2;
  const uint32_t lds0 = lds_addr(smem);
  const int64_t kv_gap = (voff - koff) * 2;  // bytes from a K row to its V row

  const int x = blockIdx.x;
  const int slot = ns == 1 ? x : (x / (8 * ns)) * 8 + (x & 7);
  const int qs = ns == 1 ? 0 : (x >> 3) % ns;
  const int stride = gridDim.x / ns;
  // one pass over the unit counts: their total, and the chunk and index of
  // this wavefront's first unit
  int total = 0, c_first = -1, gi_first = 0;
  for (int cb = 0; cb < n_chunks; cb += 64) {
    const int v = cb + lane < n_chunks ? n_units[cb + lane] : 0;
    int inc = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int tv = __shfl_up(inc, d);
      if (lane >= d) inc += tv;
    }
    const uint64_t hit = __ballot(v > 0 && total + inc - v <= slot && slot < total + inc);
    if (c_first < 0 && hit) {
      const int q = __builtin_ctzll(hit);
      c_first = cb + q;
      gi_first = slot - total - __shfl(inc - v, q);
    }
    total += __shfl(inc, 63);
  }
  total = __builtin_amdgcn_readfirstlane(total);
  for (int u = slot; u < total; u += stride) {
    int c = c_first, gi = gi_first;
    if (u != slot) locate_unit(n_units, n_chunks, u, &c, &gi);
    c = __builtin_amdgcn_readfirstlane(c);
    gi = __builtin_amdgcn_readfirstlane(gi);
    const DecodeUnit* up = units + c * b + gi;
    const int nk = __builtin_amdgcn_readfirstlane(up->nk);
    const uint64_t mask = ((uint64_t)__builtin_amdgcn_readfirstlane(up->mask_hi) << 32) |
                          (uint32_t)__builtin_amdgcn_readfirstlane(up->mask_lo);
    int tb = up->blk[lane];
    settle(tb);
    const int R = __popcll(mask) * G;  // query vectors of the unit
    const int q0 = qs * 32 * RT;       // this slice's first query vector
    if (q0 >= R) continue;             // wave-uniform: a unit with fewer slices
    const bool two = RT > 1 && R - q0 > 32;

    // the first stages go out before the query vectors are read, so that the
    // two latencies overlap (the wait for the queries below also waits for
    // these copies, which the first stage needs anyway)
    const int n_tiles = (nk + kKT - 1) / kKT;
    for (int st = 0; st < S - 1 && st < n_tiles; ++st)
      issue_stage(g, pool_kv, kv_gap, tb, st, lds0 + st * kStage * 2, lane);
    bf16x8 qf[RT][8];
    int qrow[RT], qhead[RT];
    load_q<RT>(g, qbuf, mask, R, q0, gk, lc, M, lane, qf, qrow, qhead);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) settle(qf[rt][ks]);

    floatx16 oacc[RT][4];
    float m_run[RT], l_run[RT];
    clear_state<RT>(oacc, m_run, l_run);
    for (int t = 0; t < n_tiles; ++t) {
      wait_stage(min(S - 2, n_tiles - 1 - t));
      // stage (t - 1) % S was consumed in the previous iteration
      if (t + S - 1 < n_tiles)
        issue_stage(g, pool_kv, kv_gap, tb, t + S - 1, lds0 + ((t + S - 1) % S) * kStage * 2,
                    lane);
      attend_stage<RT>(smem + (t % S) * kStage, t * kKT, nk, two, qf, oacc, m_run, l_run,
                       qk_scale_log2, lane);
    }
    write_partials<RT>(part, g, b, lc, c, n_chunks, qrow, qhead, oacc, m_run, l_run, lane);
  }
}

// Unit counts of up to 64 * kNR chunks in registers (count and inclusive
// prefix of chunk 64 r + lane), so that a wavefront finds the chunk and
// index of any unit without a memory access.
constexpr int kNR = 4;
constexpr int kPersMaxChunks = 64 * kNR;

struct UnitIndex {
  int v[kNR], inc[kNR];
};

__device__ inline int index_units(const int* __restrict__ n_units, int n_chunks, int lane,
                                  UnitIndex& ix) {
  int run = 0;
#pragma unroll
  for (int r = 0; r < kNR; ++r) {
    const int v = 64 * r + lane < n_chunks ? n_units[64 * r + lane] : 0;
    int inc = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int tv = __shfl_up(inc, d);
      if (lane >= d) inc += tv;
    }
    ix.v[r] = v;
    ix.inc[r] = run + inc;
    run += __shfl(inc, 63);
  }
  return __builtin_amdgcn_readfirstlane(run);
}

__device__ inline void find_unit(const UnitIndex& ix, int u, int* c, int* gi) {
  int cc = 0, gg = 0;
#pragma unroll
  for (int r = 0; r < kNR; ++r) {
    const uint64_t hit = __ballot(ix.v[r] > 0 && ix.inc[r] - ix.v[r] <= u && u < ix.inc[r]);
    if (hit) {
      const int q = __builtin_ctzll(hit);
      cc = 64 * r + q;
      gg = u - __shfl(ix.inc[r] - ix.v[r], q);
    }
  }
  *c = __builtin_amdgcn_readfirstlane(cc);
  *gi = __builtin_amdgcn_readfirstlane(gg);
}

// A work item: one unit x one layer x one KV head.
struct DecodeItem {
  int c, lc, gk, nk, n_tiles;
  uint64_t mask;
  const char* pool_kv;
  int tb;
};

// grid (W), block 64 NW, units of at most 32 RT NW query vectors, at most
// kPersMaxChunks chunks.  Persistent: workgroup w takes items w, w + W, w +
// 2W, ... of the list (unit, layer, KV head) in that order, units in chunk
// order, so that the full chunks of a shared context come first and the
// short last chunks fill the end.  The NW wavefronts of a workgroup share one
// LDS stage ring (each issues its share of every stage's copies; a barrier
// per stage makes the stage visible to all and frees the slot consumed
// before it) and each scores 32 RT of the unit's query vectors, so that a
// deep ring and the matrix cores of several SIMDs serve the same bytes.  The ring runs
// across items: the first stages of the next item are issued while the
// current item's last stages are consumed, so a workgroup pays the copy
// latency once, not once per item.  The next item's record (read a whole
// item ahead) and query vectors (loaded at the start of the current item)
// are waited for only at the switch between items, the one point where the
// compiler drains a wavefront's memory operations.
template <int NW, int RT, int S>
__global__ void __launch_bounds__(64 * NW)
k_decode_pers(PoolGeom g, const uint16_t* __restrict__ qbuf, AppendDesc a,
              const DecodeUnit* __restrict__ units, const int* __restrict__ n_units,
              float* __restrict__ part, int n_chunks, int l0, int lcn, float qk_scale_log2) {
  static_assert(S >= 2 && S <= 4, "stages");
  static_assert(NW == 1 || NW == 2 || NW == 4, "wavefronts per workgroup");
  __shared__ __attribute__((aligned(16))) uint16_t smem[S * kStage];
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int q0 = 32 * RT * wv;  // this wavefront's first query vector of a unit
  const int wcp = NW == 1 ? 0 : wv;  // copy share (a constant for one wavefront)
  const int G = g.Hq / g.Hkv, b = a.batch, M = b;  // T == 1
  const uint32_t lds0 = lds_addr(smem);
  const int64_t kv_gap = (tile_off(g, 0, 1, 0, 0) - tile_off(g, 0, 0, 0, 0)) * 2;
  const int W = gridDim.x;

  UnitIndex ix;
  const int total = index_units(n_units, n_chunks, lane, ix);
  const int per_u = lcn * g.Hkv;
  const int n_items = total * per_u;
  int i = blockIdx.x;
  if (i >= n_items) return;  // workgroup-uniform

  // record words of item j: lane l holds word l (header in lanes 0-3) and
  // word l + 4 (block id l)
  auto load_rec = [&](int j, int& w0, int& w1, int& c, int& lc, int& gk) {
    const int u = j / per_u, r = j - u * per_u;
    lc = r / g.Hkv;
    gk = r - lc * g.Hkv;
    int gi;
    find_unit(ix, u, &c, &gi);
    const int* wp = (const int*)(units + c * b + gi);
    w0 = wp[lane];
    w1 = wp[lane + 4];
  };
  auto make_item = [&](int w0, int w1, int c, int lc, int gk, DecodeItem& it) {
    it.c = c;
    it.lc = lc;
    it.gk = gk;
    it.nk = __builtin_amdgcn_readlane(w0, 1);
    it.mask = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane(w0, 3) << 32) |
              (uint32_t)__builtin_amdgcn_readlane(w0, 2);
    it.n_tiles = (it.nk + kKT - 1) / kKT;
    it.pool_kv = (const char*)g.pool + tile_off(g, l0 + lc, 0, gk, 0) * 2;
    it.tb = w1;
  };

  DecodeItem cur, nxt{};
  bool has_nxt;
  bf16x8 qf[RT][8], qn[RT][8];
  int qrow[RT], qhead[RT], qrow_n[RT], qhead_n[RT];
  int nw0 = 0, nw1 = 0, nc = 0, nlc = 0, ngk = 0;  // record of the item after nxt
  {
    int w0, w1, c, lc, gk;
    load_rec(i, w0, w1, c, lc, gk);
    settle(w0);
    settle(w1);
    make_item(w0, w1, c, lc, gk, cur);
    has_nxt = i + W < n_items;
    if (has_nxt) {
      load_rec(i + W, w0, w1, c, lc, gk);
      settle(w0);
      settle(w1);
      make_item(w0, w1, c, lc, gk, nxt);
    }
    load_q<RT>(g, qbuf, cur.mask, __popcll(cur.mask) * G, q0, cur.gk, cur.lc, M, lane, qf, qrow,
               qhead);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) settle(qf[rt][ks]);
  }

  int base = 0;    // stream index of cur's first stage
  int issued = 0;  // stages issued so far
  // issue this wavefront's share of the next stage of the stream (cur's
  // stages, then nxt's) if any
  auto issue_next = [&]() {
    const int s = issued;
    const uint32_t sl = lds0 + (s % S) * kStage * 2;
    if (s - base < cur.n_tiles) {
      issue_stage<NW>(g, cur.pool_kv, kv_gap, cur.tb, s - base, sl, lane, wcp);
      ++issued;
    } else if (has_nxt && s - base - cur.n_tiles < nxt.n_tiles) {
      issue_stage<NW>(g, nxt.pool_kv, kv_gap, nxt.tb, s - base - cur.n_tiles, sl, lane, wcp);
      ++issued;
    }
  };

  floatx16 oacc[RT][4];
  float m_run[RT], l_run[RT];
  for (;;) {
    // prefetch for the switch after this item: nxt's query vectors and the
    // record of the item after it (unconditional, so that no copy of a
    // pending value lands before the switch: no next item loads nothing, a
    // missing item after it re-reads the current record)
    const bool has_nn = has_nxt && i + 2 * W < n_items;
    const uint64_t qmask = has_nxt ? nxt.mask : 0;
    load_q<RT>(g, qbuf, qmask, __popcll(qmask) * G, q0, nxt.gk, nxt.lc, M, lane, qn, qrow_n,
               qhead_n);
    load_rec(has_nn ? i + 2 * W : i, nw0, nw1, nc, nlc, ngk);
    // top up the ring to S - 1 stages ahead; every slot written here was
    // consumed before the last barrier
#pragma unroll
    for (int st = 0; st < S - 1; ++st)
      if (issued - base < S - 1) issue_next();

    const int R = __popcll(cur.mask) * G;  // the unit's query vectors
    const bool active = q0 < R;              // wavefront-uniform
    const bool two = RT > 1 && R - q0 > 32;
    clear_state<RT>(oacc, m_run, l_run);
    for (int t = 0; t < cur.n_tiles; ++t) {
      const int s = base + t;
      wait_stage<NW>(issued - s - 1);
      // several wavefronts: every wavefront's copies of stage s are visible
      // and every LDS access of stage s - 1 (reads, tail zeroing) is done, so
      // its slot may be refilled.  One: the slot's reads fed products issued
      // in the previous iteration, and its tail zeroing precedes the copy
      // that refills it by a whole stage.
      if constexpr (NW > 1) lds_barrier();
      if (issued < s + S) issue_next();
      if (NW == 1 || active)
        attend_stage<RT>(smem + (s % S) * kStage, t * kKT, cur.nk, two, qf, oacc, m_run, l_run,
                         qk_scale_log2, lane);
    }
    if (!has_nxt) {
      write_partials<RT>(part, g, b, cur.lc, cur.c, n_chunks, qrow, qhead, oacc, m_run, l_run,
                         lane);
      return;
    }
    // the switch: the one wait for the prefetched values
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) settle(qn[rt][ks]);
    settle(nw0);
    settle(nw1);
    write_partials<RT>(part, g, b, cur.lc, cur.c, n_chunks, qrow, qhead, oacc, m_run, l_run,
                       lane);
    base += cur.n_tiles;
    cur = nxt;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      qrow[rt] = qrow_n[rt];
      qhead[rt] = qhead_n[rt];
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) qf[rt][ks] = qn[rt][ks];
    }
    has_nxt = has_nn;
    if (has_nn) make_item(nw0, nw1, nc, nlc, ngk, nxt);
    i += W;
  }
}

// grid (batch * Hq, lc), block 64: combine the chunk partials of one query.
// Lane i owns output channels 2i, 2i + 1; the chunk weights exp2(m_c - max)
// are computed once per chunk and broadcast through LDS.
__global__ void __launch_bounds__(64)
k_decode_merge(PoolGeom g, AppendDesc a, const float* __restrict__ part, int n_chunks, int ck,
               uint16_t* __restrict__ o, int l0) {
  __shared__ float s_w[64];
  const int sh = blockIdx.x, lc = blockIdx.y, lane = threadIdx.x;
  const int s = sh / g.Hq, h = sh % g.Hq;
  const int b = a.batch;
  const int n = a.seq[s].n_before + 1;
  const int nc = (n + ck - 1) / ck;
  const float* pp = part + (((int64_t)lc * b + s) * g.Hq + h) * n_chunks * kPart;
  float mx = -INFINITY;
  for (int c = lane; c < nc; c += 64) mx = fmaxf(mx, pp[(int64_t)c * kPart]);
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) mx = fmaxf(mx, __shfl_xor(mx, d));
  float lsum = 0.f;
  float2 acc = make_float2(0.f, 0.f);
  for (int c0 = 0; c0 < nc; c0 += 64) {
    const int c = c0 + lane;
    float w = 0.f;
    if (c < nc) {
      w = exp2f(pp[(int64_t)c * kPart] - mx);
      lsum += pp[(int64_t)c * kPart + 1] * w;
    }
    s_w[lane] = w;
    __syncthreads();
    const int cn = min(64, nc - c0);
    const float* q = pp + (int64_t)c0 * kPart + 4 + 2 * lane;
    int i = 0;
    for (; i + 4 <= cn; i += 4) {
      const float2 v0 = *(const float2*)(q + (int64_t)i * kPart);
      const float2 v1 = *(const float2*)(q + (int64_t)(i + 1) * kPart);
      const float2 v2 = *(const float2*)(q + (int64_t)(i + 2) * kPart);
      const float2 v3 = *(const float2*)(q + (int64_t)(i + 3) * kPart);
      acc.x += v0.x * s_w[i] + v1.x * s_w[i + 1] + v2.x * s_w[i + 2] + v3.x * s_w[i + 3];
      acc.y += v0.y * s_w[i] + v1.y * s_w[i + 1] + v2.y * s_w[i + 2] + v3.y * s_w[i + 3];
    }
    for (; i < cn; ++i) {
      const float2 v = *(const float2*)(q + (int64_t)i * kPart);
      acc.x += v.x * s_w[i];
      acc.y += v.y * s_w[i];
    }
    __syncthreads();
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) lsum += __shfl_xor(lsum, d);
  const float inv = 1.f / lsum;
  const int l = l0 + lc;
  *(uint32_t*)(o + (((int64_t)l * b + s) * g.Hq + h) * kDh + 2 * lane) =
      pack2(acc.x * inv, acc.y * inv);
}

}  // namespace

// Keys per chunk of a decode call.
int decode_ck(const AppendDesc& a) { return a.batch == 1 ? kCK / 2 : kCK; }

int decode_chunks(const AppendDesc& a) { return (a.max_keys + decode_ck(a) - 1) / decode_ck(a); }

bool decode_mfma_ok(const PoolGeom& g, int dtype, const AppendDesc& a) {
  // ck % B == 0 with B >= 16 a power of two: at most 64 block ids per chunk;
  // any batch (query slices of 64 vectors cover batch x G)
  return dtype == KV_DTYPE_BF16 && g.dh == kDh && a.T == 1 && a.batch <= KV_MAX_BATCH &&
         decode_ck(a) % g.B == 0 && g.B >= 16 && g.b_shift >= 0;
}

namespace {
size_t unit_bytes(const AppendDesc& a) {
  return ((size_t)decode_chunks(a) * a.batch * sizeof(DecodeUnit) + 255) & ~size_t(255);
}
}  // namespace

// Split-key partials of one layer: [batch][Hq][chunks][kPart] floats.
size_t decode_part_layer_bytes(const PoolGeom& g, const AppendDesc& a) {
  return ((size_t)a.batch * g.Hq * decode_chunks(a) * kPart * sizeof(float) + 255) & ~size_t(255);
}

// The work plan: units [chunks][batch], then the unit count of each chunk.
size_t decode_plan_bytes(const AppendDesc& a) {
  return unit_bytes(a) + (((size_t)decode_chunks(a) * sizeof(int) + 255) & ~size_t(255));
}

size_t decode_scratch_bound(int64_t L, int64_t batch, int64_t Hq, int64_t max_keys) {
  // calls of any batch up to `batch`: kCK-key chunks, or kCK / 2 for a batch of one
  size_t worst = 0;
  for (const int64_t ck : {(int64_t)kCK, (int64_t)kCK / 2}) {
    const int64_t b = ck == kCK ? batch : 1;
    const int64_t chunks = (max_keys + ck - 1) / ck;
    worst = std::max(worst, (size_t)L * b * Hq * chunks * kPart * sizeof(float) +
                                (size_t)chunks * b * sizeof(DecodeUnit) +
                                (size_t)chunks * sizeof(int) + 3 * 256);
  }
  return worst;
}

namespace {
// Resident workgroups of k_decode_pers<NW, RT, S> on the current device: CUs
// x workgroups per CU (bounded by LDS and registers), cached per device.
template <int NW, int RT, int S>
int pers_slots() {
  static int cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cache[dev] == 0) {
    int cus = 0, per = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &per, reinterpret_cast<const void*>(&k_decode_pers<NW, RT, S>), 64 * NW, 0) !=
            hipSuccess)
      return 256;
    cache[dev] = std::max(1, cus * per);
  }
  return cache[dev];
}
}  // namespace

namespace {
// Items per resident slot up to which the persistent form is used (units of
// at most 64 query vectors).
constexpr int64_t kPersItemsPerSlot = 16;

template <int NW, int RT, int S>
void launch_pers(const PoolGeom& g, const void* qbuf, const AppendDesc& a, const DecodeUnit* units,
                 const int* n_units, float* part, int nch, int l0, int lc, float sc,
                 int64_t items_max, hipStream_t s) {
  const int w = (int)std::min<int64_t>(pers_slots<NW, RT, S>(), items_max);
  k_decode_pers<NW, RT, S><<<w, 64 * NW, 0, s>>>(g, (const uint16_t*)qbuf, a, units, n_units, part,
                                             nch, l0, lc, sc);
}
}  // namespace

hipError_t launch_decode_attn(const PoolGeom& g, const void* qbuf, const AppendDesc& a,
                              void* part_area, void* plan, int lc, int l0, hipStream_t s) {
  const int G = g.Hq / g.Hkv;
  const int nch = decode_chunks(a);
  const int ck = decode_ck(a);
  float* part = (float*)part_area;
  DecodeUnit* units = (DecodeUnit*)plan;
  int* n_units = (int*)((char*)plan + unit_bytes(a));
  if (l0 == 0) {  // the grouping holds for every layer group of the call
    const size_t dyn = (size_t)a.batch * (ck / g.B) * sizeof(int);
    k_decode_plan<<<nch, 64, dyn, s>>>(g, a, units, n_units, ck);
  }
  const float sc = 1.4426950408889634f / sqrtf((float)kDh);
  int slots = std::min(nch * a.batch, 2 * nch + a.batch);
  const int ns = (a.batch * G + 63) / 64;  // query slices of 64 vectors
  if (ns > 1) slots = (slots + 7) / 8 * 8;
  dim3 grid(slots * ns, g.Hkv, lc);
  // Units of 65 to 128 query vectors (at most kPersMaxChunks chunks): the
  // persistent form with four wavefronts of 32 vectors per workgroup sharing
  // one stage ring (32 agents x 4 query heads, 8192 keys, 32 layers: 341
  // against 496 us as query slices).  At most 64 vectors: the persistent form
  // (one wavefront per resident slot) only while each slot takes at most
  // kPersItemsPerSlot items (counting every (chunk, member) as a unit, an
  // upper bound), since each switch between items costs about one refill of
  // the ring; with more (batch one over a long context, 80 layers) the
  // per-unit kernel, whose start-up other wavefronts of the CU cover, is 3-5%
  // faster, with fewer (fork4-8b decode) 4-5% slower.  Otherwise one
  // wavefront per (unit, query slice of 64 vectors, KV head, layer): three
  // stages for one query tile, two for two (15% faster than three).
  const int vec = a.batch * G;
  const int64_t items_max = (int64_t)nch * a.batch * lc * g.Hkv;
  if (vec > 64 && vec <= 128 && nch <= kPersMaxChunks) {
    launch_pers<4, 1, 2>(g, qbuf, a, units, n_units, part, nch, l0, lc, sc, items_max, s);
  } else if (vec <= 32 && nch <= kPersMaxChunks &&
             items_max <= (int64_t)kPersItemsPerSlot * pers_slots<1, 1, 3>()) {
    launch_pers<1, 1, 3>(g, qbuf, a, units, n_units, part, nch, l0, lc, sc, items_max, s);
  } else if (vec > 32 && vec <= 64 && nch <= kPersMaxChunks &&
             items_max <= (int64_t)kPersItemsPerSlot * pers_slots<1, 2, 2>()) {
    launch_pers<1, 2, 2>(g, qbuf, a, units, n_units, part, nch, l0, lc, sc, items_max, s);
  } else if (a.batch * G <= 32)
    k_decode_stream<1, 3><<<grid, 64, 0, s>>>(g, (const uint16_t*)qbuf, a, units, n_units, part,
                                              nch, ck, l0, sc, 1);
  else
    k_decode_stream<2, 2><<<grid, 64, 0, s>>>(g, (const uint16_t*)qbuf, a, units, n_units, part,
                                              nch, ck, l0, sc, ns);
  return hipGetLastError();
}

hipError_t launch_decode_merge(const PoolGeom& g, const AppendDesc& a, void* o, const void* part,
                               int l0, int lc, hipStream_t s) {
  dim3 grid(a.batch * g.Hq, lc);
  k_decode_merge<<<grid, 64, 0, s>>>(g, a, (const float*)part, decode_chunks(a), decode_ck(a), (uint16_t*)o,
                                      l0);
  return hipGetLastError();
}

}  // namespace kvs
