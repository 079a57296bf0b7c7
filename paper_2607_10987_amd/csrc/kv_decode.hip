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
// k_decode_stream runs one wavefront per (unit, query slice, KV head, layer)
// with no workgroup barriers: it streams the unit's K/V rows once, 32 keys at a time,
// through a ring of LDS stages filled by direct global->LDS copies, and scores
// all of the group's query vectors (members x the G query heads of the KV
// head) with MFMA in the transposed layout of the prefill kernel (query vector
// in the MFMA column, softmax state lane-local, V^T operands by transposed LDS
// reads).  Per (query vector, chunk) it writes a partial (running max m,
// running sum l, unnormalised output o); k_decode_merge combines the chunks of
// a query with the usual log-sum-exp rescaling.  A unit's query vectors are
// taken 64 at a time (two MFMA column tiles): a unit with more (e.g. 32
// members x 4 query heads) is split into query slices, each a wavefront of
// its own that streams the same keys; the slices of a unit are launched on
// one XCD, so the later ones find the keys in its L2.
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

// One work unit: the members in `mask` share block ids and key count `nk`
// over the chunk; `lead` is the first of them.
struct DecodeUnit {
  int32_t lead, nk;
  uint32_t mask_lo, mask_hi;
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
  if (lane < n_groups)
    units[c * b + lane] = DecodeUnit{g_lead, g_nk, (uint32_t)g_mask, (uint32_t)(g_mask >> 32)};
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
  const int lane = threadIdx.x, hl = lane >> 5, col = lane & 31;
  const int gk = blockIdx.y, lc = blockIdx.z, layer = l0 + lc;
  const int G = g.Hq / g.Hkv, b = a.batch, M = b;  // T == 1
  const uint16_t* pool = (const uint16_t*)g.pool;
  const int64_t koff = tile_off(g, layer, 0, gk, 0), voff = tile_off(g, layer, 1, gk, 0);

  int total = 0;
  for (int cb = 0; cb < n_chunks; cb += 64) {
    int v = cb + lane < n_chunks ? n_units[cb + lane] : 0;
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d);
    total += v;
  }
  total = __builtin_amdgcn_readfirstlane(total);
  const uint32_t lds0 = lds_addr(smem);
  const int64_t kv_gap = (voff - koff) * 2;  // bytes from a K row to its V row

  const int x = blockIdx.x;
  const int slot = ns == 1 ? x : (x / (8 * ns)) * 8 + (x & 7);
  const int qs = ns == 1 ? 0 : (x >> 3) % ns;
  const int stride = gridDim.x / ns;
  for (int u = slot; u < total; u += stride) {
    int c, gi;
    locate_unit(n_units, n_chunks, u, &c, &gi);
    c = __builtin_amdgcn_readfirstlane(c);
    gi = __builtin_amdgcn_readfirstlane(gi);
    const DecodeUnit* up = units + c * b + gi;
    const int nk = __builtin_amdgcn_readfirstlane(up->nk);
    const int lead = __builtin_amdgcn_readfirstlane(up->lead);
    const uint64_t mask = ((uint64_t)__builtin_amdgcn_readfirstlane(up->mask_hi) << 32) |
                          (uint32_t)__builtin_amdgcn_readfirstlane(up->mask_lo);
    const int R = __popcll(mask) * G;  // query vectors of the unit
    const int q0 = qs * 32 * RT;       // this slice's first query vector
    if (q0 >= R) continue;             // wave-uniform: a unit with fewer slices
    const bool two = RT > 1 && R - q0 > 32;
    const int c0 = c * ck;
    // lane j: block id of the leader's entry j of the chunk (0 past the end)
    const int tbl = (lane << g.b_shift) < nk
                        ? g.tables[(int64_t)a.seq[lead].slot * g.max_blocks +
                                   (c0 >> g.b_shift) + lane]
                        : 0;

    // Q^T operands: query vector r = (member rank) * G + head
    bf16x8 qf[RT][8];
    int qrow[RT], qhead[RT];
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
    int tb = tbl;
    settle(tb);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) settle(qf[rt][ks]);

    // stage loads: 8 copies of 1 KiB (4 key rows, all in one block since
    // B >= 16) per operand, block base in scalar registers, non-temporal
    // (each byte is read once per call).  Rows past the
    // unit's last key read slots of a real block; their scores are masked and
    // their V rows zeroed in LDS before use.
    auto issue = [&](int tile, int buf) {
      const uint32_t ks_lds = lds0 + buf * kStage * 2;
#pragma unroll
      for (int j = 0; j < kKT / 4; ++j) {
        const int key0 = tile * kKT + j * 4;
        const int id = __builtin_amdgcn_readlane(tb, key0 >> g.b_shift);
        const char* kb = (const char*)pool +
                         ((int64_t)id * g.block_elems + koff + (key0 & (g.B - 1)) * kDh) * 2;
        const int r = j * 4 + (lane >> 4);
        const uint32_t ko = (lane >> 4) * (kDh * 2) + (((lane & 15) ^ kswz(r)) * 16);
        const uint32_t vo = (lane >> 4) * (kDh * 2) + (((lane & 15) ^ vswz(r)) * 16);
        lds_dma16_sv_nt(kb, ko, ks_lds + j * 1024);
        lds_dma16_sv_nt(kb + kv_gap, vo, ks_lds + kKT * kDh * 2 + j * 1024);
      }
    };

    floatx16 oacc[RT][4];
    float m_run[RT], l_run[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      m_run[rt] = -INFINITY;
      l_run[rt] = 0.f;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[rt][mt][e] = 0.f;
    }

    const int n_tiles = (nk + kKT - 1) / kKT;
    for (int st = 0; st < S - 1 && st < n_tiles; ++st) issue(st, st);
    for (int t = 0; t < n_tiles; ++t) {
      // copies of this wave complete in order: stage t is ready once at most
      // the stages issued after it are pending (2 * kKT / 4 copies each)
      const int ahead = min(S - 2, n_tiles - 1 - t);
      if (ahead >= 2)
        wait_vmcnt<4 * kKT / 4>();
      else if (ahead == 1)
        wait_vmcnt<2 * kKT / 4>();
      else
        wait_vmcnt<0>();
      // stage (t - 1) % S was consumed in the previous iteration
      if (t + S - 1 < n_tiles) issue(t + S - 1, (t + S - 1) % S);
      const uint16_t* Ks = smem + (t % S) * kStage;
      const uint16_t* Vs = Ks + kKT * kDh;
      const int k0 = t * kKT;
      const bool tail = k0 + kKT > nk;  // wave-uniform
      if (tail) {  // V rows of keys >= nk may hold anything: zero them
        uint16_t* Vw = (uint16_t*)Vs;
        for (int i = (nk - k0) * (kDh / 8) + lane; i < kKT * (kDh / 8); i += 64)
          *(uint4*)(Vw + i * 8) = make_uint4(0, 0, 0, 0);
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
      // O^T += V^T P^T, V^T operands by transposed LDS reads
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

    // partials of this unit's query vectors for chunk c
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
  // one query tile: three 16 KiB stages per wave (two in flight), 3-4%
  // faster than two, while four are 9% slower; the number of bytes in flight
  // per CU, bounded by LDS, is what limits this stream.  Two query tiles (more
  // than 32 query vectors per unit): two stages, 15% faster than three.
  if (a.batch * G <= 32)
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
