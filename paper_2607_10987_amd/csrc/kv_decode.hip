// Decode attention (one new token per sequence) over the paged cache on MFMA,
// split over key chunks, reading each shared block once for the whole batch.
//
// Forked agents share the blocks of their common context (same physical ids
// in their block tables).  A workgroup owns one chunk of 512 key positions of
// one (layer, KV head); it groups the batch members whose block ids and key
// counts agree over the chunk, and for each group streams the chunk's K/V once
// while computing the scores of all of the group's query vectors (members x
// the G query heads of the KV head) with MFMA.  Per (query vector, chunk) it
// writes a partial (running max m, running sum l, unnormalised output o);
// k_decode_merge combines the chunks with the usual log-sum-exp rescaling.
//
// Inside a workgroup the chunk is walked in 4 tiles of 128 keys staged in LDS
// (K rows, V transposed on the way in, next tile prefetched into registers);
// wavefront w takes keys 32 w .. 32 w + 31 of each tile for every query
// vector, and the four wavefronts' partials are combined in LDS at the end.
// The MFMA products use the same transposed layout as the prefill kernel
// (query vector in the MFMA column, softmax state lane-local).
#include "kv_fast.h"

namespace kvs {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kDh = 128;
constexpr int kCK = 1024;        // keys per chunk (one workgroup)
constexpr int kTile = 128;       // keys per LDS tile
constexpr int kLd = kDh + 8;     // K row stride
constexpr int kVLd = kTile + 8;  // V^T row stride
constexpr int kPart = kDh + 4;   // floats per partial: m, l, pad, pad, o[128]

__device__ inline uint32_t pack2(float a, float b) {
  const __bf16 x = (__bf16)a, y = (__bf16)b;
  return (uint32_t)__builtin_bit_cast(uint16_t, x) | ((uint32_t)__builtin_bit_cast(uint16_t, y) << 16);
}

// grid (n_chunks, Hkv, lc), block 256.  RT = query-vector tiles of 32.
template <int RT>
__global__ void __launch_bounds__(256, RT == 1 ? 2 : 1)
k_decode_attn(PoolGeom g, const uint16_t* __restrict__ qbuf, AppendDesc a,
              float* __restrict__ part, int n_chunks, int l0, float qk_scale_log2) {
  constexpr int kKBytes = kTile * kLd * 2, kVBytes = kDh * kVLd * 2;
  __shared__ __attribute__((aligned(16))) char smem[kKBytes + kVBytes];
  extern __shared__ int s_tbl_dyn[];  // [batch][kCK / B] block ids of the chunk
  __shared__ int s_nk[KV_MAX_BATCH], s_lead[KV_MAX_BATCH], s_mem[KV_MAX_BATCH];
  __shared__ int s_nmem;
  uint16_t* sK = (uint16_t*)smem;
  uint16_t* sV = (uint16_t*)(smem + kKBytes);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hl = lane >> 5, col = lane & 31;
  const int c = blockIdx.x, gk = blockIdx.y, lc = blockIdx.z;
  const int G = g.Hq / g.Hkv;
  const int b = a.batch;
  const int M = b;  // T == 1
  const int c0 = c * kCK;
  const int nbc = kCK / g.B;  // table entries per chunk (B divides kCK, B >= 16)
  auto s_tbl = [&](int sq) -> int* { return s_tbl_dyn + sq * nbc; };
  const uint16_t* pool = (const uint16_t*)g.pool;
  const int layer = l0 + lc;

  // ---- key counts and block ids of each member in this chunk
  if (tid < b) {
    const int n = a.seq[tid].n_before + 1;
    s_nk[tid] = max(0, min(kCK, n - c0));
  }
  for (int i = tid; i < b * nbc; i += 256) {
    const int sq = i / nbc, j = i % nbc;
    const int n = a.seq[sq].n_before + 1;
    const int jb = c0 / g.B + j;
    s_tbl(sq)[j] = jb * g.B < n ? g.tables[(int64_t)a.seq[sq].slot * g.max_blocks + jb] : -1;
  }
  __syncthreads();
  // ---- group members with identical block ids over the chunk (leader = first)
  if (tid < b) {
    int lead = tid;
    const int nk = s_nk[tid];
    if (nk > 0) {
      const int nb = (nk + g.B - 1) / g.B;
      for (int sq = 0; sq < tid; ++sq) {
        if (s_nk[sq] != nk) continue;
        bool same = true;
        for (int j = 0; j < nb; ++j) same &= s_tbl(sq)[j] == s_tbl(tid)[j];
        if (same) {
          lead = sq;
          break;
        }
      }
    }
    s_lead[tid] = lead;
  }
  __syncthreads();

  for (int s0 = 0; s0 < b; ++s0) {
    if (s_lead[s0] != s0 || s_nk[s0] == 0) continue;  // uniform across the workgroup
    if (tid == 0) {
      int n = 0;
      for (int sq = s0; sq < b; ++sq)
        if (s_lead[sq] == s0) s_mem[n++] = sq;
      s_nmem = n;
    }
    __syncthreads();
    const int R = s_nmem * G;  // query vectors of this group (<= 32 RT)
    const int nk = s_nk[s0];
    const int* tb = s_tbl(s0);

    // Q operands: query vector r = member * G + head
    bf16x8 qf[RT][8];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int r = rt * 32 + col;
      const bool ok = r < R;
      const int mi = ok ? r / G : 0, w = ok ? r % G : 0;
      const int row = s_mem[mi];
      const uint16_t* qp = qbuf + (((int64_t)lc * M + row) * g.Hq + gk * G + w) * kDh;
#pragma unroll
      for (int ks = 0; ks < 8; ++ks)
        qf[rt][ks] = ok ? *(const bf16x8*)(qp + ks * 16 + hl * 8) : bf16x8{};
    }

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

    const int n_tiles = (nk + kTile - 1) / kTile;
    uint4 rk[8], rv[4][2];
    const int64_t koff = tile_off(g, layer, 0, gk, 0), voff = tile_off(g, layer, 1, gk, 0);
    auto kaddr = [&](int kk, int64_t base) -> const uint16_t* {
      return pool + (int64_t)tb[kk / g.B] * g.block_elems + base + (kk % g.B) * kDh;
    };
    auto gload = [&](int t) {
      const int k0 = t * kTile;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int q = tid + 256 * i, r = q >> 4, cc = q & 15;
        const int kk = k0 + r;
        rk[i] = kk < nk ? *(const uint4*)(kaddr(kk, koff) + cc * 8) : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = tid + 256 * i, kp = q & 63, cc = q >> 6;
        const int kk = k0 + 2 * kp;
        rv[i][0] = kk < nk ? *(const uint4*)(kaddr(kk, voff) + cc * 8) : make_uint4(0, 0, 0, 0);
        rv[i][1] = kk + 1 < nk ? *(const uint4*)(kaddr(kk + 1, voff) + cc * 8)
                               : make_uint4(0, 0, 0, 0);
      }
    };
    auto sstore = [&]() {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int q = tid + 256 * i, r = q >> 4, cc = q & 15;
        *(uint4*)(sK + r * kLd + cc * 8) = rk[i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = tid + 256 * i, kp = q & 63, cc = q >> 6;
        const uint32_t* a0 = (const uint32_t*)&rv[i][0];
        const uint32_t* a1 = (const uint32_t*)&rv[i][1];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t lo = (e & 1) ? (a0[e >> 1] >> 16) : (a0[e >> 1] & 0xffffu);
          const uint32_t hi = (e & 1) ? (a1[e >> 1] >> 16) : (a1[e >> 1] & 0xffffu);
          *(uint32_t*)(sV + (cc * 8 + e) * kVLd + 2 * kp) = lo | (hi << 16);
        }
      }
    };

    for (int t = 0; t < n_tiles; ++t) {
      gload(t);         // two workgroups per CU hide each other's load latency
      __syncthreads();  // previous tile fully consumed
      sstore();
      __syncthreads();
      const int kw = wave * 32;  // this wave's keys within the tile
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        floatx16 sacc;
#pragma unroll
        for (int e = 0; e < 16; ++e) sacc[e] = 0.f;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
          const bf16x8 kf = *(const bf16x8*)(sK + (kw + col) * kLd + ks * 16 + hl * 8);
          sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[rt][ks], sacc, 0, 0, 0);
        }
        float mx = -INFINITY;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int kk = t * kTile + kw + (e >> 2) * 8 + hl * 4 + (e & 3);
          float sv = sacc[e] * qk_scale_log2;
          if (kk >= nk) sv = -INFINITY;
          sacc[e] = sv;
          mx = fmaxf(mx, sv);
        }
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run[rt], mx);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = exp2f(m_run[rt] - m_use);
        float ps = 0.f;
        bf16x8 pf[2];
#pragma unroll
        for (int hs = 0; hs < 2; ++hs) {
          float p[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            p[j] = exp2f(sacc[hs * 8 + j] - m_use);
            ps += p[j];
          }
          uint32_t wds[4] = {pack2(p[0], p[1]), pack2(p[2], p[3]), pack2(p[4], p[5]),
                             pack2(p[6], p[7])};
          pf[hs] = __builtin_bit_cast(bf16x8, *(uint4*)wds);
        }
        l_run[rt] = l_run[rt] * alpha + ps;
        m_run[rt] = m_new;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
#pragma unroll
          for (int e = 0; e < 16; ++e) oacc[rt][mt][e] *= alpha;
#pragma unroll
          for (int hs = 0; hs < 2; ++hs) {
            const uint16_t* vp = sV + (mt * 32 + col) * kVLd + kw + hs * 16 + hl * 4;
            const uint2 v0 = *(const uint2*)vp;
            const uint2 v1 = *(const uint2*)(vp + 8);
            const uint4 vv = make_uint4(v0.x, v0.y, v1.x, v1.y);
            oacc[rt][mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8, vv), pf[hs], oacc[rt][mt], 0, 0, 0);
          }
        }
      }
    }

    // ---- combine the four wavefronts per query vector, write partials
    float* so = (float*)smem;             // [4 waves][32 vectors][128]
    float* sm = so + 4 * 32 * kDh;        // [4 waves][32] m, then [4][32] l
    static_assert(4 * 32 * kDh * 4 + 2 * 4 * 32 * 4 <= kKBytes + kVBytes, "combine scratch");
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      __syncthreads();  // LDS tiles (or the previous round) no longer read
      const float lt = l_run[rt] + __shfl_xor(l_run[rt], 32);
      if (hl == 0) {
        sm[wave * 32 + col] = m_run[rt];
        sm[128 + wave * 32 + col] = lt;
      }
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int dc = mt * 32 + q * 8 + hl * 4;
          *(float4*)(so + (wave * 32 + col) * kDh + dc) =
              make_float4(oacc[rt][mt][q * 4], oacc[rt][mt][q * 4 + 1], oacc[rt][mt][q * 4 + 2],
                          oacc[rt][mt][q * 4 + 3]);
        }
      __syncthreads();
      for (int i = tid; i < 32 * (kDh / 4); i += 256) {
        const int r = i / (kDh / 4), d4 = (i % (kDh / 4)) * 4;
        const int rr = rt * 32 + r;
        if (rr >= R) continue;
        float mw[4], m2 = -INFINITY;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          mw[w] = sm[w * 32 + r];
          m2 = fmaxf(m2, mw[w]);
        }
        const float mu = m2 == -INFINITY ? 0.f : m2;
        float4 acc4 = make_float4(0.f, 0.f, 0.f, 0.f);
        float l2 = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const float sc = exp2f(mw[w] - mu);
          const float4 v = *(const float4*)(so + (w * 32 + r) * kDh + d4);
          acc4.x += v.x * sc;
          acc4.y += v.y * sc;
          acc4.z += v.z * sc;
          acc4.w += v.w * sc;
          l2 += sm[128 + w * 32 + r] * sc;
        }
        const int sq = s_mem[rr / G], h = gk * G + rr % G;
        float* pp = part + ((((int64_t)lc * b + sq) * g.Hq + h) * n_chunks + c) * kPart;
        *(float4*)(pp + 4 + d4) = acc4;
        if (d4 == 0) {
          pp[0] = m2;
          pp[1] = l2;
        }
      }
    }
    __syncthreads();  // partial writes done with the LDS before the next group
  }
}

// grid (batch * Hq, lc), block 128: combine the chunk partials of one query.
__global__ void __launch_bounds__(128)
k_decode_merge(PoolGeom g, AppendDesc a, const float* __restrict__ part, int n_chunks,
               uint16_t* __restrict__ o, int l0) {
  const int sh = blockIdx.x, lc = blockIdx.y;
  const int s = sh / g.Hq, h = sh % g.Hq;
  const int b = a.batch;
  const int n = a.seq[s].n_before + 1;
  const int nc = (n + kCK - 1) / kCK;
  const float* pp = part + (((int64_t)lc * b + s) * g.Hq + h) * n_chunks * kPart;
  float mx = -INFINITY;
  for (int c = 0; c < nc; ++c) mx = fmaxf(mx, pp[c * kPart]);
  float lsum = 0.f, acc = 0.f;
  const int dc = threadIdx.x;
  for (int c = 0; c < nc; ++c) {
    const float wgt = exp2f(pp[c * kPart] - mx);
    lsum += pp[c * kPart + 1] * wgt;
    acc += pp[c * kPart + 4 + dc] * wgt;
  }
  const int l = l0 + lc;
  const float v = acc / lsum;
  const __bf16 bv = (__bf16)v;
  o[(((int64_t)l * b + s) * g.Hq + h) * kDh + dc] = __builtin_bit_cast(uint16_t, bv);
}

}  // namespace

int decode_chunks(const AppendDesc& a) { return (a.max_keys + kCK - 1) / kCK; }

bool decode_mfma_ok(const PoolGeom& g, int dtype, const AppendDesc& a) {
  const int G = g.Hq / g.Hkv;
  return dtype == KV_DTYPE_BF16 && g.dh == kDh && a.T == 1 && a.batch * G <= 64 &&
         kCK % g.B == 0 && g.B >= 16;
}

size_t decode_part_bytes(const PoolGeom& g, const AppendDesc& a) {
  return (size_t)g.L * a.batch * g.Hq * decode_chunks(a) * kPart * sizeof(float);
}

hipError_t launch_decode_attn(const PoolGeom& g, const void* qbuf, const AppendDesc& a,
                              void* part, int lc, int l0, hipStream_t s) {
  const int G = g.Hq / g.Hkv;
  const int nch = decode_chunks(a);
  const float sc = 1.4426950408889634f / sqrtf((float)kDh);
  dim3 grid(nch, g.Hkv, lc);
  const size_t dyn = (size_t)a.batch * (kCK / g.B) * sizeof(int);
  if (a.batch * G <= 32)
    k_decode_attn<1><<<grid, 256, dyn, s>>>(g, (const uint16_t*)qbuf, a, (float*)part, nch, l0,
                                            sc);
  else
    k_decode_attn<2><<<grid, 256, dyn, s>>>(g, (const uint16_t*)qbuf, a, (float*)part, nch, l0,
                                            sc);
  return hipGetLastError();
}

hipError_t launch_decode_merge(const PoolGeom& g, const AppendDesc& a, void* o, const void* part,
                               int l0, int lc, hipStream_t s) {
  dim3 grid(a.batch * g.Hq, lc);
  k_decode_merge<<<grid, 128, 0, s>>>(g, a, (const float*)part, decode_chunks(a), (uint16_t*)o,
                                      l0);
  return hipGetLastError();
}

}  // namespace kvs
