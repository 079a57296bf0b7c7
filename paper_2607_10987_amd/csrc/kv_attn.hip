// Causal grouped-query attention over the paged cache on MFMA (bf16 inputs,
// fp32 softmax and accumulation), head_dim 128.
//
// One workgroup = one sequence's tile of 32 query tokens x one KV head x one
// layer; wavefront w handles query head g * G + w, so the G heads that share
// a KV head share every K / V tile staged in LDS.  Keys are walked in tiles of
// 64 (4 paged blocks of 16, or 2 of 32), looked up through the block table.
//
// Both products keep the query token in the MFMA "column" so that every
// per-token quantity is lane-local:
//   S^T [64 keys x 32 tok] = K [keys x dh] . Q^T      (A: K rows from LDS,
//                                                     B: Q rows, registers)
//   O^T [dh x 32 tok]     += V^T [dh x keys] . P^T     (A: V^T from LDS,
//                                                     B: P from registers)
// In the C layout of v_mfma_f32_32x32x16_bf16 a lane holds keys
// {8q + 4h + r : q < 4, r < 4} of its token (h = lane / 32).  Taking the PV
// contraction over keys in the order (4h + r, 8 + 4h + r) for each group of
// 16 keys makes those registers exactly the B operand, so P never leaves the
// lane; V^T is staged in LDS (transposed on the way in) and read with the
// same key order.  Softmax: running max / running sum per token in base 2
// (scores pre-multiplied by log2(e) / sqrt(dh)), halves of a token combined
// with one lane swap.
#include "kv_dma.h"
#include "kv_fast.h"

namespace kvs {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kDh = 128;
constexpr int kQT = 32;            // query tokens per workgroup
constexpr int kKT = 64;            // keys per tile
constexpr int kKLd = kDh + 8;      // K tile row stride (elements)
constexpr int kVLd = kKT + 8;      // V^T tile row stride (elements)
constexpr int kStage = kKT * kKLd + kDh * kVLd;

__device__ inline uint32_t pack2(float a, float b) {
  const __bf16 x = (__bf16)a, y = (__bf16)b;
  return (uint32_t)__builtin_bit_cast(uint16_t, x) | ((uint32_t)__builtin_bit_cast(uint16_t, y) << 16);
}

template <int G>
__global__ void __launch_bounds__(64 * G, 8 / G)
k_attn_prefill(PoolGeom g, const uint16_t* __restrict__ qbuf, AppendDesc a,
               uint16_t* __restrict__ o, int l0, float qk_scale_log2) {
  constexpr int NT = 64 * G;
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * kStage];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hl = lane >> 5;       // lane half
  const int col = lane & 31;      // token within the tile
  const int qt_per_seq = (a.T + kQT - 1) / kQT;
  const int seq = blockIdx.x / qt_per_seq;
  const int qt = qt_per_seq - 1 - (blockIdx.x % qt_per_seq);  // long tiles first
  const int gk = blockIdx.y;
  const int lc = blockIdx.z, l = l0 + lc;
  const int M = a.batch * a.T;
  const SeqDesc sd = a.seq[seq];
  const int n_keys = sd.n_before + a.T;
  const int t0 = qt * kQT;
  const int tq = t0 + col;                      // this lane's query token
  const int uq = sd.n_before + tq;              // its key index (causal limit)
  const bool q_valid = tq < a.T;
  const int key_end = min(n_keys, sd.n_before + t0 + kQT);  // keys this tile can see
  const int n_tiles = (key_end + kKT - 1) / kKT;
  const int h = gk * G + wave;
  const int32_t* trow = g.tables + (int64_t)sd.slot * g.max_blocks;
  const uint16_t* pool = (const uint16_t*)g.pool;

  // Q^T operand: token col, dh chunk (ks * 16 + hl * 8 .. + 8), 8 k-steps
  bf16x8 qf[8];
  {
    const int row = seq * a.T + min(tq, a.T - 1);
    const uint16_t* qp = qbuf + (((int64_t)lc * M + row) * g.Hq + h) * kDh;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) qf[ks] = *(const bf16x8*)(qp + ks * 16 + hl * 8);
  }

  // tile loaders: K rows [64][128] and V transposed [128][64]
  constexpr int KCH = kKT * kDh / 8 / NT;        // 16-byte K chunks per thread
  constexpr int VIT = (kKT / 2) * (kDh / 8) / NT; // V items (key pair, 8 channels) per thread
  uint4 rk[KCH], rv[VIT][2];
  auto key_addr = [&](int kk, int kv) -> const uint16_t* {
    const int32_t blk = trow[kk / g.B];
    return pool + (int64_t)blk * g.block_elems + tile_off(g, l, kv, gk, kk % g.B);
  };
  auto gload = [&](int tile) {
    const int k0 = tile * kKT;
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int q = tid + NT * i, r = q >> 4, c = q & 15;
      const int kk = k0 + r;
      rk[i] = kk < n_keys ? *(const uint4*)(key_addr(kk, 0) + c * 8) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < VIT; ++i) {
      const int q = tid + NT * i, kp = q & 31, c = q >> 5;
      const int kk = k0 + 2 * kp;
      rv[i][0] = kk < n_keys ? *(const uint4*)(key_addr(kk, 1) + c * 8) : make_uint4(0, 0, 0, 0);
      rv[i][1] = kk + 1 < n_keys ? *(const uint4*)(key_addr(kk + 1, 1) + c * 8)
                                 : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int buf) {
    uint16_t* Ks = smem + buf * kStage;
    uint16_t* Vt = Ks + kKT * kKLd;
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int q = tid + NT * i, r = q >> 4, c = q & 15;
      *(uint4*)(Ks + r * kKLd + c * 8) = rk[i];
    }
#pragma unroll
    for (int i = 0; i < VIT; ++i) {
      const int q = tid + NT * i, kp = q & 31, c = q >> 5;
      const uint32_t* a0 = (const uint32_t*)&rv[i][0];
      const uint32_t* a1 = (const uint32_t*)&rv[i][1];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t lo = (e & 1) ? (a0[e >> 1] >> 16) : (a0[e >> 1] & 0xffffu);
        const uint32_t hi = (e & 1) ? (a1[e >> 1] >> 16) : (a1[e >> 1] & 0xffffu);
        *(uint32_t*)(Vt + (c * 8 + e) * kVLd + 2 * kp) = lo | (hi << 16);
      }
    }
  };

  floatx16 oacc[4];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[mt][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  gload(0);
  sstore(0);
  __syncthreads();
  for (int tile = 0; tile < n_tiles; ++tile) {
    const int cur = tile & 1;
    if (tile + 1 < n_tiles) gload(tile + 1);
    const uint16_t* Ks = smem + cur * kStage;
    const uint16_t* Vt = Ks + kKT * kKLd;
    const int k0 = tile * kKT;

    // S^T = K Q^T for two 32-key halves of the tile
    floatx16 sacc[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) sacc[kt][e] = 0.f;
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        const bf16x8 kf = *(const bf16x8*)(Ks + (kt * 32 + col) * kKLd + ks * 16 + hl * 8);
        sacc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], sacc[kt], 0, 0, 0);
      }
    }
    // mask, running max on raw scores (scale > 0 commutes with max)
    const bool need_mask = k0 + kKT - 1 > sd.n_before + t0 || k0 + kKT > n_keys || !q_valid;
    float mt_max = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float s = sacc[kt][e];
        if (need_mask) {
          const int kk = k0 + kt * 32 + (e >> 2) * 8 + hl * 4 + (e & 3);
          if (kk > uq || kk >= n_keys) s = -INFINITY;
        }
        sacc[kt][e] = s;
        mt_max = fmaxf(mt_max, s);
      }
    mt_max = fmaxf(mt_max, __shfl_xor(mt_max, 32)) * qk_scale_log2;
    // Lazy rescaling: the running max only moves when a score exceeds it by
    // more than 2^8 in the exponent; until then p <= 256, exact in fp32 and
    // representable in bf16, and O is not rescaled (the final division by l
    // uses the same reference, so the result is unchanged).
    const float m_new = mt_max > m_run + 8.f ? mt_max : m_run;
    const float m_use = m_new == -INFINITY ? 0.f : m_new;  // fully masked (padding) rows
    const bool moved = __ballot(m_new != m_run) != 0;
    float psum = 0.f;
    bf16x8 pf[4];  // B operands of the PV product, one per 16-key step
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int hs = 0; hs < 2; ++hs) {
        float p[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          p[j] = exp2f(fmaf(sacc[kt][hs * 8 + j], qk_scale_log2, -m_use));
          psum += p[j];
        }
        uint32_t w[4] = {pack2(p[0], p[1]), pack2(p[2], p[3]), pack2(p[4], p[5]),
                         pack2(p[6], p[7])};
        pf[kt * 2 + hs] = __builtin_bit_cast(bf16x8, *(uint4*)w);
      }
    if (moved) {
      const float alpha = exp2f(m_run - m_use);
      l_run *= alpha;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[mt][e] *= alpha;
    }
    l_run += psum;
    m_run = m_new;
    // O^T += V^T P^T; 16-key step s covers keys 16 s + {4h + r, 8 + 4h + r}
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const uint16_t* vp = Vt + (mt * 32 + col) * kVLd + s4 * 16 + hl * 4;
        const uint2 v0 = *(const uint2*)vp;
        const uint2 v1 = *(const uint2*)(vp + 8);
        const uint4 vv = make_uint4(v0.x, v0.y, v1.x, v1.y);
        oacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vv), pf[s4],
                                                           oacc[mt], 0, 0, 0);
      }
    }
    if (tile + 1 < n_tiles) sstore(cur ^ 1);
    __syncthreads();
  }

  // normalise and store: lane holds channels 32 mt + 8 q + 4 h + r of its token
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!q_valid) return;
  const float inv = 1.f / l_tot;
  const int row = seq * a.T + tq;
  uint16_t* op = o + (((int64_t)l * M + row) * g.Hq + h) * kDh;
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int c0 = mt * 32 + q * 8 + hl * 4;
      *(uint2*)(op + c0) = make_uint2(pack2(oacc[mt][q * 4] * inv, oacc[mt][q * 4 + 1] * inv),
                                      pack2(oacc[mt][q * 4 + 2] * inv, oacc[mt][q * 4 + 3] * inv));
    }
}

// ---------------------------------------------------------------------------
// Pipelined variant: K and V tiles stream straight from the paged pool into
// LDS (global_load_lds_dwordx4, three tiles in flight), unpadded 256-byte key
// rows with the 16-byte chunk c of row r stored at slot c ^ (r & 15), so that
// 16 consecutive rows read at one chunk hit 16 distinct bank groups.  V stays
// in key-major order; its MFMA operand (4 consecutive keys of one channel per
// half) is read with ds_read_b64_tr_b16: within each group of 16 lanes, lane
// i addressing row key0 + i / 4, channels c0 + 4 (i % 4) .. + 3 receives the
// 4 keys key0 .. key0 + 3 of channel c0 + i.  Eight wavefronts: G query heads
// x (8 / G) groups of 32 query tokens share every staged tile.  The block
// table slice the workgroup needs is staged in LDS once.
constexpr int kPW = 8;                 // wavefronts per workgroup
constexpr int kPS = 3;                 // pipeline stages
constexpr int kPTile = kKT * kDh;      // elements of one K (or V) tile

typedef short v4s __attribute__((ext_vector_type(4)));
#define KV_LDS4(p) ((__attribute__((address_space(3))) v4s*)(p))

template <int G>
__global__ void __launch_bounds__(64 * kPW, 1)
k_attn_pipe(PoolGeom g, const uint16_t* __restrict__ qbuf, AppendDesc a,
            uint16_t* __restrict__ o, int l0, float qk_scale_log2) {
  constexpr int TG = kPW / G;       // token groups of 32
  constexpr int QT = 32 * TG;       // query tokens per workgroup
  __shared__ __attribute__((aligned(16))) uint16_t smem[kPS * 2 * kPTile];
  extern __shared__ int s_tbl[];    // block ids of the keys this workgroup reads
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hl = lane >> 5, col = lane & 31;
  const int tg = wave / G, hw = wave % G;
  const int qt_per_seq = (a.T + QT - 1) / QT;
  const int seq = blockIdx.x / qt_per_seq;
  const int qt = qt_per_seq - 1 - (blockIdx.x % qt_per_seq);  // long tiles first
  const int gk = blockIdx.y;
  const int lc = blockIdx.z, l = l0 + lc;
  const int M = a.batch * a.T;
  const SeqDesc sd = a.seq[seq];
  const int n_keys = sd.n_before + a.T;
  const int t0 = qt * QT;
  const int tq = t0 + tg * 32 + col;
  const int uq = sd.n_before + tq;
  const bool q_valid = tq < a.T;
  const int key_end = min(n_keys, sd.n_before + t0 + QT);
  const int n_tiles = (key_end + kKT - 1) / kKT;
  const int h = gk * G + hw;
  const uint16_t* pool = (const uint16_t*)g.pool;

  // stage the block ids of keys [0, key_end) in LDS
  const int nbl = (key_end + g.B - 1) / g.B;
  const int32_t* trow = g.tables + (int64_t)sd.slot * g.max_blocks;
  for (int i = tid; i < nbl; i += 64 * kPW) s_tbl[i] = trow[i];

  // Q^T operand (registers for the whole loop)
  bf16x8 qf[8];
  {
    const int row = seq * a.T + min(tq, a.T - 1);
    const uint16_t* qp = qbuf + (((int64_t)lc * M + row) * g.Hq + h) * kDh;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) qf[ks] = *(const bf16x8*)(qp + ks * 16 + hl * 8);
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) settle(qf[ks]);
  }
  __syncthreads();  // s_tbl ready

  // tile loads: 16 instructions of 1 KiB per operand (4 key rows each); wave w
  // issues instructions w and w + 8 of K and of V
  const int64_t koff = tile_off(g, l, 0, gk, 0), voff = tile_off(g, l, 1, gk, 0);
  auto issue = [&](int tile, int buf) {
    uint16_t* Ks = smem + buf * 2 * kPTile;
    uint16_t* Vs = Ks + kPTile;
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      const int j = wave + jj * kPW;
      const int r = j * 4 + (lane >> 4);
      const int c = (lane & 15) ^ (r & 15);
      const int key = min(tile * kKT + r, key_end - 1);  // rows past the end: any staged key
      const int64_t base = (int64_t)s_tbl[key >> g.b_shift] * g.block_elems +
                           (key & (g.B - 1)) * kDh + c * 8;
      lds_dma16(pool + base + koff, Ks + j * 512);
      lds_dma16(pool + base + voff, Vs + j * 512);
    }
  };

  floatx16 oacc[4];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int e = 0; e < 16; ++e) oacc[mt][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  for (int st = 0; st < kPS - 1 && st < n_tiles; ++st) issue(st, st);
  for (int tile = 0; tile < n_tiles; ++tile) {
    if (tile + 1 < n_tiles)
      wait_vmcnt<4>();  // the next tile (4 copies per wave) may be pending
    else
      wait_vmcnt<0>();
    lds_barrier();
    if (tile + kPS - 1 < n_tiles) issue(tile + kPS - 1, (tile + kPS - 1) % kPS);
    const uint16_t* Ks = smem + (tile % kPS) * 2 * kPTile;
    const uint16_t* Vs = Ks + kPTile;
    const int k0 = tile * kKT;

    floatx16 sacc[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
      for (int e = 0; e < 16; ++e) sacc[kt][e] = 0.f;
      const int r = kt * 32 + col;
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        const bf16x8 kf = *(const bf16x8*)(Ks + r * kDh + (((ks * 2 + hl) ^ (r & 15)) * 8));
        sacc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], sacc[kt], 0, 0, 0);
      }
    }
    // wave-uniform: does any (query, key) pair of this tile need masking?
    const bool need_mask = k0 + kKT - 1 > sd.n_before + t0 + tg * 32 || k0 + kKT > n_keys ||
                           t0 + tg * 32 + 31 >= a.T;
    float mt_max = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float sv = sacc[kt][e];
        if (need_mask) {
          const int kk = k0 + kt * 32 + (e >> 2) * 8 + hl * 4 + (e & 3);
          if (kk > uq || kk >= n_keys) sv = -INFINITY;
        }
        sacc[kt][e] = sv;
        mt_max = fmaxf(mt_max, sv);
      }
    mt_max = fmaxf(mt_max, __shfl_xor(mt_max, 32)) * qk_scale_log2;
    const float m_new = mt_max > m_run + 8.f ? mt_max : m_run;
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const bool moved = __builtin_amdgcn_readfirstlane((int)(__ballot(m_new != m_run) != 0)) != 0;
    float psum = 0.f;
    bf16x8 pf[4];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int hs = 0; hs < 2; ++hs) {
        float p[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          p[j] = __builtin_amdgcn_exp2f(fmaf(sacc[kt][hs * 8 + j], qk_scale_log2, -m_use));
          psum += p[j];
        }
        uint32_t wv[4] = {pack2(p[0], p[1]), pack2(p[2], p[3]), pack2(p[4], p[5]),
                          pack2(p[6], p[7])};
        pf[kt * 2 + hs] = __builtin_bit_cast(bf16x8, *(uint4*)wv);
      }
    if (moved) {
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
      l_run *= alpha;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[mt][e] *= alpha;
    }
    l_run += psum;
    m_run = m_new;
    // O^T += V^T P^T, V^T operands by transposed LDS reads
    const int gi = lane >> 4, li = lane & 15;
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
      const int key_a = s4 * 16 + (gi >> 1) * 4 + (li >> 2);
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const int dc = mt * 32 + (gi & 1) * 16 + (li & 3) * 4;
        const int ch = dc >> 3, hf = (dc & 7);
        const v4s r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            KV_LDS4(Vs + key_a * kDh + ((ch ^ (key_a & 15)) * 8) + hf));
        const int key_b = key_a + 8;
        const v4s r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            KV_LDS4(Vs + key_b * kDh + ((ch ^ (key_b & 15)) * 8) + hf));
        const v4s vv[2] = {r0, r1};
        oacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vv), pf[s4],
                                                           oacc[mt], 0, 0, 0);
      }
    }
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!q_valid) return;
  const float inv = 1.f / l_tot;
  const int row = seq * a.T + tq;
  uint16_t* op = o + (((int64_t)l * M + row) * g.Hq + h) * kDh;
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int c0 = mt * 32 + q * 8 + hl * 4;
      *(uint2*)(op + c0) = make_uint2(pack2(oacc[mt][q * 4] * inv, oacc[mt][q * 4 + 1] * inv),
                                      pack2(oacc[mt][q * 4 + 2] * inv, oacc[mt][q * 4 + 3] * inv));
    }
}

}  // namespace

bool attn_mfma_ok(const PoolGeom& g, int dtype) {
  const int G = g.Hq / g.Hkv;
  return dtype == KV_DTYPE_BF16 && g.dh == kDh && (G == 4 || G == 8) && g.b_shift >= 0;
}

hipError_t launch_attn_prefill(const PoolGeom& g, const void* qbuf, const AppendDesc& a, void* o,
                               int l0, int lc, hipStream_t s) {
  const int G = g.Hq / g.Hkv;
  {
    const int QT = 32 * (kPW / G);
    const int qt = (a.T + QT - 1) / QT;
    dim3 grid(a.batch * qt, g.Hkv, lc);
    const float sc = 1.4426950408889634f / sqrtf((float)kDh);
    const size_t dyn = (size_t)((a.max_keys + g.B - 1) / g.B) * sizeof(int);
    if (G == 4)
      k_attn_pipe<4><<<grid, 64 * kPW, dyn, s>>>(g, (const uint16_t*)qbuf, a, (uint16_t*)o, l0,
                                                  sc);
    else
      k_attn_pipe<8><<<grid, 64 * kPW, dyn, s>>>(g, (const uint16_t*)qbuf, a, (uint16_t*)o, l0,
                                                  sc);
    return hipGetLastError();
  }
  const int qt = (a.T + kQT - 1) / kQT;
  dim3 grid(a.batch * qt, g.Hkv, lc);
  const float sc = 1.4426950408889634f / sqrtf((float)kDh);
  if (G == 4)
    k_attn_prefill<4><<<grid, 256, 0, s>>>(g, (const uint16_t*)qbuf, a, (uint16_t*)o, l0, sc);
  else
    k_attn_prefill<8><<<grid, 512, 0, s>>>(g, (const uint16_t*)qbuf, a, (uint16_t*)o, l0, sc);
  return hipGetLastError();
}

}  // namespace kvs
