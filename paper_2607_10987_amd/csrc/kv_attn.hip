// Causal grouped-query attention of an append (prefill) over the paged cache
// on MFMA: bf16 inputs, fp32 softmax and accumulation, head_dim 128.
//
// One workgroup = 8 wavefronts = the G query heads of one KV head x (8 / G)
// groups of 32 query tokens of one sequence, in one layer; all eight share
// every K / V tile of 64 keys staged in LDS.  Keys are looked up through the
// block table (its slice for this workgroup is staged in LDS once).
//
// Both products keep the query token in the MFMA column so that every
// per-token quantity is lane-local:
//   S^T [64 keys x 32 tok] = K [keys x dh] . Q^T      (A: K rows from LDS,
//                                                     B: Q rows, registers)
//   O^T [dh x 32 tok]     += V^T [dh x keys] . P^T     (A: V^T from LDS,
//                                                     B: P from registers)
// In the C layout of v_mfma_f32_32x32x16_bf16 a lane holds keys
// {8q + 4h + r : q < 4, r < 4} of its token (h = lane / 32).  Taking the PV
// contraction over keys in the order (4h + r, 8 + 4h + r) for each group of
// 16 keys makes those registers exactly the B operand, so P never leaves the
// lane.  Softmax: running max / running sum per token in base 2 (scores
// scaled by log2(e) / sqrt(dh)); the max is only moved when it grows by more
// than 8 (a factor 2^8), so the accumulator rescale is rare.
//
// Staging: K and V tiles stream straight from the pool into LDS
// (global_load_lds_dwordx4) through 4 stages as unpadded 256-byte key rows
// whose 16-byte chunks are permuted per row (kswz, vswz) so that the reads
// below hit every bank group evenly.  The four K stages come first in LDS,
// then the four V stages (16 KiB each), so that every operand read is one
// loop-invariant per-lane address register plus an immediate offset (stage,
// key group) below 64 KiB when the stage is known at compile time.  V stays
// key major; its operand (4 consecutive keys of one channel per half) is read
// with ds_read_b64_tr_b16: within each group of 16 lanes, lane i addressing
// row key0 + i / 4, channels c0 + 4 (i % 4) .. + 3 receives keys
// key0 .. key0 + 3 of channel c0 + i.
//
// Software pipeline: iteration t issues the QK^T products of tile t + 1
// before the softmax of tile t, so that the matrix cores can work on the next
// scores while the vector ALUs exponentiate the current ones; then the PV
// products of tile t, in two halves.  The loop is peeled so that its body has
// no branch between those products and the softmax (the only branch left is
// the rare accumulator rescale, placed after the exponentials): the last tile
// is handled after the loop, and the tiles that no query of the wave masks
// run in a loop of their own without mask code (the mask is applied only on
// the causal diagonal and on ragged ends), unrolled by the four stages so
// that each step's stage is a constant.  The one workgroup barrier per
// tile sits between the two PV halves, so a wave meets it with products
// still to issue; it makes tile t + 2 visible and frees the buffer of tile
// t - 1 for the copies of tile t + 3.  The block ids of a tile's copies are
// read from LDS one issue ahead.
//
// Workgroup order: consecutive workgroups are dispatched round-robin to the
// 8 XCDs, each with its own L2.  The linear workgroup id is permuted so that
// each XCD receives a contiguous range of (layer, KV head, query tile)
// triples: the query tiles of one (layer, KV head) read its K / V through
// one L2.
#include "kv_dma.h"
#include "kv_fast.h"
#include <type_traits>

namespace kvs {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef short v4s __attribute__((ext_vector_type(4)));
#define KV_LDS4(p) ((__attribute__((address_space(3))) v4s*)(p))

constexpr int kDh = 128;
constexpr int kKT = 64;             // keys per tile
constexpr int kPW = 8;              // query heads x token groups per workgroup
// Query heads per wavefront (wavefronts per workgroup: kPW / kHeadsPerWave).
// Two heads per wave share every K / V operand read from LDS between two
// products, but need ~470 registers: one wave per SIMD, and the loss of the
// second wave's overlap made it 8-20% slower (measured), so one it is.
constexpr int kHeadsPerWave = 1;
constexpr int kPS = 4;              // pipeline stages
constexpr int kPTile = kKT * kDh;   // elements of one K (or V) tile
constexpr int kXcd = 8;             // XCDs per device
constexpr size_t kLdsMax = 160 * 1024;
constexpr size_t kStaticLds = (size_t)kPS * 2 * kPTile * 2;

// Reductions over lanes l and l ^ 32 (the two halves of a token's keys) with
// v_permlane32_swap, which leaves v[l % 32] and v[l % 32 + 32] in every lane.
// max_xor32_scaled returns max(v, v of lane l ^ 32) * c for c > 0; scaling
// both swapped values before the max makes them results of arithmetic, which
// the compiler knows are not signalling NaNs, so it adds no quieting
// instructions around the max.
__device__ inline float max_xor32_scaled(float v, float c) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]) * c, __uint_as_float(r[1]) * c);
}
__device__ inline float sum_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// LDS slot permutations of a key row's 16 chunks of 16 bytes.  K rows are
// read 16 consecutive rows at one chunk: chunk c of row r sits at slot
// c ^ (r & 15).  V rows are read transposed, 8 consecutive rows x 4 adjacent
// chunks per instruction: chunk c of row r sits at slot c ^ vswz(r), with
// vswz the 2-bit rotation of r & 15, which sends those 32 (row, chunk) pairs
// to every slot exactly twice.
__device__ inline int kswz(int r) { return r & 15; }
__device__ inline int vswz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }

__device__ inline uint32_t cvt2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((floatx2){a, b}, bf16x2));
}

// Bijection of [0, n) that gives XCD x (= id % kXcd) a contiguous logical
// range.
__device__ inline int xcd_remap(int id, int n) {
  const int per = (n + kXcd - 1) / kXcd;
  const int tall = n % kXcd == 0 ? kXcd : n % kXcd;
  const int x = id % kXcd, i = id / kXcd;
  return x < tall ? x * per + i : tall * per + (x - tall) * (per - 1) + i;
}

// grid (batch x query tiles x Hkv x lc, flattened), block 64 * (8 / HP):
// each wavefront computes HP query heads of one group of 32 tokens.
template <int G, int HP>
__global__ void __launch_bounds__(64 * (kPW / HP), 1)
k_attn_pipe(PoolGeom g, const uint16_t* __restrict__ qbuf, AppendDesc a,
            uint16_t* __restrict__ o, int l0, float qk_scale_log2) {
  constexpr int NW = kPW / HP;      // wavefronts per workgroup
  constexpr int TG = kPW / G;       // token groups of 32
  constexpr int QT = 32 * TG;       // query tokens per workgroup
  constexpr int CJ = 16 / NW;       // 1 KiB copies per operand, tile and wave
  __shared__ __attribute__((aligned(16))) uint16_t smem[kPS * 2 * kPTile];
  extern __shared__ int s_tbl[];    // block ids of the keys this workgroup reads
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hl = lane >> 5, col = lane & 31;
  const int tg = wave / (G / HP), hw = wave % (G / HP);
  const int qt_per_seq = (a.T + QT - 1) / QT;
  const int nx = a.batch * qt_per_seq;
  const int lid = xcd_remap(blockIdx.x, gridDim.x);
  const int bx = lid % nx, gk = (lid / nx) % g.Hkv, lc = lid / (nx * g.Hkv);
  const int seq = bx / qt_per_seq;
  const int qt = qt_per_seq - 1 - (bx % qt_per_seq);  // long tiles first
  const int l = l0 + lc;
  const int M = a.batch * a.T;
  const SeqDesc sd = a.seq[seq];
  const int n_keys = sd.n_before + a.T;
  const int t0 = qt * QT;
  const int tq = t0 + tg * 32 + col;
  const int uq = sd.n_before + tq;
  const bool q_valid = tq < a.T;
  const int key_end = min(n_keys, sd.n_before + t0 + QT);
  const int n_tiles = (key_end + kKT - 1) / kKT;
  const int h0 = gk * G + hw * HP;  // this wave's first query head
  const uint16_t* pool = (const uint16_t*)g.pool;

  // stage the block ids of keys [0, key_end) in LDS
  const int nbl = (key_end + g.B - 1) / g.B;
  const int32_t* trow = g.tables + (int64_t)sd.slot * g.max_blocks;
  for (int i = tid; i < nbl; i += 64 * NW) s_tbl[i] = trow[i];

  // Q^T operands of the wave's heads (registers for the whole loop)
  bf16x8 qf[HP][8];
  {
    const int row = seq * a.T + min(tq, a.T - 1);
#pragma unroll
    for (int hh = 0; hh < HP; ++hh) {
      const uint16_t* qp = qbuf + (((int64_t)lc * M + row) * g.Hq + h0 + hh) * kDh;
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) qf[hh][ks] = *(const bf16x8*)(qp + ks * 16 + hl * 8);
    }
#pragma unroll
    for (int hh = 0; hh < HP; ++hh)
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) settle(qf[hh][ks]);
  }
  __syncthreads();  // s_tbl ready

  // Tile loads: 16 copies of 1 KiB (4 key rows of one block, as B >= 16) per
  // operand; wave w issues copies w, w + NW, ... of K and of V.  Full tiles
  // use a scalar block base; the last tile clamps rows past key_end to
  // key_end - 1 per lane (slots past the end of a state may hold anything).
  const int64_t koff = tile_off(g, l, 0, gk, 0), voff = tile_off(g, l, 1, gk, 0);
  const int64_t kv_gap = (voff - koff) * 2;
  const uint32_t lds0 = lds_addr(smem);
  // Full-tile copies: scalar base = K tile of this (layer, head) in the key's
  // block (one 32 x 32-bit product per copy) + the copy's first row in the
  // block; per-lane offset = row within the copy + swizzled chunk, plus the
  // K -> V distance for V.  B divides the 64 keys of a tile, so copy j's rows
  // sit at the same place in their block in every tile, and the swizzle of
  // row r = 4 j + lane / 16 depends on r mod 16 only, the same for every
  // copy of a wave (j = wave + NW jj with 4 NW a multiple of 16): the offsets
  // are loop invariants, one register each for K and V.
  static_assert((4 * NW) % 16 == 0, "one swizzle per wave");
  const char* pool_k = (const char*)pool + koff * 2;
  const uint32_t blk_bytes = (uint32_t)(g.block_elems * 2);
  const int r0 = wave * 4 + (lane >> 4);
  const uint32_t cko = (uint32_t)((lane >> 4) * (kDh * 2) + (((lane & 15) ^ kswz(r0)) * 16));
  const uint32_t cvo = (uint32_t)((lane >> 4) * (kDh * 2) + (((lane & 15) ^ vswz(r0)) * 16)) +
                       (uint32_t)kv_gap;
  // block ids of the next full tile's copies, read one issue ahead
  int nid[CJ];
  auto fetch_ids = [&](int tile) {
#pragma unroll
    for (int jj = 0; jj < CJ; ++jj)
      nid[jj] = s_tbl[min((tile * kKT + (wave + jj * NW) * 4) >> g.b_shift, nbl - 1)];
  };
  fetch_ids(0);
  auto issue = [&](int tile, int buf) {
    if ((tile + 1) * kKT <= key_end) {
      const uint32_t kl = lds0 + buf * kPTile * 2, vl = kl + kPS * kPTile * 2;
#pragma unroll
      for (int jj = 0; jj < CJ; ++jj) {
        const int j = wave + jj * NW;
        const uint32_t id = (uint32_t)__builtin_amdgcn_readfirstlane(nid[jj]);
        const char* kb = pool_k + (uint64_t)id * blk_bytes + ((j * 4) & (g.B - 1)) * (kDh * 2);
        lds_dma16_sv(kb, cko, kl + j * 1024);
        lds_dma16_sv(kb, cvo, vl + j * 1024);
      }
    } else {
      uint16_t* Ks = smem + buf * kPTile;
      uint16_t* Vs = Ks + kPS * kPTile;
#pragma unroll
      for (int jj = 0; jj < CJ; ++jj) {
        const int j = wave + jj * NW;
        const int r = j * 4 + (lane >> 4);
        const int key = min(tile * kKT + r, key_end - 1);
        const int64_t base = (int64_t)s_tbl[key >> g.b_shift] * g.block_elems +
                             (key & (g.B - 1)) * kDh;
        lds_dma16(pool + base + koff + ((lane & 15) ^ kswz(r)) * 8, Ks + j * 512);
        lds_dma16(pool + base + voff + ((lane & 15) ^ vswz(r)) * 8, Vs + j * 512);
      }
    }
    fetch_ids(tile + 1);
  };
  // Per-lane LDS byte addresses of the operand reads in stage 0: K for each
  // k-substep ks of the first 32 keys (the second 32 keys are 8 KiB further,
  // and kswz(32 + r) = kswz(r)); V for each 32-channel block mt and key half
  // of the first 16 keys (key group s4 is 4 KiB further, and vswz is the same
  // for keys r and r + 16 s4).  settle() keeps the compiler from splitting
  // them into more registers.
  uint32_t kof[8], vof[8];
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) {
    kof[ks] = lds0 + (uint32_t)(col * kDh + (((ks * 2 + hl) ^ kswz(col)) * 8)) * 2;
    settle(kof[ks]);
  }
  {
    const int gi = lane >> 4, li = lane & 15;
    const int key_a = (gi >> 1) * 4 + (li >> 2);
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const int dc = mt * 32 + (gi & 1) * 16 + (li & 3) * 4;
      const int ch = dc >> 3, hf = (dc & 7);
#pragma unroll
      for (int ab = 0; ab < 2; ++ab) {
        const int key = key_a + ab * 8;
        vof[mt * 2 + ab] = lds0 + kPS * kPTile * 2 +
                           (uint32_t)(key * kDh + ((ch ^ vswz(key)) * 8) + hf) * 2;
        settle(vof[mt * 2 + ab]);
      }
    }
  }
  // S^T of one tile for this wave's heads and 32 tokens; each K operand read
  // from LDS feeds the products of all HP heads
  auto qk = [&](int buf, floatx16 (*sacc)[2]) {
    const uint32_t kb = buf * kPTile * 2;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        const bf16x8 kf =
            *(const __attribute__((address_space(3))) bf16x8*)(kof[ks] + kb + kt * 32 * kDh * 2);
        // the first product of a chain takes a literal zero accumulator
#pragma unroll
        for (int hh = 0; hh < HP; ++hh)
          sacc[hh][kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              kf, qf[hh][ks], ks == 0 ? floatx16{} : sacc[hh][kt], 0, 0, 0);
      }
    }
  };

  floatx16 oacc[HP][4];
#pragma unroll
  for (int hh = 0; hh < HP; ++hh)
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int e = 0; e < 16; ++e) oacc[hh][mt][e] = 0.f;
  float m_run[HP], l_run[HP];
#pragma unroll
  for (int hh = 0; hh < HP; ++hh) {
    m_run[hh] = -INFINITY;
    l_run[hh] = 0.f;
  }
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

  // the step below computes QK^T of tile t + 1 before its own barrier, so
  // tile t + 1 must have been made visible one step earlier: four stages
  static_assert(kPS == 4, "stages");
  auto wait_tiles = [](int k) {  // at most k tiles of this wave's copies pending
    if (k >= 2)
      wait_vmcnt<4 * CJ>();
    else if (k == 1)
      wait_vmcnt<2 * CJ>();
    else
      wait_vmcnt<0>();
  };

  // softmax of one tile's scores per head: mask (MASKED only), running max,
  // exp2, bf16 probabilities pf and their row sum; moved[hh] = the max moved.
  // m_thr = m_run + 8, updated with m_run.
  float ps[HP], m_new[HP], m_use[HP], m_thr[HP];
#pragma unroll
  for (int hh = 0; hh < HP; ++hh) m_thr[hh] = -INFINITY;
  bool moved[HP];
  bf16x8 pf[HP][4];
  auto softmax = [&](floatx16 (*sc)[2], int tile, auto masked_c) {
    constexpr bool MASKED = decltype(masked_c)::value;
    const int k0 = tile * kKT;
#pragma unroll
    for (int hh = 0; hh < HP; ++hh) {
      if constexpr (MASKED) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int kk = k0 + kt * 32 + (e >> 2) * 8 + hl * 4 + (e & 3);
            if (kk > uq || kk >= n_keys) sc[hh][kt][e] = -INFINITY;
          }
      }
      float mt_max = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e) mt_max = fmaxf(mt_max, sc[hh][kt][e]);
      mt_max = max_xor32_scaled(mt_max, qk_scale_log2);
      m_new[hh] = mt_max > m_thr[hh] ? mt_max : m_run[hh];
      m_use[hh] = m_new[hh] == -INFINITY ? 0.f : m_new[hh];
      moved[hh] = __ballot(m_new[hh] != m_run[hh]) != 0;
      float ps0 = 0.f, ps1 = 0.f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int hs = 0; hs < 2; ++hs) {
          float p[8];
#pragma unroll
          for (int j = 0; j < 8; ++j)
            p[j] = __builtin_amdgcn_exp2f(fmaf(sc[hh][kt][hs * 8 + j], qk_scale_log2, -m_use[hh]));
          const uint32_t wv[4] = {cvt2(p[0], p[1]), cvt2(p[2], p[3]), cvt2(p[4], p[5]),
                                  cvt2(p[6], p[7])};
          ps0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, wv[0]), ones, ps0, false);
          ps1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, wv[1]), ones, ps1, false);
          ps0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, wv[2]), ones, ps0, false);
          ps1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, wv[3]), ones, ps1, false);
          pf[hh][kt * 2 + hs] = __builtin_bit_cast(bf16x8, *(const uint4*)wv);
        }
      ps[hh] = ps0 + ps1;
    }
    // pin the probabilities before the caller's rescale branches, so that the
    // exponentials stay in the straight-line region with the QK^T products
#pragma unroll
    for (int hh = 0; hh < HP; ++hh) {
#pragma unroll
      for (int i = 0; i < 4; ++i) settle(pf[hh][i]);
      settle(ps[hh]);
    }
  };
  auto finish = [&]() {
#pragma unroll
    for (int hh = 0; hh < HP; ++hh) {
      if (moved[hh]) {
        const float alpha = __builtin_amdgcn_exp2f(m_run[hh] - m_use[hh]);
        l_run[hh] *= alpha;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
          for (int e = 0; e < 16; ++e) oacc[hh][mt][e] *= alpha;
        m_thr[hh] = m_new[hh] + 8.f;
      }
      l_run[hh] += ps[hh];
      m_run[hh] = m_new[hh];
    }
  };
  // O^T += V^T P^T for keys [16 s_lo, 16 s_hi) of the tile in stage sb, V^T
  // operands by transposed LDS reads, each feeding the products of all HP heads
  auto pv = [&](int sb, int s_lo, int s_hi) {
    const uint32_t vb = sb * kPTile * 2;
#pragma unroll
    for (int s4 = s_lo; s4 < s_hi; ++s4) {
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const uint32_t so = vb + s4 * 16 * kDh * 2;
        const v4s r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            KV_LDS4(vof[mt * 2] + so));
        const v4s r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            KV_LDS4(vof[mt * 2 + 1] + so));
        const v4s vv[2] = {r0, r1};
        const bf16x8 vf = __builtin_bit_cast(bf16x8, vv);
#pragma unroll
        for (int hh = 0; hh < HP; ++hh)
          oacc[hh][mt] =
              __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[hh][s4], oacc[hh][mt], 0, 0, 0);
      }
    }
  };

  // Tiles 0 .. kPS - 2 in flight; tiles 0 and 1 visible before the loop.
  for (int st = 0; st < kPS - 1 && st < n_tiles; ++st) issue(st, st);
  wait_tiles(min(kPS - 1, n_tiles) - min(2, n_tiles));
  lds_barrier();
  floatx16 sacc[HP][2];
  qk(0, sacc);

  // One step: QK^T of tile + 1 (into snx) with the softmax of tile (scores
  // in scur), then the PV product of tile in two halves with the barrier
  // between them: it makes tile + 2 visible for the next step and frees the
  // buffer of tile - 1.  Steps run in pairs that swap the two score sets, so
  // no scores are copied between registers.  sb = the stage of tile.
  floatx16 sB[HP][2];
  auto step = [&](int tile, int sb, floatx16 (*scur)[2], floatx16 (*snx)[2], auto masked_c) {
    qk((sb + 1) % kPS, snx);
    softmax(scur, tile, masked_c);
    finish();
    pv(sb, 0, 2);
    if (tile + 2 < n_tiles) {
      // copies of one wave complete in order, 2 CJ per tile: tile + 2 is the
      // newest issued.  Every read of the buffer about to be refilled (tile
      // - 1) fed a product issued earlier, so no LDS wait is needed here.
      wait_vmcnt<0>();
      barrier_only();
      if (tile + kPS - 1 < n_tiles) issue(tile + kPS - 1, (sb + kPS - 1) % kPS);
    }
    pv(sb, 2, 4);
  };
  // a step left over after the pairs: its next scores become sacc
  auto step_copy = [&](int tile, auto masked_c) {
    step(tile, tile % kPS, sacc, sB, masked_c);
#pragma unroll
    for (int hh = 0; hh < HP; ++hh) {
      sacc[hh][0] = sB[hh][0];
      sacc[hh][1] = sB[hh][1];
    }
  };
  const int first_q = sd.n_before + t0 + tg * 32;
  const int n_free = (t0 + tg * 32 + 31 < a.T) ? min((first_q + 1) / kKT, n_keys / kKT) : 0;
  const int lim = n_tiles - 1;
  const int nf = min(n_free, lim);
  int tile = 0;
  for (; tile + 3 < nf; tile += 4) {
    step(tile, 0, sacc, sB, std::false_type{});
    step(tile + 1, 1, sB, sacc, std::false_type{});
    step(tile + 2, 2, sacc, sB, std::false_type{});
    step(tile + 3, 3, sB, sacc, std::false_type{});
  }
  for (; tile + 1 < nf; tile += 2) {
    step(tile, tile % kPS, sacc, sB, std::false_type{});
    step(tile + 1, (tile + 1) % kPS, sB, sacc, std::false_type{});
  }
  if (tile < nf) step_copy(tile++, std::false_type{});
  for (; tile + 1 < lim; tile += 2) {
    step(tile, tile % kPS, sacc, sB, std::true_type{});
    step(tile + 1, (tile + 1) % kPS, sB, sacc, std::true_type{});
  }
  if (tile < lim) step_copy(tile++, std::true_type{});
  softmax(sacc, tile, std::true_type{});
  finish();
  pv(tile % kPS, 0, 4);

  float l_tot[HP];
#pragma unroll
  for (int hh = 0; hh < HP; ++hh) l_tot[hh] = sum_xor32(l_run[hh]);
  if (!q_valid) return;
  const int row = seq * a.T + tq;
#pragma unroll
  for (int hh = 0; hh < HP; ++hh) {
    const float inv = 1.f / l_tot[hh];
    uint16_t* op = o + (((int64_t)l * M + row) * g.Hq + h0 + hh) * kDh;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c0 = mt * 32 + q * 8 + hl * 4;
        *(uint2*)(op + c0) =
            make_uint2(cvt2(oacc[hh][mt][q * 4] * inv, oacc[hh][mt][q * 4 + 1] * inv),
                       cvt2(oacc[hh][mt][q * 4 + 2] * inv, oacc[hh][mt][q * 4 + 3] * inv));
      }
  }
}

size_t table_bytes(const PoolGeom& g, int max_keys) {
  return (size_t)((max_keys + g.B - 1) / g.B) * sizeof(int);
}

}  // namespace

bool attn_mfma_ok(const PoolGeom& g, int dtype, const AppendDesc& a) {
  const int G = g.Hq / g.Hkv;
  // 16 <= B <= 64 a power of two (B divides a 64-key tile); block bytes and
  // the K -> V distance fit the 32-bit copy arithmetic
  return dtype == KV_DTYPE_BF16 && g.dh == kDh && (G == 4 || G == 8) && g.b_shift >= 0 &&
         g.B >= 16 && g.B <= kKT && g.block_elems * 2 < (int64_t)1 << 32 &&
         kStaticLds + table_bytes(g, a.max_keys) <= kLdsMax;
}

hipError_t launch_attn_prefill(const PoolGeom& g, const void* qbuf, const AppendDesc& a, void* o,
                               int l0, int lc, hipStream_t s) {
  const int G = g.Hq / g.Hkv;
  const int QT = 32 * (kPW / G);
  const int qt = (a.T + QT - 1) / QT;
  const int64_t n = (int64_t)a.batch * qt * g.Hkv * lc;
  if (n > 0x7fffffff) return hipErrorInvalidValue;
  const float sc = 1.4426950408889634f / sqrtf((float)kDh);
  const size_t dyn = table_bytes(g, a.max_keys);
  constexpr int HP = kHeadsPerWave;
  if (G == 4)
    k_attn_pipe<4, HP><<<(unsigned)n, 64 * (kPW / HP), dyn, s>>>(g, (const uint16_t*)qbuf, a,
                                                                 (uint16_t*)o, l0, sc);
  else
    k_attn_pipe<8, HP><<<(unsigned)n, 64 * (kPW / HP), dyn, s>>>(g, (const uint16_t*)qbuf, a,
                                                                 (uint16_t*)o, l0, sc);
  return hipGetLastError();
}

}  // namespace kvs
