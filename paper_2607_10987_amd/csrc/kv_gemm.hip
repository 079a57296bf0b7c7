// QKV projection on MFMA (bf16 in, fp32 accumulate) with the RoPE rotation
// and the paged K/V store fused into the epilogue.
//
// The kernel computes C^T = W_l X^T: the A operand is a 32-row slab of the
// weight rows (output channels), the B operand a 32-row slab of the token
// rows, both K-contiguous, so tiles are staged through LDS with 16-byte
// accesses and read back with one ds_read_b128 per MFMA operand.  In the
// C^T layout of v_mfma_f32_32x32x16_bf16 a lane holds, for one token, four
// consecutive output channels per group, so RoPE partners (channel i and
// i + 64 of the same head) sit in the same lane when one wavefront owns a
// whole 128-channel head, and stores are 8-byte runs of one token row.
//
// Kernels, by token count M of the call:
//   M > 32   k_qkv_dl: 256 channels (2 heads) x 256 tokens per workgroup,
//            eight waves of 128 x 64, direct global->LDS copies, RoPE in
//            registers (factors read from a copy of the table grouped by 4
//            frequencies, position-major within a group, so that one load
//            instruction reads consecutive positions), bf16 tile restaged
//            through LDS so that the final Q / K / V stores are 16-byte,
//            row-contiguous writes (the fast path requires d % 64 == 0);
//   M <= 16  k_qkv_decode_pst when d is a multiple of 256 and a column chunk
//            of the token rows fits in 32 KiB of LDS (chunks halve while
//            they are multiples of 512): each workgroup streams the weights
//            of a group of (layer, head) tiles through per-wave LDS buffers
//            without a break between tiles, token rows staged once per
//            column chunk, one accumulator per tile, RoPE in registers;
//            otherwise k_qkv_decode_lds (token rows staged in LDS, weights
//            loaded straight into registers; d a multiple of 256, e.g. 2560
//            with 13-16 rows), else k_qkv_decode<1> (token rows from global
//            memory; d a multiple of 512 whose rows do not fit, e.g. 10752);
//   M <= 32  k_qkv_decode<2> (d a multiple of 512) or k_qkv_mfma<128, 32>
//            (any other d, and M <= 16 when d is not a multiple of 256):
//            128 channels (1 head) x 32 tokens, fp32 tile in LDS for the
//            rotation.
// Q goes to the scratch buffer [lc][M][Hq * dh]; K and V rows go to
// pool[table[slot][u / B]][l][K|V][kv head][u % B][:] with u = n_before + t.
#include <atomic>

#include "kv_dma.h"
#include "kv_fast.h"

namespace kvs {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kBK = 64;
constexpr int kLd = kBK + 8;  // LDS row stride in elements (144 bytes)
constexpr int kThreads = 256;
constexpr int kDh = 128;

__device__ inline uint32_t pack_bf16x2(float a, float b) {
  const __bf16 x = (__bf16)a, y = (__bf16)b;  // round to nearest even
  return (uint32_t)__builtin_bit_cast(uint16_t, x) | ((uint32_t)__builtin_bit_cast(uint16_t, y) << 16);
}

// Row m of the token matrix -> destination description.
struct RowInfo {
  int seq, t, u, pos, slot;
};

__device__ inline RowInfo row_info(const AppendDesc& a, int row) {
  RowInfo r;
  r.seq = row / a.T;
  r.t = row - r.seq * a.T;
  const SeqDesc sd = a.seq[r.seq];
  r.u = sd.n_before + r.t;
  r.pos = sd.pos0 + r.u;
  r.slot = sd.slot;
  return r;
}

// Destination of 8 consecutive channels [c, c + 8) of layer-local head `hh`
// (0 .. Hq + 2 Hkv - 1) for token row `row`.
__device__ inline uint16_t* dest(const PoolGeom& g, const AppendDesc& a, uint16_t* qbuf, int lc,
                                 int l, int M, int row, int hh, int c) {
  if (hh < g.Hq) return qbuf + (((int64_t)lc * M + row) * g.Hq + hh) * kDh + c;
  const RowInfo r = row_info(a, row);
  const int kv = hh < g.Hq + g.Hkv ? 0 : 1;
  const int gh = hh - g.Hq - kv * g.Hkv;
  const int32_t blk = g.tables[(int64_t)r.slot * g.max_blocks + r.u / g.B];
  return (uint16_t*)g.pool + (int64_t)blk * g.block_elems + tile_off(g, l, kv, gh, r.u % g.B) + c;
}

template <int CH, int BT, int WCH, int WTK>
struct Tiling {
  static constexpr int TI = CH / WCH / 32;  // channel tiles per wave
  static constexpr int TJ = BT / WTK / 32;  // token tiles per wave
  static constexpr int WAVE_CH = CH / WCH;
  static constexpr int STAGE = (CH + BT) * kLd;            // elements per LDS stage
  static constexpr int A_LD = CH * kBK / 8 / kThreads;     // 16-byte loads per thread
  static constexpr int B_LD = (BT * kBK / 8 + kThreads - 1) / kThreads;
  static constexpr bool WAVE_HEAD = WAVE_CH == kDh;         // wave owns a whole head
  static constexpr int EPI_BYTES = WAVE_HEAD ? BT * (CH + 8) * 2 : BT * (CH + 4) * 4;
  static constexpr int MAIN_BYTES = 2 * STAGE * 2;
  static constexpr int SMEM = MAIN_BYTES > EPI_BYTES ? MAIN_BYTES : EPI_BYTES;
};

template <int CH, int BT, int WCH, int WTK>
__global__ void __launch_bounds__(kThreads)
k_qkv_mfma(PoolGeom g, const uint16_t* __restrict__ x, const uint16_t* __restrict__ w,
           int64_t w_stride, AppendDesc a, uint16_t* __restrict__ qbuf, int l0) {
  using TL = Tiling<CH, BT, WCH, WTK>;
  constexpr int TI = TL::TI, TJ = TL::TJ;
  __shared__ __attribute__((aligned(16))) char smem_raw[TL::SMEM];
  uint16_t* smem = (uint16_t*)smem_raw;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n0 = blockIdx.x * CH;  // first output channel of the layer
  const int m0 = blockIdx.y * BT;  // first token row
  const int lc = blockIdx.z, l = l0 + lc;
  const int M = a.batch * a.T, d = g.d;
  const uint16_t* wl = w + (int64_t)l * w_stride;
  const int ch0 = (wave % WCH) * TL::WAVE_CH;
  const int tk0 = (wave / WCH) * (BT / WTK);

  uint4 ra[TL::A_LD], rb[TL::B_LD];
  auto gload = [&](int kb) {
#pragma unroll
    for (int i = 0; i < TL::A_LD; ++i) {
      const int q = tid + kThreads * i, r = q >> 3, c = q & 7;
      ra[i] = *(const uint4*)(wl + (int64_t)(n0 + r) * d + kb * kBK + c * 8);
    }
#pragma unroll
    for (int i = 0; i < TL::B_LD; ++i) {
      const int q = tid + kThreads * i, r = q >> 3, c = q & 7;
      const int row = m0 + r;
      rb[i] = (r < BT && row < M) ? *(const uint4*)(x + (int64_t)row * d + kb * kBK + c * 8)
                                  : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int buf) {
    uint16_t* As = smem + buf * TL::STAGE;
    uint16_t* Bs = As + CH * kLd;
#pragma unroll
    for (int i = 0; i < TL::A_LD; ++i) {
      const int q = tid + kThreads * i, r = q >> 3, c = q & 7;
      *(uint4*)(As + r * kLd + c * 8) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < TL::B_LD; ++i) {
      const int q = tid + kThreads * i, r = q >> 3, c = q & 7;
      if (r < BT) *(uint4*)(Bs + r * kLd + c * 8) = rb[i];
    }
  };

  floatx16 acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int nk = d / kBK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kb = 0; kb < nk; ++kb) {
    const int cur = kb & 1;
    if (kb + 1 < nk) gload(kb + 1);
    const uint16_t* As = smem + cur * TL::STAGE;
    const uint16_t* Bs = As + CH * kLd;
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      bf16x8 fa[TI], fb[TJ];
      const int kof = ks * 16 + (lane >> 5) * 8;
#pragma unroll
      for (int i = 0; i < TI; ++i)
        fa[i] = *(const bf16x8*)(As + (ch0 + i * 32 + (lane & 31)) * kLd + kof);
#pragma unroll
      for (int j = 0; j < TJ; ++j)
        fb[j] = *(const bf16x8*)(Bs + (tk0 + j * 32 + (lane & 31)) * kLd + kof);
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
    if (kb + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

  const int half = kDh / 2;
  if constexpr (TL::WAVE_HEAD) {
    // ---- prefill epilogue: rotate in registers, restage bf16 rows in LDS
    constexpr int SLD = CH + 8;
    uint16_t* S = smem;
    const int hh = (n0 + ch0) / kDh;
    const bool rot = hh < g.Hq + g.Hkv;
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int tl = tk0 + j * 32 + (lane & 31);
      const int row = m0 + tl;
      const int pos = row < M ? row_info(a, row).pos : 0;
      const float* cr = g.rope_cos + (int64_t)pos * half;
      const float* sr = g.rope_sin + (int64_t)pos * half;
#pragma unroll
      for (int i = 0; i < TI / 2; ++i) {
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) {
          const int f0 = i * 32 + e4 * 8 + (lane >> 5) * 4;
          float4 cs = make_float4(1.f, 1.f, 1.f, 1.f), sn = make_float4(0.f, 0.f, 0.f, 0.f);
          if (rot) {
            cs = *(const float4*)(cr + f0);
            sn = *(const float4*)(sr + f0);
          }
          float xr[4], yr[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float xv = acc[i][j][e4 * 4 + q], yv = acc[i + 2][j][e4 * 4 + q];
            const float c = (&cs.x)[q], s = (&sn.x)[q];
            xr[q] = xv * c - yv * s;
            yr[q] = xv * s + yv * c;
          }
          uint2 px = make_uint2(pack_bf16x2(xr[0], xr[1]), pack_bf16x2(xr[2], xr[3]));
          uint2 py = make_uint2(pack_bf16x2(yr[0], yr[1]), pack_bf16x2(yr[2], yr[3]));
          *(uint2*)(S + tl * SLD + ch0 + f0) = px;
          *(uint2*)(S + tl * SLD + ch0 + half + f0) = py;
        }
      }
    }
    __syncthreads();
    constexpr int G8 = CH / 8;  // 16-byte groups per token row
    for (int q = tid; q < BT * G8; q += kThreads) {
      const int r = q / G8, c8 = q % G8;
      const int row = m0 + r;
      if (row >= M) continue;
      const uint4 v = *(const uint4*)(S + r * SLD + c8 * 8);
      const int ch = n0 + c8 * 8;
      *(uint4*)dest(g, a, qbuf, lc, l, M, row, ch / kDh, ch % kDh) = v;
    }
  } else {
    // ---- decode epilogue: fp32 tile in LDS, pairs straddle waves
    constexpr int FLD = CH + 4;
    float* Cf = (float*)smem_raw;
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j)
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) {
          const int ch = ch0 + i * 32 + e4 * 8 + (lane >> 5) * 4;
          const int tl = tk0 + j * 32 + (lane & 31);
          *(float4*)(Cf + tl * FLD + ch) =
              make_float4(acc[i][j][e4 * 4], acc[i][j][e4 * 4 + 1], acc[i][j][e4 * 4 + 2],
                          acc[i][j][e4 * 4 + 3]);
        }
    __syncthreads();
    constexpr int NH = CH / kDh;
    for (int it = tid; it < BT * NH * (half / 4); it += kThreads) {
      const int f4 = it % (half / 4);
      const int hl = (it / (half / 4)) % NH;
      const int r = it / ((half / 4) * NH);
      const int row = m0 + r;
      if (row >= M) continue;
      const int hh = (n0 / kDh) + hl;
      const float4 xv = *(const float4*)(Cf + r * FLD + hl * kDh + f4 * 4);
      const float4 yv = *(const float4*)(Cf + r * FLD + hl * kDh + half + f4 * 4);
      float4 xo = xv, yo = yv;
      if (hh < g.Hq + g.Hkv) {
        const int pos = row_info(a, row).pos;
        const float4 cs = *(const float4*)(g.rope_cos + (int64_t)pos * half + f4 * 4);
        const float4 sn = *(const float4*)(g.rope_sin + (int64_t)pos * half + f4 * 4);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float c = (&cs.x)[q], s = (&sn.x)[q];
          (&xo.x)[q] = (&xv.x)[q] * c - (&yv.x)[q] * s;
          (&yo.x)[q] = (&xv.x)[q] * s + (&yv.x)[q] * c;
        }
      }
      uint16_t* dp = dest(g, a, qbuf, lc, l, M, row, hh, f4 * 4);
      *(uint2*)dp = make_uint2(pack_bf16x2(xo.x, xo.y), pack_bf16x2(xo.z, xo.w));
      *(uint2*)(dp + half) = make_uint2(pack_bf16x2(yo.x, yo.y), pack_bf16x2(yo.z, yo.w));
    }
  }
}

// Prefill projection, main loop with direct global->LDS loads
// (global_load_lds_dwordx4: lane i of a wavefront writes LDS bytes
// [16 i, 16 i + 16) of the instruction's 1 KiB destination) and a 2-stage
// pipeline of K-steps of 64, with no register staging.  Tile 256 channels x
// 256 tokens, 8 wavefronts of 128 channels x 64 tokens (a wave owns a whole
// head, so RoPE stays in registers).  LDS rows are 128 bytes (64 k); the
// 16-byte chunk q of row r is stored at chunk slot q ^ f(r), f(r) =
// (r >> 1) & 7, so that the 16 consecutive rows an operand read serves in one
// LDS cycle (16 lanes x 16 bytes over 64 banks) cover the 16 bank groups.
//
// Operands are read one k-substep (16) ahead of the products that use them,
// and the one workgroup barrier per K-step sits between the reads and the
// products of the step's last k-substep: a wave reaches it with those
// operands already in registers, so its products keep the matrix core busy
// while the first operands of the next stage are read.  That barrier also
// frees the stage just consumed, which then receives the copies of the
// K-step after next.  Copies take a wave-uniform base (scalar registers) and
// a per-lane 32-bit offset.
__device__ inline int swz(int r) { return (r >> 1) & 7; }

constexpr int kDlBK = 64;
constexpr int kDlWaves = 8;
constexpr int kDlThreads = 64 * kDlWaves;

__global__ void __launch_bounds__(kDlThreads, 1)
k_qkv_dl(PoolGeom g, const uint16_t* __restrict__ x, const uint16_t* __restrict__ w,
         int64_t w_stride, AppendDesc a, uint16_t* __restrict__ qbuf, int l0) {
  constexpr int CH = 256, BT = 256;
  constexpr int OP = CH * kDlBK;
  constexpr int STAGE = 2 * OP;
  constexpr int SLD = CH + 8;
  constexpr int MAIN = 2 * STAGE * 2;
  constexpr int EPI = BT * SLD * 2;
  constexpr int LPW = (OP / 8) / 64 / kDlWaves;  // copies per wave per operand
  constexpr int TI = 4, TJ = 2;
  constexpr int KS = kDlBK / 16;
  __shared__ __attribute__((aligned(16))) char smem_raw[MAIN > EPI ? MAIN : EPI];
  uint16_t* smem = (uint16_t*)smem_raw;

  const int tid = threadIdx.x, lane = tid & 63, hl = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n0 = blockIdx.x * CH;
  const int m0 = blockIdx.y * BT;
  const int lc = blockIdx.z, l = l0 + lc;
  const int M = a.batch * a.T, d = g.d;
  const uint16_t* wl = w + (int64_t)l * w_stride;
  const int ch0 = (wave & 1) * 128;
  const int tk0 = (wave >> 1) * (TJ * 32);

  const uint32_t lds0 = lds_addr(smem);
  uint32_t va[LPW], vb[LPW];
#pragma unroll
  for (int j = 0; j < LPW; ++j) {
    const int c = (wave * LPW + j) * 64 + lane, r = c >> 3, q = (c & 7) ^ swz(r);
    va[j] = ((uint32_t)r * d + q * 8) * 2;
    vb[j] = ((uint32_t)min(r, M - 1 - m0) * d + q * 8) * 2;
  }
  const char* abase = (const char*)(wl + (int64_t)n0 * d);
  const char* bbase = (const char*)(x + (int64_t)m0 * d);
  auto issue = [&](int kb, int buf) {
    const uint32_t la = lds0 + buf * STAGE * 2 + wave * LPW * 1024;
    const char* sa = abase + kb * kDlBK * 2;
    const char* sb = bbase + kb * kDlBK * 2;
#pragma unroll
    for (int j = 0; j < LPW; ++j) {
      lds_dma16_sv(sa, va[j], la + j * 1024);
      lds_dma16_sv(sb, vb[j], la + OP * 2 + j * 1024);
    }
  };

  floatx16 acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  bf16x8 fa[2][TI], fb[2][TJ];
  auto load = [&](int buf, int ks, int sl) {
    const uint16_t* As = smem + buf * STAGE;
    const uint16_t* Bs = As + OP;
    const int q = ks * 2 + hl;
#pragma unroll
    for (int i = 0; i < TI; ++i) {
      const int m = ch0 + i * 32 + (lane & 31);
      fa[sl][i] = *(const bf16x8*)(As + (m * 8 + (q ^ swz(m))) * 8);
    }
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int t = tk0 + j * 32 + (lane & 31);
      fb[sl][j] = *(const bf16x8*)(Bs + (t * 8 + (q ^ swz(t))) * 8);
    }
  };

  const int nk = d / kDlBK;
  issue(0, 0);
  if (nk > 1) {
    issue(1, 1);
    wait_vmcnt<2 * LPW>();
  } else {
    wait_vmcnt<0>();
  }
  lds_barrier();
  load(0, 0, 0);
  for (int kb = 0; kb < nk; ++kb) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (ks + 1 < KS) {
        load(kb & 1, ks + 1, (ks + 1) & 1);
      } else if (kb + 1 < nk) {
        // stage kb + 1 landed (this wave's copies, then every wave's), and
        // every wave holds its last operands of stage kb in registers, so
        // its buffer takes stage kb + 2
        wait_vmcnt<0>();
        lds_barrier();
        load((kb + 1) & 1, 0, 0);
        if (kb + 2 < nk) issue(kb + 2, kb & 1);
      }
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[ks & 1][i], fb[ks & 1][j],
                                                              acc[i][j], 0, 0, 0);
    }
  }
  const int half = kDh / 2;
  const int hh = (n0 + ch0) / kDh;
  const bool rot = hh < g.Hq + g.Hkv;
  const int64_t gstride = (int64_t)g.max_pos * 4;
  // RoPE factors of token sub-tile j from the channel-group-major tables (one
  // load instruction reads 32 consecutive positions of a group: 512
  // contiguous bytes per half-wave); sub-tile 0's are requested before the
  // barrier, so that their latency overlaps the last products
  auto fetch = [&](int j, float4* cf, float4* sf) {
    const int row = m0 + tk0 + j * 32 + (lane & 31);
    const int pos = row < M ? row_info(a, row).pos : 0;
    const float* cr = g.rope_cos_g + (int64_t)pos * 4;
    const float* sr = g.rope_sin_g + (int64_t)pos * 4;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int f0 = (k >> 2) * 32 + (k & 3) * 8 + hl * 4;
      cf[k] = make_float4(1.f, 1.f, 1.f, 1.f);
      sf[k] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (rot) {
        cf[k] = *(const float4*)(cr + (f0 >> 2) * gstride);
        sf[k] = *(const float4*)(sr + (f0 >> 2) * gstride);
      }
    }
  };
  uint16_t* S = smem;
  auto rotate = [&](int j, const float4* cf, const float4* sf) {
    const int tl = tk0 + j * 32 + (lane & 31);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int i = k >> 2, e4 = k & 3;
      const int f0 = i * 32 + e4 * 8 + hl * 4;
      float xr[4], yr[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float xv = acc[i][j][e4 * 4 + q], yv = acc[i + 2][j][e4 * 4 + q];
        const float c = (&cf[k].x)[q], s = (&sf[k].x)[q];
        xr[q] = fmaf(xv, c, -(yv * s));
        yr[q] = fmaf(xv, s, yv * c);
      }
      *(uint2*)(S + tl * SLD + ch0 + f0) =
          make_uint2(pack_bf16x2(xr[0], xr[1]), pack_bf16x2(xr[2], xr[3]));
      *(uint2*)(S + tl * SLD + ch0 + half + f0) =
          make_uint2(pack_bf16x2(yr[0], yr[1]), pack_bf16x2(yr[2], yr[3]));
    }
  };
  static_assert(TJ == 2 && TI == 4, "epilogue tiling");
  float4 c0[8], s0[8], c1[8], s1[8];
  fetch(0, c0, s0);
  __syncthreads();

  rotate(0, c0, s0);
  fetch(1, c1, s1);
  rotate(1, c1, s1);
  __syncthreads();
  // coalesced stores: thread tid writes 16-byte chunk tid % G8 of rows
  // tid / G8 + k (kDlThreads / G8); all destinations (block-table lookups for
  // K / V rows) are resolved before the first store
  constexpr int G8 = CH / 8;
  constexpr int NIT = BT * G8 / kDlThreads;
  constexpr int RSTEP = kDlThreads / G8;
  static_assert(kDlThreads % G8 == 0 && (BT * G8) % kDlThreads == 0, "store tiling");
  const int c8 = tid % G8, r0 = tid / G8;
  const int ch = n0 + c8 * 8;
  uint16_t* dps[NIT];
#pragma unroll
  for (int k = 0; k < NIT; ++k) {
    const int row = m0 + r0 + k * RSTEP;
    dps[k] = row < M ? dest(g, a, qbuf, lc, l, M, row, ch / kDh, ch % kDh) : nullptr;
  }
#pragma unroll
  for (int k = 0; k < NIT; ++k)
    if (dps[k] != nullptr) *(uint4*)dps[k] = *(const uint4*)(S + (r0 + k * RSTEP) * SLD + c8 * 8);
}

typedef __bf16 bf16x8v __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// Decode-size projection (M <= 32 token rows): weight streaming.  Each weight
// element is used by one wavefront only, so operands are loaded straight from
// global memory in the v_mfma_f32_16x16x32_bf16 layout (a lane reads 16 bytes
// of one weight row; the four lanes of a row cover 64 contiguous bytes),
// sixteen k-steps of loads in flight per lane (non-temporal loads measured
// slower here).  Workgroup = one 128-channel
// head of one layer, eight waves of 16 channels (so that the launch, 1536
// workgroups for the 8B shape, fills the GPU in whole rounds); RoPE and the
// stores go through an fp32 tile in LDS.  grid (N / 128, 1, lc), block 512.
constexpr int kDecWaves = 8;

template <int TT>  // token tiles of 16
__global__ void __launch_bounds__(64 * kDecWaves)
k_qkv_decode(PoolGeom g, const uint16_t* __restrict__ x, const uint16_t* __restrict__ w,
             int64_t w_stride, AppendDesc a, uint16_t* __restrict__ qbuf, int l0) {
  constexpr int U = 16;              // k-steps of 32 per batch of loads
  constexpr int FLD = kDh + 4;
  constexpr int NT = 64 * kDecWaves;
  __shared__ __attribute__((aligned(16))) float Cf[TT * 16 * FLD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lk = (lane >> 4) * 8;
  const int n0 = blockIdx.x * kDh;
  const int lc = blockIdx.z, l = l0 + lc;
  const int M = a.batch * a.T, d = g.d;
  const uint16_t* wl = w + (int64_t)l * w_stride;
  const uint16_t* wr = wl + (int64_t)(n0 + wave * 16 + lr) * d + lk;
  const uint16_t* xr[TT];
  bool xok[TT];
#pragma unroll
  for (int j = 0; j < TT; ++j) {
    const int row = j * 16 + lr;
    xok[j] = row < M;
    xr[j] = x + (int64_t)(xok[j] ? row : 0) * d + lk;
  }
  floatx4 acc[TT];
#pragma unroll
  for (int j = 0; j < TT; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < d; k0 += 32 * U) {
    uint4 fa[U], fb[U][TT];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      fa[u] = *(const uint4*)(wr + k0 + 32 * u);
#pragma unroll
      for (int j = 0; j < TT; ++j)
        fb[u][j] = xok[j] ? *(const uint4*)(xr[j] + k0 + 32 * u) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < TT; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8v, fa[u]),
                                                         __builtin_bit_cast(bf16x8v, fb[u][j]),
                                                         acc[j], 0, 0, 0);
  }
  // C[16 ch x 16 tok]: lane holds channels 4 (lane / 16) + e of token lane % 16
#pragma unroll
  for (int j = 0; j < TT; ++j) {
    const int ch = wave * 16 + (lane >> 4) * 4;
    const int tl = j * 16 + lr;
    *(float4*)(Cf + tl * FLD + ch) = make_float4(acc[j][0], acc[j][1], acc[j][2], acc[j][3]);
  }
  __syncthreads();
  const int half = kDh / 2;
  const int hh = n0 / kDh;
  for (int it = tid; it < TT * 16 * (half / 4); it += NT) {
    const int f4 = it % (half / 4), r = it / (half / 4);
    if (r >= M) continue;
    const float4 xv = *(const float4*)(Cf + r * FLD + f4 * 4);
    const float4 yv = *(const float4*)(Cf + r * FLD + half + f4 * 4);
    float4 xo = xv, yo = yv;
    if (hh < g.Hq + g.Hkv) {
      const int pos = row_info(a, r).pos;
      const float4 cs = *(const float4*)(g.rope_cos + (int64_t)pos * half + f4 * 4);
      const float4 sn = *(const float4*)(g.rope_sin + (int64_t)pos * half + f4 * 4);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float c = (&cs.x)[q], s = (&sn.x)[q];
        (&xo.x)[q] = (&xv.x)[q] * c - (&yv.x)[q] * s;
        (&yo.x)[q] = (&xv.x)[q] * s + (&yv.x)[q] * c;
      }
    }
    uint16_t* dp = dest(g, a, qbuf, lc, l, M, r, hh, f4 * 4);
    *(uint2*)dp = make_uint2(pack_bf16x2(xo.x, xo.y), pack_bf16x2(xo.z, xo.w));
    *(uint2*)(dp + half) = make_uint2(pack_bf16x2(yo.x, yo.y), pack_bf16x2(yo.z, yo.w));
  }
}

// Decode-size projection with the token rows staged in LDS (M <= 16 rows):
// the x operand is read from LDS (row stride kc + 8 elements, so the 16 rows
// one operand read touches fall in distinct bank groups) instead of being
// fetched again from L2 by every wavefront, and the next batch of weight
// loads is issued before the products of the current one.  x is staged in
// column chunks of kc (the launcher picks the widest that lets two
// workgroups share a CU).  Same tiling as k_qkv_decode<1>; dynamic LDS:
// M * (kc + 8) bf16.
constexpr int kDecU = 8;  // k-steps of 32 per load batch (two batches in flight)

__global__ void __launch_bounds__(64 * kDecWaves)
k_qkv_decode_lds(PoolGeom g, const uint16_t* __restrict__ x, const uint16_t* __restrict__ w,
                 int64_t w_stride, AppendDesc a, uint16_t* __restrict__ qbuf, int l0, int kc) {
  constexpr int FLD = kDh + 4;
  constexpr int NT = 64 * kDecWaves;
  __shared__ __attribute__((aligned(16))) float Cf[16 * FLD];
  extern __shared__ __attribute__((aligned(16))) uint16_t xs[];  // [M][kc + 8]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lk = (lane >> 4) * 8;
  const int n0 = blockIdx.x * kDh;
  const int lc = blockIdx.z, l = l0 + lc;
  const int M = a.batch * a.T, d = g.d, xld = kc + 8;
  const uint16_t* wl = w + (int64_t)l * w_stride;
  const uint16_t* wr = wl + (int64_t)(n0 + wave * 16 + lr) * d + lk;
  const bool xok = lr < M;
  const uint16_t* xr = xs + (xok ? lr : 0) * xld + lk;

  // weights of the first batch in flight while the first x chunk is staged
  uint4 fa[kDecU], fn[kDecU];
#pragma unroll
  for (int u = 0; u < kDecU; ++u) fa[u] = *(const uint4*)(wr + 32 * u);
  floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
  const int c8 = kc / 8;
  for (int kc0 = 0; kc0 < d; kc0 += kc) {
    // token rows, columns [kc0, kc0 + kc), into LDS
    if (kc0 > 0) __syncthreads();  // the previous chunk has been read
    for (int i = tid; i < M * c8; i += NT) {
      const int r = i / c8, c = i - r * c8;
      *(uint4*)(xs + r * xld + c * 8) = *(const uint4*)(x + (int64_t)r * d + kc0 + c * 8);
    }
    __syncthreads();
    for (int k0 = kc0; k0 < kc0 + kc; k0 += 32 * kDecU) {
      const bool more = k0 + 32 * kDecU < d;
      if (more) {
#pragma unroll
        for (int u = 0; u < kDecU; ++u) fn[u] = *(const uint4*)(wr + k0 + 32 * kDecU + 32 * u);
      }
#pragma unroll
      for (int u = 0; u < kDecU; ++u) {
        const uint4 fb =
            xok ? *(const uint4*)(xr + (k0 - kc0) + 32 * u) : make_uint4(0, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8v, fa[u]),
                                                      __builtin_bit_cast(bf16x8v, fb), acc, 0, 0,
                                                      0);
      }
      if (more) {
#pragma unroll
        for (int u = 0; u < kDecU; ++u) fa[u] = fn[u];
      }
    }
  }
  // C[16 ch x 16 tok]: lane holds channels 4 (lane / 16) + e of token lane % 16
  {
    const int ch = wave * 16 + (lane >> 4) * 4;
    *(float4*)(Cf + lr * FLD + ch) = make_float4(acc[0], acc[1], acc[2], acc[3]);
  }
  __syncthreads();
  const int half = kDh / 2;
  const int hh = n0 / kDh;
  for (int it = tid; it < 16 * (half / 4); it += NT) {
    const int f4 = it % (half / 4), r = it / (half / 4);
    if (r >= M) continue;
    const float4 xv = *(const float4*)(Cf + r * FLD + f4 * 4);
    const float4 yv = *(const float4*)(Cf + r * FLD + half + f4 * 4);
    float4 xo = xv, yo = yv;
    if (hh < g.Hq + g.Hkv) {
      const int pos = row_info(a, r).pos;
      const float4 cs = *(const float4*)(g.rope_cos + (int64_t)pos * half + f4 * 4);
      const float4 sn = *(const float4*)(g.rope_sin + (int64_t)pos * half + f4 * 4);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float c = (&cs.x)[q], s = (&sn.x)[q];
        (&xo.x)[q] = (&xv.x)[q] * c - (&yv.x)[q] * s;
        (&yo.x)[q] = (&xv.x)[q] * s + (&yv.x)[q] * c;
      }
    }
    uint16_t* dp = dest(g, a, qbuf, lc, l, M, r, hh, f4 * 4);
    *(uint2*)dp = make_uint2(pack_bf16x2(xo.x, xo.y), pack_bf16x2(xo.z, xo.w));
    *(uint2*)(dp + half) = make_uint2(pack_bf16x2(yo.x, yo.y), pack_bf16x2(yo.z, yo.w));
  }
}

// Weight stream of the decode-size projection: the 16x16x32 MFMA operand
// layout asks for 16 weight rows x 64 bytes per load instruction, which reads
// half cache lines and streams ~12% slower (measured), so each copy
// instruction moves 2 rows x 512 contiguous bytes into LDS (non-temporal
// global->LDS copies) instead.  Batches of kDmaKB k-steps (16 rows x 512
// bytes), kDmaBuf per wave in LDS.  Each wave copies and reads only its own
// 16 rows, so the stream needs no workgroup barrier; within a row's 512 bytes
// the 16-byte chunk c sits in lane slot c ^ (row & 15), so that the 16 rows
// one operand read touches fall in distinct bank groups.
constexpr int kDmaKB = 8;                          // k-steps of 32 per batch
constexpr int kDmaBuf = 2;                         // batches per wave in LDS
constexpr int kDmaBatch = 16 * kDmaKB * 64;        // bytes of one batch (16 rows)
constexpr int kDmaNI = kDmaBatch / 1024;           // copy instructions per batch

// Decode-size projection, workgroup-per-tile-group form: workgroup b takes
// `tpw` consecutive (layer, head) tiles (tpw <= kPstTiles, chosen so that the
// grid fills whole rounds of CUs) and keeps one accumulator per tile in
// registers.  The token rows are staged in LDS in column chunks of kd (the
// whole row when it fits in kPstX bytes, with chunk c of row r at slot
// c ^ (r & 15)); for each chunk the workgroup runs over its tiles, so a chunk
// is staged once per workgroup rather than once per tile.  The weight stream
// (above: 2 rows x 512 bytes per non-temporal global->LDS copy, two batches
// of 16 rows x 512 bytes per wave) runs on across tile and chunk borders.  Wave w multiplies channels w * 8 .. w * 8 + 7 and their RoPE
// partners 64 + w * 8 .. 64 + w * 8 + 7, so that in the 16x16 output layout
// the partners of lane l's values sit in lane l ^ 32: the rotation runs in
// registers with factors loaded once, and each lane stores its 4 channels of
// one token (8 bytes).  grid (ceil(tiles / tpw)), block 512.
constexpr int kPstTiles = 8;
constexpr int kPstX = 32 * 1024;

__global__ void __launch_bounds__(64 * kDecWaves, 1)
k_qkv_decode_pst(PoolGeom g, const uint16_t* __restrict__ x, const uint16_t* __restrict__ w,
                 int64_t w_stride, AppendDesc a, uint16_t* __restrict__ qbuf, int l0, int n_lc,
                 int tpw, int kd) {
  constexpr int RPI = 1024 / (kDmaKB * 64);      // rows per copy instruction
  constexpr int SPR = kDmaKB * 4;                // 16-byte slots per row and batch
  __shared__ __attribute__((aligned(16))) char wbuf[kDecWaves * kDmaBuf * kDmaBatch];
  extern __shared__ __attribute__((aligned(16))) uint16_t xs[];  // [M][kd], chunk-swizzled
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lg = lane >> 4;
  const int M = a.batch * a.T, d = g.d;
  const int nt = g.Hq + 2 * g.Hkv;               // head tiles per layer
  const int t0 = (int)blockIdx.x * tpw;
  const int my = min(tpw, nt * n_lc - t0);
  if (my <= 0) return;
  const int nck = d / kd;                        // token-row chunks
  const int nbc = kd / (kDmaKB * 32);            // weight batches per tile and chunk
  const int per_chunk = my * nbc;
  const int total = nck * per_chunk;

  // copy j of a batch: local rows RPI j + lane / SPR; local row r is channel
  // r + w * 8 (+ 56 for r >= 8) of the head
  uint32_t voff[kDmaNI];
#pragma unroll
  for (int j = 0; j < kDmaNI; ++j) {
    const int r = RPI * j + lane / SPR, sl = lane % SPR;
    const int ch = r + wave * 8 + (r >= 8 ? 56 : 0);
    voff[j] = (uint32_t)ch * d * 2 + (sl ^ (r & 15)) * 16;
  }
  const uint32_t lds_w = lds_addr(wbuf) + wave * kDmaBuf * kDmaBatch;
  // batch q of the stream: chunk, tile, batch within the tile's chunk
  auto issue = [&](int q) {
    const int ch = q / per_chunk, rem = q - ch * per_chunk;
    const int k = rem / nbc, jb = rem - k * nbc;
    const int t = t0 + k;
    const int lc = t / nt, hh = t - lc * nt;
    const char* sb = (const char*)(w + (int64_t)(l0 + lc) * w_stride + (int64_t)hh * kDh * d) +
                     ((int64_t)ch * kd + (int64_t)jb * kDmaKB * 32) * 2;
    const uint32_t ld = lds_w + (q % kDmaBuf) * kDmaBatch;
#pragma unroll
    for (int j = 0; j < kDmaNI; ++j) lds_dma16_sv_nt(sb, voff[j], ld + j * 1024);
  };
  issue(0);

  // per-lane output row: token lr, channels i0 .. i0 + 3 of the x (lane < 32)
  // or y (lane >= 32) half of the head; RoPE factors are the same for every tile
  const bool xok = lr < M;
  const int half = kDh / 2;
  const int i0 = wave * 8 + 4 * (lg & 1);
  const int coff = (lg >= 2 ? half : 0) + i0;
  float4 cs = make_float4(1.f, 1.f, 1.f, 1.f), sn = make_float4(0.f, 0.f, 0.f, 0.f);
  int64_t qrow = 0, kvrow = 0;
  if (xok) {
    const RowInfo ri = row_info(a, lr);
    cs = *(const float4*)(g.rope_cos + (int64_t)ri.pos * half + i0);
    sn = *(const float4*)(g.rope_sin + (int64_t)ri.pos * half + i0);
    qrow = (int64_t)lr * g.Hq * kDh;
    const int32_t blk = g.tables[(int64_t)ri.slot * g.max_blocks + ri.u / g.B];
    kvrow = (int64_t)blk * g.block_elems + (int64_t)(ri.u % g.B) * kDh;
  }

  const char* wrd = wbuf + wave * kDmaBuf * kDmaBatch + (lr / RPI) * 1024 + (lr % RPI) * SPR * 16;
  const uint16_t* xr = xs + (xok ? lr : 0) * kd;
  const int c8n = kd / 8;
  floatx4 acc[kPstTiles];
#pragma unroll
  for (int k = 0; k < kPstTiles; ++k) acc[k] = floatx4{0.f, 0.f, 0.f, 0.f};
  int q = 0;
  for (int ch = 0; ch < nck; ++ch) {
    // token rows, columns [ch kd, ch kd + kd), into LDS
    if (ch > 0) __syncthreads();  // every wave has read the previous chunk
    for (int i = tid; i < M * c8n; i += 64 * kDecWaves) {
      const int r = i / c8n, c = i - r * c8n;
      *(uint4*)(xs + (int64_t)r * kd + ((c ^ (r & 15)) * 8)) =
          *(const uint4*)(x + (int64_t)r * d + (int64_t)ch * kd + c * 8);
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kPstTiles; ++k) {
      if (k < my) {
        for (int jb = 0; jb < nbc; ++jb, ++q) {
          // the other buffer was read by the products of batch q - 1; a
          // wave's copies complete in order, kDmaNI per batch
          if (q + 1 < total) {
            issue(q + 1);
            wait_vmcnt<kDmaNI>();
          } else {
            wait_vmcnt<0>();
          }
          const char* wb = wrd + (q % kDmaBuf) * kDmaBatch;
          const int cx = jb * kDmaKB * 4;  // first 16-byte chunk of this batch in a token row
#pragma unroll
          for (int u = 0; u < kDmaKB; ++u) {
            const int c = 4 * u + lg;
            const uint4 fa = *(const uint4*)(wb + (c ^ lr) * 16);
            const uint4 fb =
                xok ? *(const uint4*)(xr + ((cx + c) ^ lr) * 8) : make_uint4(0, 0, 0, 0);
            acc[k] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8v, fa),
                                                             __builtin_bit_cast(bf16x8v, fb),
                                                             acc[k], 0, 0, 0);
          }
        }
      }
    }
  }
  // epilogue in registers: lane l holds channels 4 (l / 16) + e (local rows)
  // of token l % 16; local rows 8 .. 15 (lanes 32 .. 63) are the partners
  // (channel + 64) of rows 0 .. 7 (lanes 0 .. 31)
#pragma unroll
  for (int k = 0; k < kPstTiles; ++k) {
    if (k < my) {
      const int t = t0 + k;
      const int lc = t / nt, hh = t - lc * nt, l = l0 + lc;
      const bool rot = hh < g.Hq + g.Hkv;
      float o[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[k][e]),
                                                        __float_as_uint(acc[k][e]), false, false);
        const float xv = __uint_as_float(r[0]), yv = __uint_as_float(r[1]);
        const float c = (&cs.x)[e], s = (&sn.x)[e];
        o[e] = !rot ? acc[k][e] : (lane < 32 ? fmaf(xv, c, -(yv * s)) : fmaf(xv, s, yv * c));
      }
      if (xok) {
        uint16_t* dp;
        if (hh < g.Hq) {
          dp = qbuf + (int64_t)lc * M * g.Hq * kDh + qrow + (int64_t)hh * kDh + coff;
        } else {
          const int kv = hh < g.Hq + g.Hkv ? 0 : 1;
          const int gh = hh - g.Hq - kv * g.Hkv;
          dp = (uint16_t*)g.pool + kvrow + tile_off(g, l, kv, gh, 0) + coff;
        }
        *(uint2*)dp = make_uint2(pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]));
      }
    }
  }
}

}  // namespace

bool qkv_mfma_ok(const PoolGeom& g, int dtype) {
  return dtype == KV_DTYPE_BF16 && g.dh == kDh && g.d % kBK == 0 &&
         ((g.Hq + 2 * g.Hkv) * kDh) % 256 == 0;
}

hipError_t launch_qkv_mfma(const PoolGeom& g, const void* x, const void* w, int64_t w_stride,
                           const AppendDesc& a, void* qbuf, int l0, int lc, hipStream_t s) {
  const int M = a.batch * a.T;
  const int N = (g.Hq + 2 * g.Hkv) * kDh;
  // x staged in column chunks of kc: the whole row if two workgroups still
  // fit in a CU's LDS, else halves, quarters, ... (multiples of the batch width)
  int kc = g.d;
  const size_t cf_bytes = 16 * (kDh + 4) * 4;
  while (kc % (2 * 32 * kDecU) == 0 && (size_t)M * (kc + 8) * 2 + cf_bytes > 80 * 1024) kc /= 2;
  const size_t x_lds = (size_t)M * (kc + 8) * 2;
  // token-row chunk of the tile-group kernel: the whole row, else halves, ...
  int kx = g.d;
  while ((size_t)M * kx * 2 > kPstX && kx % (2 * kDmaKB * 32) == 0) kx /= 2;
  if (M <= 16 && g.d % (kDmaKB * 32) == 0 && kx % (kDmaKB * 32) == 0 &&
      (size_t)M * kx * 2 <= kPstX) {
    // CU count per device, cached (calls from several threads may race to
    // store the same value)
    static std::atomic<int> cu_cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    int n_cu = cu_cache[dev].load(std::memory_order_relaxed);
    if (n_cu <= 0) {
      if (hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
          n_cu <= 0)
        return hipErrorInvalidDevice;
      cu_cache[dev].store(n_cu, std::memory_order_relaxed);
    }
    // tiles per workgroup: the most (up to kPstTiles) whose grid wastes at
    // most 3% of its last round of CUs, else the least wasteful
    const int tiles = (g.Hq + 2 * g.Hkv) * lc;
    int tpw = 1;
    double best = 2.0;
    for (int t = kPstTiles; t >= 1; --t) {
      const int64_t grid = (tiles + t - 1) / t;
      const int64_t rounds = (grid + n_cu - 1) / n_cu;
      const double waste = (double)(rounds * n_cu - grid) / (double)(rounds * n_cu);
      if (waste <= 0.03) {
        tpw = t;
        break;
      }
      if (waste < best) {
        best = waste;
        tpw = t;
      }
    }
    k_qkv_decode_pst<<<(tiles + tpw - 1) / tpw, 64 * kDecWaves, (size_t)M * kx * 2, s>>>(
        g, (const uint16_t*)x, (const uint16_t*)w, w_stride, a, (uint16_t*)qbuf, l0, lc, tpw, kx);
  } else if (M <= 16 && g.d % (32 * kDecU) == 0 && x_lds + cf_bytes <= 160 * 1024) {
    dim3 grid(N / kDh, 1, lc);
    k_qkv_decode_lds<<<grid, 64 * kDecWaves, x_lds, s>>>(g, (const uint16_t*)x, (const uint16_t*)w,
                                                         w_stride, a, (uint16_t*)qbuf, l0, kc);
  } else if (M <= 16 && g.d % 512 == 0) {
    dim3 grid(N / kDh, 1, lc);
    k_qkv_decode<1><<<grid, 64 * kDecWaves, 0, s>>>(g, (const uint16_t*)x, (const uint16_t*)w,
                                                   w_stride, a, (uint16_t*)qbuf, l0);
  } else if (M <= 32 && g.d % 512 == 0) {
    dim3 grid(N / kDh, 1, lc);
    k_qkv_decode<2><<<grid, 64 * kDecWaves, 0, s>>>(g, (const uint16_t*)x, (const uint16_t*)w,
                                                   w_stride, a, (uint16_t*)qbuf, l0);
  } else if (M <= 32) {
    dim3 grid(N / 128, 1, lc);
    k_qkv_mfma<128, 32, 4, 1><<<grid, kThreads, 0, s>>>(g, (const uint16_t*)x, (const uint16_t*)w,
                                                        w_stride, a, (uint16_t*)qbuf, l0);
  } else {  // qkv_mfma_ok: d % kDlBK == 0
    dim3 grid(N / 256, (M + 255) / 256, lc);
    k_qkv_dl<<<grid, kDlThreads, 0, s>>>(g, (const uint16_t*)x, (const uint16_t*)w, w_stride, a,
                                          (uint16_t*)qbuf, l0);
  }
  return hipGetLastError();
}

}  // namespace kvs
