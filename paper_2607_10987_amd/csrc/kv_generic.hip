// Portable append path for any head_dim <= 256 (multiple of 16) and both
// storage types: fp32 vector-ALU kernels.  This is the path of float32 pools
// and of shapes the MFMA kernels do not cover.
//
//  k_qkv_generic: one workgroup computes a 32-row x dh-column tile of
//    X W_l^T (one head of one layer), applies RoPE at each row's position
//    (pairs (i, i + dh/2), angles from the float table built in double on the
//    host), and stores Q into the scratch buffer and K/V into the row's paged
//    block: block = table[slot][(n_before + t) / B], slot = (n_before + t) % B.
//  k_attn_generic: one wavefront per (query row, query head, layer) walks the
//    row's visible keys (key index <= n_before + t) in chunks of 64 with an
//    online (running max / running sum) softmax in fp32.
#include "kv_internal.h"

namespace kvs {

namespace {

template <typename T>
__device__ inline float ld(const T* p);
template <>
__device__ inline float ld<float>(const float* p) { return *p; }
template <>
__device__ inline float ld<uint16_t>(const uint16_t* p) {
  return __uint_as_float((uint32_t)(*p) << 16);
}

template <typename T>
__device__ inline T cvt(float f);
template <>
__device__ inline float cvt<float>(float f) { return f; }
template <>
__device__ inline uint16_t cvt<uint16_t>(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

constexpr int kRows = 32;
constexpr int kKc = 32;
constexpr int kMaxDh = 256;

// grid (Hq + 2 Hkv, ceil(M / 32), lc), block 256
template <typename T>
__global__ void __launch_bounds__(256)
k_qkv_generic(PoolGeom g, const T* __restrict__ x, const T* __restrict__ w, int64_t w_stride,
              AppendDesc a, T* __restrict__ qbuf, int l0) {
  __shared__ float xs[kRows][kKc + 1];
  __shared__ float ws[kMaxDh][kKc + 1];
  __shared__ float cs[kRows][kMaxDh + 1];
  const int head = blockIdx.x;
  const int row0 = blockIdx.y * kRows;
  const int lc = blockIdx.z;
  const int l = l0 + lc;
  const int M = a.batch * a.T;
  const int dh = g.dh, d = g.d;
  const T* wl = w + (int64_t)l * w_stride + (int64_t)head * dh * d;
  const int tid = threadIdx.x;
  const int r = tid / 8, cg = tid % 8;
  const int ncol = dh / 8;  // columns per thread: cg + 8 j
  float acc[kMaxDh / 8];
#pragma unroll
  for (int j = 0; j < kMaxDh / 8; ++j) acc[j] = 0.f;
  for (int k0 = 0; k0 < d; k0 += kKc) {
    for (int e = tid; e < kRows * kKc; e += 256) {
      const int rr = e / kKc, kk = e % kKc;
      const int row = row0 + rr;
      xs[rr][kk] = (row < M && k0 + kk < d) ? ld<T>(x + (int64_t)row * d + k0 + kk) : 0.f;
    }
    for (int e = tid; e < dh * kKc; e += 256) {
      const int cc = e / kKc, kk = e % kKc;
      ws[cc][kk] = (k0 + kk < d) ? ld<T>(wl + (int64_t)cc * d + k0 + kk) : 0.f;
    }
    __syncthreads();
#pragma unroll 4
    for (int kk = 0; kk < kKc; ++kk) {
      const float xv = xs[r][kk];
#pragma unroll
      for (int j = 0; j < kMaxDh / 8; ++j)
        if (j < ncol) acc[j] += xv * ws[cg + 8 * j][kk];
    }
    __syncthreads();
  }
#pragma unroll
  for (int j = 0; j < kMaxDh / 8; ++j)
    if (j < ncol) cs[r][cg + 8 * j] = acc[j];
  __syncthreads();
  const int half = dh / 2;
  const int kind = head < g.Hq ? 0 : (head < g.Hq + g.Hkv ? 1 : 2);  // Q, K, V
  for (int e = tid; e < kRows * half; e += 256) {
    const int rr = e / half, i = e % half;
    const int row = row0 + rr;
    if (row >= M) continue;
    const int sq = row / a.T, t = row % a.T;
    const SeqDesc sd = a.seq[sq];
    const int u = sd.n_before + t;
    const int pos = sd.pos0 + u;
    float xv = cs[rr][i], yv = cs[rr][i + half];
    if (kind < 2) {
      const float c = g.rope_cos[(int64_t)pos * half + i];
      const float s = g.rope_sin[(int64_t)pos * half + i];
      const float xr = xv * c - yv * s;
      const float yr = xv * s + yv * c;
      xv = xr;
      yv = yr;
    }
    if (kind == 0) {
      T* q = qbuf + ((int64_t)lc * M + row) * (g.Hq * dh) + head * dh;
      q[i] = cvt<T>(xv);
      q[i + half] = cvt<T>(yv);
    } else {
      const int hk = kind == 1 ? head - g.Hq : head - g.Hq - g.Hkv;
      const int32_t blk = g.tables[(int64_t)sd.slot * g.max_blocks + u / g.B];
      T* p = (T*)g.pool + (int64_t)blk * g.block_elems + tile_off(g, l, kind - 1, hk, u % g.B);
      p[i] = cvt<T>(xv);
      p[i + half] = cvt<T>(yv);
    }
  }
}

__device__ inline float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ inline float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// grid (M, Hq, lc), block 64 (one wavefront)
template <typename T>
__global__ void __launch_bounds__(64)
k_attn_generic(PoolGeom g, const T* __restrict__ qbuf, AppendDesc a, T* __restrict__ o, int l0,
               float scale) {
  __shared__ float qs[kMaxDh];
  const int row = blockIdx.x, h = blockIdx.y, lc = blockIdx.z;
  const int l = l0 + lc;
  const int M = a.batch * a.T;
  const int dh = g.dh;
  const int lane = threadIdx.x;
  const int sq = row / a.T, t = row % a.T;
  const SeqDesc sd = a.seq[sq];
  const int nkeys = sd.n_before + t + 1;
  const int hk = h / (g.Hq / g.Hkv);
  const T* q = qbuf + ((int64_t)lc * M + row) * (g.Hq * dh) + h * dh;
  for (int i = lane; i < dh; i += 64) qs[i] = ld<T>(q + i);
  __syncthreads();
  const T* pool = (const T*)g.pool;
  const int32_t* trow = g.tables + (int64_t)sd.slot * g.max_blocks;
  const int nd = (dh + 63) / 64;
  float acc[kMaxDh / 64];
  for (int j = 0; j < kMaxDh / 64; ++j) acc[j] = 0.f;
  float m = -INFINITY, lsum = 0.f;
  for (int k0 = 0; k0 < nkeys; k0 += 64) {
    const int key = k0 + lane;
    float sc = -INFINITY;
    if (key < nkeys) {
      const int32_t blk = trow[key / g.B];
      const T* kp = pool + (int64_t)blk * g.block_elems + tile_off(g, l, 0, hk, key % g.B);
      float dot = 0.f;
      for (int i = 0; i < dh; ++i) dot += qs[i] * ld<T>(kp + i);
      sc = dot * scale;
    }
    const float mn = fmaxf(m, wave_max(sc));
    const float p = key < nkeys ? __expf(sc - mn) : 0.f;
    const float alpha = __expf(m - mn);
    lsum = lsum * alpha + wave_sum(p);
    for (int j = 0; j < kMaxDh / 64; ++j) acc[j] *= alpha;
    const int nk = min(64, nkeys - k0);
    for (int jk = 0; jk < nk; ++jk) {
      const float pj = __shfl(p, jk);
      const int kk = k0 + jk;
      const int32_t blk = trow[kk / g.B];
      const T* vp = pool + (int64_t)blk * g.block_elems + tile_off(g, l, 1, hk, kk % g.B);
      for (int j = 0; j < nd; ++j) {
        const int i = lane + 64 * j;
        if (i < dh) acc[j] += pj * ld<T>(vp + i);
      }
    }
    m = mn;
  }
  T* op = o + ((int64_t)l * M + row) * (g.Hq * dh) + h * dh;
  const float inv = 1.f / lsum;
  for (int j = 0; j < nd; ++j) {
    const int i = lane + 64 * j;
    if (i < dh) op[i] = cvt<T>(acc[j] * inv);
  }
}

}  // namespace

hipError_t launch_qkv_generic(const PoolGeom& g, int dtype, const void* x, const void* w,
                              int64_t w_stride, const AppendDesc& a, void* qbuf, int l0, int lc,
                              hipStream_t s) {
  const int M = a.batch * a.T;
  dim3 grid(g.Hq + 2 * g.Hkv, (M + kRows - 1) / kRows, lc);
  if (dtype == KV_DTYPE_BF16)
    k_qkv_generic<uint16_t><<<grid, 256, 0, s>>>(g, (const uint16_t*)x, (const uint16_t*)w,
                                                 w_stride, a, (uint16_t*)qbuf, l0);
  else
    k_qkv_generic<float><<<grid, 256, 0, s>>>(g, (const float*)x, (const float*)w, w_stride, a,
                                              (float*)qbuf, l0);
  return hipGetLastError();
}

hipError_t launch_attn_generic(const PoolGeom& g, int dtype, const void* qbuf,
                               const AppendDesc& a, void* o, int l0, int lc, hipStream_t s) {
  const int M = a.batch * a.T;
  dim3 grid(M, g.Hq, lc);
  const float scale = 1.0f / sqrtf((float)g.dh);
  if (dtype == KV_DTYPE_BF16)
    k_attn_generic<uint16_t><<<grid, 64, 0, s>>>(g, (const uint16_t*)qbuf, a, (uint16_t*)o, l0,
                                                 scale);
  else
    k_attn_generic<float><<<grid, 64, 0, s>>>(g, (const float*)qbuf, a, (float*)o, l0, scale);
  return hipGetLastError();
}

}  // namespace kvs
