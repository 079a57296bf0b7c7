// MFMA append path (bf16, head_dim 128).
#include "kv_fast.h"

namespace kvs {

int decode_chunks(const AppendDesc& a);
bool decode_mfma_ok(const PoolGeom& g, int dtype, const AppendDesc& a);
size_t decode_part_layer_bytes(const PoolGeom& g, const AppendDesc& a);
size_t decode_plan_bytes(const AppendDesc& a);
size_t decode_scratch_bound(int64_t L, int64_t batch, int64_t Hq, int64_t max_keys);
hipError_t launch_decode_attn(const PoolGeom& g, const void* qbuf, const AppendDesc& a,
                              void* part, void* plan, int lc, int l0, hipStream_t s);
hipError_t launch_decode_merge(const PoolGeom& g, const AppendDesc& a, void* o, const void* part,
                               int l0, int lc, hipStream_t s);

void fast_scratch_need(const PoolGeom& g, int dtype, const AppendDesc& a, size_t* per_layer,
                       size_t* fixed) {
  const bool dec = decode_mfma_ok(g, dtype, a);
  *per_layer = dec ? decode_part_layer_bytes(g, a) : 0;
  *fixed = dec ? decode_plan_bytes(a) : 0;
}

size_t fast_scratch_bound(const kv_model_cfg& c, int64_t, int32_t batch, int64_t max_keys) {
  // split-key partials and the work-unit plan of a decode call
  return decode_scratch_bound(c.n_layers, batch, c.n_q_heads, max_keys);
}

bool qkv_mfma_ok(const PoolGeom& g, int dtype);
hipError_t launch_qkv_mfma(const PoolGeom& g, const void* x, const void* w, int64_t w_stride,
                           const AppendDesc& a, void* qbuf, int l0, int lc, hipStream_t s);

hipError_t launch_qkv_fast(const PoolGeom& g, int dtype, const void* x, const void* w,
                           int64_t w_stride, const AppendDesc& a, void* qbuf, int l0, int lc,
                           hipStream_t s, bool* done) {
  *done = false;
  if (!qkv_mfma_ok(g, dtype)) return hipSuccess;
  *done = true;
  return launch_qkv_mfma(g, x, w, w_stride, a, qbuf, l0, lc, s);
}

bool attn_mfma_ok(const PoolGeom& g, int dtype, const AppendDesc& a);
hipError_t launch_attn_prefill(const PoolGeom& g, const void* qbuf, const AppendDesc& a, void* o,
                               int l0, int lc, hipStream_t s);

hipError_t launch_attn_fast(const PoolGeom& g, int dtype, const void* qbuf, const AppendDesc& a,
                            void* o, void* part, void* plan, int l0, int lc, hipStream_t s,
                            bool* done, bool* merge) {
  *done = false;
  *merge = false;
  if (decode_mfma_ok(g, dtype, a)) {
    *done = true;
    *merge = true;
    return launch_decode_attn(g, qbuf, a, part, plan, lc, l0, s);
  }
  if (!attn_mfma_ok(g, dtype, a)) return hipSuccess;
  *done = true;
  return launch_attn_prefill(g, qbuf, a, o, l0, lc, s);
}

hipError_t launch_attn_merge(const PoolGeom& g, int, const AppendDesc& a, void* o,
                             const void* part, int l0, int lc, hipStream_t s) {
  return launch_decode_merge(g, a, o, part, l0, lc, s);
}

}  // namespace kvs
