// MFMA (bf16) append path: projection GEMM with fused RoPE and paged store,
// causal prefill attention, and split-K decode attention.  Each launcher sets
// *done = false (and enqueues nothing) when the shape is not covered, in which
// case the portable kernels of kv_generic.hip run instead.
#pragma once

#include "kv_internal.h"

namespace kvs {

// Scratch bytes the fast attention needs beyond the Q buffer for this call:
// *per_layer for each layer of a group in flight (split-key partials) and
// *fixed once per call (the decode work plan), both multiples of 256.
void fast_scratch_need(const PoolGeom& g, int dtype, const AppendDesc& a, size_t* per_layer,
                       size_t* fixed);
// An upper bound of the same for calls of `tokens` new tokens over at most
// `max_keys` keys per state.
size_t fast_scratch_bound(const kv_model_cfg& c, int64_t tokens, int32_t batch, int64_t max_keys);

hipError_t launch_qkv_fast(const PoolGeom& g, int dtype, const void* x, const void* w,
                           int64_t w_stride, const AppendDesc& a, void* qbuf, int l0, int lc,
                           hipStream_t s, bool* done);
// part: per_layer bytes for each layer of the group; plan: the fixed bytes,
// written by the group that starts at layer 0 and read by every group.
// *merge = true when the launch wrote split-key partials that
// launch_attn_merge must combine into o.
hipError_t launch_attn_fast(const PoolGeom& g, int dtype, const void* qbuf, const AppendDesc& a,
                            void* o, void* part, void* plan, int l0, int lc, hipStream_t s,
                            bool* done, bool* merge);
hipError_t launch_attn_merge(const PoolGeom& g, int dtype, const AppendDesc& a, void* o,
                             const void* part, int l0, int lc, hipStream_t s);

}  // namespace kvs
