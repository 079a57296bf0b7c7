// Internal declarations shared by the host catalog (kv_api.cpp) and the HIP
// kernels (kv_*.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvstate.h"

namespace kvs {

// Device-resident allocator header (first 256 bytes of the metadata area).
// head/tail are monotone counters of the free ring: ring[(i) % P] for
// i in [head, tail) are the free block ids, oldest first.
struct DevHeader {
  int64_t head;
  int64_t tail;
  int32_t status;     // sticky: 0 or KV_ERR_INTERNAL
  int32_t n_evicted;  // result of the last release/evict kernel
  int32_t pad[58];
};
static_assert(sizeof(DevHeader) == 256, "header size");

// Geometry of one pool, passed by value to every data kernel.
struct PoolGeom {
  void* pool;             // [P][L][2][Hkv][B][dh]
  const int32_t* tables;  // [max_states][max_blocks]
  const float* rope_cos;  // [max_pos][dh/2]
  const float* rope_sin;  // [max_pos][dh/2]
  const float* rope_cos_g;  // [dh/8][max_pos][4]: channels 4q .. 4q+3 of group q
  const float* rope_sin_g;  // [dh/8][max_pos][4]
  int64_t block_elems;    // L * 2 * Hkv * B * dh
  int32_t max_blocks;
  int32_t L, Hq, Hkv, dh, B, d;
  int32_t max_pos;
  int32_t b_shift;  // log2(B) when B is a power of two, else -1
};

// Element offset of (layer, K|V, kv head, slot, channel 0) inside a block.
__host__ __device__ inline int64_t tile_off(const PoolGeom& g, int l, int kv, int h, int slot) {
  return ((((int64_t)l * 2 + kv) * g.Hkv + h) * g.B + slot) * (int64_t)g.dh;
}

// One sequence of a batched append: catalog slot, tokens already cached,
// position of token 0.
struct SeqDesc {
  int32_t slot;
  int32_t n_before;
  int32_t pos0;
  int32_t pad;
};

struct AppendDesc {
  int32_t batch;
  int32_t T;
  int32_t max_keys;  // max over the batch of n_before + T
  int32_t pad;
  SeqDesc seq[KV_MAX_BATCH];
};

// Allocation requests, processed in order: if cow > 0, copy-on-write of the
// entry `first - 1` (whose first `cow` slots hold valid tokens), then `count`
// new entries starting at `first`.  partial = valid slots of entry
// `first - 1` when it is a partial tail block (0 otherwise): with cow == 0
// the host holds that tail private, and the kernel checks that no other
// table references it.
struct AllocReq {
  int32_t slot, first, count, cow, partial;
};
struct AllocArgs {
  int32_t n_req;
  int32_t pad[3];
  AllocReq req[KV_MAX_BATCH];
};

struct ForkArgs {
  int32_t parent, nblocks, k, pad;
  int32_t child[KV_MAX_FORK];
};

// One compose segment after host planning.  Destination token u of segment i
// reads source token j = u - off; its key is re-rotated by delta.  Destination
// blocks [alias_b0, alias_b1) alias source blocks b - off / B.
struct SegDesc {
  int32_t slot;
  int32_t cum;    // first destination token of the segment
  int32_t off;
  int32_t delta;
  int32_t alias_b0, alias_b1;
  int32_t pad[2];
};
struct ComposeArgs {
  int32_t nseg, new_slot, n_tokens, n_dest_blocks;
  SegDesc seg[KV_MAX_SEGMENTS];
};

// ---------------------------------------------------------------- launchers
// Every launcher enqueues on `s` and returns hipGetLastError().

hipError_t launch_alloc(DevHeader* hdr, int32_t* ring, int32_t* rc, int32_t* tables,
                        int32_t max_blocks, int32_t P, int64_t head, const AllocArgs& a,
                        int2* cow_pairs, hipStream_t s);
hipError_t launch_fork(DevHeader* hdr, int32_t* tables, int32_t max_blocks, int32_t* rc,
                       const ForkArgs& a, hipStream_t s);
hipError_t launch_release(DevHeader* hdr, int32_t* ring, int32_t* rc, const int32_t* tables,
                          int32_t max_blocks, int32_t P, const int32_t* cand, int32_t n_cand,
                          int64_t max_alloc, int64_t head, int64_t tail, int32_t truncate,
                          int32_t* kept, hipStream_t s);
hipError_t launch_compose_meta(DevHeader* hdr, int32_t* ring, int32_t* rc, int32_t* tables,
                               int32_t max_blocks, int32_t P, int32_t B, int64_t head,
                               int32_t ncopy, const ComposeArgs& a, hipStream_t s);

// Payload checksum accumulators: pairs (s1, s2) in kSumSlots slots of the
// metadata area, zero between checksummed copies (k_csum_final clears them).
constexpr int kSumSlots = 1024;

// slots != null: also add the checksum terms of the bytes copied, the launch's
// first block starting at payload chunk (16 bytes) index base16.
hipError_t launch_pack(const PoolGeom& g, int dtype, const int32_t* trow, int64_t b0,
                       int32_t nblk, int32_t last_valid, void* dst, unsigned long long* slots,
                       int64_t base16, hipStream_t s);
hipError_t launch_unpack(const PoolGeom& g, int dtype, const int32_t* trow, int32_t nblk,
                         const void* src, unsigned long long* slots, int64_t base16,
                         hipStream_t s);
// out[0..1] = the slots' sums (s1, s2); clears the slots.
hipError_t launch_csum_final(unsigned long long* slots, unsigned long long* out, hipStream_t s);
hipError_t launch_cow(const PoolGeom& g, int dtype, const int2* cow_pairs, const AllocArgs& a,
                      hipStream_t s);
hipError_t launch_compose_copy(const PoolGeom& g, int dtype, const ComposeArgs& a,
                               hipStream_t s);

// Append path (projection + RoPE + paged store, then causal attention) for
// layers [l0, l0 + lc).  x: [M][d], w: layer 0 weights, qbuf: [lc][M][Hq*dh],
// o: [L][M][Hq*dh] with M = batch * T.
hipError_t launch_qkv_generic(const PoolGeom& g, int dtype, const void* x, const void* w,
                              int64_t w_stride, const AppendDesc& a, void* qbuf, int l0, int lc,
                              hipStream_t s);
hipError_t launch_attn_generic(const PoolGeom& g, int dtype, const void* qbuf,
                               const AppendDesc& a, void* o, int l0, int lc, hipStream_t s);

}  // namespace kvs
