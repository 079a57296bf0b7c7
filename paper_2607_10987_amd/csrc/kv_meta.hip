// Block allocator kernels: the free ring, refcounts and block tables live in
// device memory and are only changed here.
//
// Semantics (the paper's metadata catalog: a block's refcount is the number of
// logical states that share it; KV-Fork aliases blocks by raising refcounts;
// KV-Evict frees a state's blocks, shared blocks surviving while referenced):
//  - allocation pops ids from the ring head in order (FIFO), so a sequence of
//    operations has exactly one resulting set of tables;
//  - release decrements a state's blocks in logical order and appends the ids
//    reaching zero to the ring tail in that order (a workgroup prefix scan
//    assigns ring slots, no atomics), states in the given order.
// Each kernel is a single workgroup or touches disjoint ids, so results are
// deterministic.  A mismatch with the host's expected counters sets the sticky
// status KV_ERR_INTERNAL and the kernel does nothing.  k_alloc also checks the
// host's copy-on-write decisions against the refcounts in both directions (a
// tail it copies must be shared, a partial tail it appends to in place must
// not be) and sets the same status when they disagree.
#include "kv_internal.h"

namespace kvs {

namespace {

constexpr int kMetaThreads = 256;

__device__ inline bool fail_if(DevHeader* hdr, bool bad) {
  if (bad && threadIdx.x == 0) hdr->status = KV_ERR_INTERNAL;
  return bad;
}

__global__ void __launch_bounds__(kMetaThreads)
k_alloc(DevHeader* hdr, int32_t* ring, int32_t* rc, int32_t* tables, int32_t max_blocks,
        int32_t P, int64_t head, AllocArgs a, int2* cow_pairs) {
  __shared__ int ok;
  if (threadIdx.x == 0) {
    int64_t need = 0;
    for (int r = 0; r < a.n_req; ++r) need += a.req[r].count + (a.req[r].cow > 0 ? 1 : 0);
    ok = hdr->status == 0 && hdr->head == head && hdr->tail - head >= need;
  }
  __syncthreads();
  if (fail_if(hdr, !ok)) return;
  int64_t pos = head;
  for (int r = 0; r < a.n_req; ++r) {
    const AllocReq q = a.req[r];
    int32_t* trow = tables + (int64_t)q.slot * max_blocks;
    if (q.cow > 0) {
      if (threadIdx.x == 0) {
        const int32_t old = trow[q.first - 1];
        const int32_t nb = ring[pos % P];
        if (rc[old] <= 1) hdr->status = KV_ERR_INTERNAL;
        rc[old] -= 1;
        rc[nb] = 1;
        trow[q.first - 1] = nb;
        cow_pairs[r] = make_int2(old, nb);
      }
      pos += 1;
    } else if (q.partial > 0 && threadIdx.x == 0 && rc[trow[q.first - 1]] != 1) {
      // the host appends into a partial tail it holds alone; another table
      // referencing it would see the append's tokens
      hdr->status = KV_ERR_INTERNAL;
    }
    for (int i = threadIdx.x; i < q.count; i += blockDim.x) {
      const int32_t id = ring[(pos + i) % P];
      trow[q.first + i] = id;
      rc[id] = 1;
    }
    pos += q.count;
    __syncthreads();
  }
  if (threadIdx.x == 0) hdr->head = pos;
}

__global__ void k_fork(DevHeader* hdr, int32_t* tables, int32_t max_blocks, int32_t* rc,
                       ForkArgs a) {
  if (hdr->status) return;
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= a.nblocks) return;
  const int32_t b = tables[(int64_t)a.parent * max_blocks + j];
  rc[b] += a.k;  // ids within one table are distinct: no two threads share b
  for (int c = 0; c < a.k; ++c) tables[(int64_t)a.child[c] * max_blocks + j] = b;
}

// Exclusive prefix count of `flag` over the workgroup; returns the total.
__device__ inline int block_scan(int flag, int* excl, int* wave_tot) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const uint64_t m = __ballot(flag);
  const uint64_t below = lane ? (m & ((~0ull) >> (64 - lane))) : 0ull;
  const int in_wave = __popcll(below);
  if (lane == 0) wave_tot[wave] = __popcll(m);
  __syncthreads();
  int base = 0, total = 0;
  const int nw = blockDim.x >> 6;
  for (int w = 0; w < nw; ++w) {
    if (w < wave) base += wave_tot[w];
    total += wave_tot[w];
  }
  *excl = base + in_wave;
  __syncthreads();
  return total;
}

// cand: pairs (slot, n_blocks) in release order.  max_alloc < 0 releases all.
// truncate != 0: a candidate gives up only the blocks from its first unshared
// one (refcount 1) on, and kept[c] receives the number of leading blocks it
// keeps (0: released whole; n_blocks: nothing to give up, untouched).
// hdr->n_evicted = candidates visited before the budget was met.
__global__ void __launch_bounds__(kMetaThreads)
k_release(DevHeader* hdr, int32_t* ring, int32_t* rc, const int32_t* tables,
          int32_t max_blocks, int32_t P, const int32_t* cand, int32_t n_cand,
          int64_t max_alloc, int64_t head, int64_t tail, int32_t truncate, int32_t* kept) {
  __shared__ int ok;
  __shared__ int first_own;
  __shared__ int wave_tot[kMetaThreads / 64];
  if (threadIdx.x == 0) ok = hdr->status == 0 && hdr->head == head && hdr->tail == tail;
  __syncthreads();
  if (fail_if(hdr, !ok)) return;
  int n_ev = 0;
  for (int c = 0; c < n_cand; ++c) {
    if (max_alloc >= 0 && (int64_t)P - (tail - head) <= max_alloc) break;
    const int32_t slot = cand[2 * c];
    const int32_t nb = cand[2 * c + 1];
    const int32_t* trow = tables + (int64_t)slot * max_blocks;
    int start = 0;
    if (truncate) {
      if (threadIdx.x == 0) first_own = nb;
      __syncthreads();
      for (int j = threadIdx.x; j < nb; j += blockDim.x)
        if (rc[trow[j]] == 1) atomicMin(&first_own, j);
      __syncthreads();
      start = first_own;
      if (threadIdx.x == 0) kept[c] = start;
      __syncthreads();  // first_own is reset by the next candidate
      if (start == nb) {
        ++n_ev;
        continue;
      }
    }
    for (int j0 = start; j0 < nb; j0 += blockDim.x) {
      const int j = j0 + threadIdx.x;
      int flag = 0;
      int32_t b = -1;
      if (j < nb) {
        b = trow[j];
        const int32_t v = rc[b] - 1;
        rc[b] = v;
        flag = v == 0;
      }
      int excl;
      const int total = block_scan(flag, &excl, wave_tot);
      if (flag) ring[(tail + excl) % P] = b;
      tail += total;
    }
    ++n_ev;
  }
  if (threadIdx.x == 0) {
    hdr->tail = tail;
    hdr->n_evicted = n_ev;
  }
}

__global__ void __launch_bounds__(kMetaThreads)
k_compose_meta(DevHeader* hdr, int32_t* ring, int32_t* rc, int32_t* tables,
               int32_t max_blocks, int32_t P, int32_t B, int64_t head, int32_t ncopy,
               ComposeArgs a) {
  __shared__ int ok;
  if (threadIdx.x == 0) ok = hdr->status == 0 && hdr->head == head && hdr->tail - head >= ncopy;
  __syncthreads();
  if (fail_if(hdr, !ok)) return;
  int32_t* dst = tables + (int64_t)a.new_slot * max_blocks;
  for (int b = threadIdx.x; b < a.n_dest_blocks; b += blockDim.x) {
    int before = 0, seg = -1;
    for (int i = 0; i < a.nseg; ++i) {
      const int lo = a.seg[i].alias_b0, hi = a.seg[i].alias_b1;
      if (b >= lo && b < hi) seg = i;
      const int c = min(b, hi) - lo;
      before += c > 0 ? c : 0;
    }
    int32_t id;
    if (seg >= 0) {
      const SegDesc& sd = a.seg[seg];
      id = tables[(int64_t)sd.slot * max_blocks + (b - sd.off / B)];
      rc[id] += 1;  // distinct positions -> distinct source blocks
    } else {
      id = ring[(head + (b - before)) % P];
      rc[id] = 1;
    }
    dst[b] = id;
  }
  if (threadIdx.x == 0) hdr->head = head + ncopy;
}

}  // namespace

hipError_t launch_alloc(DevHeader* hdr, int32_t* ring, int32_t* rc, int32_t* tables,
                        int32_t max_blocks, int32_t P, int64_t head, const AllocArgs& a,
                        int2* cow_pairs, hipStream_t s) {
  k_alloc<<<1, kMetaThreads, 0, s>>>(hdr, ring, rc, tables, max_blocks, P, head, a, cow_pairs);
  return hipGetLastError();
}

hipError_t launch_fork(DevHeader* hdr, int32_t* tables, int32_t max_blocks, int32_t* rc,
                       const ForkArgs& a, hipStream_t s) {
  if (a.nblocks <= 0) return hipSuccess;
  const int grid = (a.nblocks + kMetaThreads - 1) / kMetaThreads;
  k_fork<<<grid, kMetaThreads, 0, s>>>(hdr, tables, max_blocks, rc, a);
  return hipGetLastError();
}

hipError_t launch_release(DevHeader* hdr, int32_t* ring, int32_t* rc, const int32_t* tables,
                          int32_t max_blocks, int32_t P, const int32_t* cand, int32_t n_cand,
                          int64_t max_alloc, int64_t head, int64_t tail, int32_t truncate,
                          int32_t* kept, hipStream_t s) {
  k_release<<<1, kMetaThreads, 0, s>>>(hdr, ring, rc, tables, max_blocks, P, cand, n_cand,
                                       max_alloc, head, tail, truncate, kept);
  return hipGetLastError();
}

hipError_t launch_compose_meta(DevHeader* hdr, int32_t* ring, int32_t* rc, int32_t* tables,
                               int32_t max_blocks, int32_t P, int32_t B, int64_t head,
                               int32_t ncopy, const ComposeArgs& a, hipStream_t s) {
  k_compose_meta<<<1, kMetaThreads, 0, s>>>(hdr, ring, rc, tables, max_blocks, P, B, head,
                                            ncopy, a);
  return hipGetLastError();
}

}  // namespace kvs
