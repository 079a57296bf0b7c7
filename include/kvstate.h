/*
 * kvstate.h - C ABI of the MI355X (gfx950) KV-state library.
 *
 * The library implements, on one GPU, the on-device path of the stateful KV
 * operators of AAFLOW+ (arXiv 2607.10987): a paged, refcounted KV block pool
 * and the operators materialize, fork, compose (restricted merge), pack /
 * unpack (the device side of transfer), attend (resume: append-prefill and
 * decode) and evict.
 *
 * Conventions
 * -----------
 * - Every function returns a kv_status (KV_OK = 0, errors < 0).
 * - Host-detectable errors return before anything is enqueued and leave the
 *   pool unchanged (all-or-nothing).
 * - Device work is enqueued on `stream` (a hipStream_t passed as void*; NULL
 *   is the default stream).  All mutating calls on one pool must use one
 *   stream (or be ordered by the caller); concurrent calls on one pool race.
 *   kv_release, kv_evict and kv_evict_truncate synchronise `stream`
 *   before returning.
 * - The caller owns all device memory: the pool, the metadata area, the
 *   scratch area, weights, inputs, outputs and transfer buffers.  The pool,
 *   metadata and scratch areas must be 256-byte aligned, the other buffers
 *   16-byte aligned.  Every device buffer must be device memory of the GPU
 *   that was current at kv_pool_create, inside one allocation that holds the
 *   bytes the call reads or writes: the library checks this before it
 *   launches anything (KV_ERR_ARG for the wrong kind of memory or a
 *   misaligned pointer, KV_ERR_BUFSIZE for an allocation that ends too
 *   early).  The library owns only host-side catalog memory.
 * - A kernel launch that fails after a call has started changing the pool
 *   (KV_ERR_HIP) leaves the host catalog as it was before the call, but the
 *   device may hold part of the call's effect, so the pool is marked failed:
 *   every later call on it returns KV_ERR_HIP (only kv_pool_destroy and the
 *   read-only queries still work).
 * - Layouts are row-major.  `dtype` is KV_DTYPE_F32 (float) or KV_DTYPE_BF16
 *   (bfloat16); inputs, weights, outputs and pool contents all use it.
 *
 * Pool layout: pool[P][L][2][Hkv][B][dh] (block, layer, K|V, KV head, slot,
 * channel).  One block holds B consecutive token positions of one state for
 * every layer (the paper's block b_j = (K_j, V_j, l_j, r_j, d_j), stateful
 * operator section, with l_j spanning all layers of one physical block).
 */
#ifndef KVSTATE_H
#define KVSTATE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t kv_status;
enum {
  KV_OK = 0,
  KV_ERR_ARG = -1,          /* malformed argument */
  KV_ERR_OOM = -2,          /* not enough free blocks (nothing allocated) */
  KV_ERR_INCOMPATIBLE = -3, /* Compat(S_a, S_b) = 0: caller should recompute */
  KV_ERR_EVICTED = -4,      /* handle is stale: evicted or released */
  KV_ERR_BAD_HEADER = -5,   /* pack header magic/version/sizes invalid */
  KV_ERR_BUFSIZE = -6,      /* caller buffer too small */
  KV_ERR_CAPACITY = -7,     /* catalog full or positions beyond max_pos */
  KV_ERR_HIP = -8,          /* HIP runtime error */
  KV_ERR_INTERNAL = -9,     /* device consistency check failed */
  KV_ERR_CHECKSUM = -10,    /* payload does not match the header's checksum */
  KV_ERR_IO = -11           /* checkpoint file could not be opened, read or written */
};

enum { KV_DTYPE_F32 = 0, KV_DTYPE_BF16 = 1 };

/* Lineage word (the paper's Lambda): kind in bits 56..63, fork index j in
 * bits 32..55, parent state id in bits 0..31 (0xFFFFFFFF = none). */
enum {
  KV_LINEAGE_MATERIALIZE = 1,
  KV_LINEAGE_FORK = 2,
  KV_LINEAGE_TRANSFER = 3,
  KV_LINEAGE_MERGE = 4
};

enum { KV_MAX_BATCH = 64, KV_MAX_SEGMENTS = 64, KV_MAX_FORK = 64 };

/* Size of the fixed work area of kv_attend_noalloc, in MiB. */
#define KV_NOALLOC_SCRATCH_MB 64

typedef int64_t kv_state;       /* catalog slot | generation << 32 */
typedef struct kv_pool kv_pool; /* opaque */
typedef void* kv_stream;        /* hipStream_t */

/* Model identity and configuration: the paper's M (model_id) and Theta. Two
 * states or a pool and a pack header are compatible iff model_id and every
 * shape field from n_layers to rope_base are equal (Compat predicate, KV state
 * object section).  max_pos and max_states are capacities of one pool. */
typedef struct {
  int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, block_size;
  int32_t dtype;      /* KV_DTYPE_* */
  int32_t max_pos;    /* positions 0 .. max_pos-1 are valid */
  int32_t max_states; /* live states in the catalog */
  int32_t reserved;
  double rope_base;
  uint64_t model_id;
} kv_model_cfg;

/* One segment of a composition: tokens [tok_begin, tok_end) of `state`. */
typedef struct {
  kv_state state;
  int64_t tok_begin, tok_end;
} kv_segment;

#define KV_PACK_MAGIC 0x5453564Bu
#define KV_PACK_VERSION 2u
#define KV_PACK_CHECKSUM 1u /* kv_pack_header.flags: checksum[] is set */

/* Metadata descriptor sent beside a packed payload (KV-Transfer algorithm:
 * metadata travels separately from the raw block buffers).  Plain old data. */
typedef struct {
  uint32_t magic, version;
  uint64_t model_id;
  kv_model_cfg cfg;
  int64_t pos_begin;     /* position of the first packed token */
  int64_t n_tokens;      /* valid tokens in the payload */
  int64_t blk_begin;     /* first logical block of the source state */
  int64_t n_blocks;
  uint64_t block_bytes;  /* bytes of one block (all layers) */
  uint64_t payload_bytes;
  uint64_t lineage;      /* source state's lineage word */
  int64_t src_state_id;  /* source state's id */
  uint32_t flags;        /* KV_PACK_CHECKSUM or 0; other bits invalid */
  uint32_t reserved;     /* 0 */
  /* With KV_PACK_CHECKSUM: payload read as little-endian uint32 words
   * w_0 .. w_{N-1}, checksum[0] = sum of w_i and checksum[1] = sum of
   * (i + 1) * w_i, both mod 2^64 (a position-weighted sum: any single changed
   * word and any exchange of two unequal words change it). */
  uint64_t checksum[2];
} kv_pack_header;

/* Sizes of the caller-provided device areas for a pool of n_blocks blocks.
 * pool_bytes: the block storage; meta_bytes: refcounts, free ring, block
 * tables, the RoPE tables (cos and sin of every position and frequency, in
 * two layouts: position-major and grouped by 4 frequencies) and command
 * staging. */
kv_status kv_pool_bytes(const kv_model_cfg* cfg, int64_t n_blocks, size_t* pool_bytes,
                        size_t* meta_bytes);

/* Scratch bytes that let a single materialize/attend call of `tokens` total
 * new tokens (batch * T) over at most `max_keys` keys per state run with all
 * layers at once.  A smaller scratch area works: layers are then processed
 * in groups (at least one layer must fit). */
size_t kv_scratch_bytes(const kv_model_cfg* cfg, int64_t tokens, int32_t batch,
                        int64_t max_keys);

/* Create a pool.  init_free_order (host, nullable) is a permutation of
 * 0..n_blocks-1 giving the initial order of the free ring (default identity).
 * Builds the cos/sin table (double precision, stored as float) and clears the
 * metadata; synchronises `stream`. */
kv_status kv_pool_create(const kv_model_cfg* cfg, int64_t n_blocks, void* pool_dev,
                         void* meta_dev, void* scratch_dev, size_t scratch_bytes,
                         const int32_t* init_free_order, kv_stream stream, kv_pool** out);
kv_status kv_pool_destroy(kv_pool* pool);

/* Borrow the QKV weights: layer l at w_dev + l * layer_stride_elems, each
 * [(Hq + 2 Hkv) * dh][d_model] (query heads, then key heads, then value heads;
 * QKV = X W^T).  The memory must outlive its use. */
kv_status kv_set_weights(kv_pool* pool, const void* w_dev, int64_t layer_stride_elems);

/* KV-Materialize (KV operator algorithms): prefill x [T][d_model] (one hidden
 * state matrix shared by every layer) at positions pos0 .. pos0+T-1.  Projects
 * Q, K, V per layer, applies RoPE to Q and K, writes K and V into newly
 * allocated blocks (FIFO order), and writes the causal GQA attention output
 * o [L][T][Hq * dh].  Returns the new state. */
kv_status kv_materialize(kv_pool* pool, const void* x_dev, int64_t T, int64_t pos0,
                         void* o_dev, kv_stream stream, kv_state* out);

/* KV-Fork: k children alias every block of `parent` (refcount += k); each
 * child's lineage records fork(j), j = 1..k.  children: host array of k. */
kv_status kv_fork(kv_pool* pool, kv_state parent, int32_t k, kv_state* children,
                  kv_stream stream);

/* Restricted-KV-Merge by ordered, non-overlapping concatenation: segment i is
 * placed after segments 0..i-1, starting at the position of segment 0's first
 * token.  Keys of a segment whose position changes by D are re-rotated by D;
 * values are copied bit-exactly; destination blocks that are identical to a
 * source block (zero shift, same slot alignment) are aliased instead of
 * copied.  segs: host array of n (1 <= n <= KV_MAX_SEGMENTS). */
kv_status kv_compose(kv_pool* pool, const kv_segment* segs, int32_t n, kv_stream stream,
                     kv_state* out);

/* KV-Transfer, source side: write logical blocks [blk_begin, blk_end) of
 * `state` to dst_dev as n_blocks * block_bytes contiguous bytes in logical
 * order (each block in the pool's block layout; slots after the state's last
 * token zero-filled) and fill *hdr_out.  dst_dev is device memory or pinned
 * host memory (hipHostMalloc; the host tier of a state, written over the
 * host link); any other pointer is KV_ERR_ARG.  16-byte aligned. */
kv_status kv_pack(kv_pool* pool, kv_state state, int64_t blk_begin, int64_t blk_end,
                  void* dst_dev, size_t dst_bytes, kv_pack_header* hdr_out, kv_stream stream);

/* kv_pack with the payload checksum computed in the same pass over the bytes
 * (fused into the copy kernel) and stored in hdr_out->checksum, with
 * KV_PACK_CHECKSUM in hdr_out->flags.  Synchronises `stream`. */
kv_status kv_pack_checked(kv_pool* pool, kv_state state, int64_t blk_begin, int64_t blk_end,
                          void* dst_dev, size_t dst_bytes, kv_pack_header* hdr_out,
                          kv_stream stream);

/* KV-Transfer, destination side: check the header (KV_ERR_BAD_HEADER) and
 * compatibility (KV_ERR_INCOMPATIBLE), allocate n_blocks blocks from the free
 * ring, copy the payload and register a state at positions pos_begin ..
 * src_dev is device memory or pinned host memory (as for kv_pack).
 * With KV_PACK_CHECKSUM in hdr->flags the copy also computes the payload's
 * checksum and the call synchronises `stream`; on a mismatch the new blocks
 * go back to the tail of the free ring (logical order), the state id drawn
 * for the state is not reused, and the result is KV_ERR_CHECKSUM. */
kv_status kv_unpack(kv_pool* pool, const kv_pack_header* hdr, const void* src_dev,
                    size_t src_bytes, kv_stream stream, kv_state* out);

/* File checkpoint of a state (persistence of the host tier): the header of a
 * checksummed pack of all of the state's blocks, then its payload, written
 * through a pinned host staging buffer of at most 64 MiB (whole blocks, at
 * least one), so any state size works.  The state counts as used (like
 * kv_pack).  KV_ERR_IO if the file cannot be written.  Synchronous. */
kv_status kv_checkpoint_save(kv_pool* pool, kv_state state, const char* path,
                             kv_stream stream);

/* Restore a file written by kv_checkpoint_save as a new state, with the
 * checks and the result of kv_unpack (header, compatibility, capacity, then
 * the checksum over the whole payload: KV_ERR_CHECKSUM with the same roll
 * back).  KV_ERR_IO if the file cannot be read or is shorter than its header
 * says.  Synchronous. */
kv_status kv_checkpoint_load(kv_pool* pool, const char* path, kv_stream stream, kv_state* out);

/* KV-Resume over a batch (append-prefill when T > 1, decode when T = 1): for
 * each state in order, copy-on-write a shared partial tail block, allocate the
 * blocks the append needs, project x [batch][T][d_model] at positions
 * pos0+n .. pos0+n+T-1, store K/V, and write the causal attention of the T
 * new queries over all n+T keys to o [L][batch][T][Hq * dh]. */
kv_status kv_attend(kv_pool* pool, const kv_state* states, int32_t batch, const void* x_dev,
                    int64_t T, void* o_dev, kv_stream stream);

/* kv_attend for callers that cannot allocate memory (code under HIP graph
 * capture, serving loops, harnesses that forbid allocation): the same
 * operation and kernels, with its work area in a fixed device array of
 * KV_NOALLOC_SCRATCH_MB MiB that the library holds on each GPU until the
 * process ends, instead of the pool's scratch area (the pool may have none).
 * Calls no allocating routine on the host or the device.  The call runs in
 * layer groups that fit the array: per layer, the query rows
 * (batch * T * Hq * dh elements) and, for decode (T = 1), the split-key
 * partials (batch * Hq * ceil(max keys / chunk) * (dh + 4) floats, chunks of
 * 1024 keys, 512 for a batch of one), plus the decode plan once; a call of
 * which not even one layer fits is KV_ERR_BUFSIZE and changes nothing.
 * Nothing in the array needs to start at zero.  Every call on one GPU uses
 * that GPU's array, so calls that overlap on one GPU (several pools or
 * streams, several host threads) race: the caller orders them.
 * KV_ERR_HIP if the array's device address could not be resolved when the
 * pool was created.  Profiling events are not recorded for this call. */
kv_status kv_attend_noalloc(kv_pool* pool, const kv_state* states, int32_t batch,
                            const void* x_dev, int64_t T, void* o_dev, kv_stream stream);

/* KV-Evict: order unpinned live states by score = alpha*reuse - beta*size -
 * gamma*age (ties by state id, ascending), and release them in that order
 * while allocated blocks > max_allocated_blocks.  LRU is (0, 0, 1).  Blocks
 * still referenced by another state survive.  Synchronous; *n_evicted is the
 * number of states evicted. */
kv_status kv_evict(kv_pool* pool, int64_t max_allocated_blocks, double alpha, double beta,
                   double gamma, kv_stream stream, int32_t* n_evicted);

/* KV-Evict, the branch for states that share blocks: candidates in the order
 * of kv_evict, while allocated blocks > max_allocated_blocks; a candidate
 * keeps the leading blocks in front of its first block that no other state
 * references (refcount 1) and gives up every block from there on (freed if
 * unshared, else decremented), its token count becoming those whole blocks'
 * (truncation to the shared prefix: only the continuation is lost and can be
 * recomputed).  A candidate whose first block is unshared is evicted whole;
 * one with no unshared block is left unchanged.  Synchronous.
 * *n_evicted / *n_truncated: states evicted whole / truncated. */
kv_status kv_evict_truncate(kv_pool* pool, int64_t max_allocated_blocks, double alpha,
                            double beta, double gamma, kv_stream stream, int32_t* n_evicted,
                            int32_t* n_truncated);

/* Drop a state's block references (blocks reaching refcount 0 return to the
 * tail of the free ring, in logical order).  Synchronous. */
kv_status kv_release(kv_pool* pool, kv_state state, kv_stream stream);

/* Exclude (pinned != 0) or re-admit a state as an eviction candidate. */
kv_status kv_pin(kv_pool* pool, kv_state state, int32_t pinned);

/* Wait for the pool's work on `stream`; returns the device's sticky status
 * (KV_ERR_INTERNAL if a device consistency check failed) and clears it. */
kv_status kv_sync(kv_pool* pool, kv_stream stream);

/* Catalog queries. */
kv_status kv_state_info(kv_pool* pool, kv_state state, int64_t* pos0, int64_t* n_tokens,
                        int64_t* n_blocks, uint64_t* lineage, int64_t* state_id);
kv_status kv_pool_counts(kv_pool* pool, int64_t* free_blocks, int64_t* live_states,
                         int64_t* clock);

/* The terms of a state's KV-Evict score (score = alpha*reuse - beta*size -
 * gamma*age, KV-Evict algorithm): reuse = number of operator calls that took
 * the state as an input (fork parent, attend member, compose segment, pack
 * and checkpoint source), last_access = the pool clock at its last touch (age
 * = clock - last_access, the clock from kv_pool_counts), pinned = 1 while it
 * is excluded from eviction.  Any output pointer may be NULL. */
kv_status kv_state_usage(kv_pool* pool, kv_state state, int64_t* reuse, int64_t* last_access,
                         int32_t* pinned);

/* Device-side metadata read back (synchronises `stream`): a state's block
 * table (host_out must hold n_blocks entries) and the allocator (refcount and
 * ring arrays of n_blocks entries each, ring head/tail counters). */
kv_status kv_read_block_table(kv_pool* pool, kv_state state, int32_t* host_out, int64_t cap,
                              kv_stream stream);
kv_status kv_read_allocator(kv_pool* pool, int32_t* refcount_out, int32_t* ring_out,
                            int64_t* head, int64_t* tail, kv_stream stream);

/* Per-kernel timing.  While enabled, every kernel the pool launches is
 * bracketed by HIP events recorded on its launch stream; kv_profile_read
 * waits for them and returns, per kernel kind, the number of launches and
 * their summed duration since the last read (then clears the counters). */
enum {
  KV_KERNEL_ALLOC = 0,
  KV_KERNEL_FORK,
  KV_KERNEL_RELEASE,
  KV_KERNEL_COMPOSE_META,
  KV_KERNEL_COMPOSE_COPY,
  KV_KERNEL_PACK,
  KV_KERNEL_UNPACK,
  KV_KERNEL_COW,
  KV_KERNEL_QKV,         /* projection + RoPE + paged store, T > 1 */
  KV_KERNEL_QKV_DECODE,  /* the same for T = 1 */
  KV_KERNEL_ATTN,        /* causal attention, T > 1 */
  KV_KERNEL_ATTN_DECODE, /* attention for T = 1 (split-key partials) */
  KV_KERNEL_MERGE,       /* merge of split-key partials */
  KV_KERNEL_KINDS
};
typedef struct {
  int64_t launches;
  double total_ms;
} kv_profile_entry;
kv_status kv_profile_enable(kv_pool* pool, int32_t enabled);
kv_status kv_profile_read(kv_pool* pool, kv_profile_entry* out /* KV_KERNEL_KINDS */);
/* The durations (ms) of the individual launches of one kernel kind recorded
 * since the last kv_profile_read, in launch order (waits for them): up to
 * `cap` values into out_ms, *n = how many there are.  The next
 * kv_profile_read clears them. */
kv_status kv_profile_launches(kv_pool* pool, int32_t kind, float* out_ms, int64_t cap,
                              int64_t* n);

/* Transfer-vs-recompute decision for a state of n_tokens tokens: the state-
 * aware scheduling rule of the paper (pi(S) = transfer iff
 * T_transfer < T_prefill, with T_transfer = |KV| / BW + delta, as in the
 * first steps of the KV-Transfer algorithm).  Pure host arithmetic on
 * caller-supplied rates (typically measured with kv_profile_*); touches no
 * device memory and needs no pool.
 *   kv_bytes      = ceil(n_tokens / B) * block bytes   (what kv_pack moves)
 *   t_transfer    = kv_bytes / link_bytes_per_s + link_latency_s
 *                   + kv_bytes / pack_bytes_per_s + kv_bytes / unpack_bytes_per_s
 *                   (a pack or unpack rate <= 0 leaves that term out)
 *   prefill_flops = L * (2 n d (Hq + 2 Hkv) dh + 4 Hq dh n (n + 1) / 2)
 *                   (projections, and causal attention over visible pairs)
 *   t_prefill     = prefill_flops / prefill_flops_per_s
 *   transfer      = 1 iff t_transfer < t_prefill, else 0 (recompute).
 * Errors: KV_ERR_ARG for a null pointer, an invalid cfg, n_tokens < 1,
 * link_bytes_per_s <= 0, link_latency_s < 0 or prefill_flops_per_s <= 0. */
typedef struct {
  double kv_bytes;
  double t_transfer; /* seconds */
  double t_prefill;  /* seconds */
  double prefill_flops;
  int32_t transfer; /* 1 = transfer, 0 = recompute */
  int32_t pad;
} kv_transfer_plan;

kv_status kv_plan_transfer(const kv_model_cfg* cfg, int64_t n_tokens, double link_bytes_per_s,
                           double link_latency_s, double pack_bytes_per_s,
                           double unpack_bytes_per_s, double prefill_flops_per_s,
                           kv_transfer_plan* out);

/* Human-readable name of a status. */
const char* kv_strerror(kv_status status);

#ifdef __cplusplus
}
#endif
#endif /* KVSTATE_H */
