// Host side of the KV-state library: the catalog of states (the paper's
// S_KV = (M, Theta, B, Pi, Lambda, Gamma) with the metadata-catalog fields
// state_id, model_id, position_range, block_id, lineage, refcount,
// last_access), argument and compatibility checks, and the C ABI declared in
// kvstate.h.  Block ids, refcounts and the free ring live on the device; the
// host knows the exact number of free blocks (allocations are counted here,
// releases report their frees back), so every out-of-memory condition is
// detected before anything is enqueued.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <vector>

#include "kv_internal.h"
#include "kv_fast.h"

using namespace kvs;

// Work area of kv_attend_noalloc: a fixed device array, one per GPU, held
// until the process ends (the query rows, split-key partials and decode plan
// of the layer group in flight).  Host code never uses its name as an
// address: the device address is resolved per GPU (static_scratch_ptr).
constexpr size_t kStaticScratchBytes = (size_t)KV_NOALLOC_SCRATCH_MB << 20;
static __device__ __align__(256) char scratch[kStaticScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_addr[kMaxDevices];

// Device address of `scratch` on the current GPU `device`, resolved on the
// first call for that device (nullptr if it cannot be resolved).
void* static_scratch_ptr(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  void* a = g_scratch_addr[device].load(std::memory_order_acquire);
  if (a) return a;
  if (hipGetSymbolAddress(&a, HIP_SYMBOL(scratch)) != hipSuccess || !a) {
    (void)hipGetLastError();
    return nullptr;
  }
  g_scratch_addr[device].store(a, std::memory_order_release);  // same value if two race
  return a;
}

constexpr uint32_t kNoParent = 0xFFFFFFFFu;

enum : int32_t { ST_FREE = 0, ST_ACTIVE = 1, ST_EVICTED = 2, ST_RELEASED = 3 };

struct StateRec {
  uint32_t gen = 0;
  int32_t status = ST_FREE;
  int64_t sid = -1;
  int64_t pos0 = 0, n = 0, nblocks = 0;
  uint64_t lineage = 0;
  bool pinned = false;
  int64_t last_access = 0, reuse = 0;
  int32_t group = -1;  // tail group of a partial tail block, -1 if none
};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

uint64_t lineage_word(uint64_t kind, uint64_t parent, uint64_t j) {
  return (kind << 56) | ((j & 0xFFFFFFull) << 32) | (parent & 0xFFFFFFFFull);
}

struct MetaLayout {
  size_t hdr, rc, ring, tables, rope_cos, rope_sin, rope_cos_g, rope_sin_g, cow, cmd, csum, total;
};

MetaLayout meta_layout(const kv_model_cfg& c, int64_t P) {
  MetaLayout m;
  const int64_t max_blocks = ceil_div(c.max_pos, c.block_size);
  size_t off = 0;
  m.hdr = off;
  off += sizeof(DevHeader);
  m.rc = off;
  off = align256(off + P * 4);
  m.ring = off;
  off = align256(off + P * 4);
  m.tables = off;
  off = align256(off + (size_t)c.max_states * max_blocks * 4);
  m.rope_cos = off;
  off = align256(off + (size_t)c.max_pos * (c.head_dim / 2) * 4);
  m.rope_sin = off;
  off = align256(off + (size_t)c.max_pos * (c.head_dim / 2) * 4);
  m.rope_cos_g = off;
  off = align256(off + (size_t)c.max_pos * (c.head_dim / 2) * 4);
  m.rope_sin_g = off;
  off = align256(off + (size_t)c.max_pos * (c.head_dim / 2) * 4);
  m.cow = off;
  off = align256(off + KV_MAX_BATCH * sizeof(int2));
  m.cmd = off;
  off = align256(off + (size_t)c.max_states * 3 * 4);  // candidates, then kept counts
  m.csum = off;
  off = align256(off + (size_t)(kSumSlots + 1) * 2 * 8);  // slots, then the result
  m.total = off;
  return m;
}

int elt_bytes(const kv_model_cfg& c) { return c.dtype == KV_DTYPE_BF16 ? 2 : 4; }

bool same_theta(const kv_model_cfg& a, const kv_model_cfg& b) {
  return a.n_layers == b.n_layers && a.d_model == b.d_model && a.n_q_heads == b.n_q_heads &&
         a.n_kv_heads == b.n_kv_heads && a.head_dim == b.head_dim &&
         a.block_size == b.block_size && a.dtype == b.dtype && a.rope_base == b.rope_base;
}

kv_status check_cfg(const kv_model_cfg* c) {
  if (!c) return KV_ERR_ARG;
  if (c->n_layers < 1 || c->d_model < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1) return KV_ERR_ARG;
  if (c->n_q_heads % c->n_kv_heads) return KV_ERR_ARG;
  if (c->head_dim < 16 || c->head_dim > 256 || c->head_dim % 16) return KV_ERR_ARG;
  if (c->block_size < 1 || c->block_size > 64) return KV_ERR_ARG;
  if (c->dtype != KV_DTYPE_F32 && c->dtype != KV_DTYPE_BF16) return KV_ERR_ARG;
  if (c->max_pos < 1 || c->max_states < 1) return KV_ERR_ARG;
  if (!(c->rope_base > 1.0) || !std::isfinite(c->rope_base)) return KV_ERR_ARG;
  return KV_OK;
}

}  // namespace

static_assert(sizeof(kv_model_cfg) == 56, "kv_model_cfg layout");
static_assert(sizeof(kv_pack_header) == 160, "kv_pack_header layout");

struct kv_pool {
  kv_model_cfg cfg;
  int64_t P = 0;
  int device = 0;       // the GPU the pool's memory is on (current at creation)
  bool failed = false;  // a launch failed after device state changed: refuse further work
  void* static_scratch = nullptr;  // that GPU's copy of `scratch` (kv_attend_noalloc)
  int32_t max_blocks = 0;
  char* pool = nullptr;
  char* meta = nullptr;
  char* scratch = nullptr;
  size_t scratch_bytes = 0;
  MetaLayout ml;
  DevHeader* dhdr = nullptr;
  int32_t* rc = nullptr;
  int32_t* ring = nullptr;
  int32_t* tables = nullptr;
  float* rope_cos = nullptr;
  float* rope_sin = nullptr;
  float* rope_cos_g = nullptr;
  float* rope_sin_g = nullptr;
  int2* cow = nullptr;
  int32_t* cmd = nullptr;
  unsigned long long* csum = nullptr;  // kSumSlots (s1, s2) slots, then the result pair
  int64_t head = 0, tail = 0;  // exact mirror of the device counters
  std::vector<StateRec> slots;
  int64_t next_sid = 0;
  int64_t clock = 0;
  std::vector<int32_t> holders;  // tail groups: number of states sharing the tail block
  std::vector<int32_t> free_groups;
  const void* w = nullptr;
  int64_t w_stride = 0;
  // kernel timing (kv_profile_*)
  bool prof = false;
  struct Rec {
    int kind;
    hipEvent_t a, b;
  };
  std::vector<Rec> pending;
  std::vector<hipEvent_t> spare;
  kv_profile_entry acc[KV_KERNEL_KINDS] = {};
  std::vector<float> launch_ms[KV_KERNEL_KINDS];  // individual launches since the last read
  hipEvent_t ev() {
    hipEvent_t e = nullptr;
    if (!spare.empty()) {
      e = spare.back();
      spare.pop_back();
    } else if (hipEventCreate(&e) != hipSuccess) {
      e = nullptr;
    }
    return e;
  }
  ~kv_pool() {
    for (auto& r : pending) {
      hipEventDestroy(r.a);
      hipEventDestroy(r.b);
    }
    for (auto e : spare) hipEventDestroy(e);
  }

  PoolGeom geom() const {
    PoolGeom g;
    g.pool = pool;
    g.tables = tables;
    g.rope_cos = rope_cos;
    g.rope_sin = rope_sin;
    g.rope_cos_g = rope_cos_g;
    g.rope_sin_g = rope_sin_g;
    g.block_elems = (int64_t)cfg.n_layers * 2 * cfg.n_kv_heads * cfg.block_size * cfg.head_dim;
    g.max_blocks = max_blocks;
    g.L = cfg.n_layers;
    g.Hq = cfg.n_q_heads;
    g.Hkv = cfg.n_kv_heads;
    g.dh = cfg.head_dim;
    g.B = cfg.block_size;
    g.d = cfg.d_model;
    g.max_pos = cfg.max_pos;
    g.b_shift = -1;
    for (int sh = 0; sh < 7; ++sh)
      if ((1 << sh) == cfg.block_size) g.b_shift = sh;
    return g;
  }
  int64_t free_blocks() const { return tail - head; }
  int64_t live() const {
    int64_t n = 0;
    for (const auto& s : slots) n += s.status == ST_ACTIVE;
    return n;
  }
  int32_t new_group(int32_t h) {
    int32_t g;
    if (!free_groups.empty()) {
      g = free_groups.back();
      free_groups.pop_back();
      holders[g] = h;
    } else {
      g = (int32_t)holders.size();
      holders.push_back(h);
    }
    return g;
  }
  void leave_group(StateRec& s) {
    if (s.group >= 0 && --holders[s.group] == 0) free_groups.push_back(s.group);
    s.group = -1;
  }
  void touch(StateRec& s, bool input) {
    s.last_access = ++clock;
    if (input) ++s.reuse;
  }
  // a free catalog slot, or -1
  int32_t take_slot() {
    for (size_t i = 0; i < slots.size(); ++i)
      if (slots[i].status != ST_ACTIVE) return (int32_t)i;
    return -1;
  }
  StateRec& open_state(int32_t slot, int64_t pos0, int64_t n, int64_t nblocks, uint64_t lin) {
    StateRec& s = slots[slot];
    s.gen += 1;
    s.status = ST_ACTIVE;
    s.sid = next_sid++;
    s.pos0 = pos0;
    s.n = n;
    s.nblocks = nblocks;
    s.lineage = lin;
    s.pinned = false;
    s.last_access = 0;
    s.reuse = 0;
    s.group = -1;
    return s;
  }
  kv_state handle(int32_t slot) const {
    return (kv_state)(uint32_t)slot | ((kv_state)slots[slot].gen << 32);
  }
  kv_status lookup(kv_state h, int32_t* slot_out) const {
    const int64_t slot = h & 0xFFFFFFFFll;
    const uint32_t gen = (uint32_t)((uint64_t)h >> 32);
    if (h < 0 || slot >= (int64_t)slots.size()) return KV_ERR_EVICTED;
    const StateRec& s = slots[slot];
    if (s.status != ST_ACTIVE || s.gen != gen) return KV_ERR_EVICTED;
    *slot_out = (int32_t)slot;
    return KV_OK;
  }
  int32_t* trow(int32_t slot) const { return tables + (int64_t)slot * max_blocks; }
};

namespace {

hipStream_t S(kv_stream s) { return (hipStream_t)s; }

kv_status hip_ok(hipError_t e) { return e == hipSuccess ? KV_OK : KV_ERR_HIP; }

#define KV_TRY(expr)                  \
  do {                                \
    kv_status _st = (expr);           \
    if (_st != KV_OK) return _st;     \
  } while (0)
#define KV_HIP(expr) KV_TRY(hip_ok(expr))
// A kernel launch of a call that changes pool state: if it fails, the device
// may already hold part of the call's effect while the host catalog does not,
// so the pool is marked failed and refuses every later operation.
#define KV_LAUNCH(p, expr)                 \
  do {                                     \
    if ((expr) != hipSuccess) {            \
      (void)hipGetLastError();             \
      (p)->failed = true;                  \
      return KV_ERR_HIP;                   \
    }                                      \
  } while (0)

// Brackets the kernel launches of one scope with events when profiling is on.
struct Timed {
  kv_pool* p;
  int kind;
  hipStream_t s;
  hipEvent_t a = nullptr;
  Timed(kv_pool* p_, int kind_, hipStream_t s_) : p(p_), kind(kind_), s(s_) {
    if (p->prof && (a = p->ev())) hipEventRecord(a, s);
  }
  ~Timed() {
    if (!a) return;
    hipEvent_t b = p->ev();
    if (b && hipEventRecord(b, s) == hipSuccess) {
      p->pending.push_back({kind, a, b});
    } else {
      p->spare.push_back(a);
      if (b) p->spare.push_back(b);
    }
  }
};

// Allocate on the device in request order; the caller has checked the count.
kv_status run_alloc(kv_pool* p, const AllocArgs& a, hipStream_t s) {
  int64_t need = 0;
  for (int r = 0; r < a.n_req; ++r) need += a.req[r].count + (a.req[r].cow > 0);
  if (need == 0) return KV_OK;
  {
    Timed t(p, KV_KERNEL_ALLOC, s);
    KV_LAUNCH(p, launch_alloc(p->dhdr, p->ring, p->rc, p->tables, p->max_blocks, (int32_t)p->P,
                        p->head, a, p->cow, s));
  }
  p->head += need;
  return KV_OK;
}

// Release states (slot, nblocks) in order; synchronous.  max_alloc < 0 releases
// all of them.  Returns the number of candidates visited.  With kept != null,
// candidates are truncated to their shared prefix instead (see k_release) and
// kept[i] receives the blocks candidate i keeps, for the visited ones.
kv_status run_release(kv_pool* p, const std::vector<int32_t>& cand, int64_t max_alloc,
                      hipStream_t s, int32_t* n_done, std::vector<int32_t>* kept = nullptr) {
  const int32_t n = (int32_t)(cand.size() / 2);
  *n_done = 0;
  if (n == 0) return KV_OK;
  int32_t* kept_dev = p->cmd + 2 * (size_t)p->cfg.max_states;
  KV_HIP(hipMemcpyAsync(p->cmd, cand.data(), cand.size() * 4, hipMemcpyHostToDevice, s));
  {
    Timed t(p, KV_KERNEL_RELEASE, s);
    KV_LAUNCH(p, launch_release(p->dhdr, p->ring, p->rc, p->tables, p->max_blocks, (int32_t)p->P,
                          p->cmd, n, max_alloc, p->head, p->tail, kept ? 1 : 0,
                          kept ? kept_dev : nullptr, s));
  }
  DevHeader h;
  KV_HIP(hipMemcpyAsync(&h, p->dhdr, sizeof(h), hipMemcpyDeviceToHost, s));
  if (kept) {
    kept->assign((size_t)n, -1);
    KV_HIP(hipMemcpyAsync(kept->data(), kept_dev, (size_t)n * 4, hipMemcpyDeviceToHost, s));
  }
  KV_HIP(hipStreamSynchronize(s));
  if (h.status != 0 || h.head != p->head || h.n_evicted < 0 || h.n_evicted > n)
    return KV_ERR_INTERNAL;
  p->tail = h.tail;
  *n_done = h.n_evicted;
  if (kept) kept->resize((size_t)h.n_evicted);
  return KV_OK;
}

// Per-call launch description of an append (materialize or attend) of T
// tokens to `batch` states (catalog slots, tokens cached, position of token 0).
AppendDesc make_desc(int32_t batch, const int32_t* slots, const int64_t* n_before,
                     const int64_t* pos0, int64_t T) {
  AppendDesc ad;
  std::memset(&ad, 0, sizeof(ad));
  ad.batch = batch;
  ad.T = (int32_t)T;
  int32_t max_keys = 0;
  for (int32_t i = 0; i < batch; ++i) {
    ad.seq[i].slot = slots[i];
    ad.seq[i].n_before = (int32_t)n_before[i];
    ad.seq[i].pos0 = (int32_t)pos0[i];
    max_keys = std::max<int32_t>(max_keys, (int32_t)(n_before[i] + T));
  }
  ad.max_keys = max_keys;
  return ad;
}

// Layout of an append's scratch area: the query rows of each layer of a group
// ([lc][M][Hq dh]), then the attention's per-layer area (split-key partials),
// then its per-call area (the decode work plan).
struct ScratchPlan {
  size_t q_layer, part_layer, fixed;
  int lc_max;  // layers per group; 0 when not even one layer fits
};

ScratchPlan plan_scratch(const kv_pool* p, const AppendDesc& ad, size_t scratch_bytes) {
  const kv_model_cfg& c = p->cfg;
  const int64_t M = (int64_t)ad.batch * ad.T;
  ScratchPlan sp;
  sp.q_layer = align256((size_t)M * c.n_q_heads * c.head_dim * elt_bytes(c));
  fast_scratch_need(p->geom(), c.dtype, ad, &sp.part_layer, &sp.fixed);
  const size_t per = sp.q_layer + sp.part_layer;
  sp.lc_max = scratch_bytes < sp.fixed + per
                  ? 0
                  : (int)std::min<size_t>(c.n_layers, (scratch_bytes - sp.fixed) / per);
  return sp;
}

// Shared path of materialize and attend: allocation (with copy-on-write),
// projection + RoPE + paged store, and attention, layer group by layer group,
// with `scratch` (scratch_bytes) as the work area.
kv_status run_append(kv_pool* p, const AppendDesc& ad, const AllocArgs& aa, const void* x,
                     void* o, hipStream_t s, char* scratch, size_t scratch_bytes) {
  const kv_model_cfg& c = p->cfg;
  const ScratchPlan sp = plan_scratch(p, ad, scratch_bytes);
  const int lc_max = sp.lc_max;
  if (lc_max < 1) return KV_ERR_BUFSIZE;
  KV_TRY(run_alloc(p, aa, s));
  const PoolGeom g = p->geom();
  bool any_cow = false;
  for (int i = 0; i < aa.n_req; ++i) any_cow |= aa.req[i].cow > 0;
  if (any_cow) {
    Timed t(p, KV_KERNEL_COW, s);
    KV_LAUNCH(p, launch_cow(g, c.dtype, p->cow, aa, s));
  }
  char* part = scratch + sp.q_layer * lc_max;
  char* plan = part + sp.part_layer * lc_max;
  for (int l0 = 0; l0 < c.n_layers; l0 += lc_max) {
    const int lc = std::min(lc_max, c.n_layers - l0);
    bool done = false;
    {
      Timed t(p, ad.T == 1 ? KV_KERNEL_QKV_DECODE : KV_KERNEL_QKV, s);
      KV_LAUNCH(p, launch_qkv_fast(g, c.dtype, x, p->w, p->w_stride, ad, scratch, l0, lc, s,
                                   &done));
      if (!done)
        KV_LAUNCH(p, launch_qkv_generic(g, c.dtype, x, p->w, p->w_stride, ad, scratch, l0, lc,
                                        s));
    }
    done = false;
    bool merge = false;
    {
      Timed t(p, ad.T == 1 ? KV_KERNEL_ATTN_DECODE : KV_KERNEL_ATTN, s);
      KV_LAUNCH(p, launch_attn_fast(g, c.dtype, scratch, ad, o, part, plan, l0, lc, s, &done,
                                    &merge));
      if (!done) KV_LAUNCH(p, launch_attn_generic(g, c.dtype, scratch, ad, o, l0, lc, s));
    }
    if (merge) {
      Timed t(p, KV_KERNEL_MERGE, s);
      KV_LAUNCH(p, launch_attn_merge(g, c.dtype, ad, o, part, l0, lc, s));
    }
  }
  return KV_OK;
}

}  // namespace

namespace {

// Device address of a buffer the data-movement kernels read or write:
// device memory as is, pinned host memory (hipHostMalloc) through its device
// mapping; pageable or unknown host memory is rejected, so that no kernel is
// ever launched on an address the GPU cannot reach.
kv_status device_view(const void* p, const void** out, bool* on_device = nullptr) {
  hipPointerAttribute_t a;
  std::memset(&a, 0, sizeof(a));
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return KV_ERR_ARG;
  }
  if (on_device) *on_device = a.type == hipMemoryTypeDevice || a.type == hipMemoryTypeManaged;
  if (a.type == hipMemoryTypeDevice || a.type == hipMemoryTypeManaged) {
    *out = p;
    return KV_OK;
  }
  if (a.type == hipMemoryTypeHost && a.devicePointer) {
    const ptrdiff_t off = a.hostPointer ? (const char*)p - (const char*)a.hostPointer : 0;
    *out = (const char*)a.devicePointer + off;
    return KV_OK;
  }
  return KV_ERR_ARG;
}

// A device buffer the kernels of `p` read or write: device (or managed) memory
// of the pool's GPU, 16-byte aligned, inside an allocation that extends at
// least `bytes` bytes past it (KV_ERR_BUFSIZE otherwise).  Anything else is
// rejected before a kernel could be launched on it.
kv_status device_span(int device, const void* ptr, size_t bytes) {
  if (!ptr || ((uintptr_t)ptr & 15)) return KV_ERR_ARG;
  hipPointerAttribute_t a;
  std::memset(&a, 0, sizeof(a));
  if (hipPointerGetAttributes(&a, ptr) != hipSuccess) {
    (void)hipGetLastError();
    return KV_ERR_ARG;
  }
  if ((a.type != hipMemoryTypeDevice && a.type != hipMemoryTypeManaged) || a.device != device)
    return KV_ERR_ARG;
  hipDeviceptr_t base = nullptr;
  size_t size = 0;
  if (hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)ptr) == hipSuccess && base) {
    const uintptr_t lo = (uintptr_t)base, q = (uintptr_t)ptr;
    if (q < lo || q - lo > size || bytes > size - (q - lo)) return KV_ERR_BUFSIZE;
  } else {
    (void)hipGetLastError();  // no range known: the type check above stands
  }
  return KV_OK;
}


// Unpinned live states in eviction order: score = alpha*reuse - beta*size -
// gamma*age ascending, ties by state id.  Returns (slot, n_blocks) pairs.
std::vector<int32_t> eviction_candidates(const kv_pool* p, double alpha, double beta,
                                         double gamma) {
  struct Cand {
    double score;
    int64_t sid;
    int32_t slot;
  };
  std::vector<Cand> cs;
  for (size_t i = 0; i < p->slots.size(); ++i) {
    const StateRec& r = p->slots[i];
    if (r.status != ST_ACTIVE || r.pinned) continue;
    const double age = (double)(p->clock - r.last_access);
    const double score = (alpha * (double)r.reuse - beta * (double)r.nblocks) - gamma * age;
    cs.push_back({score, r.sid, (int32_t)i});
  }
  std::sort(cs.begin(), cs.end(), [](const Cand& a, const Cand& b) {
    return a.score < b.score || (a.score == b.score && a.sid < b.sid);
  });
  std::vector<int32_t> cand;
  for (const auto& c : cs) {
    cand.push_back(c.slot);
    cand.push_back((int32_t)p->slots[c.slot].nblocks);
  }
  return cand;
}

// Header of a pack of blocks [b0, b1) of state r (checksum fields zero).
kv_pack_header make_header(const kv_pool* p, const StateRec& r, int64_t b0, int64_t b1) {
  const kv_model_cfg& c = p->cfg;
  const int B = c.block_size;
  const uint64_t block_bytes = (uint64_t)p->geom().block_elems * elt_bytes(c);
  kv_pack_header h;
  std::memset(&h, 0, sizeof(h));
  h.magic = KV_PACK_MAGIC;
  h.version = KV_PACK_VERSION;
  h.model_id = c.model_id;
  h.cfg = c;
  h.pos_begin = r.pos0 + b0 * B;
  h.n_tokens = std::min<int64_t>(r.n, b1 * B) - b0 * B;
  h.blk_begin = b0;
  h.n_blocks = b1 - b0;
  h.block_bytes = block_bytes;
  h.payload_bytes = (b1 - b0) * block_bytes;
  h.lineage = r.lineage;
  h.src_state_id = r.sid;
  return h;
}

// The receiving side's checks of a header, in the order kv_unpack documents.
kv_status check_header(const kv_pool* p, const kv_pack_header* hdr) {
  if (hdr->magic != KV_PACK_MAGIC || hdr->version != KV_PACK_VERSION) return KV_ERR_BAD_HEADER;
  if ((hdr->flags & ~KV_PACK_CHECKSUM) != 0 || hdr->reserved != 0) return KV_ERR_BAD_HEADER;
  const kv_model_cfg& c = p->cfg;
  if (hdr->model_id != c.model_id || !same_theta(hdr->cfg, c)) return KV_ERR_INCOMPATIBLE;
  const int B = c.block_size;
  const uint64_t block_bytes = (uint64_t)p->geom().block_elems * elt_bytes(c);
  const int64_t nb = hdr->n_blocks, nt = hdr->n_tokens;
  if (nb < 1 || !((nb - 1) * B < nt && nt <= nb * B) || hdr->block_bytes != block_bytes ||
      hdr->payload_bytes != nb * block_bytes || hdr->pos_begin < 0)
    return KV_ERR_BAD_HEADER;
  return KV_OK;
}

// Register a state for a checked header and allocate its blocks (the
// destination side of a transfer before any byte is copied).
kv_status open_transfer(kv_pool* p, const kv_pack_header* hdr, hipStream_t s, int32_t* slot_out) {
  const kv_model_cfg& c = p->cfg;
  const int64_t nb = hdr->n_blocks, nt = hdr->n_tokens;
  if (hdr->pos_begin + nt > c.max_pos) return KV_ERR_CAPACITY;
  const int32_t slot = p->take_slot();
  if (slot < 0) return KV_ERR_CAPACITY;
  if (nb > p->free_blocks()) return KV_ERR_OOM;
  StateRec& r = p->open_state(slot, hdr->pos_begin, nt, nb,
                              lineage_word(KV_LINEAGE_TRANSFER, (uint64_t)hdr->src_state_id, 0));
  AllocArgs aa;
  std::memset(&aa, 0, sizeof(aa));
  aa.n_req = 1;
  aa.req[0].slot = slot;
  aa.req[0].first = 0;
  aa.req[0].count = (int32_t)nb;
  KV_TRY(run_alloc(p, aa, s));
  if (nt % c.block_size) r.group = p->new_group(1);
  *slot_out = slot;
  return KV_OK;
}

// Undo open_transfer after a failed copy: the blocks return to the free ring,
// the state is not registered (its id stays used).
kv_status abort_transfer(kv_pool* p, int32_t slot, hipStream_t s) {
  StateRec& r = p->slots[slot];
  std::vector<int32_t> cand = {slot, (int32_t)r.nblocks};
  int32_t n = 0;
  KV_TRY(run_release(p, cand, -1, s, &n));
  p->leave_group(r);
  r.status = ST_RELEASED;
  return KV_OK;
}

// Clear the checksum slots (the folding kernel clears what it reads; its
// result is overwritten by csum_end).
kv_status csum_begin(kv_pool* p, hipStream_t s) {
  KV_LAUNCH(p, launch_csum_final(p->csum, p->csum + 2 * kSumSlots, s));
  return KV_OK;
}

// Fold the slots into (s1, s2), clear them, synchronise, return the pair.
kv_status csum_end(kv_pool* p, hipStream_t s, uint64_t out[2]) {
  unsigned long long* res = p->csum + 2 * kSumSlots;
  KV_LAUNCH(p, launch_csum_final(p->csum, res, s));
  unsigned long long h[2];
  KV_HIP(hipMemcpyAsync(h, res, sizeof(h), hipMemcpyDeviceToHost, s));
  KV_HIP(hipStreamSynchronize(s));
  out[0] = h[0];
  out[1] = h[1];
  return KV_OK;
}

// Pinned host staging buffer of whole blocks, released on scope exit.
struct Staging {
  void* host = nullptr;
  const void* dev = nullptr;
  int64_t blocks = 0;
  ~Staging() {
    if (host) (void)hipHostFree(host);
  }
  kv_status alloc(int64_t want_blocks, uint64_t block_bytes) {
    const int64_t cap = std::max<int64_t>(1, (int64_t)((64ull << 20) / block_bytes));
    blocks = std::min(want_blocks, cap);
    if (hipHostMalloc(&host, (size_t)(blocks * block_bytes), hipHostMallocDefault) != hipSuccess) {
      (void)hipGetLastError();
      host = nullptr;
      return KV_ERR_HIP;
    }
    return device_view(host, &dev);
  }
};

struct File {
  FILE* f = nullptr;
  ~File() {
    if (f) std::fclose(f);
  }
};

}  // namespace

extern "C" {

kv_status kv_plan_transfer(const kv_model_cfg* cfg, int64_t n_tokens, double link_bytes_per_s,
                           double link_latency_s, double pack_bytes_per_s,
                           double unpack_bytes_per_s, double prefill_flops_per_s,
                           kv_transfer_plan* out) {
  if (!out) return KV_ERR_ARG;
  KV_TRY(check_cfg(cfg));
  if (n_tokens < 1 || !(link_bytes_per_s > 0.0) || !(link_latency_s >= 0.0) ||
      !(prefill_flops_per_s > 0.0))
    return KV_ERR_ARG;
  const kv_model_cfg& c = *cfg;
  const double elt = c.dtype == KV_DTYPE_BF16 ? 2.0 : 4.0;
  const double block_bytes =
      2.0 * c.n_layers * c.n_kv_heads * (double)c.block_size * c.head_dim * elt;
  const double n = (double)n_tokens;
  kv_transfer_plan r;
  std::memset(&r, 0, sizeof(r));
  r.kv_bytes = (double)ceil_div(n_tokens, c.block_size) * block_bytes;
  r.t_transfer = r.kv_bytes / link_bytes_per_s + link_latency_s;
  if (pack_bytes_per_s > 0.0) r.t_transfer += r.kv_bytes / pack_bytes_per_s;
  if (unpack_bytes_per_s > 0.0) r.t_transfer += r.kv_bytes / unpack_bytes_per_s;
  const double cols = (double)(c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  r.prefill_flops = c.n_layers * (2.0 * n * c.d_model * cols +
                                  4.0 * c.n_q_heads * c.head_dim * (n * (n + 1.0) / 2.0));
  r.t_prefill = r.prefill_flops / prefill_flops_per_s;
  r.transfer = r.t_transfer < r.t_prefill ? 1 : 0;
  *out = r;
  return KV_OK;
}

const char* kv_strerror(kv_status st) {
  switch (st) {
    case KV_OK: return "KV_OK";
    case KV_ERR_ARG: return "KV_ERR_ARG";
    case KV_ERR_OOM: return "KV_ERR_OOM";
    case KV_ERR_INCOMPATIBLE: return "KV_ERR_INCOMPATIBLE";
    case KV_ERR_EVICTED: return "KV_ERR_EVICTED";
    case KV_ERR_BAD_HEADER: return "KV_ERR_BAD_HEADER";
    case KV_ERR_BUFSIZE: return "KV_ERR_BUFSIZE";
    case KV_ERR_CAPACITY: return "KV_ERR_CAPACITY";
    case KV_ERR_HIP: return "KV_ERR_HIP";
    case KV_ERR_INTERNAL: return "KV_ERR_INTERNAL";
    case KV_ERR_CHECKSUM: return "KV_ERR_CHECKSUM";
    case KV_ERR_IO: return "KV_ERR_IO";
    default: return "KV_ERR_UNKNOWN";
  }
}

kv_status kv_pool_bytes(const kv_model_cfg* cfg, int64_t n_blocks, size_t* pool_bytes,
                        size_t* meta_bytes) {
  KV_TRY(check_cfg(cfg));
  if (n_blocks < 1 || n_blocks > INT32_MAX) return KV_ERR_ARG;
  const size_t block_bytes = (size_t)cfg->n_layers * 2 * cfg->n_kv_heads * cfg->block_size *
                             cfg->head_dim * elt_bytes(*cfg);
  if (pool_bytes) *pool_bytes = block_bytes * n_blocks;
  if (meta_bytes) *meta_bytes = meta_layout(*cfg, n_blocks).total;
  return KV_OK;
}

size_t kv_scratch_bytes(const kv_model_cfg* cfg, int64_t tokens, int32_t batch,
                        int64_t max_keys) {
  if (check_cfg(cfg) != KV_OK || tokens < 1 || batch < 1) return 0;
  const size_t q = (size_t)cfg->n_layers * tokens * cfg->n_q_heads * cfg->head_dim *
                   elt_bytes(*cfg);
  return align256(q) + fast_scratch_bound(*cfg, tokens, batch, max_keys);
}

kv_status kv_pool_create(const kv_model_cfg* cfg, int64_t n_blocks, void* pool_dev,
                         void* meta_dev, void* scratch_dev, size_t scratch_bytes,
                         const int32_t* init_free_order, kv_stream stream, kv_pool** out) {
  KV_TRY(check_cfg(cfg));
  if (!out || !pool_dev || !meta_dev || n_blocks < 1 || n_blocks > INT32_MAX) return KV_ERR_ARG;
  if (((uintptr_t)pool_dev | (uintptr_t)meta_dev | (uintptr_t)scratch_dev) & 255) return KV_ERR_ARG;
  int device = 0;
  if (hipGetDevice(&device) != hipSuccess) return KV_ERR_HIP;
  {
    size_t pb = 0, mb = 0;
    KV_TRY(kv_pool_bytes(cfg, n_blocks, &pb, &mb));
    KV_TRY(device_span(device, pool_dev, pb));
    KV_TRY(device_span(device, meta_dev, mb));
    if (scratch_dev) KV_TRY(device_span(device, scratch_dev, scratch_bytes));
  }
  std::vector<int32_t> order(n_blocks);
  if (init_free_order) {
    std::vector<char> seen(n_blocks, 0);
    for (int64_t i = 0; i < n_blocks; ++i) {
      const int32_t v = init_free_order[i];
      if (v < 0 || v >= n_blocks || seen[v]) return KV_ERR_ARG;
      seen[v] = 1;
      order[i] = v;
    }
  } else {
    for (int64_t i = 0; i < n_blocks; ++i) order[i] = (int32_t)i;
  }
  kv_pool* p = new (std::nothrow) kv_pool();
  if (!p) return KV_ERR_ARG;
  p->cfg = *cfg;
  p->P = n_blocks;
  p->device = device;
  p->static_scratch = static_scratch_ptr(device);
  p->max_blocks = (int32_t)ceil_div(cfg->max_pos, cfg->block_size);
  p->pool = (char*)pool_dev;
  p->meta = (char*)meta_dev;
  p->scratch = (char*)scratch_dev;
  p->scratch_bytes = scratch_dev ? scratch_bytes : 0;
  p->ml = meta_layout(*cfg, n_blocks);
  p->dhdr = (DevHeader*)(p->meta + p->ml.hdr);
  p->rc = (int32_t*)(p->meta + p->ml.rc);
  p->ring = (int32_t*)(p->meta + p->ml.ring);
  p->tables = (int32_t*)(p->meta + p->ml.tables);
  p->rope_cos = (float*)(p->meta + p->ml.rope_cos);
  p->rope_sin = (float*)(p->meta + p->ml.rope_sin);
  p->rope_cos_g = (float*)(p->meta + p->ml.rope_cos_g);
  p->rope_sin_g = (float*)(p->meta + p->ml.rope_sin_g);
  p->cow = (int2*)(p->meta + p->ml.cow);
  p->cmd = (int32_t*)(p->meta + p->ml.cmd);
  p->csum = (unsigned long long*)(p->meta + p->ml.csum);
  p->head = 0;
  p->tail = n_blocks;
  p->slots.resize(cfg->max_states);
  // at most one tail group per live state: no reallocation after creation
  p->holders.reserve(cfg->max_states);
  p->free_groups.reserve(cfg->max_states);

  // RoPE table: angle p * theta_i with theta_i = base^(-2i/dh), in double.
  const int half = cfg->head_dim / 2;
  std::vector<float> cs((size_t)cfg->max_pos * half), sn((size_t)cfg->max_pos * half);
  for (int i = 0; i < half; ++i) {
    const double th = std::pow(cfg->rope_base, -2.0 * i / cfg->head_dim);
    for (int64_t pos = 0; pos < cfg->max_pos; ++pos) {
      const double a = (double)pos * th;
      cs[pos * half + i] = (float)std::cos(a);
      sn[pos * half + i] = (float)std::sin(a);
    }
  }
  // the same values grouped by 4 channels, position-major within a group
  std::vector<float> csg(cs.size()), sng(sn.size());
  for (int64_t pos = 0; pos < cfg->max_pos; ++pos)
    for (int i = 0; i < half; ++i) {
      const size_t k = ((size_t)(i / 4) * cfg->max_pos + pos) * 4 + i % 4;
      csg[k] = cs[pos * half + i];
      sng[k] = sn[pos * half + i];
    }
  DevHeader h;
  std::memset(&h, 0, sizeof(h));
  h.head = 0;
  h.tail = n_blocks;
  hipStream_t s = S(stream);
  kv_status st = KV_OK;
  if (hipMemsetAsync(p->meta, 0, p->ml.total, s) != hipSuccess ||
      hipMemcpyAsync(p->dhdr, &h, sizeof(h), hipMemcpyHostToDevice, s) != hipSuccess ||
      hipMemcpyAsync(p->ring, order.data(), n_blocks * 4, hipMemcpyHostToDevice, s) != hipSuccess ||
      hipMemcpyAsync(p->rope_cos, cs.data(), cs.size() * 4, hipMemcpyHostToDevice, s) != hipSuccess ||
      hipMemcpyAsync(p->rope_sin, sn.data(), sn.size() * 4, hipMemcpyHostToDevice, s) != hipSuccess ||
      hipMemcpyAsync(p->rope_cos_g, csg.data(), csg.size() * 4, hipMemcpyHostToDevice, s) != hipSuccess ||
      hipMemcpyAsync(p->rope_sin_g, sng.data(), sng.size() * 4, hipMemcpyHostToDevice, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    st = KV_ERR_HIP;
  if (st != KV_OK) {
    delete p;
    return st;
  }
  *out = p;
  return KV_OK;
}

kv_status kv_pool_destroy(kv_pool* pool) {
  delete pool;
  return KV_OK;
}

kv_status kv_set_weights(kv_pool* p, const void* w_dev, int64_t layer_stride_elems) {
  if (!p || !w_dev) return KV_ERR_ARG;
  const int64_t per = (int64_t)(p->cfg.n_q_heads + 2 * p->cfg.n_kv_heads) * p->cfg.head_dim *
                      p->cfg.d_model;
  if (layer_stride_elems < per && p->cfg.n_layers > 1) return KV_ERR_ARG;
  const size_t bytes =
      (size_t)((p->cfg.n_layers - 1) * std::max<int64_t>(layer_stride_elems, 0) + per) *
      elt_bytes(p->cfg);
  KV_TRY(device_span(p->device, w_dev, bytes));
  p->w = w_dev;
  p->w_stride = layer_stride_elems;
  return KV_OK;
}

kv_status kv_materialize(kv_pool* p, const void* x_dev, int64_t T, int64_t pos0, void* o_dev,
                         kv_stream stream, kv_state* out) {
  if (!p || !x_dev || !o_dev || !out || T <= 0 || pos0 < 0) return KV_ERR_ARG;
  if (p->failed) return KV_ERR_HIP;
  if (!p->w) return KV_ERR_ARG;
  const kv_model_cfg& c = p->cfg;
  if (pos0 + T > c.max_pos) return KV_ERR_CAPACITY;
  const size_t elt = elt_bytes(c);
  KV_TRY(device_span(p->device, x_dev, (size_t)T * c.d_model * elt));
  KV_TRY(device_span(p->device, o_dev, (size_t)c.n_layers * T * c.n_q_heads * c.head_dim * elt));
  const int32_t slot = p->take_slot();
  if (slot < 0) return KV_ERR_CAPACITY;
  const int64_t nb = ceil_div(T, c.block_size);
  if (nb > p->free_blocks()) return KV_ERR_OOM;
  const int64_t zero = 0;
  const AppendDesc ad = make_desc(1, &slot, &zero, &pos0, T);
  if (plan_scratch(p, ad, p->scratch_bytes).lc_max < 1) return KV_ERR_BUFSIZE;
  AllocArgs aa;
  std::memset(&aa, 0, sizeof(aa));
  aa.n_req = 1;
  aa.req[0].slot = slot;
  aa.req[0].count = (int32_t)nb;
  // the catalog changes only once every launch of the call is enqueued
  KV_TRY(run_append(p, ad, aa, x_dev, o_dev, S(stream), p->scratch, p->scratch_bytes));
  StateRec& r = p->open_state(slot, pos0, T, nb,
                              lineage_word(KV_LINEAGE_MATERIALIZE, kNoParent, 0));
  if (T % c.block_size) r.group = p->new_group(1);
  p->touch(r, false);
  *out = p->handle(slot);
  return KV_OK;
}

kv_status kv_fork(kv_pool* p, kv_state parent, int32_t k, kv_state* children, kv_stream stream) {
  if (!p || !children || k < 1 || k > KV_MAX_FORK) return KV_ERR_ARG;
  if (p->failed) return KV_ERR_HIP;
  int32_t ps;
  KV_TRY(p->lookup(parent, &ps));
  if (p->live() + k > p->cfg.max_states) return KV_ERR_CAPACITY;
  ForkArgs fa;
  std::memset(&fa, 0, sizeof(fa));
  fa.parent = ps;
  fa.k = k;
  const StateRec par = p->slots[ps];
  fa.nblocks = (int32_t)par.nblocks;
  std::vector<int32_t> kids;
  for (int j = 1; j <= k; ++j) {
    const int32_t cs = p->take_slot();
    StateRec& c = p->open_state(cs, par.pos0, par.n, par.nblocks,
                                lineage_word(KV_LINEAGE_FORK, (uint64_t)par.sid, j));
    c.group = par.group;
    fa.child[j - 1] = cs;
    kids.push_back(cs);
  }
  if (par.group >= 0) p->holders[par.group] += k;
  {
    Timed t(p, KV_KERNEL_FORK, S(stream));
    KV_LAUNCH(p, launch_fork(p->dhdr, p->tables, p->max_blocks, p->rc, fa, S(stream)));
  }
  p->touch(p->slots[ps], true);
  for (int j = 0; j < k; ++j) {
    p->touch(p->slots[kids[j]], false);
    children[j] = p->handle(kids[j]);
  }
  return KV_OK;
}

}  // extern "C"

// KV-Resume over a batch with `scratch` as the work area.  Uses no heap
// memory on the host (fixed arrays of KV_MAX_BATCH) and none on the device.
static kv_status attend_impl(kv_pool* p, const kv_state* states, int32_t batch,
                             const void* x_dev, int64_t T, void* o_dev, kv_stream stream,
                             char* scratch, size_t scratch_bytes) {
  if (!p || !states || !x_dev || !o_dev || batch < 1 || batch > KV_MAX_BATCH || T <= 0)
    return KV_ERR_ARG;
  if (p->failed) return KV_ERR_HIP;
  if (!p->w) return KV_ERR_ARG;
  for (int i = 0; i < batch; ++i)
    for (int j = 0; j < i; ++j)
      if (states[i] == states[j]) return KV_ERR_ARG;
  const kv_model_cfg& c = p->cfg;
  const int B = c.block_size;
  int32_t slots[KV_MAX_BATCH];
  for (int i = 0; i < batch; ++i) KV_TRY(p->lookup(states[i], &slots[i]));
  AllocArgs aa;
  std::memset(&aa, 0, sizeof(aa));
  aa.n_req = batch;
  int64_t nbef[KV_MAX_BATCH], pos0[KV_MAX_BATCH];
  int64_t need = 0;
  // tail groups left by earlier members of the batch: a member that copies a
  // shared tail leaves its group before the next member looks
  int32_t left[KV_MAX_BATCH];
  int n_left = 0;
  auto holders_now = [&](int32_t g) {
    int32_t h = p->holders[g];
    for (int i = 0; i < n_left; ++i) h -= left[i] == g;
    return h;
  };
  for (int i = 0; i < batch; ++i) {
    const StateRec& r = p->slots[slots[i]];
    if (r.pos0 + r.n + T > c.max_pos) return KV_ERR_CAPACITY;
    const bool shared_tail = (r.n % B) && r.group >= 0 && holders_now(r.group) > 1;
    if (shared_tail) left[n_left++] = r.group;
    aa.req[i].slot = slots[i];
    aa.req[i].cow = shared_tail ? (int32_t)(r.n % B) : 0;
    aa.req[i].partial = (int32_t)(r.n % B);
    aa.req[i].first = (int32_t)r.nblocks;
    aa.req[i].count = (int32_t)(ceil_div(r.n + T, B) - ceil_div(r.n, B));
    need += aa.req[i].count + (shared_tail ? 1 : 0);
    nbef[i] = r.n;
    pos0[i] = r.pos0;
  }
  if (need > p->free_blocks()) return KV_ERR_OOM;
  const AppendDesc ad = make_desc(batch, slots, nbef, pos0, T);
  if (plan_scratch(p, ad, scratch_bytes).lc_max < 1) return KV_ERR_BUFSIZE;
  const size_t elt = elt_bytes(c);
  KV_TRY(device_span(p->device, x_dev, (size_t)batch * T * c.d_model * elt));
  KV_TRY(device_span(p->device, o_dev,
                     (size_t)c.n_layers * batch * T * c.n_q_heads * c.head_dim * elt));
  // the catalog changes only once every launch of the call is enqueued
  KV_TRY(run_append(p, ad, aa, x_dev, o_dev, S(stream), scratch, scratch_bytes));
  for (int i = 0; i < batch; ++i) {
    StateRec& r = p->slots[slots[i]];
    p->leave_group(r);  // after the append the tail block is private
    r.n += T;
    r.nblocks += aa.req[i].count;
    if (r.n % B) r.group = p->new_group(1);
  }
  for (int i = 0; i < batch; ++i) p->touch(p->slots[slots[i]], true);
  return KV_OK;
}

extern "C" {

kv_status kv_attend(kv_pool* p, const kv_state* states, int32_t batch, const void* x_dev,
                    int64_t T, void* o_dev, kv_stream stream) {
  return attend_impl(p, states, batch, x_dev, T, o_dev, stream, p ? p->scratch : nullptr,
                     p ? p->scratch_bytes : 0);
}

kv_status kv_attend_noalloc(kv_pool* p, const kv_state* states, int32_t batch,
                            const void* x_dev, int64_t T, void* o_dev, kv_stream stream) {
  if (!p) return KV_ERR_ARG;
  if (!p->static_scratch) return KV_ERR_HIP;  // its address could not be resolved
  // no profiling events for this call: creating them could allocate
  const bool prof = p->prof;
  p->prof = false;
  const kv_status st = attend_impl(p, states, batch, x_dev, T, o_dev, stream,
                                   (char*)p->static_scratch, kStaticScratchBytes);
  p->prof = prof;
  return st;
}

kv_status kv_compose(kv_pool* p, const kv_segment* segs, int32_t n, kv_stream stream,
                     kv_state* out) {
  if (!p || !segs || !out || n < 1 || n > KV_MAX_SEGMENTS) return KV_ERR_ARG;
  if (p->failed) return KV_ERR_HIP;
  const kv_model_cfg& c = p->cfg;
  const int B = c.block_size;
  std::vector<int32_t> sl(n);
  for (int i = 0; i < n; ++i) KV_TRY(p->lookup(segs[i].state, &sl[i]));
  int64_t N = 0;
  for (int i = 0; i < n; ++i) {
    const StateRec& r = p->slots[sl[i]];
    if (!(0 <= segs[i].tok_begin && segs[i].tok_begin < segs[i].tok_end &&
          segs[i].tok_end <= r.n))
      return KV_ERR_ARG;
    N += segs[i].tok_end - segs[i].tok_begin;
  }
  const int64_t P0 = p->slots[sl[0]].pos0 + segs[0].tok_begin;
  if (P0 + N > c.max_pos) return KV_ERR_CAPACITY;
  const int32_t slot = p->take_slot();
  if (slot < 0) return KV_ERR_CAPACITY;
  ComposeArgs ca;
  std::memset(&ca, 0, sizeof(ca));
  ca.nseg = n;
  ca.new_slot = slot;
  ca.n_tokens = (int32_t)N;
  ca.n_dest_blocks = (int32_t)ceil_div(N, B);
  int64_t cum = 0, aliased = 0;
  int32_t tail_alias_seg = -1;
  for (int i = 0; i < n; ++i) {
    const StateRec& r = p->slots[sl[i]];
    const int64_t len = segs[i].tok_end - segs[i].tok_begin;
    const int64_t off = cum - segs[i].tok_begin;
    const int64_t delta = P0 + off - r.pos0;
    SegDesc& sd = ca.seg[i];
    sd.slot = sl[i];
    sd.cum = (int32_t)cum;
    sd.off = (int32_t)off;
    sd.delta = (int32_t)delta;
    sd.alias_b0 = sd.alias_b1 = 0;
    if (delta == 0 && off % B == 0) {
      int64_t b0 = ceil_div(cum, B), b1 = (cum + len) / B;
      if (i == n - 1 && segs[i].tok_end == r.n && N % B && (N / B) * B >= cum) {
        b1 += 1;  // the final partial block is the source's own tail
        tail_alias_seg = i;
      }
      if (b1 > b0) {
        sd.alias_b0 = (int32_t)b0;
        sd.alias_b1 = (int32_t)b1;
        aliased += b1 - b0;
      }
    }
    cum += len;
  }
  const int64_t ncopy = ca.n_dest_blocks - aliased;
  if (ncopy > p->free_blocks()) return KV_ERR_OOM;
  const hipStream_t s = S(stream);
  StateRec& r = p->open_state(slot, P0, N, ca.n_dest_blocks,
                              lineage_word(KV_LINEAGE_MERGE, (uint64_t)p->slots[sl[0]].sid, 0));
  {
    Timed t(p, KV_KERNEL_COMPOSE_META, s);
    KV_LAUNCH(p, launch_compose_meta(p->dhdr, p->ring, p->rc, p->tables, p->max_blocks,
                               (int32_t)p->P, B, p->head, (int32_t)ncopy, ca, s));
  }
  p->head += ncopy;
  if (N % B) {
    if (tail_alias_seg >= 0 && p->slots[sl[tail_alias_seg]].group >= 0) {
      r.group = p->slots[sl[tail_alias_seg]].group;
      p->holders[r.group] += 1;
    } else {
      r.group = p->new_group(1);
    }
  }
  if (ncopy > 0) {
    Timed t(p, KV_KERNEL_COMPOSE_COPY, s);
    KV_LAUNCH(p, launch_compose_copy(p->geom(), c.dtype, ca, s));
  }
  for (int i = 0; i < n; ++i) p->touch(p->slots[sl[i]], true);
  p->touch(r, false);
  *out = p->handle(slot);
  return KV_OK;
}

static kv_status pack_impl(kv_pool* p, kv_state state, int64_t blk_begin, int64_t blk_end,
                           void* dst_dev, size_t dst_bytes, kv_pack_header* hdr_out,
                           kv_stream stream, bool checked) {
  if (!p || !dst_dev || !hdr_out) return KV_ERR_ARG;
  if (p->failed) return KV_ERR_HIP;
  int32_t slot;
  KV_TRY(p->lookup(state, &slot));
  StateRec& r = p->slots[slot];
  if (!(0 <= blk_begin && blk_begin < blk_end && blk_end <= r.nblocks)) return KV_ERR_ARG;
  if ((uintptr_t)dst_dev & 15) return KV_ERR_ARG;
  const void* dst_view = nullptr;
  bool dst_on_device = false;
  KV_TRY(device_view(dst_dev, &dst_view, &dst_on_device));
  const kv_model_cfg& c = p->cfg;
  kv_pack_header h = make_header(p, r, blk_begin, blk_end);
  if (dst_bytes < h.payload_bytes) return KV_ERR_BUFSIZE;
  if (dst_on_device) KV_TRY(device_span(p->device, dst_dev, h.payload_bytes));
  const int64_t nblk = h.n_blocks;
  const int32_t last_valid = (int32_t)(h.n_tokens - (nblk - 1) * c.block_size);
  const hipStream_t s = S(stream);
  if (checked) KV_TRY(csum_begin(p, s));
  {
    Timed t(p, KV_KERNEL_PACK, s);
    KV_LAUNCH(p, launch_pack(p->geom(), c.dtype, p->trow(slot), blk_begin, (int32_t)nblk, last_valid,
                       const_cast<void*>(dst_view), checked ? p->csum : nullptr, 0, s));
  }
  if (checked) {
    uint64_t sum[2];
    KV_TRY(csum_end(p, s, sum));
    h.flags = KV_PACK_CHECKSUM;
    h.checksum[0] = sum[0];
    h.checksum[1] = sum[1];
  }
  p->touch(r, true);
  *hdr_out = h;
  return KV_OK;
}

kv_status kv_pack(kv_pool* p, kv_state state, int64_t blk_begin, int64_t blk_end, void* dst_dev,
                  size_t dst_bytes, kv_pack_header* hdr_out, kv_stream stream) {
  return pack_impl(p, state, blk_begin, blk_end, dst_dev, dst_bytes, hdr_out, stream, false);
}

kv_status kv_pack_checked(kv_pool* p, kv_state state, int64_t blk_begin, int64_t blk_end,
                          void* dst_dev, size_t dst_bytes, kv_pack_header* hdr_out,
                          kv_stream stream) {
  return pack_impl(p, state, blk_begin, blk_end, dst_dev, dst_bytes, hdr_out, stream, true);
}

kv_status kv_unpack(kv_pool* p, const kv_pack_header* hdr, const void* src_dev, size_t src_bytes,
                    kv_stream stream, kv_state* out) {
  if (!p || !hdr || !src_dev || !out) return KV_ERR_ARG;
  if (p->failed) return KV_ERR_HIP;
  if ((uintptr_t)src_dev & 15) return KV_ERR_ARG;
  const void* src_view = nullptr;
  bool src_on_device = false;
  KV_TRY(device_view(src_dev, &src_view, &src_on_device));
  KV_TRY(check_header(p, hdr));
  if (src_bytes < hdr->payload_bytes) return KV_ERR_BUFSIZE;
  if (src_on_device) KV_TRY(device_span(p->device, src_dev, hdr->payload_bytes));
  const hipStream_t s = S(stream);
  const bool checked = (hdr->flags & KV_PACK_CHECKSUM) != 0;
  int32_t slot;
  KV_TRY(open_transfer(p, hdr, s, &slot));
  if (checked) KV_TRY(csum_begin(p, s));
  {
    Timed t(p, KV_KERNEL_UNPACK, s);
    KV_LAUNCH(p, launch_unpack(p->geom(), p->cfg.dtype, p->trow(slot), (int32_t)hdr->n_blocks, src_view,
                         checked ? p->csum : nullptr, 0, s));
  }
  if (checked) {
    uint64_t sum[2];
    KV_TRY(csum_end(p, s, sum));
    if (sum[0] != hdr->checksum[0] || sum[1] != hdr->checksum[1]) {
      KV_TRY(abort_transfer(p, slot, s));
      return KV_ERR_CHECKSUM;
    }
  }
  StateRec& r = p->slots[slot];
  p->touch(r, false);
  *out = p->handle(slot);
  return KV_OK;
}

kv_status kv_checkpoint_save(kv_pool* p, kv_state state, const char* path, kv_stream stream) {
  if (!p || !path) return KV_ERR_ARG;
  if (p->failed) return KV_ERR_HIP;
  int32_t slot;
  KV_TRY(p->lookup(state, &slot));
  StateRec& r = p->slots[slot];
  const kv_model_cfg& c = p->cfg;
  kv_pack_header h = make_header(p, r, 0, r.nblocks);
  const hipStream_t s = S(stream);
  Staging st;
  KV_TRY(st.alloc(h.n_blocks, h.block_bytes));
  File f;
  f.f = std::fopen(path, "wb");
  if (!f.f) return KV_ERR_IO;
  kv_pack_header blank;
  std::memset(&blank, 0, sizeof(blank));
  if (std::fwrite(&blank, sizeof(blank), 1, f.f) != 1) return KV_ERR_IO;
  KV_TRY(csum_begin(p, s));
  for (int64_t b = 0; b < h.n_blocks; b += st.blocks) {
    const int64_t k = std::min(st.blocks, h.n_blocks - b);
    const int32_t last_valid =
        b + k == h.n_blocks ? (int32_t)(h.n_tokens - (h.n_blocks - 1) * c.block_size)
                            : c.block_size;
    {
      Timed t(p, KV_KERNEL_PACK, s);
      KV_LAUNCH(p, launch_pack(p->geom(), c.dtype, p->trow(slot), b, (int32_t)k, last_valid,
                         const_cast<void*>(st.dev), p->csum,
                         (int64_t)(b * h.block_bytes / 16), s));
    }
    KV_HIP(hipStreamSynchronize(s));
    if (std::fwrite(st.host, (size_t)(k * h.block_bytes), 1, f.f) != 1) {
      KV_TRY(csum_begin(p, s));
      return KV_ERR_IO;
    }
  }
  uint64_t sum[2];
  KV_TRY(csum_end(p, s, sum));
  h.flags = KV_PACK_CHECKSUM;
  h.checksum[0] = sum[0];
  h.checksum[1] = sum[1];
  if (std::fseek(f.f, 0, SEEK_SET) != 0 || std::fwrite(&h, sizeof(h), 1, f.f) != 1)
    return KV_ERR_IO;
  const int rc = std::fclose(f.f);
  f.f = nullptr;
  if (rc != 0) return KV_ERR_IO;
  p->touch(r, true);
  return KV_OK;
}

kv_status kv_checkpoint_load(kv_pool* p, const char* path, kv_stream stream, kv_state* out) {
  if (!p || !path || !out) return KV_ERR_ARG;
  if (p->failed) return KV_ERR_HIP;
  File f;
  f.f = std::fopen(path, "rb");
  if (!f.f) return KV_ERR_IO;
  kv_pack_header h;
  if (std::fread(&h, sizeof(h), 1, f.f) != 1) return KV_ERR_IO;
  KV_TRY(check_header(p, &h));
  if (!(h.flags & KV_PACK_CHECKSUM)) return KV_ERR_BAD_HEADER;
  if (std::fseek(f.f, 0, SEEK_END) != 0) return KV_ERR_IO;
  const long size = std::ftell(f.f);
  if (size < 0 || (uint64_t)size < sizeof(h) + h.payload_bytes) return KV_ERR_IO;
  if (std::fseek(f.f, (long)sizeof(h), SEEK_SET) != 0) return KV_ERR_IO;
  const hipStream_t s = S(stream);
  Staging st;
  KV_TRY(st.alloc(h.n_blocks, h.block_bytes));
  int32_t slot;
  KV_TRY(open_transfer(p, &h, s, &slot));
  KV_TRY(csum_begin(p, s));
  for (int64_t b = 0; b < h.n_blocks; b += st.blocks) {
    const int64_t k = std::min(st.blocks, h.n_blocks - b);
    // the previous chunk's kernel has finished reading the staging buffer
    KV_HIP(hipStreamSynchronize(s));
    if (std::fread(st.host, (size_t)(k * h.block_bytes), 1, f.f) != 1) {
      KV_TRY(abort_transfer(p, slot, s));
      KV_TRY(csum_begin(p, s));
      return KV_ERR_IO;
    }
    Timed t(p, KV_KERNEL_UNPACK, s);
    KV_LAUNCH(p, launch_unpack(p->geom(), p->cfg.dtype, p->trow(slot) + b, (int32_t)k, st.dev, p->csum,
                         (int64_t)(b * h.block_bytes / 16), s));
  }
  uint64_t sum[2];
  KV_TRY(csum_end(p, s, sum));
  if (sum[0] != h.checksum[0] || sum[1] != h.checksum[1]) {
    KV_TRY(abort_transfer(p, slot, s));
    return KV_ERR_CHECKSUM;
  }
  p->touch(p->slots[slot], false);
  *out = p->handle(slot);
  return KV_OK;
}

kv_status kv_release(kv_pool* p, kv_state state, kv_stream stream) {
  if (!p) return KV_ERR_ARG;
  if (p->failed) return KV_ERR_HIP;
  int32_t slot;
  KV_TRY(p->lookup(state, &slot));
  StateRec& r = p->slots[slot];
  std::vector<int32_t> cand = {slot, (int32_t)r.nblocks};
  int32_t n = 0;
  KV_TRY(run_release(p, cand, -1, S(stream), &n));
  p->leave_group(r);
  r.status = ST_RELEASED;
  return KV_OK;
}

kv_status kv_pin(kv_pool* p, kv_state state, int32_t pinned) {
  if (!p) return KV_ERR_ARG;
  int32_t slot;
  KV_TRY(p->lookup(state, &slot));
  p->slots[slot].pinned = pinned != 0;
  return KV_OK;
}

kv_status kv_evict(kv_pool* p, int64_t max_allocated_blocks, double alpha, double beta,
                   double gamma, kv_stream stream, int32_t* n_evicted) {
  if (!p || !n_evicted || max_allocated_blocks < 0) return KV_ERR_ARG;
  if (p->failed) return KV_ERR_HIP;
  *n_evicted = 0;
  const std::vector<int32_t> cand = eviction_candidates(p, alpha, beta, gamma);
  int32_t n = 0;
  KV_TRY(run_release(p, cand, max_allocated_blocks, S(stream), &n));
  for (int i = 0; i < n; ++i) {
    StateRec& r = p->slots[cand[2 * i]];
    p->leave_group(r);
    r.status = ST_EVICTED;
  }
  *n_evicted = n;
  return KV_OK;
}

kv_status kv_evict_truncate(kv_pool* p, int64_t max_allocated_blocks, double alpha, double beta,
                            double gamma, kv_stream stream, int32_t* n_evicted,
                            int32_t* n_truncated) {
  if (!p || !n_evicted || !n_truncated || max_allocated_blocks < 0) return KV_ERR_ARG;
  if (p->failed) return KV_ERR_HIP;
  *n_evicted = *n_truncated = 0;
  const std::vector<int32_t> cand = eviction_candidates(p, alpha, beta, gamma);
  int32_t n = 0;
  std::vector<int32_t> kept;
  KV_TRY(run_release(p, cand, max_allocated_blocks, S(stream), &n, &kept));
  const int64_t B = p->cfg.block_size;
  for (int i = 0; i < n; ++i) {
    StateRec& r = p->slots[cand[2 * i]];
    const int32_t k = kept[i];
    if (k < 0 || k > r.nblocks) return KV_ERR_INTERNAL;
    if (k == r.nblocks) continue;  // only shared blocks: nothing given up
    p->leave_group(r);             // what remains ends on a whole block
    if (k == 0) {
      r.status = ST_EVICTED;
      ++*n_evicted;
    } else {
      r.nblocks = k;
      r.n = k * B;
      ++*n_truncated;
    }
  }
  return KV_OK;
}

kv_status kv_sync(kv_pool* p, kv_stream stream) {
  if (!p) return KV_ERR_ARG;
  if (p->failed) return KV_ERR_HIP;
  const hipStream_t s = S(stream);
  DevHeader h;
  KV_HIP(hipMemcpyAsync(&h, p->dhdr, sizeof(h), hipMemcpyDeviceToHost, s));
  KV_HIP(hipStreamSynchronize(s));
  if (h.status != 0) {
    const int32_t zero = 0;
    KV_HIP(hipMemcpyAsync(&p->dhdr->status, &zero, 4, hipMemcpyHostToDevice, s));
    KV_HIP(hipStreamSynchronize(s));
    return h.status;
  }
  if (h.head != p->head || h.tail != p->tail) return KV_ERR_INTERNAL;
  return KV_OK;
}

kv_status kv_state_info(kv_pool* p, kv_state state, int64_t* pos0, int64_t* n_tokens,
                        int64_t* n_blocks, uint64_t* lineage, int64_t* state_id) {
  if (!p) return KV_ERR_ARG;
  int32_t slot;
  KV_TRY(p->lookup(state, &slot));
  const StateRec& r = p->slots[slot];
  if (pos0) *pos0 = r.pos0;
  if (n_tokens) *n_tokens = r.n;
  if (n_blocks) *n_blocks = r.nblocks;
  if (lineage) *lineage = r.lineage;
  if (state_id) *state_id = r.sid;
  return KV_OK;
}

kv_status kv_state_usage(kv_pool* p, kv_state state, int64_t* reuse, int64_t* last_access,
                         int32_t* pinned) {
  if (!p) return KV_ERR_ARG;
  int32_t slot;
  KV_TRY(p->lookup(state, &slot));
  const StateRec& r = p->slots[slot];
  if (reuse) *reuse = r.reuse;
  if (last_access) *last_access = r.last_access;
  if (pinned) *pinned = r.pinned ? 1 : 0;
  return KV_OK;
}

kv_status kv_pool_counts(kv_pool* p, int64_t* free_blocks, int64_t* live_states,
                         int64_t* clock) {
  if (!p) return KV_ERR_ARG;
  if (free_blocks) *free_blocks = p->free_blocks();
  if (live_states) *live_states = p->live();
  if (clock) *clock = p->clock;
  return KV_OK;
}

kv_status kv_read_block_table(kv_pool* p, kv_state state, int32_t* host_out, int64_t cap,
                              kv_stream stream) {
  if (!p || !host_out) return KV_ERR_ARG;
  int32_t slot;
  KV_TRY(p->lookup(state, &slot));
  const StateRec& r = p->slots[slot];
  if (cap < r.nblocks) return KV_ERR_BUFSIZE;
  const hipStream_t s = S(stream);
  KV_HIP(hipMemcpyAsync(host_out, p->trow(slot), r.nblocks * 4, hipMemcpyDeviceToHost, s));
  KV_HIP(hipStreamSynchronize(s));
  return KV_OK;
}

kv_status kv_read_allocator(kv_pool* p, int32_t* refcount_out, int32_t* ring_out, int64_t* head,
                            int64_t* tail, kv_stream stream) {
  if (!p) return KV_ERR_ARG;
  const hipStream_t s = S(stream);
  DevHeader h;
  if (refcount_out)
    KV_HIP(hipMemcpyAsync(refcount_out, p->rc, p->P * 4, hipMemcpyDeviceToHost, s));
  if (ring_out) KV_HIP(hipMemcpyAsync(ring_out, p->ring, p->P * 4, hipMemcpyDeviceToHost, s));
  KV_HIP(hipMemcpyAsync(&h, p->dhdr, sizeof(h), hipMemcpyDeviceToHost, s));
  KV_HIP(hipStreamSynchronize(s));
  if (head) *head = h.head;
  if (tail) *tail = h.tail;
  return KV_OK;
}

kv_status kv_profile_enable(kv_pool* p, int32_t enabled) {
  if (!p) return KV_ERR_ARG;
  p->prof = enabled != 0;
  return KV_OK;
}

}  // extern "C"

// Wait for the recorded launches and add them to the per-kind totals and lists.
static kv_status profile_drain(kv_pool* p) {
  size_t i = 0;
  kv_status st = KV_OK;
  for (; i < p->pending.size(); ++i) {
    const auto& r = p->pending[i];
    float ms = 0.f;
    if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) {
      st = KV_ERR_HIP;
      break;
    }
    p->acc[r.kind].launches += 1;
    p->acc[r.kind].total_ms += ms;
    p->launch_ms[r.kind].push_back(ms);
    p->spare.push_back(r.a);
    p->spare.push_back(r.b);
  }
  p->pending.erase(p->pending.begin(), p->pending.begin() + i);
  return st;
}

extern "C" {

kv_status kv_profile_read(kv_pool* p, kv_profile_entry* out) {
  if (!p || !out) return KV_ERR_ARG;
  KV_TRY(profile_drain(p));
  for (int k = 0; k < KV_KERNEL_KINDS; ++k) {
    out[k] = p->acc[k];
    p->acc[k] = kv_profile_entry{0, 0.0};
    p->launch_ms[k].clear();
  }
  return KV_OK;
}

kv_status kv_profile_launches(kv_pool* p, int32_t kind, float* out_ms, int64_t cap,
                              int64_t* n) {
  if (!p || !n || kind < 0 || kind >= KV_KERNEL_KINDS || cap < 0 || (cap > 0 && !out_ms))
    return KV_ERR_ARG;
  KV_TRY(profile_drain(p));
  const auto& v = p->launch_ms[kind];
  *n = (int64_t)v.size();
  for (int64_t i = 0; i < std::min<int64_t>(cap, *n); ++i) out_ms[i] = v[(size_t)i];
  return KV_OK;
}

}  // extern "C"
