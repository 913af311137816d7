// C ABI of the chunked MoE expert layer: argument checks, the memory-aware
// chunk planner, the per-chunk workspace layout, and the chunk driver that
// allocates, fills and releases every chunk's buffers in stream order
// (paper Section 4.1, Eq. (6)/(7); Section 4.2, Eq. (8)/(9)).
#include <algorithm>
#include <cstdlib>
#include <map>
#include <mutex>
#include <unordered_map>
#include <vector>

#include "kernels.h"
#include "memfine.h"

using namespace memfine;

namespace {

// ------------------------------------------------------------- profiling
struct ProfRecord {
  int id;
  hipEvent_t start, stop;
  double flops, bytes;
};
std::mutex g_prof_mu;
uint32_t g_prof_mask = 0;
std::vector<ProfRecord> g_prof;

class KernelTimer {
 public:
  KernelTimer(int id, hipStream_t s, double flops, double bytes)
      : id_(id), s_(s), flops_(flops), bytes_(bytes) {
    on_ = (g_prof_mask >> id) & 1u;
    if (on_) {
      on_ = hipEventCreate(&a_) == hipSuccess && hipEventCreate(&b_) == hipSuccess &&
            hipEventRecord(a_, s_) == hipSuccess;
    }
  }
  ~KernelTimer() {
    if (!on_) return;
    if (hipEventRecord(b_, s_) != hipSuccess) return;
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_prof.push_back({id_, a_, b_, flops_, bytes_});
  }

 private:
  int id_;
  hipStream_t s_;
  double flops_, bytes_;
  bool on_ = false;
  hipEvent_t a_ = nullptr, b_ = nullptr;
};

// ----------------------------------------------------------------- checks
int check_shape(const memfine_shape* s) {
  if (!s) return MEMFINE_ERR_INVALID_ARG;
  if (s->T < 0 || s->h < 64 || s->F < 64 || (s->h % 64) || (s->F % 64) || s->k < 1 || s->E < 1 ||
      s->E > 1024)
    return MEMFINE_ERR_INVALID_ARG;
  if (s->dtype != MEMFINE_BF16 && s->dtype != MEMFINE_F32) return MEMFINE_ERR_UNSUPPORTED;
  if (s->T * (int64_t)s->k >= (int64_t(1) << 31)) return MEMFINE_ERR_UNSUPPORTED;
  // the kernels address X, dY and one expert's weights with 31-bit offsets
  const int64_t es = s->dtype == MEMFINE_BF16 ? 2 : 4;
  if (s->T * (int64_t)s->h * es >= (int64_t(1) << 31) ||
      (int64_t)2 * s->F * (int64_t)s->h * es >= (int64_t(1) << 31))
    return MEMFINE_ERR_UNSUPPORTED;
  return MEMFINE_OK;
}

int64_t elem_bytes(const memfine_shape& s) { return s.dtype == MEMFINE_BF16 ? 2 : 4; }

// ------------------------------------------------------ workspace layout
// One allocation per chunk, carved into 256-byte aligned buffers.
struct Layout {
  enum {
    kBcount, kBstart, kCounts, kOffsets, kOrder, kSorted, kRowOf, kTokOf, kGateOf,
    kA, kY,                 // forward
    kU, kAg, kDxp, kDgp,    // backward
    kCtr,                   // backward: tile counters of the two weight gradients
    kOffC, kOrderC, kWexp, kWmode,  // expert-ordered chunks: the current chunk's view
    kNum
  };
  int64_t off[kNum];
  int64_t size[kNum];
  int64_t total;
};

int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

// Buffers for n slots: the routing tables of one dispatch (`tables`), the
// views of expert-ordered chunks (`views`), and the intermediates of a
// forward or backward pass over n rows (`pass`, or -1 for none).
void layout(const memfine_shape& s, int64_t n, int pass, bool tables, bool views, Layout& L) {
  const int64_t es = elem_bytes(s), E = s.E, nb = dispatch_blocks(n);
  const int64_t P = dgate_partials(s.F);
  for (int i = 0; i < Layout::kNum; ++i) L.size[i] = 0;
  if (tables) {
    L.size[Layout::kBcount] = E * nb * 4;
    L.size[Layout::kBstart] = E * nb * 4;
    L.size[Layout::kCounts] = E * 4;
    L.size[Layout::kOffsets] = (E + 1) * 4;
    L.size[Layout::kOrder] = E * 4;
    L.size[Layout::kSorted] = n * 4;
    L.size[Layout::kRowOf] = n * 4;
    L.size[Layout::kTokOf] = n * 4;
    L.size[Layout::kGateOf] = n * 4;
  }
  if (views) {
    L.size[Layout::kOffC] = (E + 1) * 4;
    L.size[Layout::kOrderC] = E * 4;
    L.size[Layout::kWexp] = 4;
    L.size[Layout::kWmode] = E * 4;
  }
  if (pass == MEMFINE_PASS_FWD) {
    L.size[Layout::kA] = n * s.F * es;
    L.size[Layout::kY] = n * s.h * es;
  } else if (pass == MEMFINE_PASS_BWD) {
    L.size[Layout::kU] = n * 2 * s.F * es;
    L.size[Layout::kAg] = n * s.F * es;
    L.size[Layout::kDxp] = n * s.h * es;
    L.size[Layout::kDgp] = n * P * 4;
    L.size[Layout::kCtr] = 2 * 4;
  }
  int64_t o = 0;
  for (int i = 0; i < Layout::kNum; ++i) {
    L.off[i] = o;
    o += align256(L.size[i]);
  }
  L.total = o;
}
// a token-range chunk of n slots: its dispatch tables and its pass buffers
void chunk_layout(const memfine_shape& s, int64_t n, int pass, Layout& L) {
  layout(s, n, pass, true, false, L);
}

// tokens in the largest chunk of the floor-balanced split of T into C
int64_t max_chunk_tokens(int64_t T, int64_t C) {
  if (T == 0) return 0;
  C = std::min(C, T);
  return (T + C - 1) / C;
}

// --------------------------------------------------------------- memory
std::mutex g_pool_mu;
std::unordered_map<int, hipMemPool_t> g_pools;

// A private stream-ordered pool per device that keeps freed memory cached,
// so releasing a chunk's buffers and allocating the next chunk's reuses the
// same memory without a trip to the driver.
hipMemPool_t device_pool() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  std::lock_guard<std::mutex> lk(g_pool_mu);
  auto it = g_pools.find(dev);
  if (it != g_pools.end()) return it->second;
  hipMemPoolProps props = {};
  props.allocType = hipMemAllocationTypePinned;
  props.location.type = hipMemLocationTypeDevice;
  props.location.id = dev;
  hipMemPool_t pool = nullptr;
  if (hipMemPoolCreate(&pool, &props) != hipSuccess) return nullptr;
  uint64_t keep = UINT64_MAX;
  hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
  g_pools[dev] = pool;
  return pool;
}

// Calls with a NULL allocator carve each chunk's buffers from one cached
// block per (device, stream) and hand it back when the chunk ends.  Kernels
// on one stream run in order, so the next chunk (or call) on that stream may
// take the block again at once, with no trip to the allocator: a
// hipFreeAsync per chunk blocked the host for up to ~1 ms here, long enough
// that the next chunk's kernels were enqueued only after the GPU had
// drained.  The block is re-allocated (from the pool, in stream order) when
// a larger workspace is asked for and kept until the process ends.  A
// request while the stream's block is taken gets a pool allocation of its
// own.
struct WsBlock {
  void* p = nullptr;
  size_t bytes = 0;
  bool busy = false;
};
std::mutex g_ws_mu;
std::map<std::pair<int, hipStream_t>, WsBlock> g_ws;

void* pool_alloc(size_t bytes, hipStream_t s) {
  hipMemPool_t pool = device_pool();
  if (!pool) return nullptr;
  void* p = nullptr;
  if (hipMallocFromPoolAsync(&p, bytes, pool, s) != hipSuccess) {
    (void)hipGetLastError();
    return nullptr;
  }
  return p;
}

void* ws_alloc(const memfine_allocator* a, size_t bytes, hipStream_t s) {
  if (bytes == 0) bytes = 256;
  if (a && a->alloc) return a->alloc(bytes, (void*)s, a->ctx);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  {
    std::lock_guard<std::mutex> lk(g_ws_mu);
    WsBlock& b = g_ws[{dev, s}];
    if (!b.busy) {
      if (b.bytes < bytes) {
        if (b.p) (void)hipFreeAsync(b.p, s);
        b.p = pool_alloc(bytes, s);
        b.bytes = b.p ? bytes : 0;
        if (!b.p) return nullptr;
      }
      b.busy = true;
      return b.p;
    }
  }
  return pool_alloc(bytes, s);
}

void ws_release(const memfine_allocator* a, void* p, size_t bytes, hipStream_t s) {
  if (!p) return;
  if (bytes == 0) bytes = 256;
  if (a && a->release) {
    a->release(p, bytes, (void*)s, a->ctx);
    return;
  }
  if (a && a->alloc) return;
  int dev = 0;
  if (hipGetDevice(&dev) == hipSuccess) {
    std::lock_guard<std::mutex> lk(g_ws_mu);
    auto it = g_ws.find({dev, s});
    if (it != g_ws.end() && it->second.p == p) {
      it->second.busy = false;
      return;
    }
  }
  (void)hipFreeAsync(p, s);
}

// Pinned host buffer per device for memfine_count's result (E + 1 ints at
// most 1025), allocated on first use and kept until the process ends.
constexpr int kMaxExperts = 1024;
std::mutex g_pinned_mu;
std::unordered_map<int, int32_t*> g_pinned;

struct ChunkBuffers {
  ChunkMeta m;
  void *a, *y, *u, *ag, *dxp;
  float* dgp;
  int32_t* ctr;  // [2] tile counters: FC1 wgrad, FC2 wgrad
  int32_t *off_c, *order_c, *wexp, *wmode;  // expert-ordered chunks: the chunk's view
};

ChunkBuffers carve(void* base, const Layout& L) {
  char* b = (char*)base;
  ChunkBuffers c;
  c.m.bcount = (int32_t*)(b + L.off[Layout::kBcount]);
  c.m.bstart = (int32_t*)(b + L.off[Layout::kBstart]);
  c.m.counts = (int32_t*)(b + L.off[Layout::kCounts]);
  c.m.offsets = (int32_t*)(b + L.off[Layout::kOffsets]);
  c.m.order = (int32_t*)(b + L.off[Layout::kOrder]);
  c.m.sorted_slot = (int32_t*)(b + L.off[Layout::kSorted]);
  c.m.row_of_slot = (int32_t*)(b + L.off[Layout::kRowOf]);
  c.m.tok_of_row = (int32_t*)(b + L.off[Layout::kTokOf]);
  c.m.gate_of_row = (float*)(b + L.off[Layout::kGateOf]);
  c.a = b + L.off[Layout::kA];
  c.y = b + L.off[Layout::kY];
  c.u = b + L.off[Layout::kU];
  c.ag = b + L.off[Layout::kAg];
  c.dxp = b + L.off[Layout::kDxp];
  c.dgp = (float*)(b + L.off[Layout::kDgp]);
  c.ctr = (int32_t*)(b + L.off[Layout::kCtr]);
  c.off_c = (int32_t*)(b + L.off[Layout::kOffC]);
  c.order_c = (int32_t*)(b + L.off[Layout::kOrderC]);
  c.wexp = (int32_t*)(b + L.off[Layout::kWexp]);
  c.wmode = (int32_t*)(b + L.off[Layout::kWmode]);
  return c;
}

// Launch options (memfine_set_launch_options): one process-wide setting,
// copied under a lock at the start of every layer call, so that a call never
// sees a half-written update.  The defaults are the measured-best choices.
std::mutex g_opts_mu;
const memfine_launch_options kDefaultOptions = {MEMFINE_TILE_AUTO, -1, 1, 0, 0, MEMFINE_CHUNK_TOKENS};
memfine_launch_options g_opts = kDefaultOptions;

memfine_launch_options launch_options() {
  std::lock_guard<std::mutex> lk(g_opts_mu);
  return g_opts;
}

// Compute units of the current device (cached per device id).
int device_cus() {
  static std::mutex mu;
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  std::lock_guard<std::mutex> lk(mu);
  if (cache[dev] == 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
      v = 256;
    cache[dev] = v;
  }
  return cache[dev];
}

int hip_status(hipError_t e) { return e == hipSuccess ? MEMFINE_OK : MEMFINE_ERR_HIP; }


// Two side streams per device (non-blocking, default priority) and the
// events of one fork/join.  `mu` is held from the fork to the join, so that
// concurrent callers on one device never interleave their uses of the
// shared events.
struct SideStreams {
  std::mutex mu;
  hipStream_t s[2] = {nullptr, nullptr};
  hipEvent_t fork = nullptr, join[2] = {nullptr, nullptr};
  bool ok = false;
};
SideStreams* side_streams() {
  static std::mutex mu;
  static SideStreams cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lk(mu);
  SideStreams& c = cache[dev];
  if (!c.ok) {
    bool ok = true;
    for (auto& st : c.s)
      if (!st) ok = ok && hipStreamCreateWithFlags(&st, hipStreamNonBlocking) == hipSuccess;
    if (!c.fork) ok = ok && hipEventCreateWithFlags(&c.fork, hipEventDisableTiming) == hipSuccess;
    for (auto& e : c.join)
      if (!e) ok = ok && hipEventCreateWithFlags(&e, hipEventDisableTiming) == hipSuccess;
    if (!ok) {
      (void)hipGetLastError();
      return nullptr;
    }
    c.ok = true;
  }
  return &c;
}

GemmArgs gemm_args(const memfine_shape& s, int64_t n, const ChunkBuffers& c,
                   const memfine_launch_options& o) {
  GemmArgs g = {};
  g.dtype = s.dtype;
  g.n = (int)n;
  g.E = s.E;
  g.h = s.h;
  g.F = s.F;
  g.offsets = c.m.offsets;
  g.order = c.m.order;
  g.tok_of_row = c.m.tok_of_row;
  g.gate_of_row = c.m.gate_of_row;
  g.a = c.a;
  g.y = c.y;
  g.u = c.u;
  g.ag = c.ag;
  g.dxp = c.dxp;
  g.dgp = c.dgp;
  g.P = dgate_partials(s.F);
  g.T_h_bytes = s.T * (int64_t)s.h * elem_bytes(s);
  g.tile_override = o.tile;
  g.raster = o.raster;
  g.cus = device_cus();
  g.split_tail = o.split_tail;
  return g;
}

// This library's backward bytes per slot, an upper bound of the slope of
// its per-chunk workspace in the chunk's slots: the intermediates u, g*a
// and the input gradient (es (3F + h)), the gate-gradient partials, the
// four per-slot routing tables, and the per-block expert counts.
int64_t beta_impl(const memfine_shape& s) {
  return elem_bytes(s) * (3 * (int64_t)s.F + s.h) + 4 * (int64_t)dgate_partials(s.F) + 16 +
         (s.E + 31) / 32;
}

// Smallest bin b with b * avail >= num (bin b splits the slots into b chunks
// of at most s''/b), or -1.
int32_t smallest_bin_admitting(const int32_t* bins, int nbins, int64_t avail, __int128 num) {
  int32_t best = INT32_MAX;
  for (int i = 0; i < nbins; ++i)
    if ((__int128)bins[i] * avail >= num) best = std::min(best, bins[i]);
  return best == INT32_MAX ? -1 : best;
}

// Smallest bin larger than b, or -1.
int32_t next_bin_above(const int32_t* bins, int nbins, int32_t b) {
  int32_t best = INT32_MAX;
  for (int i = 0; i < nbins; ++i)
    if (bins[i] > b) best = std::min(best, bins[i]);
  return best == INT32_MAX ? -1 : best;
}

// Algorithmic work of one launch, for the timing table.
struct Work {
  double flops, bytes;
};
Work dispatch_work(int64_t n) { return {0.0, 8.0 * n + 16.0 * n}; }

// ----------------------------------------------- static scratch (no-alloc)
// Working memory of memfine_moe_fwd_noalloc: a device array that the code
// object carries, so that the call allocates nothing.  In host code its name
// stands for a host-side shadow, not a device address: the address comes
// from hipGetSymbolAddress, once per device (each GPU holds its own copy),
// and is the only way host code refers to the array's memory.
constexpr int64_t kScratchBytes = MEMFINE_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kScratchBytes];

std::mutex g_scratch_mu;
std::unordered_map<int, void*> g_scratch_ptr;

// Device address of `scratch` on the current device (looked up on the first
// call on that device, with it current).
int scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MEMFINE_ERR_HIP;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  auto it = g_scratch_ptr.find(dev);
  if (it == g_scratch_ptr.end()) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress((void**)&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
      (void)hipGetLastError();
      return MEMFINE_ERR_HIP;
    }
    it = g_scratch_ptr.emplace(dev, ptr).first;
  }
  *out = it->second;
  return MEMFINE_OK;
}

int moe_fwd_impl(const memfine_shape* shape, int32_t chunks, const void* d_X,
                 const int32_t* d_idx, const float* d_gates, const void* d_W1, const void* d_W2,
                 void* d_Y, const memfine_allocator* alloc, void* fixed_ws,
                 const memfine_launch_options& opt, void* stream);

// Expert-ordered chunks (launch option chunk_order): one dispatch groups all
// T k slots by expert; chunk c is rows [c N / C, (c + 1) N / C) of that
// order.  Its routing tables and the chunk views live for the whole call.
int64_t expert_meta_bytes(const memfine_shape& s) {
  Layout L;
  layout(s, s.T * (int64_t)s.k, -1, true, true, L);
  return L.total;
}
int64_t expert_chunks(const memfine_shape& s, int32_t chunks) {
  return std::min<int64_t>(chunks, s.T);
}
int64_t expert_chunk_row(const memfine_shape& s, int64_t C, int64_t c) {
  return c * (s.T * (int64_t)s.k) / C;
}

int64_t workspace_bytes(const memfine_shape& s, int32_t chunks, int32_t pass, int32_t order) {
  if (order == MEMFINE_CHUNK_EXPERTS) {
    const int64_t N = s.T * (int64_t)s.k;
    if (N == 0) return 0;
    const int64_t C = expert_chunks(s, chunks);
    Layout L;
    layout(s, (N + C - 1) / C, pass, false, false, L);
    return expert_meta_bytes(s) + L.total;
  }
  const int64_t n = max_chunk_tokens(s.T, chunks) * s.k;
  if (n == 0) return 0;
  Layout L;
  chunk_layout(s, n, pass, L);
  return L.total;
}

}  // namespace

// =================================================================== ABI
extern "C" {

const char* memfine_status_str(int status) {
  switch (status) {
    case MEMFINE_OK: return "ok";
    case MEMFINE_ERR_INVALID_ARG: return "invalid argument";
    case MEMFINE_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case MEMFINE_ERR_BUDGET: return "memory budget too small for every allowed chunk count";
    case MEMFINE_ERR_OOM: return "device memory allocation failed";
    case MEMFINE_ERR_HIP: return "HIP runtime error";
    case MEMFINE_ERR_SCRATCH:
      return "the largest chunk needs more working memory than the static scratch holds "
             "(MEMFINE_NOALLOC_SCRATCH_BYTES); use more chunks";
    default: return "unknown status";
  }
}

int memfine_plan(const memfine_shape* shape, const int64_t* h_counts, int64_t budget_bytes,
                 int64_t fixed_bytes, int64_t beta_bytes, const int32_t* bins, int32_t nbins,
                 int32_t* chunks_out, memfine_plan_info* info) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if (!h_counts || !bins || nbins < 1 || !chunks_out || fixed_bytes < 0 || beta_bytes < 0)
    return MEMFINE_ERR_INVALID_ARG;
  int32_t bmax = 0;
  for (int i = 0; i < nbins; ++i) {
    if (bins[i] < 1) return MEMFINE_ERR_INVALID_ARG;
    bmax = std::max(bmax, bins[i]);
  }
  __int128 s2 = 0;
  for (int e = 0; e < shape->E; ++e) {
    if (h_counts[e] < 0) return MEMFINE_ERR_INVALID_ARG;
    s2 += h_counts[e];
  }
  // Table 2 rows 11-13: D_t (h + 2 g_e + h) bytes per received slot
  const int64_t beta_paper = elem_bytes(*shape) * (2 * (int64_t)shape->h + 2 * (int64_t)shape->F);
  const int64_t b_impl = beta_impl(*shape);
  const bool impl_check = beta_bytes == 0;
  const int64_t beta = beta_bytes > 0 ? beta_bytes : std::max(beta_paper, b_impl);
  const int64_t avail = budget_bytes - fixed_bytes;
  int64_t c_theory = -1;
  int32_t chosen = -1;
  int32_t paper_chosen = -1;
  if (avail > 0) {
    // Eq. (9): c = ceil(s'' / s'_max) = ceil(s'' * beta / avail)
    const __int128 num = s2 * (__int128)beta;
    const __int128 c = (num + avail - 1) / avail;
    c_theory = c > (__int128)INT64_MAX ? INT64_MAX : (int64_t)c;
    chosen = smallest_bin_admitting(bins, nbins, avail, num);
    paper_chosen = smallest_bin_admitting(bins, nbins, avail, s2 * (__int128)beta_paper);
    // Eq. (3) on the memory this library really takes: the next larger bin
    // while the chunk's workspace exceeds what is available
    while (impl_check && chosen > 0 &&
           memfine_workspace_bytes(shape, chosen, MEMFINE_PASS_BWD) > avail)
      chosen = next_bin_above(bins, nbins, chosen);
  }
  const bool fits = chosen > 0;
  if (!fits) chosen = bmax;
  *chunks_out = chosen;
  if (info) {
    info->s_recv = (int64_t)s2;
    info->beta = beta;
    info->avail = avail;
    info->s_max = avail > 0 ? (double)avail / (double)beta : 0.0;
    info->c_theory = c_theory;
    info->chunks = chosen;
    info->fits = fits ? 1 : 0;
    info->paper_peak_bytes = beta_paper * max_chunk_tokens(shape->T, chosen) * shape->k;
    info->beta_paper = beta_paper;
    info->beta_impl = b_impl;
    info->workspace_bytes = memfine_workspace_bytes(shape, chosen, MEMFINE_PASS_BWD);
    info->paper_chunks = paper_chosen > 0 ? paper_chosen : bmax;
    info->reserved = 0;
  }
  return fits ? MEMFINE_OK : MEMFINE_ERR_BUDGET;
}

int memfine_set_launch_options(const memfine_launch_options* opts) {
  memfine_launch_options o = kDefaultOptions;
  if (opts) {
    if (opts->tile < MEMFINE_TILE_AUTO || opts->tile > MEMFINE_TILE_256_REG ||
        opts->raster < -1 || opts->raster > 4 || (opts->split_tail != 0 && opts->split_tail != 1) ||
        (opts->pair != 0 && opts->pair != 1) || (opts->streams != 0 && opts->streams != 1) ||
        (opts->chunk_order != MEMFINE_CHUNK_TOKENS && opts->chunk_order != MEMFINE_CHUNK_EXPERTS))
      return MEMFINE_ERR_INVALID_ARG;
    o = *opts;
  }
  std::lock_guard<std::mutex> lk(g_opts_mu);
  g_opts = o;
  return MEMFINE_OK;
}

int memfine_get_launch_options(memfine_launch_options* opts_out) {
  if (!opts_out) return MEMFINE_ERR_INVALID_ARG;
  *opts_out = launch_options();
  return MEMFINE_OK;
}

int memfine_workspace_held(void* stream, int64_t* bytes_out) {
  if (!bytes_out) return MEMFINE_ERR_INVALID_ARG;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MEMFINE_ERR_HIP;
  std::lock_guard<std::mutex> lk(g_ws_mu);
  auto it = g_ws.find({dev, (hipStream_t)stream});
  *bytes_out = it == g_ws.end() ? 0 : (int64_t)it->second.bytes;
  return MEMFINE_OK;
}

int memfine_workspace_trim(void* stream, int64_t keep_bytes) {
  if (keep_bytes < 0) return MEMFINE_ERR_INVALID_ARG;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MEMFINE_ERR_HIP;
  hipStream_t s = (hipStream_t)stream;
  std::lock_guard<std::mutex> lk(g_ws_mu);
  auto it = g_ws.find({dev, s});
  if (it == g_ws.end()) return MEMFINE_OK;
  WsBlock& b = it->second;
  if (b.busy) return MEMFINE_ERR_INVALID_ARG;  // a call on this stream is enqueuing
  if ((int64_t)b.bytes <= keep_bytes) return MEMFINE_OK;
  if (b.p && hipFreeAsync(b.p, s) != hipSuccess) return MEMFINE_ERR_HIP;
  b.p = nullptr;
  b.bytes = 0;
  if (keep_bytes > 0) {
    b.p = pool_alloc((size_t)keep_bytes, s);
    if (!b.p) return MEMFINE_ERR_OOM;
    b.bytes = (size_t)keep_bytes;
  }
  return MEMFINE_OK;
}

int memfine_pool_high_water(int64_t* bytes_out, int32_t reset) {
  if (!bytes_out || (reset != 0 && reset != 1)) return MEMFINE_ERR_INVALID_ARG;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MEMFINE_ERR_HIP;
  hipMemPool_t pool = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_pool_mu);
    auto it = g_pools.find(dev);
    if (it != g_pools.end()) pool = it->second;
  }
  *bytes_out = 0;
  if (!pool) return MEMFINE_OK;
  uint64_t v = 0;
  if (hipMemPoolGetAttribute(pool, hipMemPoolAttrUsedMemHigh, &v) != hipSuccess)
    return MEMFINE_ERR_HIP;
  *bytes_out = (int64_t)v;
  if (reset) {
    uint64_t zero = 0;
    if (hipMemPoolSetAttribute(pool, hipMemPoolAttrUsedMemHigh, &zero) != hipSuccess)
      return MEMFINE_ERR_HIP;
  }
  return MEMFINE_OK;
}

int64_t memfine_workspace_bytes(const memfine_shape* shape, int32_t chunks, int32_t pass) {
  if (check_shape(shape)) return MEMFINE_ERR_INVALID_ARG;
  if (chunks < 1 || (pass != MEMFINE_PASS_FWD && pass != MEMFINE_PASS_BWD))
    return MEMFINE_ERR_INVALID_ARG;
  return workspace_bytes(*shape, chunks, pass, launch_options().chunk_order);
}

int memfine_count(const memfine_shape* shape, const int32_t* d_idx, int32_t* d_work,
                  int64_t* h_counts, void* stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if (!d_work || !h_counts || (shape->T > 0 && !d_idx)) return MEMFINE_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  const int64_t nslots = shape->T * shape->k;
  {
    KernelTimer kt(MEMFINE_K_COUNT, s, 0.0, 4.0 * nslots);
    if (launch_count(d_idx, nslots, shape->E, d_work, s) != hipSuccess) return MEMFINE_ERR_HIP;
  }
  // the counts come back through a pinned buffer (a direct copy; a pageable
  // destination is staged by the runtime)
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MEMFINE_ERR_HIP;
  std::lock_guard<std::mutex> lk(g_pinned_mu);
  int32_t*& host = g_pinned[dev];
  if (!host && hipHostMalloc((void**)&host, (kMaxExperts + 1) * sizeof(int32_t),
                             hipHostMallocDefault) != hipSuccess) {
    host = nullptr;
    return MEMFINE_ERR_HIP;
  }
  if (hipMemcpyAsync(host, d_work, (shape->E + 1) * sizeof(int32_t), hipMemcpyDeviceToHost, s) !=
      hipSuccess)
    return MEMFINE_ERR_HIP;
  if (hipStreamSynchronize(s) != hipSuccess) return MEMFINE_ERR_HIP;
  for (int e = 0; e < shape->E; ++e) h_counts[e] = host[e];
  return host[shape->E] ? MEMFINE_ERR_INVALID_ARG : MEMFINE_OK;
}

int memfine_dispatch(const memfine_shape* shape, const int32_t* d_idx, int64_t t0, int64_t t1,
                     int32_t* d_counts, int32_t* d_offsets, int32_t* d_sorted_slot,
                     int32_t* d_row_of_slot, const memfine_allocator* alloc, void* stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if (t0 < 0 || t1 < t0 || t1 > shape->T) return MEMFINE_ERR_INVALID_ARG;
  const int64_t n = (t1 - t0) * shape->k;
  if (!d_counts || !d_offsets || (n > 0 && (!d_idx || !d_sorted_slot || !d_row_of_slot)))
    return MEMFINE_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  const int64_t E = shape->E, nb = dispatch_blocks(n);
  // scratch: bcount, bstart, order, tok_of_row, gate_of_row
  const int64_t o_bstart = align256(E * nb * 4), o_order = o_bstart + align256(E * nb * 4);
  const int64_t o_tok = o_order + align256(E * 4), o_gate = o_tok + align256(n * 4);
  const int64_t total = o_gate + align256(n * 4);
  char* scratch = (char*)ws_alloc(alloc, (size_t)total, s);
  if (!scratch) return MEMFINE_ERR_OOM;
  ChunkMeta m;
  m.bcount = (int32_t*)scratch;
  m.bstart = (int32_t*)(scratch + o_bstart);
  m.order = (int32_t*)(scratch + o_order);
  m.tok_of_row = (int32_t*)(scratch + o_tok);
  m.gate_of_row = (float*)(scratch + o_gate);
  m.counts = d_counts;
  m.offsets = d_offsets;
  m.sorted_slot = d_sorted_slot;
  m.row_of_slot = d_row_of_slot;
  hipError_t err;
  {
    KernelTimer kt(MEMFINE_K_DISPATCH, s, 0.0, dispatch_work(n).bytes);
    err = launch_dispatch(d_idx, nullptr, t0 * shape->k, (int)n, shape->E, shape->k, m, s);
  }
  ws_release(alloc, scratch, (size_t)total, s);
  return hip_status(err);
}

int memfine_moe_fwd(const memfine_shape* shape, int32_t chunks, const void* d_X,
                    const int32_t* d_idx, const float* d_gates, const void* d_W1,
                    const void* d_W2, void* d_Y, const memfine_allocator* alloc, void* stream) {
  return moe_fwd_impl(shape, chunks, d_X, d_idx, d_gates, d_W1, d_W2, d_Y, alloc, nullptr,
                      launch_options(), stream);
}

int memfine_moe_fwd_noalloc(const memfine_shape* shape, int32_t chunks, const void* d_X,
                            const int32_t* d_idx, const float* d_gates, const void* d_W1,
                            const void* d_W2, void* d_Y, void* stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if (chunks < 1) return MEMFINE_ERR_INVALID_ARG;
  // one copy of the options for the size check and the call
  const memfine_launch_options opt = launch_options();
  if (workspace_bytes(*shape, chunks, MEMFINE_PASS_FWD, opt.chunk_order) > kScratchBytes)
    return MEMFINE_ERR_SCRATCH;
  if (shape->T == 0) return MEMFINE_OK;
  void* scratch_dev = nullptr;
  rc = scratch_address(&scratch_dev);
  if (rc) return rc;
  return moe_fwd_impl(shape, chunks, d_X, d_idx, d_gates, d_W1, d_W2, d_Y, nullptr, scratch_dev,
                      opt, stream);
}

}  // extern "C"

namespace {
// The chunked forward.  Each chunk's buffers come from `fixed_ws` when it is
// not null (it then holds the largest chunk's workspace; nothing is
// allocated or released), else from ws_alloc / ws_release.
// Profiling of expert-ordered chunks: a host copy of the layer's expert
// offsets (one synchronisation per call, only while kernel timing is on),
// for the algorithmic bytes of each chunk's launches.
std::vector<int32_t> offsets_for_profile(const int32_t* d_offsets, int E, hipStream_t s) {
  std::vector<int32_t> h;
  if (g_prof_mask == 0) return h;
  h.resize(E + 1);
  if (hipMemcpyAsync(h.data(), d_offsets, (E + 1) * sizeof(int32_t), hipMemcpyDeviceToHost, s) !=
          hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess) {
    (void)hipGetLastError();
    h.clear();
  }
  return h;
}
// experts with rows in [p0, p1), and those of them whose dW the chunk adds to
struct ChunkExperts {
  double in = 0, add = 0;
};
ChunkExperts chunk_experts(const std::vector<int32_t>& off, int E, int64_t p0, int64_t p1,
                           bool accumulate) {
  ChunkExperts c;
  if (off.empty()) {  // unknown: every expert, read and written
    c.in = c.add = E;
    return c;
  }
  for (int e = 0; e < E; ++e) {
    const int64_t lo = off[e], hi = off[e + 1];
    if (std::min(hi, p1) > std::max(lo, p0)) {
      c.in += 1;
      if (accumulate || lo < p0) c.add += 1;
    }
  }
  return c;
}

// The expert-ordered forward: the layer's dispatch, then per chunk its view,
// FC1 and FC2 over its rows, and the combine of its rows into Y.  With
// `fixed_ws` the tables and the chunk buffers are carved from it.
int moe_fwd_experts(const memfine_shape& S, int32_t chunks, const void* d_X, const int32_t* d_idx,
                    const float* d_gates, const void* d_W1, const void* d_W2, void* d_Y,
                    const memfine_allocator* alloc, void* fixed_ws,
                    const memfine_launch_options& opt, hipStream_t s) {
  const int64_t N = S.T * (int64_t)S.k, C = expert_chunks(S, chunks);
  const double es = (double)elem_bytes(S), hF = (double)S.h * S.F;
  Layout Lm;
  layout(S, N, -1, true, true, Lm);
  Layout Lmax;
  layout(S, (N + C - 1) / C, MEMFINE_PASS_FWD, false, false, Lmax);
  // The first chunk's buffers are taken before the tables, so that with the
  // library's own allocator the chunks reuse the stream's cached block.
  void* ws = fixed_ws ? (char*)fixed_ws + Lm.total : ws_alloc(alloc, (size_t)Lmax.total, s);
  if (!ws) return MEMFINE_ERR_OOM;
  void* meta = fixed_ws ? fixed_ws : ws_alloc(alloc, (size_t)Lm.total, s);
  if (!meta) {
    if (!fixed_ws) ws_release(alloc, ws, (size_t)Lmax.total, s);
    return MEMFINE_ERR_OOM;
  }
  const ChunkBuffers mb = carve(meta, Lm);
  hipError_t err;
  {
    KernelTimer kt(MEMFINE_K_DISPATCH, s, 0.0, dispatch_work(N).bytes);
    err = launch_dispatch(d_idx, d_gates, 0, (int)N, S.E, S.k, mb.m, s);
  }
  const std::vector<int32_t> hoff =
      err == hipSuccess ? offsets_for_profile(mb.m.offsets, S.E, s) : std::vector<int32_t>();
  for (int64_t c = 0; c < C && err == hipSuccess; ++c) {
    const int64_t p0 = expert_chunk_row(S, C, c), p1 = expert_chunk_row(S, C, c + 1);
    const int64_t n = p1 - p0;
    if (n == 0) continue;
    Layout L;
    layout(S, n, MEMFINE_PASS_FWD, false, false, L);
    if (!ws) ws = ws_alloc(alloc, (size_t)Lmax.total, s);
    if (!ws) {
      ws_release(alloc, meta, (size_t)Lm.total, s);
      return MEMFINE_ERR_OOM;
    }
    const ChunkBuffers cb = carve(ws, L);
    err = launch_chunk_view(mb.m.offsets, S.E, (int)p0, (int)p1, c == 0, 0, mb.off_c, mb.order_c,
                            mb.wexp, mb.wmode, s);
    GemmArgs g = gemm_args(S, n, cb, opt);
    g.offsets = mb.off_c;
    g.order = mb.order_c;
    g.tok_of_row = mb.m.tok_of_row + p0;
    g.gate_of_row = mb.m.gate_of_row + p0;
    g.X = d_X;
    g.W1 = d_W1;
    g.W2 = d_W2;
    const double nd = (double)n, Ec = chunk_experts(hoff, S.E, p0, p1, false).in;
    if (err == hipSuccess) {
      KernelTimer kt(MEMFINE_K_FC1, s, 4.0 * nd * hF, es * (nd * S.h + 2.0 * Ec * hF + nd * S.F));
      err = launch_fc1_fwd(g, s);
    }
    if (err == hipSuccess) {
      KernelTimer kt(MEMFINE_K_FC2, s, 2.0 * nd * hF, es * (nd * S.F + Ec * hF + nd * S.h));
      err = launch_fc2_fwd(g, s);
    }
    if (err == hipSuccess) {
      // the chunk's rows once, and a read and write of (at most) one Y row each
      KernelTimer kt(MEMFINE_K_COMBINE, s, 2.0 * nd * S.h,
                     es * 3.0 * nd * S.h + 4.0 * (double)N + 4.0 * nd);
      err = launch_combine_rows(S.dtype, cb.y, mb.m.row_of_slot, d_gates, S.T, S.h, S.k, (int)p0,
                                (int)p1, d_Y, s);
    }
    if (!fixed_ws) {  // the chunk's buffers go back before the next chunk takes its own
      ws_release(alloc, ws, (size_t)Lmax.total, s);
      ws = nullptr;
    }
  }
  if (!fixed_ws) {
    if (ws) ws_release(alloc, ws, (size_t)Lmax.total, s);
    ws_release(alloc, meta, (size_t)Lm.total, s);
  }
  return err == hipSuccess ? MEMFINE_OK : MEMFINE_ERR_HIP;
}

int moe_fwd_impl(const memfine_shape* shape, int32_t chunks, const void* d_X,
                 const int32_t* d_idx, const float* d_gates, const void* d_W1, const void* d_W2,
                 void* d_Y, const memfine_allocator* alloc, void* fixed_ws,
                 const memfine_launch_options& opt, void* stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if (chunks < 1) return MEMFINE_ERR_INVALID_ARG;
  const memfine_shape& S = *shape;
  if (S.T == 0) return MEMFINE_OK;
  if (!d_X || !d_idx || !d_gates || !d_W1 || !d_W2 || !d_Y) return MEMFINE_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  if (opt.chunk_order == MEMFINE_CHUNK_EXPERTS)
    return moe_fwd_experts(S, chunks, d_X, d_idx, d_gates, d_W1, d_W2, d_Y, alloc, fixed_ws, opt,
                           s);
  const int64_t C = std::min<int64_t>(chunks, S.T);
  const double es = (double)elem_bytes(S);
  for (int64_t i = 0; i < C; ++i) {
    const int64_t t0 = i * S.T / C, t1 = (i + 1) * S.T / C;
    const int64_t tokens = t1 - t0, n = tokens * S.k;
    if (n == 0) continue;
    Layout L;
    chunk_layout(S, n, MEMFINE_PASS_FWD, L);
    void* ws = fixed_ws ? fixed_ws : ws_alloc(alloc, (size_t)L.total, s);
    if (!ws) return MEMFINE_ERR_OOM;
    const ChunkBuffers cb = carve(ws, L);
    GemmArgs g = gemm_args(S, n, cb, opt);
    g.X = d_X;
    g.W1 = d_W1;
    g.W2 = d_W2;
    hipError_t err;
    {
      KernelTimer kt(MEMFINE_K_DISPATCH, s, 0.0, dispatch_work(n).bytes);
      err = launch_dispatch(d_idx, d_gates, t0 * S.k, (int)n, S.E, S.k, cb.m, s);
    }
    const double hF = (double)S.h * S.F, nd = (double)n, Ed = S.E;
    if (err == hipSuccess) {
      KernelTimer kt(MEMFINE_K_FC1, s, 4.0 * nd * hF,
                     es * (tokens * (double)S.h + 2.0 * Ed * hF + nd * S.F));
      err = launch_fc1_fwd(g, s);
    }
    if (err == hipSuccess) {
      KernelTimer kt(MEMFINE_K_FC2, s, 2.0 * nd * hF, es * (nd * S.F + Ed * hF + nd * S.h));
      err = launch_fc2_fwd(g, s);
    }
    if (err == hipSuccess) {
      KernelTimer kt(MEMFINE_K_COMBINE, s, 2.0 * nd * S.h,
                     es * (nd * S.h + tokens * (double)S.h) + 8.0 * nd);
      err = launch_combine(S.dtype, cb.y, cb.m.row_of_slot, d_gates, t0, (int)tokens, S.h, S.k,
                           d_Y, s);
    }
    if (!fixed_ws) ws_release(alloc, ws, (size_t)L.total, s);
    if (err != hipSuccess) return MEMFINE_ERR_HIP;
  }
  return MEMFINE_OK;
}
}  // namespace

namespace {
// Algorithmic work of a chunk's backward GEMMs (flops, bytes).
struct BwdWork {
  Work fc2d, rec, fc2w, fc1w, fc1d;
};
// A chunk's backward GEMMs, after its dispatch: FC2 dgrad, the FC1
// recomputation with the SwiGLU backward, the two weight gradients and the
// FC1 dgrad (the last three on side streams, or in one launch, as the
// launch options say).
hipError_t bwd_gemms(const GemmArgs& g, const ChunkBuffers& cb, const memfine_launch_options& opt,
                     const BwdWork& w, hipStream_t s) {
  hipError_t err;
  {  // dA = dY W2 of the chunk's rows (into ag)
    KernelTimer kt(MEMFINE_K_FC2_DGRAD, s, w.fc2d.flops, w.fc2d.bytes);
    err = launch_fc2_dgrad(g, s);
  }
  if (err == hipSuccess) {  // recompute F_w(X_i)'s FC1; SwiGLU backward: du, g * a, dg partials
    KernelTimer kt(MEMFINE_K_FC1_RECOMP, s, w.rec.flops, w.rec.bytes);
    err = launch_fc1_recompute(g, s);
  }
  SideStreams* ss = (!opt.pair && opt.streams) ? side_streams() : nullptr;
  if (ss) {
    // The two weight gradients and the FC1 dgrad read what the recompute
    // wrote and write disjoint outputs (dW1, dW2, the chunk's dX rows).
    // The weight gradients run on side streams beside the dgrad, so that
    // their dW read-modify-write phases overlap the dgrad's matrix work;
    // the caller's stream joins them before the unpermute (and before
    // the chunk's buffers are released, also after an error).
    std::lock_guard<std::mutex> lk(ss->mu);
    bool forked = false;
    if (err == hipSuccess) err = hipEventRecord(ss->fork, s);
    if (err == hipSuccess) {
      forked = true;
      for (int j = 0; j < 2 && err == hipSuccess; ++j) err = hipStreamWaitEvent(ss->s[j], ss->fork, 0);
    }
    if (err == hipSuccess) {
      KernelTimer kt(MEMFINE_K_FC1_WGRAD, ss->s[0], w.fc1w.flops, w.fc1w.bytes);
      GemmArgs gw = g;
      gw.tile_ctr = cb.ctr;
      err = launch_fc1_wgrad(gw, ss->s[0]);
    }
    if (err == hipSuccess) {
      KernelTimer kt(MEMFINE_K_FC2_WGRAD, ss->s[1], w.fc2w.flops, w.fc2w.bytes);
      GemmArgs gw = g;
      gw.tile_ctr = cb.ctr + 1;
      err = launch_fc2_wgrad(gw, ss->s[1]);
    }
    if (err == hipSuccess) {
      KernelTimer kt(MEMFINE_K_FC1_DGRAD, s, w.fc1d.flops, w.fc1d.bytes);
      err = launch_fc1_dgrad(g, s);
    }
    if (forked) {
      for (int j = 0; j < 2; ++j) {
        const hipError_t e1 = hipEventRecord(ss->join[j], ss->s[j]);
        const hipError_t e2 = e1 == hipSuccess ? hipStreamWaitEvent(s, ss->join[j], 0) : e1;
        if (e2 != hipSuccess) {
          // the caller's stream cannot be ordered after the side stream:
          // wait for it on the host before the buffers are released
          (void)hipStreamSynchronize(ss->s[j]);
          if (err == hipSuccess) err = e2;
        }
      }
    }
    return err;
  }
  if (err == hipSuccess) {
    KernelTimer kt(MEMFINE_K_FC2_WGRAD, s, w.fc2w.flops, w.fc2w.bytes);
    GemmArgs gw = g;
    gw.tile_ctr = cb.ctr + 1;
    err = launch_fc2_wgrad(gw, s);
  }
  if (opt.pair) {
    if (err == hipSuccess) {
      KernelTimer kt(MEMFINE_K_FC1_BWD, s, w.fc1d.flops + w.fc1w.flops,
                     w.fc1d.bytes + w.fc1w.bytes);
      err = launch_fc1_dgrad_wgrad(g, s);
    }
  } else {
    if (err == hipSuccess) {
      KernelTimer kt(MEMFINE_K_FC1_WGRAD, s, w.fc1w.flops, w.fc1w.bytes);
      GemmArgs gw = g;
      gw.tile_ctr = cb.ctr;
      err = launch_fc1_wgrad(gw, s);
    }
    if (err == hipSuccess) {
      KernelTimer kt(MEMFINE_K_FC1_DGRAD, s, w.fc1d.flops, w.fc1d.bytes);
      err = launch_fc1_dgrad(g, s);
    }
  }
  return err;
}

// The expert-ordered backward: the layer's dispatch, then per chunk its view
// (with each expert's dW mode: the chunk holding an expert's first rows
// overwrites its dW unless the caller accumulates, later chunks add), the
// backward GEMMs over its rows, and the unpermute of its rows into dX.
int moe_bwd_experts(const memfine_shape& S, int32_t chunks, const void* d_X, const int32_t* d_idx,
                    const float* d_gates, const void* d_W1, const void* d_W2, const void* d_dY,
                    void* d_dX, float* d_dW1, float* d_dW2, float* d_dgates,
                    int32_t accumulate_dW, const memfine_allocator* alloc,
                    const memfine_launch_options& opt, hipStream_t s) {
  const int64_t N = S.T * (int64_t)S.k, C = expert_chunks(S, chunks);
  const double es = (double)elem_bytes(S), hF = (double)S.h * S.F;
  Layout Lm;
  layout(S, N, -1, true, true, Lm);
  Layout Lmax;
  layout(S, (N + C - 1) / C, MEMFINE_PASS_BWD, false, false, Lmax);
  // the first chunk's buffers before the tables (as in the forward)
  void* ws = ws_alloc(alloc, (size_t)Lmax.total, s);
  if (!ws) return MEMFINE_ERR_OOM;
  void* meta = ws_alloc(alloc, (size_t)Lm.total, s);
  if (!meta) {
    ws_release(alloc, ws, (size_t)Lmax.total, s);
    return MEMFINE_ERR_OOM;
  }
  const ChunkBuffers mb = carve(meta, Lm);
  hipError_t err;
  {
    KernelTimer kt(MEMFINE_K_DISPATCH, s, 0.0, dispatch_work(N).bytes);
    err = launch_dispatch(d_idx, d_gates, 0, (int)N, S.E, S.k, mb.m, s);
  }
  const std::vector<int32_t> hoff =
      err == hipSuccess ? offsets_for_profile(mb.m.offsets, S.E, s) : std::vector<int32_t>();
  for (int64_t c = 0; c < C && err == hipSuccess; ++c) {
    const int64_t p0 = expert_chunk_row(S, C, c), p1 = expert_chunk_row(S, C, c + 1);
    const int64_t n = p1 - p0;
    if (n == 0) continue;
    Layout L;
    layout(S, n, MEMFINE_PASS_BWD, false, false, L);
    if (!ws) ws = ws_alloc(alloc, (size_t)Lmax.total, s);
    if (!ws) {
      ws_release(alloc, meta, (size_t)Lm.total, s);
      return MEMFINE_ERR_OOM;
    }
    const ChunkBuffers cb = carve(ws, L);
    err = launch_chunk_view(mb.m.offsets, S.E, (int)p0, (int)p1, c == 0, accumulate_dW, mb.off_c,
                            mb.order_c, mb.wexp, mb.wmode, s);
    GemmArgs g = gemm_args(S, n, cb, opt);
    g.offsets = mb.off_c;
    g.order = mb.order_c;
    g.tok_of_row = mb.m.tok_of_row + p0;
    g.gate_of_row = mb.m.gate_of_row + p0;
    g.wmode = mb.wmode;
    g.wexperts = mb.wexp;
    g.accumulate = accumulate_dW;
    g.X = d_X;
    g.dY = d_dY;
    g.W1 = d_W1;
    g.W2 = d_W2;
    g.dW1 = d_dW1;
    g.dW2 = d_dW2;
    const ChunkExperts ce = chunk_experts(hoff, S.E, p0, p1, accumulate_dW != 0);
    const double nd = (double)n;
    // dW: every element of the chunk's experts written, and read where added
    const double dw = 4.0 * ce.in + 4.0 * ce.add;
    const BwdWork w = {
        {2.0 * nd * hF, es * (nd * S.h + ce.in * hF + nd * S.F)},
        {4.0 * nd * hF, es * (nd * S.h + 2.0 * ce.in * hF + 4.0 * nd * S.F) + 4.0 * nd * g.P},
        {2.0 * nd * hF, es * (nd * S.h + nd * S.F) + dw * hF},
        {4.0 * nd * hF, es * (2.0 * nd * S.F + nd * S.h) + 2.0 * dw * hF},
        {4.0 * nd * hF, es * (2.0 * nd * S.F + 2.0 * ce.in * hF + nd * S.h)}};
    if (err == hipSuccess) err = bwd_gemms(g, cb, opt, w, s);
    if (err == hipSuccess) {
      KernelTimer kt(MEMFINE_K_UNPERMUTE, s, nd * S.h,
                     es * 3.0 * nd * S.h + 4.0 * (double)N + 4.0 * nd * (g.P + 1));
      err = launch_unpermute_rows(S.dtype, cb.dxp, cb.dgp, g.P, mb.m.row_of_slot, S.T, S.h, S.k,
                                  (int)p0, (int)p1, d_dX, d_dgates, s);
    }
    ws_release(alloc, ws, (size_t)Lmax.total, s);
    ws = nullptr;
  }
  if (ws) ws_release(alloc, ws, (size_t)Lmax.total, s);
  ws_release(alloc, meta, (size_t)Lm.total, s);
  return err == hipSuccess ? MEMFINE_OK : MEMFINE_ERR_HIP;
}
}  // namespace

extern "C" {

int memfine_moe_bwd(const memfine_shape* shape, int32_t chunks, const void* d_X,
                    const int32_t* d_idx, const float* d_gates, const void* d_W1,
                    const void* d_W2, const void* d_dY, void* d_dX, float* d_dW1, float* d_dW2,
                    float* d_dgates, int32_t accumulate_dW, const memfine_allocator* alloc,
                    void* stream) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if (chunks < 1 || (accumulate_dW != 0 && accumulate_dW != 1)) return MEMFINE_ERR_INVALID_ARG;
  const memfine_shape& S = *shape;
  if (!d_W1 || !d_W2 || !d_dW1 || !d_dW2) return MEMFINE_ERR_INVALID_ARG;
  if (S.T > 0 && (!d_X || !d_idx || !d_gates || !d_dY || !d_dX || !d_dgates))
    return MEMFINE_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  const double es = (double)elem_bytes(S);
  const double hF = (double)S.h * S.F, Ed = S.E;
  if (S.T == 0) {
    if (accumulate_dW) return MEMFINE_OK;
    // no rows at all: the weight gradients are zero
    const int64_t w1 = (int64_t)S.E * 2 * S.F * S.h, w2 = (int64_t)S.E * S.h * S.F;
    hipError_t err = launch_fill_i32((int32_t*)d_dW1, w1, 0, s);
    if (err == hipSuccess) err = launch_fill_i32((int32_t*)d_dW2, w2, 0, s);
    return hip_status(err);
  }
  const memfine_launch_options opt = launch_options();
  if (opt.chunk_order == MEMFINE_CHUNK_EXPERTS)
    return moe_bwd_experts(S, chunks, d_X, d_idx, d_gates, d_W1, d_W2, d_dY, d_dX, d_dW1, d_dW2,
                           d_dgates, accumulate_dW, alloc, opt, s);
  const int64_t C = std::min<int64_t>(chunks, S.T);
  bool first = true;
  for (int64_t i = 0; i < C; ++i) {
    const int64_t t0 = i * S.T / C, t1 = (i + 1) * S.T / C;
    const int64_t tokens = t1 - t0, n = tokens * S.k;
    if (n == 0) continue;
    Layout L;
    chunk_layout(S, n, MEMFINE_PASS_BWD, L);
    void* ws = ws_alloc(alloc, (size_t)L.total, s);
    if (!ws) return MEMFINE_ERR_OOM;
    const ChunkBuffers cb = carve(ws, L);
    GemmArgs g = gemm_args(S, n, cb, opt);
    g.X = d_X;
    g.dY = d_dY;
    g.W1 = d_W1;
    g.W2 = d_W2;
    g.dW1 = d_dW1;
    g.dW2 = d_dW2;
    g.accumulate = (accumulate_dW || !first) ? 1 : 0;
    const double nd = (double)n, td = (double)tokens;
    const double dw_rmw = g.accumulate ? 8.0 : 4.0;
    hipError_t err;
    {
      KernelTimer kt(MEMFINE_K_DISPATCH, s, 0.0, dispatch_work(n).bytes);
      err = launch_dispatch(d_idx, d_gates, t0 * S.k, (int)n, S.E, S.k, cb.m, s);
    }
    const BwdWork w = {
        {2.0 * nd * hF, es * (td * S.h + Ed * hF + nd * S.F)},
        {4.0 * nd * hF, es * (td * S.h + 2.0 * Ed * hF + 4.0 * nd * S.F) + 4.0 * nd * g.P},
        {2.0 * nd * hF, es * (td * S.h + nd * S.F) + dw_rmw * Ed * hF},
        {4.0 * nd * hF, es * (2.0 * nd * S.F + td * S.h) + 2.0 * dw_rmw * Ed * hF},
        {4.0 * nd * hF, es * (2.0 * nd * S.F + 2.0 * Ed * hF + nd * S.h)}};
    if (err == hipSuccess) err = bwd_gemms(g, cb, opt, w, s);
    if (err == hipSuccess) {
      KernelTimer kt(MEMFINE_K_UNPERMUTE, s, nd * S.h,
                     es * (nd * S.h + td * S.h) + 4.0 * nd * (g.P + 2));
      err = launch_unpermute(S.dtype, cb.dxp, cb.dgp, g.P, cb.m.row_of_slot, t0, (int)tokens,
                             S.h, S.k, d_dX, d_dgates, s);
    }
    ws_release(alloc, ws, (size_t)L.total, s);
    if (err != hipSuccess) return MEMFINE_ERR_HIP;
    first = false;
  }
  return MEMFINE_OK;
}

// ------------------------------------------------------------------ router
namespace {
// Width of the dense dz rows fed to the split-K weight gradient: E rounded
// up to 32 (the GEMM's M; the partials it writes scale with it).
int router_ep(int E) { return (E + 31) / 32 * 32; }

int check_router(const memfine_shape* shape) {
  int rc = check_shape(shape);
  if (rc) return rc;
  if (shape->k > 16 || shape->k > shape->E || shape->E > 256) return MEMFINE_ERR_UNSUPPORTED;
  return MEMFINE_OK;
}
}  // namespace

int memfine_router_fwd(const memfine_shape* shape, const void* d_X, const void* d_Wr,
                       int32_t* d_idx, float* d_gates, float* d_logits, void* stream) {
  int rc = check_router(shape);
  if (rc) return rc;
  const memfine_shape& S = *shape;
  if (S.T == 0) return MEMFINE_OK;
  if (!d_X || !d_Wr || !d_idx || !d_gates) return MEMFINE_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  const double es = (double)elem_bytes(S), Td = (double)S.T;
  KernelTimer kt(MEMFINE_K_ROUTER_FWD, s, 2.0 * Td * S.h * S.E,
                 es * (Td * S.h + (double)S.E * S.h) + 8.0 * Td * S.k +
                     (d_logits ? 4.0 * Td * S.E : 0.0));
  if (S.E <= 64 || S.E % 32 != 0)
    return hip_status(launch_router_fwd(S.dtype, d_X, d_Wr, S.T, S.h, S.E, S.k, d_idx, d_gates,
                                        d_logits, s));
  // Wide routers: the logits as a grouped GEMM on 256-token tiles (each tile
  // reads Wr once; one fused kernel per 32 tokens read it T / 32 times), then
  // their top-k.  Working memory: the {0, T} row offsets of the GEMM's one
  // "expert" and, without d_logits, the logits themselves.
  const int64_t off_bytes = 256, lg_bytes = d_logits ? 0 : S.T * (int64_t)S.E * 4;
  void* ws = ws_alloc(nullptr, (size_t)(off_bytes + lg_bytes), s);
  if (!ws) return MEMFINE_ERR_OOM;
  int32_t* off = (int32_t*)ws;
  float* lg = d_logits ? d_logits : (float*)((char*)ws + off_bytes);
  hipError_t err = launch_fill_i32(off, 1, 0, s);
  if (err == hipSuccess) err = launch_fill_i32(off + 1, 1, (int32_t)S.T, s);
  if (err == hipSuccess) {
    const memfine_launch_options opt = launch_options();
    GemmArgs g = {};
    g.dtype = S.dtype;
    g.n = (int)S.T;
    g.E = 1;
    g.h = S.E;   // output columns: the logits
    g.F = S.h;   // reduction: the hidden size
    g.offsets = off;
    g.a = const_cast<void*>(d_X);
    g.W2 = d_Wr;
    g.y = lg;
    g.T_h_bytes = S.T * (int64_t)S.h * elem_bytes(S);
    g.tile_override = opt.tile;
    g.raster = opt.raster;
    g.cus = device_cus();
    g.split_tail = opt.split_tail;
    err = launch_router_logits(g, s);
  }
  if (err == hipSuccess) err = launch_router_topk(lg, S.T, S.E, S.k, d_idx, d_gates, s);
  ws_release(nullptr, ws, (size_t)(off_bytes + lg_bytes), s);
  return hip_status(err);
}

int memfine_router_bwd(const memfine_shape* shape, const void* d_X, const void* d_Wr,
                       const int32_t* d_idx, const float* d_gates, const float* d_dgates,
                       void* d_dX, float* d_dWr, int32_t accumulate_dX, int32_t accumulate_dWr,
                       const memfine_allocator* alloc, void* stream) {
  int rc = check_router(shape);
  if (rc) return rc;
  if ((accumulate_dX != 0 && accumulate_dX != 1) || (accumulate_dWr != 0 && accumulate_dWr != 1))
    return MEMFINE_ERR_INVALID_ARG;
  const memfine_shape& S = *shape;
  if (!d_Wr || !d_dWr) return MEMFINE_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  if (S.T == 0) {
    if (accumulate_dWr) return MEMFINE_OK;
    return hip_status(launch_fill_i32((int32_t*)d_dWr, (int64_t)S.E * S.h, 0, s));
  }
  if (!d_X || !d_idx || !d_gates || !d_dgates || !d_dX) return MEMFINE_ERR_INVALID_ARG;
  const int64_t es = elem_bytes(S), T = S.T;
  const int EP = router_ep(S.E);
  // split-K: enough row ranges for about 256 workgroups, each at least 256 rows
  const int ntn = (S.h + 255) / 256;
  const int64_t want = (256 + ntn - 1) / ntn, most = std::max<int64_t>(1, T / 256);
  const int splits = (int)std::max<int64_t>(1, std::min(want, most));
  // dX (+)= dz Wr: per token in the dz kernel, or (E % 64 == 0, so that the
  // dense dz rows are whole K tiles) as a grouped GEMM from D, which reads
  // Wr once per 256-token tile instead of k rows of it per token
  const bool gemm_dx = S.E % 64 == 0;
  const int64_t o_meta = align256(T * EP * es);
  const int64_t o_order = o_meta + align256((splits + 1) * 4);
  const int64_t o_tok = o_order + align256(splits * 4);
  const int64_t o_off1 = o_tok + align256(T * 4);
  const int64_t o_part = o_off1 + 256;
  const int64_t total = o_part + align256((int64_t)splits * EP * S.h * 4);
  char* ws = (char*)ws_alloc(alloc, (size_t)total, s);
  if (!ws) return MEMFINE_ERR_OOM;
  void* D = ws;
  int32_t* offsets = (int32_t*)(ws + o_meta);
  int32_t* order = (int32_t*)(ws + o_order);
  int32_t* tok = (int32_t*)(ws + o_tok);
  int32_t* off1 = (int32_t*)(ws + o_off1);
  float* part = (float*)(ws + o_part);
  const double Td = (double)T, hd = (double)S.h;
  hipError_t err = launch_router_split_meta(offsets, order, tok, T, splits, s);
  if (err == hipSuccess) {
    KernelTimer kt(MEMFINE_K_ROUTER_BWD_DX, s, 2.0 * Td * (gemm_dx ? EP : S.k) * hd,
                   (double)es * (Td * hd * (accumulate_dX ? 2.0 : 1.0) +
                                 Td * EP * (gemm_dx ? 2.0 : 1.0) + (double)S.E * hd) +
                       12.0 * Td * S.k);
    err = launch_router_bwd_dx(S.dtype, d_Wr, d_idx, d_gates, d_dgates, T, S.h, S.E, S.k,
                               EP, accumulate_dX, gemm_dx ? 0 : 1, d_dX, D, s);
    if (err == hipSuccess && gemm_dx) {
      err = launch_fill_i32(off1, 1, 0, s);
      if (err == hipSuccess) err = launch_fill_i32(off1 + 1, 1, (int32_t)T, s);
      if (err == hipSuccess) {
        const memfine_launch_options opt = launch_options();
        GemmArgs g = {};
        g.dtype = S.dtype;
        g.n = (int)T;
        g.E = 1;
        g.h = EP;    // reduction: the dense dz row
        g.F = S.h;   // output columns: the hidden size
        g.offsets = off1;
        g.tok_of_row = tok;   // the identity
        g.dY = D;
        g.W2 = d_Wr;
        g.ag = d_dX;
        g.accumulate = accumulate_dX;
        g.T_h_bytes = T * (int64_t)EP * es;
        g.tile_override = opt.tile;
        g.raster = opt.raster;
        g.cus = device_cus();
        g.split_tail = opt.split_tail;
        err = launch_router_dx(g, s);
      }
    }
  }
  if (err == hipSuccess) {
    // dWr partials: the grouped weight-gradient GEMM over `splits` row ranges
    // of dz^T X (M = EP rows of the dense dz, N = h, K = the range)
    GemmArgs g = {};
    g.dtype = S.dtype;
    g.n = (int)T;
    g.E = splits;
    g.h = S.h;
    g.F = EP / 2;
    g.offsets = offsets;
    g.order = order;
    g.tok_of_row = tok;
    g.X = d_X;
    g.u = D;
    g.dW1 = part;
    g.accumulate = 0;
    g.T_h_bytes = T * (int64_t)S.h * es;
    g.cus = device_cus();
    KernelTimer kt(MEMFINE_K_ROUTER_WGRAD, s, 2.0 * Td * EP * hd,
                   (double)es * (Td * hd + Td * EP) + 4.0 * splits * EP * hd);
    err = launch_fc1_wgrad(g, s);
  }
  if (err == hipSuccess) {
    KernelTimer kt(MEMFINE_K_ROUTER_REDUCE, s, 0.0,
                   4.0 * (double)S.E * hd * (splits + (accumulate_dWr ? 2.0 : 1.0)));
    err = launch_router_reduce(part, splits, EP, S.E, S.h, accumulate_dWr, d_dWr, s);
  }
  ws_release(alloc, ws, (size_t)total, s);
  return hip_status(err);
}

int memfine_profile_begin(uint32_t mask) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto& r : g_prof) {
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  g_prof.clear();
  g_prof_mask = mask;
  return MEMFINE_OK;
}

int memfine_profile_end(memfine_kernel_stat* out) {
  if (!out) return MEMFINE_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_mask = 0;
  for (int i = 0; i < MEMFINE_K_NUM; ++i) out[i] = memfine_kernel_stat{0, 0.0, 0.0, 0.0};
  int rc = MEMFINE_OK;
  for (auto& r : g_prof) {
    float ms = 0.f;
    if (hipEventSynchronize(r.stop) != hipSuccess ||
        hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess)
      rc = MEMFINE_ERR_HIP;
    memfine_kernel_stat& st = out[r.id];
    st.launches += 1;
    st.total_ms += ms;
    st.flops += r.flops;
    st.bytes += r.bytes;
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  g_prof.clear();
  return rc;
}

}  // extern "C"
