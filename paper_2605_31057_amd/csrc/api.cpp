// api.cpp -- the C ABI declared in include/lvsa.h: argument checks, handle
// management and dispatch to the builders and kernels.
#include <climits>
#include <mutex>
#include <new>

#include "internal.h"

namespace lvsa {

lvsa_status resolve_frames(int32_t T, int32_t step, const lvsa_params* p,
                           FrameCfg* out) {
  if (!p || !out) return LVSA_EINVAL;
  if (T < 1 || T > LVSA_MAX_FRAMES || step < 0) return LVSA_EINVAL;
  if (p->window < 0 || p->window > LVSA_MAX_FRAMES) return LVSA_EINVAL;
  if (p->window_mode < LVSA_WINDOW_BASIC || p->window_mode > LVSA_WINDOW_EXPANDED)
    return LVSA_EINVAL;
  if ((p->rotate != 0 && p->rotate != 1) || (p->tie_high != 0 && p->tie_high != 1))
    return LVSA_EINVAL;
  if (p->tper < 0) return LVSA_EINVAL;
  if (p->extra_anchors < 0 || p->extra_anchors > LVSA_MAX_FRAMES) return LVSA_EINVAL;
  if (p->text_tokens < 0) return LVSA_EINVAL;
  int32_t tper = p->tper;
  if (tper == 0) {
    // Sec. 2, budget paragraph: T_per = ceil(T / (C - (2W+1))), for C > 2W+1;
    // dedicated initial anchors leave the budget first.
    const int64_t spare = (int64_t)p->budget_frames - (2 * (int64_t)p->window + 1) -
                          p->extra_anchors;
    if (p->budget_frames <= 0 || spare <= 0) return LVSA_EINVAL;
    tper = ceil_div(T, (int32_t)spare);
  }
  FrameCfg c;
  c.T = T;
  c.W = p->window;
  c.tper = tper;
  c.k = ceil_div(T, tper);
  // Eq. 3 reduces s mod T_per, then every anchor mod T (only the first
  // reduction matters when T_per <= T).
  c.s0 = p->rotate ? (step % tper) % T : 0;
  c.mode = p->window_mode;
  c.rotate = p->rotate;
  c.tie_high = p->tie_high;
  c.extra = p->extra_anchors;
  c.text = p->text_tokens;
  c.g = anchors_below(c, T);
  *out = c;
  return LVSA_OK;
}

lvsa_status check_mask_shape(int32_t T, int32_t P, int32_t B, int32_t L) {
  if (T < 1 || P < 1 || B < 1 || B > (1 << 20) || L < 0) return LVSA_EINVAL;
  const int64_t N = (int64_t)T * P + L;
  if (N + B > INT32_MAX) return LVSA_EINVAL;
  const int64_t nb = (N + B - 1) / B;
  if (nb * nb > INT32_MAX) return LVSA_EINVAL;  // nnz must fit row_ptr
  return LVSA_OK;
}

// Tile-counter pool (lvsa.h, "Tile counters").  Per device: sets of
// kTileCounters 64-bit words in chunks of device memory.  An eager launch
// takes a set whose event (recorded behind the set's last launch) has
// completed; a launch under stream capture takes a set no launch has used
// and keeps it, because the graph replays it later (no event can be queried
// or recorded during a capture).  Sets are zeroed on the launch stream by
// the attention launch itself, so their contents never matter here.
namespace {

constexpr int kMaxDevices = 64;
constexpr int32_t kChunkSets = 256;   // 16 KB per chunk

struct CounterSet {
  uint64_t* counters = nullptr;
  hipEvent_t done = nullptr;   // created on the first eager release
  bool busy = false;           // between acquire and release
  bool kept = false;           // recorded into a graph: never handed out again
  bool used = false;           // handed out at least once
};

struct CounterPool {
  std::mutex mu;
  std::vector<CounterSet> sets;
  int32_t next = 0;
};

CounterPool g_pools[kMaxDevices];

lvsa_status grow_pool(CounterPool& pool) {
  void* chunk = nullptr;
  if (hipMalloc(&chunk, sizeof(uint64_t) * kTileCounters * kChunkSets) != hipSuccess)
    return LVSA_ENOMEM;
  for (int32_t i = 0; i < kChunkSets; ++i) {
    CounterSet cs;
    cs.counters = (uint64_t*)chunk + (size_t)kTileCounters * i;
    pool.sets.push_back(cs);
  }
  return LVSA_OK;
}

}  // namespace

lvsa_status acquire_counters(hipStream_t stream, CounterLease* lease) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return LVSA_EDEVICE;
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cap) != hipSuccess) return LVSA_EDEVICE;
  const bool capturing = cap != hipStreamCaptureStatusNone;
  CounterPool& pool = g_pools[dev];
  std::lock_guard<std::mutex> lock(pool.mu);
  try {
    if (pool.sets.empty()) {
      const lvsa_status st = grow_pool(pool);
      if (st != LVSA_OK) return st;
    }
    const int32_t n = (int32_t)pool.sets.size();
    int32_t pick = -1;
    for (int32_t d = 0; d < n && pick < 0; ++d) {
      const int32_t i = (pool.next + d) % n;
      CounterSet& cs = pool.sets[i];
      if (cs.busy || cs.kept) continue;
      if (capturing) {
        if (!cs.used) pick = i;
        continue;
      }
      if (cs.done) {
        const hipError_t q = hipEventQuery(cs.done);
        if (q == hipErrorNotReady) continue;
        if (q != hipSuccess) return LVSA_EDEVICE;
      }
      pick = i;
    }
    if (pick < 0) {
      const lvsa_status st = grow_pool(pool);
      if (st != LVSA_OK) return st;
      pick = n;
    }
    CounterSet& cs = pool.sets[pick];
    cs.busy = true;
    cs.used = true;
    pool.next = (pick + 1) % (int32_t)pool.sets.size();
    lease->device = dev;
    lease->slot = pick;
    lease->counters = cs.counters;
    lease->captured = capturing;
  } catch (const std::bad_alloc&) {
    return LVSA_ENOMEM;
  }
  return LVSA_OK;
}

void release_counters(const CounterLease& lease, hipStream_t stream) {
  if (lease.slot < 0) return;
  CounterPool& pool = g_pools[lease.device];
  std::lock_guard<std::mutex> lock(pool.mu);
  CounterSet& cs = pool.sets[lease.slot];
  cs.busy = false;
  if (lease.captured) {
    cs.kept = true;
    return;
  }
  if (!cs.done && hipEventCreateWithFlags(&cs.done, hipEventDisableTiming) != hipSuccess) {
    cs.done = nullptr;
    cs.kept = true;   // no way to know when the launch ends: never reuse it
    return;
  }
  if (hipEventRecord(cs.done, stream) != hipSuccess) cs.kept = true;
}

// Allocation-free launches (lvsa_attention_noalloc): the tile counters live
// in a file-scope device array, one copy per device, whose device address is
// looked up once per device (with that device current) and kept; the
// array's name in host code is only a stand-in for the symbol, never a device
// address.  Every such launch on a device uses the same counters, zeroed by
// the launch's own zeroing kernel, so such launches must not overlap on a
// device.
constexpr int kNoAllocCounterSets = 1;
static __device__ __align__(256) uint64_t scratch[kTileCounters * kNoAllocCounterSets];

namespace {

std::mutex g_scratch_mu;
uint64_t* g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's copy of `scratch` (looked up on the first
// call on a device, with that device current).
lvsa_status noalloc_counters(uint64_t** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return LVSA_EDEVICE;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
      return LVSA_EDEVICE;
    g_scratch_ptr[dev] = (uint64_t*)ptr;
  }
  *out = g_scratch_ptr[dev];
  return LVSA_OK;
}

}  // namespace

}  // namespace lvsa

struct lvsa_csr {
  int32_t n_tokens = 0;
  int32_t block = 0;
  int32_t n_blocks = 0;
  int32_t frame_tokens = 0;
  bool has_entry = false;          // token-exact entry words built
  std::vector<int32_t> row_ptr;
  std::vector<int32_t> col_idx;
  std::vector<uint32_t> entry;
  // Device copies, allocated in stream order on the first upload.
  int32_t* d_row_ptr = nullptr;
  int32_t* d_col_idx = nullptr;
  uint32_t* d_entry = nullptr;
  hipStream_t upload_stream = nullptr;   // stream of the last upload
  hipEvent_t uploaded = nullptr;         // recorded behind the last upload
};

namespace {

// Device copy of a host array: allocated in the order of `s` on the first
// upload (the handle's arrays never change size), then copied asynchronously
// on `s`.
template <typename T>
lvsa_status upload_array(const std::vector<T>& host, T** dev, hipStream_t s) {
  if (!*dev) {
    const size_t n = host.empty() ? 1 : host.size();
    if (hipMallocAsync((void**)dev, sizeof(T) * n, s) != hipSuccess) {
      *dev = nullptr;
      return LVSA_ENOMEM;
    }
  }
  if (!host.empty() &&
      hipMemcpyAsync(*dev, host.data(), sizeof(T) * host.size(), hipMemcpyHostToDevice,
                     s) != hipSuccess)
    return LVSA_EDEVICE;
  return LVSA_OK;
}

// Host arrays of freed handles, handed to the next builds: a denoising loop
// frees step s's mask and builds step s+1's of the same shape, and reusing
// the arrays' memory skips the page faults of fresh allocations (most of a
// rebuild's cost).  At most kHostPool sets are kept.
struct HostArrays {
  std::vector<int32_t> row_ptr, col_idx;
  std::vector<uint32_t> entry;
};
constexpr size_t kHostPool = 4;
std::mutex g_host_pool_mu;
std::vector<HostArrays> g_host_pool;

void take_host_arrays(lvsa_csr* h) {
  std::lock_guard<std::mutex> lock(g_host_pool_mu);
  if (g_host_pool.empty()) return;
  HostArrays& a = g_host_pool.back();
  h->row_ptr.swap(a.row_ptr);
  h->col_idx.swap(a.col_idx);
  h->entry.swap(a.entry);
  g_host_pool.pop_back();
}

void give_host_arrays(lvsa_csr* h) {
  std::lock_guard<std::mutex> lock(g_host_pool_mu);
  if (g_host_pool.size() >= kHostPool) return;
  try {
    g_host_pool.emplace_back();
  } catch (const std::bad_alloc&) {
    return;
  }
  HostArrays& a = g_host_pool.back();
  a.row_ptr.swap(h->row_ptr);
  a.col_idx.swap(h->col_idx);
  a.entry.swap(h->entry);
}

}  // namespace

using namespace lvsa;

extern "C" {

const char* lvsa_status_str(lvsa_status s) {
  switch (s) {
    case LVSA_OK: return "ok";
    case LVSA_EINVAL: return "invalid argument";
    case LVSA_ENOMEM: return "out of memory";
    case LVSA_EDEVICE: return "device error";
    case LVSA_EUNSUPPORTED: return "unsupported shape or layout";
    default: return "unknown status";
  }
}

int32_t lvsa_version(void) { return 20000; }

void lvsa_params_default(lvsa_params* p) {
  if (!p) return;
  p->budget_frames = 21;
  p->window = 6;
  p->tper = 0;
  p->window_mode = LVSA_WINDOW_EXPANDED;
  p->rotate = 1;
  p->tie_high = 0;
  p->extra_anchors = 0;
  p->text_tokens = 0;
}

lvsa_status lvsa_frame_sets(int32_t T, int32_t step, const lvsa_params* p,
                            int32_t* tper_out, int32_t* anchors,
                            int32_t* n_anchors, int32_t* win_lo,
                            int32_t* win_hi, int32_t* growth) {
  FrameCfg c;
  const lvsa_status st = resolve_frames(T, step, p, &c);
  if (st != LVSA_OK) return st;
  if (tper_out) *tper_out = c.tper;
  int32_t n = 0;
  for (int32_t t = 0; t < T; ++t)
    if (is_anchor(c, t)) {
      if (anchors) anchors[n] = t;
      ++n;
    }
  if (n_anchors) *n_anchors = n;
  for (int32_t t = 0; t < T; ++t) {
    int32_t lo, hi;
    const int32_t g = frame_window(c, t, &lo, &hi);
    if (win_lo) win_lo[t] = lo;
    if (win_hi) win_hi[t] = hi;
    if (growth) growth[t] = g;
  }
  return LVSA_OK;
}

lvsa_status lvsa_frame_window(int32_t T, int32_t step, const lvsa_params* p,
                              int32_t t, int32_t* lo, int32_t* hi,
                              int32_t* growth) {
  FrameCfg c;
  const lvsa_status st = resolve_frames(T, step, p, &c);
  if (st != LVSA_OK) return st;
  if (t < 0 || t >= T) return LVSA_EINVAL;
  int32_t l, h;
  const int32_t g = frame_window(c, t, &l, &h);
  if (lo) *lo = l;
  if (hi) *hi = h;
  if (growth) *growth = g;
  return LVSA_OK;
}

namespace {

lvsa_status build_mask_handle(int32_t T, int32_t P, int32_t B, int32_t step,
                              int32_t layer, const lvsa_params* p,
                              bool exact, lvsa_csr** out) {
  if (!out) return LVSA_EINVAL;
  *out = nullptr;
  if (layer < 0) return LVSA_EINVAL;
  FrameCfg c;
  lvsa_status st = resolve_frames(T, step, p, &c);
  if (st != LVSA_OK) return st;
  st = check_mask_shape(T, P, B, c.text);
  if (st != LVSA_OK) return st;
  const int64_t nb = (mask_tokens(c, P) + B - 1) / B;
  if (exact && !exact_supported(P, B, nb)) return LVSA_EUNSUPPORTED;
  lvsa_csr* h = new (std::nothrow) lvsa_csr();
  if (!h) return LVSA_ENOMEM;
  h->has_entry = exact;
  take_host_arrays(h);
  if (!exact) h->entry.clear();
  try {
    build_csr_host(c, P, B, &h->row_ptr, &h->col_idx, h->has_entry ? &h->entry : nullptr);
  } catch (const std::bad_alloc&) {
    delete h;
    return LVSA_ENOMEM;
  }
  h->n_tokens = (int32_t)mask_tokens(c, P);
  h->frame_tokens = P;
  h->block = B;
  h->n_blocks = (int32_t)h->row_ptr.size() - 1;
  *out = h;
  return LVSA_OK;
}

}  // namespace

lvsa_status lvsa_build_mask(int32_t T, int32_t P, int32_t B, int32_t step,
                            int32_t layer, const lvsa_params* p,
                            lvsa_csr** out) {
  return build_mask_handle(T, P, B, step, layer, p, false, out);
}

lvsa_status lvsa_build_exact_mask(int32_t T, int32_t P, int32_t B,
                                  int32_t step, int32_t layer,
                                  const lvsa_params* p, lvsa_csr** out) {
  return build_mask_handle(T, P, B, step, layer, p, true, out);
}

lvsa_status lvsa_csr_info(const lvsa_csr* csr, int32_t* n_q_blocks,
                          int32_t* n_kv_blocks, int64_t* nnz,
                          const int32_t** row_ptr, const int32_t** col_idx) {
  if (!csr) return LVSA_EINVAL;
  if (n_q_blocks) *n_q_blocks = csr->n_blocks;
  if (n_kv_blocks) *n_kv_blocks = csr->n_blocks;
  if (nnz) *nnz = (int64_t)csr->col_idx.size();
  if (row_ptr) *row_ptr = csr->row_ptr.data();
  if (col_idx) *col_idx = csr->col_idx.data();
  return LVSA_OK;
}

lvsa_status lvsa_csr_shape(const lvsa_csr* csr, int32_t* n_tokens, int32_t* block) {
  if (!csr) return LVSA_EINVAL;
  if (n_tokens) *n_tokens = csr->n_tokens;
  if (block) *block = csr->block;
  return LVSA_OK;
}

lvsa_status lvsa_csr_upload(lvsa_csr* csr, void* stream) {
  if (!csr) return LVSA_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  // Device arrays live in the order of the stream they were allocated on;
  // a later upload on another stream first waits for that one's copies.
  if (csr->uploaded && s != csr->upload_stream &&
      hipStreamWaitEvent(s, csr->uploaded, 0) != hipSuccess)
    return LVSA_EDEVICE;
  lvsa_status st;
  if ((st = upload_array(csr->row_ptr, &csr->d_row_ptr, s)) != LVSA_OK) return st;
  if ((st = upload_array(csr->col_idx, &csr->d_col_idx, s)) != LVSA_OK) return st;
  if (csr->has_entry && (st = upload_array(csr->entry, &csr->d_entry, s)) != LVSA_OK)
    return st;
  if (!csr->uploaded &&
      hipEventCreateWithFlags(&csr->uploaded, hipEventDisableTiming) != hipSuccess) {
    csr->uploaded = nullptr;
    return LVSA_EDEVICE;
  }
  if (hipEventRecord(csr->uploaded, s) != hipSuccess) return LVSA_EDEVICE;
  csr->upload_stream = s;
  return LVSA_OK;
}

void lvsa_csr_free(lvsa_csr* csr) {
  if (!csr) return;
  // The host arrays are the source of the last upload's copies.
  if (csr->uploaded) (void)hipEventSynchronize(csr->uploaded);
  for (void* d : {(void*)csr->d_row_ptr, (void*)csr->d_col_idx, (void*)csr->d_entry})
    if (d) (void)hipFreeAsync(d, csr->upload_stream);
  if (csr->uploaded) (void)hipEventDestroy(csr->uploaded);
  give_host_arrays(csr);
  delete csr;
}

lvsa_status lvsa_csr_device_view(const lvsa_csr* csr, lvsa_block_mask* out) {
  if (!csr || !out || !csr->d_row_ptr || !csr->d_col_idx) return LVSA_EINVAL;
  out->n_tokens = csr->n_tokens;
  out->block = csr->block;
  out->n_q_blocks = csr->n_blocks;
  out->n_kv_blocks = csr->n_blocks;
  out->row_ptr = csr->d_row_ptr;
  out->col_idx = csr->d_col_idx;
  return LVSA_OK;
}

lvsa_status lvsa_csr_entries(const lvsa_csr* csr, int32_t* frame_tokens,
                             const uint32_t** entry) {
  if (!csr) return LVSA_EINVAL;
  if (!csr->has_entry) return LVSA_EUNSUPPORTED;
  if (frame_tokens) *frame_tokens = csr->frame_tokens;
  if (entry) *entry = csr->entry.data();
  return LVSA_OK;
}

lvsa_status lvsa_csr_exact_view(const lvsa_csr* csr, lvsa_exact_mask* out) {
  if (!csr || !out) return LVSA_EINVAL;
  if (!csr->has_entry) return LVSA_EUNSUPPORTED;
  if (!csr->d_row_ptr || !csr->d_entry) return LVSA_EINVAL;
  out->n_tokens = csr->n_tokens;
  out->block = csr->block;
  out->n_q_blocks = csr->n_blocks;
  out->frame_tokens = csr->frame_tokens;
  out->row_ptr = csr->d_row_ptr;
  out->entry = csr->d_entry;
  return LVSA_OK;
}

namespace {

// Common checks of the device builders; resolves the frame rules and nb.
lvsa_status check_device_build(int32_t T, int32_t P, int32_t B, int32_t step,
                               int32_t layer, const lvsa_params* p, FrameCfg* c,
                               int64_t* nb) {
  if (layer < 0) return LVSA_EINVAL;
  lvsa_status st = resolve_frames(T, step, p, c);
  if (st != LVSA_OK) return st;
  st = check_mask_shape(T, P, B, c->text);
  if (st != LVSA_OK) return st;
  *nb = (mask_tokens(*c, P) + B - 1) / B;
  return LVSA_OK;
}

}  // namespace

lvsa_status lvsa_build_mask_device(int32_t T, int32_t P, int32_t B,
                                   int32_t step, int32_t layer,
                                   const lvsa_params* p, int32_t* d_row_ptr,
                                   int32_t* d_col_idx, int64_t col_capacity,
                                   void* stream) {
  if (!d_row_ptr || !d_col_idx) return LVSA_EINVAL;
  FrameCfg c;
  int64_t nb = 0;
  const lvsa_status st = check_device_build(T, P, B, step, layer, p, &c, &nb);
  if (st != LVSA_OK) return st;
  if (!device_mask_supported(c, P, B)) return LVSA_EUNSUPPORTED;
  if (col_capacity < nb * nb) return LVSA_EINVAL;
  if (launch_build_mask_device(c, P, B, d_row_ptr, d_col_idx, nullptr,
                               (hipStream_t)stream) != hipSuccess)
    return LVSA_EDEVICE;
  return LVSA_OK;
}

lvsa_status lvsa_build_exact_mask_device(int32_t T, int32_t P, int32_t B,
                                         int32_t step, int32_t layer,
                                         const lvsa_params* p,
                                         int32_t* d_row_ptr, uint32_t* d_entry,
                                         int64_t entry_capacity, void* stream) {
  if (!d_row_ptr || !d_entry) return LVSA_EINVAL;
  FrameCfg c;
  int64_t nb = 0;
  const lvsa_status st = check_device_build(T, P, B, step, layer, p, &c, &nb);
  if (st != LVSA_OK) return st;
  if (!exact_supported(P, B, nb)) return LVSA_EUNSUPPORTED;
  if (!device_mask_supported(c, P, B)) return LVSA_EUNSUPPORTED;
  if (entry_capacity < nb * nb) return LVSA_EINVAL;
  if (launch_build_mask_device(c, P, B, d_row_ptr, nullptr, d_entry,
                               (hipStream_t)stream) != hipSuccess)
    return LVSA_EDEVICE;
  return LVSA_OK;
}

namespace {

lvsa_status check_tensor(const lvsa_tensor* t, int32_t heads, int32_t n) {
  if (!t || !t->data) return LVSA_EINVAL;
  if (t->heads != heads || t->n_tokens != n) return LVSA_EINVAL;
  if (t->head_dim != 128) return LVSA_EUNSUPPORTED;
  if (((uintptr_t)t->data) % 16 != 0) return LVSA_EUNSUPPORTED;
  if (t->stride_token < 1 || t->stride_token % 8 != 0) return LVSA_EUNSUPPORTED;
  if (t->stride_head < 0 || t->stride_head % 8 != 0) return LVSA_EUNSUPPORTED;
  return LVSA_OK;
}

// Checks the tensors against (N, B, nb) and fills the launch arguments
// except the mask and the counters.
lvsa_status attention_args(const lvsa_tensor* q, const lvsa_tensor* k,
                           const lvsa_tensor* v, int32_t n_tokens, int32_t block,
                           int32_t n_blocks, lvsa_tensor* out, AttnArgs* a) {
  if (!q || !k || !v || !out) return LVSA_EINVAL;
  if (block != 64 && block != 128) return LVSA_EUNSUPPORTED;
  const int32_t H = q->heads;
  if (H < 1 || n_tokens < 1) return LVSA_EINVAL;
  if (n_blocks != (int32_t)(((int64_t)n_tokens + block - 1) / block)) return LVSA_EINVAL;
  // Work-items per launch must stay below 2^32.
  if ((int64_t)n_blocks * H * block * 2 >= ((int64_t)1 << 32)) return LVSA_EUNSUPPORTED;
  lvsa_status st;
  if ((st = check_tensor(q, H, n_tokens)) != LVSA_OK) return st;
  if ((st = check_tensor(k, H, n_tokens)) != LVSA_OK) return st;
  if ((st = check_tensor(v, H, n_tokens)) != LVSA_OK) return st;
  if ((st = check_tensor(out, H, n_tokens)) != LVSA_OK) return st;
  // K and V rows are addressed with 32-bit byte offsets within a head.
  const int64_t rows = (int64_t)n_blocks * block;
  if (rows * k->stride_token * 2 >= ((int64_t)1 << 32) ||
      rows * v->stride_token * 2 >= ((int64_t)1 << 32))
    return LVSA_EUNSUPPORTED;
  if (out->data == q->data || out->data == k->data || out->data == v->data)
    return LVSA_EINVAL;
  a->q = q->data;
  a->k = k->data;
  a->v = v->data;
  a->o = out->data;
  a->q_sh = q->stride_head;
  a->q_st = q->stride_token;
  a->k_sh = k->stride_head;
  a->k_st = k->stride_token;
  a->v_sh = v->stride_head;
  a->v_st = v->stride_token;
  a->o_sh = out->stride_head;
  a->o_st = out->stride_token;
  a->heads = H;
  a->n_tokens = n_tokens;
  a->n_blocks = n_blocks;
  a->row_ptr = nullptr;
  a->rows = nullptr;
  a->frame_tokens = 0;
  a->counters = nullptr;
  return LVSA_OK;
}

// Launches with a counter set of the pool (lvsa.h, "Tile counters").
lvsa_status run_attention(AttnArgs& a, int32_t block, AttnMode mode, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  CounterLease lease;
  const lvsa_status st = acquire_counters(s, &lease);
  if (st != LVSA_OK) return st;
  a.counters = lease.counters;
  if (launch_attention(a, block, mode, s) != hipSuccess) {
    CounterLease unused = lease;
    unused.captured = false;
    release_counters(unused, s);
    return LVSA_EDEVICE;
  }
  release_counters(lease, s);
  return LVSA_OK;
}

}  // namespace

lvsa_status lvsa_attention(const lvsa_tensor* q, const lvsa_tensor* k,
                           const lvsa_tensor* v, const lvsa_block_mask* mask,
                           lvsa_tensor* out, void* stream) {
  if (!mask || !mask->row_ptr || !mask->col_idx) return LVSA_EINVAL;
  if (mask->n_kv_blocks != mask->n_q_blocks) return LVSA_EINVAL;
  if (mask->n_q_blocks > kMaxSparseBlocks) return LVSA_EUNSUPPORTED;
  AttnArgs a;
  const lvsa_status st = attention_args(q, k, v, mask->n_tokens, mask->block,
                                        mask->n_q_blocks, out, &a);
  if (st != LVSA_OK) return st;
  a.row_ptr = mask->row_ptr;
  a.rows = (const uint32_t*)mask->col_idx;
  return run_attention(a, mask->block, ATTN_BLOCK, stream);
}

lvsa_status lvsa_attention_noalloc(const lvsa_tensor* q, const lvsa_tensor* k,
                                   const lvsa_tensor* v, const lvsa_block_mask* mask,
                                   lvsa_tensor* out, void* stream) {
  if (!mask || !mask->row_ptr || !mask->col_idx) return LVSA_EINVAL;
  if (mask->n_kv_blocks != mask->n_q_blocks) return LVSA_EINVAL;
  if (mask->n_q_blocks > kMaxSparseBlocks) return LVSA_EUNSUPPORTED;
  AttnArgs a;
  lvsa_status st = attention_args(q, k, v, mask->n_tokens, mask->block, mask->n_q_blocks,
                                  out, &a);
  if (st != LVSA_OK) return st;
  a.row_ptr = mask->row_ptr;
  a.rows = (const uint32_t*)mask->col_idx;
  if ((st = noalloc_counters(&a.counters)) != LVSA_OK) return st;
  if (launch_attention(a, mask->block, ATTN_BLOCK, (hipStream_t)stream) != hipSuccess)
    return LVSA_EDEVICE;
  return LVSA_OK;
}

lvsa_status lvsa_attention_exact(const lvsa_tensor* q, const lvsa_tensor* k,
                                 const lvsa_tensor* v,
                                 const lvsa_exact_mask* mask, lvsa_tensor* out,
                                 void* stream) {
  if (!mask || !mask->row_ptr || !mask->entry) return LVSA_EINVAL;
  if (mask->frame_tokens < 1) return LVSA_EINVAL;
  if (!exact_supported(mask->frame_tokens, mask->block, mask->n_q_blocks) ||
      mask->n_q_blocks > kMaxSparseBlocks)
    return LVSA_EUNSUPPORTED;
  AttnArgs a;
  const lvsa_status st = attention_args(q, k, v, mask->n_tokens, mask->block,
                                        mask->n_q_blocks, out, &a);
  if (st != LVSA_OK) return st;
  a.row_ptr = mask->row_ptr;
  a.rows = mask->entry;
  a.frame_tokens = mask->frame_tokens;
  return run_attention(a, mask->block, ATTN_EXACT, stream);
}

lvsa_status lvsa_dense_attention(const lvsa_tensor* q, const lvsa_tensor* k,
                                 const lvsa_tensor* v, int32_t block,
                                 lvsa_tensor* out, void* stream) {
  if (!q) return LVSA_EINVAL;
  if (block != 64 && block != 128) return LVSA_EUNSUPPORTED;
  const int32_t n = q->n_tokens;
  if (n < 1) return LVSA_EINVAL;
  const int32_t nb = (int32_t)(((int64_t)n + block - 1) / block);
  AttnArgs a;
  const lvsa_status st = attention_args(q, k, v, n, block, nb, out, &a);
  if (st != LVSA_OK) return st;
  return run_attention(a, block, ATTN_DENSE, stream);
}

}  // extern "C"
