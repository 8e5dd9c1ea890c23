// api.cpp -- the C ABI declared in include/lvsa.h: argument checks, handle
// management and dispatch to the builders and kernels.
#include <climits>
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
  c.s0 = p->rotate ? step % tper : 0;
  c.mode = p->window_mode;
  c.rotate = p->rotate;
  c.tie_high = p->tie_high;
  c.extra = p->extra_anchors;
  c.text = p->text_tokens;
  c.g = 0;
  for (int32_t f = 0; f < T; ++f) c.g += is_anchor(c, f) ? 1 : 0;
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
  std::vector<int32_t> pair_ptr;   // pair schedule (block words, and
  std::vector<uint32_t> pair_word; // token-exact words with entry words)
  std::vector<uint32_t> pair_exact;
  // Device copies, in one allocation each, sized when first uploaded.
  int32_t* d_row_ptr = nullptr;
  int32_t* d_col_idx = nullptr;
  uint32_t* d_entry = nullptr;
  int32_t* d_pair_ptr = nullptr;
  uint32_t* d_pair_word = nullptr;
  uint32_t* d_pair_exact = nullptr;
};

namespace {

// Device copy of a host array: allocated on the first upload (the handle's
// arrays never change size), then copied asynchronously on `s`.
// Device copy of `host` followed by `zeros` zero elements (allocated on the
// first upload, reused after).
template <typename T>
lvsa_status upload_array(const std::vector<T>& host, T** dev, hipStream_t s,
                         size_t zeros = 0) {
  static const T kZeros[LVSA_PAIR_WORK] = {};
  if (zeros > LVSA_PAIR_WORK) return LVSA_EINVAL;
  if (!*dev) {
    const size_t n = (host.empty() ? 1 : host.size()) + zeros;
    if (hipMalloc(dev, sizeof(T) * n) != hipSuccess) {
      *dev = nullptr;
      return LVSA_ENOMEM;
    }
  }
  if (!host.empty() &&
      hipMemcpyAsync(*dev, host.data(), sizeof(T) * host.size(), hipMemcpyHostToDevice,
                     s) != hipSuccess)
    return LVSA_EDEVICE;
  if (zeros && hipMemcpyAsync(*dev + host.size(), kZeros, sizeof(T) * zeros,
                              hipMemcpyHostToDevice, s) != hipSuccess)
    return LVSA_EDEVICE;
  return LVSA_OK;
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

int32_t lvsa_version(void) { return 10500; }

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
                            int32_t* win_hi) {
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
    frame_window(c, t, &lo, &hi);
    if (win_lo) win_lo[t] = lo;
    if (win_hi) win_hi[t] = hi;
  }
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
  try {
    build_csr_host(c, P, B, &h->row_ptr, &h->col_idx,
                   h->has_entry ? &h->entry : nullptr);
    build_pairs_host(h->row_ptr, h->col_idx, h->has_entry ? &h->entry : nullptr,
                     &h->pair_ptr, &h->pair_word, h->has_entry ? &h->pair_exact : nullptr);
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

lvsa_status lvsa_csr_info(const lvsa_csr* csr, int32_t* n_tokens,
                          int32_t* block, int32_t* n_blocks, int64_t* nnz,
                          const int32_t** row_ptr, const int32_t** col_idx) {
  if (!csr) return LVSA_EINVAL;
  if (n_tokens) *n_tokens = csr->n_tokens;
  if (block) *block = csr->block;
  if (n_blocks) *n_blocks = csr->n_blocks;
  if (nnz) *nnz = (int64_t)csr->col_idx.size();
  if (row_ptr) *row_ptr = csr->row_ptr.data();
  if (col_idx) *col_idx = csr->col_idx.data();
  return LVSA_OK;
}

lvsa_status lvsa_csr_upload(lvsa_csr* csr, void* stream) {
  if (!csr) return LVSA_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  lvsa_status st;
  if ((st = upload_array(csr->row_ptr, &csr->d_row_ptr, s)) != LVSA_OK) return st;
  if ((st = upload_array(csr->col_idx, &csr->d_col_idx, s)) != LVSA_OK) return st;
  if ((st = upload_array(csr->pair_ptr, &csr->d_pair_ptr, s, LVSA_PAIR_WORK)) != LVSA_OK)
    return st;
  if ((st = upload_array(csr->pair_word, &csr->d_pair_word, s)) != LVSA_OK) return st;
  if (csr->has_entry) {
    if ((st = upload_array(csr->entry, &csr->d_entry, s)) != LVSA_OK) return st;
    if ((st = upload_array(csr->pair_exact, &csr->d_pair_exact, s)) != LVSA_OK) return st;
  }
  return LVSA_OK;
}

void lvsa_csr_free(lvsa_csr* csr) {
  if (!csr) return;
  void* dev[] = {csr->d_row_ptr, csr->d_col_idx, csr->d_entry,
                 csr->d_pair_ptr, csr->d_pair_word, csr->d_pair_exact};
  bool any = false;
  for (void* d : dev) any = any || d != nullptr;
  if (any) {
    (void)hipDeviceSynchronize();
    for (void* d : dev)
      if (d) (void)hipFree(d);
  }
  delete csr;
}

lvsa_status lvsa_csr_pairs(const lvsa_csr* csr, int32_t* n_pairs, int64_t* n_words,
                           const int32_t** pair_ptr, const uint32_t** pair_word,
                           const uint32_t** pair_exact) {
  if (!csr) return LVSA_EINVAL;
  if (n_pairs) *n_pairs = (int32_t)csr->pair_ptr.size() - 1;
  if (n_words) *n_words = (int64_t)csr->pair_word.size();
  if (pair_ptr) *pair_ptr = csr->pair_ptr.data();
  if (pair_word) *pair_word = csr->pair_word.data();
  if (pair_exact) *pair_exact = csr->has_entry ? csr->pair_exact.data() : nullptr;
  return LVSA_OK;
}

lvsa_status lvsa_csr_device_view(const lvsa_csr* csr, lvsa_block_mask* out) {
  if (!csr || !out || !csr->d_row_ptr || !csr->d_col_idx || !csr->d_pair_ptr ||
      !csr->d_pair_word)
    return LVSA_EINVAL;
  out->n_tokens = csr->n_tokens;
  out->block = csr->block;
  out->n_blocks = csr->n_blocks;
  out->row_ptr = csr->d_row_ptr;
  out->col_idx = csr->d_col_idx;
  out->pair_ptr = csr->d_pair_ptr;
  out->pair_word = csr->d_pair_word;
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
  if (!csr->d_row_ptr || !csr->d_entry || !csr->d_pair_ptr || !csr->d_pair_exact)
    return LVSA_EINVAL;
  out->n_tokens = csr->n_tokens;
  out->block = csr->block;
  out->n_blocks = csr->n_blocks;
  out->frame_tokens = csr->frame_tokens;
  out->row_ptr = csr->d_row_ptr;
  out->entry = csr->d_entry;
  out->pair_ptr = csr->d_pair_ptr;
  out->pair_word = csr->d_pair_exact;
  return LVSA_OK;
}

lvsa_status lvsa_build_exact_mask_device(int32_t T, int32_t P, int32_t B,
                                         int32_t step, int32_t layer,
                                         const lvsa_params* p,
                                         int32_t* d_row_ptr, uint32_t* d_entry,
                                         int64_t entry_capacity, int32_t* d_pair_ptr,
                                         uint32_t* d_pair_word, int64_t pair_capacity,
                                         void* stream) {
  if (layer < 0 || !d_row_ptr || !d_entry || !d_pair_ptr || !d_pair_word)
    return LVSA_EINVAL;
  FrameCfg c;
  lvsa_status st = resolve_frames(T, step, p, &c);
  if (st != LVSA_OK) return st;
  st = check_mask_shape(T, P, B, c.text);
  if (st != LVSA_OK) return st;
  const int64_t nb = (mask_tokens(c, P) + B - 1) / B;
  if (!exact_supported(P, B, nb)) return LVSA_EUNSUPPORTED;
  if (!device_mask_supported(c, P, B)) return LVSA_EUNSUPPORTED;
  if (entry_capacity < nb * nb || pair_capacity < (nb + 1) / 2 * nb) return LVSA_EINVAL;
  if (launch_build_mask_device(c, P, B, d_row_ptr, nullptr, d_entry, d_pair_ptr,
                               d_pair_word, true, (hipStream_t)stream) != hipSuccess)
    return LVSA_EDEVICE;
  return LVSA_OK;
}

lvsa_status lvsa_build_mask_device(int32_t T, int32_t P, int32_t B,
                                   int32_t step, int32_t layer,
                                   const lvsa_params* p, int32_t* d_row_ptr,
                                   int32_t* d_col_idx, int64_t col_capacity,
                                   int32_t* d_pair_ptr, uint32_t* d_pair_word,
                                   int64_t pair_capacity, void* stream) {
  if (layer < 0 || !d_row_ptr || !d_col_idx || !d_pair_ptr || !d_pair_word)
    return LVSA_EINVAL;
  FrameCfg c;
  lvsa_status st = resolve_frames(T, step, p, &c);
  if (st != LVSA_OK) return st;
  st = check_mask_shape(T, P, B, c.text);
  if (st != LVSA_OK) return st;
  const int64_t nb = (mask_tokens(c, P) + B - 1) / B;
  if (!device_mask_supported(c, P, B)) return LVSA_EUNSUPPORTED;
  if (col_capacity < nb * nb || pair_capacity < (nb + 1) / 2 * nb) return LVSA_EINVAL;
  if (launch_build_mask_device(c, P, B, d_row_ptr, d_col_idx, nullptr, d_pair_ptr,
                               d_pair_word, false, (hipStream_t)stream) != hipSuccess)
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

lvsa_status run_attention(const lvsa_tensor* q, const lvsa_tensor* k,
                          const lvsa_tensor* v, int32_t n_tokens,
                          int32_t block, int32_t n_blocks,
                          const int32_t* pair_ptr, const uint32_t* pair_word,
                          int32_t frame_tokens, AttnMode mode,
                          lvsa_tensor* out, void* stream) {
  if (!q || !k || !v || !out) return LVSA_EINVAL;
  if (block != 64 && block != 128) return LVSA_EUNSUPPORTED;
  const int32_t H = q->heads;
  if (H < 1 || n_tokens < 1) return LVSA_EINVAL;
  if (n_blocks != (int32_t)(((int64_t)n_tokens + block - 1) / block))
    return LVSA_EINVAL;
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
  AttnArgs a;
  a.q = q->data;
  a.k = k->data;
  a.v = v->data;
  a.o = out->data;
  a.q_sh = q->stride_head;
  a.q_st = q->stride_token;
  a.k_sh = k->stride_head;
  a.k_st = k->stride_token;
  a.v_sh = v->stride_head;
  a.v_st = v->stride_token;
  a.o_sh = out->stride_head;
  a.o_st = out->stride_token;
  a.heads = H;
  a.n_tokens = n_tokens;
  a.n_blocks = n_blocks;
  a.pair_ptr = pair_ptr;
  a.pair_word = pair_word;
  a.frame_tokens = frame_tokens;
  if (launch_attention(a, block, mode, (hipStream_t)stream) != hipSuccess)
    return LVSA_EDEVICE;
  return LVSA_OK;
}

}  // namespace

lvsa_status lvsa_attention(const lvsa_tensor* q, const lvsa_tensor* k,
                           const lvsa_tensor* v, const lvsa_block_mask* mask,
                           lvsa_tensor* out, void* stream) {
  if (!mask || !mask->pair_ptr || !mask->pair_word) return LVSA_EINVAL;
  return run_attention(q, k, v, mask->n_tokens, mask->block, mask->n_blocks,
                       mask->pair_ptr, mask->pair_word, 0, ATTN_BLOCK, out, stream);
}

lvsa_status lvsa_attention_exact(const lvsa_tensor* q, const lvsa_tensor* k,
                                 const lvsa_tensor* v,
                                 const lvsa_exact_mask* mask, lvsa_tensor* out,
                                 void* stream) {
  if (!mask || !mask->pair_ptr || !mask->pair_word) return LVSA_EINVAL;
  if (mask->frame_tokens < 1) return LVSA_EINVAL;
  if (!exact_supported(mask->frame_tokens, mask->block, mask->n_blocks))
    return LVSA_EUNSUPPORTED;
  return run_attention(q, k, v, mask->n_tokens, mask->block, mask->n_blocks,
                       mask->pair_ptr, mask->pair_word, mask->frame_tokens, ATTN_EXACT,
                       out, stream);
}

lvsa_status lvsa_dense_attention(const lvsa_tensor* q, const lvsa_tensor* k,
                                 const lvsa_tensor* v, int32_t block,
                                 lvsa_tensor* out, void* stream) {
  if (!q) return LVSA_EINVAL;
  if (block != 64 && block != 128) return LVSA_EUNSUPPORTED;
  const int32_t n = q->n_tokens;
  if (n < 1) return LVSA_EINVAL;
  const int32_t nb = (int32_t)(((int64_t)n + block - 1) / block);
  return run_attention(q, k, v, n, block, nb, nullptr, nullptr, 0, ATTN_DENSE,
                       out, stream);
}

}  // extern "C"
