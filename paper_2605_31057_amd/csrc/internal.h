// internal.h -- declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "frames.h"
#include "lvsa.h"

namespace lvsa {

// Checks the mask arguments and resolves T_per, |G^s| and s mod T_per.
lvsa_status resolve_frames(int32_t T, int32_t step, const lvsa_params* p,
                           FrameCfg* out);

// Checks (T, P, B, text tokens L) of a block mask: N = T*P + L, N + B must fit
// in int32 and nb*nb too.
lvsa_status check_mask_shape(int32_t T, int32_t P, int32_t B, int32_t L);

// Tokens of the mask: T*P video tokens and the text tokens after them.
__host__ __device__ inline int64_t mask_tokens(const FrameCfg& c, int32_t P) {
  return (int64_t)c.T * P + c.text;
}

// Host CSR construction (mask_host.cpp).  `entry` (may be null) receives the
// token-exact entry word of every kept block; callers pass it only when
// exact_supported(P, B, nb).
void build_csr_host(const FrameCfg& c, int32_t P, int32_t B,
                    std::vector<int32_t>* row_ptr,
                    std::vector<int32_t>* col_idx,
                    std::vector<uint32_t>* entry);

// Device mask construction (mask_device.hip).  Writes row_ptr and, where the
// pointer is non-null, col_idx and/or the token-exact entry words.  The
// builder holds the windows of one query-block pair's frames in LDS:
// device_mask_supported says whether a pair touches few enough frames.
bool device_mask_supported(const FrameCfg& c, int32_t P, int32_t B);
hipError_t launch_build_mask_device(const FrameCfg& c, int32_t P, int32_t B,
                                    int32_t* d_row_ptr, int32_t* d_col_idx,
                                    uint32_t* d_entry, hipStream_t stream);

// Key blocks a sparse attention launch supports: a workgroup merges the two
// CSR rows of its pair of query blocks (at most nb words) in LDS.
constexpr int32_t kMaxSparseBlocks = 8000;

// Tile counters of one attention launch: eight 64-bit words (one per XCD),
// zeroed on the launch stream before the kernel runs.
constexpr int kTileCounters = 8;

// Attention launch (attention.hip).  Pointers are bf16 tensors; strides in
// elements.  The sparse modes read the CSR rows of each pair of query blocks
// (col_idx for ATTN_BLOCK, entry words for ATTN_EXACT); row_ptr and rows are
// null for the dense pass.
struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  int64_t q_sh, q_st, k_sh, k_st, v_sh, v_st, o_sh, o_st;
  int32_t heads;
  int32_t n_tokens;
  int32_t n_blocks;
  const int32_t* row_ptr;    // [n_blocks + 1]
  const uint32_t* rows;      // col_idx (block form) or entry words (exact form)
  int32_t frame_tokens;      // P (ATTN_EXACT only)
  uint64_t* counters;        // kTileCounters words, any content (zeroed here)
};
enum AttnMode { ATTN_DENSE = 0, ATTN_BLOCK = 1, ATTN_EXACT = 2 };
hipError_t launch_attention(const AttnArgs& a, int32_t block, AttnMode mode,
                            hipStream_t stream);

// Per-device pool of tile-counter sets (api.cpp).  acquire hands out a set no
// launch in flight uses; release records, after the launch on `stream`, the
// event that frees it again (or keeps the set for good when the stream is
// being captured into a graph).
struct CounterLease {
  int device = -1;
  int32_t slot = -1;
  uint64_t* counters = nullptr;
  bool captured = false;
};
lvsa_status acquire_counters(hipStream_t stream, CounterLease* lease);
void release_counters(const CounterLease& lease, hipStream_t stream);

}  // namespace lvsa
