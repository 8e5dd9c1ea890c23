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

// Pair schedule from a CSR (mask_host.cpp): row p lists the key blocks of
// query blocks 2p and 2p+1 (lvsa.h, "pair schedule"); `pair_exact` (may be
// null, and is ignored when `entry` is null) receives the token-exact words.
void build_pairs_host(const std::vector<int32_t>& row_ptr,
                      const std::vector<int32_t>& col_idx,
                      const std::vector<uint32_t>* entry,
                      std::vector<int32_t>* pair_ptr,
                      std::vector<uint32_t>* pair_word,
                      std::vector<uint32_t>* pair_exact);

// Device mask construction (mask_device.hip).  Writes row_ptr and, where the
// pointer is non-null, col_idx and/or the token-exact entry words, then the
// pair schedule (pair_ptr and pair words, in the token-exact form when
// `exact`).  The builder holds the windows of one query-block pair's frames
// in LDS: device_mask_supported says whether a pair touches few enough frames.
bool device_mask_supported(const FrameCfg& c, int32_t P, int32_t B);
hipError_t launch_build_mask_device(const FrameCfg& c, int32_t P, int32_t B,
                                    int32_t* d_row_ptr, int32_t* d_col_idx,
                                    uint32_t* d_entry, int32_t* d_pair_ptr,
                                    uint32_t* d_pair_word, bool exact,
                                    hipStream_t stream);

// Attention launch (attention.hip).  Pointers are bf16 tensors; strides in
// elements.  pair_ptr/pair_word are null for the dense pass.
struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  int64_t q_sh, q_st, k_sh, k_st, v_sh, v_st, o_sh, o_st;
  int32_t heads;
  int32_t n_tokens;
  int32_t n_blocks;
  const int32_t* pair_ptr;   // pair schedule rows [ceil(nb/2) + 1]
  const uint32_t* pair_word; // block or token-exact (ATTN_EXACT) pair words
  int32_t frame_tokens;      // P (ATTN_EXACT only)
};
enum AttnMode { ATTN_DENSE = 0, ATTN_BLOCK = 1, ATTN_EXACT = 2 };
hipError_t launch_attention(const AttnArgs& a, int32_t block, AttnMode mode,
                            hipStream_t stream);

}  // namespace lvsa
