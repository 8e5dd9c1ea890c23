// frames.h -- LVSA frame-level rules shared by the host and device mask
// builders (LVSA paper, Sec. 2: Def. 2, Eq. 3, the adaptive window and
// Alg. 1).  Everything here is integer arithmetic on frame indices, written
// once as __host__ __device__ inline functions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lvsa.h"

namespace lvsa {

// Resolved per-step frame configuration.
struct FrameCfg {
  int32_t T;         // frames
  int32_t W;         // window half-width
  int32_t tper;      // anchor period T_per
  int32_t k;         // Eq. 3 anchors ceil(T / T_per)
  int32_t extra;     // dedicated initial anchors: frames 0..extra-1
  int32_t g;         // |G|: Eq. 3 (or Def. 2) anchors plus the extra ones
  int32_t text;      // text tokens after the T*P video tokens (segment T)
  int32_t s0;        // s mod T_per (0 for fixed anchors)
  int32_t mode;      // LVSA_WINDOW_*
  int32_t rotate;    // Eq. 3 (1) or Def. 2's fixed set (0)
  int32_t tie_high;  // Alg. 1 equal-room rule
};

__host__ __device__ inline int32_t ceil_div(int32_t a, int32_t b) {
  return (a + b - 1) / b;
}
__host__ __device__ inline int32_t imin(int32_t a, int32_t b) { return a < b ? a : b; }
__host__ __device__ inline int32_t imax(int32_t a, int32_t b) { return a > b ? a : b; }

// Membership of frame f in the anchor set.
//   rotate = 0: Def. 2, f mod T_per == 0.
//   rotate = 1: Eq. 3, f = (s0 + i*T_per) mod T for some 0 <= i < k.  The
//   unreduced value s0 + i*T_per is below k*T_per <= T + T_per - 1 < 2T, so
//   it equals either f or f + T.
//   f < extra: a dedicated initial anchor.
__host__ __device__ inline bool is_anchor(const FrameCfg& c, int32_t f) {
  if (f < c.extra) return true;
  if (!c.rotate) return f % c.tper == 0;
  if (f >= c.s0 && (f - c.s0) % c.tper == 0 && (f - c.s0) / c.tper < c.k)
    return true;
  const int32_t u = f + c.T - c.s0;
  return u % c.tper == 0 && u / c.tper < c.k;
}

// Window [lo, hi] of query frame t under the configured rule.
//   BASIC    Def. 2
//   ADAPTIVE shifted to keep 2W+1 frames (Sec. 2, "Overlapping frames")
//   EXPANDED Alg. 1: grow the adaptive window on the side with more room
//            until min(2W+1, T-|G|) of its frames are not anchors.
// Returns the number of Alg. 1 growth steps (0 for the other rules).
__host__ __device__ inline int32_t frame_window(const FrameCfg& c, int32_t t,
                                                int32_t* lo_out,
                                                int32_t* hi_out) {
  const int32_t T = c.T, W = c.W;
  int32_t lo, hi;
  if (c.mode == LVSA_WINDOW_BASIC) {
    lo = imax(0, t - W);
    hi = imin(T - 1, t + W);
    *lo_out = lo;
    *hi_out = hi;
    return 0;
  }
  lo = imax(0, imin(t - W, T - 1 - 2 * W));
  hi = imin(T - 1, imax(t + W, 2 * W));
  int32_t steps = 0;
  if (c.mode == LVSA_WINDOW_EXPANDED) {
    const int32_t target = imin(2 * W + 1, T - c.g);
    int32_t nonglobal = 0;
    for (int32_t f = lo; f <= hi; ++f) nonglobal += is_anchor(c, f) ? 0 : 1;
    while (nonglobal < target && (lo > 0 || hi < T - 1)) {
      const int32_t room_lo = lo, room_hi = T - 1 - hi;
      int32_t f;
      if (room_lo > room_hi || (room_lo == room_hi && !c.tie_high))
        f = --lo;
      else
        f = ++hi;
      nonglobal += is_anchor(c, f) ? 0 : 1;
      ++steps;
    }
  }
  *lo_out = lo;
  *hi_out = hi;
  return steps;
}

// First and last segment touched by block b (tokens b*B .. min((b+1)*B, N)-1):
// frames 0..T-1 for video tokens, segment T for the text tokens after them.
__host__ __device__ inline void block_frame_range(int32_t b, int32_t T,
                                                  int32_t P, int32_t B,
                                                  int32_t N, int32_t* first,
                                                  int32_t* last) {
  const int64_t t0 = (int64_t)b * B;
  const int64_t end = t0 + B < (int64_t)N ? t0 + B : (int64_t)N;
  *first = (int32_t)(t0 / P < T ? t0 / P : T);
  *last = (int32_t)((end - 1) / P < T ? (end - 1) / P : T);
}

// Key blocks of segment tau: frame tau's tokens tau*P .. tau*P+P-1, or the
// text tokens T*P .. N-1 for tau = T.
__host__ __device__ inline void segment_blocks(int32_t tau, int32_t T, int32_t P,
                                               int32_t B, int32_t N, int32_t* b0,
                                               int32_t* b1) {
  const int64_t first = (int64_t)tau * P;
  const int64_t last = tau < T ? first + P - 1 : (int64_t)N - 1;
  *b0 = (int32_t)(first / B);
  *b1 = (int32_t)(last / B);
}

// Token-exact entry word of a kept block pair (lvsa.h, "token-exact form").
// The query block touches segments f0..f1 and key block kb segments g0..g1,
// each at most two apart since P >= B (segment T, the text tokens, follows
// frame T-1); kb's first kfirst tokens lie in g0.  attends(t, tau) is
// "segment tau is attended by segment t": tau in A(t), or either is text.
//   bits  0..15  kb
//   bits 16..23  kfirst (B when kb lies in one frame)
//   bits 24..27  bit 2a+b: frame (b ? g1 : g0) is in A(a ? f1 : f0)
template <typename Attends>
__host__ __device__ inline uint32_t exact_word(int32_t kb, int32_t g0,
                                               int32_t g1, uint32_t kfirst,
                                               int32_t f0, int32_t f1,
                                               const Attends& attends) {
  const uint32_t pat = (attends(f0, g0) ? 1u : 0u) | (attends(f0, g1) ? 2u : 0u) |
                       (attends(f1, g0) ? 4u : 0u) | (attends(f1, g1) ? 8u : 0u);
  return (uint32_t)kb | (kfirst << 16) | (pat << 24);
}

// Segments g0..g1 of key block kb and its tokens in g0 (B if g0 == g1).
__host__ __device__ inline void key_block_split(int32_t kb, int32_t T,
                                                int32_t P, int32_t B, int32_t N,
                                                int32_t* g0, int32_t* g1,
                                                uint32_t* kfirst) {
  block_frame_range(kb, T, P, B, N, g0, g1);
  *kfirst = *g1 > *g0 ? (uint32_t)((int64_t)(*g0 + 1) * P - (int64_t)kb * B)
                      : (uint32_t)B;
}

template <typename Attends>
__host__ __device__ inline uint32_t exact_entry(int32_t kb, int32_t f0,
                                                int32_t f1, int32_t T,
                                                int32_t P, int32_t B, int32_t N,
                                                const Attends& attends) {
  int32_t g0, g1;
  uint32_t kfirst;
  key_block_split(kb, T, P, B, N, &g0, &g1, &kfirst);
  return exact_word(kb, g0, g1, kfirst, f0, f1, attends);
}

// Pair schedule words (lvsa.h, "pair schedule"): key block kb listed for the
// query-block pair (2p, 2p+1), with which of the two keeps it.
__host__ __device__ inline uint32_t pair_word_of(int32_t kb, bool kept0, bool kept1) {
  return (uint32_t)kb | (kept0 ? 1u << 30 : 0u) | (kept1 ? 1u << 31 : 0u);
}

// Token-exact pair word from the entry words e0 of (2p, kb) and e1 of
// (2p+1, kb), each 0 when that query block does not keep kb (a kept block's
// pattern is never 0): kb and kfirst, then the two 4-bit patterns.
__host__ __device__ inline uint32_t pair_exact_word(uint32_t e0, uint32_t e1) {
  const uint32_t base = (e0 != 0u ? e0 : e1) & 0xFFFFFFu;
  return base | (((e0 >> 24) & 0xFu) << 24) | (((e1 >> 24) & 0xFu) << 28);
}

// Whether a block mask of (P, B, nb) can carry exact entry words.
__host__ __device__ inline bool exact_supported(int32_t P, int32_t B,
                                                int64_t nb) {
  return P >= B && B <= 255 && nb <= 65536;
}

}  // namespace lvsa
