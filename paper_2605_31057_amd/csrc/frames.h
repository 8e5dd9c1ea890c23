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
  int32_t s0;        // (s mod T_per) mod T (0 for fixed anchors)
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
//   rotate = 1: Eq. 3, f = (s0 + i*T_per) mod T for some 0 <= i < k, with
//   s0 = (s mod T_per) mod T < T.  When T_per <= T the unreduced value
//   s0 + i*T_per stays below s0 + (k-1)*T_per <= T + T_per - 2 < 2T, so it
//   equals either f or f + T; when T_per > T, k = 1 and the only anchor is s0.
//   f < extra: a dedicated initial anchor.
__host__ __device__ inline bool is_anchor(const FrameCfg& c, int32_t f) {
  if (f < c.extra) return true;
  if (!c.rotate) return f % c.tper == 0;
  if (f >= c.s0 && (f - c.s0) % c.tper == 0 && (f - c.s0) / c.tper < c.k)
    return true;
  const int32_t u = f + c.T - c.s0;
  return u % c.tper == 0 && u / c.tper < c.k;
}

// Anchors of the period rule alone (Eq. 3 or Def. 2) among frames 0..f-1,
// 0 <= f <= T, in closed form.  Eq. 3's anchors are two ascending runs: the
// values s0 + i*T_per that stay below T (the first n_a of them), then the
// wrapped ones s0 + i*T_per - T (i = n_a..k-1), which all lie below s0.
__host__ __device__ inline int32_t period_anchors_below(const FrameCfg& c, int32_t f) {
  if (!c.rotate) return ceil_div(imin(f, c.T), c.tper);
  const int32_t n_a = imin(c.k, ceil_div(c.T - c.s0, c.tper));
  const int32_t run_a = f <= c.s0 ? 0 : imin(n_a, ceil_div(f - c.s0, c.tper));
  const int32_t run_b = imax(0, imin(c.k, ceil_div(f + c.T - c.s0, c.tper)) - n_a);
  return run_a + run_b;
}

// All anchors (the period rule's and frames 0..extra-1) among frames 0..f-1.
__host__ __device__ inline int32_t anchors_below(const FrameCfg& c, int32_t f) {
  const int32_t e = imin(imin(c.extra, c.T), f);
  return period_anchors_below(c, f) + e - period_anchors_below(c, e);
}

// Frames of [lo, hi] that are not anchors.
__host__ __device__ inline int32_t free_frames(const FrameCfg& c, int32_t lo, int32_t hi) {
  return (hi - lo + 1) - (anchors_below(c, hi + 1) - anchors_below(c, lo));
}

// Expanded window (Alg. 1).  Alg. 1 widens the adaptive window [l, h] one
// frame at a time on the side with more room (room below a = l, above
// b = T-1-h; equal room goes to the low side, or to the high side under
// tie_high) until the window holds min(2W+1, T-|G|) frames that are not
// anchors, or spans every frame.  The room rule fixes the order in which
// frames join: the roomier side alone until the two rooms are equal, then
// the two sides in turn, the tie side first.  So the window after g growth
// steps has a closed form, its count of non-anchor frames never decreases
// with g, and Alg. 1's number of steps is the least g in [0, a + b] whose
// window holds enough of them (a binary search over g).
__host__ __device__ inline void grown_window(int32_t l, int32_t h, int32_t a, int32_t b,
                                             int32_t g, bool tie_high, int32_t* lo,
                                             int32_t* hi) {
  const int32_t d = a > b ? a - b : b - a;   // steps before the rooms are equal
  int32_t grow_lo, grow_hi;
  if (g <= d) {
    grow_lo = a > b ? g : 0;
    grow_hi = a > b ? 0 : g;
  } else {
    const int32_t r = g - d;                  // steps taken in turn
    const int32_t first = (r + 1) / 2, second = r / 2;
    grow_lo = (a > b ? d : 0) + (tie_high ? second : first);
    grow_hi = (b > a ? d : 0) + (tie_high ? first : second);
  }
  *lo = l - grow_lo;
  *hi = h + grow_hi;
}

// Window [lo, hi] of query frame t under the configured rule.
//   BASIC    Def. 2
//   ADAPTIVE shifted to keep 2W+1 frames (Sec. 2, "Overlapping frames")
//   EXPANDED Alg. 1, as above
// Returns the number of Alg. 1 growth steps (0 for the other rules).
__host__ __device__ inline int32_t frame_window(const FrameCfg& c, int32_t t,
                                                int32_t* lo_out,
                                                int32_t* hi_out) {
  const int32_t T = c.T, W = c.W;
  if (c.mode == LVSA_WINDOW_BASIC) {
    *lo_out = imax(0, t - W);
    *hi_out = imin(T - 1, t + W);
    return 0;
  }
  const int32_t l = imax(0, imin(t - W, T - 1 - 2 * W));
  const int32_t h = imin(T - 1, imax(t + W, 2 * W));
  int32_t steps = 0;
  if (c.mode == LVSA_WINDOW_EXPANDED) {
    const int32_t target = imin(2 * W + 1, T - c.g);
    const int32_t a = l, b = T - 1 - h;
    int32_t g_lo = 0, g_hi = a + b;
    while (g_lo < g_hi) {
      const int32_t g = (g_lo + g_hi) / 2;
      int32_t lo, hi;
      grown_window(l, h, a, b, g, c.tie_high != 0, &lo, &hi);
      if (free_frames(c, lo, hi) >= target)
        g_hi = g;
      else
        g_lo = g + 1;
    }
    steps = g_lo;
  }
  grown_window(l, h, l, T - 1 - h, steps, c.tie_high != 0, lo_out, hi_out);
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

// Whether a block mask of (P, B, nb) can carry exact entry words.
__host__ __device__ inline bool exact_supported(int32_t P, int32_t B,
                                                int64_t nb) {
  return P >= B && B <= 255 && nb <= 65536;
}

}  // namespace lvsa
