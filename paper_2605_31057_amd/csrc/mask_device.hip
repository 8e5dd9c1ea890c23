// mask_device.hip -- LVSA mask builder as one GPU kernel.
//
// Computes the same block CSR as the host builder (the LVSA frame sets of
// Sec. 2: Def. 2, Eq. 3, Alg. 1, expanded to blocks by the any-overlap rule)
// without a host round trip, so a denoising loop can rebuild the mask for
// step s on the stream that then runs attention.
//
// One workgroup of 1024 threads:
//   1. one thread per frame: anchor flag and window bounds into LDS;
//   2. one thread per query block: count its kept key blocks into
//      row_ptr[qb + 1];
//   3. in-place exclusive scan of the counts (chunks of 1024, LDS tree);
//   4. one thread per query block: write its row of col_idx and/or of the
//      token-exact entry words.
// The metadata is tiny (T <= 4096 frames), so one workgroup keeps the whole
// build in a single launch with plain __syncthreads between phases.
#include "internal.h"

namespace lvsa {
namespace {

constexpr int kThreads = 1024;

struct Rows {
  const uint8_t* anchor;
  const int16_t* lo;
  const int16_t* hi;
  int32_t T, P, B, N, S;   // S segments: T frames, plus the text if any
};

// Visits the kept key blocks of query block qb in ascending order.  Text
// (segment T) is attended by every query; a query block touching the text
// attends to every segment.
template <typename F>
__device__ inline void for_each_kept(const Rows& r, int32_t qb, F&& emit) {
  int32_t f0, f1;
  block_frame_range(qb, r.T, r.P, r.B, r.N, &f0, &f1);
  int32_t last = -1;
  for (int32_t tau = 0; tau < r.S; ++tau) {
    bool att = tau == r.T || f1 == r.T || r.anchor[tau] != 0;
    for (int32_t t = f0; t <= f1 && !att; ++t)
      att = r.lo[t] <= tau && tau <= r.hi[t];
    if (!att) continue;
    int32_t b0, b1;
    segment_blocks(tau, r.T, r.P, r.B, r.N, &b0, &b1);
    for (int32_t b = imax(b0, last + 1); b <= b1; ++b) emit(b);
    last = imax(last, b1);
  }
}

__global__ __launch_bounds__(kThreads) void build_mask_kernel(
    FrameCfg c, int32_t P, int32_t B, int32_t* __restrict__ row_ptr,
    int32_t* __restrict__ col_idx, uint32_t* __restrict__ entry) {
  __shared__ uint8_t s_anchor[LVSA_MAX_FRAMES];
  __shared__ int16_t s_lo[LVSA_MAX_FRAMES];
  __shared__ int16_t s_hi[LVSA_MAX_FRAMES];
  __shared__ int32_t s_scan[kThreads];
  __shared__ int32_t s_carry;

  const int32_t tid = threadIdx.x;
  const int32_t T = c.T;
  const int32_t N = (int32_t)mask_tokens(c, P);
  const int32_t nb = ceil_div(N, B);

  for (int32_t t = tid; t < T; t += kThreads) {
    s_anchor[t] = is_anchor(c, t) ? 1 : 0;
    int32_t lo, hi;
    frame_window(c, t, &lo, &hi);
    s_lo[t] = (int16_t)lo;
    s_hi[t] = (int16_t)hi;
  }
  if (tid == 0) {
    s_carry = 0;
    row_ptr[0] = 0;
  }
  __syncthreads();

  const Rows r{s_anchor, s_lo, s_hi, T, P, B, N, c.text > 0 ? T + 1 : T};
  for (int32_t qb = tid; qb < nb; qb += kThreads) {
    int32_t n = 0;
    for_each_kept(r, qb, [&](int32_t) { ++n; });
    row_ptr[qb + 1] = n;
  }
  __syncthreads();

  // Inclusive scan of row_ptr[1..nb] in chunks of kThreads.
  for (int32_t base = 0; base < nb; base += kThreads) {
    const int32_t i = base + tid;
    int32_t x = i < nb ? row_ptr[i + 1] : 0;
    s_scan[tid] = x;
    __syncthreads();
    for (int32_t off = 1; off < kThreads; off <<= 1) {
      const int32_t y = tid >= off ? s_scan[tid - off] : 0;
      __syncthreads();
      s_scan[tid] += y;
      __syncthreads();
    }
    if (i < nb) row_ptr[i + 1] = s_scan[tid] + s_carry;
    __syncthreads();
    if (tid == kThreads - 1) s_carry += s_scan[tid];
    __syncthreads();
  }

  auto attends = [&](int32_t t, int32_t tau) {
    return t == T || tau == T || s_anchor[tau] != 0 || (s_lo[t] <= tau && tau <= s_hi[t]);
  };
  for (int32_t qb = tid; qb < nb; qb += kThreads) {
    const int32_t beg = row_ptr[qb];
    int32_t f0, f1;
    block_frame_range(qb, T, P, B, N, &f0, &f1);
    int32_t n = 0;
    for_each_kept(r, qb, [&](int32_t b) {
      if (col_idx) col_idx[beg + n] = b;
      if (entry) entry[beg + n] = exact_entry(b, f0, f1, T, P, B, N, attends);
      ++n;
    });
  }
}

}  // namespace

hipError_t launch_build_mask_device(const FrameCfg& c, int32_t P, int32_t B,
                                    int32_t* d_row_ptr, int32_t* d_col_idx,
                                    uint32_t* d_entry, hipStream_t stream) {
  hipLaunchKernelGGL(build_mask_kernel, dim3(1), dim3(kThreads), 0, stream, c,
                     P, B, d_row_ptr, d_col_idx, d_entry);
  return hipGetLastError();
}

}  // namespace lvsa
