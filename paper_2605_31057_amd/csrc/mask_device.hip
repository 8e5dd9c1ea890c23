// mask_device.hip -- LVSA mask builder on the GPU.
//
// Computes the same block CSR as the host builder (the LVSA frame sets of
// Sec. 2: Def. 2, Eq. 3, Alg. 1, expanded to blocks by the any-overlap rule)
// without a host round trip, so a denoising loop can rebuild the mask for
// step s on the stream that then runs attention.
//
// Three launches on the stream:
//   1. one workgroup per query block: the windows of the block's frames
//      (Alg. 1) into LDS, then every key block tested in parallel; the count
//      of kept blocks goes to row_ptr[qb + 1];
//   2. one workgroup: in-place inclusive scan of the counts (row_ptr);
//   3. one workgroup per query block: the same test again, kept key blocks
//      compacted in ascending order (wave ballots and a per-chunk prefix) and
//      written to col_idx and/or the token-exact entry words.
// Every thread tests its own candidates with closed-form rules, so a row
// costs a few passes over nb candidates whatever its length.
#include "internal.h"

namespace lvsa {
namespace {

constexpr int kRowThreads = 256;
constexpr int kRowWaves = kRowThreads / 64;
constexpr int kScanThreads = 1024;

// Query frames one workgroup can hold (a block touches at most B/P + 2
// frames; B <= 2^20 and P >= 1 give the worst case, capped here and checked
// before launch).
constexpr int kMaxRowFrames = 1024;

struct RowFrames {
  int32_t f0, f1;                  // segments touched by the query block
  int16_t lo[kMaxRowFrames];       // window of frame f0 + i
  int16_t hi[kMaxRowFrames];
};

// tau in A(t) for segments t, tau (segment T = the text tokens, attended by
// and attending to everything).
__device__ inline bool seg_attends(const FrameCfg& c, const RowFrames& rf, int32_t t,
                                   int32_t tau) {
  if (t == c.T || tau == c.T) return true;
  if (is_anchor(c, tau)) return true;
  const int32_t i = t - rf.f0;
  return rf.lo[i] <= tau && tau <= rf.hi[i];
}

__device__ inline void load_row_frames(const FrameCfg& c, int32_t qb, int32_t P,
                                       int32_t B, int32_t N, RowFrames* rf) {
  if (threadIdx.x == 0) block_frame_range(qb, c.T, P, B, N, &rf->f0, &rf->f1);
  __syncthreads();
  const int32_t last = imin(rf->f1, c.T - 1);
  for (int32_t t = rf->f0 + (int32_t)threadIdx.x; t <= last; t += kRowThreads) {
    int32_t lo, hi;
    frame_window(c, t, &lo, &hi);
    rf->lo[t - rf->f0] = (int16_t)lo;
    rf->hi[t - rf->f0] = (int16_t)hi;
  }
  __syncthreads();
}

// Whether query block qb (frames in rf) keeps key block kb.
__device__ inline bool keeps(const FrameCfg& c, const RowFrames& rf, int32_t kb,
                             int32_t P, int32_t B, int32_t N) {
  int32_t g0, g1;
  block_frame_range(kb, c.T, P, B, N, &g0, &g1);
  for (int32_t t = rf.f0; t <= rf.f1; ++t)
    for (int32_t tau = g0; tau <= g1; ++tau)
      if (seg_attends(c, rf, t, tau)) return true;
  return false;
}

__global__ __launch_bounds__(kRowThreads) void count_rows_kernel(
    FrameCfg c, int32_t P, int32_t B, int32_t* __restrict__ row_ptr) {
  __shared__ RowFrames rf;
  __shared__ int32_t s_cnt[kRowWaves];
  const int32_t N = (int32_t)mask_tokens(c, P);
  const int32_t nb = ceil_div(N, B);
  const int32_t qb = blockIdx.x;
  load_row_frames(c, qb, P, B, N, &rf);
  int32_t cnt = 0;
  for (int32_t kb = threadIdx.x; kb < nb; kb += kRowThreads) cnt += keeps(c, rf, kb, P, B, N);
  // wave sums, then the workgroup sum
  for (int off = 32; off > 0; off >>= 1) cnt += __shfl_xor(cnt, off);
  if (threadIdx.x % 64 == 0) s_cnt[threadIdx.x / 64] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t total = 0;
    for (int w = 0; w < kRowWaves; ++w) total += s_cnt[w];
    row_ptr[qb + 1] = total;
    if (qb == 0) row_ptr[0] = 0;
  }
}

// In-place inclusive scan of row_ptr[1 .. nb] (chunks of kScanThreads).
__global__ __launch_bounds__(kScanThreads) void scan_rows_kernel(int32_t nb,
                                                                 int32_t* __restrict__ row_ptr) {
  __shared__ int32_t s_scan[kScanThreads];
  __shared__ int32_t s_carry;
  const int32_t tid = threadIdx.x;
  if (tid == 0) s_carry = 0;
  __syncthreads();
  for (int32_t base = 0; base < nb; base += kScanThreads) {
    const int32_t i = base + tid;
    s_scan[tid] = i < nb ? row_ptr[i + 1] : 0;
    __syncthreads();
    for (int32_t off = 1; off < kScanThreads; off <<= 1) {
      const int32_t y = tid >= off ? s_scan[tid - off] : 0;
      __syncthreads();
      s_scan[tid] += y;
      __syncthreads();
    }
    if (i < nb) row_ptr[i + 1] = s_scan[tid] + s_carry;
    __syncthreads();
    if (tid == kScanThreads - 1) s_carry += s_scan[tid];
    __syncthreads();
  }
}

__global__ __launch_bounds__(kRowThreads) void fill_rows_kernel(
    FrameCfg c, int32_t P, int32_t B, const int32_t* __restrict__ row_ptr,
    int32_t* __restrict__ col_idx, uint32_t* __restrict__ entry) {
  __shared__ RowFrames rf;
  __shared__ int32_t s_wave[kRowWaves];
  const int32_t N = (int32_t)mask_tokens(c, P);
  const int32_t nb = ceil_div(N, B);
  const int32_t qb = blockIdx.x;
  load_row_frames(c, qb, P, B, N, &rf);
  const int32_t lane = threadIdx.x % 64, wave = threadIdx.x / 64;
  int32_t pos = row_ptr[qb];
  auto attends = [&](int32_t t, int32_t tau) { return seg_attends(c, rf, t, tau); };
  for (int32_t base = 0; base < nb; base += kRowThreads) {
    const int32_t kb = base + (int32_t)threadIdx.x;
    const bool keep = kb < nb && keeps(c, rf, kb, P, B, N);
    const uint64_t bal = __ballot(keep);
    const int32_t below = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) s_wave[wave] = __popcll(bal);
    __syncthreads();
    int32_t off = 0, total = 0;
    for (int w = 0; w < kRowWaves; ++w) {
      off += w < wave ? s_wave[w] : 0;
      total += s_wave[w];
    }
    if (keep) {
      const int32_t at = pos + off + below;
      if (col_idx) col_idx[at] = kb;
      if (entry) entry[at] = exact_entry(kb, rf.f0, rf.f1, c.T, P, B, N, attends);
    }
    pos += total;
    __syncthreads();
  }
}

}  // namespace

bool device_mask_supported(const FrameCfg& c, int32_t P, int32_t B) {
  // A block touches at most min(T, B/P + 2) frames.
  return (int64_t)B / P + 2 <= kMaxRowFrames || c.T <= kMaxRowFrames;
}

hipError_t launch_build_mask_device(const FrameCfg& c, int32_t P, int32_t B,
                                    int32_t* d_row_ptr, int32_t* d_col_idx,
                                    uint32_t* d_entry, hipStream_t stream) {
  const int32_t nb = (int32_t)((mask_tokens(c, P) + B - 1) / B);
  hipLaunchKernelGGL(count_rows_kernel, dim3(nb), dim3(kRowThreads), 0, stream, c, P, B,
                     d_row_ptr);
  hipLaunchKernelGGL(scan_rows_kernel, dim3(1), dim3(kScanThreads), 0, stream, nb,
                     d_row_ptr);
  hipLaunchKernelGGL(fill_rows_kernel, dim3(nb), dim3(kRowThreads), 0, stream, c, P, B,
                     d_row_ptr, d_col_idx, d_entry);
  return hipGetLastError();
}

}  // namespace lvsa
