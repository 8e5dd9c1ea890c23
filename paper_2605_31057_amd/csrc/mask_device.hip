// mask_device.hip -- LVSA mask builder on the GPU.
//
// Computes the same block CSR as the host builder (the LVSA frame sets of
// Sec. 2: Def. 2, Eq. 3, Alg. 1, expanded to blocks by the any-overlap rule)
// without a host round trip, so a denoising loop can rebuild the mask for
// step s on the stream that then runs attention.
//
// Three launches on the stream, each workgroup of the first and the last
// handling a pair of query blocks 2p and 2p+1 (the last pair of an odd nb has
// one), whose frames overlap, so the windows are computed once for both:
//   1. one workgroup per pair: the windows of the pair's frames (Alg. 1) into
//      LDS, then every key block tested in parallel against both query
//      blocks; the two row lengths go to row_ptr[qb + 1];
//   2. one workgroup: an in-place inclusive scan of row_ptr;
//   3. one workgroup per pair: the same tests again, kept key blocks
//      compacted in ascending order (wave ballots and a per-chunk prefix) and
//      written as block indices and/or token-exact entry words.
// Every thread tests its own candidates with closed-form rules, so a row
// costs a few passes over nb candidates whatever its length.
#include "internal.h"

namespace lvsa {
namespace {

constexpr int kRowThreads = 256;
constexpr int kRowWaves = kRowThreads / 64;
constexpr int kScanThreads = 1024;

// Query frames one workgroup can hold (a query-block pair touches at most
// 2B/P + 2 frames; checked before launch).
constexpr int kMaxRowFrames = 1024;

struct RowFrames {
  int32_t f0, f1;                  // segments touched by the pair's query blocks
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

// Windows of the frames touched by query blocks qb0..qb1 into LDS.
__device__ inline void load_row_frames(const FrameCfg& c, int32_t qb0, int32_t qb1,
                                       int32_t P, int32_t B, int32_t N, RowFrames* rf) {
  if (threadIdx.x == 0) {
    int32_t a, b;
    block_frame_range(qb0, c.T, P, B, N, &rf->f0, &a);
    block_frame_range(qb1, c.T, P, B, N, &b, &rf->f1);
  }
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

// Whether a query block touching segments t0..t1 keeps key block kb.
__device__ inline bool keeps(const FrameCfg& c, const RowFrames& rf, int32_t t0,
                             int32_t t1, int32_t kb, int32_t P, int32_t B, int32_t N) {
  int32_t g0, g1;
  block_frame_range(kb, c.T, P, B, N, &g0, &g1);
  for (int32_t t = t0; t <= t1; ++t)
    for (int32_t tau = g0; tau <= g1; ++tau)
      if (seg_attends(c, rf, t, tau)) return true;
  return false;
}

// Per-pair test: which of the pair's query blocks keep key block kb.
struct RowTest {
  int32_t qb0, qb1;          // 2p and 2p+1 (equal for the last pair of an odd nb)
  int32_t a0, a1, b0, b1;    // segments touched by qb0 and by qb1
};

__device__ inline RowTest row_test(const FrameCfg& c, int32_t p, int32_t P, int32_t B,
                                   int32_t N, int32_t nb) {
  RowTest rt;
  rt.qb0 = 2 * p;
  rt.qb1 = imin(2 * p + 1, nb - 1);
  block_frame_range(rt.qb0, c.T, P, B, N, &rt.a0, &rt.a1);
  block_frame_range(rt.qb1, c.T, P, B, N, &rt.b0, &rt.b1);
  return rt;
}

__device__ inline void kept_by(const FrameCfg& c, const RowFrames& rf, const RowTest& rt,
                               int32_t kb, int32_t P, int32_t B, int32_t N, bool* k0,
                               bool* k1) {
  *k0 = keeps(c, rf, rt.a0, rt.a1, kb, P, B, N);
  *k1 = rt.qb1 != rt.qb0 && keeps(c, rf, rt.b0, rt.b1, kb, P, B, N);
}

// Sums of two per-thread counts over the workgroup (thread 0's result).
__device__ inline void block_sum2(int32_t (&v)[2], int32_t (*s_cnt)[kRowWaves]) {
  for (int i = 0; i < 2; ++i) {
    for (int off = 32; off > 0; off >>= 1) v[i] += __shfl_xor(v[i], off);
    if (threadIdx.x % 64 == 0) s_cnt[i][threadIdx.x / 64] = v[i];
  }
  __syncthreads();
  if (threadIdx.x == 0)
    for (int i = 0; i < 2; ++i) {
      v[i] = 0;
      for (int w = 0; w < kRowWaves; ++w) v[i] += s_cnt[i][w];
    }
}

__global__ __launch_bounds__(kRowThreads) void count_rows_kernel(
    FrameCfg c, int32_t P, int32_t B, int32_t* __restrict__ row_ptr) {
  __shared__ RowFrames rf;
  __shared__ int32_t s_cnt[2][kRowWaves];
  const int32_t N = (int32_t)mask_tokens(c, P);
  const int32_t nb = ceil_div(N, B);
  const int32_t p = blockIdx.x;
  const RowTest rt = row_test(c, p, P, B, N, nb);
  load_row_frames(c, rt.qb0, rt.qb1, P, B, N, &rf);
  int32_t cnt[2] = {0, 0};   // row qb0, row qb1
  for (int32_t kb = threadIdx.x; kb < nb; kb += kRowThreads) {
    bool k0, k1;
    kept_by(c, rf, rt, kb, P, B, N, &k0, &k1);
    cnt[0] += k0 ? 1 : 0;
    cnt[1] += k1 ? 1 : 0;
  }
  block_sum2(cnt, s_cnt);
  if (threadIdx.x == 0) {
    row_ptr[rt.qb0 + 1] = cnt[0];
    if (rt.qb1 != rt.qb0) row_ptr[rt.qb1 + 1] = cnt[1];
    if (p == 0) row_ptr[0] = 0;
  }
}

// In-place inclusive scan of row_ptr[1 .. rows] (chunks of kScanThreads).
__global__ __launch_bounds__(kScanThreads) void scan_rows_kernel(int32_t rows,
                                                                 int32_t* __restrict__ row_ptr) {
  __shared__ int32_t s_scan[kScanThreads];
  __shared__ int32_t s_carry;
  const int32_t tid = threadIdx.x;
  if (tid == 0) s_carry = 0;
  __syncthreads();
  for (int32_t base = 0; base < rows; base += kScanThreads) {
    const int32_t i = base + tid;
    s_scan[tid] = i < rows ? row_ptr[i + 1] : 0;
    __syncthreads();
    for (int32_t off = 1; off < kScanThreads; off <<= 1) {
      const int32_t y = tid >= off ? s_scan[tid - off] : 0;
      __syncthreads();
      s_scan[tid] += y;
      __syncthreads();
    }
    if (i < rows) row_ptr[i + 1] = s_scan[tid] + s_carry;
    __syncthreads();
    if (tid == kScanThreads - 1) s_carry += s_scan[tid];
    __syncthreads();
  }
}

// The CSR rows of the pair's query blocks (col_idx and/or entry words,
// either may be null).
__global__ __launch_bounds__(kRowThreads) void fill_rows_kernel(
    FrameCfg c, int32_t P, int32_t B, const int32_t* __restrict__ row_ptr,
    int32_t* __restrict__ col_idx, uint32_t* __restrict__ entry) {
  __shared__ RowFrames rf;
  __shared__ int32_t s_wave[2][kRowWaves];
  const int32_t N = (int32_t)mask_tokens(c, P);
  const int32_t nb = ceil_div(N, B);
  const int32_t p = blockIdx.x;
  const RowTest rt = row_test(c, p, P, B, N, nb);
  load_row_frames(c, rt.qb0, rt.qb1, P, B, N, &rf);
  const int32_t lane = threadIdx.x % 64, wave = threadIdx.x / 64;
  int32_t pos[2] = {row_ptr[rt.qb0], row_ptr[rt.qb1]};
  auto attends = [&](int32_t t, int32_t tau) { return seg_attends(c, rf, t, tau); };
  for (int32_t base = 0; base < nb; base += kRowThreads) {
    const int32_t kb = base + (int32_t)threadIdx.x;
    bool k0 = false, k1 = false;
    if (kb < nb) kept_by(c, rf, rt, kb, P, B, N, &k0, &k1);
    const bool keep[2] = {k0, k1};
    int32_t at[2];
    for (int i = 0; i < 2; ++i) {
      const uint64_t bal = __ballot(keep[i]);
      at[i] = __popcll(bal & ((1ull << lane) - 1ull));
      if (lane == 0) s_wave[i][wave] = __popcll(bal);
    }
    __syncthreads();
    for (int i = 0; i < 2; ++i) {
      int32_t off = 0, total = 0;
      for (int w = 0; w < kRowWaves; ++w) {
        off += w < wave ? s_wave[i][w] : 0;
        total += s_wave[i][w];
      }
      at[i] += pos[i] + off;
      pos[i] += total;
    }
    if (k0) {
      if (col_idx) col_idx[at[0]] = kb;
      if (entry) entry[at[0]] = exact_entry(kb, rt.a0, rt.a1, c.T, P, B, N, attends);
    }
    if (k1) {
      if (col_idx) col_idx[at[1]] = kb;
      if (entry) entry[at[1]] = exact_entry(kb, rt.b0, rt.b1, c.T, P, B, N, attends);
    }
    __syncthreads();
  }
}

}  // namespace

bool device_mask_supported(const FrameCfg& c, int32_t P, int32_t B) {
  // A query-block pair touches at most min(T, 2B/P + 2) frames.
  return (int64_t)2 * B / P + 2 <= kMaxRowFrames || c.T <= kMaxRowFrames;
}

hipError_t launch_build_mask_device(const FrameCfg& c, int32_t P, int32_t B,
                                    int32_t* d_row_ptr, int32_t* d_col_idx,
                                    uint32_t* d_entry, hipStream_t stream) {
  const int32_t nb = (int32_t)((mask_tokens(c, P) + B - 1) / B);
  const int32_t npairs = (nb + 1) / 2;
  hipLaunchKernelGGL(count_rows_kernel, dim3(npairs), dim3(kRowThreads), 0, stream, c, P, B,
                     d_row_ptr);
  hipLaunchKernelGGL(scan_rows_kernel, dim3(1), dim3(kScanThreads), 0, stream, nb, d_row_ptr);
  hipLaunchKernelGGL(fill_rows_kernel, dim3(npairs), dim3(kRowThreads), 0, stream, c, P, B,
                     d_row_ptr, d_col_idx, d_entry);
  return hipGetLastError();
}

}  // namespace lvsa
