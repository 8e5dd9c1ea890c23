// mask_device.hip -- LVSA mask builder on the GPU.
//
// Computes the same block CSR as the host builder (the LVSA frame sets of
// Sec. 2: Def. 2, Eq. 3, Alg. 1, expanded to blocks by the any-overlap rule)
// and the pair schedule the attention kernel reads, without a host round
// trip, so a denoising loop can rebuild the mask for step s on the stream
// that then runs attention.
//
// Two rounds of three launches on the stream, first over the CSR rows (one
// per query block), then over the pair rows (one per query-block pair 2p,
// 2p+1: a key block is listed when either block keeps it):
//   1. one workgroup per row: the windows of the row's frames (Alg. 1) into
//      LDS, then every key block tested in parallel; the count of listed
//      blocks goes to row_ptr[r + 1];
//   2. one workgroup: in-place inclusive scan of the counts;
//   3. one workgroup per row: the same test again, listed key blocks
//      compacted in ascending order (wave ballots and a per-chunk prefix) and
//      written as block indices, token-exact entry words or pair words.
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
  int32_t f0, f1;                  // segments touched by the row's query blocks
  int16_t lo[kMaxRowFrames];       // window of frame f0 + i
  int16_t hi[kMaxRowFrames];
};

// The query blocks of row r: r itself (CSR rows), or 2r and 2r+1 (pair rows;
// the last pair of an odd nb has one block, qb1 == qb0).
__device__ inline void row_blocks(bool pair, int32_t r, int32_t nb, int32_t* qb0,
                                  int32_t* qb1) {
  *qb0 = pair ? 2 * r : r;
  *qb1 = pair ? imin(2 * r + 1, nb - 1) : r;
}

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

// Per-row test: which of the row's query blocks keep key block kb.
struct RowTest {
  int32_t qb0, qb1;          // query blocks (equal for a CSR row)
  int32_t a0, a1, b0, b1;    // segments touched by qb0 and by qb1
};

__device__ inline RowTest row_test(const FrameCfg& c, bool pair, int32_t r, int32_t P,
                                   int32_t B, int32_t N, int32_t nb) {
  RowTest rt;
  row_blocks(pair, r, nb, &rt.qb0, &rt.qb1);
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

template <bool PAIR>
__global__ __launch_bounds__(kRowThreads) void count_rows_kernel(
    FrameCfg c, int32_t P, int32_t B, int32_t* __restrict__ row_ptr) {
  __shared__ RowFrames rf;
  __shared__ int32_t s_cnt[kRowWaves];
  const int32_t N = (int32_t)mask_tokens(c, P);
  const int32_t nb = ceil_div(N, B);
  const int32_t r = blockIdx.x;
  const RowTest rt = row_test(c, PAIR, r, P, B, N, nb);
  load_row_frames(c, rt.qb0, rt.qb1, P, B, N, &rf);
  int32_t cnt = 0;
  for (int32_t kb = threadIdx.x; kb < nb; kb += kRowThreads) {
    bool k0, k1;
    kept_by(c, rf, rt, kb, P, B, N, &k0, &k1);
    cnt += (k0 || k1) ? 1 : 0;
  }
  // wave sums, then the workgroup sum
  for (int off = 32; off > 0; off >>= 1) cnt += __shfl_xor(cnt, off);
  if (threadIdx.x % 64 == 0) s_cnt[threadIdx.x / 64] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t total = 0;
    for (int w = 0; w < kRowWaves; ++w) total += s_cnt[w];
    row_ptr[r + 1] = total;
    if (r == 0) row_ptr[0] = 0;
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

// CSR rows: col_idx and/or entry words (either may be null).  Pair rows:
// pair words into `words`, in the token-exact form when `exact`.
template <bool PAIR>
__global__ __launch_bounds__(kRowThreads) void fill_rows_kernel(
    FrameCfg c, int32_t P, int32_t B, const int32_t* __restrict__ row_ptr,
    int32_t* __restrict__ col_idx, uint32_t* __restrict__ words, bool exact) {
  __shared__ RowFrames rf;
  __shared__ int32_t s_wave[kRowWaves];
  const int32_t N = (int32_t)mask_tokens(c, P);
  const int32_t nb = ceil_div(N, B);
  const int32_t r = blockIdx.x;
  const RowTest rt = row_test(c, PAIR, r, P, B, N, nb);
  load_row_frames(c, rt.qb0, rt.qb1, P, B, N, &rf);
  const int32_t lane = threadIdx.x % 64, wave = threadIdx.x / 64;
  int32_t pos = row_ptr[r];
  auto attends = [&](int32_t t, int32_t tau) { return seg_attends(c, rf, t, tau); };
  for (int32_t base = 0; base < nb; base += kRowThreads) {
    const int32_t kb = base + (int32_t)threadIdx.x;
    bool k0 = false, k1 = false;
    if (kb < nb) kept_by(c, rf, rt, kb, P, B, N, &k0, &k1);
    const bool keep = k0 || k1;
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
      if (!PAIR) {
        if (col_idx) col_idx[at] = kb;
        if (words) words[at] = exact_entry(kb, rt.a0, rt.a1, c.T, P, B, N, attends);
      } else if (exact) {
        const uint32_t e0 = k0 ? exact_entry(kb, rt.a0, rt.a1, c.T, P, B, N, attends) : 0u;
        const uint32_t e1 = k1 ? exact_entry(kb, rt.b0, rt.b1, c.T, P, B, N, attends) : 0u;
        words[at] = pair_exact_word(e0, e1);
      } else {
        words[at] = pair_word_of(kb, k0, k1);
      }
    }
    pos += total;
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
                                    uint32_t* d_entry, int32_t* d_pair_ptr,
                                    uint32_t* d_pair_word, bool exact,
                                    hipStream_t stream) {
  const int32_t nb = (int32_t)((mask_tokens(c, P) + B - 1) / B);
  const int32_t npairs = (nb + 1) / 2;
  hipLaunchKernelGGL(count_rows_kernel<false>, dim3(nb), dim3(kRowThreads), 0, stream, c, P,
                     B, d_row_ptr);
  hipLaunchKernelGGL(scan_rows_kernel, dim3(1), dim3(kScanThreads), 0, stream, nb, d_row_ptr);
  hipLaunchKernelGGL(fill_rows_kernel<false>, dim3(nb), dim3(kRowThreads), 0, stream, c, P, B,
                     d_row_ptr, d_col_idx, d_entry, false);
  hipLaunchKernelGGL(count_rows_kernel<true>, dim3(npairs), dim3(kRowThreads), 0, stream, c,
                     P, B, d_pair_ptr);
  hipLaunchKernelGGL(scan_rows_kernel, dim3(1), dim3(kScanThreads), 0, stream, npairs,
                     d_pair_ptr);
  hipLaunchKernelGGL(fill_rows_kernel<true>, dim3(npairs), dim3(kRowThreads), 0, stream, c, P,
                     B, d_pair_ptr, nullptr, d_pair_word, exact);
  return hipGetLastError();
}

}  // namespace lvsa
