// mask_host.cpp -- host LVSA mask builder: frame sets -> block CSR.
//
// The paper builds the index metadata on the CPU once per denoising step
// (Sec. 2, cost remark after Alg. 1 and the end of "Rotating periodic global
// frames").  Query block qb keeps key block kb iff some frame t touched by qb
// and some frame tau touched by kb have tau in A(t), where
// A(t) = G^s U [lo(t), hi(t)].
//
// For each query block the attended frames are gathered into a flag array,
// then each attended frame contributes its block range
// [tau*P/B, ((tau+1)*P-1)/B]; ranges come in ascending order and overlap only
// at a shared straddling block, so a running "last emitted" index keeps the
// row ascending and free of repeats.  Consecutive query blocks that touch
// the same frames have identical rows, which are copied.
//
// Text tokens (dual-stream models) follow the video tokens as one more
// segment T: every query attends to them and a query block touching them
// attends to every segment.
//
// The token-exact entry words (lvsa.h) are built alongside when asked for:
// one word per kept block, from the two (at most) frames of each side.
//
// A rebuild runs once per denoising step, so its cost is mostly that of
// touching fresh memory: the working arrays are per-thread and kept between
// calls, and the output arrays come from the handles the caller has freed
// (api.cpp), so a loop that frees step s's mask before building step s+1's
// allocates nothing after the first step.
#include <algorithm>
#include <cstring>

#include "internal.h"

namespace lvsa {

namespace {

// Working arrays of one thread's builds, kept between calls.
struct HostScratch {
  std::vector<int32_t> lo, hi, kg0, kg1, uniq;
  std::vector<uint32_t> kfirst, uniq_e;
  std::vector<int64_t> src;
  std::vector<uint8_t> anchor, attended;
};

HostScratch& host_scratch() {
  thread_local HostScratch s;
  return s;
}

// Room for `more` values past `used` (grown geometrically, so rarely).
template <typename V>
void ensure(std::vector<V>& v, size_t used, size_t more) {
  if (used + more > v.size()) v.resize(std::max(2 * v.size(), used + more));
}

}  // namespace

void build_csr_host(const FrameCfg& c, int32_t P, int32_t B,
                    std::vector<int32_t>* row_ptr,
                    std::vector<int32_t>* col_idx,
                    std::vector<uint32_t>* entry) {
  const int32_t T = c.T;
  const int32_t N = (int32_t)mask_tokens(c, P);
  const int32_t nb = ceil_div(N, B);
  const int32_t S = c.text > 0 ? T + 1 : T;   // segments: frames, then text
  HostScratch& hs = host_scratch();
  hs.lo.resize(T);
  hs.hi.resize(T);
  hs.anchor.resize(T);
  int32_t* const lo = hs.lo.data();
  int32_t* const hi = hs.hi.data();
  uint8_t* const anchor = hs.anchor.data();
  for (int32_t t = 0; t < T; ++t) {
    anchor[t] = is_anchor(c, t) ? 1 : 0;
    frame_window(c, t, &lo[t], &hi[t]);
  }
  auto attends = [&](int32_t t, int32_t tau) {
    return t == T || tau == T || anchor[tau] != 0 || (lo[t] <= tau && tau <= hi[t]);
  };
  // Per key block: its frames and split point, so an entry word costs four
  // table lookups.
  if (entry) {
    hs.kg0.resize(nb);
    hs.kg1.resize(nb);
    hs.kfirst.resize(nb);
    for (int32_t b = 0; b < nb; ++b)
      key_block_split(b, T, P, B, N, &hs.kg0[b], &hs.kg1[b], &hs.kfirst[b]);
  }
  const int32_t* const kg0 = hs.kg0.data();
  const int32_t* const kg1 = hs.kg1.data();
  const uint32_t* const kfirst = hs.kfirst.data();

  // Pass 1: the distinct rows (one per run of query blocks touching the same
  // frames) into the working arrays, and every row's length.
  hs.src.resize(nb);
  hs.attended.resize(S);
  int64_t* const src = hs.src.data();
  uint8_t* const attended = hs.attended.data();
  row_ptr->assign(nb + 1, 0);
  int32_t* const rp = row_ptr->data();
  size_t used = 0;
  int32_t prev_first = -1, prev_last = -1;
  int64_t prev_begin = 0, prev_len = 0;
  for (int32_t qb = 0; qb < nb; ++qb) {
    int32_t f0, f1;
    block_frame_range(qb, T, P, B, N, &f0, &f1);
    if (f0 != prev_first || f1 != prev_last) {
      ensure(hs.uniq, used, nb);
      if (entry) ensure(hs.uniq_e, used, nb);
      int32_t* const u = hs.uniq.data();
      uint32_t* const ue = hs.uniq_e.data();
      prev_begin = (int64_t)used;
      if (f1 == T) {
        std::memset(attended, 1, S);                      // text queries: all
      } else {
        std::memcpy(attended, anchor, T);
        for (int32_t t = f0; t <= f1; ++t) std::memset(attended + lo[t], 1, hi[t] - lo[t] + 1);
        if (S > T) attended[T] = 1;                       // text keys: all
      }
      int32_t last = -1;
      for (int32_t tau = 0; tau < S; ++tau) {
        if (!attended[tau]) continue;
        int32_t b0, b1;
        segment_blocks(tau, T, P, B, N, &b0, &b1);
        const int32_t from = std::max(b0, last + 1);
        if (entry) {
          // A block inside segment tau has the same word as its neighbours
          // but for kb: the 2x2 pattern collapses to tau's two rows.
          const uint32_t q0 = attends(f0, tau) ? 3u : 0u, q1 = attends(f1, tau) ? 12u : 0u;
          const uint32_t inner = ((uint32_t)B << 16) | ((q0 | q1) << 24);
          for (int32_t b = from; b <= b1; ++b)
            ue[used + (b - from)] = kg0[b] == kg1[b]
                                        ? (uint32_t)b | inner
                                        : exact_word(b, kg0[b], kg1[b], kfirst[b], f0, f1, attends);
        }
        for (int32_t b = from; b <= b1; ++b) u[used++] = b;
        last = std::max(last, b1);
      }
      prev_len = (int64_t)used - prev_begin;
      prev_first = f0;
      prev_last = f1;
    }
    src[qb] = prev_begin;
    rp[qb + 1] = rp[qb] + (int32_t)prev_len;
  }

  // Pass 2: one allocation of the final size, rows copied in.
  const int64_t nnz = rp[nb];
  col_idx->resize(nnz);
  if (entry) entry->resize(nnz);
  const int32_t* const u = hs.uniq.data();
  const uint32_t* const ue = hs.uniq_e.data();
  for (int32_t qb = 0; qb < nb; ++qb) {
    const int64_t dst = rp[qb], len = rp[qb + 1] - dst;
    std::memcpy(col_idx->data() + dst, u + src[qb], len * sizeof(int32_t));
    if (entry) std::memcpy(entry->data() + dst, ue + src[qb], len * sizeof(uint32_t));
  }
}

}  // namespace lvsa
