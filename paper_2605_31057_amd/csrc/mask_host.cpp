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
// The attention kernel walks query blocks in pairs; build_pairs_host merges
// each pair of CSR rows into the pair schedule it reads.
#include <algorithm>
#include <climits>
#include <cstring>

#include "internal.h"

namespace lvsa {

void build_csr_host(const FrameCfg& c, int32_t P, int32_t B,
                    std::vector<int32_t>* row_ptr,
                    std::vector<int32_t>* col_idx,
                    std::vector<uint32_t>* entry) {
  const int32_t T = c.T;
  const int32_t N = (int32_t)mask_tokens(c, P);
  const int32_t nb = ceil_div(N, B);
  const int32_t S = c.text > 0 ? T + 1 : T;   // segments: frames, then text
  std::vector<int32_t> lo(T), hi(T);
  std::vector<uint8_t> anchor(T);
  for (int32_t t = 0; t < T; ++t) {
    anchor[t] = is_anchor(c, t) ? 1 : 0;
    frame_window(c, t, &lo[t], &hi[t]);
  }
  auto attends = [&](int32_t t, int32_t tau) {
    return t == T || tau == T || anchor[tau] != 0 || (lo[t] <= tau && tau <= hi[t]);
  };
  // Per key block: its frames and split point, so an entry word costs four
  // table lookups.
  std::vector<int32_t> kg0, kg1;
  std::vector<uint32_t> kfirst;
  if (entry) {
    kg0.resize(nb);
    kg1.resize(nb);
    kfirst.resize(nb);
    for (int32_t b = 0; b < nb; ++b)
      key_block_split(b, T, P, B, N, &kg0[b], &kg1[b], &kfirst[b]);
  }

  // Pass 1: the distinct rows (one per run of query blocks touching the same
  // frames) into small scratch arrays, and every row's length.
  std::vector<int32_t> uniq;
  std::vector<uint32_t> uniq_e;
  std::vector<int64_t> src(nb);
  row_ptr->assign(nb + 1, 0);
  std::vector<uint8_t> attended(S);
  int32_t prev_first = -1, prev_last = -1;
  int64_t prev_begin = 0, prev_len = 0;
  for (int32_t qb = 0; qb < nb; ++qb) {
    int32_t f0, f1;
    block_frame_range(qb, T, P, B, N, &f0, &f1);
    if (f0 != prev_first || f1 != prev_last) {
      prev_begin = (int64_t)uniq.size();
      if (f1 == T) {
        std::fill(attended.begin(), attended.end(), 1);   // text queries: all
      } else {
        std::memcpy(attended.data(), anchor.data(), T);
        for (int32_t t = f0; t <= f1; ++t)
          std::fill(attended.begin() + lo[t], attended.begin() + hi[t] + 1, 1);
        if (S > T) attended[T] = 1;                       // text keys: all
      }
      int32_t last = -1;
      for (int32_t tau = 0; tau < S; ++tau) {
        if (!attended[tau]) continue;
        int32_t b0, b1;
        segment_blocks(tau, T, P, B, N, &b0, &b1);
        for (int32_t b = std::max(b0, last + 1); b <= b1; ++b) {
          uniq.push_back(b);
          if (entry)
            uniq_e.push_back(exact_word(b, kg0[b], kg1[b], kfirst[b], f0, f1, attends));
        }
        last = std::max(last, b1);
      }
      prev_len = (int64_t)uniq.size() - prev_begin;
      prev_first = f0;
      prev_last = f1;
    }
    src[qb] = prev_begin;
    (*row_ptr)[qb + 1] = (*row_ptr)[qb] + (int32_t)prev_len;
  }

  // Pass 2: one allocation of the final size, rows copied in.
  const int64_t nnz = (*row_ptr)[nb];
  col_idx->resize(nnz);
  if (entry) entry->resize(nnz);
  for (int32_t qb = 0; qb < nb; ++qb) {
    const int64_t dst = (*row_ptr)[qb], len = (*row_ptr)[qb + 1] - dst;
    std::memcpy(col_idx->data() + dst, uniq.data() + src[qb], len * sizeof(int32_t));
    if (entry)
      std::memcpy(entry->data() + dst, uniq_e.data() + src[qb], len * sizeof(uint32_t));
  }
}

// Pair schedule: rows 2p and 2p+1 of the CSR merged (both ascending, no
// repeats), each key block tagged with the rows that hold it.  Two passes
// (row lengths, then the words into arrays of the final size); rows that are
// equal, the common case (the two query blocks touch the same frames), are
// copied with both tags instead of merged.
void build_pairs_host(const std::vector<int32_t>& row_ptr,
                      const std::vector<int32_t>& col_idx,
                      const std::vector<uint32_t>* entry,
                      std::vector<int32_t>* pair_ptr,
                      std::vector<uint32_t>* pair_word,
                      std::vector<uint32_t>* pair_exact) {
  const int32_t nb = (int32_t)row_ptr.size() - 1;
  const int32_t npairs = (nb + 1) / 2;
  const bool exact = entry != nullptr && pair_exact != nullptr;
  const int32_t* ci = col_idx.data();
  // Rows of pair p: [i0, i1) and [k0, k1) (empty for the second row of an
  // odd nb's last pair).
  auto rows = [&](int32_t p, int64_t* i0, int64_t* i1, int64_t* k0, int64_t* k1) {
    *i0 = row_ptr[2 * p];
    *i1 = row_ptr[2 * p + 1];
    *k0 = 2 * p + 1 < nb ? row_ptr[2 * p + 1] : 0;
    *k1 = 2 * p + 1 < nb ? row_ptr[2 * p + 2] : 0;
  };
  auto same = [&](int64_t i0, int64_t i1, int64_t k0, int64_t k1) {
    return k1 - k0 == i1 - i0 &&
           std::memcmp(ci + i0, ci + k0, sizeof(int32_t) * (size_t)(i1 - i0)) == 0;
  };
  // Pass 1: row lengths.
  pair_ptr->assign(npairs + 1, 0);
  for (int32_t p = 0; p < npairs; ++p) {
    int64_t i, ie, k, ke;
    rows(p, &i, &ie, &k, &ke);
    int64_t len = 0;
    if (same(i, ie, k, ke)) {
      len = ie - i;
    } else {
      while (i < ie && k < ke) {
        const int32_t x = ci[i], y = ci[k];
        i += x <= y;
        k += y <= x;
        ++len;
      }
      len += (ie - i) + (ke - k);
    }
    (*pair_ptr)[p + 1] = (*pair_ptr)[p] + (int32_t)len;
  }
  // Pass 2: the words.
  pair_word->resize((size_t)(*pair_ptr)[npairs]);
  if (exact) pair_exact->resize(pair_word->size());
  uint32_t* w = pair_word->data();
  uint32_t* we = exact ? pair_exact->data() : nullptr;
  const uint32_t* en = exact ? entry->data() : nullptr;
  for (int32_t p = 0; p < npairs; ++p) {
    int64_t i, ie, k, ke;
    rows(p, &i, &ie, &k, &ke);
    int64_t o = (*pair_ptr)[p];
    if (same(i, ie, k, ke)) {
      for (int64_t n = 0; n < ie - i; ++n) w[o + n] = pair_word_of(ci[i + n], true, true);
      if (exact)
        for (int64_t n = 0; n < ie - i; ++n) we[o + n] = pair_exact_word(en[i + n], en[k + n]);
      continue;
    }
    while (i < ie || k < ke) {
      const int32_t x = i < ie ? ci[i] : INT32_MAX;
      const int32_t y = k < ke ? ci[k] : INT32_MAX;
      const int32_t kb = x < y ? x : y;
      const bool in0 = x == kb, in1 = y == kb;
      w[o] = pair_word_of(kb, in0, in1);
      if (exact) we[o] = pair_exact_word(in0 ? en[i] : 0u, in1 ? en[k] : 0u);
      ++o;
      if (in0) ++i;
      if (in1) ++k;
    }
  }
}

}  // namespace lvsa
