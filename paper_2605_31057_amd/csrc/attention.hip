// attention.hip -- block-sparse and dense flash-attention forward for gfx950.
//
// Computes Eq. 2 of the LVSA paper (softmax attention restricted to a key
// set) with the key set of every query block given by a block CSR, and Eq. 1
// (all keys) with the same kernel visiting every key block.
//
// Work decomposition
//   A tile is (head, pair of query blocks 2p and 2p+1): 2*BLOCK query rows,
//   NW = 2*BLOCK/32 waves (8 at BLOCK = 128) of 32 rows each; waves
//   0..NW/2-1 hold rows of query block 2p, the others rows of 2p+1.  The
//   workgroup walks the union of the two blocks' key lists one key block per
//   step, and every wave takes all BLOCK keys of the step for its rows.
//   Adjacent query blocks mostly keep the same key blocks (they touch the
//   same frames), so each K/V tile brought from HBM/L2 into LDS serves
//   2*BLOCK query rows; a key block that only one of the two keeps is masked
//   out (no valid keys) for the other's waves.  One persistent workgroup per
//   compute unit takes tiles through atomic counters (fetch_tile).
//
// The merged walk
//   A tile's key blocks are the union of CSR rows 2p and 2p+1, walked in
//   descending order, each key block once with a flag per query block.  At
//   the start of the tile the workgroup merges the two rows in LDS: every
//   entry's position in the union is its index in its own row plus the
//   entries of the other row above it (a binary search) minus the entries
//   above it that both rows hold (a ballot count), and the step words are
//   written there.  The step loop then reads one word per step, three steps
//   ahead (K tiles are loaded two steps ahead).  The sparse modes take at most
//   WALK_CAP key blocks (checked before launch), so one merge covers any
//   pair.  Dense attention up to WALK_CAP key blocks runs the block mode with
//   no CSR: the words are written directly instead of merged.  The mask is
//   only read, so any number of launches can share it.
//
// Schedule ("ping-pong", one key block per step)
//   Waves w and w + NW/2 (which share a SIMD when NW = 8) run half a step
//   apart: while one is in its GEMM phase (O += P(j) V(j), S(j+1) = K(j+1)
//   Q^T: MFMA with fragments from LDS) the other is in its softmax phase (row
//   max, exponentials, P in bf16: VALU), so the matrix
//   core and the VALU of each SIMD are busy at the same time.  A barrier ends
//   every half step.  LDS holds two K stages and two V stages (slab layout,
//   see below); K(j+2) and V(j+1) stream from HBM/L2 into the stages freed by
//   step j-1 with buffer loads that write LDS directly, issued during the
//   first half of step j and waited for at its end.  The buffer resource's
//   size bound turns rows at or past N (ragged last block) into zeros.
//   Row sums (RowSums): in the block mode, 64 fp32 adds per step in the
//   softmax phase; in the other modes the matrix core, where a 16x16x32 MFMA
//   with a constant 0/1 A operand adds up each 16-key step of P for all 32
//   rows of the wave in the GEMM phase (8 small MFMAs per step, summing
//   exactly the bf16 P that multiplies V).
//   A whole key block per step keeps the per-step costs (two barriers, the
//   loop, the load set-up) small against the step's 72 MFMAs per wave; S
//   (64 registers) and P (32) then fill the register file, so the GEMM
//   phase finishes P(j) before it produces S(j+1), and masks run only in a
//   wave-uniform branch, one compare into VCC and one select per score.
//
// Contractions (bf16 MFMA 32x32x16, fp32 accumulate)
//     S^T = K Q^T     A = K rows (LDS, ds_read_b128), B = Q rows (registers)
//     O^T += V^T P^T  A = V^T (LDS, ds_read_b64_tr_b16), B = P (registers)
//   The transposed products put one query row per lane (lanes l and l^32
//   share row l%32), so row statistics are in-lane reductions plus one
//   permlane32 exchange, and P never leaves registers.
//   MFMA 32x32 lane layout (lane l, half h = l/32, i = l%32): A row i and B
//   column i carry k-slots 8h..8h+7; C register r holds row 8*(r/4)+4h+(r%4),
//   column i.  k-slot order only has to agree between A and B, so the key
//   held by S^T's C register r is paired with the V^T element of that key.
//
// Online softmax (fp32, base 2): m = running max of s*log2(e)/sqrt(d),
// p = exp2(s*log2(e)/sqrt(d) - m), l = sum p.  The running max is raised only
// when a new row max exceeds it by more than 8 (p then stays below 2^8), which
// skips most rescales of O; the result is exact either way because O and l
// always use the same m.
#include <atomic>

#include "internal.h"

namespace lvsa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int D = 128;             // head_dim
constexpr float RESCALE_SLACK = 8.f;

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base,
                                                            uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0,
                                           bytes, 0x00020000);
}

__device__ __forceinline__ float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x),
                                            __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// LDS tile layout ("slabs").  A BLOCK x 128 tile (one key block) is stored
// as 4 slabs of 32 columns; a slab row is 64 bytes (4 chunks of 16 bytes) and
// rows follow each other, so tile byte (slab, row, chunk) =
// slab*BLOCK*64 + row*64 + chunk*16.
// The chunk is XORed with x(row) = (row/4) % 4.  With 64 banks of 4 bytes:
//   - ds_read_b128 (served 16 lanes at a time) reads 16 consecutive rows at
//     one logical chunk: 4 rows share a bank window and the XOR separates them;
//   - ds_read_b64_tr_b16 (served 32 lanes at a time) reads 4 consecutive rows
//     x 4 chunks, i.e. 256 contiguous bytes.
// Both are free of bank conflicts, and every fragment address an unrolled loop
// needs is one of two per-lane bases plus an immediate offset.
constexpr int SLAB_ROW = 64;
__device__ __forceinline__ int xsw(int row) { return (row >> 2) & 3; }

template <int BLOCK>
struct Tile {
  static constexpr int NW = 2 * BLOCK / 32;         // waves (32 query rows each)
  static constexpr int NT = NW * 64;                // threads
  static constexpr int KTW = BLOCK / 32;            // 32-key tiles per step
  static constexpr int SLAB = BLOCK * SLAB_ROW;     // bytes per slab
  static constexpr int BYTES = 4 * SLAB;            // bytes per tile
  static constexpr int INSTR = BYTES / 1024;        // 1 KiB wave loads per tile
  static constexpr int LOADS = INSTR / NW;          // per wave per tile
  static constexpr int IPS = SLAB / 1024;           // wave loads per slab
  static_assert(LOADS * NW == INSTR, "tile load mapping");
};

// One wave load (1 KiB) of a K or V tile into LDS at byte address lds_dst:
// `rsrc` starts at the tile's first row, `voff` = the lane's part of the
// global byte offset plus the load's uniform part (LoadPlan).  Rows at or
// past N fall outside the buffer resource and read as zeros.  The loads are
// issued from inline assembly so the compiler does not track them: they are
// waited for explicitly (vmcnt(0) plus a barrier) at the end of the step, and
// no compiler-inserted wait can stall the phases in between.  The nop is the
// wait state gfx9 needs between an SALU write of M0 and an LDS-DMA
// instruction (the compiler cannot see into the statement to add it).
__device__ __forceinline__ void issue_load(uint32_t lds_dst, __amdgpu_buffer_rsrc_t rsrc,
                                           uint32_t voff) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %1, %2, 0 offen lds"
      :
      : "s"(lds_dst), "v"(voff), "s"(rsrc)
      : "memory", "m0");
}

// Buffer resource over rows kb*BLOCK .. N-1 of one head of K or V; a key
// block index outside [0, nb) yields an empty resource (all loads read 0).
template <int BLOCK>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const __bf16* head_base,
                                                            int64_t row_elems,
                                                            uint32_t head_bytes,
                                                            int kb, int nb) {
  const bool ok = (uint32_t)kb < (uint32_t)nb;
  const int64_t skip = ok ? (int64_t)kb * BLOCK * row_elems : 0;
  const uint32_t bytes = ok ? head_bytes - (uint32_t)(skip * 2) : 0u;
  return make_rsrc(head_base + skip, bytes);
}

// Per-wave load plan: wave w's load j of a tile fills tile bytes
// 1024*(w + NW*j): slab j, rows 16*w + lane/4 (NW = IPS: one wave per 16-row
// band of a slab), physical chunk lane%4, which holds logical chunk
// (lane%4) ^ x(row) = (lane%4) ^ (lane/16).  Global offset: lane_off plus
// 64*j; LDS offset: lds_w plus 1024*NW*j.
template <int BLOCK>
struct LoadPlan {
  uint32_t lane_off;   // (16*w + lane/4)*row_bytes + 16*((lane%4) ^ (lane/16))
  uint32_t lds_w;      // 1024*w (uniform)
};

template <int BLOCK>
__device__ __forceinline__ LoadPlan<BLOCK> load_plan(uint32_t row_bytes, int wave,
                                                     int lane) {
  using TL = Tile<BLOCK>;
  static_assert(TL::NW == TL::IPS, "one wave per 16-row band of a slab");
  LoadPlan<BLOCK> lp;
  lp.lane_off = (uint32_t)(16 * wave + lane / 4) * row_bytes +
                16u * (uint32_t)((lane % 4) ^ (lane / 16));
  lp.lds_w = (uint32_t)__builtin_amdgcn_readfirstlane(1024u * (uint32_t)wave);
  return lp;
}

template <int BLOCK>
__device__ __forceinline__ void issue_tile(uint32_t lds, __amdgpu_buffer_rsrc_t rsrc,
                                           const LoadPlan<BLOCK>& lp) {
  using TL = Tile<BLOCK>;
#pragma unroll
  for (int j = 0; j < TL::LOADS; ++j)
    issue_load(lds + lp.lds_w + 1024u * TL::NW * j, rsrc, lp.lane_off + 64u * j);
}

// The loads of one pipeline step: the next K tile and the next V tile, spread
// over the first phase of the step so the wave never stalls on issuing them.
// Issued unconditionally: near the end of a row the key-block indices repeat
// the last block and the loads land in slots no later step reads.
template <int BLOCK>
struct StepLoads {
  uint32_t k_dst, v_dst;                 // LDS tile addresses
  __amdgpu_buffer_rsrc_t rk, rv;         // resources starting at the tiles
  const LoadPlan<BLOCK>* kp;
  const LoadPlan<BLOCK>* vp;
};

template <int BLOCK>
__device__ __forceinline__ void issue_step_load(const StepLoads<BLOCK>& sl, int i) {
  using TL = Tile<BLOCK>;
  if (i < TL::LOADS)
    issue_load(sl.k_dst + sl.kp->lds_w + 1024u * TL::NW * i, sl.rk, sl.kp->lane_off + 64u * i);
  else
    issue_load(sl.v_dst + sl.vp->lds_w + 1024u * TL::NW * (i - TL::LOADS), sl.rv,
               sl.vp->lane_off + 64u * (i - TL::LOADS));
}

__device__ __forceinline__ void wait_loads_and_sync() {
  __builtin_amdgcn_s_waitcnt(0);  // vmcnt(0) expcnt(0) lgkmcnt(0)
  __syncthreads();
}

template <int BLOCK>
struct Scores {
  f32x16 s[Tile<BLOCK>::KTW];   // one 32-key tile each
};

// Per-lane LDS byte offsets (within a tile) of the K and V fragments.
struct FragAddr {
  uint32_t k_even, k_odd;   // K rows of this lane, d-steps 2t / 2t+1
  uint32_t v_lo, v_hi;      // V rows for k-slots 0..3 / 4..7 (transposing read)
};

__device__ __forceinline__ FragAddr frag_addr(int lane) {
  const int hl = lane / 32, li = lane % 32;
  FragAddr f;
  // K: row 32*kt + li, d = 16*stp + 8*hl: slab stp/2, logical chunk
  // 2*(stp%2) + hl.  x(row) = (li/4)%4 for every kt.
  const int krow = li;
  const int kx = xsw(krow);
  f.k_even = krow * SLAB_ROW + ((hl ^ kx) * 16);
  f.k_odd = krow * SLAB_ROW + (((2 + hl) ^ kx) * 16);
  // V: the transposing read gives lane (group g = lane/16, j = lane%16)
  // element e of the group's chunk 4e + j/4, entry j%4.  Source lane
  // sl = 4e + q points at V row (key e of its half: 4*(g/2) + sl/4) and
  // columns 16*(g%2) + 4q .. +3 of the slab (logical chunk 2*(g%2) + q/2,
  // byte half q%2).  Rows +8 hold k-slots 4..7.
  const int g = lane / 16, sl = lane % 16;
  const int vrow = 4 * (g / 2) + sl / 4;
  const int lc = 2 * (g % 2) + (sl % 4) / 2;
  const int half = (sl % 2) * 8;
  f.v_lo = vrow * SLAB_ROW + ((lc ^ xsw(vrow)) * 16) + half;
  f.v_hi = (vrow + 8) * SLAB_ROW + ((lc ^ xsw(vrow + 8)) * 16) + half;
  return f;
}

// S^T = K Q^T for the keys of one step (K tile at lds_k).
template <int BLOCK>
__device__ __forceinline__ void compute_scores(const char* lds_k, const bf16x8 (&qf)[8],
                                               Scores<BLOCK>& sc, const FragAddr& fa) {
  using TL = Tile<BLOCK>;
#pragma unroll
  for (int kt = 0; kt < TL::KTW; ++kt) {
    f32x16 acc = f32x16{};
#pragma unroll
    for (int stp = 0; stp < 8; ++stp) {
      const uint32_t off = ((stp & 1) ? fa.k_odd : fa.k_even) +
                           (stp / 2) * TL::SLAB + kt * 32 * SLAB_ROW;
      const bf16x8 a = *(const bf16x8*)(lds_k + off);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[stp], acc, 0, 0, 0);
    }
    sc.s[kt] = acc;
  }
}

// Row sums l are kept one of two ways (RSUM): on the matrix core, as a
// 16x16 MFMA accumulator that the GEMM phase adds each step's bf16 P into
// (lane c < 16 holds rows c and c + 16), or on the VALU, as two partial sums
// per lane of the fp32 probabilities of the lane's own keys that the softmax
// phase adds into (lanes l and l^32 hold the two halves of a row's keys).
// Timed interleaved on one board, the VALU form is 0.4-0.7% faster in the
// block mode (four workloads), and slower in the dense mode (0.4-0.9%: long
// walks) and in the token-exact mode (0.4%: its masking adds VALU work to the
// same phases).
enum RowSums { RSUM_MFMA = 0, RSUM_VALU = 1 };

struct WaveState {
  f32x16 o[4];   // O^T tiles [d tile]: d = 32*dt + C row
  float m;       // running max (log2 domain), shared by lanes l, l^32
  f32x4 l;       // RSUM_MFMA: row sums (16x16 C tile)
  float l0, l1;  // RSUM_VALU: partial row sums of the lane's keys
};

// Keys at or past N (ragged last block) do not exist: their scores become
// -inf.  `valid` = N - first key of the block (0: no key is valid).  Per
// score one compare of a constant into VCC and one select, a scheduling
// barrier every 4 scores so that few compare results are live at once.
template <int BLOCK>
__device__ __forceinline__ void mask_tail(Scores<BLOCK>& sc, int lane, int valid) {
  using TL = Tile<BLOCK>;
  const int hl = lane / 32;
  if (valid < BLOCK) {
    const int lim = valid - 4 * hl;   // key 4*hl + c is valid iff c < lim
#pragma unroll
    for (int kt = 0; kt < TL::KTW; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        if (r % 4 == 0) __builtin_amdgcn_sched_barrier(0);
        const int c = 32 * kt + 8 * (r / 4) + (r % 4);
        sc.s[kt][r] = c < lim ? sc.s[kt][r] : -__builtin_inff();
      }
  }
}

// Token-exact form: the 4-bit pattern of the wave's query block for this key
// block says which query-frame / key-frame parts are attended (bit 2a+b, a =
// the lane's query row lies in the query block's second frame, b = the key
// lies in the key block's second frame, which starts kfirst keys in; 0 = the
// query block does not keep the key block).  A row's kept keys are then one
// range [klo, khi) of the block, also clipped at `valid` = N minus the
// block's first key.  Scores outside the range become -inf.  Blocks whose
// every part is attended and that are not ragged skip the masking.
//
// Key kbase + c is kept iff the unsigned c + kbase - klo is below the range's
// width: per score one add of a constant, one compare into VCC and one
// select.  A scheduling barrier every 4 scores keeps the compiler from
// computing many compare results ahead (each holds an SGPR pair).
//
// The lane's query row lies in the second frame iff its row index within the
// wave's 32 rows reaches `sec_from` (wave-uniform); the lane index is
// recomputed here rather than held in a register through the loop.
template <int BLOCK>
__device__ __forceinline__ void mask_exact(Scores<BLOCK>& sc, uint32_t pat, int kfirst,
                                           int valid, int sec_from) {
  using TL = Tile<BLOCK>;
  if (pat != 0xFu || valid < BLOCK) {
    const int lane = (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
    const int hl = lane / 32, li = lane % 32;
    const uint32_t bits = li >= sec_from ? pat >> 2 : pat;
    const int klo = (bits & 1u) ? 0 : kfirst;
    const int khi = (bits & 2u) ? valid : min(kfirst, valid);
    const uint32_t shift = (uint32_t)(4 * hl - klo);
    const uint32_t width = (uint32_t)max(khi - klo, 0);
#pragma unroll
    for (int kt = 0; kt < TL::KTW; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        if (r % 4 == 0) __builtin_amdgcn_sched_barrier(0);
        const uint32_t c = (uint32_t)(32 * kt + 8 * (r / 4) + (r % 4));
        sc.s[kt][r] = c + shift < width ? sc.s[kt][r] : -__builtin_inff();
      }
  }
}

template <int BLOCK>
struct Probs {
  bf16x8 p[Tile<BLOCK>::KTW][2];   // [key tile][k-step half]
};

// Softmax phase of the ping-pong schedule: block j's scores (in `sc`) become
// its probabilities P (bf16, in `pr`), with the running max and, when the
// max is raised, the rescale of O and l done here so that the next GEMM phase
// only multiplies (with RSUM_VALU, P is also added into l here; with
// RSUM_MFMA the GEMM phase does it).  `sl` (may be null) carries tile
// loads to issue along the way.  Scheduling barriers every 8 scores keep the
// compiler from hoisting many exponentials at once (S, P, O and Q already
// fill the register file).
template <int BLOCK, int RSUM>
__device__ __forceinline__ void softmax_phase(const Scores<BLOCK>& sc, WaveState& st,
                                              Probs<BLOCK>& pr, float scale_log2,
                                              const StepLoads<BLOCK>* sl) {
  using TL = Tile<BLOCK>;
  constexpr int NE = 16 * TL::KTW;   // scores per lane
  constexpr int NLOADS = 2 * TL::LOADS;
  constexpr int LOAD_EVERY = NE / NLOADS >= 2 ? NE / NLOADS : 2;   // scores per load
  int issued = 0;
  float mx = -__builtin_inff();
#pragma unroll
  for (int e = 0; e < NE; ++e) mx = fmaxf(mx, sc.s[e / 16][e % 16]);
  const float m = pair_max(mx) * scale_log2;
  const bool raise = m > st.m + RESCALE_SLACK;
  if (__builtin_amdgcn_ballot_w64(raise)) {
    const float a = raise ? __builtin_amdgcn_exp2f(st.m - m) : 1.f;
    st.m = raise ? m : st.m;
    if constexpr (RSUM == RSUM_MFMA) {
      // l tile: register 0 of lane c holds row c, register 1 row c + 16.
      const float a16 = __shfl_xor(a, 16);
      st.l[0] *= a;
      st.l[1] *= a16;
    } else {
      st.l0 *= a;
      st.l1 *= a;
    }
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) st.o[dt] *= a;
  }
  const float msub = st.m == -__builtin_inff() ? 0.f : st.m;
#pragma unroll
  for (int el = 0; el < NE; el += 2) {
    if (el % 8 == 0) __builtin_amdgcn_sched_barrier(0);
    if (sl && el % LOAD_EVERY == 0 && issued < NLOADS) issue_step_load<BLOCK>(*sl, issued++);
    const float a =
        __builtin_amdgcn_exp2f(__builtin_fmaf(sc.s[el / 16][el % 16], scale_log2, -msub));
    const float b = __builtin_amdgcn_exp2f(
        __builtin_fmaf(sc.s[(el + 1) / 16][(el + 1) % 16], scale_log2, -msub));
    if constexpr (RSUM == RSUM_VALU) {
      if (el % 4 == 0) st.l0 += a + b; else st.l1 += a + b;
    }
    const bf16x2 pk = {(__bf16)a, (__bf16)b};
    pr.p[el / 16][(el % 16) / 8][el % 8] = pk[0];
    pr.p[el / 16][(el % 16) / 8][el % 8 + 1] = pk[1];
  }
  if (sl)
    for (; issued < NLOADS; ++issued) issue_step_load<BLOCK>(*sl, issued);
}

// GEMM phase of the ping-pong schedule: with RSUM_MFMA, l += the row sums of
// P(j) (one 16x16x32 MFMA per 16-key step, `ones` its A operand); then
// O += P(j) V(j) and S(j+1) = K(j+1) Q^T into `sc`, with K and V fragments
// read AHEAD MFMAs early and the tile loads in `sl` (may be null) spread over
// the phase.  The row-sum MFMAs come first: their operands are already in
// registers, so they run while the first fragments arrive from LDS (0.2-1.2%
// faster than after P V, interleaved on one board).
template <int BLOCK, int RSUM>
__device__ __forceinline__ void gemm_phase(const char* lds_k, const char* lds_v,
                                           const bf16x8 (&qf)[8], Scores<BLOCK>& sc,
                                           const Probs<BLOCK>& pr, WaveState& st,
                                           const FragAddr& fa, const bf16x8& ones,
                                           const StepLoads<BLOCK>* sl) {
  using TL = Tile<BLOCK>;
  constexpr int NS = 8 * TL::KTW;   // S MFMAs: (key tile, d-step)
  constexpr int NP = 8 * TL::KTW;   // PV fragments: (d tile, key tile, k-step half)
  constexpr int NF = NS + NP;
  constexpr int AHEAD = 3;
  constexpr int NLOADS = 2 * TL::LOADS;
  // Fragment i < NP: V^T, d tile i/(2*KTW), key tile (i/2)%KTW, k-step half
  // i%2.  Fragment NP + f: K, key tile f/8, d-step f%8.  MFMAs on one
  // accumulator follow each other, and P(j) (with its row sums) is done
  // before S(j+1) is produced, so the two are never live together.
  auto frag = [&](int i) -> bf16x8 {
    if (i >= NP) {
      const int f = i - NP;
      const int kt = f / 8, stp = f % 8;
      const uint32_t off = ((stp & 1) ? fa.k_odd : fa.k_even) + (stp / 2) * TL::SLAB +
                           kt * 32 * SLAB_ROW;
      return *(const bf16x8*)(lds_k + off);
    }
    const int dt = i / (2 * TL::KTW), kt = (i / 2) % TL::KTW, c = i % 2;
    const uint32_t off = dt * TL::SLAB + (32 * kt + 16 * c) * SLAB_ROW;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(lds_v + fa.v_lo + off));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(lds_v + fa.v_hi + off));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };
  bf16x8 fr[NF];
#pragma unroll
  for (int i = 0; i < AHEAD; ++i) fr[i] = frag(i);
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (RSUM == RSUM_MFMA) {
#pragma unroll
    for (int kt2 = 0; kt2 < TL::KTW; ++kt2)
#pragma unroll
      for (int c2 = 0; c2 < 2; ++c2) {
        st.l = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pr.p[kt2][c2], st.l, 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
  }
#pragma unroll
  for (int i = 0; i < NF; ++i) {
    if (i + AHEAD < NF) fr[i + AHEAD] = frag(i + AHEAD);
    if (sl && i % (NF / NLOADS) == 0) issue_step_load<BLOCK>(*sl, i / (NF / NLOADS));
    if (i < NP) {
      const int dt = i / (2 * TL::KTW), kt = (i / 2) % TL::KTW, c = i % 2;
      st.o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[i], pr.p[kt][c], st.o[dt], 0, 0, 0);
    } else {
      const int f = i - NP;
      const int kt = f / 8, stp = f % 8;
      sc.s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[i], qf[stp],
                                                         stp == 0 ? f32x16{} : sc.s[kt], 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// LDS of the merged walk: the step words of the tile's pair of query blocks
// (kept for the whole tile) and per-wave counts of the merge.  The merge's
// inputs, the two CSR rows, are staged in the K/V tile buffers, which are
// idle at the start of a tile.  A pair's union has at most nb words, so
// nb <= WALK_CAP (checked before launch) lets one merge cover the tile.
constexpr int WALK_CAP = 8000;
struct WalkLds {
  uint32_t w[WALK_CAP];       // step words, in walk order
  int32_t cnt[2][16][5];      // per-wave counts of a merge pass (double-buffered)
};
static_assert(2 * WALK_CAP * 4 <= 4 * Tile<64>::BYTES, "rows staged in the tile buffers");

// Step words.  Block form (row entries are key blocks): kb in bits 0..29,
// bit 30 / 31 set when row 0 / row 1 keeps kb.  Token-exact form (row
// entries are entry words): bits 0..23 kb and kfirst, bits 24..27 / 28..31
// the patterns of row 0 / row 1, 0 where that row does not keep kb.  A key
// block outside [0, nb) gives a word that masks every key (and whose loads
// read zeros).
template <bool EXACT>
__device__ __forceinline__ int32_t entry_key(uint32_t e) {
  return EXACT ? (int32_t)(e & 0xFFFFu) : (int32_t)e;
}
template <bool EXACT>
__device__ __forceinline__ uint32_t step_word(uint32_t e0, uint32_t e1, bool in0, bool in1,
                                              int32_t nb) {
  const int32_t kb = entry_key<EXACT>(in0 ? e0 : e1);
  if (kb < 0 || kb >= nb) return EXACT ? 0xFFFFu : 0x3FFFFFFFu;
  if constexpr (EXACT)
    return ((in0 ? e0 : e1) & 0xFFFFFFu) | (in0 ? e0 & 0x0F000000u : 0u) |
           (in1 ? (e1 & 0x0F000000u) << 4 : 0u);
  return (uint32_t)kb | (in0 ? 1u << 30 : 0u) | (in1 ? 1u << 31 : 0u);
}

// Merges CSR rows 2p ("row 0": entries lo0 .. hi0-1) and 2p+1 ("row 1":
// lo1 .. hi1-1) into L.w, largest key first (every thread of the workgroup
// takes part; starts and ends with a barrier).  Both rows are staged in
// `stage` from their ends down; an entry's position in the union is its
// index in its own row, plus the entries of the other row with a larger key
// (a binary search), minus the keys above it that both rows hold (a count of
// its row's duplicates before it).  Returns the number of words.  Rows of up
// to WALK_CAP entries are merged whole (more are cut); rows that are not
// strictly ascending give some order of their entries, never a write outside
// L.w.
template <int NT, bool EXACT>
__device__ __forceinline__ int32_t merge_pair(WalkLds& L, uint32_t* stage,
                                              const uint32_t* __restrict__ rows,
                                              int32_t lo0, int32_t hi0, int32_t lo1,
                                              int32_t hi1, int32_t nb) {
  const int tid = threadIdx.x, lane = tid % 64, wave = tid / 64;
  constexpr int NWAVE = NT / 64;
  uint32_t* const sa = stage;              // row 0, largest key first
  uint32_t* const sb = stage + WALK_CAP;   // row 1
  const int na = max(0, min(hi0 - lo0, WALK_CAP));
  const int nc = max(0, min(hi1 - lo1, WALK_CAP));
  __syncthreads();   // the stage buffers are idle
  for (int t = tid; t < na; t += NT) sa[t] = rows[hi0 - 1 - t];
  for (int t = tid; t < nc; t += NT) sb[t] = rows[hi1 - 1 - t];
  __syncthreads();
  int dup_base0 = 0, dup_base1 = 0, words = 0;
  const int passes = (max(na, nc) + NT - 1) / NT;
  for (int ps = 0; ps < passes; ++ps) {
    const int t = ps * NT + tid;
    // Entries of the other row with a larger key: the first index whose key
    // is not larger (the staged rows descend), by binary search.
    int above0 = 0, above1 = 0;
    bool dup0 = false, dup1 = false;
    uint32_t e0 = 0u, e1 = 0u, p0 = 0u;
    if (t < na) {
      e0 = sa[t];
      const int32_t x = entry_key<EXACT>(e0);
      int lo = 0, hi = nc;
      while (lo < hi) {
        const int mid = (lo + hi) / 2;
        if (entry_key<EXACT>(sb[mid]) > x) lo = mid + 1; else hi = mid;
      }
      above0 = lo;
      if (lo < nc) {
        p0 = sb[lo];
        dup0 = entry_key<EXACT>(p0) == x;
      }
    }
    if (t < nc) {
      e1 = sb[t];
      const int32_t y = entry_key<EXACT>(e1);
      int lo = 0, hi = na;
      while (lo < hi) {
        const int mid = (lo + hi) / 2;
        if (entry_key<EXACT>(sa[mid]) > y) lo = mid + 1; else hi = mid;
      }
      above1 = lo;
      dup1 = lo < na && entry_key<EXACT>(sa[lo]) == y;
    }
    // Keys held by both rows above each entry: its row's duplicates before it.
    const uint64_t m0 = __ballot(dup0), m1 = __ballot(dup1);
    const uint64_t below = (1ull << lane) - 1ull;
    if (lane == 0) {
      L.cnt[ps & 1][wave][0] = __popcll(m0);
      L.cnt[ps & 1][wave][1] = __popcll(m1);
    }
    __syncthreads();
    int before0 = dup_base0 + __popcll(m0 & below), before1 = dup_base1 + __popcll(m1 & below);
    for (int w = 0; w < NWAVE; ++w) {
      const int v0 = L.cnt[ps & 1][w][0], v1 = L.cnt[ps & 1][w][1];
      before0 += w < wave ? v0 : 0;
      before1 += w < wave ? v1 : 0;
      dup_base0 += v0;
      dup_base1 += v1;
    }
    if (t < na) {
      const int r = t + above0 - before0;
      if (r >= 0 && r < WALK_CAP) L.w[r] = step_word<EXACT>(e0, p0, true, dup0, nb);
    }
    if (t < nc && !dup1) {
      const int r = t + above1 - before1;
      if (r >= 0 && r < WALK_CAP) L.w[r] = step_word<EXACT>(0u, e1, false, true, nb);
    }
    words = na + nc - dup_base1;
  }
  __syncthreads();   // the words are written; the stage buffers are free again
  return __builtin_amdgcn_readfirstlane(min(words, WALK_CAP));
}

// MODE: ATTN_DENSE (every key block), ATTN_BLOCK (CSR rows of key blocks),
// ATTN_EXACT (CSR rows of token-exact entry words).
// One tile: head `tile / npairs`, pair of query blocks from `tile % npairs`,
// using the workgroup's LDS stages `lds` (K slots 0-1, V slots 0-1).
template <int BLOCK, int MODE>
__device__ __forceinline__ void attn_tile(
    char* lds, WalkLds& walk, int tile, const __bf16* __restrict__ qg, const __bf16* __restrict__ kg,
    const __bf16* __restrict__ vg, __bf16* __restrict__ og, int64_t q_sh,
    int64_t q_st, int64_t k_sh, int64_t k_st, int64_t v_sh, int64_t v_st,
    int64_t o_sh, int64_t o_st, int32_t H, int32_t N, int32_t nb,
    const int32_t* __restrict__ row_ptr, const uint32_t* __restrict__ rows,
    int32_t P, float scale_log2) {
  using TL = Tile<BLOCK>;
  constexpr bool SPARSE = MODE != ATTN_DENSE;
  constexpr bool EXACT = MODE == ATTN_EXACT;
  const uint32_t lds_base = (uint32_t)(uintptr_t)(lds_void*)lds;

  const int tid = threadIdx.x;
  const int wave = tid / 64;
  const int lane = tid % 64;
  const int hl = lane / 32;
  const int li = lane % 32;

  const int npairs = (nb + 1) / 2;
  const int head = tile / npairs;
  // Pairs of a head go last to first: rows that attend every key block (text
  // tokens, placed after the video tokens) are the longest tiles, and taking
  // them first keeps them out of the grid's tail (each row's key blocks are
  // then walked in descending order, which keeps neighbouring workgroups'
  // shared blocks in L2).
  const int pq = npairs - 1 - tile % npairs;    // query blocks 2pq, 2pq+1
  const bool upper = wave >= TL::NW / 2;        // rows of query block 2pq+1
  const int qb = 2 * pq + (upper ? 1 : 0);
  const int rows0 = 32 * (wave % (TL::NW / 2));   // first row within qb

  const __bf16* qh = qg + head * q_sh;
  __bf16* oh = og + head * o_sh;
  const __bf16* const kh_base = kg + head * k_sh;
  const __bf16* const vh_base = vg + head * v_sh;
  const uint32_t k_bytes = (uint32_t)(((int64_t)(N - 1) * k_st + D) * 2);
  const uint32_t v_bytes = (uint32_t)(((int64_t)(N - 1) * v_st + D) * 2);
  const LoadPlan<BLOCK> kp = load_plan<BLOCK>((uint32_t)(k_st * 2), wave, lane);
  const LoadPlan<BLOCK> vp = load_plan<BLOCK>((uint32_t)(v_st * 2), wave, lane);
  // Step words: key block in bits 0..29 (block form) or 0..15 (exact form).
  auto kb_of = [&](uint32_t w) {
    return (int)(EXACT ? (w & 0xFFFFu) : (w & 0x3FFFFFFFu));
  };
  auto rk_at = [&](uint32_t w) {
    return tile_rsrc<BLOCK>(kh_base, k_st, k_bytes, kb_of(w), nb);
  };
  auto rv_at = [&](uint32_t w) {
    return tile_rsrc<BLOCK>(vh_base, v_st, v_bytes, kb_of(w), nb);
  };
  const FragAddr fa = frag_addr(lane);

  // Q fragments: row qrow, k-slots d = 16*stp + 8*hl + 0..7.
  const int qrow = qb * BLOCK + rows0 + li;
  bf16x8 qf[8];
#pragma unroll
  for (int stp = 0; stp < 8; ++stp)
    qf[stp] = qrow < N ? *(const bf16x8*)(qh + (int64_t)qrow * q_st + 16 * stp + 8 * hl)
                       : bf16x8{};

  // Exact mode: the first of the wave's 32 rows that lies in the query
  // block's second frame (the first frame holds the block's first qfirst
  // rows; P >= BLOCK, so there are at most two); wave-uniform.
  int sec_from = 32;
  if constexpr (EXACT) {
    const int qfirst = P - (int)(((int64_t)qb * BLOCK) % P);
    sec_from = __builtin_amdgcn_readfirstlane(qfirst - rows0);
  }
  // Masks the scores of the key block of step word w for this wave's query
  // block: a key block that block does not keep has no valid keys.
  const uint32_t kept_bit = upper ? 31u : 30u;       // block form
  const uint32_t pat_shift = upper ? 28u : 24u;      // exact form
  auto mask_block = [&](Scores<BLOCK>& sc, uint32_t w) {
    const int kb = kb_of(w);
    if constexpr (EXACT)
      mask_exact<BLOCK>(sc, (w >> pat_shift) & 0xFu, (int)((w >> 16) & 0xFFu),
                        N - kb * BLOCK, sec_from);
    else
      mask_tail<BLOCK>(sc, lane, ((w >> kept_bit) & 1u) ? N - kb * BLOCK : 0);
  };

  // The walk (sparse modes) or the key blocks nb-1 .. 0 (dense): n steps.
  // Words of steps past the last one repeat it: their loads land in slots
  // that no later step reads.
  int n = nb;
  uint32_t w0 = 0u, w1 = 0u, w2 = 0u;
  // Dense: the words nb-1 .. 0 (both query blocks keep every key block),
  // written to LDS and read from there like the merged walk's (timed faster
  // than computing them in the loop: 1.7% at the Wan-1.3B 6x shape and 2.9%
  // at 40 heads, interleaved on one board); steps past WALK_CAP compute
  // theirs.  The block mode runs dense attention this way when it is given
  // no CSR (row_ptr null, nb <= WALK_CAP): the same code as a full mask's
  // walk, without the merge.
  auto dense_words = [&]() {
    __syncthreads();
    for (int t = threadIdx.x; t < min(nb, WALK_CAP); t += TL::NT)
      walk.w[t] = (uint32_t)(nb - 1 - t) | 0xC0000000u;
    __syncthreads();
    w0 = (uint32_t)(nb - 1) | 0xC0000000u;
    w1 = (uint32_t)max(nb - 2, 0) | 0xC0000000u;
    w2 = (uint32_t)max(nb - 3, 0) | 0xC0000000u;
  };
  if constexpr (SPARSE) {
    if (EXACT || row_ptr != nullptr) {
      const int32_t r0 = __builtin_amdgcn_readfirstlane(row_ptr[2 * pq]);
      const int32_t r1 = __builtin_amdgcn_readfirstlane(row_ptr[2 * pq + 1]);
      const int32_t r2 =
          2 * pq + 1 < nb ? __builtin_amdgcn_readfirstlane(row_ptr[2 * pq + 2]) : r1;
      n = merge_pair<TL::NT, EXACT>(walk, (uint32_t*)lds, rows, r0, r1, r1, r2, nb);
      if (n > 0) {
        w0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)walk.w[0]);
        w1 = (uint32_t)__builtin_amdgcn_readfirstlane((int)walk.w[min(1, n - 1)]);
        w2 = (uint32_t)__builtin_amdgcn_readfirstlane((int)walk.w[min(2, n - 1)]);
      }
    } else {
      dense_words();
    }
  } else {
    dense_words();
  }

  WaveState ws;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) ws.o[dt] = f32x16{};
  ws.m = -__builtin_inff();
  ws.l = f32x4{};
  ws.l0 = 0.f;
  ws.l1 = 0.f;
  constexpr int RSUM = MODE == ATTN_BLOCK ? RSUM_VALU : RSUM_MFMA;
  // A operand of the row-sum MFMA (16x16x32): read as P^T's B operand, lane
  // group g = lane/16 of the 32x32 P register holds q rows 16*(g%2) + 0..15,
  // so A row 0 takes groups 0 and 2 (rows 0-15) and row 1 groups 1 and 3.
  bf16x8 ones;
  {
    const int ai = lane % 16, ag = lane / 16;
    const bool one = (ai == 0 && ag % 2 == 0) || (ai == 1 && ag % 2 == 1);
#pragma unroll
    for (int e = 0; e < 8; ++e) ones[e] = one ? (__bf16)1.f : (__bf16)0.f;
  }

  if (n > 0) {
    // LDS stages: K(b) in K slot b % 2, V(b) in V slot b % 2.
    const uint32_t k_slot0 = lds_base, v_slot0 = lds_base + 2 * TL::BYTES;
    const char* const k_lds = lds;
    const char* const v_lds = lds + 2 * TL::BYTES;

    // Ping-pong schedule.  The waves of query block 2pq ("leaders") run half
    // a step ahead of those of 2pq+1, so on each SIMD one wave is in its GEMM
    // phase (O += P(j) V(j), S(j+1) = K(j+1) Q^T: MFMA) while the other is in
    // its softmax phase (VALU): half-period 2j is the leaders' GEMM j and the
    // others' softmax j, half-period 2j+1 the leaders' softmax j+1 and the
    // others' GEMM j.  A barrier ends every half-period.  K(j+1) and V(j) stay
    // resident through half-periods 2j and 2j+1; K(j+2) and V(j+1) are issued
    // in half-period 2j (into the slots of K(j) and V(j-1), free since
    // half-period 2j-1) and waited for at the end of 2j+1.
    const bool lead = !upper;
    issue_tile<BLOCK>(k_slot0, rk_at(w0), kp);
    issue_tile<BLOCK>(v_slot0, rv_at(w0), vp);
    issue_tile<BLOCK>(k_slot0 + TL::BYTES, rk_at(w1), kp);
    wait_loads_and_sync();
    Scores<BLOCK> sc;
    compute_scores<BLOCK>(k_lds, qf, sc, fa);   // S(0)
    mask_block(sc, w0);
    Probs<BLOCK> pr;
    if (lead) softmax_phase<BLOCK, RSUM>(sc, ws, pr, scale_log2, nullptr);   // P(0)
    __syncthreads();
    for (int j = 0; j < n; ++j) {
      // Word of step j+3 from the walk's LDS, read now and used at the end of
      // the step (the last word again past the end of the walk; a sparse
      // walk never passes WALK_CAP words, nb <= WALK_CAP).
      const int g3 = min(j + 3, n - 1);
      const uint32_t w3v = walk.w[min(g3, WALK_CAP - 1)];
      const StepLoads<BLOCK> sl{
          (uint32_t)__builtin_amdgcn_readfirstlane(k_slot0 + (uint32_t)(j & 1) * TL::BYTES),
          (uint32_t)__builtin_amdgcn_readfirstlane(v_slot0 + (uint32_t)((j + 1) & 1) * TL::BYTES),
          rk_at(w2), rv_at(w1), &kp, &vp};
      const char* const kj1 = k_lds + ((j + 1) & 1) * TL::BYTES;   // K(j+1)
      const char* const vj = v_lds + (j & 1) * TL::BYTES;          // V(j)
      // half-period 2j
      if (lead) {
        gemm_phase<BLOCK, RSUM>(kj1, vj, qf, sc, pr, ws, fa, ones, &sl);
        mask_block(sc, w1);
      } else {
        softmax_phase<BLOCK, RSUM>(sc, ws, pr, scale_log2, &sl);
      }
      __syncthreads();
      // half-period 2j+1
      if (lead) {
        if (j + 1 < n) softmax_phase<BLOCK, RSUM>(sc, ws, pr, scale_log2, nullptr);
      } else {
        gemm_phase<BLOCK, RSUM>(kj1, vj, qf, sc, pr, ws, fa, ones, nullptr);
        mask_block(sc, w1);
      }
      wait_loads_and_sync();
      w1 = w2;
      w2 = SPARSE || g3 < WALK_CAP ? (uint32_t)__builtin_amdgcn_readfirstlane((int)w3v)
                                   : (uint32_t)(nb - 1 - g3) | 0xC0000000u;
    }
    __syncthreads();
  }

  // Every wave holds whole rows: O / l, rounded to bf16.  The l tile holds
  // row c in register 0 of lane c and row c + 16 in register 1 (c < 16).
  float lsum;
  if constexpr (RSUM == RSUM_MFMA) {
    const float r0s = __shfl(ws.l[0], li), r1s = __shfl(ws.l[1], li & 15);
    lsum = li < 16 ? r0s : r1s;
  } else {
    const float lpart = ws.l0 + ws.l1;
    lsum = lpart + __shfl_xor(lpart, 32);
  }
  const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
  if (qrow < N) {
    __bf16* orow = oh + (int64_t)qrow * o_st;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
        bf16x4 w;
#pragma unroll
        for (int b = 0; b < 4; ++b) w[b] = (__bf16)(ws.o[dt][4 * a + b] * inv);
        *(bf16x4*)(orow + 32 * dt + 8 * a + 4 * hl) = w;
      }
  }
}

// First tile and tile count of XCD x's share of `total` tiles: contiguous
// shares, the first total % 8 of them one tile larger.
__device__ __forceinline__ int xcd_first(int x, int total) {
  const int per = total / 8, rem = total % 8;
  return x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per;
}
__device__ __forceinline__ int xcd_count(int x, int total) {
  return total / 8 + (x < total % 8 ? 1 : 0);
}

// Next tile for a workgroup on XCD `xcd`, or -1 when every tile is handed
// out.  Tiles are dealt to the XCDs in contiguous shares; a workgroup takes
// the next tile from the front of its own XCD's share and, once that share
// is handed out, the last one left at the back of another XCD's share, so
// XCDs that clock faster take on more tiles while each share is still
// worked from its front by its own XCD (neighbouring tiles, whose key lists
// overlap, stay together in that XCD's L2).  Counter word x holds in bits
// 0..31 the takes from the front of share x and in bits 32..63 those from
// its back; a take gets a tile iff the two counts before it sum to less
// than the share's size, so each tile goes out once.  Every call makes at
// most 8 atomic adds, so a workgroup's loop ends after at most total + 8
// calls.
__device__ __forceinline__ int fetch_tile(uint64_t* ctr, int xcd, int total) {
  for (int d = 0; d < 8; ++d) {
    const int x = (xcd + d) % 8;
    const uint64_t cnt = (uint64_t)xcd_count(x, total);
    const uint64_t seen =
        __hip_atomic_load(&ctr[x], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if ((seen & 0xFFFFFFFFull) + (seen >> 32) >= cnt) continue;
    const uint64_t old = __hip_atomic_fetch_add(&ctr[x], d == 0 ? 1ull : 1ull << 32,
                                                __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint64_t front = old & 0xFFFFFFFFull, back = old >> 32;
    if (front + back < cnt)
      return xcd_first(x, total) + (d == 0 ? (int)front : (int)(cnt - 1 - back));
  }
  return -1;
}

// Kernel arguments, passed as one struct so that the persistent loop can
// read them again for every tile instead of holding them in registers.
struct KArgs {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  __bf16* o;
  int64_t q_sh, q_st, k_sh, k_st, v_sh, v_st, o_sh, o_st;
  const int32_t* row_ptr;
  const uint32_t* rows;
  uint64_t* counters;
  int32_t H, N, nb, P;
  float scale_log2;
};

template <int BLOCK, int MODE>
__device__ __forceinline__ void attn_tile_args(char* lds, WalkLds& walk, int tile,
                                               const KArgs& a) {
  attn_tile<BLOCK, MODE>(lds, walk, tile, a.q, a.k, a.v, a.o, a.q_sh, a.q_st, a.k_sh, a.k_st,
                         a.v_sh, a.v_st, a.o_sh, a.o_st, a.H, a.N, a.nb, a.row_ptr,
                         a.rows, a.P, a.scale_log2);
}

// Persistent workgroups, at most one per CU, take tiles until all are done
// (fetch_tile), through the launch's own counters, zeroed by
// zero_counters_kernel just before on the same stream.
template <int BLOCK, int MODE>
__global__ __launch_bounds__(Tile<BLOCK>::NT) void attn_fwd_kernel(const KArgs args) {
  __shared__ __attribute__((aligned(1024))) char lds[4 * Tile<BLOCK>::BYTES];
  __shared__ WalkLds walk;
  __shared__ int next_tile;
  const int total = (args.nb + 1) / 2 * args.H;
  // Workgroups are dispatched round-robin over the 8 XCDs.
  const int xcd = blockIdx.x % 8;
  for (;;) {
    if (threadIdx.x == 0) next_tile = fetch_tile(args.counters, xcd, total);
    __syncthreads();
    const int tile = __builtin_amdgcn_readfirstlane(next_tile);
    __syncthreads();   // every wave has read next_tile before it is rewritten
    if (tile < 0) break;
    // The arguments are the first kernel argument; an offset the compiler
    // cannot see to be zero makes every tile load them afresh (scalar
    // loads), so they are not live across tiles.
    int zero = 0;
    asm volatile("" : "+v"(zero));
    zero = __builtin_amdgcn_readfirstlane(zero);
    const KArgs* ap = (const KArgs*)((const char*)__builtin_amdgcn_kernarg_segment_ptr() + zero);
    attn_tile_args<BLOCK, MODE>(lds, walk, tile, *ap);
  }
}

__global__ __launch_bounds__(64) void zero_counters_kernel(uint64_t* __restrict__ ctr) {
  if (threadIdx.x < kTileCounters) ctr[threadIdx.x] = 0;
}

// Compute units of the current device (cached per device).
int cu_count() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
      n = 256;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

template <int BLOCK, int MODE>
hipError_t launch_t(const AttnArgs& a, hipStream_t stream) {
  const float scale_log2 = 1.4426950408889634f / __builtin_sqrtf((float)D);
  const int tiles = (a.n_blocks + 1) / 2 * a.heads;
  // One persistent workgroup per CU (each takes 160 KB of LDS at BLOCK =
  // 128, so one fits a CU), or one per tile when there are fewer tiles.
  const int grid = tiles < cu_count() ? tiles : cu_count();
  KArgs k;
  k.q = (const __bf16*)a.q;
  k.k = (const __bf16*)a.k;
  k.v = (const __bf16*)a.v;
  k.o = (__bf16*)a.o;
  k.q_sh = a.q_sh; k.q_st = a.q_st; k.k_sh = a.k_sh; k.k_st = a.k_st;
  k.v_sh = a.v_sh; k.v_st = a.v_st; k.o_sh = a.o_sh; k.o_st = a.o_st;
  k.row_ptr = a.row_ptr;
  k.rows = a.rows;
  k.counters = a.counters;
  k.H = a.heads; k.N = a.n_tokens; k.nb = a.n_blocks; k.P = a.frame_tokens;
  k.scale_log2 = scale_log2;
  hipLaunchKernelGGL(zero_counters_kernel, dim3(1), dim3(64), 0, stream, a.counters);
  hipLaunchKernelGGL((attn_fwd_kernel<BLOCK, MODE>), dim3(grid), dim3(Tile<BLOCK>::NT), 0,
                     stream, k);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, int32_t block, AttnMode mode,
                            hipStream_t stream) {
  // Dense attention over at most WALK_CAP key blocks runs the block mode's
  // kernel without a CSR: the same code as the block-sparse kernel with a
  // full mask, which it matched or beat only that way (the separate dense
  // instantiation timed 0.6% slower than the full-mask launch at the
  // Wan-1.3B 6x shape, interleaved on one board, for no difference in its
  // step loop but the layout of its branches).
  if (mode == ATTN_DENSE && a.n_blocks <= WALK_CAP) {
    AttnArgs d = a;
    d.row_ptr = nullptr;
    d.rows = nullptr;
    return launch_attention(d, block, ATTN_BLOCK, stream);
  }
  if (block == 128) {
    if (mode == ATTN_EXACT) return launch_t<128, ATTN_EXACT>(a, stream);
    if (mode == ATTN_BLOCK) return launch_t<128, ATTN_BLOCK>(a, stream);
    return launch_t<128, ATTN_DENSE>(a, stream);
  }
  if (mode == ATTN_EXACT) return launch_t<64, ATTN_EXACT>(a, stream);
  if (mode == ATTN_BLOCK) return launch_t<64, ATTN_BLOCK>(a, stream);
  return launch_t<64, ATTN_DENSE>(a, stream);
}

}  // namespace lvsa
