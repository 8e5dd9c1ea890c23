// attention.hip -- block-sparse and dense flash-attention forward for gfx950.
//
// Computes Eq. 2 of the LVSA paper (softmax attention restricted to a key
// set) with the key set of every query block given by a block CSR, and Eq. 1
// (all keys) with the same kernel visiting every key block.
//
// Work decomposition
//   One workgroup per (head, query block of BLOCK rows), 2*BLOCK/32 waves
//   (two per SIMD at BLOCK = 128).  Wave w owns query rows 32*(w % R) ..+31
//   (R = BLOCK/32 row groups) and key half w / R of every key block: the two
//   waves of a row group run independent online softmaxes over disjoint keys
//   and are merged once at the end.  Two waves per SIMD let one wave's MFMAs
//   overlap the other's softmax arithmetic.
//
// Data movement
//   Key blocks are visited in CSR order.  K and V tiles (BLOCK x 128 bf16,
//   row-major) go HBM/L2 -> LDS by buffer loads that write LDS directly (no
//   register staging), double-buffered: the next key block is in flight while
//   the current one is consumed.  The buffer resource's size bound turns rows
//   at or past N (the ragged last block) into zeros.  16-byte chunks of each
//   LDS row are XOR-swizzled so both the K reads (ds_read_b128) and the V
//   reads (ds_read_b64_tr_b16) are free of bank conflicts.
//
// Contractions (bf16 MFMA 32x32x16, fp32 accumulate)
//     S^T = K Q^T     A = K rows (LDS), B = Q rows (registers, loaded once)
//     O^T += V^T P^T  A = V^T via the transposing LDS read, B = P from S^T's
//                     registers
//   The transposed products put one query row per lane (lanes l and l^32
//   share row l%32), so softmax row statistics are in-lane reductions plus
//   one permlane32 exchange, and P never leaves registers.
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
#include "internal.h"

namespace lvsa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int D = 128;             // head_dim
constexpr int ROW_BYTES = D * 2;   // one K/V row in LDS
constexpr float RESCALE_SLACK = 8.f;


typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

__device__ inline int xcd_remap(int bid, int total) {
  // Workgroups are dispatched round-robin over the 8 XCDs; give each XCD a
  // contiguous range of logical tiles so that neighbouring query blocks of a
  // head, whose key lists overlap, share that XCD's L2.
  const int per = total / 8, rem = total % 8;
  const int xcd = bid % 8, idx = bid / 8;
  return (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) +
         idx;
}

// Swizzle of the 16-byte chunk index within a 256-byte LDS row.  LDS has 64
// banks of 4 bytes.  ds_read_b128 is served 16 lanes at a time: here 16
// consecutive rows at one logical chunk, which the swizzle spreads over all
// 16 chunk positions.  ds_read_b64_tr_b16 is served 32 lanes at a time: here
// 4 consecutive rows x 4 adjacent logical chunks, which the swizzle places in
// 4 disjoint groups of 4 chunk positions (bits 2-3 of the XOR follow row%4).
__device__ inline int swz(int row) { return ((row & 3) << 2) | ((row >> 2) & 3); }

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base,
                                                   uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0,
                                           bytes, 0x00020000);
}

__device__ inline float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x),
                                            __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x),
                                            __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int BLOCK>
struct Tile {
  static constexpr int R = BLOCK / 32;          // row groups
  static constexpr int NW = 2 * R;              // waves
  static constexpr int NT = NW * 64;            // threads
  static constexpr int KH = BLOCK / 2;          // keys per wave per block
  static constexpr int KTW = KH / 32;           // 32-key tiles per wave
  static constexpr int CHUNKS = BLOCK * 16;     // 16-byte chunks per tile
  static constexpr int LOADS = CHUNKS / NT;     // per thread per tile
  static constexpr int TILE_BYTES = BLOCK * ROW_BYTES;
  static_assert(LOADS * NT == CHUNKS, "tile load mapping");
};

// One LDS stage: K tile then V tile.
template <int BLOCK>
struct Stage {
  __bf16 k[BLOCK * D];
  __bf16 v[BLOCK * D];
};

// Issues the direct-to-LDS loads of K and V rows kb*BLOCK .. +BLOCK-1.
// Load j of wave w fills LDS chunks 64*(w + NW*j) + lane: row (that index)/16,
// physical chunk lane%16, which holds logical chunk (lane%16) ^ swz(row).
template <int BLOCK>
__device__ inline void issue_tile(__bf16* lds_k, __bf16* lds_v,
                                  __amdgpu_buffer_rsrc_t rk,
                                  __amdgpu_buffer_rsrc_t rv, int64_t k_row_bytes,
                                  int64_t v_row_bytes, int kb, int wave,
                                  int lane) {
  using TL = Tile<BLOCK>;
#pragma unroll
  for (int j = 0; j < TL::LOADS; ++j) {
    const int slot0 = 64 * (wave + TL::NW * j);
    const int row = (slot0 + lane) / 16;
    const int chunk = (lane % 16) ^ swz(row);
    const int grow = kb * BLOCK + row;
    const uint32_t koff = (uint32_t)(grow * k_row_bytes + chunk * 16);
    const uint32_t voff = (uint32_t)(grow * v_row_bytes + chunk * 16);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void*)(lds_k + slot0 * 8),
                                             16, koff, 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void*)(lds_v + slot0 * 8),
                                             16, voff, 0, 0, 0);

  }
}

template <int BLOCK>
struct WaveState {
  using TL = Tile<BLOCK>;
  f32x16 o[4];       // O^T tiles: d = 32*dt + C row, query = lane%32
  float m;           // running max (log2 domain), shared by lanes l, l^32
  float l;           // partial row sum of this lane's keys
};

// Consumes one key block from LDS (K at lds_k, V at lds_v).
template <int BLOCK>
__device__ inline void consume(const __bf16* lds_k, const __bf16* lds_v,
                               const bf16x8 (&qf)[8], WaveState<BLOCK>& st,
                               int kh, int lane, int valid, float scale_log2) {
  using TL = Tile<BLOCK>;
  const int hl = lane / 32;
  const int li = lane % 32;
  const char* kbase = (const char*)lds_k;
  const char* vbase = (const char*)lds_v;

  // S^T = K Q^T for this wave's KH keys.
  f32x16 s[TL::KTW];
#pragma unroll
  for (int kt = 0; kt < TL::KTW; ++kt) {
    const int row = TL::KH * kh + 32 * kt + li;
    const char* rp = kbase + row * ROW_BYTES;
    const int sw = swz(row);
    f32x16 acc = f32x16{};
#pragma unroll
    for (int stp = 0; stp < 8; ++stp) {
      const bf16x8 a = *(const bf16x8*)(rp + (((2 * stp + hl) ^ sw) * 16));
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[stp], acc, 0, 0, 0);
    }
    s[kt] = acc;
  }

  // Keys at or past N (ragged last block) do not exist.
  if (valid < BLOCK) {
#pragma unroll
    for (int kt = 0; kt < TL::KTW; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = TL::KH * kh + 32 * kt + 8 * (r / 4) + 4 * hl + (r % 4);
        if (key >= valid) s[kt][r] = -__builtin_inff();
      }
  }

  float mx = s[0][0];
#pragma unroll
  for (int kt = 0; kt < TL::KTW; ++kt)
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kt][r]);
  mx = pair_max(mx) * scale_log2;
  const bool raise = mx > st.m + RESCALE_SLACK;
  if (__builtin_amdgcn_ballot_w64(raise)) {
    const float alpha = raise ? __builtin_amdgcn_exp2f(st.m - mx) : 1.f;
    st.m = raise ? mx : st.m;
    st.l *= alpha;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) st.o[dt] *= alpha;
  }
  const float m_sub = st.m == -__builtin_inff() ? 0.f : st.m;

  // P = exp2(s*scale - m), packed to bf16 in MFMA B-operand order.
  bf16x8 pf[TL::KTW][2];
  float psum = 0.f;
#pragma unroll
  for (int kt = 0; kt < TL::KTW; ++kt)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float p = __builtin_amdgcn_exp2f(
            __builtin_fmaf(s[kt][8 * c + e], scale_log2, -m_sub));
        psum += p;
        pf[kt][c][e] = (__bf16)p;
      }
  st.l += psum;

  // O^T += V^T P^T.  k-step (kt, c) holds keys 32kt + 16c + {4h..4h+3,
  // 8+4h..8+4h+3} (C registers 8c..8c+7 of S^T tile kt).  The transposing
  // read gives lane (group g = lane/16, j = lane%16) element e of the 16-lane
  // group's chunk 4e + j/4, entry j%4, so source lane sl = 4e + q points at
  // V row (key e of its half) and the 4 columns 4q..4q+3 of its 16-column
  // group.
  const int g = lane / 16;
  const int sl = lane % 16;
  const int vrow0 = TL::KH * kh + 4 * (g / 2) + sl / 4;
  const int cb = 2 * (g % 2) + (sl % 4) / 2;
  const int half = (sl % 2) * 8;
  const int f0 = swz(vrow0);
  const int f1 = swz(vrow0 + 8);
#pragma unroll
  for (int kt = 0; kt < TL::KTW; ++kt)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int row = vrow0 + 32 * kt + 16 * c;
      const char* r0 = vbase + row * ROW_BYTES + half;
      const char* r1 = r0 + 8 * ROW_BYTES;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
        const int pc0 = (4 * dt + cb) ^ f0;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_i16x4*)(r0 + pc0 * 16));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_i16x4*)(r1 + ((4 * dt + cb) ^ f1) * 16));
        const bf16x8 a = __builtin_bit_cast(
            bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        st.o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[kt][c],
                                                           st.o[dt], 0, 0, 0);
      }
    }
}

template <int BLOCK, bool SPARSE>
__global__ __launch_bounds__(Tile<BLOCK>::NT) void attn_fwd_kernel(
    const __bf16* __restrict__ qg, const __bf16* __restrict__ kg,
    const __bf16* __restrict__ vg, __bf16* __restrict__ og, int64_t q_sh,
    int64_t q_st, int64_t k_sh, int64_t k_st, int64_t v_sh, int64_t v_st,
    int64_t o_sh, int64_t o_st, int32_t H, int32_t N, int32_t nb,
    const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ col_idx,
    float scale_log2) {
  using TL = Tile<BLOCK>;
  __shared__ __attribute__((aligned(1024))) Stage<BLOCK> st0;
  __shared__ __attribute__((aligned(1024))) Stage<BLOCK> st1;

  const int tid = threadIdx.x;
  const int wave = tid / 64;
  const int lane = tid % 64;
  const int hl = lane / 32;
  const int li = lane % 32;
  const int rg = wave % TL::R;   // row group
  const int kh = wave / TL::R;   // key half

  const int tile = xcd_remap(blockIdx.x, nb * H);
  const int head = tile / nb;
  const int qb = tile % nb;

  const __bf16* qh = qg + head * q_sh;
  __bf16* oh = og + head * o_sh;
  const __amdgpu_buffer_rsrc_t rk =
      make_rsrc(kg + head * k_sh, (uint32_t)(((int64_t)(N - 1) * k_st + D) * 2));
  const __amdgpu_buffer_rsrc_t rv =
      make_rsrc(vg + head * v_sh, (uint32_t)(((int64_t)(N - 1) * v_st + D) * 2));
  const int64_t k_row_bytes = k_st * 2;
  const int64_t v_row_bytes = v_st * 2;

  // Q fragments: row qrow, k-slots d = 16*stp + 8*hl + 0..7.
  const int qrow = qb * BLOCK + rg * 32 + li;
  bf16x8 qf[8];
#pragma unroll
  for (int stp = 0; stp < 8; ++stp)
    qf[stp] = qrow < N ? *(const bf16x8*)(qh + (int64_t)qrow * q_st + 16 * stp + 8 * hl)
                       : bf16x8{};

  int it = 0, it_end = nb;
  if constexpr (SPARSE) {
    it = row_ptr[qb];
    it_end = row_ptr[qb + 1];
  }

  WaveState<BLOCK> ws;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) ws.o[dt] = f32x16{};
  ws.m = -__builtin_inff();
  ws.l = 0.f;

  auto kb_at = [&](int i) { return SPARSE ? col_idx[i] : i; };
  if (it < it_end)
    issue_tile<BLOCK>(st0.k, st0.v, rk, rv, k_row_bytes, v_row_bytes, kb_at(it),
                      wave, lane);

  // Two key blocks per trip so that each LDS stage is a distinct object: the
  // loads into one stage are then known not to alias reads of the other.
  while (it < it_end) {
    {
      const int kb = kb_at(it);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (it + 1 < it_end)
        issue_tile<BLOCK>(st1.k, st1.v, rk, rv, k_row_bytes, v_row_bytes,
                          kb_at(it + 1), wave, lane);
      consume<BLOCK>(st0.k, st0.v, qf, ws, kh, lane, N - kb * BLOCK, scale_log2);
      ++it;
    }
    if (it >= it_end) break;
    {
      const int kb = kb_at(it);
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (it + 1 < it_end)
        issue_tile<BLOCK>(st0.k, st0.v, rk, rv, k_row_bytes, v_row_bytes,
                          kb_at(it + 1), wave, lane);
      consume<BLOCK>(st1.k, st1.v, qf, ws, kh, lane, N - kb * BLOCK, scale_log2);
      ++it;
    }
  }

  // Merge the two key halves of each row group: the second-half wave leaves
  // its state in LDS (O as [register][lane] floats, conflict-free), the
  // first-half wave combines and stores.
  __syncthreads();
  float* mo = (float*)&st0;                 // [R][64 regs][64 lanes]
  float* mm = (float*)&st1;                 // [R][64 lanes] max
  float* ml = mm + TL::R * 64;              // [R][64 lanes] pair sums
  const float lsum = pair_sum(ws.l);
  if (kh == 1) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mo[(rg * 64 + dt * 16 + r) * 64 + lane] = ws.o[dt][r];
    mm[rg * 64 + lane] = ws.m;
    ml[rg * 64 + lane] = lsum;
  }
  __syncthreads();
  if (kh == 0) {
    const float m1 = mm[rg * 64 + lane];
    const float l1 = ml[rg * 64 + lane];
    const float m = fmaxf(ws.m, m1);
    const float a0 = ws.m == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(ws.m - m);
    const float a1 = m1 == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(m1 - m);
    const float ltot = lsum * a0 + l1 * a1;
    const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
    const float c0 = a0 * inv, c1 = a1 * inv;
    if (qrow < N) {
      __bf16* orow = oh + (int64_t)qrow * o_st;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
          bf16x4 w;
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const int r = 4 * a + b;
            w[b] = (__bf16)(ws.o[dt][r] * c0 + mo[(rg * 64 + dt * 16 + r) * 64 + lane] * c1);
          }
          *(bf16x4*)(orow + 32 * dt + 8 * a + 4 * hl) = w;
        }
    }
  }
}

template <int BLOCK, bool SPARSE>
hipError_t launch_t(const AttnArgs& a, hipStream_t stream) {
  const float scale_log2 = 1.4426950408889634f / __builtin_sqrtf((float)D);
  const int grid = a.n_blocks * a.heads;
  hipLaunchKernelGGL((attn_fwd_kernel<BLOCK, SPARSE>), dim3(grid),
                     dim3(Tile<BLOCK>::NT), 0, stream, (const __bf16*)a.q,
                     (const __bf16*)a.k, (const __bf16*)a.v, (__bf16*)a.o,
                     a.q_sh, a.q_st, a.k_sh, a.k_st, a.v_sh, a.v_st, a.o_sh,
                     a.o_st, a.heads, a.n_tokens, a.n_blocks, a.row_ptr,
                     a.col_idx, scale_log2);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, int32_t block, bool sparse,
                            hipStream_t stream) {
  if (block == 128)
    return sparse ? launch_t<128, true>(a, stream) : launch_t<128, false>(a, stream);
  return sparse ? launch_t<64, true>(a, stream) : launch_t<64, false>(a, stream);
}

}  // namespace lvsa
