// attention.hip -- block-sparse and dense flash-attention forward for gfx950.
//
// Computes Eq. 2 of the LVSA paper (softmax attention restricted to a key
// set) with the key set given per query block by a block CSR, and Eq. 1
// (all keys) with the same kernel visiting every key block.
//
// Work decomposition
//   One workgroup per (head, query block of BLOCK rows); BLOCK/32 waves, each
//   wave owns 32 query rows.  The kept key blocks are visited in CSR order;
//   each is staged through LDS (K row-major with a 16-byte XOR swizzle, V
//   transposed) and consumed with bf16 MFMA 32x32x16:
//     S^T = K Q^T     (A = K rows from LDS, B = Q rows held in registers)
//     O^T += V^T P^T  (A = V^T from LDS,   B = P straight from S^T's registers)
//   Computing the transposed products puts one query per lane (lane l and
//   l^32 share query l%32), so the softmax row max / row sum are in-lane
//   reductions plus one exchange with the partner lane, and P feeds the second
//   MFMA without leaving registers.
//
// MFMA 32x32 operand layout (lane l, half h = l/32, i = l%32):
//   A: row i, 8 consecutive k-slots of half h;  B: column i, same k-slots;
//   C: column i, rows 8*(r/4) + 4*h + (r%4) for register r = 0..15.
// The k-slot order only has to agree between A and B, so for P.V the key
// owned by C register r of S^T is paired with the V^T element of that key.
//
// Online softmax (fp32, base-2): m = running max of s*scale*log2(e),
// p = exp2(s*scale*log2(e) - m), l = sum p; O and l are rescaled by
// exp2(m_old - m_new) when the max grows.  Keys at or beyond N in the last
// (ragged) block get s = -inf, and their K/V rows are loaded as zeros.
#include "internal.h"

namespace lvsa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int D = 128;           // head_dim
constexpr int CHUNKS = D / 8;    // 16-byte chunks per row
constexpr int VPAD = 4;          // V^T row padding (elements): bank spread

__device__ inline int xcd_remap(int bid, int total) {
  // Workgroups are dispatched round-robin over the 8 XCDs; give each XCD a
  // contiguous range of logical tiles so that tiles sharing key blocks share
  // that XCD's L2.
  const int per = total / 8, rem = total % 8;
  const int xcd = bid % 8, idx = bid / 8;
  return (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) +
         idx;
}

__device__ inline uint32_t pack2(__bf16 a, __bf16 b) {
  return (uint32_t)__builtin_bit_cast(uint16_t, a) |
         ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

template <int BLOCK, bool SPARSE>
__global__ __launch_bounds__(BLOCK * 2) void attn_fwd_kernel(
    const __bf16* __restrict__ qg, const __bf16* __restrict__ kg,
    const __bf16* __restrict__ vg, __bf16* __restrict__ og, int64_t q_sh,
    int64_t q_st, int64_t k_sh, int64_t k_st, int64_t v_sh, int64_t v_st,
    int64_t o_sh, int64_t o_st, int32_t H, int32_t N, int32_t nb,
    const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ col_idx,
    float scale_log2) {
  constexpr int NW = BLOCK / 32;       // waves
  constexpr int NT = NW * 64;          // threads
  constexpr int KT = BLOCK / 32;       // 32-key tiles per key block
  constexpr int VROW = BLOCK + VPAD;   // V^T row length (elements)
  constexpr int KLOADS = BLOCK * CHUNKS / NT;       // 16B K chunks per thread
  constexpr int VGROUPS = BLOCK * CHUNKS / (4 * NT);  // 4-key V groups/thread
  static_assert(KLOADS == 8 && VGROUPS == 2, "tile mapping");

  __shared__ __attribute__((aligned(16))) __bf16 s_k[BLOCK * D];
  __shared__ __attribute__((aligned(16))) __bf16 s_vt[D * VROW];

  const int tid = threadIdx.x;
  const int wave = tid / 64;
  const int lane = tid % 64;
  const int hl = lane / 32;  // half of the wave
  const int li = lane % 32;

  const int tile = xcd_remap(blockIdx.x, nb * H);
  const int head = tile / nb;
  const int qb = tile % nb;

  const __bf16* qh = qg + head * q_sh;
  const __bf16* kh = kg + head * k_sh;
  const __bf16* vh = vg + head * v_sh;
  __bf16* oh = og + head * o_sh;

  // Q fragments (B operand of S^T = K Q^T): query row qrow, k-slots are
  // d = 16*step + 8*hl + 0..7.
  const int qrow = qb * BLOCK + wave * 32 + li;
  bf16x8 qf[8];
#pragma unroll
  for (int st = 0; st < 8; ++st) {
    if (qrow < N)
      qf[st] = *(const bf16x8*)(qh + (int64_t)qrow * q_st + 16 * st + 8 * hl);
    else
      qf[st] = bf16x8{};
  }

  int it = 0, it_end = nb;
  if constexpr (SPARSE) {
    it = row_ptr[qb];
    it_end = row_ptr[qb + 1];
  }

  // Global -> register staging of one key block.
  //   K: thread covers chunk tid%16 of keys tid/16 + (NT/16)*j.
  //   V: thread covers chunk tid%16 of 4 consecutive keys 4*(tid/16 + (NT/16)*g) + r.
  const int cchunk = tid % 16;
  const int crow = tid / 16;
  bf16x8 kreg[KLOADS];
  bf16x8 vreg[VGROUPS][4];
  auto load_block = [&](int kb) {
    const int base = kb * BLOCK;
#pragma unroll
    for (int j = 0; j < KLOADS; ++j) {
      const int key = base + crow + (NT / 16) * j;
      kreg[j] = (unsigned)key < (unsigned)N ? *(const bf16x8*)(kh + (int64_t)key * k_st + 8 * cchunk)
                        : bf16x8{};
    }
#pragma unroll
    for (int g = 0; g < VGROUPS; ++g)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = base + 4 * (crow + (NT / 16) * g) + r;
        vreg[g][r] = (unsigned)key < (unsigned)N
                         ? *(const bf16x8*)(vh + (int64_t)key * v_st + 8 * cchunk)
                         : bf16x8{};
      }
  };
  auto store_block = [&]() {
#pragma unroll
    for (int j = 0; j < KLOADS; ++j) {
      const int key = crow + (NT / 16) * j;
      *(bf16x8*)(s_k + key * D + 8 * (cchunk ^ (key & 15))) = kreg[j];
    }
#pragma unroll
    for (int g = 0; g < VGROUPS; ++g) {
      const int key0 = 4 * (crow + (NT / 16) * g);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        u32x2 w;
        w[0] = pack2(vreg[g][0][e], vreg[g][1][e]);
        w[1] = pack2(vreg[g][2][e], vreg[g][3][e]);
        *(u32x2*)(s_vt + (8 * cchunk + e) * VROW + key0) = w;
      }
    }
  };

  f32x16 o_acc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) o_acc[dt] = f32x16{};
  float m_run = -__builtin_inff();
  float l_run = 0.f;

  if (it < it_end) load_block(SPARSE ? col_idx[it] : it);

  for (; it < it_end; ++it) {
    const int kb = SPARSE ? col_idx[it] : it;
    __syncthreads();
    store_block();
    __syncthreads();
    if (it + 1 < it_end) load_block(SPARSE ? col_idx[it + 1] : it + 1);

    // S^T tiles: keys 32*kt + (row of C), query li.
    f32x16 s[KT];
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      f32x16 acc = f32x16{};
      const int key = 32 * kt + li;
#pragma unroll
      for (int st = 0; st < 8; ++st) {
        const int ch = 2 * st + hl;
        const bf16x8 a = *(const bf16x8*)(s_k + key * D + 8 * (ch ^ (key & 15)));
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[st], acc, 0, 0, 0);
      }
      s[kt] = acc;
    }

    // Ragged last block: keys >= N do not exist.
    const int valid = N - kb * BLOCK;
    if (valid < BLOCK) {
#pragma unroll
      for (int kt = 0; kt < KT; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = 32 * kt + 8 * (r / 4) + 4 * hl + (r % 4);
          if (key >= valid) s[kt][r] = -__builtin_inff();
        }
    }

    float mx = -__builtin_inff();
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kt][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx * scale_log2);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;

    float psum = 0.f;
    bf16x8 pf[KT][2];
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float p =
              __builtin_amdgcn_exp2f(__builtin_fmaf(s[kt][8 * c + e], scale_log2, -m_new));
          psum += p;
          pf[kt][c][e] = (__bf16)p;
        }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) o_acc[dt] *= alpha;

    // O^T += V^T P^T.  k-step (kt, c) covers keys 32kt + 16c + {4hl+0..3,
    // 8+4hl+0..3}, the keys of C registers 8c..8c+7 of S^T tile kt.
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const __bf16* vrow = s_vt + (32 * dt + li) * VROW;
#pragma unroll
      for (int kt = 0; kt < KT; ++kt)
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const int k0 = 32 * kt + 16 * c + 4 * hl;
          const u32x2 lo = *(const u32x2*)(vrow + k0);
          const u32x2 hi = *(const u32x2*)(vrow + k0 + 8);
          const u32x4 w = {lo[0], lo[1], hi[0], hi[1]};
          const bf16x8 a = __builtin_bit_cast(bf16x8, w);
          o_acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[kt][c], o_acc[dt], 0, 0, 0);
        }
    }
  }

  // Finalize: each query's sum is split over lanes l and l^32.
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (qrow < N) {
    __bf16* orow = oh + (int64_t)qrow * o_st;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        u32x2 w;
        w[0] = pack2((__bf16)(o_acc[dt][4 * a + 0] * inv), (__bf16)(o_acc[dt][4 * a + 1] * inv));
        w[1] = pack2((__bf16)(o_acc[dt][4 * a + 2] * inv), (__bf16)(o_acc[dt][4 * a + 3] * inv));
        *(u32x2*)(orow + 32 * dt + 8 * a + 4 * hl) = w;
      }
  }
}

template <int BLOCK, bool SPARSE>
hipError_t launch_t(const AttnArgs& a, hipStream_t stream) {
  const float scale_log2 = 1.4426950408889634f / __builtin_sqrtf((float)D);
  const int grid = a.n_blocks * a.heads;
  hipLaunchKernelGGL((attn_fwd_kernel<BLOCK, SPARSE>), dim3(grid),
                     dim3(BLOCK * 2), 0, stream, (const __bf16*)a.q,
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
