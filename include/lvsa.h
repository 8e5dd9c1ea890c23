/*
 * lvsa.h -- C ABI of the LVSA block-sparse video attention library (gfx950).
 *
 * LVSA ("Training-Free Sparse Attention for Long Video Diffusion") restricts
 * the self-attention of a video diffusion transformer, taken over the N = T*P
 * tokens of T latent frames with P spatial tokens each, to a per-query-frame
 * set of attended frames A(t) (Sec. 2, Def. 1 and Eq. 2).  LVSA's A(t) is the
 * union of periodic global anchor frames, rotated with the denoising step
 * (Def. 2, Eq. 3), and a local window of frames around t, shifted and expanded
 * so every frame attends to the same number of frames (Sec. 2 "Overlapping
 * frames", Alg. 1).
 *
 * The library has two halves:
 *   - mask builders that turn (T, P, block, step, params) into per-query-block
 *     lists of kept key blocks (a block CSR), on the host (lvsa_build_mask)
 *     or on the device (lvsa_build_mask_device);
 *   - a block-sparse flash-attention forward pass that visits only the kept
 *     blocks of any block CSR (lvsa_attention), and a dense pass of the same
 *     design over every block (lvsa_dense_attention, Eq. 1) used as the speed
 *     baseline.
 *
 * Conventions for every call:
 *   - Every function returns an lvsa_status (int32_t).  No C++ exception
 *     crosses this boundary.  Arguments are checked before anything is
 *     launched; on an error nothing is launched and no output is written.
 *   - Device pointers are HIP device addresses on the current device.
 *     Streams are hipStream_t passed as void* (NULL = the default stream).
 *   - Calls that launch work are asynchronous on the given stream; launch
 *     failures are reported as LVSA_EDEVICE.
 *   - All sizes are in elements unless stated otherwise.
 */
#ifndef LVSA_H
#define LVSA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------ status ---- */

typedef int32_t lvsa_status;
#define LVSA_OK 0
#define LVSA_EINVAL (-1)        /* an argument is out of range or inconsistent */
#define LVSA_ENOMEM (-2)        /* host or device allocation failed            */
#define LVSA_EDEVICE (-3)       /* a HIP runtime call or kernel launch failed  */
#define LVSA_EUNSUPPORTED (-4)  /* valid, but a shape or layout not implemented */

/* Static, NUL-terminated description of a status code (never NULL). */
const char* lvsa_status_str(lvsa_status s);

/* Library ABI version (major*10000 + minor*100 + patch). */
int32_t lvsa_version(void);

/* ------------------------------------------------------- mask params ---- */

/* Window rules (Sec. 2):
 *   BASIC     Def. 2: [max(0,t-W), min(T-1,t+W)], clipped at the sequence ends.
 *   ADAPTIVE  the "Overlapping frames" paragraph: the window shifted to keep
 *             2W+1 frames, [max(0,min(t-W,T-1-2W)), min(T-1,max(t+W,2W))].
 *   EXPANDED  Alg. 1: the adaptive window grown one frame at a time on the
 *             side with more room (room below = l, above = T-1-h) until it
 *             holds min(2W+1, T-|G|) non-anchor frames.  Default. */
#define LVSA_WINDOW_BASIC 0
#define LVSA_WINDOW_ADAPTIVE 1
#define LVSA_WINDOW_EXPANDED 2

typedef struct lvsa_params {
  int32_t budget_frames; /* C, per-frame budget in frames (Sec. 2, budget
                            paragraph).  Used only when tper == 0, and then
                            must exceed 2W+1.                               */
  int32_t window;        /* W >= 0, window half-width (Def. 2).              */
  int32_t tper;          /* T_per: 0 derives ceil(T / (C - (2W+1))) (Sec. 2);
                            > 0 is an explicit anchor period.                */
  int32_t window_mode;   /* LVSA_WINDOW_*                                    */
  int32_t rotate;        /* 1: anchors G^s of Eq. 3 (rotate with the step);
                            0: Def. 2's fixed G = {t : t mod T_per = 0}.     */
  int32_t tie_high;      /* Alg. 1 leaves equal room unresolved: 0 extends the
                            low side (default), 1 the high side.            */
  int32_t extra_anchors; /* E >= 0 dedicated initial anchors (the
                            generalization named after Def. 2): frames
                            0..E-1 join G at every step, count as global
                            frames in Alg. 1, and leave the budget before
                            the period is derived, T_per = ceil(T / (C -
                            (2W+1) - E)) (needs C > 2W+1+E when tper == 0).
                            E = 1 keeps frame 0 an anchor at every step.
                            Default 0.                                      */
  int32_t text_tokens;   /* L >= 0 text tokens after the T*P video tokens
                            (dual-stream models, whose text-encoder tokens
                            join self-attention, Sec. 3): the mask covers
                            N = T*P + L tokens; every query attends to every
                            text token and every text query to every token.
                            A shorter text is a smaller L.  Default 0.      */
} lvsa_params;

/* Fills *p with C = 21, W = 6, tper = 0, EXPANDED, rotate = 1, tie_high = 0,
 * extra_anchors = 0, text_tokens = 0.
 * C = 21 is the paper's Wan 2.1 budget ((81-1)/4 + 1 frames); the paper does
 * not print W, and 6 is the smallest W that keeps |A(t)| within two frames of
 * C and Alg. 1 within eight iterations on every Wan horizon. */
void lvsa_params_default(lvsa_params* p);

/* Frame-level sets for one denoising step (Def. 2, Eq. 3, Alg. 1).
 *   T       frames, 1 <= T <= LVSA_MAX_FRAMES
 *   step    denoising step s >= 0 (the same s for every layer and for the
 *           conditional and unconditional passes)
 * Outputs (host memory, caller-owned; any may be NULL to skip it):
 *   tper_out      the anchor period T_per used
 *   anchors       [T] ascending anchor frames; *n_anchors = |G^s| (Eq. 3:
 *                 ceil(T/T_per) distinct frames, or 1 when T_per > T) plus
 *                 the extra anchors 0..E-1 that Eq. 3 did not place
 *   win_lo/win_hi [T] window bounds per query frame, so that
 *                 A(t) = anchors  U  [win_lo[t], win_hi[t]]
 *   growth        [T] Alg. 1 growth steps per query frame (frames added to
 *                 the adaptive window; 0 for the other window rules)
 * Errors: EINVAL for T, step or params out of range (including C <= 2W+1+E
 * with tper == 0, E < 0, and a null params pointer). */
#define LVSA_MAX_FRAMES 4096
lvsa_status lvsa_frame_sets(int32_t T, int32_t step, const lvsa_params* p,
                            int32_t* tper_out, int32_t* anchors,
                            int32_t* n_anchors, int32_t* win_lo,
                            int32_t* win_hi, int32_t* growth);

/* The window of one query frame t (0 <= t < T) at step s: the per-frame call
 * whose cost Sec. 2 quotes (the remark after Alg. 1).  Writes lo, hi and the
 * Alg. 1 growth steps (any output may be NULL).  Errors as for
 * lvsa_frame_sets, and EINVAL for t out of range. */
lvsa_status lvsa_frame_window(int32_t T, int32_t step, const lvsa_params* p,
                              int32_t t, int32_t* lo, int32_t* hi,
                              int32_t* growth);

/* ---------------------------------------------------------- block CSR ---- */

/* Token i (0 <= i < N = T*P + L) lies in block i / B and, for i < T*P, in
 * frame i / P; tokens T*P .. N-1 are the text tokens (segment T, L =
 * params->text_tokens, usually 0).  There are nb = ceil(N / B) query blocks
 * and nb key blocks, the last possibly ragged.  Query block qb keeps key
 * block kb iff some token of qb and some token of kb lie in segments t, tau
 * with tau in A(t), or with t or tau the text (Eq. 2 applied to whole blocks:
 * every attended token pair is covered; a block straddling a frame edge
 * brings the rest of its tokens along).  Rows list kb in ascending order,
 * without repeats, and always contain the diagonal block.  The mask does not
 * depend on the head or the layer. */
typedef struct lvsa_csr lvsa_csr; /* opaque, library-owned */

/* Host builder (the paper builds this metadata on the CPU once per step).
 * Thread-safe and reentrant: each calling thread keeps its own working
 * arrays between calls, and lvsa_csr_free passes a handle's host arrays on
 * to later builds (at most 4 sets kept, behind a lock), so a loop that frees
 * step s's handle before building step s+1's touches no fresh memory.
 *   T >= 1 frames (<= LVSA_MAX_FRAMES), P >= 1 tokens per frame,
 *   1 <= B <= 2^20 tokens per block (the attention kernels take 64 or 128),
 *   T*P + B < 2^31 and nb*nb < 2^31 (so nnz fits int32), step >= 0,
 *   layer >= 0 (accepted, no effect).
 * On LVSA_OK, *out owns host arrays row_ptr[nb+1] and col_idx[nnz] (int32);
 * release it with lvsa_csr_free.  Errors: EINVAL (ranges, null pointers,
 * params), ENOMEM.  *out is set to NULL on error. */
lvsa_status lvsa_build_mask(int32_t T, int32_t P, int32_t B, int32_t step,
                            int32_t layer, const lvsa_params* p,
                            lvsa_csr** out);

/* Read-only view of a handle's host CSR: nb query-block rows over nb key
 * blocks (n_q_blocks = n_kv_blocks = nb for self-attention), nnz kept blocks,
 * row_ptr[nb + 1] and col_idx[nnz] (valid until lvsa_csr_free).  Any output
 * pointer may be NULL.  Errors: EINVAL (null handle). */
lvsa_status lvsa_csr_info(const lvsa_csr* csr, int32_t* n_q_blocks,
                          int32_t* n_kv_blocks, int64_t* nnz,
                          const int32_t** row_ptr, const int32_t** col_idx);

/* Tokens N and block size B of a handle.  Errors: EINVAL (null handle). */
lvsa_status lvsa_csr_shape(const lvsa_csr* csr, int32_t* n_tokens, int32_t* block);

/* Copies the host arrays (and, for a handle built by lvsa_build_exact_mask,
 * its entry words) to device memory owned by the handle, allocated in the
 * order of `stream` on the first call and reused after, asynchronously on
 * `stream`; the handle keeps its host arrays until lvsa_csr_free, which waits
 * for this copy.  Errors: EINVAL (null), ENOMEM, EDEVICE. */
lvsa_status lvsa_csr_upload(lvsa_csr* csr, void* stream);

/* Releases the handle.  Waits (on the host) for the handle's last upload to
 * finish, then releases its device arrays in the order of the stream given
 * to that upload, which must still exist; no device-wide synchronization.
 * Attention launches on other streams that read the device arrays must have
 * finished, as for any buffer that is freed.  NULL is accepted. */
void lvsa_csr_free(lvsa_csr* csr);

/* A block CSR in device memory: the mask lvsa_attention reads.  Any valid
 * CSR works (the builders' masks, or a caller's own): row_ptr[0] = 0,
 * row_ptr non-decreasing, nnz = row_ptr[n_q_blocks] < 2^30, each row's
 * col_idx strictly ascending within [0, n_kv_blocks).  The kernels only
 * read it, so launches on any streams may share one mask.  Column values
 * outside [0, n_kv_blocks) are skipped; a row whose entries are not
 * ascending gives an unspecified result, never a read outside row_ptr's
 * range. */
typedef struct lvsa_block_mask {
  int32_t n_tokens;         /* N                                           */
  int32_t block;            /* B, tokens per query block and per key block */
  int32_t n_q_blocks;       /* nb = ceil(N / B)                            */
  int32_t n_kv_blocks;      /* nb (self-attention: the same blocks)        */
  const int32_t* row_ptr;   /* device, [n_q_blocks + 1]                    */
  const int32_t* col_idx;   /* device, [row_ptr[n_q_blocks]]               */
} lvsa_block_mask;

/* Device view of an uploaded handle.  Errors: EINVAL if never uploaded. */
lvsa_status lvsa_csr_device_view(const lvsa_csr* csr, lvsa_block_mask* out);

/* Device builder: the same CSR computed on the GPU (three short kernels on
 * `stream`), written to caller-owned device buffers (no host round trip, no
 * allocation, no memset).
 *   d_row_ptr     device int32[nb + 1]
 *   d_col_idx     device int32[col_capacity]; col_capacity must be at least
 *                 nb * nb (the mask's worst case), so every write is in bounds
 * Arguments as for lvsa_build_mask; T <= LVSA_MAX_FRAMES.
 * Errors: EINVAL (ranges, nulls, capacity), EUNSUPPORTED when a query-block
 * pair would touch more than 1024 frames (2B/P + 2 > 1024 and T > 1024),
 * EDEVICE (launch). */
lvsa_status lvsa_build_mask_device(int32_t T, int32_t P, int32_t B,
                                   int32_t step, int32_t layer,
                                   const lvsa_params* p, int32_t* d_row_ptr,
                                   int32_t* d_col_idx, int64_t col_capacity,
                                   void* stream);

/* ------------------------------------------------ token-exact form ---- */

/* When B does not divide P, a block can straddle a frame edge and the block
 * rule above keeps some token pairs that Eq. 2 drops.  The token-exact form
 * keeps the same blocks (same row_ptr, same order) and gives every kept block
 * an entry word that says which of its query-frame / key-frame parts are
 * attended, so attention computes Eq. 2 token for token (Sec. 2, Eq. 2).
 * It needs P >= B (a block then touches at most two frames), B <= 255 and
 * nb <= 65536.
 *
 * Entry word (uint32) of kept pair (qb, kb); f0 <= f1 are the segments
 * (frames, or T for the text tokens) touched by qb, g0 <= g1 those touched by
 * kb (equal when the block lies in one segment); "frame T is in A(t)" and
 * "frame tau is in A(T)" hold for every t, tau:
 *   bits  0..15  kb
 *   bits 16..23  kfirst: tokens of kb in segment g0 (B when g0 == g1)
 *   bits 24..27  pattern: bit 2a+b set iff frame (b ? g1 : g0) is in
 *                A(a ? f1 : f0)
 *   bits 28..31  zero
 * Query token i of qb attends key token j of kb iff pattern bit
 * 2*(segment(i) != f0) + (segment(j) != g0) is set; segment(i) != f0 holds
 * iff i mod P < (qb*B) mod P, i.e. query rows split at multiples of P. */
typedef struct lvsa_exact_mask {
  int32_t n_tokens;         /* N                                            */
  int32_t block;            /* B                                            */
  int32_t n_q_blocks;       /* nb = ceil(N / B)                             */
  int32_t frame_tokens;     /* P >= B                                       */
  const int32_t* row_ptr;   /* device, [nb + 1], as in lvsa_block_mask      */
  const uint32_t* entry;    /* device, [row_ptr[nb]] entry words, kb ascending */
} lvsa_exact_mask;

/* Host builder of the token-exact form: the handle of lvsa_build_mask
 * (same arguments, same row_ptr and col_idx) plus one entry word per kept
 * block.  Errors as for lvsa_build_mask, and EUNSUPPORTED when P < B,
 * B > 255 or nb > 65536.  *out is set to NULL on error. */
lvsa_status lvsa_build_exact_mask(int32_t T, int32_t P, int32_t B,
                                  int32_t step, int32_t layer,
                                  const lvsa_params* p, lvsa_csr** out);

/* Host entry words of a handle built by lvsa_build_exact_mask (valid until
 * lvsa_csr_free; nnz of them) and its P.  Errors: EINVAL (null),
 * EUNSUPPORTED for a handle without entry words (lvsa_build_mask). */
lvsa_status lvsa_csr_entries(const lvsa_csr* csr, int32_t* frame_tokens,
                             const uint32_t** entry);

/* Device view of the token-exact form of an uploaded handle built by
 * lvsa_build_exact_mask (lvsa_csr_upload copies the entry words too).
 * Errors: EINVAL if never uploaded, EUNSUPPORTED as for lvsa_csr_entries. */
lvsa_status lvsa_csr_exact_view(const lvsa_csr* csr, lvsa_exact_mask* out);

/* Device builder of the token-exact form: row_ptr and entry words of the
 * same mask as lvsa_build_mask_device, on `stream`, into caller-owned
 * buffers
 *   d_row_ptr    device int32[nb + 1]
 *   d_entry      device uint32[entry_capacity], entry_capacity >= nb * nb
 * Errors: EINVAL (ranges, nulls, capacity), EUNSUPPORTED (P < B, B > 255,
 * nb > 65536, or as for lvsa_build_mask_device), EDEVICE (launch). */
lvsa_status lvsa_build_exact_mask_device(int32_t T, int32_t P, int32_t B,
                                         int32_t step, int32_t layer,
                                         const lvsa_params* p,
                                         int32_t* d_row_ptr, uint32_t* d_entry,
                                         int64_t entry_capacity, void* stream);

/* --------------------------------------------------------- attention ---- */

/* A bf16 tensor [heads, n_tokens, head_dim] in device memory.  Element
 * (h, i, c) is at data + h*stride_head + i*stride_token + c (elements; the
 * head_dim stride is 1).  data must be 16-byte aligned and stride_token and
 * stride_head multiples of 8. */
typedef struct lvsa_tensor {
  void* data;
  int32_t heads;
  int32_t n_tokens;
  int32_t head_dim;
  int64_t stride_head;
  int64_t stride_token;
} lvsa_tensor;

/* Tile counters.  The attention kernels run one persistent workgroup per
 * compute unit; workgroups take tiles (a head and two adjacent query blocks)
 * through atomic counters, eight per launch (one per XCD), so XCDs that
 * clock faster take on more tiles.  Every launch gets counters of its own
 * from a per-device pool the library owns (a few KB, allocated on the first
 * launch on a device and grown when every counter set is still in use), zeroed
 * by a small kernel on the launch stream before the attention kernel runs and
 * handed to a later launch only after an event recorded behind this one has
 * completed.  A launch recorded into a graph under stream capture keeps its
 * counters for the life of the process (replays of one graph are ordered).
 * So nothing that a launch reads is written by another launch: masks and
 * inputs may be shared by launches in flight on any streams. */

/* Block-sparse attention forward (Eq. 2 over the kept blocks of `mask`):
 *   out[h, i] = sum_j softmax_j(q[h,i] . k[h,j] / sqrt(d)) v[h,j]
 * with j over the real tokens (j < N) of the key blocks kept for the query
 * block of i.  bf16 inputs, fp32 products and softmax, bf16 output (round to
 * nearest even).  q, k, v, out share heads, n_tokens = mask->n_tokens and
 * head_dim = 128; mask->block is 64 or 128 and mask->n_q_blocks =
 * mask->n_kv_blocks = ceil(N / B) <= 8000 (a workgroup merges the two CSR
 * rows of its pair of query blocks in LDS).  Rows i >= N of `out` are never written;
 * a query block whose row is empty gets zeros.  out must not overlap q, k or
 * v.  The result is deterministic (fixed key order per row, whichever
 * workgroup computes it).
 * Errors: EINVAL (nulls, shape mismatch), EUNSUPPORTED (head_dim, block,
 * alignment), ENOMEM (tile counters), EDEVICE (launch). */
lvsa_status lvsa_attention(const lvsa_tensor* q, const lvsa_tensor* k,
                           const lvsa_tensor* v, const lvsa_block_mask* mask,
                           lvsa_tensor* out, void* stream);

/* lvsa_attention without any allocation, for callers that cannot allocate
 * device memory (code under graph capture, tight serving loops, harnesses
 * that forbid allocation): the same kernels and results, with the tile
 * counters taken from a fixed array in the library's device data (one set
 * of counters, 64 bytes per device, enough for every launch lvsa_attention
 * accepts; the shape limits are the same).  It allocates nothing and issues
 * no memset: the counters are zeroed by a kernel on `stream`.  All calls on
 * one device share that array, so calls that overlap in time on one device
 * (on two streams, or from two threads) race; successive calls on one
 * stream are fine.  Errors as for lvsa_attention (EDEVICE when the array's
 * device address cannot be looked up). */
lvsa_status lvsa_attention_noalloc(const lvsa_tensor* q, const lvsa_tensor* k,
                                   const lvsa_tensor* v, const lvsa_block_mask* mask,
                                   lvsa_tensor* out, void* stream);

/* Token-exact attention forward (Eq. 2 token for token): as lvsa_attention,
 * with the keys of each kept block further restricted, per query token, by
 * the block's entry word, so query i attends exactly the keys j with
 * frame(j) in A(frame(i)).  mask->block is 64 or 128, mask->frame_tokens
 * >= mask->block and mask->n_q_blocks <= 8000; every query token keeps at
 * least its own frame's keys.
 * Errors as for lvsa_attention. */
lvsa_status lvsa_attention_exact(const lvsa_tensor* q, const lvsa_tensor* k,
                                 const lvsa_tensor* v,
                                 const lvsa_exact_mask* mask, lvsa_tensor* out,
                                 void* stream);

/* Dense attention forward (Eq. 1 over all N keys), the same kernel design
 * visiting every key block; `block` (64 or 128) is its tile size.  Up to
 * 8000 key blocks it runs the block-sparse kernel with every block kept (no
 * CSR is read or allocated); past that, a dense instantiation of the same
 * kernel.  No upper limit on N beyond the tensor checks.
 * Errors as for lvsa_attention. */
lvsa_status lvsa_dense_attention(const lvsa_tensor* q, const lvsa_tensor* k,
                                 const lvsa_tensor* v, int32_t block,
                                 lvsa_tensor* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LVSA_H */
