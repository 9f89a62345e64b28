/*
 * umem.h -- C ABI of the UltraMem memory-layer forward on AMD Instinct MI355X (gfx950).
 *
 * The layer is the ultra-sparse memory layer of "Ultra-Sparse Memory Network" (Huang et al.):
 *   a1  axis scores        Sec. 3.1 eq. (2); Sec. 3.2 TDQKR eq. (4)
 *   a2  rank-1 reduction   Sec. 3.2 TDQKR eqs. (6)-(9), (11)  (Tucker grid only)
 *   a3  per-axis top-k     eq. (2) sigma_TopM; eqs. (8), (9) I_TopM
 *   a4  grid scores        eq. (3) (additive); eq. (10) (Tucker core, exact on the candidates)
 *   a5  global top-m       eq. (3) / eq. (10); weights raw (Sec. 3.2 Trick 1) or SoftMax (eq. (3))
 *   a6  IVE address map    Sec. 3.2 IVE eqs. (13), (14)
 *   a7  gather-sum         eq. (1) o = V^T s; eq. (15) per virtual block; heads add (Sec. 3.1)
 *   a8  projection         eq. (15) sum_p W_p^T (.); Sec. 3.2 Trick 6 output linear
 *
 * Conventions shared by every entry point:
 *   - All array arguments are DEVICE pointers owned by the caller, dense and row-major, unless
 *     stated otherwise.  The library never allocates, frees or synchronises; it only enqueues
 *     kernels on `stream` (NULL = the default stream).  Scratch memory comes from the caller
 *     (`ws`, sized by umem_workspace_size).
 *   - Calls are asynchronous.  The returned status covers argument validation and launch
 *     errors only.  Every argument is validated before the first launch: on a validation error
 *     (UMEM_ERR_INVALID_ARG, UMEM_ERR_UNSUPPORTED, UMEM_ERR_WORKSPACE) nothing is enqueued and
 *     no output is written.  UMEM_ERR_HIP reports a launch that the HIP runtime refused; in an
 *     entry point that launches several kernels, the kernels enqueued before that one stay
 *     enqueued and may write outputs and scratch.  Device-side faults (e.g. an index out of
 *     range in a caller-supplied bag) are not detected.  A HIP error that an earlier call left
 *     pending in the calling thread is cleared, unreported, before a call launches its kernels.
 *   - Ties: every selection orders by (score desc, index asc) -- the per-axis key index, or the
 *     logical flat index i*n + j on the grid; -0.0 equals +0.0; NaN ranks below -inf.
 *     Selections are returned sorted in that order.
 *   - Indices are int32 (n*n < 2^31); byte offsets into the value table are 64-bit.
 *   - Alignment: q/k/core 16 bytes, values and fp32 outputs 16 bytes, other arrays 4 bytes.
 *   - T == 0 is a no-op once the descriptor is valid.
 *   - Functions are reentrant; calls on one stream run in order.
 */
#ifndef UMEM_H
#define UMEM_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define UMEM_API __attribute__((visibility("default")))

typedef enum umem_status {
  UMEM_OK = 0,
  UMEM_ERR_INVALID_ARG = -1, /* a null pointer, a bad size or a misaligned buffer */
  UMEM_ERR_UNSUPPORTED = -2, /* valid for the paper, beyond this library's limits (below) */
  UMEM_ERR_WORKSPACE = -3,   /* ws too small or misaligned */
  UMEM_ERR_HIP = -4,         /* a HIP launch failed */
  UMEM_ERR_SCRATCH_LIMIT = -5 /* umem_forward_noalloc: the call needs more scratch than
                               * UMEM_STATIC_SCRATCH_BYTES */
} umem_status;

enum { UMEM_F32 = 0, UMEM_BF16 = 1 };             /* value-table element type */
enum { UMEM_GRID_ADD = 0, UMEM_GRID_TUCKER = 1 }; /* eq. (3) / eq. (10) */
enum { UMEM_W_RAW = 0, UMEM_W_SOFTMAX = 1 };      /* Trick 1 (raw scores) / eq. (3) SoftMax */

/* Shape of one memory layer.
 * Requirements (UMEM_ERR_INVALID_ARG otherwise): every count >= 1; dk % rank == 0;
 *   rank == 1 for UMEM_GRID_ADD; topk <= n_keys; topm <= topk^2; expand a perfect square with
 *   n_values * expand == n_keys^2; dv_virt > 0 when expand > 1; cores (h) of 0 or 1, or h >= 2
 *   with the Tucker grid, raw weights and dv % h == 0.
 * Limits of this library (UMEM_ERR_UNSUPPORTED beyond them): max(n_keys, topk^2) <= 8192;
 *   topk <= 90 (64 for the Tucker grid); topm <= 256; rank <= 4; (dk / rank) % 4 == 0; dk <= 1024; heads <= 64;
 *   heads * topm <= 2048; expand <= 64; a value row (dv * element size) of 16 * 2^j <= 1024
 *   bytes or a multiple of 1024 up to 8192 bytes; T <= 2^20; cores <= 8, each core's column
 *   slice (dv / h elements) a multiple of 16 bytes; dv_virt and d_out multiples of 8 (weight
 *   rows of 16-byte pieces). */
typedef struct umem_desc {
  int32_t heads;    /* H: key sets (each with its own keys and core) sharing one value table */
  int32_t dk;       /* query/key dimension per axis per head */
  int32_t n_keys;   /* n keys per axis; the logical grid has N = n*n slots */
  int32_t rank;     /* Tucker rank r: dk is read as r contiguous slices of dk/r (eq. (4)) */
  int32_t topk;     /* k: per-axis top-k */
  int32_t topm;     /* m: global top-m per head; each token's bag holds heads*topm slots */
  int32_t grid;     /* UMEM_GRID_ADD or UMEM_GRID_TUCKER */
  int32_t weight;   /* UMEM_W_RAW or UMEM_W_SOFTMAX */
  int64_t n_values; /* N_p physical value rows (= N / expand) */
  int32_t dv;       /* physical value dimension */
  int32_t vdtype;   /* UMEM_F32 or UMEM_BF16 */
  int32_t expand;   /* E: implicit value expansion (1 = none) */
  int32_t dv_virt;  /* D'v: IVE projector width (0 = no projection; required when expand > 1) */
  int32_t d_out;    /* output linear width (0 = none) */
  int32_t cores;    /* h: multi-core scoring (Sec. 3.2 MCS, eqs. (16), (17)); 0 or 1 = one core.
                     * With h >= 2 each head's Tucker core is given as h component cores
                     * [H, h, r, r]; selection runs on their sum, every selected slot carries
                     * the h component scores as weights [.., m, h], and column slice i of each
                     * value row (dv / h columns; physical rows with IVE) takes weight i. */
} umem_desc;

/* Bytes of scratch `ws` that umem_score_topk / umem_forward need for T tokens (a multiple of
 * 256; pass ws aligned to 256 bytes).  Writes 0 to *bytes and returns an error for an invalid
 * descriptor. */
UMEM_API umem_status umem_workspace_size(const umem_desc* desc, int32_t T, size_t* bytes);

/* a1 + a2: per-axis selection scores -- eq. (2) for the additive grid; u^T S_row and
 * t^T S_col of eqs. (6), (8), (9) for the Tucker grid, with (u, t) the leading singular pair of
 * each head's core (eq. (11)), the sign fixed so that u's largest-magnitude component is
 * positive and t = C^T u / sigma_1.  The singular pair is computed on the device, in fp64.
 *   q_row, q_col  fp32 [T, H, dk]  the two queries; may be the same pointer (Trick 5)
 *   k_row, k_col  fp32 [H, n, dk]  keys; with rank r each dk row holds r contiguous slices
 *   core          fp32 [H, r, r]   Tucker cores (NULL for UMEM_GRID_ADD); [H, h, r, r] component
 *                                  cores with multi-core scoring (their sum is the core)
 *   sel           fp32 [2, T, H, n] out: [0] row scores, [1] column scores
 *   ws            256-byte aligned scratch: the singular vectors (Tucker grid, 2 KiB), then for
 *                 T > 64 tokens the fp16 planes of the many-token kernel and their rows'
 *                 exponents (2 * 2 * (T + n_keys) * heads * dk * 2 + 2 * (T + n_keys) * heads * 4
 *                 bytes where dk % 32 == 0, (dk / rank) % 8 == 0 and n_keys % 4 == 0); a
 *                 workspace sized by umem_workspace_size suffices; may be NULL where neither is
 *                 needed */
UMEM_API umem_status umem_axis_scores(const umem_desc* desc, int32_t T, const float* q_row,
                                      const float* q_col, const float* k_row, const float* k_col,
                                      const float* core, float* sel, void* ws, size_t ws_bytes,
                                      hipStream_t stream);

/* a3 + a4 + a5 from selection scores: per-axis top-k, grid scores of the k*k candidates
 * (additive eq. (3); Tucker eq. (10) with the per-slice scores recomputed exactly for the
 * candidates, non-candidates excluded), global top-m and weights; optionally a7 as well.
 *   sel       fp32 [2, T, H, n] as written by umem_axis_scores, 16-byte aligned
 *   q_*, k_*, core  as above; read only for UMEM_GRID_TUCKER (may be NULL for ADD)
 *   idx       int32 [T, H, m] out: logical slot i*n + j, sorted by (score desc, index asc)
 *   w         fp32 [T, H, m] out: the weight of each slot (raw grid score, or SoftMax); with
 *             multi-core scoring [T, H, m, h]: the h component scores of each slot (eq. (16))
 *   axis_idx  int32 [2, T, H, k] out, optional (NULL): per-axis top-k, sorted
 *   values, pooled  optional (both NULL or both set): the value table [n_values, dv] and fp32
 *             [T, dv] (16-byte aligned); the selected rows are pooled as umem_gather_sum pools
 *             them (eq. (1)) and ADDED to pooled, which the caller clears beforehand.  Only for
 *             layers without expansion, with heads <= 2, topm <= 64 and value rows of 1 or
 *             2 KiB (UMEM_ERR_UNSUPPORTED otherwise); with two heads the result does not depend
 *             on their order (two adds onto zero commute exactly).  umem_forward uses this form
 *             where it applies and T <= 128, instead of a separate gather launch. */
UMEM_API umem_status umem_select(const umem_desc* desc, int32_t T, const float* sel, const float* q_row,
                        const float* q_col, const float* k_row, const float* k_col,
                        const float* core, int32_t* idx, float* w, int32_t* axis_idx,
                        const void* values, float* pooled, hipStream_t stream);

/* a1 .. a5: umem_axis_scores followed by umem_select, the scores kept in `ws`
 * (ws_bytes >= umem_workspace_size(desc, T)). */
UMEM_API umem_status umem_score_topk(const umem_desc* desc, int32_t T, const float* q_row,
                            const float* q_col, const float* k_row, const float* k_col,
                            const float* core, int32_t* idx, float* w, int32_t* axis_idx,
                            void* ws, size_t ws_bytes, hipStream_t stream);

/* a6 + a7: score-weighted gather-sum (embedding bag) of value rows -- eq. (1), eq. (15).
 *   values  [n_values, dv] of vdtype, 16-byte aligned
 *   idx     int32 [T, bag]: logical slots; without perm and with expand == 1 they are physical
 *           rows (Sec. 3.1: slot (i, j) lives at row n*i + j)
 *   w       fp32 [T, bag], or [T, bag, cores]: with cores = h >= 2 column slice i of each row
 *           (dv / h columns) takes weight i (multi-core scoring, eq. (17))
 *   perm    int32 [expand * n_values] or NULL: the IVE shuffle (eq. (14)); slot x goes to virtual
 *           slot v = perm[x], block p = v / n_values, physical row v % n_values
 *   cores   1 (or 0), or the h of multi-core scoring: dv % h == 0, each slice a multiple of
 *           16 bytes, h <= 8
 *   out     fp32 [T, expand, dv], 16-byte aligned: out[t, p, :] = sum over the bag entries of
 *           block p of w * values[row, :] (fp32 accumulation; repeated rows add)
 * Every index must be in range ([0, n_values) without perm, [0, expand*n_values) with it). */
UMEM_API umem_status umem_gather_sum(int64_t n_values, int32_t dv, int32_t vdtype, const void* values,
                            int32_t T, int32_t bag, const int32_t* idx, const float* w,
                            const int32_t* perm, int32_t expand, int32_t cores, float* out,
                            hipStream_t stream);

/* Scratch bytes umem_project needs for these sizes (the intermediate of the output linear and
 * the partial sums of split reductions over long K); dv_virt == 0 sizes the output linear alone.
 * Same shape requirements as umem_project. */
UMEM_API umem_status umem_project_workspace_size(int32_t T, int32_t expand, int32_t dv, int32_t dv_virt,
                                        int32_t d_out, size_t* bytes);

/* a8: y = sum_p pooled[:, p, :] W_p (eq. (15)), then y W_out (Trick 6).  bf16 operands (the
 * fp32 pooled sums and the intermediate are rounded to bf16, nearest even), fp32 accumulation.
 * The weights are stored output-major, as a linear layer's weight ([out features, in features]):
 *   pooled  fp32 [T, E, dv]
 *   w_proj  bf16 bits [dv_virt, E * dv]: element (j, p * dv + c) is W_p[c][j]
 *   w_out   bf16 bits [d_out, dv_virt] (element (o, j) is W_out[j][o]), or NULL
 *   out     fp32 [T, d_out] (or [T, dv_virt] without w_out).  With w_proj NULL (dv_virt 0,
 *           expand 1) the output linear alone: out = pooled [T, dv] by w_out [d_out, dv]^T
 *   ws      16-byte aligned scratch of umem_project_workspace_size(...) bytes (NULL if 0)
 * The result does not depend on timing (split reductions add their partials in a fixed order).
 * UMEM_ERR_UNSUPPORTED unless pooled, w_proj and w_out are 16-byte aligned, expand * dv,
 * dv_virt and d_out are multiples of 8, each weight is below 2 GiB and each GEMM's inner
 * dimension (expand * dv, dv_virt) is at most 2^20. */
UMEM_API umem_status umem_project(int32_t T, int32_t expand, int32_t dv, int32_t dv_virt, int32_t d_out,
                         const float* pooled, const uint16_t* w_proj, const uint16_t* w_out,
                         float* out, void* ws, size_t ws_bytes, hipStream_t stream);

/* a1 .. a8: the whole forward of the layer for T tokens.
 *   values, perm     as for umem_gather_sum (perm required iff expand > 1)
 *   w_proj, w_out    as for umem_project (w_proj required iff dv_virt > 0; w_out iff d_out > 0;
 *                    16-byte aligned, else UMEM_ERR_UNSUPPORTED)
 *   out              fp32: [T, dv] without projection, else [T, d_out] (or [T, dv_virt])
 *   idx_out, w_out_scores  optional (NULL) copies of the selection, [T, H, m] each
 *                    (w_out_scores [T, H, m, h] with multi-core scoring)
 * ws_bytes >= umem_workspace_size(desc, T). */
UMEM_API umem_status umem_forward(const umem_desc* desc, int32_t T, const float* q_row, const float* q_col,
                         const float* k_row, const float* k_col, const float* core,
                         const void* values, const int32_t* perm, const uint16_t* w_proj,
                         const uint16_t* w_out, float* out, int32_t* idx_out,
                         float* w_out_scores, void* ws, size_t ws_bytes, hipStream_t stream);

/* Bytes of the library's static scratch array (one per GPU), which umem_forward_noalloc uses in
 * place of a workspace argument. */
#define UMEM_STATIC_SCRATCH_BYTES ((size_t)64 << 20)

/* umem_forward for callers that cannot allocate memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): the same kernels and results, with the
 * workspace taken from a static array of UMEM_STATIC_SCRATCH_BYTES in each GPU's memory instead
 * of the caller.  Neither this call nor the kernels it enqueues allocate or free memory.
 *   Arguments as for umem_forward, without ws and ws_bytes.
 *   UMEM_ERR_SCRATCH_LIMIT (nothing enqueued) when umem_workspace_size(desc, T) exceeds
 *   UMEM_STATIC_SCRATCH_BYTES (the 20.07M-slot decode layer fits up to 779 tokens).
 *   The array of a GPU is created with the library's code on that GPU and held until the process
 *   ends; the first call on a device looks up its address (UMEM_ERR_HIP if that fails).  `stream`
 *   must belong to the calling thread's current device.  Every call on one GPU uses the same
 *   array and leaves its contents behind (nothing in it needs clearing between calls): calls
 *   that may run at the same time on one GPU (other streams, other threads) race on it and must
 *   be serialised by the caller. */
UMEM_API umem_status umem_forward_noalloc(const umem_desc* desc, int32_t T, const float* q_row,
                                          const float* q_col, const float* k_row,
                                          const float* k_col, const float* core,
                                          const void* values, const int32_t* perm,
                                          const uint16_t* w_proj, const uint16_t* w_out,
                                          float* out, int32_t* idx_out, float* w_out_scores,
                                          hipStream_t stream);

/* Backward of the gather-sum (eq. (1); eq. (15) per virtual block; eq. (17) per column slice),
 * for training: with the selection of the forward held fixed,
 *   dw[t, b(, c)] = <d_pooled[t, p, slice c], V[row, slice c]>   (written)
 *   d_values[row, slice c] += sum over the entries (t, b) on that row of w[t, b(, c)] d_pooled[t, p, slice c]
 * where (p, row) is the entry's virtual block and physical row (as umem_gather_sum maps them).
 *   values, idx, w, perm, expand, cores  as for umem_gather_sum (the forward's selection)
 *   d_pooled  fp32 [T, expand, dv], 16-byte aligned: the gradient of the pooled rows
 *   d_values  fp32 [n_values, dv], 16-byte aligned: accumulated into (only the rows the bag
 *             touches change; clear it between steps as the optimiser needs)
 *   dw        fp32 [T, bag] or [T, bag, cores]
 *   ws        16-byte aligned scratch of umem_gather_backward_workspace_size(T, bag, dv) bytes
 * Entries on one row are summed in a fixed order (in segments of their bag order, then the
 * segments in order), so the result does not depend on timing.  T * bag <= 2^22
 * (UMEM_ERR_UNSUPPORTED beyond). */
UMEM_API umem_status umem_gather_backward_workspace_size(int32_t T, int32_t bag, int32_t dv, size_t* bytes);
UMEM_API umem_status umem_gather_backward(int64_t n_values, int32_t dv, int32_t vdtype, const void* values,
                                 int32_t T, int32_t bag, const int32_t* idx, const float* w,
                                 const int32_t* perm, int32_t expand, int32_t cores,
                                 const float* d_pooled, float* d_values, float* dw, void* ws,
                                 size_t ws_bytes, hipStream_t stream);

/* The same backward (eq. (1); eq. (15); eq. (17)) with the value-row gradients returned
 * compactly, one row per distinct physical row the bag touches, instead of added into a dense
 * [n_values, dv] table (41 GB of fp32 for a 20M-slot table of 512-wide rows):
 *   rows      int32 [T * bag] (capacity): the distinct physical rows, ascending; the first
 *             *n_rows are written
 *   d_rows    fp32 [T * bag, dv] (capacity), 16-byte aligned: d_rows[r] = sum over the entries
 *             on rows[r] of w d_pooled (written, not accumulated; rows past *n_rows untouched)
 *   n_rows    int32 [1], device memory: the number of distinct rows (written)
 *   dw, everything else  as for umem_gather_backward; ws of umem_gather_backward_workspace_size
 * d_rows[r] equals, bit for bit, what umem_gather_backward adds into a zeroed d_values row
 * rows[r].  The dense gradient row is neither read nor written, so the call moves the value rows,
 * d_pooled and the compact rows only.  T == 0 writes nothing (n_rows included). */
UMEM_API umem_status umem_gather_backward_rows(int64_t n_values, int32_t dv, int32_t vdtype,
                                      const void* values, int32_t T, int32_t bag,
                                      const int32_t* idx, const float* w, const int32_t* perm,
                                      int32_t expand, int32_t cores, const float* d_pooled,
                                      int32_t* rows, float* d_rows, int32_t* n_rows, float* dw,
                                      void* ws, size_t ws_bytes, hipStream_t stream);

/* Backward of the scores (eqs. (2)-(4), (10), (16)) with the forward's selection held fixed: the
 * gradient reaches q, K and C only through the selected slots' scores (the top-k and top-m are
 * piecewise constant; the rank-1 factors only select).  Weight gradients become grid-score
 * gradients (eq. (3)'s SoftMax Jacobian with UMEM_W_SOFTMAX), then
 *   additive: dS_row[i] += dg, dS_col[j] += dg;  Tucker (per core c with multi-core scoring):
 *   dS_row[:, i] += dg C S_col[:, j], dS_col[:, j] += dg C^T S_row[:, i], dC += dg S_row[:, i] S_col[:, j]^T
 *   dq[slice r] = sum_i dS[r, i] K[i, slice r]  (written), dK[i, slice r] += dS[r, i] q[slice r]
 *   desc, q_row, q_col, k_row, k_col, core  as for the forward
 *   idx     int32 [T, H, m]: the forward's selection; w fp32 [T, H, m]: its weights (needed with
 *           UMEM_W_SOFTMAX, else may be NULL)
 *   dw      fp32 [T, H, m] (or [T, H, m, h] with multi-core scoring): the weight gradients
 *   dq_row, dq_col  fp32 [T, H, dk] (written); dk_row, dk_col fp32 [H, n_keys, dk], 16-byte
 *           aligned (accumulated); dcore fp32 [H, r, r] or [H, h, r, r] (accumulated; Tucker
 *           grid only, else NULL)
 *   ws      16-byte aligned scratch of umem_score_backward_workspace_size(desc, T) bytes
 * Sums over tokens (dK, dC) run in a fixed order.  T * H * 2 * m <= 2^22. */
UMEM_API umem_status umem_score_backward_workspace_size(const umem_desc* desc, int32_t T, size_t* bytes);
UMEM_API umem_status umem_score_backward(const umem_desc* desc, int32_t T, const float* q_row,
                                const float* q_col, const float* k_row, const float* k_col,
                                const float* core, const int32_t* idx, const float* w,
                                const float* dw, float* dq_row, float* dq_col, float* dk_row,
                                float* dk_col, float* dcore, void* ws, size_t ws_bytes,
                                hipStream_t stream);

/* The query front-end of the layer (Sec. 3.2 bag of tricks): a causal depthwise convolution
 * of the hidden states (Trick 4), the query linear of eq. (2), and a LayerNorm of each head's
 * query (Trick 2); with `shared` one query serves both key sets (Trick 5). */
typedef struct umem_query_desc {
  int32_t d_model;  /* width d of the hidden states */
  int32_t conv_k;   /* K_c: convolution taps per channel, tap 0 the current token */
  int32_t heads;    /* H */
  int32_t dk;       /* D_k per head */
  int32_t shared;   /* 1: one query per head for both key sets; 0: row and column queries */
  float eps;        /* LayerNorm epsilon */
} umem_query_desc;
/* Requirements (UMEM_ERR_INVALID_ARG otherwise): every count >= 1, shared 0 or 1, eps >= 0.
 * Limits (UMEM_ERR_UNSUPPORTED beyond them): d_model % 8 == 0; conv_k <= 8; dk <= 1024;
 *   (shared ? 1 : 2) * heads * dk a multiple of 8; the query weight below 2 GiB; d_model <= 2^20. */

/* Scratch bytes umem_query needs for B sequences of L tokens. */
UMEM_API umem_status umem_query_workspace_size(const umem_query_desc* qd, int32_t B, int32_t L,
                                      size_t* bytes);

/* Queries of T = B * L tokens (token t = b * L + l of sequence b) from their hidden states.
 *   x       fp32 [B, L, d_model], 16-byte aligned
 *   x_hist  fp32 [B, conv_k - 1, d_model], 16-byte aligned: the hidden states before each
 *           sequence's first token here (oldest first), or NULL for zeros (a sequence start)
 *   conv_w  fp32 [conv_k, d_model], 16-byte aligned (no bias)
 *   w_q     bf16 bits [A * heads * dk, d_model] (output-major, as a linear layer's weight),
 *           16-byte aligned, A = 1 if shared else 2: the row queries of the H heads, then (A = 2)
 *           the column queries; the convolved rows are rounded to bf16 (nearest even) for this
 *           product, fp32 accumulation.  d_model a multiple of 8, w_q below 2 GiB
 *   gamma, beta  fp32 [A, heads, dk]: the LayerNorm of each (axis, head)
 *   q_row   fp32 [T, heads, dk]; q_col the same, or NULL when shared (pass q_row for both
 *           key sets to the scoring then)
 *   ws      16-byte aligned scratch of umem_query_workspace_size(...) bytes */
UMEM_API umem_status umem_query(const umem_query_desc* qd, int32_t B, int32_t L, const float* x,
                       const float* x_hist, const float* conv_w, const uint16_t* w_q,
                       const float* gamma, const float* beta, float* q_row, float* q_col,
                       void* ws, size_t ws_bytes, hipStream_t stream);

/* The LayerNorm of a key set (Trick 2), computed once since keys are parameters: each of the
 * heads * n rows of dk elements of keys [heads, n, dk] is normalised (population variance, eps)
 * and scaled and shifted by its head's gamma, beta [heads, dk].  out may equal keys.
 * dk <= 1024 (UMEM_ERR_UNSUPPORTED beyond). */
UMEM_API umem_status umem_key_norm(int32_t heads, int32_t n, int32_t dk, const float* keys,
                          const float* gamma, const float* beta, float eps, float* out,
                          hipStream_t stream);

/* A static, human-readable name of a status code. */
UMEM_API const char* umem_status_string(umem_status status);

#ifdef __cplusplus
}
#endif

#endif /* UMEM_H */
