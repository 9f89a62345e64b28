// The C ABI of libumem: argument validation, workspace layout and kernel sequencing.
// Every entry point validates everything before it enqueues anything.
#include <stdint.h>

#include <cmath>

#include <algorithm>
#include <mutex>

#include "umem_internal.h"

using namespace umem;

namespace {

constexpr size_t kAlign = 256;

size_t round_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int64_t isqrt64(int64_t x) {
  int64_t r = 0;
  while ((r + 1) * (r + 1) <= x) ++r;
  return r;
}

umem_status check_desc(const umem_desc* d) {
  if (d == nullptr) return UMEM_ERR_INVALID_ARG;
  if (d->heads < 1 || d->dk < 1 || d->n_keys < 1 || d->rank < 1 || d->topk < 1 || d->topm < 1 ||
      d->dv < 1 || d->expand < 1 || d->n_values < 1 || d->dv_virt < 0 || d->d_out < 0)
    return UMEM_ERR_INVALID_ARG;
  if (d->grid != UMEM_GRID_ADD && d->grid != UMEM_GRID_TUCKER) return UMEM_ERR_INVALID_ARG;
  if (d->weight != UMEM_W_RAW && d->weight != UMEM_W_SOFTMAX) return UMEM_ERR_INVALID_ARG;
  if (d->vdtype != UMEM_F32 && d->vdtype != UMEM_BF16) return UMEM_ERR_INVALID_ARG;
  if (d->cores < 0) return UMEM_ERR_INVALID_ARG;
  if (d->cores > 1) {
    if (d->grid != UMEM_GRID_TUCKER || d->weight != UMEM_W_RAW || d->dv % d->cores != 0)
      return UMEM_ERR_INVALID_ARG;
    if (!cores_supported(d->dv, d->vdtype, d->cores)) return UMEM_ERR_UNSUPPORTED;
  }
  if (d->dk % d->rank != 0) return UMEM_ERR_INVALID_ARG;
  if (d->grid == UMEM_GRID_ADD && d->rank != 1) return UMEM_ERR_INVALID_ARG;
  if (d->topk > d->n_keys) return UMEM_ERR_INVALID_ARG;
  if (static_cast<int64_t>(d->topm) > static_cast<int64_t>(d->topk) * d->topk)
    return UMEM_ERR_INVALID_ARG;
  const int64_t e = isqrt64(d->expand);
  if (e * e != d->expand) return UMEM_ERR_INVALID_ARG;
  if (d->expand > 1 && d->dv_virt == 0) return UMEM_ERR_INVALID_ARG;
  if (d->n_keys > kMaxSelect) return UMEM_ERR_UNSUPPORTED;   // also keeps n*n < 2^31
  if (static_cast<int64_t>(d->n_keys) * d->n_keys != d->n_values * d->expand)
    return UMEM_ERR_INVALID_ARG;
  if (d->topk > kMaxTopK || d->topk * d->topk > kMaxSelect || d->topm > kMaxTopM)
    return UMEM_ERR_UNSUPPORTED;
  if (d->grid == UMEM_GRID_TUCKER && d->topk > kMaxTopKTucker) return UMEM_ERR_UNSUPPORTED;
  if (d->grid == UMEM_GRID_ADD && additive_candidates(d->topk, d->topm) > 2048) return UMEM_ERR_UNSUPPORTED;
  if (d->rank > kMaxRank || (d->dk / d->rank) % 4 != 0 || d->dk > kMaxDk) return UMEM_ERR_UNSUPPORTED;
  if (d->heads > kMaxHeads || d->heads * d->topm > kMaxBag) return UMEM_ERR_UNSUPPORTED;
  if (d->expand > kMaxExpand) return UMEM_ERR_UNSUPPORTED;
  if (!gather_row_supported(d->dv, d->vdtype)) return UMEM_ERR_UNSUPPORTED;
  if (d->dv_virt % 8 != 0 || d->d_out % 8 != 0) return UMEM_ERR_UNSUPPORTED;   // 16-byte weight rows
  if (d->dv_virt > 0 && ((static_cast<int64_t>(d->expand) * d->dv) % 8 != 0 ||
                         !gemm_weight_supported(d->dv_virt, static_cast<int64_t>(d->expand) * d->dv) ||
                         !gemm_weight_supported(d->d_out, d->dv_virt)))
    return UMEM_ERR_UNSUPPORTED;
  // the output linear alone reads the pooled rows (bf16) in 16-byte pieces of 8
  if (d->dv_virt == 0 && d->d_out > 0 && (d->dv % 8 != 0 || !gemm_weight_supported(d->d_out, d->dv)))
    return UMEM_ERR_UNSUPPORTED;
  return UMEM_OK;
}

umem_status check_tokens(int32_t T) {
  if (T < 0) return UMEM_ERR_INVALID_ARG;
  if (T > kMaxTokens) return UMEM_ERR_UNSUPPORTED;
  return UMEM_OK;
}

umem_status check_scoring_ptrs(const umem_desc* d, const float* q_row, const float* q_col,
                               const float* k_row, const float* k_col, const float* core) {
  if (!q_row || !q_col || !k_row || !k_col) return UMEM_ERR_INVALID_ARG;
  if (!aligned(q_row, 16) || !aligned(q_col, 16) || !aligned(k_row, 16) || !aligned(k_col, 16))
    return UMEM_ERR_INVALID_ARG;
  if (d->grid == UMEM_GRID_TUCKER && (core == nullptr || !aligned(core, 4))) return UMEM_ERR_INVALID_ARG;
  return UMEM_OK;
}

struct Layout {
  size_t factors, sel, idx, w, pooled, proj, total;
};

// Workspace: [rank-1 factors (Tucker)] [selection scores] [idx] [w] [pooled, bf16] [projection
// scratch: the intermediate and split-K partials; before the projection, the scoring's fp16
// planes of queries and keys, dead once the scores are written]
Layout layout(const umem_desc* d, int32_t T) {
  Layout L{};
  const size_t th = static_cast<size_t>(T) * d->heads;
  size_t off = 0;
  L.factors = off;
  if (d->grid == UMEM_GRID_TUCKER) off += round_up(kFactorBytes);
  L.sel = off;
  off += round_up(2 * th * d->n_keys * sizeof(float));
  L.idx = off;
  off += round_up(th * d->topm * sizeof(int32_t));
  L.w = off;
  off += round_up(th * d->topm * n_cores(*d) * sizeof(float));
  L.pooled = off;
  if (d->dv_virt > 0 || d->d_out > 0)
    off += round_up(static_cast<size_t>(T) * d->expand * d->dv * sizeof(uint16_t));
  L.proj = off;
  const size_t proj = (d->dv_virt > 0 || d->d_out > 0)
                          ? project_workspace_bytes(T, d->expand, d->dv, d->dv_virt, d->d_out) : 0;
  off += round_up(std::max(proj, score_planes_bytes(*d, T)));
  L.total = off;
  return L;
}

umem_status check_ws(const umem_desc* d, int32_t T, const void* ws, size_t ws_bytes) {
  const Layout L = layout(d, T);
  if (L.total > 0 && (ws == nullptr || !aligned(ws, kAlign) || ws_bytes < L.total))
    return UMEM_ERR_WORKSPACE;
  return UMEM_OK;
}

umem_status hip_status(hipError_t e) { return e == hipSuccess ? UMEM_OK : UMEM_ERR_HIP; }

umem_status check_gather(int64_t n_values, int32_t dv, int32_t vdtype, const void* values,
                         int32_t T, int32_t bag, const int32_t* idx, const float* w,
                         int32_t expand, int32_t cores, const float* out) {
  if (n_values < 1 || dv < 1 || bag < 1 || expand < 1 || cores < 0) return UMEM_ERR_INVALID_ARG;
  if (cores > 1 && dv % cores != 0) return UMEM_ERR_INVALID_ARG;
  if (vdtype != UMEM_F32 && vdtype != UMEM_BF16) return UMEM_ERR_INVALID_ARG;
  umem_status st = check_tokens(T);
  if (st != UMEM_OK || T == 0) return st;
  if (!values || !idx || !w || !out) return UMEM_ERR_INVALID_ARG;
  if (!aligned(values, 16) || !aligned(out, 16) || !aligned(idx, 4) || !aligned(w, 4))
    return UMEM_ERR_INVALID_ARG;
  const int64_t esize = vdtype == UMEM_F32 ? 4 : 2;
  if (n_values > (INT64_C(1) << 62) / (static_cast<int64_t>(dv) * esize)) return UMEM_ERR_INVALID_ARG;
  if (n_values * expand > (INT64_C(1) << 31)) return UMEM_ERR_UNSUPPORTED;
  if (bag > kMaxBag || expand > kMaxExpand) return UMEM_ERR_UNSUPPORTED;
  if (!gather_row_supported(dv, vdtype)) return UMEM_ERR_UNSUPPORTED;
  if (cores > 1 && !cores_supported(dv, vdtype, cores)) return UMEM_ERR_UNSUPPORTED;
  return UMEM_OK;
}

// The shape of a projection: w_proj given iff dv_virt > 0 (else the output linear alone, which
// needs expand == 1 and d_out > 0); w_out given iff d_out > 0.
umem_status check_project_shape(int32_t expand, int32_t dv, int32_t dv_virt, int32_t d_out,
                                bool has_proj, bool has_out) {
  if (expand < 1 || dv < 1 || dv_virt < 0 || d_out < 0) return UMEM_ERR_INVALID_ARG;
  if (has_proj != (dv_virt > 0) || has_out != (d_out > 0)) return UMEM_ERR_INVALID_ARG;
  if (!has_proj && (expand != 1 || d_out == 0)) return UMEM_ERR_INVALID_ARG;
  // the GEMMs read 16-byte pieces of rows of K: 4 fp32 of a pooled row, 8 bf16 of a weight row
  const int64_t k1 = static_cast<int64_t>(expand) * dv;
  if (k1 % 8 != 0 || dv_virt % 8 != 0 || d_out % 8 != 0) return UMEM_ERR_UNSUPPORTED;
  if (has_proj ? !gemm_weight_supported(dv_virt, k1) || (has_out && !gemm_weight_supported(d_out, dv_virt))
               : !gemm_weight_supported(d_out, dv))
    return UMEM_ERR_UNSUPPORTED;
  return UMEM_OK;
}

umem_status check_project(int32_t T, int32_t expand, int32_t dv, int32_t dv_virt, int32_t d_out,
                          const float* pooled, const uint16_t* w_proj, const uint16_t* w_out,
                          const float* out, const void* ws, size_t ws_bytes) {
  umem_status st = check_project_shape(expand, dv, dv_virt, d_out, w_proj != nullptr, w_out != nullptr);
  if (st == UMEM_OK) st = check_tokens(T);
  if (st != UMEM_OK || T == 0) return st;
  if (!pooled || !out) return UMEM_ERR_INVALID_ARG;
  const size_t need = project_workspace_bytes(T, expand, dv, dv_virt, d_out);
  if (need > 0 && (ws == nullptr || !aligned(ws, 16) || ws_bytes < need)) return UMEM_ERR_WORKSPACE;
  if (!aligned(pooled, 16) || !aligned(w_proj, 16) || !aligned(w_out, 16)) return UMEM_ERR_UNSUPPORTED;
  return UMEM_OK;
}

hipError_t run_project(int32_t T, int32_t expand, int32_t dv, int32_t dv_virt, int32_t d_out,
                       const float* pooled, const uint16_t* w_proj, const uint16_t* w_out,
                       float* out, void* ws, hipStream_t s) {
  return launch_project(T, expand, dv, dv_virt, d_out, pooled, w_proj, w_out, out, ws, s);
}

}  // namespace

extern "C" {

UMEM_API umem_status umem_workspace_size(const umem_desc* desc, int32_t T, size_t* bytes) {
  if (bytes == nullptr) return UMEM_ERR_INVALID_ARG;
  *bytes = 0;
  umem_status st = check_desc(desc);
  if (st == UMEM_OK) st = check_tokens(T);
  if (st != UMEM_OK) return st;
  *bytes = layout(desc, T).total;
  return UMEM_OK;
}

UMEM_API umem_status umem_axis_scores(const umem_desc* desc, int32_t T, const float* q_row,
                                      const float* q_col, const float* k_row, const float* k_col,
                                      const float* core, float* sel, void* ws, size_t ws_bytes,
                                      hipStream_t stream) {
  umem_status st = check_desc(desc);
  if (st == UMEM_OK) st = check_tokens(T);
  if (st != UMEM_OK || T == 0) return st;
  if (st == UMEM_OK) st = check_scoring_ptrs(desc, q_row, q_col, k_row, k_col, core);
  if (st == UMEM_OK && (sel == nullptr || !aligned(sel, 4))) st = UMEM_ERR_INVALID_ARG;
  const bool tucker = desc->grid == UMEM_GRID_TUCKER;
  // [factors (Tucker)] [fp16 planes of the many-token path]
  const size_t planes_at = tucker ? round_up(kFactorBytes) : 0;
  const size_t planes = score_planes_bytes(*desc, T);
  const size_t need = planes > 0 ? planes_at + planes : (tucker ? kFactorBytes : 0);
  if (st == UMEM_OK && need > 0 && (ws == nullptr || !aligned(ws, kAlign) || ws_bytes < need))
    st = UMEM_ERR_WORKSPACE;
  if (st != UMEM_OK) return st;
  float* factors = tucker ? static_cast<float*>(ws) : nullptr;
  hipError_t e = tucker ? launch_rank1(*desc, core, factors, stream) : hipSuccess;
  if (e == hipSuccess)
    e = launch_axis_scores(*desc, T, q_row, q_col, k_row, k_col, factors, sel, nullptr, 0,
                           planes > 0 ? static_cast<char*>(ws) + planes_at : nullptr, stream);
  return hip_status(e);
}

UMEM_API umem_status umem_select(const umem_desc* desc, int32_t T, const float* sel,
                                 const float* q_row, const float* q_col, const float* k_row,
                                 const float* k_col, const float* core, int32_t* idx, float* w,
                                 int32_t* axis_idx, const void* values, float* pooled,
                                 hipStream_t stream) {
  umem_status st = check_desc(desc);
  if (st == UMEM_OK) st = check_tokens(T);
  if (st != UMEM_OK || T == 0) return st;
  if (st == UMEM_OK && desc->grid == UMEM_GRID_TUCKER)
    st = check_scoring_ptrs(desc, q_row, q_col, k_row, k_col, core);
  if (st == UMEM_OK && (!sel || !idx || !w || !aligned(sel, 16) || !aligned(idx, 4) || !aligned(w, 4) ||
                        !aligned(axis_idx, 4)))
    st = UMEM_ERR_INVALID_ARG;
  if (st == UMEM_OK && (values == nullptr) != (pooled == nullptr)) st = UMEM_ERR_INVALID_ARG;
  if (st == UMEM_OK && pooled != nullptr) {
    if (!aligned(values, 16) || !aligned(pooled, 16)) st = UMEM_ERR_INVALID_ARG;
    else if (!select_pools(*desc)) st = UMEM_ERR_UNSUPPORTED;
  }
  if (st != UMEM_OK) return st;
  return hip_status(launch_select(*desc, T, sel, q_row, q_col, k_row, k_col, core, idx, w,
                                  axis_idx, values, pooled, stream));
}

UMEM_API umem_status umem_score_topk(const umem_desc* desc, int32_t T, const float* q_row,
                                     const float* q_col, const float* k_row, const float* k_col,
                                     const float* core, int32_t* idx, float* w, int32_t* axis_idx,
                                     void* ws, size_t ws_bytes, hipStream_t stream) {
  umem_status st = check_desc(desc);
  if (st == UMEM_OK) st = check_tokens(T);
  if (st != UMEM_OK || T == 0) return st;
  if (st == UMEM_OK) st = check_scoring_ptrs(desc, q_row, q_col, k_row, k_col, core);
  if (st == UMEM_OK && (!idx || !w || !aligned(idx, 4) || !aligned(w, 4) || !aligned(axis_idx, 4)))
    st = UMEM_ERR_INVALID_ARG;
  if (st == UMEM_OK) st = check_ws(desc, T, ws, ws_bytes);
  if (st != UMEM_OK) return st;
  const Layout L = layout(desc, T);
  float* sel = reinterpret_cast<float*>(static_cast<char*>(ws) + L.sel);
  float* factors = reinterpret_cast<float*>(static_cast<char*>(ws) + L.factors);
  const bool tucker = desc->grid == UMEM_GRID_TUCKER;
  hipError_t e = tucker ? launch_rank1(*desc, core, factors, stream) : hipSuccess;
  if (e == hipSuccess)
    e = launch_axis_scores(*desc, T, q_row, q_col, k_row, k_col, tucker ? factors : nullptr, sel,
                           nullptr, 0, static_cast<char*>(ws) + L.proj, stream);
  if (e == hipSuccess)
    e = launch_select(*desc, T, sel, q_row, q_col, k_row, k_col, core, idx, w, axis_idx, nullptr,
                      nullptr, stream);
  return hip_status(e);
}

UMEM_API umem_status umem_gather_sum(int64_t n_values, int32_t dv, int32_t vdtype,
                                     const void* values, int32_t T, int32_t bag,
                                     const int32_t* idx, const float* w, const int32_t* perm,
                                     int32_t expand, int32_t cores, float* out,
                                     hipStream_t stream) {
  umem_status st = check_gather(n_values, dv, vdtype, values, T, bag, idx, w, expand, cores, out);
  if (st != UMEM_OK || T == 0) return st;
  if (st == UMEM_OK && perm != nullptr && !aligned(perm, 4)) st = UMEM_ERR_INVALID_ARG;
  if (st != UMEM_OK) return st;
  return hip_status(launch_gather(n_values, dv, vdtype, values, T, bag, idx, w, perm, expand,
                                  cores > 1 ? cores : 1, out, stream));
}

UMEM_API umem_status umem_project_workspace_size(int32_t T, int32_t expand, int32_t dv,
                                                 int32_t dv_virt, int32_t d_out, size_t* bytes) {
  if (bytes == nullptr) return UMEM_ERR_INVALID_ARG;
  *bytes = 0;
  // the output linear alone has dv_virt == 0; with dv_virt > 0 the projector is given
  umem_status st = check_project_shape(expand, dv, dv_virt, d_out, dv_virt > 0, d_out > 0);
  if (st == UMEM_OK) st = check_tokens(T);
  if (st != UMEM_OK) return st;
  *bytes = project_workspace_bytes(T, expand, dv, dv_virt, d_out);
  return UMEM_OK;
}

UMEM_API umem_status umem_project(int32_t T, int32_t expand, int32_t dv, int32_t dv_virt,
                                  int32_t d_out, const float* pooled, const uint16_t* w_proj,
                                  const uint16_t* w_out, float* out, void* ws, size_t ws_bytes,
                                  hipStream_t stream) {
  umem_status st = check_project(T, expand, dv, dv_virt, d_out, pooled, w_proj, w_out, out, ws,
                                 ws_bytes);
  if (st != UMEM_OK || T == 0) return st;
  return hip_status(run_project(T, expand, dv, dv_virt, d_out, pooled, w_proj, w_out, out, ws, stream));
}

}  // extern "C"

namespace {

umem_status check_query_desc(const umem_query_desc* qd) {
  if (qd == nullptr) return UMEM_ERR_INVALID_ARG;
  if (qd->d_model < 1 || qd->conv_k < 1 || qd->heads < 1 || qd->dk < 1) return UMEM_ERR_INVALID_ARG;
  if ((qd->shared != 0 && qd->shared != 1) || !(qd->eps >= 0.0f) || qd->eps == INFINITY)
    return UMEM_ERR_INVALID_ARG;
  const int64_t nq = static_cast<int64_t>(qd->shared ? 1 : 2) * qd->heads * qd->dk;
  if (qd->d_model % 8 != 0 || qd->conv_k > 8 || qd->dk > 1024 || nq % 8 != 0 || nq > (1 << 24) ||
      !gemm_weight_supported(nq, qd->d_model))
    return UMEM_ERR_UNSUPPORTED;
  return UMEM_OK;
}

umem_status check_query_tokens(int32_t B, int32_t L) {
  if (B < 0 || L < 0) return UMEM_ERR_INVALID_ARG;
  if (static_cast<int64_t>(B) * L > kMaxTokens) return UMEM_ERR_UNSUPPORTED;
  return UMEM_OK;
}

}  // namespace

extern "C" {

UMEM_API umem_status umem_query_workspace_size(const umem_query_desc* qd, int32_t B, int32_t L,
                                               size_t* bytes) {
  if (bytes == nullptr) return UMEM_ERR_INVALID_ARG;
  *bytes = 0;
  umem_status st = check_query_desc(qd);
  if (st == UMEM_OK) st = check_query_tokens(B, L);
  if (st != UMEM_OK) return st;
  *bytes = query_workspace_bytes(*qd, static_cast<int64_t>(B) * L);
  return UMEM_OK;
}

UMEM_API umem_status umem_query(const umem_query_desc* qd, int32_t B, int32_t L, const float* x,
                                const float* x_hist, const float* conv_w, const uint16_t* w_q,
                                const float* gamma, const float* beta, float* q_row, float* q_col,
                                void* ws, size_t ws_bytes, hipStream_t stream) {
  umem_status st = check_query_desc(qd);
  if (st == UMEM_OK) st = check_query_tokens(B, L);
  if (st != UMEM_OK) return st;
  if (static_cast<int64_t>(B) * L == 0) return UMEM_OK;
  if (!x || !conv_w || !w_q || !gamma || !beta || !q_row) return UMEM_ERR_INVALID_ARG;
  if ((q_col == nullptr) != (qd->shared == 1)) return UMEM_ERR_INVALID_ARG;
  if (!aligned(x, 16) || !aligned(x_hist, 16) || !aligned(conv_w, 16) || !aligned(w_q, 16))
    return UMEM_ERR_INVALID_ARG;
  if (!aligned(gamma, 4) || !aligned(beta, 4) || !aligned(q_row, 4) || !aligned(q_col, 4))
    return UMEM_ERR_INVALID_ARG;
  const size_t need = query_workspace_bytes(*qd, static_cast<int64_t>(B) * L);
  if (ws == nullptr || !aligned(ws, 16) || ws_bytes < need) return UMEM_ERR_WORKSPACE;
  return hip_status(launch_query(*qd, B, L, x, x_hist, conv_w, w_q, gamma, beta, q_row, q_col, ws,
                                 stream));
}

UMEM_API umem_status umem_key_norm(int32_t heads, int32_t n, int32_t dk, const float* keys,
                                   const float* gamma, const float* beta, float eps, float* out,
                                   hipStream_t stream) {
  if (heads < 1 || n < 1 || dk < 1 || !(eps >= 0.0f) || eps == INFINITY) return UMEM_ERR_INVALID_ARG;
  if (!keys || !gamma || !beta || !out) return UMEM_ERR_INVALID_ARG;
  if (!aligned(keys, 4) || !aligned(gamma, 4) || !aligned(beta, 4) || !aligned(out, 4))
    return UMEM_ERR_INVALID_ARG;
  if (dk > 1024 || static_cast<int64_t>(heads) * n > (INT64_C(1) << 31)) return UMEM_ERR_UNSUPPORTED;
  return hip_status(launch_key_norm(heads, n, dk, keys, gamma, beta, eps, out, stream));
}

constexpr int64_t kMaxBackwardEntries = INT64_C(1) << 22;   // pairs the backward sorts at once

UMEM_API umem_status umem_gather_backward_workspace_size(int32_t T, int32_t bag, int32_t dv,
                                                         size_t* bytes) {
  if (bytes == nullptr) return UMEM_ERR_INVALID_ARG;
  *bytes = 0;
  if (T < 0 || bag < 1 || dv < 1) return UMEM_ERR_INVALID_ARG;
  if (static_cast<int64_t>(T) * bag > kMaxBackwardEntries) return UMEM_ERR_UNSUPPORTED;
  *bytes = gather_backward_workspace_bytes(T, bag, dv);
  return UMEM_OK;
}

UMEM_API umem_status umem_gather_backward(int64_t n_values, int32_t dv, int32_t vdtype,
                                          const void* values, int32_t T, int32_t bag,
                                          const int32_t* idx, const float* w, const int32_t* perm,
                                          int32_t expand, int32_t cores, const float* d_pooled,
                                          float* d_values, float* dw, void* ws, size_t ws_bytes,
                                          hipStream_t stream) {
  umem_status st = check_gather(n_values, dv, vdtype, values, T, bag, idx, w, expand, cores, d_values);
  if (st != UMEM_OK || T == 0) return st;
  if (!d_pooled || !dw || !aligned(d_pooled, 16) || !aligned(dw, 4)) return UMEM_ERR_INVALID_ARG;
  if ((expand > 1) != (perm != nullptr) || !aligned(perm, 4)) return UMEM_ERR_INVALID_ARG;
  if (static_cast<int64_t>(T) * bag > kMaxBackwardEntries) return UMEM_ERR_UNSUPPORTED;
  const size_t need = gather_backward_workspace_bytes(T, bag, dv);
  if (ws == nullptr || !aligned(ws, 16) || ws_bytes < need) return UMEM_ERR_WORKSPACE;
  return hip_status(launch_gather_backward(n_values, dv, vdtype, values, T, bag, idx, w, perm,
                                           expand, cores, d_pooled, d_values, dw, nullptr, nullptr,
                                           ws, stream));
}

UMEM_API umem_status umem_gather_backward_rows(int64_t n_values, int32_t dv, int32_t vdtype,
                                               const void* values, int32_t T, int32_t bag,
                                               const int32_t* idx, const float* w,
                                               const int32_t* perm, int32_t expand, int32_t cores,
                                               const float* d_pooled, int32_t* rows, float* d_rows,
                                               int32_t* n_rows, float* dw, void* ws,
                                               size_t ws_bytes, hipStream_t stream) {
  umem_status st = check_gather(n_values, dv, vdtype, values, T, bag, idx, w, expand, cores, d_rows);
  if (st != UMEM_OK || T == 0) return st;
  if (!rows || !n_rows || !aligned(rows, 4) || !aligned(n_rows, 4)) return UMEM_ERR_INVALID_ARG;
  if (!d_pooled || !dw || !aligned(d_pooled, 16) || !aligned(dw, 4)) return UMEM_ERR_INVALID_ARG;
  if ((expand > 1) != (perm != nullptr) || !aligned(perm, 4)) return UMEM_ERR_INVALID_ARG;
  if (static_cast<int64_t>(T) * bag > kMaxBackwardEntries) return UMEM_ERR_UNSUPPORTED;
  const size_t need = gather_backward_workspace_bytes(T, bag, dv);
  if (ws == nullptr || !aligned(ws, 16) || ws_bytes < need) return UMEM_ERR_WORKSPACE;
  return hip_status(launch_gather_backward(n_values, dv, vdtype, values, T, bag, idx, w, perm,
                                           expand, cores, d_pooled, d_rows, dw, rows, n_rows, ws,
                                           stream));
}

UMEM_API umem_status umem_score_backward_workspace_size(const umem_desc* desc, int32_t T,
                                                        size_t* bytes) {
  if (bytes == nullptr) return UMEM_ERR_INVALID_ARG;
  *bytes = 0;
  umem_status st = check_desc(desc);
  if (st == UMEM_OK) st = check_tokens(T);
  if (st != UMEM_OK) return st;
  if (static_cast<int64_t>(T) * desc->heads * 2 * desc->topm > kMaxBackwardEntries)
    return UMEM_ERR_UNSUPPORTED;
  *bytes = score_backward_workspace_bytes(*desc, T);
  return UMEM_OK;
}

UMEM_API umem_status umem_score_backward(const umem_desc* desc, int32_t T, const float* q_row,
                                         const float* q_col, const float* k_row,
                                         const float* k_col, const float* core,
                                         const int32_t* idx, const float* w, const float* dw,
                                         float* dq_row, float* dq_col, float* dk_row,
                                         float* dk_col, float* dcore, void* ws, size_t ws_bytes,
                                         hipStream_t stream) {
  umem_status st = check_desc(desc);
  if (st == UMEM_OK) st = check_tokens(T);
  if (st != UMEM_OK || T == 0) return st;
  st = check_scoring_ptrs(desc, q_row, q_col, k_row, k_col, core);
  if (st != UMEM_OK) return st;
  const bool softmax = desc->weight == UMEM_W_SOFTMAX;
  if (!idx || !dw || (softmax && !w)) return UMEM_ERR_INVALID_ARG;
  if (!aligned(idx, 4) || !aligned(dw, 4) || !aligned(w, 4)) return UMEM_ERR_INVALID_ARG;
  if (!dq_row || !dq_col || !dk_row || !dk_col) return UMEM_ERR_INVALID_ARG;
  if (!aligned(dq_row, 4) || !aligned(dq_col, 4) || !aligned(dk_row, 16) || !aligned(dk_col, 16))
    return UMEM_ERR_INVALID_ARG;
  if ((desc->grid == UMEM_GRID_TUCKER) != (dcore != nullptr) || !aligned(dcore, 4))
    return UMEM_ERR_INVALID_ARG;
  if (static_cast<int64_t>(T) * desc->heads * 2 * desc->topm > kMaxBackwardEntries)
    return UMEM_ERR_UNSUPPORTED;
  const size_t need = score_backward_workspace_bytes(*desc, T);
  if (ws == nullptr || !aligned(ws, 16) || ws_bytes < need) return UMEM_ERR_WORKSPACE;
  return hip_status(launch_score_backward(*desc, T, q_row, q_col, k_row, k_col, core, idx, w, dw,
                                          dq_row, dq_col, dk_row, dk_col, dcore, ws, stream));
}

}  // extern "C"

namespace {

umem_status forward_into(const umem_desc* desc, int32_t T, const float* q_row, const float* q_col,
                         const float* k_row, const float* k_col, const float* core,
                         const void* values, const int32_t* perm, const uint16_t* w_proj,
                         const uint16_t* w_out, float* out, int32_t* idx_out, float* w_out_scores,
                         void* ws, size_t ws_bytes, hipStream_t stream) {
  umem_status st = check_desc(desc);
  if (st == UMEM_OK) st = check_tokens(T);
  if (st != UMEM_OK || T == 0) return st;
  if (st == UMEM_OK) st = check_scoring_ptrs(desc, q_row, q_col, k_row, k_col, core);
  if (st == UMEM_OK) st = check_ws(desc, T, ws, ws_bytes);
  if (st != UMEM_OK) return st;
  const bool project = desc->dv_virt > 0 || desc->d_out > 0;
  if ((desc->expand > 1) != (perm != nullptr)) return UMEM_ERR_INVALID_ARG;
  if ((desc->dv_virt > 0) != (w_proj != nullptr) || (desc->d_out > 0) != (w_out != nullptr))
    return UMEM_ERR_INVALID_ARG;
  if (!aligned(idx_out, 4) || !aligned(w_out_scores, 4) || !aligned(perm, 4))
    return UMEM_ERR_INVALID_ARG;
  if (!aligned(w_proj, 16) || !aligned(w_out, 16)) return UMEM_ERR_UNSUPPORTED;
  const int bag = desc->heads * desc->topm;
  const Layout L = layout(desc, T);
  char* base = static_cast<char*>(ws);
  float* sel = reinterpret_cast<float*>(base + L.sel);
  int32_t* idx = idx_out ? idx_out : reinterpret_cast<int32_t*>(base + L.idx);
  float* w = w_out_scores ? w_out_scores : reinterpret_cast<float*>(base + L.w);
  // with a projection the pooled rows go to the workspace in bf16, as its GEMM takes them
  uint16_t* pooled = reinterpret_cast<uint16_t*>(base + L.pooled);
  st = check_gather(desc->n_values, desc->dv, desc->vdtype, values, T, bag, idx, w, desc->expand,
                    n_cores(*desc), out);
  if (st != UMEM_OK) return st;

  float* factors = reinterpret_cast<float*>(base + L.factors);
  const bool tucker = desc->grid == UMEM_GRID_TUCKER;
  hipError_t e = tucker ? launch_rank1(*desc, core, factors, stream) : hipSuccess;
  // For decode-sized batches without expansion or projection the selection pools the rows
  // itself (scoring clears out first); otherwise the gather kernel, with more rows in flight per
  // CU, pools them after it.
  const bool fused = !project && select_pools(*desc) && T <= kMaxPoolTokens;
  if (e == hipSuccess)
    e = launch_axis_scores(*desc, T, q_row, q_col, k_row, k_col, tucker ? factors : nullptr, sel,
                           fused ? out : nullptr, static_cast<size_t>(T) * desc->dv,
                           base + L.proj, stream);
  if (e == hipSuccess)
    e = launch_select(*desc, T, sel, q_row, q_col, k_row, k_col, core, idx, w, nullptr,
                      fused ? values : nullptr, fused ? out : nullptr, stream);
  if (e == hipSuccess && !fused && !project)
    e = launch_gather(desc->n_values, desc->dv, desc->vdtype, values, T, bag, idx, w, perm,
                      desc->expand, n_cores(*desc), out, stream);
  if (e == hipSuccess && project)
    e = launch_gather_bf16(desc->n_values, desc->dv, desc->vdtype, values, T, bag, idx, w, perm,
                           desc->expand, n_cores(*desc), pooled, stream);
  if (e == hipSuccess && project)
    e = launch_project(T, desc->expand, desc->dv, desc->dv_virt, desc->d_out, pooled, w_proj,
                       w_out, out, base + L.proj, stream);
  return hip_status(e);
}

// The scratch of umem_forward_noalloc: one array in each GPU's memory, loaded with the library's
// code and held until the process ends.  Host code must not pass its name to a kernel (on the
// host it is only a stand-in for the device symbol); the device address of each GPU's copy is
// looked up once per device and kept in static_scratch_ptr.
static __device__ __align__(256) unsigned char scratch[UMEM_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::once_flag scratch_once[kMaxDevices];
void* scratch_ptr[kMaxDevices];
hipError_t scratch_err[kMaxDevices];

// The address of the current device's copy of `scratch` (its first call on a device looks it
// up, with that device current).
hipError_t static_scratch_ptr(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::call_once(scratch_once[dev], [dev] {
    void* p = nullptr;
    const hipError_t r = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    scratch_err[dev] = r;
    scratch_ptr[dev] = r == hipSuccess ? p : nullptr;
  });
  *ptr = scratch_ptr[dev];
  return scratch_err[dev];
}

}  // namespace

extern "C" {

UMEM_API umem_status umem_forward(const umem_desc* desc, int32_t T, const float* q_row,
                                  const float* q_col, const float* k_row, const float* k_col,
                                  const float* core, const void* values, const int32_t* perm,
                                  const uint16_t* w_proj, const uint16_t* w_out, float* out,
                                  int32_t* idx_out, float* w_out_scores, void* ws,
                                  size_t ws_bytes, hipStream_t stream) {
  return forward_into(desc, T, q_row, q_col, k_row, k_col, core, values, perm, w_proj, w_out, out,
                      idx_out, w_out_scores, ws, ws_bytes, stream);
}

UMEM_API umem_status umem_forward_noalloc(const umem_desc* desc, int32_t T, const float* q_row,
                                          const float* q_col, const float* k_row,
                                          const float* k_col, const float* core,
                                          const void* values, const int32_t* perm,
                                          const uint16_t* w_proj, const uint16_t* w_out,
                                          float* out, int32_t* idx_out, float* w_out_scores,
                                          hipStream_t stream) {
  umem_status st = check_desc(desc);
  if (st == UMEM_OK) st = check_tokens(T);
  if (st != UMEM_OK || T == 0) return st;
  // no kernel of the forward needs its scratch cleared beforehand: every part is written before
  // it is read, so the contents a previous call left behind do not matter
  if (layout(desc, T).total > UMEM_STATIC_SCRATCH_BYTES) return UMEM_ERR_SCRATCH_LIMIT;
  st = check_scoring_ptrs(desc, q_row, q_col, k_row, k_col, core);
  if (st != UMEM_OK) return st;
  void* ws = nullptr;
  if (static_scratch_ptr(&ws) != hipSuccess) return UMEM_ERR_HIP;
  return forward_into(desc, T, q_row, q_col, k_row, k_col, core, values, perm, w_proj, w_out, out,
                      idx_out, w_out_scores, ws, UMEM_STATIC_SCRATCH_BYTES, stream);
}

UMEM_API const char* umem_status_string(umem_status status) {
  switch (status) {
    case UMEM_OK: return "ok";
    case UMEM_ERR_INVALID_ARG: return "invalid argument";
    case UMEM_ERR_UNSUPPORTED: return "unsupported by this library";
    case UMEM_ERR_WORKSPACE: return "workspace too small or misaligned";
    case UMEM_ERR_HIP: return "HIP launch error";
    case UMEM_ERR_SCRATCH_LIMIT: return "needs more scratch than the static buffer holds";
  }
  return "unknown status";
}

}  // extern "C"
