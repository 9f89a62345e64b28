// Internal declarations and device helpers of libumem (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "umem.h"

namespace umem {

constexpr int kWave = 64;            // CDNA wavefront width
constexpr int kMaxSelect = 8192;     // max(n, k*k): one selection's keys in 32 KiB of LDS
constexpr int kMaxTopK = 90;         // k*k <= kMaxSelect
constexpr int kMaxTopKTucker = 64;   // Tucker: the k*k candidate keys in 16 KiB of LDS
constexpr int kMaxTopM = 256;
constexpr int kMaxCores = 8;          // multi-core scoring: component cores per head
constexpr int kMaxPoolTopM = 64;      // the selection kernel pools rows itself up to this topm
constexpr int kMaxPoolTokens = 128;   // ... and umem_forward lets it up to this many tokens
constexpr int kMaxRank = 4;
constexpr int kMaxBag = 2048;
constexpr int kMaxTokens = 1 << 20;
constexpr int kMaxHeads = 64;
constexpr int kMaxExpand = 64;
constexpr int kMaxDk = 1024;
constexpr size_t kFactorBytes = static_cast<size_t>(kMaxHeads) * 2 * 4 * sizeof(float);

bool gather_row_supported(int dv, int vdtype);
size_t select_lds_bytes(int n_cand, int tucker, int pool_dv);
int additive_candidates(int k, int m);
constexpr int kMaxRowBytes = 8192;

// ---------------------------------------------------------------- host-side launchers

// Tucker grid: leading singular pair of every head's core, factors[h][0] = u, factors[h][1] = t,
// each padded to kMaxRank floats.
// Launchers report hipGetLastError() after their launches; an error that an earlier, unrelated
// HIP call left in the calling thread is cleared first, so that it is not taken for theirs.
inline void clear_stale_error() { (void)hipGetLastError(); }

hipError_t launch_rank1(const umem_desc& d, const float* core, float* factors, hipStream_t s);

// Selection scores; factors is the output of launch_rank1 (Tucker) or NULL (additive).  With
// zero_out set the same grid also clears zero_out[0, zero_floats) (a multiple of 4 floats).
// Scratch of the many-token scoring path (fp16 planes of queries and keys and their rows'
// exponents), or 0 where the shape takes another kernel; launch_axis_scores needs it as planes
// then.
size_t score_planes_bytes(const umem_desc& d, int T);
hipError_t launch_axis_scores(const umem_desc& d, int T, const float* q_row, const float* q_col,
                              const float* k_row, const float* k_col, const float* factors,
                              float* sel, float* zero_out, size_t zero_floats, void* planes,
                              hipStream_t s);

// Per-axis top-k, grid, top-m and weights.  With pooled set (only where select_pools(d)), each
// (token, head) workgroup also pools its m value rows into pooled[t, :] with atomic adds, which
// must start from zero (launch_axis_scores clears it).
hipError_t launch_select(const umem_desc& d, int T, const float* sel, const float* q_row,
                         const float* q_col, const float* k_row, const float* k_col,
                         const float* core, int32_t* idx, float* w, int32_t* axis_idx,
                         const void* values, float* pooled, hipStream_t s);

// Whether the selection kernel can pool the rows itself: no expansion, at most two heads (two
// atomic adds onto zero give the same bits in either order), topm <= 64 and rows of 1 or 2 KiB.
bool select_pools(const umem_desc& d);

// cores: 1, or the h of multi-core scoring (w is then [T, bag, h]; column slice i takes w[.., i]).
hipError_t launch_gather(int64_t n_values, int dv, int vdtype, const void* values, int T,
                         int bag, const int32_t* idx, const float* w, const int32_t* perm,
                         int expand, int cores, float* out, hipStream_t s);
// The same with the pooled rows rounded to bf16 (nearest even) as they are stored, for the
// projection, whose GEMM rounds its A operand the same way: out [T, expand, dv] bf16 bits.
hipError_t launch_gather_bf16(int64_t n_values, int dv, int vdtype, const void* values, int T,
                              int bag, const int32_t* idx, const float* w, const int32_t* perm,
                              int expand, int cores, uint16_t* out, hipStream_t s);

// Multi-core scoring: the number of component cores of a layer (0 counts as 1), and whether
// rows of this shape can be split into h column slices (each slice whole 16-byte chunks).
inline int n_cores(const umem_desc& d) { return d.cores > 1 ? d.cores : 1; }
bool cores_supported(int dv, int vdtype, int cores);

// C [M, N] = bf16(A [M, K]) B[N, K]^T on MFMA with fp32 accumulation (A fp32, B bf16 bits stored
// output-major like a linear layer's weight, all 16-byte aligned, K % 8 == 0, N % 4 == 0);
// part: gemm_partial_bytes(M, N, K) bytes of scratch for the split-K partial sums (unused when
// that is 0).  gemm_weight_supported: B's bytes within the loads' 32-bit range, and K small
// enough that a band of 128 rows of A does too (A is launched in bands below 2 GiB).
size_t gemm_partial_bytes(int M, int N, int K);
inline bool gemm_weight_supported(int64_t N, int64_t K) {
  return N * K * 2 < (INT64_C(1) << 31) && K <= (INT64_C(1) << 20);
}
hipError_t gemm_bf16(const float* A, const uint16_t* B, float* C, int M, int N, int K, float* part,
                     hipStream_t s);
// The same with A already bf16 bits (16-byte aligned rows of K): the product is the one the fp32
// form computes from the fp32 values that round to this A.
hipError_t gemm_bf16(const uint16_t* A, const uint16_t* B, float* C, int M, int N, int K,
                     float* part, hipStream_t s);
// The same, but a GEMM split over K (in one band of rows) leaves its *splits partial products in
// part ([*splits][M][N], to be added in split order) instead of adding them into C; *splits = 1
// means C holds the product.
hipError_t gemm_bf16_parts(const uint16_t* A, const uint16_t* B, float* C, int M, int N, int K,
                           float* part, hipStream_t s, int* splits);

// Stable sort of M (key, value) pairs with keys < 2^bits (sort.hip); the inputs are reordered
// through ws (sort_workspace_bytes(M) bytes, 4-byte aligned) and the sorted arrays returned
// (either the inputs or part of ws).
size_t sort_workspace_bytes(int M);
// Exclusive prefix sums of v[0, n) in place (n <= 2^24); sums: scan_workspace_bytes(n) bytes of
// scratch for the per-chunk sums.
size_t scan_workspace_bytes(int n);
hipError_t scan_exclusive(uint32_t* v, int n, uint32_t* sums, hipStream_t s);
hipError_t sort_pairs(uint32_t* keys, uint32_t* vals, int M, int bits, void* ws, hipStream_t s,
                      uint32_t** keys_sorted, uint32_t** vals_sorted);

// Backward of the gather-sum and of the scores (backward.hip).
size_t gather_backward_workspace_bytes(int T, int bag, int dv);
hipError_t launch_gather_backward(int64_t n_values, int dv, int vdtype, const void* values, int T,
                                  int bag, const int32_t* idx, const float* w, const int32_t* perm,
                                  int expand, int cores, const float* d_pooled, float* d_values,
                                  float* dw, int32_t* rows_out, int32_t* n_rows, void* ws,
                                  hipStream_t s);
size_t score_backward_workspace_bytes(const umem_desc& d, int T);
hipError_t launch_score_backward(const umem_desc& d, int T, const float* q_row, const float* q_col,
                                 const float* k_row, const float* k_col, const float* core,
                                 const int32_t* idx, const float* w, const float* dw,
                                 float* dq_row, float* dq_col, float* dk_row, float* dk_col,
                                 float* dcore, void* ws, hipStream_t s);

// The query front-end and the key LayerNorm (query.hip).  ws: query_workspace_bytes bytes.
size_t query_workspace_bytes(const umem_query_desc& qd, int64_t T);
hipError_t launch_query(const umem_query_desc& qd, int B, int L, const float* x,
                        const float* x_hist, const float* conv_w, const uint16_t* w_q,
                        const float* gamma, const float* beta, float* q_row, float* q_col,
                        void* ws, hipStream_t s);
hipError_t launch_key_norm(int heads, int n, int dk, const float* keys, const float* gamma,
                           const float* beta, float eps, float* out, hipStream_t s);

// a8.  ws: project_workspace_bytes(...) bytes, 256-byte aligned (the intermediate and the
// split-K partials); w_proj == nullptr is the output linear alone ([T, dv] by [dv, d_out]).
size_t project_workspace_bytes(int T, int expand, int dv, int dv_virt, int d_out);
hipError_t launch_project(int T, int expand, int dv, int dv_virt, int d_out, const float* pooled,
                          const uint16_t* w_proj, const uint16_t* w_out, float* out, void* ws,
                          hipStream_t s);
// The same from pooled rows already rounded to bf16 (launch_gather_bf16): the same result.
hipError_t launch_project(int T, int expand, int dv, int dv_virt, int d_out, const uint16_t* pooled,
                          const uint16_t* w_proj, const uint16_t* w_out, float* out, void* ws,
                          hipStream_t s);

// ---------------------------------------------------------------- device helpers

// Monotone map of a float to an unsigned key: larger float -> larger key.  -0.0 maps like +0.0
// and NaN maps to 0, below every number including -inf.
__device__ __forceinline__ uint32_t order_key(float x) {
  if (x != x) return 0u;
  uint32_t u = __float_as_uint(x);
  if ((u << 1) == 0u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ int wave_inclusive_scan(int v) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    int y = __shfl_up(v, off, kWave);
    if (lane >= off) v += y;
  }
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & (kWave - 1);
  return (lane == 0) ? 0ull : (~0ull >> (kWave - lane));
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// fp32 -> bf16, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Leading singular pair (u, t) of an r x r core (r <= 4), in fp64: cyclic Jacobi on the
// symmetric C^T C (padded with zeros to 4 x 4), t1 = its leading eigenvector, u = C t1 / |C t1|,
// then the sign fixed so that u's largest-magnitude component (lowest index among equals) is
// positive, and t = C^T u / sigma_1.  Writes u and t to u_out[0, r) and t_out[0, r).
// Single-thread routine; all indexing is static.
__device__ inline void rank1_factors(const float* C, int r, int parts, float* u_out, float* t_out) {
  double c[4][4];      // the core: the sum, in fp64, of its `parts` component cores [parts][r][r]
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      double x = 0.0;
      if (i < r && j < r)
        for (int p = 0; p < parts; ++p) x += static_cast<double>(C[(p * r + i) * r + j]);
      c[i][j] = x;
    }
  double m[4][4], v[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      double acc = 0.0;
#pragma unroll
      for (int k = 0; k < 4; ++k) acc += c[k][i] * c[k][j];
      m[i][j] = acc;
      v[i][j] = (i == j) ? 1.0 : 0.0;
    }
  // A rotation is skipped once its off-diagonal element is below 2^-60 of both diagonal
  // elements (it would move them by less than their last bit); the sweeps end when one skips all
  // six.  An exact zero (the padding, a zero column of C) is always skipped.
  for (int sweep = 0; sweep < 12; ++sweep) {
    bool rotated = false;
#pragma unroll
    for (int p = 0; p < 3; ++p)
#pragma unroll
      for (int q = p + 1; q < 4; ++q) {
        const double apq = m[p][q];
        if (fabs(apq) <= 1e-300 || fabs(apq) <= 0x1p-60 * fmin(fabs(m[p][p]), fabs(m[q][q]))) continue;
        rotated = true;
        const double theta = (m[q][q] - m[p][p]) / (2.0 * apq);
        const double tt = (theta >= 0.0 ? 1.0 : -1.0) / (fabs(theta) + sqrt(theta * theta + 1.0));
        const double cs = 1.0 / sqrt(tt * tt + 1.0);
        const double sn = tt * cs;
        // m <- J^T m J with J the (p, q) rotation; v <- v J
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const double mkp = m[k][p], mkq = m[k][q];
          m[k][p] = cs * mkp - sn * mkq;
          m[k][q] = sn * mkp + cs * mkq;
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const double mpk = m[p][k], mqk = m[q][k];
          m[p][k] = cs * mpk - sn * mqk;
          m[q][k] = sn * mpk + cs * mqk;
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const double vkp = v[k][p], vkq = v[k][q];
          v[k][p] = cs * vkp - sn * vkq;
          v[k][q] = sn * vkp + cs * vkq;
        }
      }
    if (!rotated) break;
  }
  int best = 0;
  double lam = m[0][0];
#pragma unroll
  for (int j = 1; j < 4; ++j)
    if (m[j][j] > lam) { lam = m[j][j]; best = j; }
  double t1[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    double x = v[i][0];
#pragma unroll
    for (int j = 1; j < 4; ++j) x = (j == best) ? v[i][j] : x;
    t1[i] = x;
  }
  double u[4], nu = 0.0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    double acc = 0.0;
#pragma unroll
    for (int k = 0; k < 4; ++k) acc += c[i][k] * t1[k];
    u[i] = acc;
    nu += acc * acc;
  }
  const double sigma = sqrt(nu);
  int jmax = 0;
  double amax = fabs(u[0]);
#pragma unroll
  for (int i = 1; i < 4; ++i)
    if (fabs(u[i]) > amax) { amax = fabs(u[i]); jmax = i; }
  double sgn = 1.0;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (i == jmax && u[i] < 0.0) sgn = -1.0;
#pragma unroll
  for (int i = 0; i < 4; ++i) u[i] = sgn * u[i] / sigma;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    double acc = 0.0;
#pragma unroll
    for (int k = 0; k < 4; ++k) acc += c[k][i] * u[k];
    if (i < r) {
      u_out[i] = static_cast<float>(u[i]);
      t_out[i] = static_cast<float>(acc / sigma);
    }
  }
}

}  // namespace umem
