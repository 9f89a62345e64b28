// a1 + a2: per-axis selection scores.
//
// For head h and axis (row or column), S_rho[t, i] = sum_{d in slice rho} K[h, i, d] q[t, h, d]
// (eq. (2); with rank r the key/query dim holds r contiguous slices, eq. (4)).  The selection
// score is sum_rho f[rho] S_rho[t, i] with f = u (rows) or t (columns), the leading singular pair
// of the head's Tucker core (eqs. (6), (8), (9)); for the additive grid f = [1].
//
// Tiling: one workgroup computes a TT x TN block (tokens x keys) of one (head, axis), streaming
// the key and query tiles through LDS in chunks of DC dims.  Each key is read from HBM once per
// token tile; at decode (T <= TT) once in total.
#include "umem_internal.h"

namespace umem {
namespace {

constexpr int TT = 32;       // tokens per tile
constexpr int TN = 64;       // keys per tile
constexpr int DC = 32;       // dims per LDS chunk
constexpr int LDS_STRIDE = DC + 4;   // floats per LDS row: float4-aligned, conflict-free b128 reads
constexpr int THREADS = 256;

__global__ __launch_bounds__(THREADS) void axis_scores_kernel(
    const float* __restrict__ q_row, const float* __restrict__ q_col,
    const float* __restrict__ k_row, const float* __restrict__ k_col,
    const float* __restrict__ core, float* __restrict__ sel, int T, int H, int n, int dk,
    int rank) {
  const int axis = blockIdx.z & 1;
  const int h = blockIdx.z >> 1;
  const float* __restrict__ q = axis ? q_col : q_row;
  const float* __restrict__ K = axis ? k_col : k_row;
  const int i0 = blockIdx.x * TN;
  const int t0 = blockIdx.y * TT;
  const int tid = threadIdx.x;

  __shared__ float4 sk4[TN * LDS_STRIDE / 4];
  __shared__ float4 sq4[TT * LDS_STRIDE / 4];
  __shared__ float fvec[kMaxRank];
  float* sk = reinterpret_cast<float*>(sk4);
  float* sq = reinterpret_cast<float*>(sq4);

  if (tid == 0) {
    if (core != nullptr) {
      float u[kMaxRank], tv[kMaxRank];
      rank1_factors(core + static_cast<size_t>(h) * rank * rank, rank, u, tv);
      for (int j = 0; j < rank; ++j) fvec[j] = axis ? tv[j] : u[j];
    } else {
      fvec[0] = 1.0f;
    }
  }

  // micro-tile: keys kx + 16 c (c < 4), tokens 2 ty + {0, 1}
  const int kx = tid & 15;
  const int ty = tid >> 4;
  float acc[2][4];
  float out[2][4];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int c = 0; c < 4; ++c) out[a][c] = 0.0f;

  const int width = dk / rank;
  // loader mapping: 8 lanes cover one 32-float row segment with float4 loads
  const int ld_row = tid >> 3;   // 0..31
  const int ld_col = (tid & 7) * 4;

  for (int rho = 0; rho < rank; ++rho) {
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[a][c] = 0.0f;
    const int dbeg = rho * width;
    const int dend = dbeg + width;
    for (int d0 = dbeg; d0 < dend; d0 += DC) {
      __syncthreads();
      const int d = d0 + ld_col;
      // keys: TN rows, two passes of 32 rows
#pragma unroll
      for (int p = 0; p < TN / 32; ++p) {
        const int i = ld_row + 32 * p;
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (i0 + i < n && d < dend)
          v = *reinterpret_cast<const float4*>(K + (static_cast<size_t>(h) * n + i0 + i) * dk + d);
        *reinterpret_cast<float4*>(sk + i * LDS_STRIDE + ld_col) = v;
      }
      {
        const int t = ld_row;
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (t0 + t < T && d < dend)
          v = *reinterpret_cast<const float4*>(q + (static_cast<size_t>(t0 + t) * H + h) * dk + d);
        *reinterpret_cast<float4*>(sq + t * LDS_STRIDE + ld_col) = v;
      }
      __syncthreads();
#pragma unroll
      for (int dd = 0; dd < DC; dd += 4) {
        float4 kv[4], qv[2];
#pragma unroll
        for (int c = 0; c < 4; ++c)
          kv[c] = *reinterpret_cast<const float4*>(sk + (kx + 16 * c) * LDS_STRIDE + dd);
#pragma unroll
        for (int a = 0; a < 2; ++a)
          qv[a] = *reinterpret_cast<const float4*>(sq + (2 * ty + a) * LDS_STRIDE + dd);
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            float s = acc[a][c];
            s = fmaf(kv[c].x, qv[a].x, s);
            s = fmaf(kv[c].y, qv[a].y, s);
            s = fmaf(kv[c].z, qv[a].z, s);
            s = fmaf(kv[c].w, qv[a].w, s);
            acc[a][c] = s;
          }
      }
    }
    if (core != nullptr) {
      const float f = fvec[rho];
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int c = 0; c < 4; ++c) out[a][c] = fmaf(f, acc[a][c], out[a][c]);
    } else {
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int c = 0; c < 4; ++c) out[a][c] = acc[a][c];
    }
  }

#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const int t = t0 + 2 * ty + a;
    if (t >= T) continue;
    float* dst = sel + ((static_cast<size_t>(axis) * T + t) * H + h) * n;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int i = i0 + kx + 16 * c;
      if (i < n) dst[i] = out[a][c];
    }
  }
}

}  // namespace

hipError_t launch_axis_scores(const umem_desc& d, int T, const float* q_row, const float* q_col,
                              const float* k_row, const float* k_col, const float* core,
                              float* sel, hipStream_t s) {
  if (T == 0) return hipSuccess;
  dim3 grid((d.n_keys + TN - 1) / TN, (T + TT - 1) / TT, d.heads * 2);
  const float* c = (d.grid == UMEM_GRID_TUCKER) ? core : nullptr;
  hipLaunchKernelGGL(axis_scores_kernel, grid, dim3(THREADS), 0, s, q_row, q_col, k_row, k_col, c,
                     sel, T, d.heads, d.n_keys, d.dk, d.rank);
  return hipGetLastError();
}

}  // namespace umem
