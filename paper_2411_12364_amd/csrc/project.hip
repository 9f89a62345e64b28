// a8: IVE projection and output linear, C = bf16(A) B with fp32 accumulation on MFMA.
//
// y = sum_p pooled[:, p, :] W_p (eq. (15)) is one GEMM of [T, E*Dv] by [E*Dv, D'v] because
// pooled [T, E, Dv] and W_proj [E, Dv, D'v] are both contiguous; the output linear of Trick 6 is
// a second GEMM of y by W_out [D'v, d_out].  A (fp32) is rounded to bf16 (nearest even) as it is
// staged into LDS; B is bf16.  Tiles: 64 x 64 per workgroup, four waves of 32 x 32, K in steps
// of 32, v_mfma_f32_16x16x16_bf16.
#include "umem_internal.h"

namespace umem {
namespace {

constexpr int BM = 64, BN = 64, BK = 32;
constexpr int THREADS = 256;
constexpr int APAD = 4;   // bf16 elements of padding per LDS row

typedef short bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(THREADS) void gemm_bf16_kernel(const float* __restrict__ A,
                                                            const uint16_t* __restrict__ B,
                                                            float* __restrict__ C, int M, int N,
                                                            int K) {
  __shared__ uint16_t As[BM][BK + APAD];   // [m][k]
  __shared__ uint16_t Bs[BN][BK + APAD];   // [n][k]
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;

  f32x4 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = 0; k0 < K; k0 += BK) {
    // A tile: 64 x 32 fp32 -> bf16; each thread 8 consecutive k of one row
    {
      const int r = tid >> 2, c = (tid & 3) * 8;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int gm = m0 + r, gk = k0 + c + e;
        const float x = (gm < M && gk < K) ? A[static_cast<size_t>(gm) * K + gk] : 0.0f;
        As[r][c + e] = f32_to_bf16(x);
      }
    }
    // B tile: 32 x 64 bf16, stored transposed; each thread 8 consecutive n of one k
    {
      const int kk = tid >> 3, c = (tid & 7) * 8;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int gk = k0 + kk, gn = n0 + c + e;
        Bs[c + e][kk] = (gk < K && gn < N) ? B[static_cast<size_t>(gk) * N + gn] : uint16_t(0);
      }
    }
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < BK; ks += 16) {
      bf16x4 af[2], bfr[2];
#pragma unroll
      for (int a = 0; a < 2; ++a) {
        const uint16_t* p = &As[wm * 32 + a * 16 + (lane & 15)][ks + 4 * (lane >> 4)];
        af[a] = *reinterpret_cast<const bf16x4*>(p);
      }
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const uint16_t* p = &Bs[wn * 32 + b * 16 + (lane & 15)][ks + 4 * (lane >> 4)];
        bfr[b] = *reinterpret_cast<const bf16x4*>(p);
      }
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(af[a], bfr[b], acc[a][b], 0, 0, 0);
    }
    __syncthreads();
  }
  // D layout: lane holds rows 4*(lane/16) + r of column lane%16
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int gm = m0 + wm * 32 + a * 16 + 4 * (lane >> 4) + r;
        const int gn = n0 + wn * 32 + b * 16 + (lane & 15);
        if (gm < M && gn < N) C[static_cast<size_t>(gm) * N + gn] = acc[a][b][r];
      }
}

hipError_t gemm(const float* A, const uint16_t* B, float* C, int M, int N, int K, hipStream_t s) {
  dim3 grid((N + BN - 1) / BN, (M + BM - 1) / BM);
  hipLaunchKernelGGL(gemm_bf16_kernel, grid, dim3(THREADS), 0, s, A, B, C, M, N, K);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_project(int T, int expand, int dv, int dv_virt, int d_out, const float* pooled,
                          const uint16_t* w_proj, const uint16_t* w_out, float* out, float* tmp,
                          hipStream_t s) {
  clear_stale_error();
  if (T == 0) return hipSuccess;
  if (w_out == nullptr) return gemm(pooled, w_proj, out, T, dv_virt, expand * dv, s);
  hipError_t e = gemm(pooled, w_proj, tmp, T, dv_virt, expand * dv, s);
  if (e != hipSuccess) return e;
  return gemm(tmp, w_out, out, T, d_out, dv_virt, s);
}

}  // namespace umem
