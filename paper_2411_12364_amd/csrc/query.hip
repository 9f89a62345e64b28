// The query front-end (Sec. 3.2, Tricks 2, 4, 5) and the key LayerNorm (Trick 2).
//
// hidden states x [B, L, d] -> causal depthwise convolution (K_c taps per channel, history before
// each sequence's first token in this batch) -> query linear (bf16 MFMA GEMM, fp32 accumulation)
// -> LayerNorm of each (axis, head) query over its D_k elements -> q_row (and q_col unless the
// query is shared).
//
// * conv_kernel: one thread per 4 consecutive channels of a token, the K_c source rows read as
//   16-byte pieces (neighbouring tokens' rows are L2 hits), fp32 accumulation.  The convolved
//   rows feed only the query linear, whose GEMM takes its operands in bf16, so they are stored
//   rounded to bf16 (nearest even, the rounding the GEMM would apply to fp32 rows).
// * the query linear is the projection's GEMM (split over K where few tiles would leave CUs
//   idle).  A split GEMM leaves its partial sums to the LayerNorm, which adds them in split order
//   as it loads a row (the order the GEMM's own sum kernel uses): one launch and one round trip
//   of the raw queries fewer.
// * ln_kernel: one wave per (token, axis, head) row, the row held in registers (PER values per
//   lane), mean and population variance by wave reductions, fp32; the same kernel normalises the
//   rows of a key set.
#include <algorithm>

#include "umem_internal.h"

namespace umem {
namespace {

constexpr int THREADS = 256;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// y: the convolved rows as bf16 bits [T, d]
__global__ __launch_bounds__(THREADS) void conv_kernel(const float* __restrict__ x,
                                                       const float* __restrict__ hist,
                                                       const float* __restrict__ w,
                                                       uint16_t* __restrict__ y, int L, int d, int kc,
                                                       size_t n4) {
  const int d4 = d >> 2;
  for (size_t i = static_cast<size_t>(blockIdx.x) * THREADS + threadIdx.x; i < n4;
       i += static_cast<size_t>(gridDim.x) * THREADS) {
    const size_t t = i / d4;
    const int c = static_cast<int>(i - t * d4) * 4;
    const size_t b = t / L;
    const int l = static_cast<int>(t - b * L);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < kc; ++j) {
      const int src = l - j;
      f32x4 v = {0.f, 0.f, 0.f, 0.f};
      if (src >= 0)
        v = *reinterpret_cast<const f32x4*>(x + (t - j) * d + c);
      else if (hist != nullptr)
        v = *reinterpret_cast<const f32x4*>(hist + (b * (kc - 1) + (kc - 1 + src)) * d + c);
      const f32x4 wj = *reinterpret_cast<const f32x4*>(w + static_cast<size_t>(j) * d + c);
      acc.x = fmaf(wj.x, v.x, acc.x);
      acc.y = fmaf(wj.y, v.y, acc.y);
      acc.z = fmaf(wj.z, v.z, acc.z);
      acc.w = fmaf(wj.w, v.w, acc.w);
    }
    *reinterpret_cast<u32x2*>(y + t * d + c) =
        u32x2{__builtin_bit_cast(uint32_t, bf16x2{static_cast<__bf16>(acc.x), static_cast<__bf16>(acc.y)}),
              __builtin_bit_cast(uint32_t, bf16x2{static_cast<__bf16>(acc.z), static_cast<__bf16>(acc.w)})};
  }
}

__device__ __forceinline__ float wave_sum_f(float v) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

// Row r of `in` (dk floats) normalised with parameters p (gamma, beta at p * dk).  With
// splits > 1 `in` holds that many partial sums of the rows, split_stride floats apart, and a row
// is their sum in split order.
// Query layout (KEYS false): r = t * period + blk, blk = a * H + h; written to (a ? out1 : out0)
// at (t * H + h) * dk, parameters blk.  Key layout: r = h * period + i; written in place of
// r * dk, parameters h.
template <int PER, bool KEYS>
// (in and out0 may be the same rows: each lane writes only the elements it has read)
__global__ __launch_bounds__(THREADS) void ln_kernel(const float* in, int splits, size_t split_stride,
                                                     float* out0, float* out1,
                                                     const float* __restrict__ gamma,
                                                     const float* __restrict__ beta, size_t rows,
                                                     int dk, int period, int H, float eps) {
  const int lane = threadIdx.x & (kWave - 1);
  const size_t r = static_cast<size_t>(blockIdx.x) * (THREADS / kWave) + threadIdx.x / kWave;
  if (r >= rows) return;                             // whole waves: no barrier in this kernel
  const float* src = in + r * dk;
  // the partial sums are loaded SB at a time, all in flight together, then added in split order
  constexpr int SB = PER >= 16 ? 4 : 8;
  float v[PER];
  for (int sp0 = 0; sp0 < splits; sp0 += SB) {
    float part[SB][PER];
#pragma unroll
    for (int u = 0; u < SB; ++u)
#pragma unroll
      for (int p = 0; p < PER; ++p) {
        const int e = lane + kWave * p;
        part[u][p] = sp0 + u < splits && e < dk ? src[static_cast<size_t>(sp0 + u) * split_stride + e] : 0.0f;
      }
#pragma unroll
    for (int u = 0; u < SB; ++u)
#pragma unroll
      for (int p = 0; p < PER; ++p) {
        if (sp0 + u == 0) v[p] = part[u][p];
        else if (sp0 + u < splits) v[p] += part[u][p];
      }
  }
  float s = 0.0f;
#pragma unroll
  for (int p = 0; p < PER; ++p) s += v[p];
  const float mean = wave_sum_f(s) / static_cast<float>(dk);
  float q = 0.0f;
#pragma unroll
  for (int p = 0; p < PER; ++p) {
    const int e = lane + kWave * p;
    const float dv = e < dk ? v[p] - mean : 0.0f;
    q = fmaf(dv, dv, q);
  }
  const float inv = 1.0f / sqrtf(wave_sum_f(q) / static_cast<float>(dk) + eps);
  size_t pidx;
  float* dst;
  if (KEYS) {
    pidx = r / period;
    dst = out0 + r * dk;
  } else {
    const size_t t = r / period;
    const int blk = static_cast<int>(r - t * period);
    const int a = blk / H, h = blk - a * H;
    pidx = blk;
    dst = (a ? out1 : out0) + (t * H + h) * dk;
  }
  const float* g = gamma + pidx * dk;
  const float* bt = beta + pidx * dk;
#pragma unroll
  for (int p = 0; p < PER; ++p) {
    const int e = lane + kWave * p;
    if (e < dk) dst[e] = fmaf((v[p] - mean) * inv, g[e], bt[e]);
  }
}

template <bool KEYS>
hipError_t launch_ln(const float* in, int splits, size_t split_stride, float* out0, float* out1,
                     const float* gamma, const float* beta, size_t rows, int dk, int period, int H,
                     float eps, hipStream_t s) {
  const unsigned blocks = static_cast<unsigned>((rows + THREADS / kWave - 1) / (THREADS / kWave));
  const int per = (dk + kWave - 1) / kWave;
#define UMEM_LN(P)                                                                               \
  hipLaunchKernelGGL((ln_kernel<P, KEYS>), dim3(blocks), dim3(THREADS), 0, s, in, splits,       \
                     split_stride, out0, out1, gamma, beta, rows, dk, period, H, eps)
  if (per <= 1) UMEM_LN(1);
  else if (per <= 2) UMEM_LN(2);
  else if (per <= 4) UMEM_LN(4);
  else if (per <= 8) UMEM_LN(8);
  else if (per <= 16) UMEM_LN(16);
  else return hipErrorInvalidValue;
#undef UMEM_LN
  return hipGetLastError();
}

size_t round_up256(size_t x) { return (x + 255) / 256 * 256; }

}  // namespace

size_t query_workspace_bytes(const umem_query_desc& qd, int64_t T) {
  if (T == 0) return 0;
  const int nq = (qd.shared ? 1 : 2) * qd.heads * qd.dk;
  return round_up256(static_cast<size_t>(T) * qd.d_model * sizeof(uint16_t)) +
         round_up256(static_cast<size_t>(T) * nq * sizeof(float)) +
         gemm_partial_bytes(static_cast<int>(T), nq, qd.d_model);
}

hipError_t launch_query(const umem_query_desc& qd, int B, int L, const float* x,
                        const float* x_hist, const float* conv_w, const uint16_t* w_q,
                        const float* gamma, const float* beta, float* q_row, float* q_col,
                        void* ws, hipStream_t s) {
  clear_stale_error();
  const int T = B * L;
  if (T == 0) return hipSuccess;
  const int A = qd.shared ? 1 : 2;
  const int nq = A * qd.heads * qd.dk;
  char* base = static_cast<char*>(ws);
  uint16_t* y = reinterpret_cast<uint16_t*>(base);
  float* q_raw = reinterpret_cast<float*>(base + round_up256(static_cast<size_t>(T) * qd.d_model * sizeof(uint16_t)));
  float* part = reinterpret_cast<float*>(reinterpret_cast<char*>(q_raw) +
                                         round_up256(static_cast<size_t>(T) * nq * sizeof(float)));
  const size_t n4 = static_cast<size_t>(T) * qd.d_model / 4;
  const unsigned blocks = static_cast<unsigned>(std::min<size_t>((n4 + THREADS - 1) / THREADS, 4096));
  hipLaunchKernelGGL(conv_kernel, dim3(blocks), dim3(THREADS), 0, s, x,
                     qd.conv_k > 1 ? x_hist : nullptr, conv_w, y, L, qd.d_model, qd.conv_k, n4);
  hipError_t e = hipGetLastError();
  int splits = 1;
  if (e == hipSuccess) e = gemm_bf16_parts(y, w_q, q_raw, T, nq, qd.d_model, part, s, &splits);
  if (e == hipSuccess)
    e = launch_ln<false>(splits > 1 ? part : q_raw, splits, static_cast<size_t>(T) * nq, q_row,
                         qd.shared ? q_row : q_col, gamma, beta,
                         static_cast<size_t>(T) * A * qd.heads, qd.dk, A * qd.heads, qd.heads,
                         qd.eps, s);
  return e;
}

hipError_t launch_key_norm(int heads, int n, int dk, const float* keys, const float* gamma,
                           const float* beta, float eps, float* out, hipStream_t s) {
  clear_stale_error();
  return launch_ln<true>(keys, 1, 0, out, nullptr, gamma, beta, static_cast<size_t>(heads) * n, dk,
                         n, heads, eps, s);
}

}  // namespace umem
