// a6 + a7: score-weighted gather-sum of value rows (embedding bag), eq. (1) and eq. (15).
//
// One workgroup per token.  A value row is read with 16-byte loads, L lanes per row and CPL
// 16-byte chunks per lane (row bytes = 16 * L * CPL); a wave keeps U rows in flight, so a
// workgroup has 4 * U rows outstanding.  Accumulation is fp32 in registers; partial sums of the
// sub-rows of a wave are combined with shuffles and those of the 4 waves in LDS, in a fixed
// order (the result does not depend on timing).  With implicit value expansion the bag is first
// split by virtual block p (a stable partition, order within a block kept) and each block's
// rows are pooled into out[t, p, :].
#include "umem_internal.h"

namespace umem {
namespace {

constexpr int THREADS = 256;
constexpr int NWAVES = THREADS / kWave;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <typename Elem>
struct ElemTraits;
template <>
struct ElemTraits<float> {
  static constexpr int kPerChunk = 4;
  __device__ static inline void widen(const u32x4& r, float* x) {
    x[0] = __uint_as_float(r.x);
    x[1] = __uint_as_float(r.y);
    x[2] = __uint_as_float(r.z);
    x[3] = __uint_as_float(r.w);
  }
};
template <>
struct ElemTraits<uint16_t> {   // bf16 bit patterns
  static constexpr int kPerChunk = 8;
  __device__ static inline void widen(const u32x4& r, float* x) {
    x[0] = __uint_as_float(r.x << 16);
    x[1] = __uint_as_float(r.x & 0xFFFF0000u);
    x[2] = __uint_as_float(r.y << 16);
    x[3] = __uint_as_float(r.y & 0xFFFF0000u);
    x[4] = __uint_as_float(r.z << 16);
    x[5] = __uint_as_float(r.z & 0xFFFF0000u);
    x[6] = __uint_as_float(r.w << 16);
    x[7] = __uint_as_float(r.w & 0xFFFF0000u);
  }
};

template <typename Elem, int L, int CPL>
__global__ __launch_bounds__(THREADS) void gather_kernel(
    const Elem* __restrict__ values, int64_t n_values, int dv, int bag,
    const int32_t* __restrict__ idx, const float* __restrict__ w, const int32_t* __restrict__ perm,
    int expand, float* __restrict__ out) {
  using TR = ElemTraits<Elem>;
  constexpr int EPC = TR::kPerChunk;
  constexpr int SUB = kWave / L;                   // rows a wave reads at once
  constexpr int U = (CPL >= 16) ? 1 : 16 / CPL;    // row batches in flight per wave
  extern __shared__ int32_t smem[];
  int32_t* rows = smem;                            // [bag]
  float* wts = reinterpret_cast<float*>(smem + bag);   // [bag]
  int32_t* blk = smem + 2 * bag;                   // [bag]
  int32_t* order = smem + 3 * bag;                 // [bag]
  float* red = reinterpret_cast<float*>(smem + 4 * bag);   // [dv]
  __shared__ int bstart[65], bcount[64];

  const int t = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int sub = lane / L;
  const int cl = lane % L;

  for (int s = tid; s < bag; s += THREADS) {
    const int64_t x = idx[static_cast<size_t>(t) * bag + s];
    const int64_t v = perm ? static_cast<int64_t>(perm[x]) : x;
    const int p = expand > 1 ? static_cast<int>(v / n_values) : 0;
    rows[s] = static_cast<int32_t>(v - static_cast<int64_t>(p) * n_values);
    wts[s] = w[static_cast<size_t>(t) * bag + s];
    blk[s] = p;
  }
  __syncthreads();
  if (expand > 1) {
    if (wave == 0) {
      const uint64_t lt = lanemask_lt();
      int pos = 0;
      for (int p = 0; p < expand; ++p) {
        if (lane == 0) bstart[p] = pos;
        for (int base = 0; base < bag; base += kWave) {
          const int s = base + lane;
          const bool hit = s < bag && blk[s] == p;
          const uint64_t m = __ballot(hit);
          if (hit) order[pos + __popcll(m & lt)] = s;
          pos += __popcll(m);
        }
        if (lane == 0) bcount[p] = pos - bstart[p];
      }
    }
  } else {
    for (int s = tid; s < bag; s += THREADS) order[s] = s;
    if (tid == 0) {
      bstart[0] = 0;
      bcount[0] = bag;
    }
  }
  __syncthreads();

  const int row_elems = dv;
  for (int p = 0; p < expand; ++p) {
    const int beg = bstart[p];
    const int cnt = bcount[p];
    float acc[CPL][EPC];
#pragma unroll
    for (int c = 0; c < CPL; ++c)
#pragma unroll
      for (int e = 0; e < EPC; ++e) acc[c][e] = 0.0f;

    // rows j = wave*SUB + sub + (NWAVES*SUB) * i
    constexpr int STEP = NWAVES * SUB;
    for (int j0 = wave * SUB + sub; j0 < cnt; j0 += STEP * U) {
      u32x4 raw[U][CPL];
      float wt[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int j = j0 + u * STEP;
        if (j < cnt) {
          const int s = order[beg + j];
          wt[u] = wts[s];
          const Elem* src = values + static_cast<int64_t>(rows[s]) * row_elems;
#pragma unroll
          for (int c = 0; c < CPL; ++c)
            raw[u][c] = *reinterpret_cast<const u32x4*>(src + (cl + L * c) * EPC);
        } else {
          wt[u] = 0.0f;
#pragma unroll
          for (int c = 0; c < CPL; ++c) raw[u][c] = u32x4{0u, 0u, 0u, 0u};
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          float x[EPC];
          TR::widen(raw[u][c], x);
#pragma unroll
          for (int e = 0; e < EPC; ++e) acc[c][e] = fmaf(wt[u], x[e], acc[c][e]);
        }
    }
    // combine the SUB sub-rows of this wave (lanes cl, cl + L, ...) with shuffles
#pragma unroll
    for (int off = L; off < kWave; off <<= 1)
#pragma unroll
      for (int c = 0; c < CPL; ++c)
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[c][e] += __shfl_xor(acc[c][e], off, kWave);
    // combine the waves in LDS, wave 0 first
    for (int v = 0; v < NWAVES; ++v) {
      if (wave == v && sub == 0) {
#pragma unroll
        for (int c = 0; c < CPL; ++c)
#pragma unroll
          for (int e = 0; e < EPC; ++e) {
            const int col = (cl + L * c) * EPC + e;
            red[col] = (v == 0) ? acc[c][e] : red[col] + acc[c][e];
          }
      }
      __syncthreads();
    }
    float* dst = out + (static_cast<size_t>(t) * expand + p) * dv;
    for (int col = tid * 4; col < dv; col += THREADS * 4)
      *reinterpret_cast<float4*>(dst + col) = *reinterpret_cast<const float4*>(red + col);
    __syncthreads();
  }
}

template <typename Elem>
hipError_t launch_typed(const Elem* values, int64_t n_values, int dv, int T, int bag,
                        const int32_t* idx, const float* w, const int32_t* perm, int expand,
                        float* out, hipStream_t s) {
  const int chunks = dv * static_cast<int>(sizeof(Elem)) / 16;
  const size_t lds = static_cast<size_t>(bag) * 16 + static_cast<size_t>(dv) * 4;
  const dim3 grid(T), block(THREADS);
#define UMEM_GATHER(LL, CC)                                                                  \
  hipLaunchKernelGGL((gather_kernel<Elem, LL, CC>), grid, block, lds, s, values, n_values, dv, \
                     bag, idx, w, perm, expand, out)
  switch (chunks) {
    case 1: UMEM_GATHER(1, 1); break;
    case 2: UMEM_GATHER(2, 1); break;
    case 4: UMEM_GATHER(4, 1); break;
    case 8: UMEM_GATHER(8, 1); break;
    case 16: UMEM_GATHER(16, 1); break;
    case 32: UMEM_GATHER(32, 1); break;
    case 64: UMEM_GATHER(64, 1); break;
    case 128: UMEM_GATHER(64, 2); break;
    case 192: UMEM_GATHER(64, 3); break;
    case 256: UMEM_GATHER(64, 4); break;
    case 320: UMEM_GATHER(64, 5); break;
    case 384: UMEM_GATHER(64, 6); break;
    case 448: UMEM_GATHER(64, 7); break;
    case 512: UMEM_GATHER(64, 8); break;
    default: return hipErrorInvalidValue;
  }
#undef UMEM_GATHER
  return hipGetLastError();
}

}  // namespace

bool gather_row_supported(int dv, int vdtype) {
  const int bytes = dv * (vdtype == UMEM_F32 ? 4 : 2);
  if (bytes % 16 != 0 || bytes > kMaxRowBytes) return false;
  const int chunks = bytes / 16;
  if (chunks <= 64) return (chunks & (chunks - 1)) == 0;
  return chunks % 64 == 0;
}

hipError_t launch_gather(int64_t n_values, int dv, int vdtype, const void* values, int T,
                         int bag, const int32_t* idx, const float* w, const int32_t* perm,
                         int expand, float* out, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (vdtype == UMEM_F32)
    return launch_typed(static_cast<const float*>(values), n_values, dv, T, bag, idx, w, perm,
                        expand, out, s);
  return launch_typed(static_cast<const uint16_t*>(values), n_values, dv, T, bag, idx, w, perm,
                      expand, out, s);
}

}  // namespace umem
