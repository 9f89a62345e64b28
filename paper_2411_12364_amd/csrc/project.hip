// a8: IVE projection and output linear, C = bf16(A) B with fp32 accumulation on MFMA.
//
// y = sum_p pooled[:, p, :] W_p (eq. (15)) is one GEMM of [T, E*Dv] by [E*Dv, D'v] because
// pooled [T, E, Dv] and W_proj [E, Dv, D'v] are both contiguous; the output linear of Trick 6 is
// a second GEMM of y by W_out [D'v, d_out].
//
// Tiles of 128 x 64 per workgroup, four waves of 64 x 32 (4 x 2 v_mfma_f32_16x16x16_bf16
// tiles), K in steps of 32.  A (fp32) is read with 16-byte loads and rounded to bf16 (nearest
// even) as it is staged into LDS; B (bf16, rows of N) with 16-byte loads, transposed into LDS
// so that each lane's four k of one column are contiguous.  The next K-slice is fetched into
// registers while the current one is multiplied.  Workgroups are dealt round-robin to the
// eight XCDs, so tile t is given to workgroup (t mod per) * 8 + t / per: each XCD takes a
// contiguous band of M-blocks across all N-tiles and finds A's rows and B in its own L2.
//
// Few tiles over a long K (a decode batch against the E * Dv rows of the IVE projectors) would
// leave most CUs idle, each workgroup walking hundreds of K-steps: there K is split S ways
// (S a power of two, until tiles * S >= 512 or a split would fall below 8 K-steps), each split
// writes its partial tile to the workspace, and a second kernel adds the S partials in split
// order, so the result does not depend on timing.
#include <algorithm>

#include "umem_internal.h"

namespace umem {
namespace {

constexpr int BM = 128, BN = 64, BK = 32;
constexpr int THREADS = 256;
constexpr int LDA = BK + 8;   // LDS pitch of A's rows in bf16 (80 B: fragment reads conflict-free)
constexpr int LDB = BK + 4;   // LDS pitch of B's columns in bf16 (72 B)
constexpr int kXcds = 8;

typedef short bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// One K-slice of the operands in registers: four 16-byte pieces of A (thread t, piece i: row
// (t + 256 i) / 8, k (t % 8) * 4) and one of B (row k t / 8, columns (t % 8) * 8 ...).
struct Slice {
  f32x4 a[4];
  u32x4 b;
};

// K-range [.., k_end) of this split; lda = K, the row length of A.
__device__ __forceinline__ void fetch(const float* __restrict__ A, const uint16_t* __restrict__ B,
                                      int M, int N, int lda, int k_end, int m0, int n0, int k0,
                                      int tid, Slice& sl) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int f = tid + THREADS * i;
    const int gm = m0 + (f >> 3), gk = k0 + (f & 7) * 4;
    sl.a[i] = (gm < M && gk < k_end)
                  ? *reinterpret_cast<const f32x4*>(A + static_cast<size_t>(gm) * lda + gk)
                  : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const int gk = k0 + (tid >> 3), gn = n0 + (tid & 7) * 8;
  sl.b = (gk < k_end && gn < N) ? *reinterpret_cast<const u32x4*>(B + static_cast<size_t>(gk) * N + gn)
                                : u32x4{0u, 0u, 0u, 0u};
}

__device__ __forceinline__ void stage(const Slice& sl, uint16_t* As, uint16_t* Bs, int tid) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int f = tid + THREADS * i;
    u32x2 v;
    v.x = static_cast<uint32_t>(f32_to_bf16(sl.a[i].x)) | (static_cast<uint32_t>(f32_to_bf16(sl.a[i].y)) << 16);
    v.y = static_cast<uint32_t>(f32_to_bf16(sl.a[i].z)) | (static_cast<uint32_t>(f32_to_bf16(sl.a[i].w)) << 16);
    *reinterpret_cast<u32x2*>(As + (f >> 3) * LDA + (f & 7) * 4) = v;
  }
  const int kk = tid >> 3, nc = (tid & 7) * 8;
  const uint32_t w[4] = {sl.b.x, sl.b.y, sl.b.z, sl.b.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    Bs[(nc + 2 * e) * LDB + kk] = static_cast<uint16_t>(w[e] & 0xFFFFu);
    Bs[(nc + 2 * e + 1) * LDB + kk] = static_cast<uint16_t>(w[e] >> 16);
  }
}

__global__ __launch_bounds__(THREADS) void gemm_bf16_kernel(const float* __restrict__ A,
                                                            const uint16_t* __restrict__ B,
                                                            float* __restrict__ C, int M, int N,
                                                            int K, int n_tiles_n, int per_xcd,
                                                            int n_tiles, int k_chunk) {
  __shared__ __align__(16) uint16_t As[BM * LDA];   // [m][k]
  __shared__ __align__(16) uint16_t Bs[BN * LDB];   // [n][k]
  const int tile = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
  if (tile >= n_tiles) return;                     // the whole workgroup: no barrier is skipped
  const int m0 = (tile / n_tiles_n) * BM, n0 = (tile % n_tiles_n) * BN;
  // split blockIdx.y covers K-range [k_begin, k_end) and writes its own partial C
  const int k_begin = blockIdx.y * k_chunk, k_end = min(K, k_begin + k_chunk);
  C += static_cast<size_t>(blockIdx.y) * M * N;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;         // this wave's 64 x 32 block of the tile

  f32x4 acc[4][2];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  Slice sl;
  fetch(A, B, M, N, K, k_end, m0, n0, k_begin, tid, sl);
  for (int k0 = k_begin; k0 < k_end; k0 += BK) {
    stage(sl, As, Bs, tid);
    __syncthreads();
    if (k0 + BK < k_end) fetch(A, B, M, N, K, k_end, m0, n0, k0 + BK, tid, sl);
#pragma unroll
    for (int ks = 0; ks < BK; ks += 16) {
      // lane: row (or column) lane % 16 of a 16-block, k = ks + 4 (lane / 16) ... + 3
      bf16x4 af[4], bfr[2];
#pragma unroll
      for (int a = 0; a < 4; ++a)
        af[a] = *reinterpret_cast<const bf16x4*>(As + (wm * 64 + a * 16 + (lane & 15)) * LDA + ks + 4 * (lane >> 4));
#pragma unroll
      for (int b = 0; b < 2; ++b)
        bfr[b] = *reinterpret_cast<const bf16x4*>(Bs + (wn * 32 + b * 16 + (lane & 15)) * LDB + ks + 4 * (lane >> 4));
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(af[a], bfr[b], acc[a][b], 0, 0, 0);
    }
    __syncthreads();
  }
  // D layout: lane holds rows 4 (lane / 16) + r of column lane % 16
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int gm = m0 + wm * 64 + a * 16 + 4 * (lane >> 4) + r;
        const int gn = n0 + wn * 32 + b * 16 + (lane & 15);
        if (gm < M && gn < N) C[static_cast<size_t>(gm) * N + gn] = acc[a][b][r];
      }
}

// C = sum over s < S of part[s] (n4 16-byte pieces each), in split order.
__global__ __launch_bounds__(THREADS) void sum_splits_kernel(const f32x4* __restrict__ part,
                                                             f32x4* __restrict__ C, size_t n4,
                                                             int S) {
  for (size_t i = static_cast<size_t>(blockIdx.x) * THREADS + threadIdx.x; i < n4;
       i += static_cast<size_t>(gridDim.x) * THREADS) {
    f32x4 acc = part[i];
    for (int sp = 1; sp < S; ++sp) acc += part[sp * n4 + i];
    C[i] = acc;
  }
}

int n_tiles(int M, int N) { return ((M + BM - 1) / BM) * ((N + BN - 1) / BN); }

int split_count(int M, int N, int K) {
  int S = 1;
  while (static_cast<int64_t>(n_tiles(M, N)) * S < 512 && K / (2 * S) >= 8 * BK) S *= 2;
  return S;
}

size_t round_up256(size_t x) { return (x + 255) / 256 * 256; }

}  // namespace

size_t gemm_partial_bytes(int M, int N, int K) {
  const int S = split_count(M, N, K);
  return S > 1 ? round_up256(static_cast<size_t>(S) * M * N * sizeof(float)) : 0;
}

hipError_t gemm_bf16(const float* A, const uint16_t* B, float* C, int M, int N, int K, float* part,
                     hipStream_t s) {
  const int tn = (N + BN - 1) / BN;
  const int tiles = n_tiles(M, N);
  const int per = (tiles + kXcds - 1) / kXcds;
  const int S = split_count(M, N, K);
  const int k_chunk = S > 1 ? ((K + S - 1) / S + BK - 1) / BK * BK : K;
  hipLaunchKernelGGL(gemm_bf16_kernel, dim3(per * kXcds, S), dim3(THREADS), 0, s, A, B,
                     S > 1 ? part : C, M, N, K, tn, per, tiles, k_chunk);
  if (S > 1) {
    const size_t n4 = static_cast<size_t>(M) * N / 4;     // N % 8 == 0
    const unsigned blocks = static_cast<unsigned>(std::min<size_t>((n4 + THREADS - 1) / THREADS, 2048));
    hipLaunchKernelGGL(sum_splits_kernel, dim3(blocks), dim3(THREADS), 0, s,
                       reinterpret_cast<const f32x4*>(part), reinterpret_cast<f32x4*>(C), n4, S);
  }
  return hipGetLastError();
}

size_t project_workspace_bytes(int T, int expand, int dv, int dv_virt, int d_out) {
  if (T == 0) return 0;
  if (dv_virt == 0) return gemm_partial_bytes(T, d_out, dv);          // the output linear alone
  const size_t tmp = d_out > 0 ? round_up256(static_cast<size_t>(T) * dv_virt * sizeof(float)) : 0;
  const size_t p1 = gemm_partial_bytes(T, dv_virt, expand * dv);
  const size_t p2 = d_out > 0 ? gemm_partial_bytes(T, d_out, dv_virt) : 0;
  return tmp + std::max(p1, p2);
}

hipError_t launch_project(int T, int expand, int dv, int dv_virt, int d_out, const float* pooled,
                          const uint16_t* w_proj, const uint16_t* w_out, float* out, void* ws,
                          hipStream_t s) {
  clear_stale_error();
  if (T == 0) return hipSuccess;
  char* base = static_cast<char*>(ws);
  if (w_proj == nullptr)   // the output linear alone: [T, dv] by [dv, d_out]
    return gemm_bf16(pooled, w_out, out, T, d_out, dv, reinterpret_cast<float*>(base), s);
  if (w_out == nullptr)
    return gemm_bf16(pooled, w_proj, out, T, dv_virt, expand * dv, reinterpret_cast<float*>(base), s);
  // the two GEMMs use the partial scratch one after the other, in stream order
  float* tmp = reinterpret_cast<float*>(base);
  float* part = reinterpret_cast<float*>(base + round_up256(static_cast<size_t>(T) * dv_virt * sizeof(float)));
  hipError_t e = gemm_bf16(pooled, w_proj, tmp, T, dv_virt, expand * dv, part, s);
  if (e != hipSuccess) return e;
  return gemm_bf16(tmp, w_out, out, T, d_out, dv_virt, part, s);
}

}  // namespace umem
