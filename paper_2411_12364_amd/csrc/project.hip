// a8: IVE projection and output linear, C = bf16(A) B^T with fp32 accumulation on MFMA.
//
// y = sum_p pooled[:, p, :] W_p (eq. (15)) is one GEMM of [T, E*Dv] by [E*Dv, D'v] because
// pooled [T, E, Dv] is contiguous and the projectors are stored output-major, as a linear
// layer's weight: w_proj [D'v, E*Dv] holds W_p[c][j] at (j, p*Dv + c).  The output linear of
// Trick 6 is a second GEMM of y by w_out [d_out, D'v].  Both operands are then rows of K.
//
// Tiles of 128 x 128 per workgroup, four waves of 64 x 64 (4 x 4 v_mfma_f32_16x16x32_bf16
// tiles), K in steps of 64.  A (fp32, or bf16 when the producer already rounded it) and B (bf16)
// are read with 16-byte buffer loads, whose range check returns zeros past the rows of the
// matrix, so edge tiles need no branches; fp32 A is rounded to bf16 (nearest even) as it is
// staged into LDS, bf16 A and B are copied.  The operand tiles are
// double-buffered in LDS: while slice k is multiplied, slice k + 1 (fetched into registers
// during step k - 1) is staged into the other buffer, and slice k + 2 is fetched after the
// step's one barrier.  The output tile leaves through LDS as whole 128-byte lines.
//
// Workgroups are dealt round-robin to the eight XCDs, so work item i (split-major: i = split *
// tiles + tile) is given to workgroup (i mod per) * 8 + i / per: each XCD takes a contiguous run
// of items, a band of M-blocks across all N-tiles without a split, or one K-range of all tiles
// with one, and finds its slices of A and B in its own L2.
//
// Few tiles over a long K (a decode batch against the E * Dv rows of the IVE projectors) would
// leave most CUs idle, each workgroup walking hundreds of K-steps: there K is split S ways
// (S a power of two, until tiles * S >= 512 or a split would fall below 4 K-steps), each split
// writes its partial tile to the workspace, and a second kernel adds the S partials in split
// order, so the result does not depend on timing.
#include <algorithm>

#include "umem_internal.h"

namespace umem {
namespace {

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int THREADS = 256;
constexpr int LDA = BK + 8;   // LDS pitch of A's and B's rows in bf16 (144 B: fragment reads conflict-free)
constexpr int LDC = 64 + 4;   // LDS pitch of a wave's output rows in fp32 (epilogue)
constexpr int kTileElems = (BM + BN) * LDA;      // one buffer of both operand tiles, bf16
constexpr int kXcds = 8;
constexpr uint32_t kOutOfRange = 0x80000000u;     // a buffer offset past any valid record
static_assert(4 * 32 * LDC * 4 <= 2 * kTileElems * 2, "epilogue staging fits the tiles' LDS");

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// One K-slice of the operands in registers: of fp32 A eight 16-byte pieces (thread t, piece i:
// row (t + 256 i) / 16, k ((t + 256 i) % 16) * 4), of bf16 A and of B four (row (t + 256 i) / 8,
// k ((t + 256 i) % 8) * 8).
template <typename AT>
struct Slice {
  static constexpr int kA = sizeof(AT) == 4 ? 8 : 4;
  u32x4 a[kA];
  u32x4 b[4];
};

// Buffer resource of a raw byte range (stride 0; 32-bit data format, as buffer loads need).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), static_cast<short>(0),
                                           static_cast<int>(bytes), 0x00020000);
}

// K-range [.., k_end) of this split; rows of K elements.  Rows past the matrix read as zeros by
// the buffer range check; k past k_end is sent out of range explicitly.
template <typename AT>
__device__ __forceinline__ void fetch(__amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rb, int K,
                                      int k_end, int m0, int n0, int k0, int tid, Slice<AT>& sl) {
  constexpr int kPer = 16 / sizeof(AT);            // A elements per 16-byte piece
#pragma unroll
  for (int i = 0; i < Slice<AT>::kA; ++i) {
    const int f = tid + THREADS * i;
    const int gk = k0 + (f % (BK / kPer)) * kPer;
    const uint32_t off = static_cast<uint32_t>((m0 + f / (BK / kPer)) * K + gk) * sizeof(AT);
    sl.a[i] = __builtin_amdgcn_raw_buffer_load_b128(ra, gk < k_end ? off : kOutOfRange, 0, 0);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int f = tid + THREADS * i;
    const int gk = k0 + (f & 7) * 8;
    const uint32_t off = static_cast<uint32_t>((n0 + (f >> 3)) * K + gk) * 2u;
    sl.b[i] = __builtin_amdgcn_raw_buffer_load_b128(rb, gk < k_end ? off : kOutOfRange, 0, 0);
  }
}

// Two floats rounded to bf16 (nearest even, one v_cvt_pk_bf16_f32), lo in the low half.
__device__ __forceinline__ uint32_t pack_bf16(uint32_t lo, uint32_t hi) {
  return __builtin_bit_cast(uint32_t, bf16x2{static_cast<__bf16>(__uint_as_float(lo)),
                                              static_cast<__bf16>(__uint_as_float(hi))});
}

template <typename AT>
__device__ __forceinline__ void stage(const Slice<AT>& sl, uint16_t* As, uint16_t* Bs, int tid) {
#pragma unroll
  for (int i = 0; i < Slice<AT>::kA; ++i) {
    const int f = tid + THREADS * i;
    if constexpr (sizeof(AT) == 4)
      *reinterpret_cast<u32x2*>(As + (f >> 4) * LDA + (f & 15) * 4) =
          u32x2{pack_bf16(sl.a[i].x, sl.a[i].y), pack_bf16(sl.a[i].z, sl.a[i].w)};
    else
      *reinterpret_cast<u32x4*>(As + (f >> 3) * LDA + (f & 7) * 8) = sl.a[i];
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int f = tid + THREADS * i;
    *reinterpret_cast<u32x4*>(Bs + (f >> 3) * LDA + (f & 7) * 8) = sl.b[i];
  }
}

// A fp32 or bf16 [M, K], B bf16 [N, K] (both rows of K, 16-byte aligned), C fp32 [M, N]; the
// bytes of A and of B below 2^31.
template <typename AT>
__global__ __launch_bounds__(THREADS) __attribute__((amdgpu_waves_per_eu(2, 2))) void gemm_bf16_kernel(
    const AT* __restrict__ A, const uint16_t* __restrict__ B, float* __restrict__ C, int M,
    int N, int K, int n_tiles_n, int per_xcd, int n_tiles, int n_items, int k_chunk) {
  __shared__ __align__(16) uint16_t smem[2 * kTileElems];
  // item = split * n_tiles + tile; XCD x takes items [x per, (x + 1) per)
  const int item = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
  if (item >= n_items) return;                     // the whole workgroup: no barrier is skipped
  const int split = item / n_tiles, tile = item % n_tiles;
  const int m0 = (tile / n_tiles_n) * BM, n0 = (tile % n_tiles_n) * BN;
  // this split covers K-range [k_begin, k_end) and writes its own partial C
  const int k_begin = split * k_chunk, k_end = min(K, k_begin + k_chunk);
  C += static_cast<size_t>(split) * M * N;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;         // this wave's 64 x 64 block of the tile
  const __amdgpu_buffer_rsrc_t ra = rsrc(A, static_cast<uint32_t>(M) * K * static_cast<uint32_t>(sizeof(AT)));
  const __amdgpu_buffer_rsrc_t rb = rsrc(B, static_cast<uint32_t>(N) * K * 2u);

  f32x4 acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  Slice<AT> sl;
  fetch(ra, rb, K, k_end, m0, n0, k_begin, tid, sl);
  stage(sl, smem, smem + BM * LDA, tid);
  __syncthreads();
  if (k_begin + BK < k_end) fetch(ra, rb, K, k_end, m0, n0, k_begin + BK, tid, sl);
  int buf = 0;
  for (int k0 = k_begin; k0 < k_end; k0 += BK) {
    const uint16_t* As = smem + buf * kTileElems;   // [m][k]
    const uint16_t* Bs = As + BM * LDA;             // [n][k]
#pragma unroll
    for (int ks = 0; ks < BK; ks += 32) {
      // lane: row (or column) lane % 16 of a 16-block, k = ks + 8 (lane / 16) ... + 7
      bf16x8 af[4], bfr[4];
#pragma unroll
      for (int a = 0; a < 4; ++a)
        af[a] = *reinterpret_cast<const bf16x8*>(As + (wm * 64 + a * 16 + (lane & 15)) * LDA + ks + 8 * (lane >> 4));
#pragma unroll
      for (int b = 0; b < 4; ++b)
        bfr[b] = *reinterpret_cast<const bf16x8*>(Bs + (wn * 64 + b * 16 + (lane & 15)) * LDA + ks + 8 * (lane >> 4));
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
    }
    if (k0 + BK < k_end) {
      uint16_t* An = smem + (buf ^ 1) * kTileElems;
      stage(sl, An, An + BM * LDA, tid);
    }
    __syncthreads();
    if (k0 + 2 * BK < k_end) fetch(ra, rb, K, k_end, m0, n0, k0 + 2 * BK, tid, sl);
    buf ^= 1;
  }
  // D layout: lane holds rows 4 (lane / 16) + r of column lane % 16.  Each wave's 64 x 64 block
  // goes out in two halves of 32 rows through LDS (the operand tiles' space, free after the last
  // barrier), read back as 16-byte pieces so that every row is written as whole 128-byte lines.
  float* Cs = reinterpret_cast<float*>(smem) + wave * 32 * LDC;
#pragma unroll
  for (int half = 0; half < 2; ++half) {
#pragma unroll
    for (int a2 = 0; a2 < 2; ++a2)
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          Cs[(a2 * 16 + 4 * (lane >> 4) + r) * LDC + b * 16 + (lane & 15)] = acc[half * 2 + a2][b][r];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int row = (lane >> 4) + 4 * i, c4 = (lane & 15) * 4;
      const int gm = m0 + wm * 64 + half * 32 + row, gn = n0 + wn * 64 + c4;
      const f32x4 v = *reinterpret_cast<const f32x4*>(Cs + row * LDC + c4);
      if (gm < M && gn < N) *reinterpret_cast<f32x4*>(C + static_cast<size_t>(gm) * N + gn) = v;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
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
  while (static_cast<int64_t>(n_tiles(M, N)) * S < 512 && K / (2 * S) >= 4 * BK) S *= 2;
  return S;
}

size_t round_up256(size_t x) { return (x + 255) / 256 * 256; }

// A's buffer range is 32-bit: a GEMM is launched in bands of at most this many rows of A, whose
// bytes stay below 2^31 (a multiple of BM).
int64_t band_rows(int K) {
  return std::max<int64_t>(BM, (((INT64_C(1) << 31) - 1) / (static_cast<int64_t>(K) * 4)) / BM * BM);
}

// Partial-sum bytes of one launch (one band) of `rows` rows.
size_t band_partial_bytes(int rows, int N, int K) {
  const int S = split_count(rows, N, K);
  return S > 1 ? round_up256(static_cast<size_t>(S) * rows * N * sizeof(float)) : 0;
}

}  // namespace

// Each band chooses its own split count from its own tile count, and a band of fewer rows may
// split more ways than the whole matrix would (fewer tiles), so the scratch is the largest of
// the bands' needs: the full bands and the last, shorter one.  The bands run one after the
// other on one stream and share it.
size_t gemm_partial_bytes(int M, int N, int K) {
  const int64_t band = band_rows(K);
  if (M <= band) return band_partial_bytes(M, N, K);
  const int last = static_cast<int>(M - (M - 1) / band * band);
  return std::max(band_partial_bytes(static_cast<int>(band), N, K), band_partial_bytes(last, N, K));
}

namespace {

// The bands are sized for fp32 A whatever A's type, so that the scratch of the split-K partials
// (gemm_partial_bytes) is the same for both.
template <typename AT>
hipError_t gemm_any(const AT* A, const uint16_t* B, float* C, int M, int N, int K, float* part,
                    hipStream_t s) {
  const int64_t band = band_rows(K);
  if (M > band) {
    for (int64_t m = 0; m < M; m += band) {
      const int rows = static_cast<int>(std::min<int64_t>(band, M - m));
      hipError_t e = gemm_any(A + m * K, B, C + m * N, rows, N, K, part, s);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
  const int tn = (N + BN - 1) / BN;
  const int tiles = n_tiles(M, N);
  const int S = split_count(M, N, K);
  const int per = (tiles * S + kXcds - 1) / kXcds;
  const int k_chunk = S > 1 ? ((K + S - 1) / S + BK - 1) / BK * BK : K;
  hipLaunchKernelGGL(gemm_bf16_kernel<AT>, dim3(per * kXcds), dim3(THREADS), 0, s, A, B,
                     S > 1 ? part : C, M, N, K, tn, per, tiles, tiles * S, k_chunk);
  if (S > 1) {
    const size_t n4 = static_cast<size_t>(M) * N / 4;     // N % 8 == 0
    const unsigned blocks = static_cast<unsigned>(std::min<size_t>((n4 + THREADS - 1) / THREADS, 2048));
    hipLaunchKernelGGL(sum_splits_kernel, dim3(blocks), dim3(THREADS), 0, s,
                       reinterpret_cast<const f32x4*>(part), reinterpret_cast<f32x4*>(C), n4, S);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t gemm_bf16(const float* A, const uint16_t* B, float* C, int M, int N, int K, float* part,
                     hipStream_t s) {
  return gemm_any(A, B, C, M, N, K, part, s);
}

hipError_t gemm_bf16(const uint16_t* A, const uint16_t* B, float* C, int M, int N, int K,
                     float* part, hipStream_t s) {
  return gemm_any(A, B, C, M, N, K, part, s);
}

hipError_t gemm_bf16_parts(const uint16_t* A, const uint16_t* B, float* C, int M, int N, int K,
                           float* part, hipStream_t s, int* splits) {
  const int S = split_count(M, N, K);
  if (M > band_rows(K) || S == 1) {
    *splits = 1;
    return gemm_any(A, B, C, M, N, K, part, s);
  }
  *splits = S;
  const int tiles = n_tiles(M, N);
  const int per = (tiles * S + kXcds - 1) / kXcds;
  const int k_chunk = ((K + S - 1) / S + BK - 1) / BK * BK;
  hipLaunchKernelGGL(gemm_bf16_kernel<uint16_t>, dim3(per * kXcds), dim3(THREADS), 0, s, A, B, part,
                     M, N, K, (N + BN - 1) / BN, per, tiles, tiles * S, k_chunk);
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

namespace {

template <typename PT>
hipError_t project_any(int T, int expand, int dv, int dv_virt, int d_out, const PT* pooled,
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

}  // namespace

hipError_t launch_project(int T, int expand, int dv, int dv_virt, int d_out, const float* pooled,
                          const uint16_t* w_proj, const uint16_t* w_out, float* out, void* ws,
                          hipStream_t s) {
  return project_any(T, expand, dv, dv_virt, d_out, pooled, w_proj, w_out, out, ws, s);
}

hipError_t launch_project(int T, int expand, int dv, int dv_virt, int d_out, const uint16_t* pooled,
                          const uint16_t* w_proj, const uint16_t* w_out, float* out, void* ws,
                          hipStream_t s) {
  return project_any(T, expand, dv, dv_virt, d_out, pooled, w_proj, w_out, out, ws, s);
}

}  // namespace umem
