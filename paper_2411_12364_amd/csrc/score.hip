// a1 + a2: per-axis selection scores.
//
// For head h and axis (row or column), S_rho[t, i] = sum_{d in slice rho} K[h, i, d] q[t, h, d]
// (eq. (2); with rank r the key/query dim holds r contiguous slices, eq. (4)).  The selection
// score is sum_rho f[rho] S_rho[t, i] with f = u (rows) or t (columns), the leading singular pair
// of the head's Tucker core (eqs. (6), (8), (9)); for the additive grid f = [1].
//
// Four kernels compute the same scores (dk in {64, 128, 256} take one of the first three):
//  * axis_scores_split (T <= 16): a workgroup covers 16 keys x 16 tokens of one (head, axis) on
//    v_mfma_f32_16x16x4_f32, and its 4 waves split the key/query dim into quarters.  Each lane
//    loads its key and query fragments straight into registers, so nothing waits on a barrier
//    before the MFMAs; the four partial tiles meet once in LDS.  Many small workgroups keep
//    several in flight per CU, which hides the memory latency that bounds small T.
//  * axis_scores_wide (16 < T <= 64): the same split of the dim, on v_mfma_f32_32x32x2f32 over
//    32 keys x 32 tokens: half the query fetches per key, and stores of 128-byte runs.
//  * axis_scores_mfma (larger T): a workgroup covers 64 keys x 16*MT tokens; each of its 4 waves
//    owns 16 keys and loads their key rows straight into registers, while the query tile is
//    staged once in LDS and shared by the waves.  Each key is read once per token tile.
//  * axis_scores_valu (any shape): a TT x TN tile on the vector ALUs, key and query tiles
//    streamed through LDS in chunks of DC dims.
// With a rank-r core each slice's partial scores are multiplied by their factor (u or t) before
// they are summed; for the additive grid the factor is 1.
#include <algorithm>

#include "umem_internal.h"

namespace umem {
namespace {

constexpr int TT = 32;       // tokens per tile
constexpr int TN = 64;       // keys per tile
constexpr int DC = 32;       // dims per LDS chunk
constexpr int LDS_STRIDE = DC + 4;   // floats per LDS row: float4-aligned, conflict-free b128 reads
constexpr int THREADS = 256;

// Clears zero[0, n4) (float4s) with every thread of the grid: the forward pools both heads into
// its output with atomic adds in the kernel that follows this one.
__device__ __forceinline__ void clear_with_grid(float4* __restrict__ zero, int n4) {
  if (zero == nullptr) return;
  const size_t nt = static_cast<size_t>(gridDim.x) * gridDim.y * gridDim.z * blockDim.x;
  const size_t gid = ((static_cast<size_t>(blockIdx.z) * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x) *
                         blockDim.x + threadIdx.x;
  for (size_t i = gid; i < static_cast<size_t>(n4); i += nt) zero[i] = make_float4(0.f, 0.f, 0.f, 0.f);
}

__global__ __launch_bounds__(THREADS) void axis_scores_valu(
    const float* __restrict__ q_row, const float* __restrict__ q_col,
    const float* __restrict__ k_row, const float* __restrict__ k_col,
    const float* __restrict__ factors, float* __restrict__ sel, int T, int H, int n, int dk,
    int rank, float4* __restrict__ zero, int zero_n4) {
  clear_with_grid(zero, zero_n4);
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

  if (tid < kMaxRank) fvec[tid] = factors ? factors[(h * 2 + axis) * kMaxRank + tid] : 1.0f;

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
    if (factors != nullptr) {
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


typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int MT, int NCH>
__global__ __launch_bounds__(THREADS) void axis_scores_mfma(
    const float* __restrict__ q_row, const float* __restrict__ q_col,
    const float* __restrict__ k_row, const float* __restrict__ k_col,
    const float* __restrict__ factors, float* __restrict__ sel, int T, int H, int n, int dk,
    int rank, float4* __restrict__ zero, int zero_n4) {
  clear_with_grid(zero, zero_n4);
  constexpr int TM = 16 * MT;
  extern __shared__ __align__(16) float qs[];    // [TM][dk + 4]
  __shared__ float fvec[kMaxRank];
  const int axis = blockIdx.z & 1;
  const int h = blockIdx.z >> 1;
  const float* __restrict__ q = axis ? q_col : q_row;
  const float* __restrict__ K = axis ? k_col : k_row;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int j = lane & 15;        // key within the wave's 16 (B column, D column)
  const int g = lane >> 4;        // 4-dim group within a 16-dim chunk
  const int key0 = blockIdx.x * 64 + wave * 16;
  const int t0 = blockIdx.y * TM;
  const int ldq = dk + 4;
  const int width = dk / rank;

  // this lane's key-row fragments: dims 16 c + 4 g .. + 3 of key key0 + j, all chunks
  const int key = key0 + j;
  const float* krow = K + (static_cast<size_t>(h) * n + (key < n ? key : 0)) * dk + 4 * g;
  float4 kf[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c)
    kf[c] = (key < n) ? *reinterpret_cast<const float4*>(krow + 16 * c)
                                 : make_float4(0.f, 0.f, 0.f, 0.f);
  // the query tile, shared by the four waves
  const int vec_per_row = dk / 4;
  for (int v = tid; v < TM * vec_per_row; v += THREADS) {
    const int r = v / vec_per_row, c4 = v - r * vec_per_row;
    float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
    if (t0 + r < T) x = *reinterpret_cast<const float4*>(q + (static_cast<size_t>(t0 + r) * H + h) * dk + 4 * c4);
    *reinterpret_cast<float4*>(qs + r * ldq + 4 * c4) = x;
  }
  if (tid < kMaxRank) fvec[tid] = factors ? factors[(h * 2 + axis) * kMaxRank + tid] : 1.0f;
  __syncthreads();

  f32x4 out[MT], acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    out[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  int rho = 0;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    {
      if (c > 0 && (16 * c) % width == 0) {     // a slice ends: fold it with its factor
        const float f = fvec[rho++];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          out[mt] += f * acc[mt];
          acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const float4 qf = *reinterpret_cast<const float4*>(qs + (mt * 16 + j) * ldq + 16 * c + 4 * g);
        acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(qf.x, kf[c].x, acc[mt], 0, 0, 0);
        acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(qf.y, kf[c].y, acc[mt], 0, 0, 0);
        acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(qf.z, kf[c].z, acc[mt], 0, 0, 0);
        acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(qf.w, kf[c].w, acc[mt], 0, 0, 0);
      }
    }
  }
  const float f = fvec[rho];
  // lane holds D[4 g + r][j]: token t0 + 16 mt + 4 g + r, key key0 + j
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    out[mt] += f * acc[mt];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = t0 + mt * 16 + 4 * g + r;
      // nontemporal: the scores stream through once, the keys should stay in L2
      if (t < T && key < n)
        __builtin_nontemporal_store(out[mt][r], sel + ((static_cast<size_t>(axis) * T + t) * H + h) * n + key);
    }
  }
}

template <int MT, int CPW>
__global__ __launch_bounds__(THREADS) void axis_scores_split(
    const float* __restrict__ q_row, const float* __restrict__ q_col,
    const float* __restrict__ k_row, const float* __restrict__ k_col,
    const float* __restrict__ factors, float* __restrict__ sel, int T, int H, int n, int dk,
    int rank, float4* __restrict__ zero, int zero_n4) {
  clear_with_grid(zero, zero_n4);
  constexpr int TM = 16 * MT;
  __shared__ f32x4 part[3][MT][kWave];       // partial D fragments of waves 1..3
  const int axis = blockIdx.z & 1;
  const int h = blockIdx.z >> 1;
  const float* __restrict__ q = axis ? q_col : q_row;
  const float* __restrict__ K = axis ? k_col : k_row;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int j = lane & 15;        // key within the 16 (B and D column); token within 16 for A
  const int g = lane >> 4;        // 4-dim group within a 16-dim chunk
  const int key = blockIdx.x * 16 + j;
  const int t0 = blockIdx.y * TM;
  const int d0 = wave * 16 * CPW + 4 * g;    // this lane's first dim

  // fragments: key rows of the 16 keys and query rows of the TM tokens, this wave's dims only
  f32x4 kf[CPW], qf[MT][CPW];
  const float* krow = K + (static_cast<size_t>(h) * n + (key < n ? key : n - 1)) * dk + d0;
#pragma unroll
  for (int c = 0; c < CPW; ++c) kf[c] = *reinterpret_cast<const f32x4*>(krow + 16 * c);
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int t = t0 + 16 * mt + j;
    const float* qrow = q + (static_cast<size_t>(t < T ? t : T - 1) * H + h) * dk + d0;
#pragma unroll
    for (int c = 0; c < CPW; ++c) qf[mt][c] = *reinterpret_cast<const f32x4*>(qrow + 16 * c);
  }
  f32x4 acc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < CPW; ++c) {
      acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(qf[mt][c].x, kf[c].x, acc[mt], 0, 0, 0);
      acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(qf[mt][c].y, kf[c].y, acc[mt], 0, 0, 0);
      acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(qf[mt][c].z, kf[c].z, acc[mt], 0, 0, 0);
      acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(qf[mt][c].w, kf[c].w, acc[mt], 0, 0, 0);
    }
  }
  // a wave's quarter of the dims lies in one slice (the launcher checks 4 % rank == 0): fold it
  if (factors != nullptr) {
    const float f = factors[(h * 2 + axis) * kMaxRank + (wave * 16 * CPW) / (dk / rank)];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] *= f;
  }
  if (wave > 0) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) part[wave - 1][mt][lane] = acc[mt];
  }
  __syncthreads();
  if (wave == 0) {
    // lane holds D[4 g + r][j]: token t0 + 16 mt + 4 g + r, key blockIdx.x * 16 + j
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const f32x4 o = ((acc[mt] + part[0][mt][lane]) + part[1][mt][lane]) + part[2][mt][lane];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = t0 + mt * 16 + 4 * g + r;
        if (t < T && key < n)
          __builtin_nontemporal_store(o[r], sel + ((static_cast<size_t>(axis) * T + t) * H + h) * n + key);
      }
    }
  }
}

typedef float f32x16 __attribute__((ext_vector_type(16)));

// Decode-sized T on v_mfma_f32_32x32x2f32: a workgroup covers 32 keys x 32 tokens of one (head,
// axis) and its 8 waves split the dim into eighths of DW = dk / 8.  Lane l (token / key l % 32,
// half l / 32) holds dims d0 + (l / 32) * DW/2 .. + DW/2 - 1 of its token and of its key, so
// MFMA i pairs dims d0 + i and d0 + DW/2 + i.  The eight partial tiles meet in LDS; wave w adds
// them (in wave order) for D registers 2w, 2w + 1 and stores 128-byte runs of keys.  Eight
// waves rather than four (or sixteen) halve each wave's chain of dependent MFMAs and loads
// (measured at decode-20M: 5.50 us with four, 5.19 with eight, 5.77 with sixteen).
constexpr int kWideWaves = 8;
template <int NV4>
__global__ __launch_bounds__(kWideWaves * kWave) void axis_scores_wide(
    const float* __restrict__ q_row, const float* __restrict__ q_col,
    const float* __restrict__ k_row, const float* __restrict__ k_col,
    const float* __restrict__ factors, float* __restrict__ sel, int T, int H, int n, int dk,
    int rank, float4* __restrict__ zero, int zero_n4) {
  clear_with_grid(zero, zero_n4);
  constexpr int HALF = 4 * NV4;                 // DW / 2 dims per lane
  __shared__ float part[kWideWaves][16][kWave];   // the waves' D fragments
  const int axis = blockIdx.z & 1;
  const int h = blockIdx.z >> 1;
  const float* __restrict__ q = axis ? q_col : q_row;
  const float* __restrict__ K = axis ? k_col : k_row;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int c = lane & 31, hh = lane >> 5;
  const int key = blockIdx.x * 32 + c;
  const int tok = blockIdx.y * 32 + c;
  const int d0 = wave * 2 * HALF + hh * HALF;
  f32x4 kf[NV4], qf[NV4];
  const float* krow = K + (static_cast<size_t>(h) * n + (key < n ? key : n - 1)) * dk + d0;
  const float* qrow = q + (static_cast<size_t>(tok < T ? tok : T - 1) * H + h) * dk + d0;
#pragma unroll
  for (int i = 0; i < NV4; ++i) kf[i] = *reinterpret_cast<const f32x4*>(krow + 4 * i);
#pragma unroll
  for (int i = 0; i < NV4; ++i) qf[i] = *reinterpret_cast<const f32x4*>(qrow + 4 * i);
  f32x16 acc;
#pragma unroll
  for (int j = 0; j < 16; ++j) acc[j] = 0.0f;
#pragma unroll
  for (int i = 0; i < NV4; ++i) {
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qf[i].x, kf[i].x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qf[i].y, kf[i].y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qf[i].z, kf[i].z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qf[i].w, kf[i].w, acc, 0, 0, 0);
  }
  // a wave's eighth of the dims lies in one slice (the launcher checks 8 % rank == 0): fold it
  if (factors != nullptr) {
    const float f = factors[(h * 2 + axis) * kMaxRank + (wave * 2 * HALF) / (dk / rank)];
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[j] *= f;
  }
#pragma unroll
  for (int j = 0; j < 16; ++j) part[wave][j][lane] = acc[j];
  __syncthreads();
  // D register j of lane l: token 8 (j / 4) + 4 (l / 32) + j % 4, key l % 32
#pragma unroll
  for (int jj = 0; jj < 16 / kWideWaves; ++jj) {
    const int j = (16 / kWideWaves) * wave + jj;
    float o = part[0][j][lane];
#pragma unroll
    for (int v = 1; v < kWideWaves; ++v) o += part[v][j][lane];
    const int t = blockIdx.y * 32 + 8 * (j / 4) + 4 * hh + j % 4;
    // nontemporal: the selection reads the scores from other XCDs, so this XCD's L2 has no use
    // for them (measured: decode-20M step 16.53 -> 16.29 us)
    if (t < T && key < n)
      __builtin_nontemporal_store(o, sel + ((static_cast<size_t>(axis) * T + t) * H + h) * n + key);
  }
}

// ---------------------------------------------------------------- scores on fp16 matrix cores
// For many tokens the scores are one GEMM per (head, axis): with the slice factors folded into
// the query (sum_rho f_rho sum_{d in rho} q_d K_d = sum_d (f_rho(d) q_d) K_d), S = Q' K^T with
// both operands rows of dk.  fp32 MFMA runs at 1/16 of the fp16 rate, so the GEMM is done on
// fp16 MFMA in fp32 precision.  Each row is first scaled by a power of two 2^s (exact) that puts
// its largest magnitude in [2^14, 2^15), which keeps every part below fp16's largest value and
// its small parts clear of fp16's subnormals; then each scaled x is split into two fp16 parts,
// x1 = fp16(x) (11 significant bits) and x2 = fp16(x - x1) (x - x1 is exact; x2 keeps its next
// 11 bits, so x - x1 - x2 is below 2^-22 |x|).  q . k = 2^-(s_q + s_k) (q1 k1 + q1 k2 + q2 k1):
// each product of two fp16 is exact in fp32, the MFMA accumulates in fp32, and the dropped
// product q2 k2 and the split's remainders are of order 2^-22 of the terms, below the fp32
// rounding of a plain fp32 product sum (measured on the workloads' inputs: 4e-8 to 1.1e-7 of
// sum |q_d k_d| against 2e-7 to 3.3e-7 for plain fp32).  The three products cost 3/16 of the
// fp32 MFMA time.
//
// split_planes_kernel writes the two planes of Q' and K and every row's exponent s in the
// workspace, per (axis, plane, head) a [rows, dk] block; axis_scores_planes is a 128 x 128 tile
// of (tokens x keys) per workgroup, four waves of 64 x 64 (4 x 4 v_mfma_f32_16x16x32_f16 tiles
// x 3 products), dk in steps of 32 through two LDS buffers (slice k + 1, prefetched into
// registers, is staged into one while slice k is multiplied from the other; one barrier per
// step), and the scores leave through LDS as whole 128-byte lines (nontemporal), each multiplied
// by its 2^-(s_q + s_k) on the way out.
constexpr int XT = 128, XN = 128, XK = 32;
constexpr int XLD = XK;                       // LDS pitch in fp16 (64-byte rows, chunks swizzled)
constexpr int XLDC = 64 + 4;                  // LDS pitch of the epilogue's fp32 rows
constexpr int XPL = 2;                        // fp16 planes per operand

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// The workspace blocks of the planes: Qp[axis][p][h][t][dk], Kp[axis][p][h][i][dk] (fp16 bits),
// then the rows' exponents Qs[axis][h][t], Ks[axis][h][i].
struct PlaneLayout {
  uint16_t* Qp;
  uint16_t* Kp;
  int32_t* Qs;
  int32_t* Ks;
};
__host__ __device__ inline size_t plane_elems(int T, int H, int n, int dk) {
  return static_cast<size_t>(2) * XPL * (static_cast<size_t>(T) + n) * H * dk;
}
PlaneLayout plane_layout(void* planes, int T, int H, int n, int dk) {
  PlaneLayout L;
  L.Qp = static_cast<uint16_t*>(planes);
  L.Kp = L.Qp + static_cast<size_t>(2) * XPL * T * H * dk;
  L.Qs = reinterpret_cast<int32_t*>(L.Qp + plane_elems(T, H, n, dk));
  L.Ks = L.Qs + static_cast<size_t>(2) * H * T;
  return L;
}

// One row per group of G lanes (G = 4 .. 64, a power of two, G >= dk / 8 unless dk > 512):
// queries (both axes, scaled by their slice factors) first, then keys.  A lane holds 8 dims per
// chunk, chunks c = lane + G j; the group's largest magnitude sets the row's exponent.
template <int G>
__global__ __launch_bounds__(THREADS) void split_planes_kernel(
    const float* __restrict__ q_row, const float* __restrict__ q_col,
    const float* __restrict__ k_row, const float* __restrict__ k_col,
    const float* __restrict__ factors, int T, int H, int n, int dk, int width, PlaneLayout L) {
  constexpr int kMaxChunks = 2;                    // dk <= 1024: at most 128 chunks of 8 over 64 lanes
  const int d8n = dk / 8;
  const int lg = threadIdx.x & (G - 1);
  const size_t nq = static_cast<size_t>(2) * T * H, rows_all = nq + static_cast<size_t>(2) * H * n;
  const size_t groups = static_cast<size_t>(gridDim.x) * (THREADS / G);
  for (size_t r = static_cast<size_t>(blockIdx.x) * (THREADS / G) + threadIdx.x / G; r < rows_all;
       r += groups) {
    // (the loop bound is uniform over a group: its G lanes take the same rows)
    const bool query = r < nq;
    int axis, h;
    size_t src_row, dst_row, rows;
    if (query) {
      h = static_cast<int>(r % H);
      const size_t at = r / H;
      axis = static_cast<int>(at / T);
      const size_t t = at % T;
      src_row = t * H + h;
      dst_row = static_cast<size_t>(h) * T + t;
      rows = static_cast<size_t>(H) * T;
    } else {
      const size_t y = r - nq;
      axis = static_cast<int>(y / (static_cast<size_t>(H) * n));
      src_row = y % (static_cast<size_t>(H) * n);
      h = static_cast<int>(src_row / n);
      dst_row = src_row;
      rows = static_cast<size_t>(H) * n;
    }
    const float* src = (query ? (axis ? q_col : q_row) : (axis ? k_col : k_row)) + src_row * dk;
    float v[kMaxChunks][8];
    float mx = 0.0f;
#pragma unroll
    for (int j = 0; j < kMaxChunks; ++j) {
      const int c = lg + G * j;
      if (c < d8n) {
        const float4 v0 = *reinterpret_cast<const float4*>(src + 8 * c);
        const float4 v1 = *reinterpret_cast<const float4*>(src + 8 * c + 4);
        float f = 1.0f;
        if (query && factors != nullptr) f = factors[(h * 2 + axis) * kMaxRank + (8 * c) / width];
        v[j][0] = v0.x * f; v[j][1] = v0.y * f; v[j][2] = v0.z * f; v[j][3] = v0.w * f;
        v[j][4] = v1.x * f; v[j][5] = v1.y * f; v[j][6] = v1.z * f; v[j][7] = v1.w * f;
#pragma unroll
        for (int e = 0; e < 8; ++e) mx = fmaxf(mx, fabsf(v[j][e]));
      }
    }
#pragma unroll
    for (int off = 1; off < G; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, kWave));
    // mx in [2^(k-1), 2^k) (frexp's exponent k): 2^(15 - k) puts it in [2^14, 2^15)
    const int sc = mx > 0.0f ? 15 - __builtin_amdgcn_frexp_expf(mx) : 0;
#pragma unroll
    for (int j = 0; j < kMaxChunks; ++j) {
      const int c = lg + G * j;
      if (c < d8n) {
        f16x8 p[XPL];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float x = ldexpf(v[j][e], sc);                       // exact
          const _Float16 a = static_cast<_Float16>(x);
          p[0][e] = a;
          p[1][e] = static_cast<_Float16>(x - static_cast<float>(a));   // x - a is exact
        }
        uint16_t* dst = query ? L.Qp : L.Kp;
#pragma unroll
        for (int pl = 0; pl < XPL; ++pl)
          *reinterpret_cast<f16x8*>(dst + ((static_cast<size_t>(axis) * XPL + pl) * rows + dst_row) * dk + 8 * c) = p[pl];
      }
    }
    if (lg == 0) (query ? L.Qs : L.Ks)[static_cast<size_t>(axis) * rows + dst_row] = sc;
  }
}

// One 16-byte piece per thread and plane-row chunk: piece f of 2 * 128 * 4 (plane f / 512, row
// (f % 512) / 4, dims 8 (f % 4) ..), four per thread per operand.
struct XSlice {
  u32x4 a[2 * XPL], b[2 * XPL];
};

// Where 16-byte chunk ch of tile row `row` sits in LDS: the chunk index is XORed with row bits
// 1..3, so that the eight (or sixteen) lanes an LDS cycle serves, rows r..r+7 of one chunk when
// fragments are read and rows r, r+1 (r..r+3) of all four chunks when tiles are staged, fall on
// distinct banks with 32 (or 64) banks of 4 bytes.
__device__ __forceinline__ int x_pos(int row, int ch) {
  return row * XLD + 8 * (ch ^ (((row >> 1) ^ (row >> 3)) & 3));
}

// The tile's next K-slice (32 dims) of the two planes of Q' (tokens t0..) and K (keys i0..) into
// registers.  Buffer loads over one (axis, plane, head) block each: rows past T (or n) fall
// outside the block's range and read as zeros, and the addresses are 32-bit lane offsets on
// scalar bases (no 64-bit address per load to keep live).
__device__ __forceinline__ void x_fetch(const uint16_t* __restrict__ Qa, const uint16_t* __restrict__ Kb,
                                        size_t qplane, size_t kplane, int T, int n, int dk,
                                        int t0, int i0, int k0, int tid, XSlice& sl) {
  static_assert(THREADS == 256, "a thread's pieces: planes j / 2, rows tid / 4 + 64 (j % 2)");
  const uint32_t qbytes = static_cast<uint32_t>(T) * dk * 2u, kbytes = static_cast<uint32_t>(n) * dk * 2u;
#pragma unroll
  for (int j = 0; j < 2 * XPL; ++j) {
    const int pl = j >> 1, row = (tid >> 2) + 64 * (j & 1), col = k0 + 8 * (tid & 3);
    const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(Qa + pl * qplane), static_cast<short>(0), static_cast<int>(qbytes), 0x00020000);
    const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(Kb + pl * kplane), static_cast<short>(0), static_cast<int>(kbytes), 0x00020000);
    sl.a[j] = __builtin_amdgcn_raw_buffer_load_b128(ra, static_cast<uint32_t>((t0 + row) * dk + col) * 2u, 0, 0);
    sl.b[j] = __builtin_amdgcn_raw_buffer_load_b128(rb, static_cast<uint32_t>((i0 + row) * dk + col) * 2u, 0, 0);
  }
}

__global__ __launch_bounds__(THREADS) void axis_scores_planes(
    PlaneLayout L, float* __restrict__ sel, int T, int H, int n, int dk, float4* __restrict__ zero,
    int zero_n4) {
  clear_with_grid(zero, zero_n4);
  // two buffers of [A | B][plane][row][k] during the K-steps, the waves' fp32 output rows in the
  // epilogue
  constexpr int kTileElems = 2 * XPL * XT * XLD, kOutElems = 4 * 32 * XLDC * 2;
  __shared__ __align__(16) uint16_t smem[2 * kTileElems > kOutElems ? 2 * kTileElems : kOutElems];
  __shared__ int32_t sexp[XT + XN];                               // the tile's row exponents
  // Tiles in (key tile, token tile, head/axis) order, dealt to the eight XCDs in contiguous runs
  // (workgroups go to XCDs round-robin): each XCD walks its own token tiles against every key tile
  // of a head and axis, so both operands' planes are reused from its L2.  The grid is persistent
  // (8 gx workgroups, gx per XCD): workgroup s of an XCD takes the XCD's tiles s, s + gx, ...; the
  // first slice of the next tile and its row exponents are fetched during the last K-step.
  const int nx = (n + XN - 1) / XN, ny = (T + XT - 1) / XT;
  const int ntiles = nx * ny * 2 * H;
  const int xcd = blockIdx.x & 7, gx = gridDim.x >> 3, per = ntiles >> 3, extra = ntiles & 7;
  const int first = xcd * per + min(xcd, extra), cnt = per + (xcd < extra ? 1 : 0);
  int jt = blockIdx.x >> 3;                              // this workgroup's tiles: jt, jt + gx, ...
  if (jt >= cnt) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;              // 64 tokens x 64 keys of the tile
  const size_t qplane = static_cast<size_t>(H) * T * dk, kplane = static_cast<size_t>(H) * n * dk;
  auto coords = [&](int u, int& axis, int& h, int& i0, int& t0, const uint16_t*& Qa, const uint16_t*& Kb) {
    const int tz = u / (nx * ny), txy = u - tz * (nx * ny);
    axis = tz & 1;
    h = tz >> 1;
    i0 = (txy % nx) * XN;
    t0 = (txy / nx) * XT;
    Qa = L.Qp + static_cast<size_t>(axis) * XPL * qplane + static_cast<size_t>(h) * T * dk;
    Kb = L.Kp + static_cast<size_t>(axis) * XPL * kplane + static_cast<size_t>(h) * n * dk;
  };
  // thread tid's row exponent of a tile: token row t0 + tid (tid < XT), key row i0 + tid - XT
  auto exponent = [&](int axis, int h, int i0, int t0) {
    const int rr = tid < XT ? t0 + tid : i0 + tid - XT;
    if (tid < XT ? rr >= T : rr >= n) return 0;
    return tid < XT ? L.Qs[(static_cast<size_t>(axis) * H + h) * T + rr]
                    : L.Ks[(static_cast<size_t>(axis) * H + h) * n + rr];
  };
  auto stage = [&](const XSlice& sl, uint16_t* buf) {
#pragma unroll
    for (int j = 0; j < 2 * XPL; ++j) {
      const int f = tid + THREADS * j;
      const int pl = f >> 9, row = (f & 511) >> 2, ch = f & 3;
      *reinterpret_cast<u32x4*>(buf + pl * XT * XLD + x_pos(row, ch)) = sl.a[j];
      *reinterpret_cast<u32x4*>(buf + XPL * XT * XLD + pl * XN * XLD + x_pos(row, ch)) = sl.b[j];
    }
  };
  int axis, h, i0, t0;
  const uint16_t *Qa, *Kb;
  coords(first + jt, axis, h, i0, t0, Qa, Kb);
  XSlice sl;
  x_fetch(Qa, Kb, qplane, kplane, T, n, dk, t0, i0, 0, tid, sl);
  int32_t e_mine = exponent(axis, h, i0, t0);
  while (true) {
    const bool has_next = jt + gx < cnt;
    int naxis = 0, nh = 0, ni0 = 0, nt0 = 0;
    const uint16_t *nQa = Qa, *nKb = Kb;
    if (has_next) coords(first + jt + gx, naxis, nh, ni0, nt0, nQa, nKb);
    stage(sl, smem);                                    // slice 0 (fetched earlier) into buffer 0
    sexp[tid] = e_mine;
    __syncthreads();
    if (XK < dk) x_fetch(Qa, Kb, qplane, kplane, T, n, dk, t0, i0, XK, tid, sl);
    else if (has_next) x_fetch(nQa, nKb, qplane, kplane, T, n, dk, nt0, ni0, 0, tid, sl);
    if (has_next) e_mine = exponent(naxis, nh, ni0, nt0);
    f32x4 acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
    int buf = 0;
    for (int k0 = 0; k0 < dk; k0 += XK) {
      const uint16_t* As = smem + buf * kTileElems;
      const uint16_t* Bs = As + XPL * XT * XLD;
      // lane: row (token or key) lane % 16 of a 16-block, dims 8 (lane / 16) ... + 7
      f16x8 af[XPL][4], bfr[XPL][4];
#pragma unroll
      for (int pl = 0; pl < XPL; ++pl)
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          af[pl][a] = *reinterpret_cast<const f16x8*>(As + pl * XT * XLD + x_pos(wm * 64 + a * 16 + (lane & 15), lane >> 4));
          bfr[pl][a] = *reinterpret_cast<const f16x8*>(Bs + pl * XN * XLD + x_pos(wn * 64 + a * 16 + (lane & 15), lane >> 4));
        }
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          // the three products of significance 2^-11 and above, smaller ones first
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[1][a], bfr[0][b], acc[a][b], 0, 0, 0);
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[0][a], bfr[1][b], acc[a][b], 0, 0, 0);
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_f16(af[0][a], bfr[0][b], acc[a][b], 0, 0, 0);
        }
      // slice k + 1 (in registers) into the other buffer while these MFMAs run; one barrier
      if (k0 + XK < dk) stage(sl, smem + (buf ^ 1) * kTileElems);
      __syncthreads();
      if (k0 + 2 * XK < dk) x_fetch(Qa, Kb, qplane, kplane, T, n, dk, t0, i0, k0 + 2 * XK, tid, sl);
      else if (k0 + XK < dk && has_next) x_fetch(nQa, nKb, qplane, kplane, T, n, dk, nt0, ni0, 0, tid, sl);
      buf ^= 1;
    }
    // D layout: lane holds tokens 4 (lane / 16) + r of key lane % 16.  Each wave's 64 x 64 block
    // leaves in two halves of 32 tokens through LDS (free after the last barrier), as 16-byte
    // pieces: every token's 64 keys are 256 contiguous bytes of sel.
    float* Cs = reinterpret_cast<float*>(smem) + wave * 32 * XLDC;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
#pragma unroll
      for (int a2 = 0; a2 < 2; ++a2)
#pragma unroll
        for (int b = 0; b < 4; ++b)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            Cs[(a2 * 16 + 4 * (lane >> 4) + r) * XLDC + b * 16 + (lane & 15)] = acc[half * 2 + a2][b][r];
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
      for (int it = 0; it < 8; ++it) {
        const int row = (lane >> 4) + 4 * it, c4 = (lane & 15) * 4;
        const int tl = wm * 64 + half * 32 + row, kl = wn * 64 + c4;
        const int t = t0 + tl, key = i0 + kl;
        f32x4 v = *reinterpret_cast<const f32x4*>(Cs + row * XLDC + c4);
        const int eq = sexp[tl];
        v.x = ldexpf(v.x, -(eq + sexp[XT + kl]));                     // exact
        v.y = ldexpf(v.y, -(eq + sexp[XT + kl + 1]));
        v.z = ldexpf(v.z, -(eq + sexp[XT + kl + 2]));
        v.w = ldexpf(v.w, -(eq + sexp[XT + kl + 3]));
        if (t < T && key < n)      // n % 4 == 0: the piece is whole
          __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(sel + ((static_cast<size_t>(axis) * T + t) * H + h) * n + key));
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    if (!has_next) break;
    jt += gx;
    axis = naxis;
    h = nh;
    i0 = ni0;
    t0 = nt0;
    Qa = nQa;
    Kb = nKb;
    __syncthreads();          // the epilogue's LDS rows and sexp are free before the next tile
  }
}

bool scores_use_planes(const umem_desc& d, int T) {
  return T > 64 && d.dk % XK == 0 && d.n_keys % 4 == 0 && (d.dk / d.rank) % 8 == 0;
}

}  // namespace

// One thread per head; with multi-core scoring the head's component cores are summed first
// (eq. (16)): the singular pair of the whole core drives the retrieval.
__global__ void rank1_kernel(const float* __restrict__ core, int H, int r, int parts,
                             float* __restrict__ factors) {
  const int h = threadIdx.x;
  if (h < H) {
    float* f = factors + h * 2 * kMaxRank;
    rank1_factors(core + static_cast<size_t>(h) * parts * r * r, r, parts, f, f + kMaxRank);
  }
}

hipError_t launch_rank1(const umem_desc& d, const float* core, float* factors, hipStream_t s) {
  clear_stale_error();
  hipLaunchKernelGGL(rank1_kernel, dim3(1), dim3(kWave), 0, s, core, d.heads, d.rank, n_cores(d),
                     factors);
  return hipGetLastError();
}

size_t score_planes_bytes(const umem_desc& d, int T) {
  if (!scores_use_planes(d, T)) return 0;
  return plane_elems(T, d.heads, d.n_keys, d.dk) * sizeof(uint16_t) +
         static_cast<size_t>(2) * (static_cast<size_t>(T) + d.n_keys) * d.heads * sizeof(int32_t);
}

hipError_t launch_axis_scores(const umem_desc& d, int T, const float* q_row, const float* q_col,
                              const float* k_row, const float* k_col, const float* factors,
                              float* sel, float* zero_out, size_t zero_floats, void* planes,
                              hipStream_t s) {
  float4* zero = reinterpret_cast<float4*>(zero_out);
  const int zero_n4 = zero_out ? static_cast<int>(zero_floats / 4) : 0;
  clear_stale_error();
  if (T == 0) return hipSuccess;
  const float* c = (d.grid == UMEM_GRID_TUCKER) ? factors : nullptr;
  const int width = d.dk / d.rank;
  if ((d.dk == 64 || d.dk == 128 || d.dk == 256) && width % 16 == 0 && T <= 16 &&
      4 % d.rank == 0) {
    dim3 grid((d.n_keys + 15) / 16, 1, d.heads * 2);
#define UMEM_SPLIT(CPW)                                                                          \
  hipLaunchKernelGGL((axis_scores_split<1, CPW>), grid, dim3(THREADS), 0, s, q_row, q_col,       \
                     k_row, k_col, c, sel, T, d.heads, d.n_keys, d.dk, d.rank, zero, zero_n4)
    if (d.dk == 64) UMEM_SPLIT(1);
    else if (d.dk == 128) UMEM_SPLIT(2);
    else UMEM_SPLIT(4);
#undef UMEM_SPLIT
    return hipGetLastError();
  }
  if ((d.dk == 64 || d.dk == 128 || d.dk == 256) && T > 16 && T <= 64 && kWideWaves % d.rank == 0) {
    dim3 grid((d.n_keys + 31) / 32, (T + 31) / 32, d.heads * 2);
#define UMEM_WIDE(NV4)                                                                            \
  hipLaunchKernelGGL((axis_scores_wide<NV4>), grid, dim3(kWideWaves * kWave), 0, s, q_row,       \
                     q_col, k_row, k_col, c, sel, T, d.heads, d.n_keys, d.dk, d.rank, zero,     \
                     zero_n4)
    if (d.dk == 64) UMEM_WIDE(1);
    else if (d.dk == 128) UMEM_WIDE(2);
    else UMEM_WIDE(4);
#undef UMEM_WIDE
    return hipGetLastError();
  }
  // (the plane kernel stores 16-byte pieces of sel)
  if (scores_use_planes(d, T) && planes != nullptr && reinterpret_cast<uintptr_t>(sel) % 16 == 0) {
    const PlaneLayout L = plane_layout(planes, T, d.heads, d.n_keys, d.dk);
    const size_t rows = static_cast<size_t>(2) * (static_cast<size_t>(T) + d.n_keys) * d.heads;
    const int d8n = d.dk / 8;                      // 4 .. 128 (dk % 32 == 0, dk <= 1024)
    const int G = d8n <= 4 ? 4 : (d8n <= 8 ? 8 : (d8n <= 16 ? 16 : (d8n <= 32 ? 32 : 64)));
    const unsigned blocks = static_cast<unsigned>(std::min<size_t>((rows * G + THREADS - 1) / THREADS, 8192));
#define UMEM_SPLIT_PLANES(GG)                                                                      \
  hipLaunchKernelGGL(split_planes_kernel<GG>, dim3(blocks), dim3(THREADS), 0, s, q_row, q_col,      \
                     k_row, k_col, c, T, d.heads, d.n_keys, d.dk, d.dk / d.rank, L)
    if (G == 4) UMEM_SPLIT_PLANES(4);
    else if (G == 8) UMEM_SPLIT_PLANES(8);
    else if (G == 16) UMEM_SPLIT_PLANES(16);
    else if (G == 32) UMEM_SPLIT_PLANES(32);
    else UMEM_SPLIT_PLANES(64);
#undef UMEM_SPLIT_PLANES
    // a persistent grid of 8 gx workgroups (two per CU, as registers allow), gx per XCD
    const long long ntiles = static_cast<long long>((d.n_keys + XN - 1) / XN) * ((T + XT - 1) / XT) * d.heads * 2;
    const dim3 grid(static_cast<unsigned>(8 * std::min<long long>((ntiles + 7) / 8, 64)));
    hipLaunchKernelGGL(axis_scores_planes, grid, dim3(THREADS), 0, s, L, sel, T, d.heads, d.n_keys,
                       d.dk, zero, zero_n4);
    return hipGetLastError();
  }
  // the key widths of the paper's UltraMem models (Kdim 256, 384, 448) and smaller powers of two
  if ((d.dk == 64 || d.dk == 128 || d.dk == 256 || d.dk == 384 || d.dk == 448) && width % 16 == 0) {
    int mt = T <= 16 ? 1 : (T <= 32 ? 2 : 4);
    while (mt > 1 && static_cast<size_t>(16 * mt) * (d.dk + 4) * 4 > 65536) mt /= 2;
    const size_t lds = static_cast<size_t>(16 * mt) * (d.dk + 4) * 4;
    dim3 grid((d.n_keys + 63) / 64, (T + 16 * mt - 1) / (16 * mt), d.heads * 2);
#define UMEM_SCORE(MT, NCH)                                                                      \
  hipLaunchKernelGGL((axis_scores_mfma<MT, NCH>), grid, dim3(THREADS), lds, s, q_row, q_col,     \
                     k_row, k_col, c, sel, T, d.heads, d.n_keys, d.dk, d.rank, zero, zero_n4)
#define UMEM_SCORE_DK(MT)                  \
  if (d.dk == 64) UMEM_SCORE(MT, 4);       \
  else if (d.dk == 128) UMEM_SCORE(MT, 8); \
  else if (d.dk == 256) UMEM_SCORE(MT, 16); \
  else if (d.dk == 384) UMEM_SCORE(MT, 24); \
  else UMEM_SCORE(MT, 28)
    if (mt == 1) { UMEM_SCORE_DK(1); }
    else if (mt == 2) { UMEM_SCORE_DK(2); }
    else { UMEM_SCORE_DK(4); }
#undef UMEM_SCORE_DK
#undef UMEM_SCORE
    return hipGetLastError();
  }
  dim3 grid((d.n_keys + TN - 1) / TN, (T + TT - 1) / TT, d.heads * 2);
  hipLaunchKernelGGL(axis_scores_valu, grid, dim3(THREADS), 0, s, q_row, q_col, k_row, k_col, c,
                     sel, T, d.heads, d.n_keys, d.dk, d.rank, zero, zero_n4);
  return hipGetLastError();
}

}  // namespace umem
