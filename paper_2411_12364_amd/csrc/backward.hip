// Backward of the gather-sum (eq. (1), eq. (15) per virtual block, eq. (17) per column slice):
// the weight gradients dw[e] = <d_pooled[t_e, p_e], V[row_e]> (per slice with multi-core
// scoring) and the value-row gradients dV[row] += sum over the entries e on that row of
// w_e d_pooled[t_e, p_e].
//
// The T * bag entries are keyed by physical row and stably sorted (sort.hip), so the entries of
// one row form a run in their original order.  The first wave of each run reads V[row] once,
// 16 bytes per lane at a time, and for each entry of the run in order computes its weight
// gradient (a wave reduction per core) and adds w_e d_pooled into an fp32 accumulator; then it
// adds the accumulator into dV[row].  Every row has one writer and a fixed summation order: the
// result does not depend on timing, and no atomics are needed.
//
// Backward of the scores (eqs. (2)-(4), (10), (16)) with the selection held fixed: one
// workgroup per (token, head) turns the weight gradients into grid-score gradients (SoftMax
// Jacobian where eq. (3)'s SoftMax weights), recomputes the selected slots' per-slice scores
// (Tucker), forms each slot's contribution to dS_row / dS_col and to dC, adds the contributions
// of slots that share a row (or column) in slot order, and writes dq = sum_i dS[i] K[i].  The key
// gradients dK[i] += dS[i] q are sums over tokens: each (token, head, axis) emits one entry per
// distinct key, the entries are stably sorted by key, and one wave per key sums them in order.
// dC sums its per-token partials in a fixed order (chunks of tokens, then the chunks).
#include <algorithm>

#include "umem_internal.h"

namespace umem {
namespace {

constexpr int THREADS = 256;
constexpr int NWAVES = THREADS / kWave;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(THREADS) void bwd_keys_kernel(const int32_t* __restrict__ idx,
                                                           const int32_t* __restrict__ perm,
                                                           int64_t n_values, int M,
                                                           uint32_t* __restrict__ keys,
                                                           uint32_t* __restrict__ vals) {
  for (int e = blockIdx.x * THREADS + threadIdx.x; e < M; e += gridDim.x * THREADS) {
    const int32_t x = idx[e];
    keys[e] = perm != nullptr ? static_cast<uint32_t>(perm[x] % n_values) : static_cast<uint32_t>(x);
    vals[e] = static_cast<uint32_t>(e);
  }
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

template <typename Elem>
struct Chunk;
template <>
struct Chunk<float> {
  static constexpr int kElems = 4;
  __device__ static inline void load(const float* p, float* x) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(p);
    x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
  }
};
template <>
struct Chunk<uint16_t> {   // bf16 bit patterns
  static constexpr int kElems = 8;
  __device__ static inline void load(const uint16_t* p, float* x) {
    const u32x4 r = *reinterpret_cast<const u32x4*>(p);
    const uint32_t q[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(q[i] << 16);
      x[2 * i + 1] = __uint_as_float(q[i] & 0xFFFF0000u);
    }
  }
};

template <typename Elem>
__global__ __launch_bounds__(THREADS) void gather_bwd_run_kernel(
    const uint32_t* __restrict__ rows, const uint32_t* __restrict__ ents, int M,
    const Elem* __restrict__ values, int dv, const int32_t* __restrict__ idx,
    const float* __restrict__ w, const int32_t* __restrict__ perm, int64_t n_values, int expand,
    int cores, int bag, const float* __restrict__ d_pooled, float* __restrict__ d_values,
    float* __restrict__ dw) {
  constexpr int EPC = Chunk<Elem>::kElems;            // elements per 16-byte piece
  const int lane = threadIdx.x & (kWave - 1);
  const int i = blockIdx.x * NWAVES + static_cast<int>(threadIdx.x) / kWave;
  if (i >= M) return;                                 // whole waves: no barrier in this kernel
  const uint32_t row = rows[i];
  if (i > 0 && rows[i - 1] == row) return;            // not the first entry of its run
  int end = i + 1;                                    // the run is [i, end)
  for (int base = i + 1; base < M; base += kWave) {
    const int pos = base + lane;
    const uint64_t same = __ballot(pos < M && rows[pos] == row);
    if (same != ~0ull) {
      end = base + __builtin_ctzll(~same);
      break;
    }
    end = min(M, base + kWave);
  }
  const int slice_w = dv / cores;
  const Elem* vrow = values + static_cast<size_t>(row) * dv;
  float* grow = d_values + static_cast<size_t>(row) * dv;
  for (int c0 = 0; c0 < dv; c0 += kWave * EPC) {
    const int col = c0 + lane * EPC;
    const bool active = col < dv;
    const int sl = active ? col / slice_w : 0;        // a piece lies in one column slice
    float x[EPC];
    if (active) {
      Chunk<Elem>::load(vrow + col, x);
    } else {
#pragma unroll
      for (int k = 0; k < EPC; ++k) x[k] = 0.0f;
    }
    float acc[EPC];
#pragma unroll
    for (int k = 0; k < EPC; ++k) acc[k] = 0.0f;
    for (int e = i; e < end; ++e) {
      const int ent = static_cast<int>(ents[e]);
      const int t = ent / bag;
      const int p = perm != nullptr ? static_cast<int>(perm[idx[ent]] / n_values) : 0;
      float g[EPC];
      float dot = 0.0f;
      if (active) {
        const float* src = d_pooled + (static_cast<size_t>(t) * expand + p) * dv + col;
#pragma unroll
        for (int k = 0; k < EPC; k += 4) {
          const f32x4 v = *reinterpret_cast<const f32x4*>(src + k);
          g[k] = v.x; g[k + 1] = v.y; g[k + 2] = v.z; g[k + 3] = v.w;
        }
#pragma unroll
        for (int k = 0; k < EPC; ++k) dot = fmaf(g[k], x[k], dot);
      } else {
#pragma unroll
        for (int k = 0; k < EPC; ++k) g[k] = 0.0f;
      }
      const float wt = active ? w[static_cast<size_t>(ent) * cores + sl] : 0.0f;
#pragma unroll
      for (int k = 0; k < EPC; ++k) acc[k] = fmaf(wt, g[k], acc[k]);
      for (int c = 0; c < cores; ++c) {
        const float s = wave_sum(sl == c ? dot : 0.0f);
        if (lane == 0) {
          float* d = dw + static_cast<size_t>(ent) * cores + c;
          *d = c0 == 0 ? s : *d + s;                  // this wave is the entry's only writer
        }
      }
    }
    if (active) {
#pragma unroll
      for (int k = 0; k < EPC; k += 4) {
        f32x4* dst = reinterpret_cast<f32x4*>(grow + col + k);
        f32x4 v = *dst;
        v.x += acc[k]; v.y += acc[k + 1]; v.z += acc[k + 2]; v.w += acc[k + 3];
        *dst = v;
      }
    }
  }
}

// ---------------------------------------------------------------- score backward

constexpr int kDcChunk = 256;          // tokens per first-level dC partial sum

struct ScoreBwdShared {
  int ii[kMaxTopM], jj[kMaxTopM];                  // row, column of each selected slot
  float dg[kMaxTopM * kMaxCores];                  // grid-score gradient per slot (and core)
  float srow[kMaxTopM][kMaxRank], scol[kMaxTopM][kMaxRank];   // the slots' per-slice scores
  float cr[kMaxTopM][kMaxRank], cc[kMaxTopM][kMaxRank];       // a slot's dS_row, dS_col terms
  int lead_r[kMaxTopM], lead_c[kMaxTopM];          // first slot with the same row / column
  int dist_r[kMaxTopM], dist_c[kMaxTopM];          // distinct rows / columns, in slot order
  int pos_r[kMaxTopM], pos_c[kMaxTopM];            // a leader's place in that list
  float dsr[kMaxTopM][kMaxRank], dsc[kMaxTopM][kMaxRank];     // dS per distinct row / column
  float core[kMaxCores][kMaxRank * kMaxRank];
  float red[THREADS];
  int nr, nc;
};

__global__ __launch_bounds__(THREADS) void score_bwd_kernel(
    const float* __restrict__ q_row, const float* __restrict__ q_col,
    const float* __restrict__ k_row, const float* __restrict__ k_col,
    const float* __restrict__ core_all, const int32_t* __restrict__ idx,
    const float* __restrict__ w, const float* __restrict__ dw, int T, int H, int n, int dk,
    int rank, int m, int tucker, int softmax, int hc, float* __restrict__ dq_row,
    float* __restrict__ dq_col, uint32_t* __restrict__ ekeys, uint32_t* __restrict__ evals,
    float* __restrict__ edS, float* __restrict__ dc_part) {
  __shared__ ScoreBwdShared sh;
  const int tid = threadIdx.x;
  const int t = blockIdx.x / H, h = blockIdx.x % H;
  const size_t th = static_cast<size_t>(t) * H + h;
  for (int s = tid; s < m; s += THREADS) {
    const int flat = idx[th * m + s];
    sh.ii[s] = flat / n;
    sh.jj[s] = flat % n;
  }
  if (tucker)
    for (int x = tid; x < hc * rank * rank; x += THREADS)
      sh.core[x / (rank * rank)][x % (rank * rank)] =
          core_all[static_cast<size_t>(h) * hc * rank * rank + x];
  // ---- weight gradients -> grid-score gradients
  if (softmax) {
    float p = 0.0f;
    for (int s = tid; s < m; s += THREADS) p = fmaf(w[th * m + s], dw[th * m + s], p);
    sh.red[tid] = p;
    __syncthreads();
    for (int off = THREADS / 2; off > 0; off >>= 1) {     // fixed-order tree
      if (tid < off) sh.red[tid] += sh.red[tid + off];
      __syncthreads();
    }
    const float wdot = sh.red[0];
    for (int s = tid; s < m; s += THREADS) sh.dg[s] = w[th * m + s] * (dw[th * m + s] - wdot);
  } else {
    for (int x = tid; x < m * hc; x += THREADS) sh.dg[x] = dw[th * m * hc + x];
  }
  __syncthreads();
  // ---- Tucker: the selected slots' per-slice scores, four lanes per (axis, slot) key row
  if (tucker) {
    const int width = dk / rank, n4 = dk >> 2;
    for (int job = tid; job < 8 * m; job += THREADS) {   // whole quads: 8m is a multiple of 4
      const int part = job & 3, row = job >> 2;
      const int axis = row >= m, s = row - (axis ? m : 0);
      const int key = axis ? sh.jj[s] : sh.ii[s];
      const float4* kr = reinterpret_cast<const float4*>((axis ? k_col : k_row) + (static_cast<size_t>(h) * n + key) * dk);
      const float4* qr = reinterpret_cast<const float4*>((axis ? q_col : q_row) + th * dk);
      float acc[kMaxRank] = {0.0f, 0.0f, 0.0f, 0.0f};
      const int f1 = ((part + 1) * n4) >> 2;
      for (int f = (part * n4) >> 2; f < f1; ++f) {
        const float4 kv = kr[f], qv = qr[f];
        float d = kv.x * qv.x;
        d = fmaf(kv.y, qv.y, d);
        d = fmaf(kv.z, qv.z, d);
        d = fmaf(kv.w, qv.w, d);
        const int rho = (4 * f) / width;
#pragma unroll
        for (int r = 0; r < kMaxRank; ++r) acc[r] += rho == r ? d : 0.0f;
      }
#pragma unroll
      for (int r = 0; r < kMaxRank; ++r) {
        acc[r] += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, acc[r]), 0xB1, 0xF, 0xF, false));
        acc[r] += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, acc[r]), 0x4E, 0xF, 0xF, false));
      }
      if (part == 0)
        for (int r = 0; r < rank; ++r) (axis ? sh.scol : sh.srow)[s][r] = acc[r];
    }
    __syncthreads();
  }
  // ---- each slot's dS terms, and which slot first holds its row / column
  for (int s = tid; s < m; s += THREADS) {
    if (!tucker) {
      sh.cr[s][0] = sh.dg[s];
      sh.cc[s][0] = sh.dg[s];
    } else {
      for (int r = 0; r < rank; ++r) {
        float a = 0.0f, b = 0.0f;
        for (int c = 0; c < hc; ++c) {
          float ca = 0.0f, cb = 0.0f;
          for (int x = 0; x < rank; ++x) {
            ca = fmaf(sh.core[c][r * rank + x], sh.scol[s][x], ca);   // (C S_col)[r]
            cb = fmaf(sh.core[c][x * rank + r], sh.srow[s][x], cb);   // (C^T S_row)[r]
          }
          a = fmaf(sh.dg[s * hc + c], ca, a);
          b = fmaf(sh.dg[s * hc + c], cb, b);
        }
        sh.cr[s][r] = a;
        sh.cc[s][r] = b;
      }
    }
    int lr = s, lc = s;
    for (int x = s - 1; x >= 0; --x) {
      if (sh.ii[x] == sh.ii[s]) lr = x;
      if (sh.jj[x] == sh.jj[s]) lc = x;
    }
    sh.lead_r[s] = lr;
    sh.lead_c[s] = lc;
  }
  __syncthreads();
  if (tucker)       // dC partial of this (token, head): slots in order
    for (int x = tid; x < hc * rank * rank; x += THREADS) {
      const int c = x / (rank * rank), r = (x / rank) % rank, z = x % rank;
      float a = 0.0f;
      for (int s = 0; s < m; ++s) a = fmaf(sh.dg[s * hc + c], sh.srow[s][r] * sh.scol[s][z], a);
      dc_part[th * hc * rank * rank + x] = a;
    }
  for (int s = tid; s < m; s += THREADS) {
    if (sh.lead_r[s] == s) {
      int pos = 0;
      for (int x = 0; x < s; ++x) pos += sh.lead_r[x] == x;
      sh.pos_r[s] = pos;
      sh.dist_r[pos] = sh.ii[s];
    }
    if (sh.lead_c[s] == s) {
      int pos = 0;
      for (int x = 0; x < s; ++x) pos += sh.lead_c[x] == x;
      sh.pos_c[s] = pos;
      sh.dist_c[pos] = sh.jj[s];
    }
  }
  if (tid == 0) {
    int a = 0, b = 0;
    for (int s = 0; s < m; ++s) {
      a += sh.lead_r[s] == s;
      b += sh.lead_c[s] == s;
    }
    sh.nr = a;
    sh.nc = b;
  }
  __syncthreads();
  // ---- dS per distinct row / column: its slots' terms in slot order
  for (int s = tid; s < m; s += THREADS) {
    if (sh.lead_r[s] == s)
      for (int r = 0; r < rank; ++r) {
        float a = 0.0f;
        for (int x = s; x < m; ++x) a += sh.lead_r[x] == s ? sh.cr[x][r] : 0.0f;
        sh.dsr[sh.pos_r[s]][r] = a;
      }
    if (sh.lead_c[s] == s)
      for (int r = 0; r < rank; ++r) {
        float a = 0.0f;
        for (int x = s; x < m; ++x) a += sh.lead_c[x] == s ? sh.cc[x][r] : 0.0f;
        sh.dsc[sh.pos_c[s]][r] = a;
      }
  }
  __syncthreads();
  // ---- dq = sum over distinct keys of dS K (eq. (2) / (4) transposed)
  const int width = dk / rank;
  for (int d = tid; d < 2 * dk; d += THREADS) {
    const int axis = d >= dk, e = d - (axis ? dk : 0);
    const int r = e / width;
    const float* K = axis ? k_col : k_row;
    const int nk = axis ? sh.nc : sh.nr;
    float a = 0.0f;
    for (int k = 0; k < nk; ++k) {
      const int key = axis ? sh.dist_c[k] : sh.dist_r[k];
      const float ds = axis ? sh.dsc[k][r] : sh.dsr[k][r];
      a = fmaf(ds, K[(static_cast<size_t>(h) * n + key) * dk + e], a);
    }
    (axis ? dq_col : dq_row)[th * dk + e] = a;
  }
  // ---- key-gradient entries: slot ((t H + h) 2 + axis) m + k for the k-th distinct key
  const uint32_t sentinel = static_cast<uint32_t>(2 * H) * n;
  for (int x = tid; x < 2 * m; x += THREADS) {
    const int axis = x >= m, k = x - (axis ? m : 0);
    const size_t slot = (th * 2 + axis) * m + k;
    const int nk = axis ? sh.nc : sh.nr;
    evals[slot] = static_cast<uint32_t>(slot);
    if (k < nk) {
      const int key = axis ? sh.dist_c[k] : sh.dist_r[k];
      ekeys[slot] = static_cast<uint32_t>((axis * H + h) * n + key);
      for (int r = 0; r < rank; ++r) edS[slot * rank + r] = axis ? sh.dsc[k][r] : sh.dsr[k][r];
    } else {
      ekeys[slot] = sentinel;
    }
  }
}

// One wave per run of equal keys: dK[key] += sum over the run's entries (in order) of dS q.
__global__ __launch_bounds__(THREADS) void key_bwd_run_kernel(
    const uint32_t* __restrict__ keys, const uint32_t* __restrict__ slots, int M, uint32_t sentinel,
    const float* __restrict__ edS, const float* __restrict__ q_row, const float* __restrict__ q_col,
    float* __restrict__ dk_row, float* __restrict__ dk_col, int H, int n, int dk, int rank, int m) {
  const int lane = threadIdx.x & (kWave - 1);
  const int i = blockIdx.x * NWAVES + static_cast<int>(threadIdx.x) / kWave;
  if (i >= M) return;
  const uint32_t key = keys[i];
  if (key == sentinel || (i > 0 && keys[i - 1] == key)) return;
  int end = i + 1;
  for (int base = i + 1; base < M; base += kWave) {
    const int pos = base + lane;
    const uint64_t same = __ballot(pos < M && keys[pos] == key);
    if (same != ~0ull) {
      end = base + __builtin_ctzll(~same);
      break;
    }
    end = min(M, base + kWave);
  }
  const int axis = static_cast<int>(key / (static_cast<uint32_t>(H) * n));
  const int rem = static_cast<int>(key - static_cast<uint32_t>(axis) * H * n);
  const int h = rem / n, kidx = rem % n;
  const float* q = axis ? q_col : q_row;
  float* dK = (axis ? dk_col : dk_row) + (static_cast<size_t>(h) * n + kidx) * dk;
  const int width = dk / rank;
  for (int d0 = 0; d0 < dk; d0 += kWave * 4) {
    const int d = d0 + lane * 4;
    if (d >= dk) continue;                         // no cross-lane operation below
    const int r = d / width;                       // four consecutive dims lie in one slice
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int e = i; e < end; ++e) {
      const size_t slot = slots[e];
      const size_t t = slot / (static_cast<size_t>(2) * H * m);
      const f32x4 qv = *reinterpret_cast<const f32x4*>(q + (t * H + h) * dk + d);
      const float ds = edS[slot * rank + r];
      acc.x = fmaf(ds, qv.x, acc.x);
      acc.y = fmaf(ds, qv.y, acc.y);
      acc.z = fmaf(ds, qv.z, acc.z);
      acc.w = fmaf(ds, qv.w, acc.w);
    }
    f32x4* dst = reinterpret_cast<f32x4*>(dK + d);
    f32x4 v = *dst;
    v += acc;
    *dst = v;
  }
}

// out[k][c] = sum over rows j of chunk k (rows k*chunk .. min(R, (k+1)*chunk) - 1, in order) of
// in[j][c]; with accumulate, out[0][c] += that sum (one chunk only).
__global__ __launch_bounds__(THREADS) void sum_rows_kernel(const float* __restrict__ in,
                                                           float* __restrict__ out, int R, int C,
                                                           int chunk, int accumulate) {
  const int chunks = (R + chunk - 1) / chunk;
  for (int x = blockIdx.x * THREADS + threadIdx.x; x < chunks * C; x += gridDim.x * THREADS) {
    const int k = x / C, c = x % C;
    float a = 0.0f;
    for (int j = k * chunk; j < min(R, (k + 1) * chunk); ++j) a += in[static_cast<size_t>(j) * C + c];
    if (accumulate) out[c] += a;
    else out[x] = a;
  }
}

size_t round_up256(size_t x) { return (x + 255) / 256 * 256; }

int bits_for(int64_t n) {
  int b = 0;
  while (b < 31 && (INT64_C(1) << b) < n) ++b;
  return b;
}

}  // namespace

size_t gather_backward_workspace_bytes(int T, int bag) {
  const int M = T * bag;
  if (M == 0) return 0;
  return 2 * round_up256(static_cast<size_t>(M) * sizeof(uint32_t)) + round_up256(sort_workspace_bytes(M));
}

hipError_t launch_gather_backward(int64_t n_values, int dv, int vdtype, const void* values, int T,
                                  int bag, const int32_t* idx, const float* w, const int32_t* perm,
                                  int expand, int cores, const float* d_pooled, float* d_values,
                                  float* dw, void* ws, hipStream_t s) {
  clear_stale_error();
  const int M = T * bag;
  if (M == 0) return hipSuccess;
  char* base = static_cast<char*>(ws);
  uint32_t* keys = reinterpret_cast<uint32_t*>(base);
  uint32_t* vals = reinterpret_cast<uint32_t*>(base + round_up256(static_cast<size_t>(M) * sizeof(uint32_t)));
  void* sws = base + 2 * round_up256(static_cast<size_t>(M) * sizeof(uint32_t));
  const unsigned kb = static_cast<unsigned>(std::min((M + THREADS - 1) / THREADS, 4096));
  hipLaunchKernelGGL(bwd_keys_kernel, dim3(kb), dim3(THREADS), 0, s, idx,
                     expand > 1 ? perm : nullptr, n_values, M, keys, vals);
  uint32_t *rows_sorted, *ents_sorted;
  hipError_t e = sort_pairs(keys, vals, M, bits_for(n_values), sws, s, &rows_sorted, &ents_sorted);
  if (e != hipSuccess) return e;
  const dim3 grid((M + NWAVES - 1) / NWAVES);
  const int c = cores > 1 ? cores : 1;
  if (vdtype == UMEM_F32)
    hipLaunchKernelGGL(gather_bwd_run_kernel<float>, grid, dim3(THREADS), 0, s, rows_sorted,
                       ents_sorted, M, static_cast<const float*>(values), dv, idx, w,
                       expand > 1 ? perm : nullptr, n_values, expand, c, bag, d_pooled, d_values, dw);
  else
    hipLaunchKernelGGL(gather_bwd_run_kernel<uint16_t>, grid, dim3(THREADS), 0, s, rows_sorted,
                       ents_sorted, M, static_cast<const uint16_t*>(values), dv, idx, w,
                       expand > 1 ? perm : nullptr, n_values, expand, c, bag, d_pooled, d_values, dw);
  return hipGetLastError();
}

size_t score_backward_workspace_bytes(const umem_desc& d, int T) {
  if (T == 0) return 0;
  const size_t th = static_cast<size_t>(T) * d.heads;
  const int Mk = static_cast<int>(th * 2 * d.topm);
  const int hc = d.cores > 1 ? d.cores : 1;
  const size_t dc = d.grid == UMEM_GRID_TUCKER ? static_cast<size_t>(hc) * d.rank * d.rank : 0;
  const size_t chunks = (static_cast<size_t>(T) + kDcChunk - 1) / kDcChunk;
  return 2 * round_up256(static_cast<size_t>(Mk) * sizeof(uint32_t)) +
         round_up256(static_cast<size_t>(Mk) * d.rank * sizeof(float)) +
         round_up256(th * dc * sizeof(float)) + round_up256(chunks * d.heads * dc * sizeof(float)) +
         round_up256(sort_workspace_bytes(Mk));
}

hipError_t launch_score_backward(const umem_desc& d, int T, const float* q_row, const float* q_col,
                                 const float* k_row, const float* k_col, const float* core,
                                 const int32_t* idx, const float* w, const float* dw,
                                 float* dq_row, float* dq_col, float* dk_row, float* dk_col,
                                 float* dcore, void* ws, hipStream_t s) {
  clear_stale_error();
  if (T == 0) return hipSuccess;
  const int H = d.heads, m = d.topm, r = d.rank;
  const size_t th = static_cast<size_t>(T) * H;
  const int Mk = static_cast<int>(th * 2 * m);
  const bool tucker = d.grid == UMEM_GRID_TUCKER;
  const int hc = d.cores > 1 ? d.cores : 1;
  const int dc = tucker ? hc * r * r : 0;
  char* base = static_cast<char*>(ws);
  uint32_t* ekeys = reinterpret_cast<uint32_t*>(base);
  base += round_up256(static_cast<size_t>(Mk) * sizeof(uint32_t));
  uint32_t* evals = reinterpret_cast<uint32_t*>(base);
  base += round_up256(static_cast<size_t>(Mk) * sizeof(uint32_t));
  float* edS = reinterpret_cast<float*>(base);
  base += round_up256(static_cast<size_t>(Mk) * r * sizeof(float));
  float* dc_part = reinterpret_cast<float*>(base);
  base += round_up256(th * dc * sizeof(float));
  float* dc_chunks = reinterpret_cast<float*>(base);
  const size_t chunks = (static_cast<size_t>(T) + kDcChunk - 1) / kDcChunk;
  base += round_up256(chunks * H * dc * sizeof(float));
  void* sws = base;
  hipLaunchKernelGGL(score_bwd_kernel, dim3(static_cast<unsigned>(th)), dim3(THREADS), 0, s, q_row,
                     q_col, k_row, k_col, core, idx, w, dw, T, H, d.n_keys, d.dk, r, m,
                     tucker ? 1 : 0, d.weight == UMEM_W_SOFTMAX ? 1 : 0, hc, dq_row, dq_col, ekeys,
                     evals, edS, dc_part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const uint32_t sentinel = static_cast<uint32_t>(2 * H) * d.n_keys;
  uint32_t *ks, *vs;
  e = sort_pairs(ekeys, evals, Mk, bits_for(static_cast<int64_t>(sentinel) + 1), sws, s, &ks, &vs);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(key_bwd_run_kernel, dim3((Mk + NWAVES - 1) / NWAVES), dim3(THREADS), 0, s, ks,
                     vs, Mk, sentinel, edS, q_row, q_col, dk_row, dk_col, H, d.n_keys, d.dk, r, m);
  if (tucker) {
    // dC: per-token partials [T][H dc] -> chunks of kDcChunk tokens -> the chunks, added to dcore
    const int C = H * dc;
    const unsigned b1 = static_cast<unsigned>(std::min<size_t>((chunks * C + THREADS - 1) / THREADS, 1024));
    hipLaunchKernelGGL(sum_rows_kernel, dim3(b1), dim3(THREADS), 0, s, dc_part, dc_chunks, T, C,
                       kDcChunk, 0);
    hipLaunchKernelGGL(sum_rows_kernel, dim3((C + THREADS - 1) / THREADS), dim3(THREADS), 0, s,
                       dc_chunks, dcore, static_cast<int>(chunks), C, static_cast<int>(chunks), 1);
  }
  return hipGetLastError();
}

}  // namespace umem
