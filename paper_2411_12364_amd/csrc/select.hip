// a3 + a4 + a5: per-axis top-k, grid scores of the k*k candidates, global top-m and weights.
//
// One workgroup per (token, head).  Selections are radix selects on order-preserving 32-bit
// keys held in LDS: four 8-bit digit passes find the k-th largest key exactly, then one
// ordered pass keeps every key above it plus the lowest-positioned keys equal to it, so ties go
// to the lower position.  The per-axis selections come out in ascending index order; the
// candidate (a, b) = (a-th selected row, b-th selected column) then sits at position a*k + b,
// and that order is the order of the logical flat index i*n + j, so the same tie rule gives the
// lower flat index on the grid (eq. (3) / eq. (10) with ties to the lower index).
#include "umem_internal.h"

namespace umem {
namespace {

constexpr int THREADS = 256;
constexpr int NWAVES = THREADS / kWave;

struct SelectShared {
  int hist[256];
  int wave_cnt[NWAVES][2];
  int digit;
  int remaining;
  int32_t I[2][kMaxTopK];                  // selected indices, ascending
  float s_sel[2][kMaxTopK];                // their selection scores
  float s_ex[2][kMaxRank][kMaxTopK];       // Tucker: exact per-slice scores of the selected
  float p_col[kMaxRank][kMaxTopK];         // Tucker: (C S_col)[rho, b]
  int32_t cand[kMaxTopM];                  // selected candidate positions, ascending
  float cand_g[kMaxTopM];
  float e[kMaxTopM];
  float core[kMaxRank * kMaxRank];
  float gmax, esum;
};

// Positions (ascending) of the k largest of keys[0, len); ties go to the lower position.
__device__ void block_select(const uint32_t* keys, int len, int k, int32_t* out, SelectShared& sh) {
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  uint32_t prefix = 0u, mask = 0u;
  int remaining = k;
  for (int shift = 24; shift >= 0; shift -= 8) {
    sh.hist[tid] = 0;
    __syncthreads();
    for (int i = tid; i < len; i += THREADS) {
      const uint32_t x = keys[i];
      if ((x & mask) == prefix) atomicAdd(&sh.hist[(x >> shift) & 255u], 1);
    }
    __syncthreads();
    if (wave == 0) {
      // lane l owns bins 255-4l .. 252-4l, scanned from the top
      const int b0 = 255 - 4 * lane;
      const int c0 = sh.hist[b0], c1 = sh.hist[b0 - 1], c2 = sh.hist[b0 - 2], c3 = sh.hist[b0 - 3];
      const int sum = c0 + c1 + c2 + c3;
      const int incl = wave_inclusive_scan(sum);
      const int excl = incl - sum;
      if (excl < remaining && remaining <= incl) {
        int acc = excl, dig;
        if (remaining <= acc + c0) {
          dig = b0;
        } else if (remaining <= acc + c0 + c1) {
          acc += c0;
          dig = b0 - 1;
        } else if (remaining <= acc + c0 + c1 + c2) {
          acc += c0 + c1;
          dig = b0 - 2;
        } else {
          acc += c0 + c1 + c2;
          dig = b0 - 3;
        }
        sh.digit = dig;
        sh.remaining = remaining - acc;
      }
    }
    __syncthreads();
    prefix |= static_cast<uint32_t>(sh.digit) << shift;
    mask |= 255u << shift;
    remaining = sh.remaining;
    __syncthreads();
  }
  const uint32_t thr = prefix;
  const int need_eq = remaining;   // keys equal to thr that are kept (>= 1)

  // each wave scans one contiguous quarter of the array, 64 positions at a time
  const int seg = ((len + NWAVES - 1) / NWAVES + kWave - 1) / kWave * kWave;
  const int beg = wave * seg;
  const int end = min(len, beg + seg);
  int gt_cnt = 0, eq_cnt = 0;
  for (int base = beg; base < end; base += kWave) {
    const int i = base + lane;
    const uint32_t x = (i < end) ? keys[i] : 0u;
    gt_cnt += __popcll(__ballot(i < end && x > thr));
    eq_cnt += __popcll(__ballot(i < end && x == thr));
  }
  if (lane == 0) {
    sh.wave_cnt[wave][0] = gt_cnt;
    sh.wave_cnt[wave][1] = eq_cnt;
  }
  __syncthreads();
  int eq_base = 0, taken_base = 0;
  for (int v = 0; v < wave; ++v) {
    const int g = sh.wave_cnt[v][0], e = sh.wave_cnt[v][1];
    taken_base += g + min(max(need_eq - eq_base, 0), e);
    eq_base += e;
  }
  const uint64_t lt = lanemask_lt();
  for (int base = beg; base < end; base += kWave) {
    const int i = base + lane;
    const uint32_t x = (i < end) ? keys[i] : 0u;
    const bool gt = i < end && x > thr;
    const bool eq = i < end && x == thr;
    const uint64_t m_eq = __ballot(eq);
    const int eq_rank = eq_base + __popcll(m_eq & lt);
    const bool take = gt || (eq && eq_rank < need_eq);
    const uint64_t m_take = __ballot(take);
    if (take) out[taken_base + __popcll(m_take & lt)] = i;
    eq_base += __popcll(m_eq);
    taken_base += __popcll(m_take);
  }
  __syncthreads();
}

__global__ __launch_bounds__(THREADS) void select_kernel(
    const float* __restrict__ sel, const float* __restrict__ q_row,
    const float* __restrict__ q_col, const float* __restrict__ k_row,
    const float* __restrict__ k_col, const float* __restrict__ core_all,
    int32_t* __restrict__ idx_out, float* __restrict__ w_out, int32_t* __restrict__ axis_out,
    int T, int H, int n, int dk, int rank, int k, int m, int tucker, int softmax) {
  extern __shared__ uint32_t keys[];     // max(n, k*k) keys
  __shared__ SelectShared sh;
  const int tid = threadIdx.x;
  const int t = blockIdx.x / H;
  const int h = blockIdx.x % H;

  if (tucker && tid < rank * rank) sh.core[tid] = core_all[static_cast<size_t>(h) * rank * rank + tid];

  // ---- a3: per-axis top-k on the selection scores
  for (int axis = 0; axis < 2; ++axis) {
    const float* src = sel + ((static_cast<size_t>(axis) * T + t) * H + h) * n;
    for (int i = tid; i < n; i += THREADS) keys[i] = order_key(src[i]);
    __syncthreads();
    block_select(keys, n, k, sh.I[axis], sh);
    for (int a = tid; a < k; a += THREADS) sh.s_sel[axis][a] = src[sh.I[axis][a]];
    __syncthreads();
    if (axis_out != nullptr) {
      // rank by (score desc, index asc); I is ascending so a lower slot means a lower index
      for (int a = tid; a < k; a += THREADS) {
        const uint32_t ka = order_key(sh.s_sel[axis][a]);
        int r = 0;
        for (int b = 0; b < k; ++b) {
          const uint32_t kb = order_key(sh.s_sel[axis][b]);
          r += (kb > ka) || (kb == ka && b < a);
        }
        axis_out[((static_cast<size_t>(axis) * T + t) * H + h) * k + r] = sh.I[axis][a];
      }
    }
  }

  // ---- a4: candidate scores
  if (tucker) {
    // exact per-slice scores of the selected keys (eq. (4)), recomputed in fp32
    const int width = dk / rank;
    for (int job = tid; job < 2 * rank * k; job += THREADS) {
      const int axis = job / (rank * k);
      const int rho = (job / k) % rank;
      const int a = job % k;
      const float* K = axis ? k_col : k_row;
      const float* q = axis ? q_col : q_row;
      const float* kr = K + (static_cast<size_t>(h) * n + sh.I[axis][a]) * dk + rho * width;
      const float* qr = q + (static_cast<size_t>(t) * H + h) * dk + rho * width;
      float s = 0.0f;
      for (int d = 0; d < width; d += 4) {
        const float4 kv = *reinterpret_cast<const float4*>(kr + d);
        const float4 qv = *reinterpret_cast<const float4*>(qr + d);
        s = fmaf(kv.x, qv.x, s);
        s = fmaf(kv.y, qv.y, s);
        s = fmaf(kv.z, qv.z, s);
        s = fmaf(kv.w, qv.w, s);
      }
      sh.s_ex[axis][rho][a] = s;
    }
    __syncthreads();
    for (int job = tid; job < rank * k; job += THREADS) {
      const int rho = job / k, b = job % k;
      float p = 0.0f;
      for (int sg = 0; sg < rank; ++sg) p = fmaf(sh.core[rho * rank + sg], sh.s_ex[1][sg][b], p);
      sh.p_col[rho][b] = p;
    }
    __syncthreads();
  }
  const int ncand = k * k;
  for (int c = tid; c < ncand; c += THREADS) {
    const int a = c / k, b = c - (c / k) * k;
    float g;
    if (tucker) {
      g = 0.0f;
      for (int rho = 0; rho < rank; ++rho) g = fmaf(sh.s_ex[0][rho][a], sh.p_col[rho][b], g);
    } else {
      g = sh.s_sel[0][a] + sh.s_sel[1][b];
    }
    keys[c] = order_key(g);
  }
  __syncthreads();

  // ---- a5: global top-m, sorted by (score desc, flat index asc), and weights
  block_select(keys, ncand, m, sh.cand, sh);
  for (int j = tid; j < m; j += THREADS) {
    const int c = sh.cand[j];
    const int a = c / k, b = c - (c / k) * k;
    float g;
    if (tucker) {
      g = 0.0f;
      for (int rho = 0; rho < rank; ++rho) g = fmaf(sh.s_ex[0][rho][a], sh.p_col[rho][b], g);
    } else {
      g = sh.s_sel[0][a] + sh.s_sel[1][b];
    }
    sh.cand_g[j] = g;
  }
  __syncthreads();
  int my_rank = -1;
  if (tid < m) {
    const uint32_t kj = keys[sh.cand[tid]];
    int r = 0;
    for (int l = 0; l < m; ++l) {
      const uint32_t kl = keys[sh.cand[l]];
      r += (kl > kj) || (kl == kj && l < tid);
    }
    my_rank = r;
    if (r == 0) sh.gmax = sh.cand_g[tid];
  }
  __syncthreads();
  if (softmax) {
    if (tid < m) sh.e[my_rank] = __expf(sh.cand_g[tid] - sh.gmax);
    __syncthreads();
    if (tid < kWave) {
      float s = 0.0f;
      for (int j = tid; j < m; j += kWave) s += sh.e[j];
      s = wave_sum(s);
      if (tid == 0) sh.esum = s;
    }
    __syncthreads();
  }
  if (tid < m) {
    const int c = sh.cand[tid];
    const int a = c / k, b = c - (c / k) * k;
    const size_t o = (static_cast<size_t>(t) * H + h) * m + my_rank;
    idx_out[o] = sh.I[0][a] * n + sh.I[1][b];
    w_out[o] = softmax ? sh.e[my_rank] / sh.esum : sh.cand_g[tid];
  }
}

}  // namespace

hipError_t launch_select(const umem_desc& d, int T, const float* sel, const float* q_row,
                         const float* q_col, const float* k_row, const float* k_col,
                         const float* core, int32_t* idx, float* w, int32_t* axis_idx,
                         hipStream_t s) {
  if (T == 0) return hipSuccess;
  const int cap = d.n_keys > d.topk * d.topk ? d.n_keys : d.topk * d.topk;
  const size_t lds = static_cast<size_t>(cap) * sizeof(uint32_t);
  const int tucker = d.grid == UMEM_GRID_TUCKER;
  hipLaunchKernelGGL(select_kernel, dim3(static_cast<unsigned>(T) * d.heads), dim3(THREADS), lds, s,
                     sel, q_row, q_col, k_row, k_col, core, idx, w, axis_idx, T, d.heads, d.n_keys,
                     d.dk, d.rank, d.topk, d.topm, tucker, d.weight == UMEM_W_SOFTMAX);
  return hipGetLastError();
}

}  // namespace umem
