// a3 + a4 + a5: per-axis top-k, grid scores of the candidates, global top-m and weights.
//
// One workgroup (256 threads) per (token, head).  Every selection is exact under the order
// (score desc, index asc):
//
//  1. Threshold.  Each thread holds its elements in registers and takes their maximum.  The k-th
//     largest of the 256 thread maxima, L, is found by a 32-step ballot search in one wave.  The
//     k largest maxima are k distinct elements >= L, so the k-th largest element is >= L and
//     every element of the top-k (ties included) is >= L.
//  2. Survivors {x >= L} (typically a few dozen) are appended to LDS with one atomic per wave.
//  3. Each survivor's rank is the number of survivors ordered before it; ranks < k are the
//     answer, already sorted.
//  If the survivors overflow their buffer (massive ties), a radix select on the 32-bit keys
//  with lowest-position tie-break takes over.
//
// Additive grid (eq. (3)): with both axis lists sorted, candidate (a, b) (a-th best row, b-th
// best column) is preceded in the order by the (a+1)(b+1)-1 candidates (a' <= a, b' <= b), so
// only (a+1)(b+1) <= m can reach the top-m.  Candidate scores are summed in fp64, where the sum
// of two fp32 scores is exact, so this dominance holds exactly.
// Tucker grid (eq. (10)): all k*k candidates, exact per-slice scores recomputed for the selected
// keys, scores in fp64, the threshold filter of step 1 on their fp32 roundings.
#include "umem_internal.h"

namespace umem {
namespace {

constexpr int THREADS = 256;
constexpr int NWAVES = THREADS / kWave;
constexpr int SMAX = 2048;        // survivor buffer

struct SelectShared {
  uint32_t mx[THREADS];               // thread maxima
  int hist[256];                      // fallback radix histogram
  int wave_cnt[NWAVES][2];
  int digit, remaining, count;
  uint32_t thr;
  int32_t ax_idx[2][kMaxTopK];        // axis top-k, sorted by (score desc, index asc)
  float ax_sc[2][kMaxTopK];
  uint64_t tmp_comp[kMaxTopK];        // fallback: the k picked positions, re-ranked
  int32_t tmp_pos[kMaxTopM];
  int32_t inv[2][kMaxTopK];           // Tucker fallback: index-sorted position -> sorted position
  float s_ex[2][kMaxRank][kMaxTopK];  // Tucker: exact per-slice scores of the selected keys
  double p_col[kMaxRank][kMaxTopK];   // Tucker: (C S_col)[rho, b] in fp64
  float core[kMaxRank * kMaxRank];
  int32_t out_flat[kMaxTopM];         // final top-m, by rank
  double out_g[kMaxTopM];
  float e[kMaxTopM];
  double gmax;
  float esum;
};

__device__ __forceinline__ uint64_t order_key64(double x) {
  if (x != x) return 0ull;
  if (x == 0.0) x = 0.0;                      // -0.0 ranks as +0.0
  const uint64_t u = static_cast<uint64_t>(__double_as_longlong(x));
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// Slot for an appended element: all lanes of the wave call this; returns -1 where !pred.
__device__ __forceinline__ int wave_append(bool pred, int* counter) {
  const uint64_t m = __ballot(pred);
  if (m == 0ull) return -1;
  int base = 0;
  if ((threadIdx.x & (kWave - 1)) == 0) base = atomicAdd(counter, static_cast<int>(__popcll(m)));
  base = __shfl(base, 0, kWave);
  return pred ? base + static_cast<int>(__popcll(m & lanemask_lt())) : -1;
}

// k-th largest of the 256 thread maxima (wave 0 only; 4 values per lane).
__device__ __forceinline__ uint32_t kth_largest_of_maxima(const uint32_t* mx, int k) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t v0 = mx[lane], v1 = mx[lane + 64], v2 = mx[lane + 128], v3 = mx[lane + 192];
  uint32_t prefix = 0u;
  for (int b = 31; b >= 0; --b) {
    const uint32_t c = prefix | (1u << b);
    const int cnt = __popcll(__ballot(v0 >= c)) + __popcll(__ballot(v1 >= c)) +
                    __popcll(__ballot(v2 >= c)) + __popcll(__ballot(v3 >= c));
    if (cnt >= k) prefix = c;
  }
  return prefix;
}

// Positions (ascending) of the k largest of keys[0, len); ties go to the lower position.
// Radix select, four 8-bit digits.  Used only when the threshold filter overflows.
__device__ void radix_select(const uint32_t* keys, int len, int k, int32_t* out, SelectShared& sh) {
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
  const int need_eq = remaining;
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

// Composite 64-bit key of an axis element: larger = earlier in (score desc, index asc).
__device__ __forceinline__ uint64_t axis_comp(uint32_t key, int idx) {
  return (static_cast<uint64_t>(key) << 32) | static_cast<uint64_t>(0xFFFFFFFFu - static_cast<uint32_t>(idx));
}

// Top-k of one axis whose n scores sit in registers (element tid + 256 j in x[j]).
template <int NPT>
__device__ void select_axis(const float (&x)[NPT], int n, int k, int axis, SelectShared& sh,
                            unsigned char* dyn) {
  const int tid = threadIdx.x;
  uint64_t* comp = reinterpret_cast<uint64_t*>(dyn);     // [SMAX] survivors
  uint32_t mx = 0u;
  uint32_t key[NPT];
#pragma unroll
  for (int j = 0; j < NPT; ++j) {
    const int i = tid + THREADS * j;
    key[j] = (i < n) ? order_key(x[j]) : 0u;
    if (i < n) mx = max(mx, key[j]);
  }
  sh.mx[tid] = mx;
  if (tid == 0) sh.count = 0;
  __syncthreads();
  if (tid < kWave) {
    const uint32_t L = kth_largest_of_maxima(sh.mx, k);
    if (tid == 0) sh.thr = L;
  }
  __syncthreads();
  const uint32_t L = sh.thr;
#pragma unroll
  for (int j = 0; j < NPT; ++j) {
    const int i = tid + THREADS * j;
    const bool pred = i < n && key[j] >= L;
    const int pos = wave_append(pred, &sh.count);
    if (pos >= 0 && pos < SMAX) comp[pos] = axis_comp(key[j], i);
  }
  __syncthreads();
  const int S = sh.count;
  if (S <= SMAX) {
    for (int s = tid; s < S; s += THREADS) {
      const uint64_t c = comp[s];
      int r = 0;
      for (int t = 0; t < S; ++t) r += comp[t] > c;
      if (r < k) {
        const int idx = static_cast<int>(0xFFFFFFFFu - static_cast<uint32_t>(c & 0xFFFFFFFFull));
        sh.ax_idx[axis][r] = idx;
      }
    }
  } else {
    // fallback: exact radix select over all n keys, then order the k picked
    uint32_t* keys = reinterpret_cast<uint32_t*>(dyn);
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
      const int i = tid + THREADS * j;
      if (i < n) keys[i] = key[j];
    }
    __syncthreads();
    radix_select(keys, n, k, sh.tmp_pos, sh);
    for (int a = tid; a < k; a += THREADS) sh.tmp_comp[a] = axis_comp(keys[sh.tmp_pos[a]], sh.tmp_pos[a]);
    __syncthreads();
    for (int a = tid; a < k; a += THREADS) {
      const uint64_t c = sh.tmp_comp[a];
      int r = 0;
      for (int b = 0; b < k; ++b) r += sh.tmp_comp[b] > c;
      sh.ax_idx[axis][r] = sh.tmp_pos[a];
    }
  }
  __syncthreads();
}

template <int NPT>
__global__ __launch_bounds__(THREADS) void select_kernel(
    const float* __restrict__ sel, const float* __restrict__ q_row,
    const float* __restrict__ q_col, const float* __restrict__ k_row,
    const float* __restrict__ k_col, const float* __restrict__ core_all,
    int32_t* __restrict__ idx_out, float* __restrict__ w_out, int32_t* __restrict__ axis_out,
    int T, int H, int n, int dk, int rank, int k, int m, int tucker, int softmax) {
  extern __shared__ __align__(16) unsigned char dyn[];
  __shared__ SelectShared sh;
  const int tid = threadIdx.x;
  const int t = blockIdx.x / H;
  const int h = blockIdx.x % H;

  // both axes' selection scores, one memory round trip
  float xr[NPT], xc[NPT];
  const float* src_r = sel + ((static_cast<size_t>(0) * T + t) * H + h) * n;
  const float* src_c = sel + ((static_cast<size_t>(1) * T + t) * H + h) * n;
#pragma unroll
  for (int j = 0; j < NPT; ++j) {
    const int i = tid + THREADS * j;
    xr[j] = (i < n) ? src_r[i] : 0.0f;
    xc[j] = (i < n) ? src_c[i] : 0.0f;
  }
  if (tucker && tid < rank * rank) sh.core[tid] = core_all[static_cast<size_t>(h) * rank * rank + tid];

  // ---- a3: per-axis top-k
  select_axis<NPT>(xr, n, k, 0, sh, dyn);
  select_axis<NPT>(xc, n, k, 1, sh, dyn);
  for (int a = tid; a < 2 * k; a += THREADS) {
    const int axis = a / k, r = a % k;
    const float* src = axis ? src_c : src_r;
    sh.ax_sc[axis][r] = src[sh.ax_idx[axis][r]];
    if (axis_out != nullptr)
      axis_out[((static_cast<size_t>(axis) * T + t) * H + h) * k + r] = sh.ax_idx[axis][r];
  }
  __syncthreads();

  uint64_t* ckey = reinterpret_cast<uint64_t*>(dyn);                 // [SMAX] candidate keys
  int32_t* cflat = reinterpret_cast<int32_t*>(dyn + SMAX * 8);       // [SMAX] candidate slots
  if (tid == 0) sh.count = 0;
  __syncthreads();

  if (!tucker) {
    // ---- a4 (additive): candidates with (a+1)(b+1) <= m, scores summed exactly in fp64
    const int kk = k * k;
    for (int c0 = 0; c0 < kk; c0 += THREADS) {
      const int c = c0 + tid;
      const int a = c / k, b = c - (c / k) * k;
      const bool pred = c < kk && (a + 1) * (b + 1) <= m;
      const int pos = wave_append(pred, &sh.count);
      if (pos >= 0 && pos < SMAX) {   // at most m * H(k) < SMAX candidates (host-checked)
        const double g = static_cast<double>(sh.ax_sc[0][a]) + static_cast<double>(sh.ax_sc[1][b]);
        ckey[pos] = order_key64(g);
        cflat[pos] = sh.ax_idx[0][a] * n + sh.ax_idx[1][b];
      }
    }
    __syncthreads();
  } else {
    // ---- a4 (Tucker): exact per-slice scores of the selected keys (eq. (4)), in fp32
    const int width = dk / rank;
    for (int job = tid; job < 2 * rank * k; job += THREADS) {
      const int axis = job / (rank * k);
      const int rho = (job / k) % rank;
      const int a = job % k;
      const float* K = axis ? k_col : k_row;
      const float* q = axis ? q_col : q_row;
      const float* kr = K + (static_cast<size_t>(h) * n + sh.ax_idx[axis][a]) * dk + rho * width;
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
      double p = 0.0;
      for (int sg = 0; sg < rank; ++sg)
        p += static_cast<double>(sh.core[rho * rank + sg]) * static_cast<double>(sh.s_ex[1][sg][b]);
      sh.p_col[rho][b] = p;
    }
    __syncthreads();
    auto gscore = [&](int a, int b) {
      double g = 0.0;
      for (int rho = 0; rho < rank; ++rho) g += static_cast<double>(sh.s_ex[0][rho][a]) * sh.p_col[rho][b];
      return g;
    };
    const int kk = k * k;
    uint32_t mx = 0u;
    for (int c = tid; c < kk; c += THREADS) mx = max(mx, order_key(static_cast<float>(gscore(c / k, c % k))));
    sh.mx[tid] = mx;
    __syncthreads();
    if (tid < kWave) {
      const uint32_t L = kth_largest_of_maxima(sh.mx, m);
      if (tid == 0) sh.thr = L;
    }
    __syncthreads();
    const uint32_t L = sh.thr;
    for (int c0 = 0; c0 < kk; c0 += THREADS) {
      const int c = c0 + tid;
      const int a = c / k, b = c - (c / k) * k;
      double g = 0.0;
      bool pred = false;
      if (c < kk) {
        g = gscore(a, b);
        pred = order_key(static_cast<float>(g)) >= L;
      }
      const int pos = wave_append(pred, &sh.count);
      if (pos >= 0 && pos < SMAX) {
        ckey[pos] = order_key64(g);
        cflat[pos] = sh.ax_idx[0][a] * n + sh.ax_idx[1][b];
      }
    }
    __syncthreads();
    if (sh.count > SMAX) {
      // fallback: radix select on the fp32-rounded scores laid out in flat-index order
      uint32_t* keys = reinterpret_cast<uint32_t*>(dyn);
      for (int a = tid; a < 2 * k; a += THREADS) {
        const int axis = a / k, r = a % k;
        int p = 0;
        for (int b = 0; b < k; ++b) p += sh.ax_idx[axis][b] < sh.ax_idx[axis][r];
        sh.inv[axis][p] = r;
      }
      __syncthreads();
      for (int c = tid; c < kk; c += THREADS)
        keys[c] = order_key(static_cast<float>(gscore(sh.inv[0][c / k], sh.inv[1][c % k])));
      __syncthreads();
      radix_select(keys, kk, m, sh.tmp_pos, sh);
      if (tid == 0) sh.count = m;
      __syncthreads();
      for (int j = tid; j < m; j += THREADS) {
        const int c = sh.tmp_pos[j];
        const int a = sh.inv[0][c / k], b = sh.inv[1][c % k];
        ckey[j] = order_key64(gscore(a, b));
        cflat[j] = sh.ax_idx[0][a] * n + sh.ax_idx[1][b];
      }
      __syncthreads();
    }
  }

  // ---- a5: rank the candidates by (score desc, flat index asc); ranks < m are the answer
  const int C = sh.count;
  for (int s = tid; s < C; s += THREADS) {
    const uint64_t ks = ckey[s];
    const int fs = cflat[s];
    int r = 0;
    for (int u = 0; u < C; ++u) {
      const uint64_t ku = ckey[u];
      r += (ku > ks) || (ku == ks && cflat[u] < fs);
    }
    if (r < m) {
      sh.out_flat[r] = fs;
      const uint64_t raw = (ks >> 63) ? (ks & 0x7FFFFFFFFFFFFFFFull) : ~ks;
      sh.out_g[r] = __longlong_as_double(static_cast<long long>(raw));
    }
  }
  __syncthreads();
  if (softmax) {
    if (tid < m) sh.e[tid] = __expf(static_cast<float>(sh.out_g[tid] - sh.out_g[0]));
    __syncthreads();
    if (tid < kWave) {
      float s = 0.0f;
      for (int j = tid; j < m; j += kWave) s += sh.e[j];
      s = wave_sum(s);
      if (tid == 0) sh.esum = s;
    }
    __syncthreads();
  }
  for (int j = tid; j < m; j += THREADS) {
    const size_t o = (static_cast<size_t>(t) * H + h) * m + j;
    idx_out[o] = sh.out_flat[j];
    w_out[o] = softmax ? sh.e[j] / sh.esum : static_cast<float>(sh.out_g[j]);
  }
}

}  // namespace

int additive_candidates(int k, int m) {
  int c = 0;
  for (int a = 0; a < k; ++a) c += min(k, m / (a + 1));
  return c;
}

size_t select_lds_bytes(int n, int k) {
  size_t a = static_cast<size_t>(n) * 4, b = static_cast<size_t>(SMAX) * 12, c = static_cast<size_t>(k) * k * 4;
  return a > b ? (a > c ? a : c) : (b > c ? b : c);
}

hipError_t launch_select(const umem_desc& d, int T, const float* sel, const float* q_row,
                         const float* q_col, const float* k_row, const float* k_col,
                         const float* core, int32_t* idx, float* w, int32_t* axis_idx,
                         hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (d.grid == UMEM_GRID_ADD && additive_candidates(d.topk, d.topm) > SMAX) return hipErrorInvalidValue;
  const size_t lds = select_lds_bytes(d.n_keys, d.topk);
  const int tucker = d.grid == UMEM_GRID_TUCKER;
  const dim3 grid(static_cast<unsigned>(T) * d.heads), block(THREADS);
#define UMEM_SELECT(NPT)                                                                          \
  hipLaunchKernelGGL(select_kernel<NPT>, grid, block, lds, s, sel, q_row, q_col, k_row, k_col,   \
                     core, idx, w, axis_idx, T, d.heads, d.n_keys, d.dk, d.rank, d.topk, d.topm,  \
                     tucker, d.weight == UMEM_W_SOFTMAX)
  const int npt = (d.n_keys + THREADS - 1) / THREADS;
  if (npt <= 1) UMEM_SELECT(1);
  else if (npt <= 2) UMEM_SELECT(2);
  else if (npt <= 4) UMEM_SELECT(4);
  else if (npt <= 8) UMEM_SELECT(8);
  else if (npt <= 16) UMEM_SELECT(16);
  else if (npt <= 32) UMEM_SELECT(32);
  else return hipErrorInvalidValue;
#undef UMEM_SELECT
  return hipGetLastError();
}

}  // namespace umem
