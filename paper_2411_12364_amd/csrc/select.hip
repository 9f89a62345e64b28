// a3 + a4 + a5: per-axis top-k, grid scores of the candidates, global top-m and weights.
//
// One workgroup of eight waves per (token, head): waves 0-3 select on the row axis and waves
// 4-7 on the column axis, at the same time.  Every selection is exact under the order
// (score desc, index asc), in three steps:
//
//  1. Threshold.  Each thread holds its elements in registers and takes their maximum; the
//     maxima of four threads are merged per lane, and L is the largest value whose low 16 key
//     bits are zero such that at least k of those 64 merged maxima are >= L (8 radix-4 steps of
//     ballots, which each wave of the axis runs for itself).  They are maxima of disjoint sets, so at least k elements are >= L:
//     the whole top-k is >= L.
//  2. Survivors {x >= L} (typically a few dozen) are compacted into LDS: a DPP wave scan places
//     them within the wave's range, which one LDS atomic reserves (the ranks below do not depend
//     on the order of the ranges, so the result is deterministic).
//  3. A survivor's rank is the number of survivors ordered before it, counted by P threads per
//     survivor (as many as the group has to spare) and summed over those lanes; ranks < k are
//     the answer, already sorted.
//  If an axis's survivors overflow their buffer (massive ties), an exact threshold search over
//  all elements of the axis (32 steps of group-wide counts) takes over.
//
// Additive grid (eq. (3)): with both axis lists sorted, candidate (a, b) (a-th best row, b-th
// best column) is preceded in the order by the (a+1)(b+1)-1 candidates (a' <= a, b' <= b), so
// only (a+1)(b+1) <= m can reach the top-m.  Candidate scores are summed in fp64, where the sum
// of two fp32 scores is exact (or monotone), so this dominance holds.  Further, for r <= k rows
// and c = ceil(m / r) <= k columns the r x c corner of the grid holds at least m pairs, all
// scoring >= A[r-1] + B[c-1]: theta, the largest such bound over r, is <= the m-th best score,
// and only candidates >= theta are ranked (typically a third of them).
// For the forward without expansion (at most two heads, rows of 1 or 2 KiB) the workgroup also
// pools its m rows (eq. (1)) and adds them into the token's output: the decode path then needs
// no separate gather launch.
// With multi-core scoring (eqs. (16), (17)) the selection runs on the summed core and, for the
// m selected slots, each component core's exact score is computed (fp64) as its weight.
// Tucker grid (eq. (10)): all k*k candidates, the exact per-slice scores recomputed for the
// selected keys, candidate scores in fp64; the threshold of step 1 runs on their fp32 roundings
// (rounding is monotone, so the survivors still contain the top-m) and the ranks on fp64.
#include "umem_internal.h"

namespace umem {
namespace {

constexpr int THREADS = 512;
constexpr int NWAVES = THREADS / kWave;
constexpr int GROUP = 256;          // threads per axis
constexpr int SMAX_AX = 512;        // survivors per axis
constexpr int SMAX_S = 512;         // grid survivors (Tucker)
constexpr int KK_MAX = 4096;        // Tucker: k*k candidates
constexpr int ADD_MAX = 2048;       // additive candidates (a+1)(b+1) <= m, a, b < k
constexpr int CPT = KK_MAX / THREADS;   // Tucker candidates per thread

// Kernel variants: kModePool pools the value rows when given them and takes the grid from its
// argument; its row loads in flight take many registers.  kModeAdd and kModeTucker never pool
// and are specialised to one grid: fewer registers, more workgroups per CU for many tokens.
constexpr int kModePool = 0, kModeAdd = 1, kModeTucker = 2;

typedef float f32x4 __attribute__((ext_vector_type(4)));

struct SelectShared {
  uint32_t mx[THREADS];               // thread maxima (both axes, or the grid)
  int wave_tot[NWAVES];
  int ax_cnt[2];                      // survivors of each axis (LDS-atomic ranges per wave)
  uint32_t thr[2];
  int32_t ax_idx[2][kMaxTopK];        // axis top-k, sorted by (score desc, index asc)
  float ax_sc[2][kMaxTopK];
  int grid_cnt;                       // additive grid: candidates kept for ranking
  int grid_total;                     // additive grid: (a+1)(b+1) <= m candidates
  uint16_t grid_ab[ADD_MAX];          // ... their (a << 8) | b, row by row
  uint8_t th_col[kMaxTopK + 1];       // ceil(m / r) for the corner bound of r rows (0: beyond k)
  float s_ex[2][kMaxRank][kMaxTopK];  // Tucker: exact per-slice scores of the selected keys
  double p_col[kMaxRank][kMaxTopK];   // Tucker: (C S_col)[rho, b] in fp64
  double core[kMaxRank * kMaxRank];              // Tucker: the core (sum of its components)
  float core_parts[kMaxCores][kMaxRank * kMaxRank];   // multi-core scoring: the components
  int32_t out_ab[kMaxTopM];                      // Tucker: (a << 8) | b of each selected slot
  float w_core[kMaxTopM * kMaxCores];            // multi-core scoring: weights [m][cores]
  int32_t out_flat[kMaxTopM];         // final top-m, by rank
  double out_g[kMaxTopM];
  float e[kMaxTopM];
  float esum;
};

__device__ __forceinline__ uint64_t order_key64(double x) {
  if (x != x) return 0ull;
  if (x == 0.0) x = 0.0;                      // -0.0 ranks as +0.0
  const uint64_t u = static_cast<uint64_t>(__double_as_longlong(x));
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

__device__ __forceinline__ double key64_value(uint64_t k) {
  const uint64_t raw = (k >> 63) ? (k & 0x7FFFFFFFFFFFFFFFull) : ~k;
  return __longlong_as_double(static_cast<long long>(raw));
}

__device__ __forceinline__ float key32_value(uint32_t k) {
  return __uint_as_float((k >> 31) ? (k & 0x7FFFFFFFu) : ~k);
}

// Composite key of an axis element: larger = earlier in (score desc, index asc).
__device__ __forceinline__ uint64_t axis_comp(uint32_t key, int idx) {
  return (static_cast<uint64_t>(key) << 32) |
         static_cast<uint64_t>(0xFFFFFFFFu - static_cast<uint32_t>(idx));
}

// Inclusive prefix sum over the 64 lanes of a wave (DPP row shifts and row broadcasts).
__device__ __forceinline__ int wave_scan_dpp(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, true);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, true);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, true);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, true);   // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);  // row_bcast:15
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return x;
}

// Maximum of a 64-bit value over the 64 lanes of a wave (DPP row shifts and row broadcasts on
// both halves; lanes outside a step's source read 0, the identity), returned to every lane.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t x) {
#define UMEM_MAX_STEP(CTRL, ROWS, BC)                                                        \
  {                                                                                          \
    const uint32_t lo = __builtin_amdgcn_update_dpp(0, static_cast<uint32_t>(x), CTRL, ROWS, 0xF, BC);  \
    const uint32_t hi = __builtin_amdgcn_update_dpp(0, static_cast<uint32_t>(x >> 32), CTRL, ROWS, 0xF, BC); \
    const uint64_t y = (static_cast<uint64_t>(hi) << 32) | lo;                               \
    x = y > x ? y : x;                                                                       \
  }
  UMEM_MAX_STEP(0x111, 0xF, true)    // row_shr:1
  UMEM_MAX_STEP(0x112, 0xF, true)    // row_shr:2
  UMEM_MAX_STEP(0x114, 0xF, true)    // row_shr:4
  UMEM_MAX_STEP(0x118, 0xF, true)    // row_shr:8
  UMEM_MAX_STEP(0x142, 0xA, false)   // row_bcast:15
  UMEM_MAX_STEP(0x143, 0xC, false)   // row_bcast:31
#undef UMEM_MAX_STEP
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(x), kWave - 1);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<uint32_t>(x >> 32), kWave - 1);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Sum over aligned groups of 2^lp consecutive lanes (every lane of a group gets the sum): the
// quad swaps, the half-row and row mirrors of DPP, then shuffles across rows.
__device__ __forceinline__ int group_sum(int r, int lp) {
  if (lp >= 1) r += __builtin_amdgcn_update_dpp(0, r, 0xB1, 0xF, 0xF, false);   // quad_perm 1,0,3,2
  if (lp >= 2) r += __builtin_amdgcn_update_dpp(0, r, 0x4E, 0xF, 0xF, false);   // quad_perm 2,3,0,1
  if (lp >= 3) r += __builtin_amdgcn_update_dpp(0, r, 0x141, 0xF, 0xF, false);  // row_half_mirror
  if (lp >= 4) r += __builtin_amdgcn_update_dpp(0, r, 0x140, 0xF, 0xF, false);  // row_mirror
  if (lp >= 5) r += __shfl_xor(r, 16, kWave);
  if (lp >= 6) r += __shfl_xor(r, 32, kWave);
  return r;
}

// The same for floats (IEEE addition commutes, so every lane of a group gets the same bits).
__device__ __forceinline__ float group_sum_f(float x, int lp) {
  int r = __builtin_bit_cast(int, x);
#define UMEM_FSTEP(CTRL) \
  r = __builtin_bit_cast(int, __builtin_bit_cast(float, r) + \
                         __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, r, CTRL, 0xF, 0xF, false)))
  if (lp >= 1) UMEM_FSTEP(0xB1);
  if (lp >= 2) UMEM_FSTEP(0x4E);
  if (lp >= 3) UMEM_FSTEP(0x141);
  if (lp >= 4) UMEM_FSTEP(0x140);
#undef UMEM_FSTEP
  return __builtin_bit_cast(float, r);
}

// Exclusive offset of each thread's count within waves [w0, w0 + nw), and their total.
// Called by every thread of the workgroup (it holds two barriers).
__device__ __forceinline__ int2 group_offsets(int cnt, int w0, int nw, SelectShared& sh) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int incl = wave_scan_dpp(cnt);
  if (lane == kWave - 1) sh.wave_tot[wave] = incl;
  __syncthreads();
  int base = 0, total = 0;
  for (int w = w0; w < w0 + nw; ++w) {
    const int tw = sh.wave_tot[w];
    base += (w < wave) ? tw : 0;
    total += tw;
  }
  __syncthreads();
  return make_int2(base + incl - cnt, total);
}

// Largest L with zero low 16 bits such that at least k of the wave's 64 G values v[] are
// >= L (k <= 64 G): eight radix-4 steps, each of three independent ballots.
template <int G>
__device__ __forceinline__ uint32_t wave_kth_largest16(const uint32_t (&v)[G], int k) {
  uint32_t p = 0u;
  for (int b = 30; b >= 16; b -= 2) {
    const uint32_t c1 = p | (1u << b), c2 = p | (2u << b), c3 = p | (3u << b);
    int n1 = 0, n2 = 0, n3 = 0;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      n1 += __popcll(__ballot(v[g] >= c1));
      n2 += __popcll(__ballot(v[g] >= c2));
      n3 += __popcll(__ballot(v[g] >= c3));
    }
    p = n3 >= k ? c3 : (n2 >= k ? c2 : (n1 >= k ? c1 : p));
  }
  return p;
}

// A valid threshold for a top-k from V maxima per lane (maxima of disjoint sets) in LDS:
// lane-wise they are merged into G = ceil(k / 32) (at most V) maxima of unions (still disjoint
// sets), and L, the k-th largest of those 64 G values with its low 16 bits cleared, has at
// least k elements >= L.  With at least two groups per wanted element L stays close to the
// k-th largest element (with one, it falls to the best of the worst group).  One wave.
template <int V>
__device__ __forceinline__ uint32_t threshold_from_maxima(const uint32_t* vals, int k) {
  const int lane = threadIdx.x & (kWave - 1);
  uint32_t v[V];
#pragma unroll
  for (int q = 0; q < V; ++q) v[q] = vals[lane + kWave * q];
  if (k <= kWave / 2) {
    uint32_t r[1] = {0u};
#pragma unroll
    for (int q = 0; q < V; ++q) r[0] = max(r[0], v[q]);
    return wave_kth_largest16<1>(r, k);
  }
  if (V >= 4 && k <= kWave) {
    uint32_t r[2] = {0u, 0u};
#pragma unroll
    for (int q = 0; q < V; ++q) r[q & 1] = max(r[q & 1], v[q]);
    return wave_kth_largest16<2>(r, k);
  }
  uint32_t r[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int q = 0; q < V; ++q) r[q & 3] = max(r[q & 3], v[q]);
  return wave_kth_largest16<4>(r, k);
}

// ---------------------------------------------------------------- per-axis top-k

// Element i of an axis is held by thread g of its group (g = threadIdx.x % 256) as key[j]:
// VEC == 4 (n % 4 == 0): i = 1024 j + 4 g + e, key[4 j + e]; VEC == 1: i = 256 j + g.
template <int VEC>
__device__ __forceinline__ int elem_index(int g, int j, int e) {
  return VEC == 4 ? 1024 * j + 4 * g + e : GROUP * j + g;
}

// Rank the S survivors of one axis in comp[0, S) with the axis's 256 threads: P = 2^lp threads
// per survivor (consecutive lanes), each counting the survivors before it among every P-th
// entry; ranks < k go to the axis list.
__device__ __forceinline__ void rank_axis(const uint64_t* comp, int S, int axis, int k, int g,
                                          SelectShared& sh) {
  int lp = 0;
  while (lp < 6 && (S << (lp + 1)) <= GROUP) ++lp;
  const int P = 1 << lp;
  for (int base = 0; base < (S << lp); base += GROUP) {
    const int slot = base + g;
    const int e = slot >> lp, part = slot & (P - 1);
    uint64_t me = 0ull;
    int r = 0;
    if (e < S) {
      me = comp[e];
      int u = part;
      for (; u + 3 * P < S; u += 4 * P) {
        const uint64_t b0 = comp[u], b1 = comp[u + P], b2 = comp[u + 2 * P], b3 = comp[u + 3 * P];
        r += static_cast<int>(b0 > me) + static_cast<int>(b1 > me) + static_cast<int>(b2 > me) +
             static_cast<int>(b3 > me);
      }
      for (; u < S; u += P) r += comp[u] > me;
    }
    r = group_sum(r, lp);
    if (part == 0 && e < S && r < k) {
      sh.ax_idx[axis][r] = static_cast<int>(0xFFFFFFFFu - static_cast<uint32_t>(me & 0xFFFFFFFFull));
      sh.ax_sc[axis][r] = key32_value(static_cast<uint32_t>(me >> 32));
    }
  }
}

// Both axes' top-k into sh.ax_idx / sh.ax_sc.
// The additive grid's candidates (a+1)(b+1) <= m as a table, row by row, and ceil(m / r) for
// the corner bound; one wave, while the score loads are in flight.
__device__ __forceinline__ void additive_tables(int k, int m, SelectShared& sh) {
  const int lane = threadIdx.x & (kWave - 1);
  const int R = min(k, m);
  int carry = 0;
  for (int a0 = 0; a0 < R; a0 += kWave) {
    const int a = a0 + lane;
    const int len = a < R ? min(k, m / (a + 1)) : 0;
    const int first = carry + wave_scan_dpp(len) - len;
    for (int b = 0; b < len; ++b) sh.grid_ab[first + b] = static_cast<uint16_t>((a << 8) | b);
    if (a < R) {
      const int c = (m + a) / (a + 1);                   // ceil(m / r), r = a + 1
      sh.th_col[a + 1] = static_cast<uint8_t>(c <= k ? c : 0);
    }
    carry = __shfl(first + len, kWave - 1, kWave);   // first already counts the earlier rows
  }
  if (lane == 0) sh.grid_total = carry;
}

// MODE only gives each kernel variant its own copy (with a single caller, the inliner treats it
// as it would in a single-variant build).
template <int NV, int VEC, int MODE>
__device__ void select_axes(const float* __restrict__ sel, int T, int H, int t, int h, int n, int k,
                            int m, bool tables, uint64_t* comp_all, SelectShared& sh) {
  constexpr int NE = NV * VEC;
  const int tid = threadIdx.x;
  const int axis = tid / GROUP;
  const int g = tid % GROUP;
  const int lane = tid & (kWave - 1);
  const float* src = sel + ((static_cast<size_t>(axis) * T + t) * H + h) * n;
  uint64_t* comp = comp_all + axis * SMAX_AX;
  uint32_t key[NE];
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    // the scores are read nontemporally: they stream through once (the keys the Tucker grid
    // reads back should stay in L2), and they were written from other XCDs (measured at decode:
    // 10.32 -> 10.06 us against plain loads)
    if (VEC == 4) {
      const f32x4* p = reinterpret_cast<const f32x4*>(src + min(1024 * j + 4 * g, n - 4));
      const f32x4 v = __builtin_nontemporal_load(p);
      key[4 * j + 0] = order_key(v.x);
      key[4 * j + 1] = order_key(v.y);
      key[4 * j + 2] = order_key(v.z);
      key[4 * j + 3] = order_key(v.w);
    } else {
      const float* p = src + min(GROUP * j + g, n - 1);
      key[j] = order_key(__builtin_nontemporal_load(p));
    }
  }
  if (tables && tid < kWave) additive_tables(k, m, sh);
  uint32_t mx = 0u;
#pragma unroll
  for (int j = 0; j < NV; ++j)
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const bool ok = elem_index<VEC>(g, j, e) < n;
      key[j * VEC + e] = ok ? key[j * VEC + e] : 0u;      // masked tail: below every element
      mx = ok ? max(mx, key[j * VEC + e]) : mx;
    }
  sh.mx[tid] = mx;
  __syncthreads();
  const uint32_t L = threshold_from_maxima<4>(sh.mx + axis * GROUP, k);   // in every wave
  uint32_t hit = 0u;                                      // bit j*VEC+e: element survives
#pragma unroll
  for (int j = 0; j < NV; ++j)
#pragma unroll
    for (int e = 0; e < VEC; ++e)
      hit |= static_cast<uint32_t>((elem_index<VEC>(g, j, e) < n) & (key[j * VEC + e] >= L)) << (j * VEC + e);
  const int cnt = __popc(hit);
  const int incl = wave_scan_dpp(cnt);
  const int tot = __shfl(incl, kWave - 1, kWave);
  int wbase = 0;
  if (lane == 0) wbase = atomicAdd(&sh.ax_cnt[axis], tot);
  wbase = __shfl(wbase, 0, kWave);
  if (wbase + tot <= SMAX_AX) {
    int pos = wbase + incl - cnt;
#pragma unroll
    for (int j = 0; j < NV; ++j)
#pragma unroll
      for (int e = 0; e < VEC; ++e)
        if ((hit >> (j * VEC + e)) & 1u) comp[pos++] = axis_comp(key[j * VEC + e], elem_index<VEC>(g, j, e));
  }
  __syncthreads();
  int S = sh.ax_cnt[axis];
  if (max(sh.ax_cnt[0], sh.ax_cnt[1]) > SMAX_AX) {
    // Massive ties on one axis: the exact k-th largest key theta over all its elements, then
    // the elements above it and the lowest-indexed elements equal to it.  Both groups run the
    // loop (its barriers are shared); only an overflowing axis writes.
    const bool overflow = S > SMAX_AX;
    uint32_t prefix = 0u;
    for (int b = 31; b >= 0; --b) {
      const uint32_t c = prefix | (1u << b);
      int cl = 0;
#pragma unroll
      for (int j = 0; j < NE; ++j) cl += key[j] >= c;       // masked keys are 0
      if (group_offsets(cl, axis * 4, 4, sh).y >= k) prefix = c;
    }
    const uint32_t theta = prefix;
    int gl = 0;
#pragma unroll
    for (int j = 0; j < NE; ++j) gl += key[j] > theta;
    const int need = k - group_offsets(gl, axis * 4, 4, sh).y;
    int pos = 0, eq_seen = 0;
    // element order: chunk j, then thread g, then e
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      int eq_l = 0;
#pragma unroll
      for (int e = 0; e < VEC; ++e) eq_l += (elem_index<VEC>(g, j, e) < n) & (key[j * VEC + e] == theta);
      const int2 oe = group_offsets(eq_l, axis * 4, 4, sh);
      int eq_rank = eq_seen + oe.x;
      int take_l = 0;
      bool take[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const bool ok = elem_index<VEC>(g, j, e) < n;
        const bool eq = ok & (key[j * VEC + e] == theta);
        take[e] = (ok & (key[j * VEC + e] > theta)) | (eq & (eq_rank < need));
        eq_rank += eq;
        take_l += take[e];
      }
      const int2 otk = group_offsets(take_l, axis * 4, 4, sh);
      if (overflow) {
        int p = pos + otk.x;
#pragma unroll
        for (int e = 0; e < VEC; ++e)
          if (take[e]) comp[p++] = axis_comp(key[j * VEC + e], elem_index<VEC>(g, j, e));
      }
      pos += otk.y;
      eq_seen += oe.y;
    }
    if (overflow) S = k;
    __syncthreads();
  }
  rank_axis(comp, S, axis, k, g, sh);
  __syncthreads();
}

// ---------------------------------------------------------------- top-m of candidates

// A candidate: its fp64 order key and its flat slot, in one 16-byte LDS record.
struct Cand {
  uint64_t key;
  int32_t id;
  int32_t pad;
};

__device__ __forceinline__ int before(const Cand& a, uint64_t ks, int is) {
  return static_cast<int>(a.key > ks) + static_cast<int>((a.key == ks) & (a.id < is));
}

// Rank the S candidates (key desc, id asc) with the whole workgroup: P = 2^lp threads per
// candidate (consecutive lanes), each counting the candidates before it among every P-th one;
// ranks < m go to sh.out_flat / sh.out_g.
__device__ __forceinline__ void rank_candidates(const Cand* cand, int S, int m, SelectShared& sh) {
  int lp = 0;
  while (lp < 6 && (S << (lp + 1)) <= THREADS) ++lp;
  const int P = 1 << lp;
  for (int base = 0; base < (S << lp); base += THREADS) {
    const int slot = base + static_cast<int>(threadIdx.x);
    const int e = slot >> lp, part = slot & (P - 1);
    uint64_t ks = 0ull;
    int is = 0, ab = 0, r = 0;
    if (e < S) {
      ks = cand[e].key;
      is = cand[e].id;
      ab = cand[e].pad;
      int u = part;
      for (; u + 3 * P < S; u += 4 * P) {
        const Cand b0 = cand[u], b1 = cand[u + P], b2 = cand[u + 2 * P], b3 = cand[u + 3 * P];
        r += before(b0, ks, is) + before(b1, ks, is) + before(b2, ks, is) + before(b3, ks, is);
      }
      for (; u < S; u += P) r += before(cand[u], ks, is);
    }
    r = group_sum(r, lp);
    if (part == 0 && e < S && r < m) {
      sh.out_flat[r] = is;
      sh.out_g[r] = key64_value(ks);
      sh.out_ab[r] = ab;
    }
  }
  __syncthreads();
}

// ---------------------------------------------------------------- a7 fused (decode)

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kPoolRowsPerWave = kMaxPoolTopM / NWAVES;

// This (token, head)'s m rows pooled into out_t[0, dv) with fp32 atomic adds.  Wave v reads rows
// v, v + 8, ... with 16-byte nontemporal loads (64 lanes x cpl chunks of a 1 or 2 KiB row, all
// of the wave's rows in flight), the 8 partial rows meet in LDS and are added in wave order, and
// each element takes one atomic add per head.
template <bool BF16>
__device__ void pool_rows(const void* __restrict__ values, int dv, int m, bool softmax, int cores,
                          const SelectShared& sh, float* red, float* __restrict__ out_t) {
  constexpr int EPC = BF16 ? 8 : 4;                  // elements per 16-byte chunk
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int cpl = dv * (BF16 ? 2 : 4) / 1024;        // 16-byte chunks per lane: 1 or 2
  const char* base = static_cast<const char*>(values);
  const size_t row_bytes = static_cast<size_t>(dv) * (BF16 ? 2 : 4);
  // with multi-core scoring a lane's chunk c takes the weight of the column slice it lies in
  // (a second chunk past a 1 KiB row is never loaded; its slice is clamped to a real one)
  int slice[2];
#pragma unroll
  for (int c = 0; c < 2; ++c)
    slice[c] = cores > 1 ? min(((kWave * c + lane) * EPC) / (dv / cores), cores - 1) : 0;
  u32x4 raw[kPoolRowsPerWave][2];
  float wt[kPoolRowsPerWave][2];
#pragma unroll
  for (int i = 0; i < kPoolRowsPerWave; ++i) {
    const int r = wave + NWAVES * i;
    wt[i][0] = wt[i][1] = 0.0f;
    raw[i][0] = raw[i][1] = u32x4{0u, 0u, 0u, 0u};
    if (r < m) {
      if (cores > 1) {
        wt[i][0] = sh.w_core[r * cores + slice[0]];
        wt[i][1] = sh.w_core[r * cores + slice[1]];
      } else {
        wt[i][0] = wt[i][1] = softmax ? sh.e[r] / sh.esum : static_cast<float>(sh.out_g[r]);
      }
      const u32x4* src = reinterpret_cast<const u32x4*>(base + static_cast<size_t>(sh.out_flat[r]) * row_bytes);
      raw[i][0] = __builtin_nontemporal_load(src + lane);
      if (cpl > 1) raw[i][1] = __builtin_nontemporal_load(src + kWave + lane);
    }
  }
  float acc[2][EPC];
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[c][e] = 0.0f;
#pragma unroll
  for (int i = 0; i < kPoolRowsPerWave; ++i)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const uint32_t q[4] = {raw[i][c].x, raw[i][c].y, raw[i][c].z, raw[i][c].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (BF16) {
          acc[c][2 * e] = fmaf(wt[i][c], __uint_as_float(q[e] << 16), acc[c][2 * e]);
          acc[c][2 * e + 1] = fmaf(wt[i][c], __uint_as_float(q[e] & 0xFFFF0000u), acc[c][2 * e + 1]);
        } else {
          acc[c][e] = fmaf(wt[i][c], __uint_as_float(q[e]), acc[c][e]);
        }
      }
    }
  // lane holds elements (64 c + lane) * EPC .. + EPC - 1 of chunk c
#pragma unroll
  for (int c = 0; c < 2; ++c)
    if (c < cpl) {
#pragma unroll
      for (int e = 0; e < EPC; e += 4)
        *reinterpret_cast<float4*>(red + wave * dv + (kWave * c + lane) * EPC + e) =
            make_float4(acc[c][e], acc[c][e + 1], acc[c][e + 2], acc[c][e + 3]);
    }
  __syncthreads();
  for (int col = tid; col < dv; col += THREADS) {
    float v = red[col];
#pragma unroll
    for (int u = 1; u < NWAVES; ++u) v += red[u * dv + col];
    atomicAdd(out_t + col, v);
  }
}

// ---------------------------------------------------------------- the kernel

template <int NV, int VEC, int MODE>
__global__ __launch_bounds__(THREADS) void select_kernel(
    const float* __restrict__ sel, const float* __restrict__ q_row,
    const float* __restrict__ q_col, const float* __restrict__ k_row,
    const float* __restrict__ k_col, const float* __restrict__ core_all,
    int32_t* __restrict__ idx_out, float* __restrict__ w_out, int32_t* __restrict__ axis_out,
    const void* __restrict__ values, int vbf16, int dv, float* __restrict__ pooled,
    int T, int H, int n, int dk, int rank, int k, int m, int grid_tucker, int softmax, int n_cand,
    int cores) {
  extern __shared__ __align__(16) unsigned char dyn[];
  __shared__ SelectShared sh;
  const int tucker = MODE == kModePool ? grid_tucker : MODE == kModeTucker;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int t = blockIdx.x / H;
  const int h = blockIdx.x % H;

  // ---- a3: the two axes, four waves each
  if (tucker && tid < rank * rank) {
    const float* ch = core_all + static_cast<size_t>(h) * cores * rank * rank;
    double c = 0.0;
    for (int i = 0; i < cores; ++i) {
      const float x = ch[i * rank * rank + tid];
      c += static_cast<double>(x);                 // eq. (16): the core is the sum
      if (cores > 1) sh.core_parts[i][tid] = x;
    }
    sh.core[tid] = c;
  }
  if (tid < 2) sh.ax_cnt[tid] = 0;
  if (tid == 0) sh.grid_cnt = 0;
  // Tucker: the token's two query rows (2 dk / 4 <= THREADS 16-byte pieces), loaded now, staged
  // in LDS for the exact per-slice scores once the axes are done with it
  const int n4 = dk >> 2;
  f32x4 q_piece = {0.0f, 0.0f, 0.0f, 0.0f};
  if (tucker && tid < 2 * n4) {
    const int ax = tid >= n4;
    q_piece = reinterpret_cast<const f32x4*>((ax ? q_col : q_row) + (static_cast<size_t>(t) * H + h) * dk)[tid - (ax ? n4 : 0)];
  }
  select_axes<NV, VEC, MODE>(sel, T, H, t, h, n, k, m, !tucker, reinterpret_cast<uint64_t*>(dyn), sh);
  if (axis_out != nullptr)
    for (int a = tid; a < 2 * k; a += THREADS)
      axis_out[((static_cast<size_t>(a / k) * T + t) * H + h) * k + a % k] = sh.ax_idx[a / k][a % k];

  Cand* cand = reinterpret_cast<Cand*>(dyn);                 // candidates, after the axes
  int S;
  if (!tucker) {
    // ---- a4 (additive): (a, b) with a, b < k and (a+1)(b+1) <= m, scores exact in fp64; every
    // wave first takes theta, the corner bound, itself
    const int R = min(k, m);
    uint64_t th = 0ull;
    for (int r0 = 1; r0 <= R; r0 += kWave) {
      const int r = r0 + lane;
      const int c = r <= R ? sh.th_col[r] : 0;
      if (c > 0)
        th = max(th, order_key64(static_cast<double>(sh.ax_sc[0][r - 1]) + static_cast<double>(sh.ax_sc[1][c - 1])));
    }
    th = wave_max_u64(th);
    const int C = sh.grid_total;
    for (int c0 = wave * kWave; c0 < C; c0 += THREADS) {
      const int c = c0 + lane;
      uint64_t key = 0ull;
      bool keep = false;
      int a = 0, b = 0;
      if (c < C) {
        const int ab = sh.grid_ab[c];
        a = ab >> 8;
        b = ab & 0xFF;
        key = order_key64(static_cast<double>(sh.ax_sc[0][a]) + static_cast<double>(sh.ax_sc[1][b]));
        keep = key >= th;
      }
      const uint64_t bal = __ballot(keep);
      int wbase = 0;
      if (lane == 0 && bal) wbase = atomicAdd(&sh.grid_cnt, static_cast<int>(__popcll(bal)));
      wbase = __shfl(wbase, 0, kWave);
      if (keep) {
        const int pos = wbase + static_cast<int>(__popcll(bal & lanemask_lt()));
        cand[pos].key = key;
        cand[pos].id = sh.ax_idx[0][a] * n + sh.ax_idx[1][b];
      }
    }
    __syncthreads();
    S = sh.grid_cnt;
  } else {
    // ---- a4 (Tucker): exact per-slice scores of the selected keys (eq. (4)), in fp32.  G = 4, 8
    // or 16 lanes per (axis, key) row, as many as 2k rows leave in the workgroup (one pass), and
    // L = G / 4, G / 2 or G lanes per slice of the row (rank 3 or 4, 2, 1): lane sub of a slice
    // takes its 16-byte pieces sub, sub + L, ... (the L lanes read contiguous 16L-byte runs),
    // eight loads in flight before any is used, and the L partial sums meet through DPP.
    {
      const f32x4* qs = reinterpret_cast<const f32x4*>(dyn);          // [2][n4] query pieces
      if (tid < 2 * n4) reinterpret_cast<f32x4*>(dyn)[tid] = q_piece;
      __syncthreads();
      constexpr int kPieces = 8;
      const int wp = n4 / rank;                                        // pieces per slice
      const int lg = 2 * k <= 32 ? 4 : (2 * k <= 64 ? 3 : 2);
      const int ls = rank == 1 ? lg : (rank == 2 ? lg - 1 : lg - 2);
      for (int job = tid; job < (2 * k) << lg; job += THREADS) {   // whole groups: G | THREADS
        const int part = job & ((1 << lg) - 1), row = job >> lg;
        const int axis = row >= k, a = row - (axis ? k : 0);
        const int rho = part >> ls, sub = part & ((1 << ls) - 1);
        const int cnt = rho < rank ? (wp - sub + (1 << ls) - 1) >> ls : 0;
        const int first = rho * wp + sub;
        const f32x4* kr = reinterpret_cast<const f32x4*>(
            (axis ? k_col : k_row) + (static_cast<size_t>(h) * n + sh.ax_idx[axis][a]) * dk) + first;
        const f32x4* qr = qs + axis * n4 + first;
        float acc = 0.0f;
        for (int i0 = 0; i0 < cnt; i0 += kPieces) {
          f32x4 kv[kPieces];
#pragma unroll
          for (int i = 0; i < kPieces; ++i)
            if (i0 + i < cnt) kv[i] = kr[(i0 + i) << ls];
#pragma unroll
          for (int i = 0; i < kPieces; ++i)
            if (i0 + i < cnt) {
              const f32x4 qv = qr[(i0 + i) << ls];
              acc = fmaf(kv[i].x, qv.x, acc);
              acc = fmaf(kv[i].y, qv.y, acc);
              acc = fmaf(kv[i].z, qv.z, acc);
              acc = fmaf(kv[i].w, qv.w, acc);
            }
        }
        acc = group_sum_f(acc, ls);
        if (rho < rank && sub == 0) sh.s_ex[axis][rho][a] = acc;
      }
    }
    __syncthreads();
    for (int job = tid; job < rank * k; job += THREADS) {
      const int rho = job / k, b = job % k;
      double p = 0.0;
      for (int sg = 0; sg < rank; ++sg)
        p += sh.core[rho * rank + sg] * static_cast<double>(sh.s_ex[1][sg][b]);
      sh.p_col[rho][b] = p;
    }
    __syncthreads();
    // Candidates in registers: thread tid < R k takes column b = tid mod k and rows a0 + R j
    // (a0 = tid / k, R = 512 / k, j < CPT; R >= 8 as k <= 64, so CPT = 8 rows cover a column).
    const int R = THREADS / k;
    const int b = tid % k, a0 = tid / k;
    const bool on = tid < R * k;
    double pc[kMaxRank];
#pragma unroll
    for (int r = 0; r < kMaxRank; ++r) pc[r] = (on && r < rank) ? sh.p_col[r][b] : 0.0;
    uint64_t k64[CPT];
    uint32_t k32[CPT];
    uint32_t valid = 0u;                              // bit j: row a0 + R j exists
    uint32_t mx = 0u;
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
      const int a = a0 + R * j;
      k64[j] = 0ull;
      k32[j] = 0u;
      if (on && a < k) {
        double gv = 0.0;
#pragma unroll
        for (int rho = 0; rho < kMaxRank; ++rho)            // pc[] indexed at compile time
          if (rho < rank) gv += static_cast<double>(sh.s_ex[0][rho][a]) * pc[rho];
        k64[j] = order_key64(gv);
        k32[j] = order_key(static_cast<float>(gv));
        mx = max(mx, k32[j]);
        valid |= 1u << j;
      }
    }
    sh.mx[tid] = mx;
    __syncthreads();
    // The threshold from all 512 thread maxima, unmerged (each covers up to 8 candidates of one
    // column): their m-th largest lies close to the m-th largest candidate.  Merged lane-wise
    // they would be column maxima, whose m-th largest (m = k) is the best score of the worst
    // column, below most of the grid.  One wave takes it, the others wait at the barrier.
    if (wave == 0) {
      uint32_t mxs[CPT];
#pragma unroll
      for (int q = 0; q < CPT; ++q) mxs[q] = sh.mx[lane + kWave * q];
      const uint32_t L0 = wave_kth_largest16<CPT>(mxs, m);
      if (lane == 0) sh.thr[0] = L0;
    }
    __syncthreads();
    const uint32_t L = sh.thr[0];
    int cnt = 0;
#pragma unroll
    for (int j = 0; j < CPT; ++j) cnt += ((valid >> j) & 1u) & (k32[j] >= L);
    const int2 o = group_offsets(cnt, 0, NWAVES, sh);
    if (o.y <= SMAX_S) {
      int pos = o.x;
#pragma unroll
      for (int j = 0; j < CPT; ++j) {
        const int a = a0 + R * j;
        if (((valid >> j) & 1u) && k32[j] >= L) {
          cand[pos].key = k64[j];
          cand[pos].id = sh.ax_idx[0][a] * n + sh.ax_idx[1][b];
          cand[pos].pad = (a << 8) | b;
          ++pos;
        }
      }
      __syncthreads();
      S = o.y;
    } else {
      // Massive ties: exact m-th largest fp64 key theta, then the lowest flat indices among
      // the candidates equal to it.
      int32_t fl[CPT];
#pragma unroll
      for (int j = 0; j < CPT; ++j)
        fl[j] = ((valid >> j) & 1u) ? sh.ax_idx[0][a0 + R * j] * n + sh.ax_idx[1][b] : 0x7FFFFFFF;
      uint64_t prefix = 0ull;
      for (int bit = 63; bit >= 0; --bit) {
        const uint64_t cb = prefix | (1ull << bit);
        int cl = 0;
#pragma unroll
        for (int j = 0; j < CPT; ++j) cl += ((valid >> j) & 1u) & (k64[j] >= cb);
        if (group_offsets(cl, 0, NWAVES, sh).y >= m) prefix = cb;
      }
      const uint64_t theta = prefix;
      int gl = 0;
#pragma unroll
      for (int j = 0; j < CPT; ++j) gl += ((valid >> j) & 1u) & (k64[j] > theta);
      const int need = m - group_offsets(gl, 0, NWAVES, sh).y;
      uint32_t ylim = 0u;     // the need-th smallest flat index among the keys equal to theta
      for (int bit = 31; bit >= 0; --bit) {
        const uint32_t cb = ylim | (1u << bit);
        int cl = 0;
#pragma unroll
        for (int j = 0; j < CPT; ++j)
          cl += ((valid >> j) & 1u) & (k64[j] == theta) & (static_cast<uint32_t>(fl[j]) < cb);
        if (group_offsets(cl, 0, NWAVES, sh).y < need) ylim = cb;
      }
      int tk = 0;
      uint32_t take = 0u;
#pragma unroll
      for (int j = 0; j < CPT; ++j) {
        const bool ok = ((valid >> j) & 1u) &&
                        ((k64[j] > theta) | ((k64[j] == theta) & (static_cast<uint32_t>(fl[j]) <= ylim)));
        take |= static_cast<uint32_t>(ok) << j;
        tk += ok;
      }
      const int2 ot = group_offsets(tk, 0, NWAVES, sh);
      int pos = ot.x;
#pragma unroll
      for (int j = 0; j < CPT; ++j) {
        if ((take >> j) & 1u) {
          cand[pos].key = k64[j];
          cand[pos].id = fl[j];
          cand[pos].pad = ((a0 + R * j) << 8) | b;
          ++pos;
        }
      }
      __syncthreads();
      S = m;
    }
  }

  // ---- a5: rank the candidates by (score desc, flat index asc); ranks < m are the answer
  rank_candidates(cand, S, m, sh);
  if (softmax) {
    for (int j = tid; j < m; j += THREADS) sh.e[j] = __expf(static_cast<float>(sh.out_g[j] - sh.out_g[0]));
    __syncthreads();
    if (wave == 0) {
      float s = 0.0f;
      for (int j = lane; j < m; j += kWave) s += sh.e[j];
      s = wave_sum(s);
      if (lane == 0) sh.esum = s;
    }
    __syncthreads();
  }
  for (int j = tid; j < m; j += THREADS) {
    const size_t o = (static_cast<size_t>(t) * H + h) * m + j;
    idx_out[o] = sh.out_flat[j];
    if (cores == 1) w_out[o] = softmax ? sh.e[j] / sh.esum : static_cast<float>(sh.out_g[j]);
  }
  if (cores > 1) {
    // multi-core scoring (eq. (16)): each core's exact score of every selected slot, in fp64
    for (int x = tid; x < m * cores; x += THREADS) {
      const int j = x / cores, i = x - (x / cores) * cores;
      const int a = sh.out_ab[j] >> 8, b = sh.out_ab[j] & 0xFF;
      double g = 0.0;
      for (int rho = 0; rho < rank; ++rho) {
        double p = 0.0;
        for (int sg = 0; sg < rank; ++sg)
          p += static_cast<double>(sh.core_parts[i][rho * rank + sg]) * static_cast<double>(sh.s_ex[1][sg][b]);
        g += static_cast<double>(sh.s_ex[0][rho][a]) * p;
      }
      sh.w_core[x] = static_cast<float>(g);
      w_out[((static_cast<size_t>(t) * H + h) * m + j) * cores + i] = static_cast<float>(g);
    }
    __syncthreads();
  }
  // ---- a7 fused: pool this head's rows into the token's output (the axes' LDS is free now)
  // (a run-time test also in the pooling variant: the decode kernel measured faster with it than
  // with the branch resolved at compile time)
  if (MODE == kModePool && pooled != nullptr) {
    float* red = reinterpret_cast<float*>(dyn);
    float* out_t = pooled + static_cast<size_t>(t) * dv;
    if (vbf16) pool_rows<true>(values, dv, m, softmax, cores, sh, red, out_t);
    else pool_rows<false>(values, dv, m, softmax, cores, sh, red, out_t);
  }
}

}  // namespace

int additive_candidates(int k, int m) {
  int c = 0;
  for (int a = 0; a < k && a < m; ++a) c += min(k, m / (a + 1));
  return c;
}

size_t select_lds_bytes(int n_cand, int tucker, int pool_dv) {
  const size_t axes = 2 * static_cast<size_t>(SMAX_AX) * 8;
  const size_t grid = static_cast<size_t>(tucker ? SMAX_S : 2 * n_cand) * sizeof(Cand);
  const size_t pool = static_cast<size_t>(NWAVES) * pool_dv * 4;
  return axes > grid ? (axes > pool ? axes : pool) : (grid > pool ? grid : pool);
}

bool select_pools(const umem_desc& d) {
  const int row_bytes = d.dv * (d.vdtype == UMEM_F32 ? 4 : 2);
  return d.expand == 1 && d.heads <= 2 && d.topm <= kMaxPoolTopM &&
         (row_bytes == 1024 || row_bytes == 2048);
}

hipError_t launch_select(const umem_desc& d, int T, const float* sel, const float* q_row,
                         const float* q_col, const float* k_row, const float* k_col,
                         const float* core, int32_t* idx, float* w, int32_t* axis_idx,
                         const void* values, float* pooled, hipStream_t s) {
  clear_stale_error();
  if (pooled != nullptr && !select_pools(d)) return hipErrorInvalidValue;
  if (T == 0) return hipSuccess;
  const int tucker = d.grid == UMEM_GRID_TUCKER;
  const int n_cand = tucker ? d.topk * d.topk : additive_candidates(d.topk, d.topm);
  if (tucker && n_cand > KK_MAX) return hipErrorInvalidValue;
  const size_t lds = select_lds_bytes(n_cand, tucker, pooled ? d.dv : 0);
  const dim3 grid(static_cast<unsigned>(T) * d.heads), block(THREADS);
#define UMEM_SELECT_P(NV, VEC, MODE)                                                              \
  hipLaunchKernelGGL((select_kernel<NV, VEC, MODE>), grid, block, lds, s, sel, q_row, q_col,     \
                     k_row, k_col, core, idx, w, axis_idx, values, d.vdtype == UMEM_BF16, d.dv,   \
                     pooled, T, d.heads, d.n_keys, d.dk, d.rank, d.topk,                         \
                     d.topm, tucker, d.weight == UMEM_W_SOFTMAX, n_cand, n_cores(d))
#define UMEM_SELECT(NV, VEC)                                                                      \
  do {                                                                                            \
    if (pooled != nullptr) UMEM_SELECT_P(NV, VEC, kModePool);                                     \
    else if (tucker) UMEM_SELECT_P(NV, VEC, kModeTucker);                                         \
    else UMEM_SELECT_P(NV, VEC, kModeAdd);                                                        \
  } while (0)
  const int n = d.n_keys;
  if (n % 4 == 0) {
    const int nv = (n + 1023) / 1024;
    if (nv <= 1) UMEM_SELECT(1, 4);
    else if (nv <= 2) UMEM_SELECT(2, 4);
    else if (nv <= 3) UMEM_SELECT(3, 4);
    else if (nv <= 4) UMEM_SELECT(4, 4);
    else if (nv <= 5) UMEM_SELECT(5, 4);
    else if (nv <= 6) UMEM_SELECT(6, 4);
    else if (nv <= 8) UMEM_SELECT(8, 4);
    else return hipErrorInvalidValue;
  } else {
    const int nv = (n + GROUP - 1) / GROUP;
    if (nv <= 1) UMEM_SELECT(1, 1);
    else if (nv <= 2) UMEM_SELECT(2, 1);
    else if (nv <= 4) UMEM_SELECT(4, 1);
    else if (nv <= 8) UMEM_SELECT(8, 1);
    else if (nv <= 16) UMEM_SELECT(16, 1);
    else if (nv <= 24) UMEM_SELECT(24, 1);
    else if (nv <= 32) UMEM_SELECT(32, 1);
    else return hipErrorInvalidValue;
  }
#undef UMEM_SELECT
#undef UMEM_SELECT_P
  return hipGetLastError();
}

}  // namespace umem
