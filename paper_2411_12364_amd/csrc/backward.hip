// Backward of the gather-sum (eq. (1), eq. (15) per virtual block, eq. (17) per column slice):
// the weight gradients dw[e] = <d_pooled[t_e, p_e], V[row_e]> (per slice with multi-core
// scoring) and the value-row gradients dV[row] += sum over the entries e on that row of
// w_e d_pooled[t_e, p_e].
//
// The T * bag entries are keyed by physical row and stably sorted (sort.hip), so the entries of
// one row form a run in their original order.  Runs are cut into pieces of at most 64 entries;
// a wave takes a piece, reads V[row] 16 bytes per lane at a time, and for each entry of the
// piece in order computes its weight gradient (a wave reduction per core) and adds w_e d_pooled
// into an fp32 accumulator, which it adds into dV[row] (a whole run) or stores as a partial row
// that a second pass adds in order.  Every row has one writer and a fixed summation order: the
// result does not depend on timing, and no atomics are needed.  The compact form writes one
// gradient row per run (distinct row) from zero instead of adding into a dense table.
//
// Backward of the scores (eqs. (2)-(4), (10), (16)) with the selection held fixed: one wave
// per (token, head) turns the weight gradients into grid-score gradients (SoftMax Jacobian where
// eq. (3)'s SoftMax weights), finds the distinct rows and columns of its slots (ballots over the
// key bits), recomputes their per-slice scores (Tucker), forms each slot's contribution to
// dS_row / dS_col and to dC, adds the contributions of slots that share a row (or column) in
// slot order, and writes dq = sum_i dS[i] K[i].  The key
// gradients dK[i] += dS[i] q are sums over tokens: each (token, head, axis) emits one entry per
// distinct key, the entries are stably sorted by key, and the key's pieces are summed in a fixed
// order as above.  dC sums its per-token partials in a fixed order (per thread, then a tree over
// the threads).
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

// The run [i, end) of sorted entries that starts at sorted position i (wave-uniform).
__device__ __forceinline__ int run_end(const uint32_t* __restrict__ keys, int i, int M, uint32_t key) {
  const int lane = threadIdx.x & (kWave - 1);
  for (int base = i + 1; base < M; base += kWave) {
    const int pos = base + lane;
    const uint64_t same = __ballot(pos < M && keys[pos] == key);
    if (same != ~0ull) return base + __builtin_ctzll(~same);
  }
  return M;
}

// The sorted entries are cut into pieces at the starts of runs and at every kSeg-th position, and
// each piece is one wave's work, so that a row chosen by thousands of tokens does not leave one
// wave walking them all while a row chosen once still gets a wave of its own.  The piece starts
// are listed first (counted per chunk, the counts scanned, then written in order), and a fixed
// grid of waves walks the list.  A piece that is a
// whole run adds its sum into its row; a piece cut by a segment edge (segment g = positions
// [g kSeg, (g + 1) kSeg)) stores its partial row: slot 2 g + 1 for the last piece of segment g
// when it starts its run, slot 2 g for the first piece of segment g when it continues one.  A
// second pass adds, for each run spanning segments, its head piece and then the first piece of
// each later segment, in that order.
constexpr int kSeg = kWave;

// The piece starting at sorted position i, if one does ([i, *pe), with whether it starts and
// ends its run); false for positions inside a piece.  Wave-uniform.
__device__ __forceinline__ bool piece_at(const uint32_t* __restrict__ keys, int i, int M,
                                         uint32_t key, int* pe, bool* run_start, bool* run_end) {
  const int lane = threadIdx.x & (kWave - 1);
  *run_start = i == 0 || keys[i - 1] != key;
  if (!*run_start && i % kSeg != 0) return false;
  const int seg_end = min(M, (i / kSeg + 1) * kSeg);
  const int pos = i + 1 + lane;
  const uint64_t diff = __ballot(pos < seg_end && keys[pos] != key);
  *pe = diff != 0ull ? i + 1 + __builtin_ctzll(diff) : seg_end;
  *run_end = *pe == M || keys[*pe] != key;
  return true;
}

constexpr int kListWaves = 8192;        // waves of the grids that walk the key lists (b2)
// ... and the value-row lists (b1): four waves per SIMD, which the piece kernel's registers allow;
// more value-row loads in flight pay where rows repeat (measured at tucker-ive-4M: 473 -> 453 us)
constexpr int kValueListWaves = 16384;
constexpr int kInFlight = 4;            // a piece's entries whose loads are issued together

constexpr int kListPer = 16;                           // positions per thread
constexpr int kListChunk = THREADS * kListPer;          // positions per workgroup

__device__ __forceinline__ bool is_piece_start(const uint32_t* __restrict__ keys, int i, int M,
                                               uint32_t sentinel) {
  if (i >= M) return false;
  const uint32_t k = keys[i];
  return k != sentinel && (i % kSeg == 0 || keys[i - 1] != k);
}

// Exclusive prefix of v over the workgroup's threads, in thread order (every thread calls it).
__device__ __forceinline__ uint32_t block_prefix(uint32_t v, uint32_t* lds, uint32_t* total) {
  const int tid = threadIdx.x;
  lds[tid] = v;
  __syncthreads();
  for (int off = 1; off < THREADS; off <<= 1) {
    const uint32_t add = tid >= off ? lds[tid - off] : 0u;
    __syncthreads();
    lds[tid] += add;
    __syncthreads();
  }
  const uint32_t incl = lds[tid];
  *total = lds[THREADS - 1];
  __syncthreads();
  return incl - v;
}

// A run of the sorted keys starts here (the compact row output numbers runs, not rows).
__device__ __forceinline__ bool is_run_start(const uint32_t* __restrict__ keys, int i, int M) {
  return i < M && (i == 0 || keys[i - 1] != keys[i]);
}

// Per chunk of kListChunk positions: its piece starts into offs[chunk] and, with runs wanted, its
// run starts into offs[chunks + chunk]; one exclusive scan over both halves follows.
__global__ __launch_bounds__(THREADS) void piece_count_kernel(const uint32_t* __restrict__ keys,
                                                              int M, uint32_t sentinel,
                                                              uint32_t* __restrict__ offs,
                                                              int runs) {
  __shared__ uint32_t lds[THREADS];
  const int beg = blockIdx.x * kListChunk + threadIdx.x * kListPer;
  uint32_t c = 0, cr = 0;
  for (int k = 0; k < kListPer; ++k) {
    c += is_piece_start(keys, beg + k, M, sentinel);
    if (runs) cr += is_run_start(keys, beg + k, M);
  }
  uint32_t total;
  block_prefix(c, lds, &total);
  if (threadIdx.x == 0) offs[blockIdx.x] = total;
  if (runs) {
    block_prefix(cr, lds, &total);
    if (threadIdx.x == 0) offs[gridDim.x + blockIdx.x] = total;
  }
}

// offs: the scanned counts.  Writes the piece starts in order into list, their number into
// counts[0] (counts[1] cleared); with run_of given also every position's run number, each run's
// key into rows_out[run] (ascending) and the number of runs into *n_runs.
__global__ __launch_bounds__(THREADS) void piece_write_kernel(const uint32_t* __restrict__ keys,
                                                              int M, uint32_t sentinel,
                                                              const uint32_t* __restrict__ offs,
                                                              uint32_t* __restrict__ list,
                                                              uint32_t* __restrict__ counts,
                                                              uint32_t* __restrict__ run_of,
                                                              int32_t* __restrict__ rows_out,
                                                              int32_t* __restrict__ n_runs) {
  __shared__ uint32_t lds[THREADS];
  const int beg = blockIdx.x * kListChunk + threadIdx.x * kListPer;
  uint32_t c = 0;
  for (int k = 0; k < kListPer; ++k) c += is_piece_start(keys, beg + k, M, sentinel);
  uint32_t total;
  uint32_t at = offs[blockIdx.x] + block_prefix(c, lds, &total);
  for (int k = 0; k < kListPer; ++k)
    if (is_piece_start(keys, beg + k, M, sentinel)) list[at++] = static_cast<uint32_t>(beg + k);
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) {
    counts[0] = offs[blockIdx.x] + total;
    counts[1] = 0u;                                       // the spanning runs, appended later
  }
  if (run_of == nullptr) return;                          // (uniform over the grid)
  uint32_t cr = 0;
  for (int k = 0; k < kListPer; ++k) cr += is_run_start(keys, beg + k, M);
  const uint32_t pieces = offs[gridDim.x];                // the scan's offset of the run half
  uint32_t total_r;
  uint32_t r = offs[gridDim.x + blockIdx.x] - pieces + block_prefix(cr, lds, &total_r);
  for (int k = 0; k < kListPer && beg + k < M; ++k) {
    if (is_run_start(keys, beg + k, M)) rows_out[r++] = static_cast<int32_t>(keys[beg + k]);
    run_of[beg + k] = r - 1;                              // position 0 starts a run: r >= 1 here
  }
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0)
    *n_runs = static_cast<int32_t>(offs[gridDim.x + blockIdx.x] - pieces + total_r);
}

size_t list_workspace_bytes(int M) {
  const size_t chunks = (static_cast<size_t>(M) + kListChunk - 1) / kListChunk;
  return (2 * chunks + 1) * sizeof(uint32_t) + scan_workspace_bytes(static_cast<int>(2 * chunks)) + 64;
}

// The piece starts of the sorted keys into list (in order) and their number into counts[0];
// counts[1] cleared.  With run_of given (keys without the sentinel), also the runs as
// piece_write_kernel states.  ws: list_workspace_bytes(M).
hipError_t list_pieces(const uint32_t* keys, int M, uint32_t sentinel, uint32_t* list,
                       uint32_t* counts, void* ws, hipStream_t s, uint32_t* run_of = nullptr,
                       int32_t* rows_out = nullptr, int32_t* n_runs = nullptr) {
  const int chunks = (M + kListChunk - 1) / kListChunk;
  const int runs = run_of != nullptr ? 1 : 0;
  uint32_t* offs = static_cast<uint32_t*>(ws);
  uint32_t* sums = offs + 2 * chunks + 1;
  hipLaunchKernelGGL(piece_count_kernel, dim3(chunks), dim3(THREADS), 0, s, keys, M, sentinel, offs,
                     runs);
  hipError_t e = scan_exclusive(offs, (1 + runs) * chunks, sums, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(piece_write_kernel, dim3(chunks), dim3(THREADS), 0, s, keys, M, sentinel, offs,
                     list, counts, run_of, rows_out, n_runs);
  return hipGetLastError();
}

// With run_of given (compact row output), a row's gradient goes to out[run_of[position] * dv],
// written from zero; otherwise it is added into out[row * dv].  Either way the value stored is
// (the row's previous value, or 0) + the row's sum, so a compact row holds exactly what the
// dense form adds into a zeroed row.
template <typename Elem>
__global__ __launch_bounds__(THREADS) void gather_bwd_seg_kernel(
    const uint32_t* __restrict__ rows, const uint32_t* __restrict__ ents, int M,
    const Elem* __restrict__ values, int dv, const int32_t* __restrict__ idx,
    const float* __restrict__ w, const int32_t* __restrict__ perm, int64_t n_values, int expand,
    int cores, int bag, const float* __restrict__ d_pooled, float* __restrict__ d_values,
    float* __restrict__ dw, float* __restrict__ partial, const uint32_t* __restrict__ list,
    uint32_t* __restrict__ counts, uint32_t* __restrict__ heads, const uint32_t* __restrict__ run_of) {
  constexpr int EPC = Chunk<Elem>::kElems;            // elements per 16-byte piece
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t n_pieces = counts[0];
  for (uint32_t k = blockIdx.x * NWAVES + threadIdx.x / kWave; k < n_pieces;
       k += gridDim.x * NWAVES) {                     // wave-uniform: no barrier in this kernel
  const int ps = static_cast<int>(list[k]);
  const uint32_t row = rows[ps];
  int pe;
  bool run_start, run_end;
  piece_at(rows, ps, M, row, &pe, &run_start, &run_end);
  if (run_start && !run_end && lane == 0)            // a run spanning segments: list its head
    heads[atomicAdd(counts + 1, 1u)] = static_cast<uint32_t>(ps);
  const int g = ps / kSeg;
  const int slice_w = dv / cores;
  // the piece's entries, one per lane: entry number and the d_pooled row (token, virtual block)
  const int n_e = pe - ps;
  int my_ent = 0, my_prow = 0;
  if (lane < n_e) {
    my_ent = static_cast<int>(ents[ps + lane]);
    const int p = perm != nullptr ? static_cast<int>(perm[idx[my_ent]] / n_values) : 0;
    my_prow = (my_ent / bag) * expand + p;
  }
  const Elem* vrow = values + static_cast<size_t>(row) * dv;
  float* drow = d_values + static_cast<size_t>(run_of != nullptr ? run_of[ps] : row) * dv;
  // lane j holds entry j's weight gradient per core, summed over the column steps in order and
  // written once at the end of the piece
  float my_dw[kMaxCores];
#pragma unroll
  for (int c = 0; c < kMaxCores; ++c) my_dw[c] = 0.0f;
  for (int c0 = 0; c0 < dv; c0 += kWave * EPC) {
    const int col = c0 + lane * EPC;
    const bool active = col < dv;
    const int sl = active ? col / slice_w : 0;        // a piece lies in one column slice
    float x[EPC], acc[EPC];
#pragma unroll
    for (int k = 0; k < EPC; ++k) {
      x[k] = 0.0f;
      acc[k] = 0.0f;
    }
    if (active) Chunk<Elem>::load(vrow + col, x);
    // a whole run adds into its gradient row: read that row now, under the entries' loads
    // (a compact row starts from zero)
    const bool whole = run_start && run_end;
    f32x4 old[EPC / 4];
#pragma unroll
    for (int k = 0; k < EPC / 4; ++k)
      old[k] = (active && whole && run_of == nullptr) ? *reinterpret_cast<const f32x4*>(drow + col + 4 * k)
                                                      : f32x4{0.f, 0.f, 0.f, 0.f};
    for (int j0 = 0; j0 < n_e; j0 += kInFlight) {    // wave-uniform
      int ent[kInFlight];
      float wt[kInFlight];
      f32x4 v[kInFlight][EPC / 4];
#pragma unroll
      for (int u = 0; u < kInFlight; ++u) {          // all loads first
        const int j = min(j0 + u, n_e - 1);
        ent[u] = __builtin_amdgcn_readlane(my_ent, j);
        const int prow = __builtin_amdgcn_readlane(my_prow, j);
        wt[u] = 0.0f;
#pragma unroll
        for (int k = 0; k < EPC / 4; ++k) v[u][k] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        if (active && j0 + u < n_e) {                // (past the piece's end: no loads)
          wt[u] = w[static_cast<size_t>(ent[u]) * cores + sl];
          const f32x4* src = reinterpret_cast<const f32x4*>(d_pooled + static_cast<size_t>(prow) * dv + col);
#pragma unroll
          for (int k = 0; k < EPC / 4; ++k) v[u][k] = src[k];
        }
      }
#pragma unroll
      for (int u = 0; u < kInFlight; ++u) {          // then the entries in order
        if (j0 + u >= n_e) break;
        float dot = 0.0f;
#pragma unroll
        for (int k = 0; k < EPC; k += 4) {
          const f32x4 vv = v[u][k / 4];
          dot = fmaf(vv.x, x[k], dot);
          dot = fmaf(vv.y, x[k + 1], dot);
          dot = fmaf(vv.z, x[k + 2], dot);
          dot = fmaf(vv.w, x[k + 3], dot);
          acc[k] = fmaf(wt[u], vv.x, acc[k]);
          acc[k + 1] = fmaf(wt[u], vv.y, acc[k + 1]);
          acc[k + 2] = fmaf(wt[u], vv.z, acc[k + 2]);
          acc[k + 3] = fmaf(wt[u], vv.w, acc[k + 3]);
        }
#pragma unroll
        for (int c = 0; c < kMaxCores; ++c) {
          if (c >= cores) break;
          const float sc = wave_sum(sl == c ? dot : 0.0f);
          if (lane == j0 + u) my_dw[c] = c0 == 0 ? sc : my_dw[c] + sc;
        }
      }
    }
    if (!active) continue;
    if (whole) {                                      // a whole run: add into its row
#pragma unroll
      for (int k = 0; k < EPC; k += 4) {
        f32x4 v = old[k / 4];
        v.x += acc[k]; v.y += acc[k + 1]; v.z += acc[k + 2]; v.w += acc[k + 3];
        *reinterpret_cast<f32x4*>(drow + col + k) = v;
      }
    } else {                                          // cut by a segment edge: its partial row
      float* dst = partial + (static_cast<size_t>(2) * g + (run_start ? 1 : 0)) * dv + col;
#pragma unroll
      for (int k = 0; k < EPC; k += 4)
        *reinterpret_cast<f32x4*>(dst + k) = f32x4{acc[k], acc[k + 1], acc[k + 2], acc[k + 3]};
    }
  }
  if (lane < n_e) {                                   // this wave is the entries' only writer
#pragma unroll
    for (int c = 0; c < kMaxCores; ++c) {
      if (c >= cores) break;
      dw[static_cast<size_t>(my_ent) * cores + c] = my_dw[c];
    }
  }
  }
}

// One wave per run that spans segments: its partial rows, in segment order, added into the row.
__global__ __launch_bounds__(THREADS) void seg_join_kernel(const uint32_t* __restrict__ keys, int M,
                                                           int width, const float* __restrict__ partial,
                                                           float* __restrict__ out,
                                                           const uint32_t* __restrict__ heads,
                                                           const uint32_t* __restrict__ counts,
                                                           int H, int n, float* __restrict__ out2,
                                                           const uint32_t* __restrict__ run_of) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t n_heads = counts[1];
  for (uint32_t hk = blockIdx.x * NWAVES + threadIdx.x / kWave; hk < n_heads;
       hk += gridDim.x * NWAVES) {
  const int i = static_cast<int>(heads[hk]);
  const uint32_t key = keys[i];
  const int g0 = i / kSeg;
  const int end = run_end(keys, i, M, key);
  const int g1 = (end - 1) / kSeg;
  // the row of this key: value rows directly, or (out2 given) key rows of the two axes
  float* dst;
  if (run_of != nullptr) {                           // compact rows: written from zero
    dst = out + static_cast<size_t>(run_of[i]) * width;
  } else if (out2 == nullptr) {
    dst = out + static_cast<size_t>(key) * width;
  } else {
    const int axis = static_cast<int>(key / (static_cast<uint32_t>(H) * n));
    dst = (axis ? out2 : out) + static_cast<size_t>(key - static_cast<uint32_t>(axis) * H * n) * width;
  }
  for (int c = lane * 4; c < width; c += kWave * 4) {
    f32x4 acc = *reinterpret_cast<const f32x4*>(partial + (static_cast<size_t>(2) * g0 + 1) * width + c);
    for (int g = g0 + 1; g <= g1; ++g)
      acc += *reinterpret_cast<const f32x4*>(partial + static_cast<size_t>(2) * g * width + c);
    f32x4* d = reinterpret_cast<f32x4*>(dst + c);
    f32x4 v = run_of != nullptr ? f32x4{0.f, 0.f, 0.f, 0.f} : *d;
    v += acc;
    *d = v;
  }
  }
}

// ---------------------------------------------------------------- score backward

// One wave per (token, head); slot s = g * 64 + lane for the NG groups g of a lane.  The waves
// of a workgroup share nothing, so the kernel has no workgroup barrier; each wave's own LDS
// traffic is ordered by wave_sync.
template <int NG>
struct ScoreBwdLds {
  int dist[2][NG * kWave];                     // distinct rows / columns, in slot order
  float sd[2][NG * kWave][kMaxRank];           // per distinct key: its per-slice score, then its dS
  float cs[2][NG * kWave][kMaxRank];           // per slot: its dS_row / dS_col term
};

template <int NG>
constexpr int score_bwd_waves() { return NG >= 4 ? 2 : 4; }

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The lanes whose key_other (valid_other) equals this lane's key: one ballot per key bit.
__device__ __forceinline__ uint64_t key_match(uint32_t key, uint32_t key_other, bool valid_other,
                                              int bits) {
  uint64_t mask = __ballot(valid_other);
  for (int b = 0; b < bits; ++b) {
    const uint64_t ones = __ballot(valid_other && ((key_other >> b) & 1u));
    mask &= ((key >> b) & 1u) ? ones : ~ones;
  }
  return mask;
}

template <int NG>
__global__ __launch_bounds__(score_bwd_waves<NG>() * kWave) void score_bwd_kernel(
    const float* __restrict__ q_row, const float* __restrict__ q_col,
    const float* __restrict__ k_row, const float* __restrict__ k_col,
    const float* __restrict__ core_all, const int32_t* __restrict__ idx,
    const float* __restrict__ w, const float* __restrict__ dw, int T, int H, int n, int key_bits,
    int dk, int rank, int m, int tucker, int softmax, int hc, float* __restrict__ dq_row,
    float* __restrict__ dq_col, uint32_t* __restrict__ ekeys, uint32_t* __restrict__ evals,
    float* __restrict__ edS, float* __restrict__ dc_part) {
  constexpr int W = score_bwd_waves<NG>();
  __shared__ ScoreBwdLds<NG> lds[W];
  const int lane = threadIdx.x & (kWave - 1);
  ScoreBwdLds<NG>& sh = lds[threadIdx.x / kWave];
  // (token, head) pairs in head-major order, dealt to the eight XCDs in contiguous runs
  // (workgroups go to XCDs round-robin): an XCD's pairs then share few heads, and their key rows
  // stay in its L2 for the two passes over them below
  const int64_t pairs = static_cast<int64_t>(T) * H;
  const int64_t nwg = gridDim.x, per = nwg >> 3, extra = nwg & 7;
  const int64_t xcd = blockIdx.x & 7;
  const int64_t wg = xcd * per + (xcd < extra ? xcd : extra) + (blockIdx.x >> 3);
  const int64_t q = wg * W + threadIdx.x / kWave;
  if (q >= pairs) return;                             // wave-uniform
  const int h = static_cast<int>(q / T);
  const size_t th = static_cast<size_t>(q % T) * H + h;
  const int R = tucker ? rank : 1;
  bool valid[NG];
  uint32_t key[2][NG];                                 // row, column of each slot
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int s = g * kWave + lane;
    valid[g] = s < m;
    const uint32_t flat = valid[g] ? static_cast<uint32_t>(idx[th * m + s]) : 0u;
    key[0][g] = flat / static_cast<uint32_t>(n);
    key[1][g] = flat % static_cast<uint32_t>(n);
  }
  // ---- weight gradients -> grid-score gradients (SoftMax Jacobian where eq. (3) weights)
  float dg[NG][kMaxCores];
  if (softmax) {
    float p = 0.0f;
#pragma unroll
    for (int g = 0; g < NG; ++g)
      if (valid[g]) p = fmaf(w[th * m + g * kWave + lane], dw[th * m + g * kWave + lane], p);
    const float wdot = wave_sum(p);                    // identical in every lane
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const size_t x = th * m + g * kWave + lane;
      dg[g][0] = valid[g] ? w[x] * (dw[x] - wdot) : 0.0f;
    }
  } else {
#pragma unroll
    for (int g = 0; g < NG; ++g)
#pragma unroll
      for (int c = 0; c < kMaxCores; ++c)
        dg[g][c] = valid[g] && c < hc ? dw[(th * m + g * kWave + lane) * hc + c] : 0.0f;
  }
  // ---- distinct keys per axis: a slot leads its key when no earlier slot holds it; pos is the
  // number of leaders before the key's leader
  int first[2][NG], pos[2][NG], nd[2];
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    uint64_t lead[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      int f = -1;
#pragma unroll
      for (int g2 = 0; g2 <= g; ++g2) {
        const uint64_t mm = key_match(key[a][g], key[a][g2], valid[g2], key_bits);
        if (f < 0 && mm != 0ull) f = g2 * kWave + __builtin_ctzll(mm);
      }
      first[a][g] = f;
      lead[g] = __ballot(valid[g] && f == g * kWave + lane);
    }
    int total = 0;
#pragma unroll
    for (int g = 0; g < NG; ++g) total += __popcll(lead[g]);
    nd[a] = total;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const int f = valid[g] ? first[a][g] : 0;
      int p = 0;
#pragma unroll
      for (int g2 = 0; g2 < NG; ++g2) {
        if (g2 < f / kWave) p += __popcll(lead[g2]);
        if (g2 == f / kWave) p += __popcll(lead[g2] & ((1ull << (f % kWave)) - 1ull));
      }
      pos[a][g] = p;
      if (valid[g] && f == g * kWave + lane) sh.dist[a][p] = static_cast<int>(key[a][g]);
    }
  }
  wave_sync();
  // ---- Tucker: per-slice scores of the distinct keys, four lanes per key row.  The quad is
  // split into one group per slice (4, 2 or 1 lanes for rank 1, 2, 3-4; rank 3 leaves a lane
  // idle); a lane strides its slice's 16-byte pieces by the group width, eight loads in flight,
  // and the group's partial sums meet through DPP in a fixed order.
  float sr[NG][kMaxRank] = {}, sc[NG][kMaxRank] = {};
  if (tucker) {
    constexpr int kPieces = 8;
    const int n4 = dk >> 2, wp = n4 / rank;                   // pieces per row, per slice
    const int part = lane & 3;
    const int ls = rank == 1 ? 2 : (rank == 2 ? 1 : 0);       // log2 lanes per slice
    const int rho = part >> ls, sub = part & ((1 << ls) - 1);
    const int cnt = rho < rank ? (wp - sub + (1 << ls) - 1) >> ls : 0;
    const int first = rho * wp + sub;
    const int jobs = nd[0] + nd[1];
    for (int j0 = 0; j0 < jobs; j0 += kWave / 4) {     // wave-uniform trip count
      const int kk = j0 + lane / 4;
      const bool ok = kk < jobs;                       // uniform across each quad
      const int a = kk >= nd[0] ? 1 : 0;
      const int k = kk - (a ? nd[0] : 0);
      float acc = 0.0f;
      if (ok) {
        const float4* kr = reinterpret_cast<const float4*>(
            (a ? k_col : k_row) + (static_cast<size_t>(h) * n + sh.dist[a][k]) * dk) + first;
        const float4* qr = reinterpret_cast<const float4*>((a ? q_col : q_row) + th * dk) + first;
        for (int i0 = 0; i0 < cnt; i0 += kPieces) {
          float4 kv[kPieces];
#pragma unroll
          for (int i = 0; i < kPieces; ++i)
            if (i0 + i < cnt) kv[i] = kr[(i0 + i) << ls];
#pragma unroll
          for (int i = 0; i < kPieces; ++i)
            if (i0 + i < cnt) {
              const float4 qv = qr[(i0 + i) << ls];
              acc = fmaf(kv[i].x, qv.x, acc);
              acc = fmaf(kv[i].y, qv.y, acc);
              acc = fmaf(kv[i].z, qv.z, acc);
              acc = fmaf(kv[i].w, qv.w, acc);
            }
        }
      }
      // the slice group's sum (every lane takes part)
      if (ls >= 1) acc += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, acc), 0xB1, 0xF, 0xF, false));
      if (ls >= 2) acc += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, acc), 0x4E, 0xF, 0xF, false));
      if (ok && rho < rank && sub == 0) sh.sd[a][k][rho] = acc;
      if (ok && part == 0)
        for (int r = rank; r < kMaxRank; ++r) sh.sd[a][k][r] = 0.0f;
    }
    wave_sync();
#pragma unroll
    for (int g = 0; g < NG; ++g)
#pragma unroll
      for (int r = 0; r < kMaxRank; ++r) {
        sr[g][r] = valid[g] ? sh.sd[0][pos[0][g]][r] : 0.0f;
        sc[g][r] = valid[g] ? sh.sd[1][pos[1][g]][r] : 0.0f;
      }
  }
  // ---- each slot's dS terms: d score / d s_row = C s_col, d score / d s_col = C^T s_row (eq. (10))
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    if (!valid[g]) continue;
    const int s = g * kWave + lane;
    if (!tucker) {
      sh.cs[0][s][0] = dg[g][0];
      sh.cs[1][s][0] = dg[g][0];
      continue;
    }
    for (int r = 0; r < rank; ++r) {
      float x0 = 0.0f, x1 = 0.0f;
#pragma unroll
      for (int c = 0; c < kMaxCores; ++c) {
        if (c >= hc) break;
        const float* C = core_all + (static_cast<size_t>(h) * hc + c) * rank * rank;
        float ca = 0.0f, cb = 0.0f;
#pragma unroll
        for (int x = 0; x < kMaxRank; ++x) {
          if (x >= rank) break;
          ca = fmaf(C[r * rank + x], sc[g][x], ca);
          cb = fmaf(C[x * rank + r], sr[g][x], cb);
        }
        x0 = fmaf(dg[g][c], ca, x0);
        x1 = fmaf(dg[g][c], cb, x1);
      }
      sh.cs[0][s][r] = x0;
      sh.cs[1][s][r] = x1;
    }
  }
  // ---- dC partial of this (token, head): sum over slots of dg s_row s_col^T (a wave sum)
  if (tucker) {
    for (int x = 0; x < hc * rank * rank; ++x) {    // wave-uniform
      const int c = x / (rank * rank), r = (x / rank) % rank, z = x % rank;
      float v = 0.0f;
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        float d = 0.0f, a = 0.0f, b = 0.0f;
#pragma unroll
        for (int cc = 0; cc < kMaxCores; ++cc) d = cc == c ? dg[g][cc] : d;
#pragma unroll
        for (int q = 0; q < kMaxRank; ++q) {
          a = q == r ? sr[g][q] : a;
          b = q == z ? sc[g][q] : b;
        }
        v = fmaf(d, a * b, v);
      }
      v = wave_sum(v);
      if (lane == 0) dc_part[th * hc * rank * rank + x] = v;
    }
  }
  wave_sync();
  // ---- dS per distinct key: its slots' terms in slot order, summed by the leading slot
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const bool leads = valid[g] && first[a][g] == g * kWave + lane;
      float acc[kMaxRank] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int g2 = g; g2 < NG; ++g2) {
        uint64_t mm = key_match(key[a][g], key[a][g2], valid[g2], key_bits);
        if (!leads) continue;
        while (mm != 0ull) {
          const int x = g2 * kWave + __builtin_ctzll(mm);
          mm &= mm - 1ull;
#pragma unroll
          for (int r = 0; r < kMaxRank; ++r)
            if (r < R) acc[r] += sh.cs[a][x][r];
        }
      }
      if (leads)
#pragma unroll
        for (int r = 0; r < kMaxRank; ++r) sh.sd[a][pos[a][g]][r] = acc[r];
    }
  wave_sync();
  // ---- dq = sum over distinct keys of dS K (eqs. (2) / (4) transposed)
  const int width = dk / R;
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    const float* Kh = (a ? k_col : k_row) + static_cast<size_t>(h) * n * dk;
    float* dq = (a ? dq_col : dq_row) + th * dk;
    const int nk = nd[a];
    if (dk % 4 == 0 && (dk > 2 * kWave || (dk & (dk - 1)) == 0) &&
        (reinterpret_cast<uintptr_t>(dq) & 15u) == 0) {
      // four dims per lane (16-byte loads); rows of at most 128 dims take S = 64 / (dk / 4) keys
      // per load, lane group s summing keys s, s + S, ... in order, the groups then meeting by a
      // fixed butterfly of shuffles; wider rows go in passes of 256 dims, each lane's sum in key
      // order
      const int G = dk <= 2 * kWave ? dk / 4 : kWave, S = kWave / G;
      const int sub = lane / G;
      for (int d0 = 0; d0 < dk; d0 += 4 * G) {
        const int e = d0 + (lane % G) * 4;
        const bool active = e < dk;
        const int r = active ? e / width : 0;         // four consecutive dims lie in one slice
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        for (int k0 = 0; k0 < nk; k0 += 4 * S) {      // four 16-byte loads in flight per lane
          f32x4 kv[4];
          float sd[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int k = k0 + S * u + sub;
            const bool ok = active && k < nk;
            kv[u] = ok ? *reinterpret_cast<const f32x4*>(Kh + static_cast<size_t>(sh.dist[a][k]) * dk + e)
                       : f32x4{0.f, 0.f, 0.f, 0.f};
            sd[u] = ok ? sh.sd[a][k][r] : 0.0f;
          }
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            if (k0 + S * u >= nk) break;              // wave-uniform: no key for any group
            acc.x = fmaf(sd[u], kv[u].x, acc.x);
            acc.y = fmaf(sd[u], kv[u].y, acc.y);
            acc.z = fmaf(sd[u], kv[u].z, acc.z);
            acc.w = fmaf(sd[u], kv[u].w, acc.w);
          }
        }
        for (int off = G; off < kWave; off <<= 1) {
          acc.x += __shfl_xor(acc.x, off, kWave);
          acc.y += __shfl_xor(acc.y, off, kWave);
          acc.z += __shfl_xor(acc.z, off, kWave);
          acc.w += __shfl_xor(acc.w, off, kWave);
        }
        if (sub == 0 && active) *reinterpret_cast<f32x4*>(dq + e) = acc;
      }
      continue;
    }
    for (int e = lane; e < dk; e += kWave) {
      const int r = e / width;
      float acc = 0.0f;
      int k = 0;
      for (; k + 8 <= nk; k += 8) {     // eight key loads in flight, the sum still in key order
        float kv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) kv[u] = Kh[static_cast<size_t>(sh.dist[a][k + u]) * dk + e];
#pragma unroll
        for (int u = 0; u < 8; ++u) acc = fmaf(sh.sd[a][k + u][r], kv[u], acc);
      }
      for (; k < nk; ++k) acc = fmaf(sh.sd[a][k][r], Kh[static_cast<size_t>(sh.dist[a][k]) * dk + e], acc);
      dq[e] = acc;
    }
  }
  // ---- key-gradient entries: slot ((t H + h) 2 + axis) m + k for the k-th distinct key; the
  // rest of the axis' m slots hold the sentinel
  const uint32_t sentinel = static_cast<uint32_t>(2 * H) * n;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      if (!valid[g]) continue;
      const int s = g * kWave + lane;
      const size_t base = (th * 2 + a) * m;
      if (first[a][g] == s) {
        const size_t slot = base + pos[a][g];
        evals[slot] = static_cast<uint32_t>(slot);
        ekeys[slot] = static_cast<uint32_t>((a * H + h) * n) + key[a][g];
        for (int r = 0; r < rank; ++r) edS[slot * rank + r] = sh.sd[a][pos[a][g]][r];
      }
      if (s >= nd[a]) {
        evals[base + s] = static_cast<uint32_t>(base + s);
        ekeys[base + s] = sentinel;
      }
    }
}

// Key gradients by segments of sorted entries (as the value rows): dK[key] += sum over the
// entries of its run, in order, of dS[entry][slice] q[t, h, :]; pieces cut by a segment store
// their partial row for seg_join_kernel.
__global__ __launch_bounds__(THREADS) void key_bwd_seg_kernel(
    const uint32_t* __restrict__ keys, const uint32_t* __restrict__ slots, int M, uint32_t sentinel,
    const float* __restrict__ edS, const float* __restrict__ q_row, const float* __restrict__ q_col,
    float* __restrict__ dk_row, float* __restrict__ dk_col, int H, int n, int dk, int rank, int m,
    float* __restrict__ partial, const uint32_t* __restrict__ list,
    uint32_t* __restrict__ counts, uint32_t* __restrict__ heads) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t n_pieces = counts[0];
  // The pieces (in (axis, head, key) order) are split into eight contiguous ranges, one per XCD
  // (workgroups go to XCDs round-robin), so that an XCD's waves read the query rows of few
  // (axis, head) blocks and find them in its L2.
  const uint32_t xcd = blockIdx.x & 7u, groups = gridDim.x < 8u ? gridDim.x : 8u;
  const uint32_t lo = static_cast<uint32_t>(static_cast<uint64_t>(n_pieces) * xcd / groups);
  const uint32_t hi = static_cast<uint32_t>(static_cast<uint64_t>(n_pieces) * (xcd + 1) / groups);
  const uint32_t xcd_waves = ((gridDim.x - xcd + 7u) >> 3) * NWAVES;   // this XCD's waves
  for (uint32_t pk = lo + (blockIdx.x >> 3) * NWAVES + threadIdx.x / kWave; pk < hi;
       pk += xcd_waves) {
  const int ps = static_cast<int>(list[pk]);
  const uint32_t key = keys[ps];                     // never the sentinel: not listed
  int pe;
  bool run_start, run_end;
  piece_at(keys, ps, M, key, &pe, &run_start, &run_end);
  if (run_start && !run_end && lane == 0)
    heads[atomicAdd(counts + 1, 1u)] = static_cast<uint32_t>(ps);
  const int g = ps / kSeg;
  const int axis = static_cast<int>(key / (static_cast<uint32_t>(H) * n));
  const int rem = static_cast<int>(key - static_cast<uint32_t>(axis) * H * n);
  const int h = rem / n;
  const float* q = axis ? q_col : q_row;
  float* dK = (axis ? dk_col : dk_row) + static_cast<size_t>(rem) * dk;
  const int width = dk / rank;
  const int n_e = pe - ps;
  const uint32_t my_slot = lane < n_e ? slots[ps + lane] : 0u;   // one entry per lane
  const bool whole = run_start && run_end;
  float* const part_row = partial + (static_cast<size_t>(2) * g + (run_start ? 1 : 0)) * dk;
  if (dk <= 2 * kWave && (dk & (dk - 1)) == 0) {
    // Rows of at most 128 dims fill a fraction of the wave: G = dk / 4 lanes take one entry, and
    // the wave's S = 64 / G lane groups take entries s, s + S, s + 2 S, ... of the piece, each
    // group in order; the groups' sums then meet by a fixed butterfly of shuffles.
    const int G = dk / 4, S = kWave / G;
    const int sub = lane / G, d = (lane % G) * 4;
    const int r = d / width;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    const f32x4 old = (whole && sub == 0) ? *reinterpret_cast<const f32x4*>(dK + d) : f32x4{0.f, 0.f, 0.f, 0.f};
    for (int j0 = 0; j0 < n_e; j0 += S * kInFlight) {   // wave-uniform
      f32x4 qv[kInFlight];
      float ds[kInFlight];
#pragma unroll
      for (int u = 0; u < kInFlight; ++u) {              // all loads first
        const int j = j0 + S * u + sub;
        const size_t slot = static_cast<uint32_t>(__shfl(static_cast<int>(my_slot), min(j, n_e - 1), kWave));
        const size_t t = slot / (static_cast<size_t>(2) * H * m);
        qv[u] = f32x4{0.f, 0.f, 0.f, 0.f};
        ds[u] = 0.0f;
        if (j < n_e) {
          qv[u] = *reinterpret_cast<const f32x4*>(q + (t * H + h) * dk + d);
          ds[u] = edS[slot * rank + r];
        }
      }
#pragma unroll
      for (int u = 0; u < kInFlight; ++u) {              // then this group's entries in order
        acc.x = fmaf(ds[u], qv[u].x, acc.x);
        acc.y = fmaf(ds[u], qv[u].y, acc.y);
        acc.z = fmaf(ds[u], qv[u].z, acc.z);
        acc.w = fmaf(ds[u], qv[u].w, acc.w);
      }
    }
    for (int off = G; off < kWave; off <<= 1) {
      acc.x += __shfl_xor(acc.x, off, kWave);
      acc.y += __shfl_xor(acc.y, off, kWave);
      acc.z += __shfl_xor(acc.z, off, kWave);
      acc.w += __shfl_xor(acc.w, off, kWave);
    }
    if (sub == 0) {
      if (whole) *reinterpret_cast<f32x4*>(dK + d) = old + acc;
      else *reinterpret_cast<f32x4*>(part_row + d) = acc;
    }
    continue;
  }
  for (int d0 = 0; d0 < dk; d0 += kWave * 4) {
    const int d = d0 + lane * 4;
    const bool active = d < dk;
    const int r = active ? d / width : 0;             // four consecutive dims lie in one slice
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    // a whole run adds into its key's gradient row: read it now, under the entries' loads
    const f32x4 old = (active && whole) ? *reinterpret_cast<const f32x4*>(dK + d) : f32x4{0.f, 0.f, 0.f, 0.f};
    for (int j0 = 0; j0 < n_e; j0 += 2 * kInFlight) {  // wave-uniform
      f32x4 qv[2 * kInFlight];
      float ds[2 * kInFlight];
#pragma unroll
      for (int u = 0; u < 2 * kInFlight; ++u) {      // all loads first
        const size_t slot = static_cast<uint32_t>(
            __builtin_amdgcn_readlane(static_cast<int>(my_slot), min(j0 + u, n_e - 1)));
        const size_t t = slot / (static_cast<size_t>(2) * H * m);
        qv[u] = f32x4{0.f, 0.f, 0.f, 0.f};
        ds[u] = 0.0f;
        if (active && j0 + u < n_e) {                 // (past the piece's end: no loads)
          qv[u] = *reinterpret_cast<const f32x4*>(q + (t * H + h) * dk + d);
          ds[u] = edS[slot * rank + r];
        }
      }
#pragma unroll
      for (int u = 0; u < 2 * kInFlight; ++u) {      // then the entries in order
        if (j0 + u >= n_e) break;
        acc.x = fmaf(ds[u], qv[u].x, acc.x);
        acc.y = fmaf(ds[u], qv[u].y, acc.y);
        acc.z = fmaf(ds[u], qv[u].z, acc.z);
        acc.w = fmaf(ds[u], qv[u].w, acc.w);
      }
    }
    if (!active) continue;
    if (whole) *reinterpret_cast<f32x4*>(dK + d) = old + acc;
    else *reinterpret_cast<f32x4*>(part_row + d) = acc;
  }
  }
}

// out[c] += sum over the R rows of in[.][c]: one workgroup per column, thread i adding rows i,
// i + 256, ... in order, then a fixed tree over the threads.
__global__ __launch_bounds__(THREADS) void sum_cols_kernel(const float* __restrict__ in,
                                                           float* __restrict__ out, int R, int C) {
  __shared__ float red[THREADS];
  const int c = blockIdx.x, tid = threadIdx.x;
  float a = 0.0f;
  for (int j = tid; j < R; j += THREADS) a += in[static_cast<size_t>(j) * C + c];
  red[tid] = a;
  __syncthreads();
  for (int off = THREADS / 2; off > 0; off >>= 1) {
    if (tid < off) red[tid] += red[tid + off];
    __syncthreads();
  }
  if (tid == 0) out[c] += red[0];
}

size_t round_up256(size_t x) { return (x + 255) / 256 * 256; }

int bits_for(int64_t n) {
  int b = 0;
  while (b < 31 && (INT64_C(1) << b) < n) ++b;
  return b;
}

}  // namespace

size_t gather_backward_workspace_bytes(int T, int bag, int dv) {
  const int M = T * bag;
  if (M == 0) return 0;
  const size_t nseg = (static_cast<size_t>(M) + kSeg - 1) / kSeg;
  return 4 * round_up256(static_cast<size_t>(M) * sizeof(uint32_t)) + round_up256(nseg * sizeof(uint32_t)) +
         256 + round_up256(2 * nseg * dv * sizeof(float)) + round_up256(sort_workspace_bytes(M)) +
         round_up256(list_workspace_bytes(M));
}

// rows_out == nullptr: d_values is the dense [n_values, dv] gradient, added into.  Otherwise the
// compact form: d_values is [T * bag, dv], row r the gradient of rows_out[r], the r-th distinct
// row (ascending), and *n_rows the number of distinct rows.
hipError_t launch_gather_backward(int64_t n_values, int dv, int vdtype, const void* values, int T,
                                  int bag, const int32_t* idx, const float* w, const int32_t* perm,
                                  int expand, int cores, const float* d_pooled, float* d_values,
                                  float* dw, int32_t* rows_out, int32_t* n_rows, void* ws,
                                  hipStream_t s) {
  clear_stale_error();
  const int M = T * bag;
  if (M == 0) return hipSuccess;
  char* base = static_cast<char*>(ws);
  uint32_t* keys = reinterpret_cast<uint32_t*>(base);
  uint32_t* vals = reinterpret_cast<uint32_t*>(base + round_up256(static_cast<size_t>(M) * sizeof(uint32_t)));
  const size_t nseg = (static_cast<size_t>(M) + kSeg - 1) / kSeg;
  char* p0 = base + 2 * round_up256(static_cast<size_t>(M) * sizeof(uint32_t));
  uint32_t* list = reinterpret_cast<uint32_t*>(p0);
  p0 += round_up256(static_cast<size_t>(M) * sizeof(uint32_t));
  uint32_t* heads = reinterpret_cast<uint32_t*>(p0);
  p0 += round_up256(nseg * sizeof(uint32_t));
  uint32_t* counts = reinterpret_cast<uint32_t*>(p0);
  p0 += 256;
  float* partial = reinterpret_cast<float*>(p0);
  void* sws = p0 + round_up256(2 * nseg * dv * sizeof(float));
  void* lws = static_cast<char*>(sws) + round_up256(sort_workspace_bytes(M));
  uint32_t* run_of = reinterpret_cast<uint32_t*>(static_cast<char*>(lws) + round_up256(list_workspace_bytes(M)));
  const unsigned kb = static_cast<unsigned>(std::min((M + THREADS - 1) / THREADS, 4096));
  hipLaunchKernelGGL(bwd_keys_kernel, dim3(kb), dim3(THREADS), 0, s, idx,
                     expand > 1 ? perm : nullptr, n_values, M, keys, vals);
  uint32_t *rows_sorted, *ents_sorted;
  hipError_t e = sort_pairs(keys, vals, M, bits_for(n_values), sws, s, &rows_sorted, &ents_sorted);
  if (e != hipSuccess) return e;
  const int c = cores > 1 ? cores : 1;
  const dim3 list_grid(kValueListWaves / NWAVES);
  // row indices are below 2^31: the sentinel never occurs
  const bool compact = rows_out != nullptr;
  e = list_pieces(rows_sorted, M, 0xFFFFFFFFu, list, counts, lws, s, compact ? run_of : nullptr,
                  rows_out, n_rows);
  if (e != hipSuccess) return e;
  const uint32_t* ro = compact ? run_of : nullptr;
  if (vdtype == UMEM_F32)
    hipLaunchKernelGGL(gather_bwd_seg_kernel<float>, list_grid, dim3(THREADS), 0, s, rows_sorted,
                       ents_sorted, M, static_cast<const float*>(values), dv, idx, w,
                       expand > 1 ? perm : nullptr, n_values, expand, c, bag, d_pooled, d_values, dw,
                       partial, list, counts, heads, ro);
  else
    hipLaunchKernelGGL(gather_bwd_seg_kernel<uint16_t>, list_grid, dim3(THREADS), 0, s, rows_sorted,
                       ents_sorted, M, static_cast<const uint16_t*>(values), dv, idx, w,
                       expand > 1 ? perm : nullptr, n_values, expand, c, bag, d_pooled, d_values, dw,
                       partial, list, counts, heads, ro);
  hipLaunchKernelGGL(seg_join_kernel, list_grid, dim3(THREADS), 0, s, rows_sorted, M, dv, partial,
                     d_values, heads, counts, 0, 0, nullptr, ro);
  return hipGetLastError();
}

size_t score_backward_workspace_bytes(const umem_desc& d, int T) {
  if (T == 0) return 0;
  const size_t th = static_cast<size_t>(T) * d.heads;
  const int Mk = static_cast<int>(th * 2 * d.topm);
  const int hc = d.cores > 1 ? d.cores : 1;
  const size_t dc = d.grid == UMEM_GRID_TUCKER ? static_cast<size_t>(hc) * d.rank * d.rank : 0;
  const size_t nseg = (static_cast<size_t>(Mk) + kSeg - 1) / kSeg;
  return 3 * round_up256(static_cast<size_t>(Mk) * sizeof(uint32_t)) + round_up256(nseg * sizeof(uint32_t)) +
         256 + round_up256(static_cast<size_t>(Mk) * d.rank * sizeof(float)) +
         round_up256(2 * nseg * d.dk * sizeof(float)) + round_up256(list_workspace_bytes(Mk)) +
         round_up256(th * dc * sizeof(float)) + round_up256(sort_workspace_bytes(Mk));
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
  const size_t nseg = (static_cast<size_t>(Mk) + kSeg - 1) / kSeg;
  float* kpart = reinterpret_cast<float*>(base);
  base += round_up256(2 * nseg * d.dk * sizeof(float));
  uint32_t* list = reinterpret_cast<uint32_t*>(base);
  base += round_up256(static_cast<size_t>(Mk) * sizeof(uint32_t));
  uint32_t* heads = reinterpret_cast<uint32_t*>(base);
  base += round_up256(nseg * sizeof(uint32_t));
  uint32_t* counts = reinterpret_cast<uint32_t*>(base);
  base += 256;
  void* lws = base;
  base += round_up256(list_workspace_bytes(Mk));
  float* dc_part = reinterpret_cast<float*>(base);
  base += round_up256(th * dc * sizeof(float));
  void* sws = base;
  const int key_bits = bits_for(d.n_keys);
  const int sm = d.weight == UMEM_W_SOFTMAX ? 1 : 0;
#define UMEM_SCORE_BWD(NG)                                                                       \
  hipLaunchKernelGGL(score_bwd_kernel<NG>,                                                      \
                     dim3(static_cast<unsigned>((th + score_bwd_waves<NG>() - 1) / score_bwd_waves<NG>())), \
                     dim3(score_bwd_waves<NG>() * kWave), 0, s, q_row, q_col, k_row, k_col, core, \
                     idx, w, dw, T, H, d.n_keys, key_bits, d.dk, r, m, tucker ? 1 : 0, sm, hc,   \
                     dq_row, dq_col, ekeys, evals, edS, dc_part)
  if (m <= kWave) UMEM_SCORE_BWD(1);
  else if (m <= 2 * kWave) UMEM_SCORE_BWD(2);
  else UMEM_SCORE_BWD(4);
#undef UMEM_SCORE_BWD
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const uint32_t sentinel = static_cast<uint32_t>(2 * H) * d.n_keys;
  uint32_t *ks, *vs;
  e = sort_pairs(ekeys, evals, Mk, bits_for(static_cast<int64_t>(sentinel) + 1), sws, s, &ks, &vs);
  if (e != hipSuccess) return e;
  const dim3 list_grid(kListWaves / NWAVES);
  e = list_pieces(ks, Mk, sentinel, list, counts, lws, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(key_bwd_seg_kernel, list_grid, dim3(THREADS), 0, s, ks, vs, Mk, sentinel, edS,
                     q_row, q_col, dk_row, dk_col, H, d.n_keys, d.dk, r, m, kpart, list, counts, heads);
  hipLaunchKernelGGL(seg_join_kernel, list_grid, dim3(THREADS), 0, s, ks, Mk, d.dk, kpart, dk_row,
                     heads, counts, H, d.n_keys, dk_col, nullptr);
  if (tucker)   // dC: the per-token partials [T][H dc], summed over tokens into dcore
    hipLaunchKernelGGL(sum_cols_kernel, dim3(H * dc), dim3(THREADS), 0, s, dc_part, dcore, T, H * dc);
  return hipGetLastError();
}

}  // namespace umem
