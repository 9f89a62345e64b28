// a6 + a7: score-weighted gather-sum of value rows (embedding bag), eq. (1) and eq. (15).
//
// One workgroup of four waves per token; each wave pools a contiguous quarter of the bag.  A
// value row is read with 16-byte loads, L lanes per row and CPL 16-byte chunks per lane (row
// bytes = 16 * L * CPL); a wave keeps U rows in flight.  The loads are nontemporal unless the
// launch reads at least a quarter as many rows as the table holds: then rows repeat (more than
// one read in nine even if slots were drawn uniformly, far more with clustered queries) and are
// worth keeping in L2 and the MALL.  Accumulation is fp32 in registers; the sub-rows of a wave
// are combined with shuffles, and the four waves' partial rows in LDS behind one barrier, always
// in wave order (the result does not depend on timing).  Pooled rows are written with plain
// stores: with implicit value expansion the projection reads them next and finds them cached.
// With implicit value expansion the bag is first mapped through the shuffle and split by
// virtual block p (a stable partition), and each block's rows are pooled into out[t, p, :]; with
// a multiple of four blocks each wave pools whole blocks, first entry to last, so the blocks
// stream side by side with no barrier between them.  From 2048 tokens on (without expansion) a
// wave per token does the same work without LDS or barriers.  Pooled rows leave as fp32, or, for
// the forward's projection, rounded to bf16 (nearest even) by the same instruction with which
// the projection GEMM rounds its A operand while staging it: the GEMM then reads half the bytes
// and computes exactly what it computed from the fp32 rows.
#include "umem_internal.h"

namespace umem {
namespace {

constexpr int THREADS = 256;
constexpr int NWAVES = THREADS / kWave;
constexpr int kWaveTokensMin = 2048;   // from here on, a wave per token
constexpr int kWaveBatch = 8;          // 16-byte loads per lane per batch of the wave-per-token form

// Partial rows the waves of one token combine in LDS: none when each wave pools whole virtual
// blocks (expand a multiple of the wave count); else one per wave, or two for rows over 2048
// elements (waves 2, 3 are folded into 0, 1 first).
__host__ __device__ constexpr int reduce_rows(int dv, int expand) {
  return expand > 1 && expand % NWAVES == 0 ? 0 : (dv <= 2048 ? NWAVES : 2);
}
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Four pooled values stored as fp32, or as bf16 bits (one v_cvt_pk_bf16_f32 per pair).
template <bool NT>
__device__ __forceinline__ void put4(float* dst, f32x4 v) {
  if constexpr (NT) __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(dst));
  else *reinterpret_cast<f32x4*>(dst) = v;
}
template <bool NT>
__device__ __forceinline__ void put4(uint16_t* dst, f32x4 v) {
  const u32x2 p{__builtin_bit_cast(uint32_t, bf16x2{static_cast<__bf16>(v.x), static_cast<__bf16>(v.y)}),
                __builtin_bit_cast(uint32_t, bf16x2{static_cast<__bf16>(v.z), static_cast<__bf16>(v.w)})};
  if constexpr (NT) __builtin_nontemporal_store(p, reinterpret_cast<u32x2*>(dst));
  else *reinterpret_cast<u32x2*>(dst) = p;
}

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

// One wave's weighted sum of entries [wbeg, wend) into acc: sub-group `sub` of the wave (L
// lanes) reads entries wbeg + SUB * i + sub in order, and the sub-rows are added by shuffles at
// the end.  `slot(j)` gives entry j's position in idx / w (after the block partition, if any).
// With multi-core scoring (cores > 1) entry s has cores weights, w_of[s * cores + i], and a
// lane's 16-byte chunk takes the weight of the column slice it lies in.
template <typename Elem, int L, int CPL, bool KEEP, typename Slot>
__device__ __forceinline__ void wave_rows(const Elem* __restrict__ values, int dv, int wbeg, int wend,
                                          const Slot& slot, const int32_t* __restrict__ rows_of,
                                          const float* __restrict__ w_of, int cores,
                                          float (&acc)[CPL][ElemTraits<Elem>::kPerChunk]) {
  using TR = ElemTraits<Elem>;
  constexpr int EPC = TR::kPerChunk;
  constexpr int SUB = kWave / L;                   // rows a wave reads at once
  constexpr int U = (CPL >= 16) ? 1 : 16 / CPL;    // row batches in flight per wave
  const int lane = threadIdx.x & (kWave - 1);
  const int sub = lane / L;
  const int cl = lane % L;
  int slice[CPL];                                  // this lane's chunks' core (0 with one core)
#pragma unroll
  for (int c = 0; c < CPL; ++c) slice[c] = cores > 1 ? ((cl + L * c) * EPC) / (dv / cores) : 0;

#pragma unroll
  for (int c = 0; c < CPL; ++c)
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[c][e] = 0.0f;
  for (int j0 = wbeg; j0 < wend; j0 += SUB * U) {
    u32x4 raw[U][CPL];
    float wt[U][CPL];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + SUB * u + sub;
      if (j < wend) {
        const int s = slot(j);
        const Elem* src = values + static_cast<int64_t>(rows_of[s]) * dv;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          wt[u][c] = w_of[static_cast<size_t>(s) * cores + slice[c]];
          const u32x4* p = reinterpret_cast<const u32x4*>(src + (cl + L * c) * EPC);
          // (a compile-time choice: a run-time select of the two loads is merged into a plain one)
          if constexpr (KEEP) raw[u][c] = *p;
          else raw[u][c] = __builtin_nontemporal_load(p);
        }
      } else {
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          wt[u][c] = 0.0f;
          raw[u][c] = u32x4{0u, 0u, 0u, 0u};
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int c = 0; c < CPL; ++c) {
        float x[EPC];
        TR::widen(raw[u][c], x);
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[c][e] = fmaf(wt[u][c], x[e], acc[c][e]);
      }
  }
  // combine the SUB sub-rows of this wave (lanes cl, cl + L, ...) with shuffles
#pragma unroll
  for (int off = L; off < kWave; off <<= 1)
#pragma unroll
    for (int c = 0; c < CPL; ++c)
#pragma unroll
      for (int e = 0; e < EPC; ++e) acc[c][e] += __shfl_xor(acc[c][e], off, kWave);
}

// Rows of one bag (or of one virtual block of it) split into NWAVES contiguous ranges, one per
// wave, and the waves' sums combined into one pooled row.
template <typename Elem, int L, int CPL, bool KEEP, typename Out, typename Slot>
__device__ __forceinline__ void pool_rows(const Elem* __restrict__ values, int dv, int cnt,
                                          const Slot& slot, const int32_t* __restrict__ rows_of,
                                          const float* __restrict__ w_of, int cores, float* red,
                                          Out* __restrict__ dst) {
  constexpr int EPC = ElemTraits<Elem>::kPerChunk;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int sub = lane / L;
  const int cl = lane % L;
  const int per_wave = (cnt + NWAVES - 1) / NWAVES;
  const int wbeg = wave * per_wave;
  const int wend = min(cnt, wbeg + per_wave);
  float acc[CPL][EPC];
  wave_rows<Elem, L, CPL, KEEP>(values, dv, wbeg, wend, slot, rows_of, w_of, cores, acc);
  // The waves' partial rows meet in LDS and every thread adds, in wave order, the partials of
  // its columns, then stores them.  Rows of up to 2048 elements use NWAVES partial rows; longer
  // rows (up to 4096) first fold waves 2, 3 into 0, 1, within half the space.
  const bool one_stage = dv <= 2048;
  if (sub == 0 && (one_stage || wave >= 2)) {
    float* r = red + (one_stage ? wave : wave - 2) * dv;
#pragma unroll
    for (int c = 0; c < CPL; ++c)
#pragma unroll
      for (int e = 0; e < EPC; e += 4)
        *reinterpret_cast<float4*>(r + (cl + L * c) * EPC + e) =
            make_float4(acc[c][e], acc[c][e + 1], acc[c][e + 2], acc[c][e + 3]);
  }
  __syncthreads();
  if (!one_stage) {
    if (sub == 0 && wave < 2) {
      float* r = red + wave * dv;
#pragma unroll
      for (int c = 0; c < CPL; ++c)
#pragma unroll
        for (int e = 0; e < EPC; e += 4) {
          float4* q = reinterpret_cast<float4*>(r + (cl + L * c) * EPC + e);
          const float4 x = *q;
          *q = make_float4(acc[c][e] + x.x, acc[c][e + 1] + x.y, acc[c][e + 2] + x.z, acc[c][e + 3] + x.w);
        }
    }
    __syncthreads();
  }
  const int parts = one_stage ? NWAVES : 2;
  for (int col = tid * 4; col < dv; col += THREADS * 4) {
    float4 r = *reinterpret_cast<const float4*>(red + col);
    for (int v = 1; v < parts; ++v) {
      const float4 x = *reinterpret_cast<const float4*>(red + v * dv + col);
      r.x += x.x;
      r.y += x.y;
      r.z += x.z;
      r.w += x.w;
    }
    // plain stores: the projection that follows reads the pooled rows from cache
    put4<false>(dst + col, f32x4{r.x, r.y, r.z, r.w});
  }
}

// Without expansion the bag is read straight from idx / w (for rows of 64 lanes a wave's row
// index is uniform and lives in scalar registers).  With expansion the bag is first mapped
// through perm and stably partitioned by virtual block in LDS.
template <typename Elem, int L, int CPL, bool KEEP, typename Out>
__global__ __launch_bounds__(THREADS) void gather_kernel(
    const Elem* __restrict__ values, int64_t n_values, int dv, int bag,
    const int32_t* __restrict__ idx, const float* __restrict__ w, const int32_t* __restrict__ perm,
    int expand, int cores, Out* __restrict__ out) {
  extern __shared__ __align__(16) float red[];               // [red_rows][dv], then the bag
  const int t = blockIdx.x;
  const int32_t* __restrict__ idx_t = idx + static_cast<size_t>(t) * bag;
  const float* __restrict__ w_t = w + static_cast<size_t>(t) * bag * cores;
  if (expand == 1) {
    pool_rows<Elem, L, CPL, KEEP, Out>(values, dv, bag, [](int j) { return j; }, idx_t, w_t, cores,
                                       red, out + static_cast<size_t>(t) * dv);
    return;
  }
  int32_t* rows = reinterpret_cast<int32_t*>(red + reduce_rows(dv, expand) * dv);   // [bag]
  int32_t* blk = rows + bag;                                       // [bag]
  int32_t* order = blk + bag;                                      // [bag]
  __shared__ int bstart[kMaxExpand + 1], bcount[kMaxExpand];
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  for (int s = tid; s < bag; s += THREADS) {
    const int64_t v = static_cast<int64_t>(perm[idx_t[s]]);
    const int p = static_cast<int>(v / n_values);
    rows[s] = static_cast<int32_t>(v - static_cast<int64_t>(p) * n_values);
    blk[s] = p;
  }
  __syncthreads();
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
  __syncthreads();
  if (expand % NWAVES == 0) {
    // a whole block per wave: the blocks stream side by side, with no barrier between them, and
    // each pooled row leaves from its wave's registers
    using TR = ElemTraits<Elem>;
    constexpr int EPC = TR::kPerChunk;
    const int w0 = __builtin_amdgcn_readfirstlane(wave);
    const int cl = lane % L;
    for (int p = w0; p < expand; p += NWAVES) {
      const int beg = __builtin_amdgcn_readfirstlane(bstart[p]);
      const int cnt = __builtin_amdgcn_readfirstlane(bcount[p]);
      float acc[CPL][EPC];
      wave_rows<Elem, L, CPL, KEEP>(values, dv, 0, cnt, [=](int j) { return order[beg + j]; },
                                    rows, w_t, cores, acc);
      if (lane < L) {
        Out* dst = out + (static_cast<size_t>(t) * expand + p) * dv;
#pragma unroll
        for (int c = 0; c < CPL; ++c)
#pragma unroll
          for (int e = 0; e < EPC; e += 4)
            put4<false>(dst + (cl + L * c) * EPC + e, f32x4{acc[c][e], acc[c][e + 1], acc[c][e + 2], acc[c][e + 3]});
      }
    }
    return;
  }
  for (int p = 0; p < expand; ++p) {
    const int beg = bstart[p];
    pool_rows<Elem, L, CPL, KEEP, Out>(values, dv, bcount[p], [=](int j) { return order[beg + j]; },
                                       rows, w_t, cores, red,
                                       out + (static_cast<size_t>(t) * expand + p) * dv);
    __syncthreads();
  }
}

// Many tokens without expansion: one wave per token, which reads the token's whole bag itself
// and needs no LDS and no barrier.  The bag's indices and weights are loaded 64 at a time, one
// per lane, and each row's index taken from its lane (readlane; a shuffle for sub-rows).  The
// rows are read in batches of kWaveBatch 16-byte loads per lane, each batch issued whole and then
// accumulated.  Single batches keep the kernel at 59 VGPRs, eight waves per SIMD: with thousands
// of tokens the CUs then hold many such waves at once, and that, not a second batch in flight
// per wave (double buffering: 103 VGPRs, four waves), keeps the most rows in flight (measured:
// 8,192 decode tokens 93.9 -> 92.7 us; prefill-1M's 2,048 tokens of 2 KiB rows 46.9 -> 46.0 us).
template <typename Elem, int L, int CPL, typename Out>
__global__ __launch_bounds__(THREADS) void gather_wave_kernel(
    const Elem* __restrict__ values, int dv, int T, int bag, const int32_t* __restrict__ idx,
    const float* __restrict__ w, Out* __restrict__ out) {
  using TR = ElemTraits<Elem>;
  constexpr int EPC = TR::kPerChunk;
  constexpr int SUB = kWave / L;
  constexpr int U = (CPL >= kWaveBatch) ? 1 : kWaveBatch / CPL;   // row steps per batch
  constexpr int BATCH = SUB * U;                       // rows per batch (divides 64)
  const int lane = threadIdx.x & (kWave - 1);
  const int t = blockIdx.x * NWAVES + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if (t >= T) return;
  const int sub = lane / L;
  const int cl = lane % L;
  const int32_t* __restrict__ idx_t = idx + static_cast<size_t>(t) * bag;
  const float* __restrict__ w_t = w + static_cast<size_t>(t) * bag;
  float acc[CPL][EPC];
#pragma unroll
  for (int c = 0; c < CPL; ++c)
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[c][e] = 0.0f;

  u32x4 buf[U][CPL];
  float wt[U];
  for (int base = 0; base < bag; base += kWave) {
    const int n_here = min(kWave, bag - base);           // entries of this chunk
    const int my_row = lane < n_here ? idx_t[base + lane] : 0;
    const float my_w = lane < n_here ? w_t[base + lane] : 0.0f;
    const int nb = (n_here + BATCH - 1) / BATCH;
    // rows of batch b: chunk entries b * BATCH + SUB * u + sub
    auto issue = [&](int b, u32x4 (&bb)[U][CPL], float (&ww)[U]) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int jl = b * BATCH + SUB * u;               // uniform part of the entry
        int row;
        float wj;
        if (SUB == 1) {
          row = __builtin_amdgcn_readlane(my_row, jl);
          wj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(my_w), jl));
        } else {
          row = __shfl(my_row, jl + sub, kWave);
          wj = __shfl(my_w, jl + sub, kWave);
        }
        const bool ok = jl + sub < n_here;
        ww[u] = ok ? wj : 0.0f;
        const Elem* src = values + static_cast<int64_t>(ok ? row : 0) * dv;
#pragma unroll
        for (int c = 0; c < CPL; ++c)
          bb[u][c] = ok ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + (cl + L * c) * EPC))
                        : u32x4{0u, 0u, 0u, 0u};
      }
    };
    auto consume = [&](const u32x4 (&bb)[U][CPL], const float (&ww)[U]) {
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
          float x[EPC];
          TR::widen(bb[u][c], x);
#pragma unroll
          for (int e = 0; e < EPC; ++e) acc[c][e] = fmaf(ww[u], x[e], acc[c][e]);
        }
    };
    for (int b = 0; b < nb; ++b) {
      issue(b, buf, wt);
      consume(buf, wt);
    }
  }
#pragma unroll
  for (int off = L; off < kWave; off <<= 1)
#pragma unroll
    for (int c = 0; c < CPL; ++c)
#pragma unroll
      for (int e = 0; e < EPC; ++e) acc[c][e] += __shfl_xor(acc[c][e], off, kWave);
  if (sub == 0) {
    Out* dst = out + static_cast<size_t>(t) * dv;
#pragma unroll
    for (int c = 0; c < CPL; ++c)
#pragma unroll
      for (int e = 0; e < EPC; e += 4)
        put4<true>(dst + (cl + L * c) * EPC + e, f32x4{acc[c][e], acc[c][e + 1], acc[c][e + 2], acc[c][e + 3]});
  }
}

template <typename Elem, typename Out>
hipError_t launch_typed(const Elem* values, int64_t n_values, int dv, int T, int bag,
                        const int32_t* idx, const float* w, const int32_t* perm, int expand,
                        int cores, Out* out, hipStream_t s) {
  const int chunks = dv * static_cast<int>(sizeof(Elem)) / 16;
  const size_t lds = static_cast<size_t>(reduce_rows(dv, expand)) * dv * 4 +
                    (expand > 1 ? static_cast<size_t>(bag) * 12 : 0);
  const dim3 block(THREADS);
  // thousands of tokens without expansion (or multi-core weights): a wave per token
  const bool per_wave = expand == 1 && cores == 1 && T >= kWaveTokensMin;
  const dim3 grid(per_wave ? (T + NWAVES - 1) / NWAVES : T);
  // temporal row loads when rows will repeat: T * bag row reads against n_values rows
  const bool keep = 4 * static_cast<int64_t>(T) * bag >= n_values;
#define UMEM_GATHER(LL, CC)                                                                      \
  if (per_wave)                                                                                  \
    hipLaunchKernelGGL((gather_wave_kernel<Elem, LL, CC, Out>), grid, block, 0, s, values, dv, T, \
                       bag, idx, w, out);                                                        \
  else if (keep)                                                                                 \
    hipLaunchKernelGGL((gather_kernel<Elem, LL, CC, true, Out>), grid, block, lds, s, values,      \
                       n_values, dv, bag, idx, w, perm, expand, cores, out);                     \
  else                                                                                           \
    hipLaunchKernelGGL((gather_kernel<Elem, LL, CC, false, Out>), grid, block, lds, s, values,     \
                       n_values, dv, bag, idx, w, perm, expand, cores, out)
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

template <typename Out>
hipError_t launch_any(int64_t n_values, int dv, int vdtype, const void* values, int T, int bag,
                      const int32_t* idx, const float* w, const int32_t* perm, int expand,
                      int cores, Out* out, hipStream_t s) {
  clear_stale_error();
  if (T == 0) return hipSuccess;
  if (vdtype == UMEM_F32)
    return launch_typed(static_cast<const float*>(values), n_values, dv, T, bag, idx, w, perm,
                        expand, cores, out, s);
  return launch_typed(static_cast<const uint16_t*>(values), n_values, dv, T, bag, idx, w, perm,
                      expand, cores, out, s);
}

}  // namespace

bool gather_row_supported(int dv, int vdtype) {
  const int bytes = dv * (vdtype == UMEM_F32 ? 4 : 2);
  if (bytes % 16 != 0 || bytes > kMaxRowBytes) return false;
  const int chunks = bytes / 16;
  if (chunks <= 64) return (chunks & (chunks - 1)) == 0;
  return chunks % 64 == 0;
}

bool cores_supported(int dv, int vdtype, int cores) {
  if (cores < 1 || cores > kMaxCores || dv % cores != 0) return false;
  return (dv / cores) * (vdtype == UMEM_F32 ? 4 : 2) % 16 == 0;   // whole 16-byte chunks
}

hipError_t launch_gather(int64_t n_values, int dv, int vdtype, const void* values, int T,
                         int bag, const int32_t* idx, const float* w, const int32_t* perm,
                         int expand, int cores, float* out, hipStream_t s) {
  return launch_any(n_values, dv, vdtype, values, T, bag, idx, w, perm, expand, cores, out, s);
}

hipError_t launch_gather_bf16(int64_t n_values, int dv, int vdtype, const void* values, int T,
                              int bag, const int32_t* idx, const float* w, const int32_t* perm,
                              int expand, int cores, uint16_t* out, hipStream_t s) {
  return launch_any(n_values, dv, vdtype, values, T, bag, idx, w, perm, expand, cores, out, s);
}

}  // namespace umem
