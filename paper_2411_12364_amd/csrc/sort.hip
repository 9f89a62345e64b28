// Stable sort of (key, value) pairs of 32-bit unsigned keys: least-significant-digit radix sort
// in as few passes of at most 11-bit digits as the key width needs (ceil(bits / 11) passes of
// ceil(bits / passes) bits: 20-bit row keys in two passes of 10).  The backward passes use it to
// bring all contributions to one value row (or key row) together, in their original order, so
// that one wave sums them in a fixed order and the gradient does not depend on timing.
//
// Per pass, over tiles of 4096 pairs (256 threads x 16 steps), with 2^D digit values:
//  * sort_hist_kernel: the tile's digit histogram (LDS atomics), stored digit-major
//    [2^D][tiles];
//  * scan_exclusive turns the 2^D * tiles counts into exclusive offsets (digit by digit, tile by
//    tile: the order the stable pass writes in): chunk sums, then each chunk rescanned from the
//    sum of the chunks before it;
//  * sort_scatter_kernel: the tile again (all of its pairs loaded up front), 256 consecutive
//    pairs per step; a pair's place is its digit's running offset in this tile + the count of
//    equal digits in earlier waves of this step + its rank among equal digits in its own wave
//    (D ballots match the digit).  Each wave's first pair of a digit posts the wave's count of
//    it, and after the step adds it to the digit's running offset and clears its post, so a step
//    costs the same whatever 2^D is.
#include <utility>

#include "umem_internal.h"

namespace umem {
namespace {

constexpr int kThreads = 256;
constexpr int kSteps = 16;
constexpr int kTile = kThreads * kSteps;
constexpr int kWaves = kThreads / kWave;
constexpr int kMaxDigitBits = 11;
constexpr int kMaxDigits = 1 << kMaxDigitBits;

__device__ __forceinline__ uint64_t lanes_below() {
  const unsigned lane = threadIdx.x & (kWave - 1);
  return lane == 0 ? 0ull : (~0ull >> (kWave - lane));
}

__global__ __launch_bounds__(kThreads) void sort_hist_kernel(const uint32_t* __restrict__ keys,
                                                             int M, int shift, int dbits,
                                                             uint32_t* __restrict__ hist,
                                                             int tiles) {
  __shared__ uint32_t cnt[kMaxDigits];
  const int nd = 1 << dbits;
  const uint32_t mask = static_cast<uint32_t>(nd - 1);
  for (int d = threadIdx.x; d < nd; d += kThreads) cnt[d] = 0;
  __syncthreads();
  const int base = blockIdx.x * kTile;
  for (int q = 0; q < kSteps; ++q) {
    const int pos = base + q * kThreads + threadIdx.x;
    if (pos < M) atomicAdd(&cnt[(keys[pos] >> shift) & mask], 1u);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < nd; d += kThreads)
    hist[static_cast<size_t>(d) * tiles + blockIdx.x] = cnt[d];
}

// ---------------------------------------------------------------- exclusive scan
// Over chunks of kScanChunk counts: each chunk's sum (scan_sums_kernel, skipped for one chunk),
// then each chunk rescanned from the sum of the chunk sums before it (scan_apply_kernel).  Thread
// t of a chunk owns its 16 consecutive counts.  Integer sums: exact in any order.

constexpr int kScanPer = 16;
constexpr int kScanChunk = kThreads * kScanPer;

// Exclusive prefix of v over the workgroup's threads (every thread calls it), and the total.
__device__ __forceinline__ uint32_t block_exclusive(uint32_t v, uint32_t* lds, uint32_t* total) {
  const int tid = threadIdx.x;
  lds[tid] = v;
  __syncthreads();
  for (int off = 1; off < kThreads; off <<= 1) {          // Hillis-Steele inclusive scan
    const uint32_t add = tid >= off ? lds[tid - off] : 0u;
    __syncthreads();
    lds[tid] += add;
    __syncthreads();
  }
  const uint32_t incl = lds[tid];
  *total = lds[kThreads - 1];
  __syncthreads();
  return incl - v;
}

__global__ __launch_bounds__(kThreads) void scan_sums_kernel(const uint32_t* __restrict__ v, int n,
                                                             uint32_t* __restrict__ sums) {
  __shared__ uint32_t lds[kThreads];
  const int beg = blockIdx.x * kScanChunk + threadIdx.x * kScanPer;
  uint32_t a = 0;
#pragma unroll
  for (int k = 0; k < kScanPer; ++k) a += beg + k < n ? v[beg + k] : 0u;
  uint32_t total;
  block_exclusive(a, lds, &total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// sums: the chunk sums (read only by chunks after the first; nb <= 256 * 16).
__global__ __launch_bounds__(kThreads) void scan_apply_kernel(uint32_t* __restrict__ v, int n,
                                                              const uint32_t* __restrict__ sums) {
  __shared__ uint32_t lds[kThreads];
  uint32_t before = 0;
  for (int j = threadIdx.x; j < static_cast<int>(blockIdx.x); j += kThreads) before += sums[j];
  uint32_t offset;
  block_exclusive(before, lds, &offset);                  // offset: all threads' parts summed
  const int beg = blockIdx.x * kScanChunk + threadIdx.x * kScanPer;
  uint32_t loc[kScanPer];
  uint32_t a = 0;
#pragma unroll
  for (int k = 0; k < kScanPer; ++k) {
    loc[k] = beg + k < n ? v[beg + k] : 0u;
    a += loc[k];
  }
  uint32_t total;
  uint32_t run = offset + block_exclusive(a, lds, &total);
#pragma unroll
  for (int k = 0; k < kScanPer; ++k) {
    if (beg + k < n) v[beg + k] = run;
    run += loc[k];
  }
}

__global__ __launch_bounds__(kThreads) void sort_scatter_kernel(
    const uint32_t* __restrict__ keys_in, const uint32_t* __restrict__ vals_in,
    uint32_t* __restrict__ keys_out, uint32_t* __restrict__ vals_out, int M, int shift, int dbits,
    const uint32_t* __restrict__ offs, int tiles) {
  __shared__ uint32_t base[kMaxDigits];
  __shared__ uint32_t wcnt[kWaves][kMaxDigits];
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  const int nd = 1 << dbits;
  const uint32_t mask = static_cast<uint32_t>(nd - 1);
  for (int d = tid; d < nd; d += kThreads) {
    base[d] = offs[static_cast<size_t>(d) * tiles + blockIdx.x];
#pragma unroll
    for (int w = 0; w < kWaves; ++w) wcnt[w][d] = 0;
  }
  const int tile0 = blockIdx.x * kTile;
  uint32_t kin[kSteps], vin[kSteps];
#pragma unroll
  for (int q = 0; q < kSteps; ++q) {
    const int pos = tile0 + q * kThreads + tid;
    kin[q] = pos < M ? keys_in[pos] : 0u;
    vin[q] = pos < M ? vals_in[pos] : 0u;
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < kSteps; ++q) {
    const int pos = tile0 + q * kThreads + tid;
    const bool valid = pos < M;
    const uint32_t key = kin[q];
    const uint32_t digit = (key >> shift) & mask;
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int b = 0; b < kMaxDigitBits; ++b) {
      if (b < dbits) {
        const uint64_t ones = __ballot(valid && ((digit >> b) & 1u));
        peers &= ((digit >> b) & 1u) ? ones : ~ones;
      }
    }
    const uint32_t rank = static_cast<uint32_t>(__popcll(peers & lanes_below()));
    const uint32_t here = static_cast<uint32_t>(__popcll(peers));
    const bool leader = valid && rank == 0;
    if (leader) wcnt[wave][digit] = here;
    __syncthreads();
    if (valid) {
      uint32_t dst = base[digit] + rank;
      for (int w = 0; w < wave; ++w) dst += wcnt[w][digit];
      keys_out[dst] = key;
      vals_out[dst] = vin[q];
    }
    __syncthreads();
    // the digit's running offset takes every wave's count (LDS atomics: an integer sum, exact in
    // any order); each post is cleared by the wave that made it.  No barrier is needed before the
    // next step: every read of this step's offsets and posts came before the barrier above, the
    // next step's posts go to the posting wave's own row (after its own clears, in program
    // order), and the next step reads offsets and posts only after its own first barrier.
    if (leader) {
      atomicAdd(&base[digit], here);
      wcnt[wave][digit] = 0;
    }
  }
}

}  // namespace

size_t scan_workspace_bytes(int n) {
  return (static_cast<size_t>(n) / kScanChunk + 2) * sizeof(uint32_t);
}

hipError_t scan_exclusive(uint32_t* v, int n, uint32_t* sums, hipStream_t s) {
  const int nb = (n + kScanChunk - 1) / kScanChunk;
  if (nb > kScanChunk) return hipErrorInvalidValue;
  if (nb == 0) return hipSuccess;
  if (nb > 1) hipLaunchKernelGGL(scan_sums_kernel, dim3(nb), dim3(kThreads), 0, s, v, n, sums);
  hipLaunchKernelGGL(scan_apply_kernel, dim3(nb), dim3(kThreads), 0, s, v, n, sums);
  return hipGetLastError();
}

size_t sort_workspace_bytes(int M) {
  const size_t tiles = (static_cast<size_t>(M) + kTile - 1) / kTile;
  return 2 * static_cast<size_t>(M) * sizeof(uint32_t) + kMaxDigits * tiles * sizeof(uint32_t) +
         scan_workspace_bytes(static_cast<int>(kMaxDigits * tiles)) + 256;
}

hipError_t sort_pairs(uint32_t* keys, uint32_t* vals, int M, int bits, void* ws, hipStream_t s,
                      uint32_t** keys_sorted, uint32_t** vals_sorted) {
  uint32_t* k2 = static_cast<uint32_t*>(ws);
  uint32_t* v2 = k2 + M;
  uint32_t* hist = v2 + M;
  uint32_t* sums = hist + kMaxDigits * static_cast<size_t>((M + kTile - 1) / kTile);
  uint32_t *ka = keys, *va = vals, *kb = k2, *vb = v2;
  const int tiles = (M + kTile - 1) / kTile;
  const int passes = (M <= 1 || bits <= 0) ? 0 : (bits + kMaxDigitBits - 1) / kMaxDigitBits;
  const int dbits = passes > 0 ? (bits + passes - 1) / passes : 0;      // <= kMaxDigitBits
  if (static_cast<int64_t>(tiles) << dbits > static_cast<int64_t>(kScanChunk) * kScanChunk)
    return hipErrorInvalidValue;                          // beyond the scan (M of 2^25 and more)
  for (int pass = 0; pass < passes; ++pass) {
    const int shift = dbits * pass;
    hipLaunchKernelGGL(sort_hist_kernel, dim3(tiles), dim3(kThreads), 0, s, ka, M, shift, dbits,
                       hist, tiles);
    hipError_t e = scan_exclusive(hist, tiles << dbits, sums, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(sort_scatter_kernel, dim3(tiles), dim3(kThreads), 0, s, ka, va, kb, vb, M,
                       shift, dbits, hist, tiles);
    std::swap(ka, kb);
    std::swap(va, vb);
  }
  *keys_sorted = ka;     // the input arrays or the scratch copies, by the number of passes
  *vals_sorted = va;
  return hipGetLastError();
}

}  // namespace umem
