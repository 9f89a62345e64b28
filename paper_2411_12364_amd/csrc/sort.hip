// Stable sort of (key, value) pairs of 32-bit unsigned keys: least-significant-digit radix sort
// with 8-bit digits, ceil(bits / 8) passes.  The backward passes use it to bring all
// contributions to one value row (or key row) together, in their original order, so that one
// wave sums them in a fixed order and the gradient does not depend on timing.
//
// Per pass, over tiles of 4096 pairs (256 threads x 16 steps):
//  * sort_hist_kernel: the tile's digit histogram (LDS atomics), stored digit-major [256][tiles];
//  * sort_scan_kernel: one workgroup turns the 256 * tiles counts into exclusive offsets (digit
//    by digit, tile by tile: the order the stable pass writes in);
//  * sort_scatter_kernel: the tile again, 256 consecutive pairs per step; a pair's place is its
//    digit's running offset in this tile + the count of equal digits in earlier waves of this
//    step + its rank among equal digits in its own wave (eight ballots match the digit).
#include <utility>

#include "umem_internal.h"

namespace umem {
namespace {

constexpr int kThreads = 256;
constexpr int kSteps = 16;
constexpr int kTile = kThreads * kSteps;
constexpr int kWaves = kThreads / kWave;
constexpr int kScanThreads = 1024;

__device__ __forceinline__ uint64_t lanes_below() {
  const unsigned lane = threadIdx.x & (kWave - 1);
  return lane == 0 ? 0ull : (~0ull >> (kWave - lane));
}

__global__ __launch_bounds__(kThreads) void sort_hist_kernel(const uint32_t* __restrict__ keys,
                                                             int M, int shift,
                                                             uint32_t* __restrict__ hist,
                                                             int tiles) {
  __shared__ uint32_t cnt[256];
  cnt[threadIdx.x] = 0;
  __syncthreads();
  const int base = blockIdx.x * kTile;
  for (int q = 0; q < kSteps; ++q) {
    const int pos = base + q * kThreads + threadIdx.x;
    if (pos < M) atomicAdd(&cnt[(keys[pos] >> shift) & 255u], 1u);
  }
  __syncthreads();
  hist[static_cast<size_t>(threadIdx.x) * tiles + blockIdx.x] = cnt[threadIdx.x];
}

// Exclusive scan of n counts in place, one workgroup: each thread sums a contiguous chunk, the
// chunk sums are scanned in LDS, and each thread rewrites its chunk with running offsets.
__global__ __launch_bounds__(kScanThreads) void sort_scan_kernel(uint32_t* __restrict__ v, int n) {
  __shared__ uint32_t part[kScanThreads];
  const int per = (n + kScanThreads - 1) / kScanThreads;
  const int beg = threadIdx.x * per, end = min(n, beg + per);
  uint32_t s = 0;
  for (int i = beg; i < end; ++i) s += v[i];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int off = 1; off < kScanThreads; off <<= 1) {      // Hillis-Steele inclusive scan
    const uint32_t add = threadIdx.x >= off ? part[threadIdx.x - off] : 0u;
    __syncthreads();
    part[threadIdx.x] += add;
    __syncthreads();
  }
  uint32_t run = part[threadIdx.x] - s;                    // exclusive
  for (int i = beg; i < end; ++i) {
    const uint32_t c = v[i];
    v[i] = run;
    run += c;
  }
}

__global__ __launch_bounds__(kThreads) void sort_scatter_kernel(
    const uint32_t* __restrict__ keys_in, const uint32_t* __restrict__ vals_in,
    uint32_t* __restrict__ keys_out, uint32_t* __restrict__ vals_out, int M, int shift,
    const uint32_t* __restrict__ offs, int tiles) {
  __shared__ uint32_t base[256];
  __shared__ uint32_t wcnt[kWaves][256];
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  base[tid] = offs[static_cast<size_t>(tid) * tiles + blockIdx.x];
  const int tile0 = blockIdx.x * kTile;
  for (int q = 0; q < kSteps; ++q) {
#pragma unroll
    for (int w = 0; w < kWaves; ++w) wcnt[w][tid] = 0;
    __syncthreads();
    const int pos = tile0 + q * kThreads + tid;
    const bool valid = pos < M;
    const uint32_t key = valid ? keys_in[pos] : 0u;
    const uint32_t val = valid ? vals_in[pos] : 0u;
    const uint32_t digit = (key >> shift) & 255u;
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const uint64_t ones = __ballot(valid && ((digit >> b) & 1u));
      peers &= ((digit >> b) & 1u) ? ones : ~ones;
    }
    const uint32_t rank = static_cast<uint32_t>(__popcll(peers & lanes_below()));
    if (valid && rank == 0) wcnt[wave][digit] = static_cast<uint32_t>(__popcll(peers));
    __syncthreads();
    if (valid) {
      uint32_t dst = base[digit] + rank;
      for (int w = 0; w < wave; ++w) dst += wcnt[w][digit];
      keys_out[dst] = key;
      vals_out[dst] = val;
    }
    __syncthreads();
    uint32_t add = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) add += wcnt[w][tid];
    base[tid] += add;
    // the next step's clearing of wcnt follows this read only after its own barrier
    __syncthreads();
  }
}

}  // namespace

size_t sort_workspace_bytes(int M) {
  const size_t tiles = (static_cast<size_t>(M) + kTile - 1) / kTile;
  return 2 * static_cast<size_t>(M) * sizeof(uint32_t) + 256 * tiles * sizeof(uint32_t) + 256;
}

hipError_t sort_pairs(uint32_t* keys, uint32_t* vals, int M, int bits, void* ws, hipStream_t s,
                      uint32_t** keys_sorted, uint32_t** vals_sorted) {
  uint32_t* k2 = static_cast<uint32_t*>(ws);
  uint32_t* v2 = k2 + M;
  uint32_t* hist = v2 + M;
  uint32_t *ka = keys, *va = vals, *kb = k2, *vb = v2;
  const int tiles = (M + kTile - 1) / kTile;
  const int passes = (M <= 1 || bits <= 0) ? 0 : (bits + 7) / 8;
  for (int pass = 0; pass < passes; ++pass) {
    const int shift = 8 * pass;
    hipLaunchKernelGGL(sort_hist_kernel, dim3(tiles), dim3(kThreads), 0, s, ka, M, shift, hist, tiles);
    hipLaunchKernelGGL(sort_scan_kernel, dim3(1), dim3(kScanThreads), 0, s, hist, 256 * tiles);
    hipLaunchKernelGGL(sort_scatter_kernel, dim3(tiles), dim3(kThreads), 0, s, ka, va, kb, vb, M,
                       shift, hist, tiles);
    std::swap(ka, kb);
    std::swap(va, vb);
  }
  *keys_sorted = ka;     // the input arrays or the scratch copies, by the number of passes
  *vals_sorted = va;
  return hipGetLastError();
}

}  // namespace umem
