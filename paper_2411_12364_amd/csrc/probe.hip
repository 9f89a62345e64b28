// Read-bandwidth probes for the benchmark (libumem_probe.so; not part of the layer or its ABI).
//
// They measure how fast this GPU delivers HBM reads in the two access patterns of the
// gather-sum, with nothing else in the kernel: long sequential runs, and whole value rows at the
// addresses of a real bag.  The gather's achieved rate is reported as a fraction of these
// ceilings beside the vendor peak.  Loads are 16 bytes per lane and nontemporal, as the gather's
// are for rows that are read once; the data is folded with XOR, and a wave writes only if the fold
// hits a value it never takes here, so that the loads stay live without any store traffic.
#include <hip/hip_runtime.h>
#include <stdint.h>

#define UMEM_PROBE_API extern "C" __attribute__((visibility("default")))

namespace {

constexpr int THREADS = 256;
constexpr int WAVES = THREADS / 64;
constexpr int ROWS_PER_WAVE = 64;     // one bag of a decode token (2 heads x top-32)
constexpr int IN_FLIGHT = 16;         // row loads per lane before the first is folded
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t fold(u32x4 v) { return v.x ^ v.y ^ v.z ^ v.w; }

// rows[0, n_rows): each wave reads 64 consecutive entries' rows, CPL 16-byte chunks per lane
// (row_bytes = 1024 CPL).
template <int CPL>
__global__ __launch_bounds__(THREADS) void read_rows_kernel(const char* __restrict__ table,
                                                            const int32_t* __restrict__ rows,
                                                            int64_t n_rows, uint32_t* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = static_cast<int64_t>(blockIdx.x) * WAVES + threadIdx.x / 64;
  const int64_t beg = wave * ROWS_PER_WAVE;
  if (beg >= n_rows) return;
  const int64_t end = beg + ROWS_PER_WAVE < n_rows ? beg + ROWS_PER_WAVE : n_rows;
  const int my_row = beg + lane < end ? rows[beg + lane] : 0;
  uint32_t acc = 0u;
  for (int64_t j0 = beg; j0 < end; j0 += IN_FLIGHT) {
    u32x4 v[IN_FLIGHT][CPL];
#pragma unroll
    for (int u = 0; u < IN_FLIGHT; ++u) {
      const int64_t j = j0 + u;
      const int r = __shfl(my_row, static_cast<int>(j - beg) & 63, 64);
      const u32x4* src = reinterpret_cast<const u32x4*>(table + static_cast<int64_t>(r) * (1024 * CPL));
#pragma unroll
      for (int c = 0; c < CPL; ++c)
        v[u][c] = j < end ? __builtin_nontemporal_load(src + 64 * c + lane) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < IN_FLIGHT; ++u)
#pragma unroll
      for (int c = 0; c < CPL; ++c) acc ^= fold(v[u][c]);
  }
  if (acc == 0x9E3779B9u) sink[wave & 1023] = acc;
}

// A sequential read of n16 16-byte chunks, grid-stride, eight loads in flight per lane.
__global__ __launch_bounds__(THREADS) void read_seq_kernel(const u32x4* __restrict__ p, int64_t n16,
                                                           uint32_t* __restrict__ sink) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * THREADS;
  uint32_t acc = 0u;
  int64_t i = static_cast<int64_t>(blockIdx.x) * THREADS + threadIdx.x;
  for (; i + 7 * stride < n16; i += 8 * stride) {
    u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
    for (int u = 0; u < 8; ++u) acc ^= fold(v[u]);
  }
  for (; i < n16; i += stride) acc ^= fold(__builtin_nontemporal_load(p + i));
  if (acc == 0x9E3779B9u) sink[blockIdx.x & 1023] = acc;
}

}  // namespace

// Reads the rows rows[0, n_rows) of a table of row_bytes-byte rows (1024 or 2048; table 16-byte
// aligned, every index in range).  sink: 4 KiB of device memory that is almost never written.
// Returns 0, -1 for bad arguments, or -1000 - the HIP error of the launch.
UMEM_PROBE_API int umem_probe_read_rows(const void* table, int row_bytes, const int32_t* rows,
                                        int64_t n_rows, uint32_t* sink, hipStream_t s) {
  if (!table || !rows || !sink || n_rows < 0 || (row_bytes != 1024 && row_bytes != 2048)) return -1;
  if (n_rows == 0) return 0;
  (void)hipGetLastError();
  const int64_t waves = (n_rows + ROWS_PER_WAVE - 1) / ROWS_PER_WAVE;
  const dim3 grid(static_cast<unsigned>((waves + WAVES - 1) / WAVES));
  if (row_bytes == 1024)
    hipLaunchKernelGGL(read_rows_kernel<1>, grid, dim3(THREADS), 0, s, static_cast<const char*>(table), rows, n_rows, sink);
  else
    hipLaunchKernelGGL(read_rows_kernel<2>, grid, dim3(THREADS), 0, s, static_cast<const char*>(table), rows, n_rows, sink);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : -1000 - static_cast<int>(e);
}

// Reads bytes (a multiple of 16, 16-byte aligned) sequentially with `blocks` workgroups.
UMEM_PROBE_API int umem_probe_read_seq(const void* p, int64_t bytes, int blocks, uint32_t* sink,
                                       hipStream_t s) {
  if (!p || !sink || bytes < 0 || bytes % 16 != 0 || blocks < 1) return -1;
  if (bytes == 0) return 0;
  (void)hipGetLastError();
  hipLaunchKernelGGL(read_seq_kernel, dim3(blocks), dim3(THREADS), 0, s, static_cast<const u32x4*>(p),
                     bytes / 16, sink);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : -1000 - static_cast<int>(e);
}
