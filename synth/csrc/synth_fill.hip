// Device twin of the seeded generator: fills a buffer with the same bits as synth.normal_f32
// (and its bf16 rounding), for tables too large to draw on the host.  It draws numbers only.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

__device__ __forceinline__ uint64_t fmix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ float draw(uint64_t key, uint64_t e, float scale) {
  const uint64_t z = fmix(key + (e + 1ull) * kGamma);
  const int64_t c = static_cast<int64_t>((z & 0xFFFFull) + ((z >> 16) & 0xFFFFull) +
                                         ((z >> 32) & 0xFFFFull) + (z >> 48)) - 131070;
  return __fmul_rn(static_cast<float>(c), scale);
}

__device__ __forceinline__ uint16_t to_bf16(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Each thread writes 8 consecutive elements [8 g, 8 g + 8) of dst, a grid-stride loop over g.
__global__ void fill_kernel(uint64_t key, float scale, uint64_t start, int64_t count, int bf16,
                            void* dst) {
  const int64_t groups = (count + 7) / 8;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t g = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; g < groups;
       g += stride) {
    const int64_t i0 = g * 8;
    const int64_t n = (count - i0) < 8 ? (count - i0) : 8;
    if (bf16) {
      uint16_t* d = static_cast<uint16_t*>(dst) + i0;
      for (int64_t j = 0; j < n; ++j) d[j] = to_bf16(draw(key, start + i0 + j, scale));
    } else {
      float* d = static_cast<float*>(dst) + i0;
      for (int64_t j = 0; j < n; ++j) d[j] = draw(key, start + i0 + j, scale);
    }
  }
}

}  // namespace

// Returns 0, -1 for bad arguments, or -(1000 + hipError_t) when the launch fails.
extern "C" __attribute__((visibility("default"))) int synth_fill_normal(
    uint64_t key, float scale, uint64_t start, int64_t count, int bf16, void* dst,
    hipStream_t stream) {
  if (count < 0 || (count > 0 && dst == nullptr)) return -1;
  if (count == 0) return 0;
  const int64_t groups = (count + 7) / 8;
  const int64_t blocks = (groups + 255) / 256 < 65536 ? (groups + 255) / 256 : 65536;
  (void)hipGetLastError();     // an error left pending by an earlier call is not this launch's
  hipLaunchKernelGGL(fill_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, key,
                     scale, start, count, bf16, dst);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : -(1000 + static_cast<int>(e));
}
