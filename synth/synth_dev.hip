// Device side of the seeded input generator: fills a dense block whose element
// i has logical index base + sum_k coord_k(i) * stride_k with the same
// counter-mode SplitMix64 / Irwin-Hall draw as the host generator, so that
// host and device produce identical bits.  Holds no arithmetic of the method.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

struct Layout {
  int ndim;
  int64_t shape[6];
  int64_t stride[6];
};

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__global__ void fill_normal_kernel(void* out, int bf16, int64_t n, Layout lay, int64_t base,
                                   uint64_t key, float scale) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= n) return;
  int64_t rem = i, idx = base;
  for (int k = lay.ndim - 1; k >= 0; --k) {
    idx += (rem % lay.shape[k]) * lay.stride[k];
    rem /= lay.shape[k];
  }
  const uint64_t z = mix64(key + (static_cast<uint64_t>(idx) + 1ull) * 0x9E3779B97F4A7C15ull);
  const int32_t s = static_cast<int32_t>((z & 0xFFFF) + ((z >> 16) & 0xFFFF) + ((z >> 32) & 0xFFFF) +
                                         (z >> 48)) - 2 * 65535;
  const float f = static_cast<float>(s) * scale;
  if (bf16) {
    uint32_t b = __float_as_uint(f);
    b += 0x7FFFu + ((b >> 16) & 1u);
    static_cast<uint16_t*>(out)[i] = static_cast<uint16_t>(b >> 16);
  } else {
    static_cast<float*>(out)[i] = f;
  }
}

// Plain 16-byte copy: the reference kernel of known traffic against which
// hardware byte counters are calibrated.
__global__ void copy16_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, int64_t n) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride)
    dst[i] = src[i];
}

}  // namespace

extern "C" int synth_copy(void* dst, const void* src, int64_t bytes, hipStream_t stream) {
  if (!dst || !src || bytes < 0 || bytes % 16) return 1;
  const int64_t n = bytes / 16;
  if (n == 0) return 0;
  const int64_t want = (n + 255) / 256;
  const unsigned blocks = static_cast<unsigned>(want < 8192 ? want : 8192);
  hipLaunchKernelGGL(copy16_kernel, dim3(blocks), dim3(256), 0, stream,
                     static_cast<const uint4*>(src), static_cast<uint4*>(dst), n);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

extern "C" int synth_fill_normal(void* out, int bf16, int ndim, const int64_t* shape,
                                 const int64_t* stride, int64_t base, uint64_t key, float scale,
                                 hipStream_t stream) {
  if (!out || ndim < 1 || ndim > 6) return 1;
  Layout lay{};
  lay.ndim = ndim;
  int64_t n = 1;
  for (int k = 0; k < ndim; ++k) {
    if (shape[k] <= 0) return 0;
    lay.shape[k] = shape[k];
    lay.stride[k] = stride[k];
    n *= shape[k];
  }
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(fill_normal_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream,
                     out, bf16, n, lay, base, key, scale);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}
