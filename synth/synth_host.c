/* Host side of the seeded input generator, in C for speed: element i of a
 * dense block has logical index base + sum_k coord_k(i) * stride_k and value
 * normal(key, index) exactly as defined in synth/__init__.py (counter-mode
 * SplitMix64, Irwin-Hall sum of the four 16-bit fields, one fp32 multiply,
 * round-to-nearest-even to bf16).  Holds no arithmetic of the method. */
#include <stdint.h>
#include <string.h>

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

static inline float draw_normal(uint64_t key, int64_t idx, float scale) {
  const uint64_t z = mix64(key + ((uint64_t)idx + 1ull) * 0x9E3779B97F4A7C15ull);
  const int32_t s = (int32_t)((z & 0xFFFF) + ((z >> 16) & 0xFFFF) + ((z >> 32) & 0xFFFF) +
                              (z >> 48)) - 2 * 65535;
  return (float)s * scale;
}

static inline uint16_t to_bf16(float f) {
  uint32_t b;
  memcpy(&b, &f, 4);
  b += 0x7FFFu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}

/* out, dense in the block's shape: float32 values (bf16 == 0), bf16 bits
 * (bf16 == 1), or the bf16-rounded values widened back to float32 (bf16 == 2). */
int synth_host_fill(void* out, int bf16, int ndim, const int64_t* shape, const int64_t* stride,
                    int64_t base, uint64_t key, float scale) {
  if (!out || ndim < 1 || ndim > 8) return 1;
  int64_t n = 1;
  for (int k = 0; k < ndim; ++k) {
    if (shape[k] <= 0) return 0;
    n *= shape[k];
  }
  const int64_t inner = shape[ndim - 1], rows = n / inner, st_in = stride[ndim - 1];
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    int64_t rem = r, idx = base;
    for (int k = ndim - 2; k >= 0; --k) {
      idx += (rem % shape[k]) * stride[k];
      rem /= shape[k];
    }
    if (bf16 == 2) {
      float* o = (float*)out + r * inner;
      for (int64_t c = 0; c < inner; ++c) {
        const uint32_t b = (uint32_t)to_bf16(draw_normal(key, idx + c * st_in, scale)) << 16;
        memcpy(o + c, &b, 4);
      }
    } else if (bf16) {
      uint16_t* o = (uint16_t*)out + r * inner;
      for (int64_t c = 0; c < inner; ++c) o[c] = to_bf16(draw_normal(key, idx + c * st_in, scale));
    } else {
      float* o = (float*)out + r * inner;
      for (int64_t c = 0; c < inner; ++c) o[c] = draw_normal(key, idx + c * st_in, scale);
    }
  }
  return 0;
}
