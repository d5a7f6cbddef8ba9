/* Seeded, counter-based synthetic value generator shared by the CPU oracle and
 * the GPU path as *input data*.  It holds none of DFlow's arithmetic.
 *
 * Element i of a tensor with 64-bit key k is derived from splitmix64
 * (Steele, Lea & Flood, "Fast splittable pseudorandom number generators",
 * OOPSLA 2014; finaliser constants as in Vigna's public reference code)
 * applied to the counter k + (i+1)*golden_gamma.  The four 16-bit lanes of
 * the hash are summed (Irwin-Hall with n = 4) and standardised, giving an
 * approximately normal variate with mean 0 and variance 1 using integer
 * arithmetic and one float multiply, so the bytes are identical on every
 * host, libm and thread count.
 */
#include <stdint.h>
#include <string.h>

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static inline float std_variate(uint64_t key, int64_t i) {
  uint64_t h = mix64(key + (uint64_t)(i + 1) * 0x9E3779B97F4A7C15ULL);
  int64_t s = (int64_t)(h & 0xFFFF) + (int64_t)((h >> 16) & 0xFFFF) +
              (int64_t)((h >> 32) & 0xFFFF) + (int64_t)(h >> 48);
  /* sum of four (l+0.5)/65536 has mean 2 and variance 1/3; shift/scale */
  double c = 2.0 * 65536.0 - 2.0; /* 4*0.5 offset folded in: sum(l)+2 - 2*65536 */
  return (float)(((double)s - c) * (1.7320508075688772 / 65536.0));
}

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

void wl_fill_f32(float* out, int64_t n, uint64_t key, float mean, float std) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = mean + std * std_variate(key, i);
}

void wl_fill_bf16(uint16_t* out, int64_t n, uint64_t key, float mean, float std) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) out[i] = f32_to_bf16_rne(mean + std * std_variate(key, i));
}

void wl_bf16_to_f32(const uint16_t* in, float* out, int64_t n) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    uint32_t u = (uint32_t)in[i] << 16;
    memcpy(&out[i], &u, 4);
  }
}
