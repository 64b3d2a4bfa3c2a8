/* Host side of the seeded input generator, in C with OpenMP: the same
 * counter-based SplitMix64 stream, quantile table, single fp32 multiply and
 * integer round-to-nearest-even to bf16 as synth/gen.py (the reference
 * definition) and synth/fill.hip (device).  Input generation only. */
#include <stdint.h>

static const uint64_t kGamma = 0x9E3779B97F4A7C15ull;

static inline uint64_t mix64(uint64_t z) {
  z ^= z >> 30;
  z *= 0xBF58476D1CE4E5B9ull;
  z ^= z >> 27;
  z *= 0x94D049BB133111EBull;
  z ^= z >> 31;
  return z;
}

static inline float round_bf16(float v) {
  union { float f; uint32_t u; } x;
  x.f = v;
  x.u = ((x.u + 0x7FFFu + ((x.u >> 16) & 1u)) >> 16) << 16;
  return x.f;
}

/* out[i] = element i0+i of stream `key`; as_bf16: value rounded to bf16
 * (returned as its fp32 value). */
void synth_host_normal(uint64_t key, uint64_t i0, int64_t n, const float* table, float sigma,
                       int as_bf16, float* out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    const uint64_t u = mix64(key + (i0 + (uint64_t)i + 1ull) * kGamma);
    const float v = table[u >> 48] * sigma;
    out[i] = as_bf16 ? round_bf16(v) : v;
  }
}
