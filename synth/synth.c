/*
 * Seeded synthetic inputs shared by the GPU path's tests/bench and by the
 * CPU oracle.  This file holds no arithmetic of the action-expert method:
 * it only turns (seed, tensor name, element index) into a normal deviate.
 *
 *   key      = FNV-1a-64(name)
 *   u1, u2   = U(splitmix64(seed + key + 2j)), U(splitmix64(seed + key + 2j + 1))
 *   U(x)     = ((x >> 11) + 1) * 2^-53            in (0, 1]
 *   z_j      = sqrt(-2 ln u1) * cos(2 pi u2) * std (Box-Muller, 1958)
 *
 * splitmix64 is the output function of Steele, Lea & Flood (2014),
 * applied to (counter + golden gamma).  Values are produced in fp64 and
 * rounded once to fp32 (round-to-nearest-even); the bf16 helper rounds the
 * fp32 value once more (RNE), so every consumer sees identical bits.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static uint64_t fnv1a64(const char* s) {
  uint64_t h = 0xcbf29ce484222325ULL;
  for (; *s; ++s) {
    h ^= (uint8_t)(*s);
    h *= 0x100000001b3ULL;
  }
  return h;
}

static inline uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9e3779b97f4a7c15ULL;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

static inline double unit_open0(uint64_t x) {
  return (double)((x >> 11) + 1) * (1.0 / 9007199254740992.0);
}

uint64_t jpi_synth_key(const char* name) { return fnv1a64(name); }

/* out[j] = fp32(std * z_j) for j in [0, n). */
void jpi_synth_normal_f32(uint64_t seed, const char* name, double stddev,
                          float* out, int64_t n) {
  const uint64_t base = seed + fnv1a64(name);
  const double two_pi = 6.283185307179586476925286766559;
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j) {
    const uint64_t c = base + 2u * (uint64_t)j;
    const double u1 = unit_open0(splitmix64(c));
    const double u2 = unit_open0(splitmix64(c + 1u));
    const double z = sqrt(-2.0 * log(u1)) * cos(two_pi * u2);
    out[j] = (float)(stddev * z);
  }
}

/* fp32 -> bf16 bits, round to nearest even (NaN kept quiet). */
void jpi_synth_f32_to_bf16(const float* in, uint16_t* out, int64_t n) {
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j) {
    uint32_t u;
    memcpy(&u, &in[j], 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) {
      out[j] = (uint16_t)((u >> 16) | 0x40u);
    } else {
      u += 0x7fffu + ((u >> 16) & 1u);
      out[j] = (uint16_t)(u >> 16);
    }
  }
}
