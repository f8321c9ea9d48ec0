// Counter-based parameter generator of the library (host side).
//
// SplitMix64 (Steele, Lea & Flood, OOPSLA 2014) read as "output i of the
// stream whose state starts at s", with s derived from (seed, tensor name):
//   key      = mix64((seed ^ fnv1a64(name)) + GAMMA)
//   draw(i)  = mix64(key + (i + 1) * GAMMA)
// Normal values use Irwin-Hall(4) on the four 16-bit fields of one draw:
//   z = ((S + 2) * 2^-16 - 2) * (sqrt(3) * sigma),  value = fp32(mu + z),
// each operation rounded once in fp64 (this file is built without
// floating-point contraction so no step is fused).
#include "gen.h"

#include <algorithm>
#include <thread>
#include <vector>

#pragma STDC FP_CONTRACT OFF

namespace vla {

static const uint64_t GAMMA = 0x9E3779B97F4A7C15ull;
static const double SQRT3 = 1.7320508075688772;

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

uint64_t fnv1a64(const char* s) {
  uint64_t h = 0xCBF29CE484222325ull;
  for (; *s; ++s) {
    h ^= (uint8_t)*s;
    h *= 0x100000001B3ull;
  }
  return h;
}

uint64_t stream_key(uint64_t seed, const char* name) { return mix64((seed ^ fnv1a64(name)) + GAMMA); }

static void normal_range(uint64_t key, size_t b, size_t e, double mean, double stdv, float* out) {
  const double c = SQRT3 * stdv;
  for (size_t i = b; i < e; ++i) {
    const uint64_t h = mix64(key + (uint64_t)(i + 1) * GAMMA);
    const uint64_t s = (h & 0xFFFF) + ((h >> 16) & 0xFFFF) + ((h >> 32) & 0xFFFF) + (h >> 48);
    double z = (double)(s + 2) * (1.0 / 65536.0);
    z = z - 2.0;
    z = z * c;
    if (mean != 0.0) {
      volatile double zz = z;  // keep the product rounded before the sum
      z = mean + zz;
    }
    out[i] = (float)z;
  }
}

void gen_normal(uint64_t seed, const char* name, size_t n, double mean, double stdv, float* out) {
  const uint64_t key = stream_key(seed, name);
  unsigned nt = std::max(1u, std::min(16u, std::thread::hardware_concurrency()));
  if (n < (size_t)1 << 20) nt = 1;
  if (nt == 1) {
    normal_range(key, 0, n, mean, stdv, out);
    return;
  }
  std::vector<std::thread> th;
  const size_t chunk = (n + nt - 1) / nt;
  for (unsigned t = 0; t < nt; ++t) {
    const size_t b = t * chunk, e = std::min(n, b + chunk);
    if (b >= e) break;
    th.emplace_back(normal_range, key, b, e, mean, stdv, out);
  }
  for (auto& x : th) x.join();
}

uint16_t bf16_bits(float f) {
  uint32_t u;
  __builtin_memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

float bf16_value(uint16_t h) {
  const uint32_t u = (uint32_t)h << 16;
  float f;
  __builtin_memcpy(&f, &u, 4);
  return f;
}

}  // namespace vla
