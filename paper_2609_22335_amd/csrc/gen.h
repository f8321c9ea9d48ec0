// Host-side counter-based parameter generator (see gen.cpp).
#pragma once
#include <stddef.h>
#include <stdint.h>

namespace vla {
uint64_t fnv1a64(const char* s);
uint64_t stream_key(uint64_t seed, const char* name);
// out[i] = value i of the named stream, N(mean, stdv) stand-in, fp32.
void gen_normal(uint64_t seed, const char* name, size_t n, double mean, double stdv, float* out);
uint16_t bf16_bits(float f);  // round to nearest even
float bf16_value(uint16_t h);
}  // namespace vla
