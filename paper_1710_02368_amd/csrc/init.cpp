// Initial parameters: He-normal weights N(0, 2/d_in), zero biases.
//
// Random source: the SplitMix64 generator (Steele, Lea and Flood, OOPSLA
// 2014), whose output number i (i = 0, 1, ...) for a seed s is the
// finaliser applied to s + (i+1)*0x9E3779B97F4A7C15.  Weight number w (in
// the packed order W_0 row-major, W_1, ...) uses outputs 2w and 2w+1 as
// u1 = ((x >> 11) + 1) * 2^-53 in (0,1] and u2 = (x >> 11) * 2^-53 in [0,1),
// and the Box-Muller transform sqrt(-2 ln u1) cos(2 pi u2), evaluated in
// double precision, times sqrt(2/d_in), rounded once to float.
#include <cmath>
#include <cstdint>

#include "agn_internal.h"

namespace agn {
namespace {

inline uint64_t splitmix64_at(uint64_t seed, uint64_t i) {
  uint64_t z = seed + (i + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

}  // namespace

void he_normal_init(const int32_t* dims, int32_t L, uint64_t seed, float* packed) {
  const double two_pi = 2.0 * M_PI;
  uint64_t w = 0;    // global weight counter
  int64_t off = 0;   // packed offset
  for (int l = 0; l < L; ++l) {
    const int64_t fan_in = dims[l], fan_out = dims[l + 1];
    const double scale = std::sqrt(2.0 / (double)fan_in);
    const int64_t cnt = fan_in * fan_out;
    for (int64_t e = 0; e < cnt; ++e, ++w) {
      const uint64_t x1 = splitmix64_at(seed, 2 * w), x2 = splitmix64_at(seed, 2 * w + 1);
      const double u1 = ((double)(x1 >> 11) + 1.0) * 0x1.0p-53;
      const double u2 = (double)(x2 >> 11) * 0x1.0p-53;
      const double z = std::sqrt(-2.0 * std::log(u1)) * std::cos(two_pi * u2);
      packed[off + e] = (float)(z * scale);
    }
    off += cnt;
    for (int64_t e = 0; e < fan_out; ++e) packed[off + e] = 0.f;
    off += fan_out;
  }
}

}  // namespace agn
