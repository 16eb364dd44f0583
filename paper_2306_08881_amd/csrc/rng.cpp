// Counter-based draw of the initial factors P_0, Q_0 (i.i.d. standard normal, Section IV-A,
// "Error-feedback").  SplitMix64's finaliser (Steele, Lea and Flood, OOPSLA 2014; Stafford's
// mix variant 13 constants) keys every element by (seed, tensor, factor, index), so the draw is
// independent of the bucket layout; Box-Muller (1958) turns two uniforms into one normal in
// float64 with the C library's log and cos, rounded once to float32.
//
// Built without fast-math or FMA contraction so that the float64 expression is evaluated as
// written.
#include <cmath>
#include <cstdint>

#include "plan.hpp"

namespace acp {

static constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

uint64_t splitmix64_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

void draw_init_factor(uint64_t seed, int32_t tid, int32_t f, int64_t count, float* out) {
  const uint64_t s = splitmix64_mix(seed ^ splitmix64_mix(2ull * static_cast<uint64_t>(tid) +
                                                          static_cast<uint64_t>(f)));
  const double two_pi = 2.0 * M_PI;
  for (int64_t i = 0; i < count; ++i) {
    const uint64_t ui = static_cast<uint64_t>(i);
    const uint64_t a = splitmix64_mix(s + (2ull * ui + 1ull) * kGamma);
    const uint64_t b = splitmix64_mix(s + (2ull * ui + 2ull) * kGamma);
    const double u1 = static_cast<double>((a >> 11) + 1ull) * 0x1.0p-53;
    const double u2 = static_cast<double>(b >> 11) * 0x1.0p-53;
    const double rad = std::sqrt(-2.0 * std::log(u1));
    const double ang = std::cos(two_pi * u2);
    out[i] = static_cast<float>(rad * ang);
  }
}

}  // namespace acp
