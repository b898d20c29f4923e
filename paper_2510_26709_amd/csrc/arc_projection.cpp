// Shared Gaussian projection V_t of ARC-Top-K (Sec. IV, Alg. 1: every node
// derives the same V in R^{n x r}, vec(V) ~ N(0, I), from a shared seed).
//
// Generator: SplitMix64 (Steele, Lea & Flood, OOPSLA 2014).  Its state starts
// at the seed and advances by the golden gamma before each output, which is
// the state passed through the variant-13 mixer.  Entry (j, k) of step t uses
// outputs 2c and 2c+1 of the stream, c = (t*n + j)*r + k, as two 53-bit
// uniforms u1 in (0, 1] and u2 in [0, 1), and the cosine branch of the
// Box-Muller transform in binary64, rounded once to binary32.  The result is
// fully determined by (seed, t, n, r) and is identical on every node.
#include <cmath>
#include <cstdint>

#include "arc_internal.h"

namespace arc {
namespace {

constexpr uint64_t kGoldenGamma = 0x9E3779B97F4A7C15ull;

inline uint64_t splitmix_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Generator positioned just before output number x of the seeded stream.
struct SplitMix64 {
  uint64_t state;
  SplitMix64(uint64_t seed, uint64_t x) : state(seed + x * kGoldenGamma) {}
  uint64_t next() {
    state += kGoldenGamma;
    return splitmix_mix(state);
  }
};

}  // namespace

void generate_projection(uint64_t seed, int64_t t, int64_t n, int32_t r,
                         float* V) {
  constexpr double kTwoPi = 6.283185307179586476925286766559;
  constexpr double kTwoToMinus53 = 1.0 / 9007199254740992.0;
  const uint64_t un = static_cast<uint64_t>(n), ur = static_cast<uint64_t>(r);
  const uint64_t row0 = static_cast<uint64_t>(t) * un;
  for (uint64_t j = 0; j < un; ++j) {
    for (uint64_t k = 0; k < ur; ++k) {
      const uint64_t c = (row0 + j) * ur + k;
      SplitMix64 gen(seed, 2 * c);
      const uint64_t w1 = gen.next();
      const uint64_t w2 = gen.next();
      const double u1 = static_cast<double>((w1 >> 11) + 1) * kTwoToMinus53;
      const double u2 = static_cast<double>(w2 >> 11) * kTwoToMinus53;
      const double radius = std::sqrt(-2.0 * std::log(u1));
      const double z = radius * std::cos(kTwoPi * u2);
      V[j * ur + k] = static_cast<float>(z);
    }
  }
}

}  // namespace arc
