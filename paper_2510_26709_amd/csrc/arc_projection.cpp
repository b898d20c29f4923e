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
#include <mutex>
#include <thread>
#include <vector>

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

void generate_projection_rows(uint64_t seed, int64_t t, int64_t n, int32_t r, int64_t j0,
                              int64_t j1, float* V) {
  constexpr double kTwoPi = 6.283185307179586476925286766559;
  constexpr double kTwoToMinus53 = 1.0 / 9007199254740992.0;
  const uint64_t un = static_cast<uint64_t>(n), ur = static_cast<uint64_t>(r);
  const uint64_t row0 = static_cast<uint64_t>(t) * un;
  for (uint64_t j = static_cast<uint64_t>(j0); j < static_cast<uint64_t>(j1); ++j) {
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

void generate_projection(uint64_t seed, int64_t t, int64_t n, int32_t r, float* V) {
  generate_projection_rows(seed, t, n, r, 0, n, V);
}

// ---------------------------------------------------------------------------
// ProjectionPool: the rows of every width's V_t split evenly over a few
// threads.  Each entry is a pure function of (seed, t, j, k), so the split
// changes no value.
// ---------------------------------------------------------------------------
ProjectionPool::ProjectionPool(int threads) {
  if (threads < 1) threads = 1;
  // Each thread gets the count by value: threads_ is still growing while the
  // first ones start.
  threads_.reserve(static_cast<size_t>(threads));
  for (int i = 0; i < threads; ++i) threads_.emplace_back([this, i, threads] { run(i, threads); });
}

ProjectionPool::~ProjectionPool() {
  {
    std::lock_guard<std::mutex> lk(mu_);
    quit_ = true;
  }
  cv_job_.notify_all();
  for (std::thread& th : threads_) th.join();
}

void ProjectionPool::start(uint64_t seed, int64_t t, int32_t r,
                           const std::vector<ProjectionBlock>* blocks, float* dst) {
  wait();
  std::lock_guard<std::mutex> lk(mu_);
  seed_ = seed;
  t_ = t;
  r_ = r;
  blocks_ = blocks;
  dst_ = dst;
  total_rows_ = 0;
  for (const ProjectionBlock& b : *blocks) total_rows_ += b.width;
  remaining_ = static_cast<int>(threads_.size());
  ++job_;
  cv_job_.notify_all();
}

void ProjectionPool::wait() {
  std::unique_lock<std::mutex> lk(mu_);
  cv_done_.wait(lk, [this] { return remaining_ == 0; });
}

void ProjectionPool::run(int id, int nthreads) {
  uint64_t seen = 0;
  for (;;) {
    std::unique_lock<std::mutex> lk(mu_);
    cv_job_.wait(lk, [&] { return quit_ || job_ != seen; });
    if (quit_) return;
    seen = job_;
    const uint64_t seed = seed_;
    const int64_t t = t_, total = total_rows_;
    const int32_t r = r_;
    const std::vector<ProjectionBlock>& blocks = *blocks_;
    float* dst = dst_;
    lk.unlock();
    // This thread's share [lo, hi) of the rows of all widths, in block order.
    const int64_t lo = total * id / nthreads, hi = total * (id + 1) / nthreads;
    int64_t first = 0;
    for (const ProjectionBlock& b : blocks) {
      const int64_t j0 = lo > first ? lo - first : 0;
      const int64_t j1 = hi - first < b.width ? hi - first : b.width;
      if (j0 < j1) generate_projection_rows(seed, t, b.width, r, j0, j1, dst + b.offset);
      first += b.width;
    }
    lk.lock();
    if (--remaining_ == 0) cv_done_.notify_all();
  }
}

}  // namespace arc
