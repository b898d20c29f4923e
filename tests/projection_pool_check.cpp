// Host-only check of the library's projection thread pool (built by
// tests/test_projection_pool.py under ThreadSanitizer): for several thread
// counts and steps, the pool's V_t over ten widths must equal the
// single-threaded generator bit for bit; a second start() must wait for the
// first; destroying a pool right after a start must be clean.
#include <cstdio>
#include <cstring>
#include <vector>

#include "arc_internal.h"

int main() {
  const std::vector<int64_t> widths = {64, 128, 147, 256, 512, 576, 1000, 1152, 2304, 4608};
  const int r = 4;
  std::vector<arc::ProjectionBlock> blocks;
  int64_t off = 0;
  for (int64_t w : widths) {
    blocks.push_back({w, off});
    off += w * r;
  }
  std::vector<float> want(off), got(off);
  int bad = 0;
  for (int threads : {1, 2, 3, 5, 8}) {
    arc::ProjectionPool pool(threads);
    for (int64_t t = 0; t < 6; ++t) {
      for (const auto& b : blocks) arc::generate_projection(77, t, b.width, r, want.data() + b.offset);
      std::memset(got.data(), 0xff, got.size() * sizeof(float));
      pool.start(77, t, r, &blocks, got.data());
      pool.wait();
      if (std::memcmp(want.data(), got.data(), off * sizeof(float)) != 0) {
        ++bad;
        std::printf("mismatch: %d threads, t = %ld\n", threads, static_cast<long>(t));
      }
    }
    pool.start(77, 9, r, &blocks, got.data());
    pool.start(77, 10, r, &blocks, got.data());
    pool.wait();
    for (const auto& b : blocks) arc::generate_projection(77, 10, b.width, r, want.data() + b.offset);
    if (std::memcmp(want.data(), got.data(), off * sizeof(float)) != 0) {
      ++bad;
      std::printf("mismatch after a second start: %d threads\n", threads);
    }
  }
  {
    arc::ProjectionPool pool(4);
    pool.start(1, 2, r, &blocks, got.data());
  }
  std::printf("%s\n", bad ? "FAIL" : "ok");
  return bad != 0;
}
