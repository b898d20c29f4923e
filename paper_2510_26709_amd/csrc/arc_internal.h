// Internal declarations shared by the libarctopk host code and its kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace arc {

// Rows of the importance vector handled by one block of the selection
// kernels (256 threads x 8 consecutive rows).
constexpr int kSelectThreads = 256;
constexpr int kRowsPerThread = 8;
constexpr int kRowsPerSelectBlock = kSelectThreads * kRowsPerThread;
// Radix digits over the 32 key bits: [31:21], [20:10], [9:0].
constexpr int kRadixBins = 2048;
constexpr int kRadixPasses = 3;

enum BucketMode : int32_t { kSelectNone = 0, kSelectAll = 1, kSelectRadix = 2 };

struct BucketDesc {
  int64_t lo, hi;     // rows [lo, hi)
  int64_t k;          // rows to keep, already clamped to [0, hi - lo]
  int64_t out_off;    // first output position of this bucket
  int32_t mode;       // BucketMode
  int32_t first_blk;  // first selection block of this bucket
  int32_t nblk;       // selection blocks of this bucket
  int32_t pad;
};

struct BlockDesc {
  int64_t lo, hi;  // rows [lo, hi), hi - lo <= kRowsPerSelectBlock
  int32_t bucket;
  int32_t pad;
};

// Running radix state of one bucket: the high bits found so far (prefix under
// mask) and how many rows are still to be taken among the rows that share
// them.  After the last pass prefix is the threshold key and kleft the number
// of rows equal to it that are kept.
struct BucketState {
  uint32_t prefix, mask;
  int64_t kleft;
};

struct SelectWorkspace {
  const BucketDesc* buckets;
  const BlockDesc* blocks;
  BucketState* state;
  uint32_t* ghist;      // [nb][kRadixBins], zero between passes
  uint32_t* counter;    // last-block election counter, zero between kernels
  uint32_t* blockcnt;   // [nblk][2]: rows above / equal to the threshold
  uint32_t* blockbase;  // [nblk][2]: exclusive prefix of blockcnt per bucket
  int32_t nb, nblk;
};

// ---- launchers (arc_kernels.hip); each returns hipGetLastError() ----

// Momentum + residual + per-worker sketch over rows [row_lo, row_hi) of
// every worker.  fast != 0 selects the vectorised kernel (requires n % 32 ==
// 0, d % 4 == 0, 16-byte aligned pointers, r in {1,2,4,8}, full rows).
hipError_t launch_sketch(bool fast, const void* grad, int32_t grad_bf16,
                         float* h, const float* g, const float* V, float* S,
                         int64_t d, int64_t n, int64_t m, int32_t N, int32_t r,
                         int64_t row_lo, int64_t row_hi, float eta, float a,
                         hipStream_t stream);

// P = sum_i S[i] (ascending i), sigma = row norm squared of P.  Also resets
// the per-bucket radix state for this step.
hipError_t launch_reduce_importance(const float* S, float* sigma, int64_t m,
                                    int32_t N, int32_t r,
                                    const SelectWorkspace& ws,
                                    hipStream_t stream);

// Per-bucket arg-top-K of sigma into out_idx (ascending per bucket).
hipError_t launch_select(const float* sigma, const SelectWorkspace& ws,
                         int32_t* out_idx, hipStream_t stream);

// Gather of the selected rows, worker sum into agg, g += Delta on them.
hipError_t launch_gather_update(bool fast, const float* h, float* g,
                                const int32_t* idx, float* agg, int64_t K_total,
                                int64_t d, int64_t n, int64_t m, int32_t N,
                                hipStream_t stream);

// ---- host projection (arc_projection.cpp) ----
// V_t (n x r, row-major) for the shared seed and step t.
void generate_projection(uint64_t seed, int64_t t, int64_t n, int32_t r,
                         float* V);

}  // namespace arc
