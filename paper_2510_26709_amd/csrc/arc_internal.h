// Internal declarations shared by the libarctopk host code and its kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace arc {

// Workers one block of the fused sketch kernel can hold (one wave each).
constexpr int kMaxFusedWorkers = 8;

// Selection kernels: 256 threads per block; radix digits over the 32 key bits
// [31:21], [20:10], [9:0].
constexpr int kSelectThreads = 256;
constexpr int kRadixBins = 2048;
constexpr int kRadixPasses = 3;
// A selection block covers kSelectThreads * rows_per_thread rows; a bucket
// uses at most kMaxBlocksPerBucket blocks and at least kMinRowsPerThread rows
// per thread.
constexpr int kMinRowsPerThread = 32;
constexpr int kMaxBlocksPerBucket = 256;

enum BucketMode : int32_t { kSelectNone = 0, kSelectAll = 1, kSelectRadix = 2 };

struct BucketDesc {
  int64_t lo, hi;           // rows [lo, hi)
  int64_t k;                // rows to keep, already clamped to [0, hi - lo]
  int64_t out_off;          // first output position of this bucket
  int64_t rows_per_thread;  // rows per selection thread in this bucket
  int32_t mode;             // BucketMode
  int32_t first_blk;        // first selection block of this bucket
  int32_t nblk;             // selection blocks of this bucket
  int32_t pad;
};

struct BlockDesc {
  int64_t lo, hi;  // rows [lo, hi)
  int32_t bucket;
  int32_t pad;
};

// Radix state of one bucket: the high bits fixed so far (prefix under mask)
// and how many rows are still to be taken among the rows that share them.
// After the last digit, prefix is the threshold key and kleft the number of
// rows equal to it that are kept.
struct BucketState {
  uint32_t prefix, mask;
  int64_t kleft;
};

struct SelectWorkspace {
  const BucketDesc* buckets;
  const BlockDesc* blocks;
  BucketState* state;
  uint32_t* hist;      // [kRadixPasses][nb][kRadixBins], zero between steps
  uint32_t* blockcnt;  // [nblk][2]: keys above / equal to the threshold
  int32_t nb, nblk;
  int32_t any_radix;   // some bucket needs the radix passes
  int32_t any_output;  // some bucket selects at least one row
};

// ---- launchers; each returns hipGetLastError() ----

// Bytes of LDS one block of the fused sketch kernel uses for N workers.
size_t fused_sketch_lds_bytes(int32_t N);

// Momentum + residual + per-worker sketch + worker sum + importance over full
// rows [row_lo, row_hi), one block per 64 rows holding all N <= 8 workers.
// Requires n % 32 == 0, d % 4 == 0, 16-byte aligned pointers, r in {1,2,4,8}.
hipError_t launch_sketch_fused(const void* grad, int32_t grad_bf16, float* h,
                               const float* g, const float* V, float* S,
                               float* sigma, int64_t d, int64_t n, int64_t m,
                               int32_t N, int32_t r, int64_t row_lo,
                               int64_t row_hi, float eta, float a,
                               hipStream_t stream);

// Momentum + residual + per-worker sketch into S over rows [row_lo, row_hi).
// fast != 0 selects the vectorised per-worker kernel (same requirements as
// the fused one, any N); otherwise one thread per (row, worker).
hipError_t launch_sketch(bool fast, const void* grad, int32_t grad_bf16,
                         float* h, const float* g, const float* V, float* S,
                         int64_t d, int64_t n, int64_t m, int32_t N, int32_t r,
                         int64_t row_lo, int64_t row_hi, float eta, float a,
                         hipStream_t stream);

// P = sum_i S[i] (ascending i), sigma = row norm squared of P, rows
// [row_lo, row_hi).
hipError_t launch_reduce_importance(const float* S, float* sigma, int64_t m,
                                    int32_t N, int32_t r, int64_t row_lo,
                                    int64_t row_hi, hipStream_t stream);

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
