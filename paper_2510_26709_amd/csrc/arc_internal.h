// Internal declarations shared by the libarctopk host code and its kernels.
#pragma once

#include <condition_variable>
#include <mutex>
#include <thread>
#include <vector>

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace arc {


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

// A group of up to 64 rows of one view, `stride` rows apart (one wave's rows
// in the sketch kernels; the vectorised kernels take groups of 64, 32, 16 or
// 8 rows).  Rows are `cols` wide; local row l starts elem_off + l*stride*cols
// coordinates into each worker's vector and is global row row0 + l*stride;
// their projection is V[v_off .. v_off + cols*r).
struct RowGroup {
  int64_t elem_off;  // coordinate of the group's first element
  int64_t row0;      // global index of the group's first row
  int64_t v_off;     // offset of this width's projection in the V buffer
  int32_t rows;      // 1..64
  int32_t cols;      // row width
  int32_t last_len;  // valid columns of the last row (< cols for a ragged tail)
  int32_t stride;    // rows between local rows: 1, or more in vectorised groups
};

// One tensor (selection bucket) of the per-tensor mode, for the gather.
struct GatherBucket {
  int64_t row0;      // global row of the tensor's first row
  int64_t elem_off;  // coordinate of the tensor's first element
  int64_t out_off;   // first position in out_idx
  int64_t agg_off;   // first element in out_agg
  int64_t work_off;  // first work item (one item = one row x 4 columns)
  int64_t rows;      // rows of the tensor
  int32_t cols;
  int32_t k;         // rows kept
  int32_t vec;       // 16-byte aligned rows and payload: float4 path
  int32_t pad;
};

struct SelectWorkspace {
  const BucketDesc* buckets;
  const BlockDesc* blocks;
  BucketState* state;  // [kRadixPasses][nb]: slot q holds the state after digit q
  uint32_t* hist;      // [kRadixPasses][nb][kRadixBins], zero between steps
  uint32_t* blockcnt;  // [nblk][2]: keys above / equal to the threshold
  int32_t nb, nblk;
  int32_t any_radix;   // some bucket needs the radix passes
  int32_t any_output;  // some bucket selects at least one row
  int32_t small;       // every bucket has at most kSmallBucketRows rows
  int32_t small_rows;  // rows of the largest bucket that needs the radix passes
};

// Buckets of at most this many rows are selected by one workgroup each, in
// one launch for the whole step (no global histograms or block counts), with
// the bucket's keys held in LDS (up to 132 KiB).  Against the five
// multi-block launches, on one MI355X: 22,832 rows (ResNet-18) 9 us less a
// step, the 201 tensors of TinyLlama-1.1B (at most 32,000 rows) 15 us less.
constexpr int kSmallSelectThreads = 1024;
constexpr int kSmallKeysPerThread = 32;
constexpr int64_t kSmallBucketRows = kSmallKeysPerThread * kSmallSelectThreads;
// LDS words that hold r keys: one word of padding after every 32 keys.
constexpr int64_t small_key_words(int64_t r) { return r + r / 32 + 1; }

// ---- launchers; each returns hipGetLastError() ----

// Row groups of group_rows rows take chunks of vector_chunk_cols(group_rows)
// columns in the vectorised sketch kernels.
constexpr int32_t vector_chunk_cols(int32_t group_rows) { return 2048 / group_rows; }

// LDS of one compute unit of the MI355X (gfx950).
constexpr int32_t kLdsPerCu = 160 * 1024;

// Shape of one launch of the vectorised sketch kernels: workgroups of `waves`
// waves (2 or 4, one row group per wave), and, with one_per_cu, a dynamic LDS
// reservation that makes every workgroup hold more than half of a compute
// unit's LDS, so that at most one runs per compute unit.
struct SketchOccupancy {
  int32_t waves;
  int32_t one_per_cu;
};

// Momentum + residual + per-worker sketch into S for the row groups
// groups[0 .. ngroups), any N.  Every group must be vectorisable for
// group_rows in {64, 32, 16, 8}: at most group_rows rows, cols a multiple of
// 4 and at most 2^22, 16-byte aligned rows, r in {1, 2, 4, 8}.
hipError_t launch_sketch_per_worker(int32_t group_rows, const void* grad, int32_t grad_bf16,
                                    float* h, const float* g, const float* V,
                                    const RowGroup* groups, int64_t ngroups, float* S,
                                    int64_t d, int64_t m, int32_t N, int32_t r, float eta,
                                    float a, SketchOccupancy occ, hipStream_t stream);

// The same for any row group (any width, r <= ARC_MAX_R, element alignment,
// ragged last row), one wave per (group, worker).  norm (r = 1): S holds each
// row's squared norm of Delta instead of its sketch.
hipError_t launch_sketch_general(const void* grad, int32_t grad_bf16, float* h,
                                 const float* g, const float* V, const RowGroup* groups,
                                 int64_t ngroups, float* S, int64_t d, int64_t m, int32_t N,
                                 int32_t r, float eta, float a, bool norm, hipStream_t stream);

// Momentum + residual + per-worker squared row norms of Delta into
// norms[N][m] (Top-K), vectorisable groups as for launch_sketch_per_worker.
hipError_t launch_row_norms(int32_t group_rows, const void* grad, int32_t grad_bf16, float* h,
                            const float* g, const float* V, const RowGroup* groups,
                            int64_t ngroups, float* norms, int64_t d, int64_t m, int32_t N,
                            float eta, float a, SketchOccupancy occ, hipStream_t stream);

// ---- comparison compressors (arc_compare.hip) ----

// Eq. (11a) alone over all N*d coordinates (Rand-K needs no residual pass).
hipError_t launch_momentum(bool vec, const void* grad, int32_t grad_bf16, float* h,
                           int64_t count, float eta, float a, hipStream_t stream);

// Rand-K keys of rows [0, m) at step t: (float)(SplitMix64(seed, t*m + p) >> 40).
hipError_t launch_randk_keys(uint64_t seed, int64_t t, int64_t m, float* keys,
                             hipStream_t stream);

// Top-K gather: work item w in [0, N*work) is node w / work's item w % work of
// the bucket table; sel holds the selection over the N*m norms (node i's rows
// offset by i*m).  Writes node i's local rows to out_idx[i*K_total + q], its
// rows of Delta to agg[i*payload + ...] (+0 past d), g^(i) += Delta there.
// With a non-null mark ([N*m]), tags node i's kept row p as
// mark[i*m + p] = stamp << 32 | (its position in the bucket's list).
hipError_t launch_topk_gather(const float* h, float* g, const int32_t* sel, int32_t* out_idx,
                              float* agg, const GatherBucket* buckets, int32_t nb,
                              int64_t work, int64_t K_total, int64_t payload, int64_t d,
                              int64_t m, int32_t N, bool vec, uint64_t* mark, uint32_t stamp,
                              hipStream_t stream);

// Top-K merge after the gather with the same stamp: G += the ascending-node
// sum of the kept values of every kept coordinate.  vec: the gather's
// 16-byte condition holds and G is 16-byte aligned.
hipError_t launch_topk_merge(const float* agg, const int32_t* sel, const uint64_t* mark,
                             uint32_t stamp, const GatherBucket* buckets, int32_t nb,
                             int64_t work, int64_t K_total, int64_t payload, int64_t d,
                             int64_t m, int32_t N, float* G, bool vec, hipStream_t stream);

// p[0 .. n) = 0.
hipError_t launch_zero_u64(uint64_t* p, int64_t n, hipStream_t stream);

// dst[0 .. n) = src[0 .. n), src a device mapping of pinned host memory (the
// projection staging buffer of one step).
hipError_t launch_stage_projection(const float* src, float* dst, int64_t n, hipStream_t stream);

// P = sum_i S[i] (ascending i), sigma = row norm squared of P, for every row
// 0 .. m-1 (one thread per row).
hipError_t launch_reduce_rows(const float* S, float* sigma, int64_t m, int32_t N, int32_t r,
                              hipStream_t stream);

// Per-bucket arg-top-K of sigma into out_idx (ascending per bucket).
hipError_t launch_select(const float* sigma, const SelectWorkspace& ws,
                         int32_t* out_idx, hipStream_t stream);

// Gather of the selected rows, worker sum into agg, g += Delta on them, and
// G += agg there when G is non-null (fast: G 16-byte aligned as well).
hipError_t launch_gather_update(bool fast, const float* h, float* g,
                                const int32_t* idx, float* agg, float* G, int64_t K_total,
                                int64_t d, int64_t n, int64_t m, int32_t N,
                                hipStream_t stream);

// Per-tensor mode gather: buckets[0 .. nb), work items total_work.
hipError_t launch_gather_update_tensors(const float* h, float* g,
                                        const int32_t* idx, float* agg, float* G,
                                        const GatherBucket* buckets, int32_t nb,
                                        int64_t total_work, int64_t d, int32_t N,
                                        bool allow_vec, hipStream_t stream);

// Model step (arc_model.hip).  Dense step: Eq. (11a), (11b) with the identity
// compressor, payload added into G, every coordinate (vec: 16-byte aligned
// pointers and d % 4 == 0).
hipError_t launch_dense_step(bool vec, const void* grad, int32_t grad_bf16, float* h,
                             float* g, float* G, int64_t d, int32_t N, float eta, float a,
                             hipStream_t stream);

// Optimiser constants of one x update (host-computed).
struct OptimizerArgs {
  int32_t kind;        // 0 SGD, 1 MSGD, 2 Adam
  float neg_lr;        // -lr
  float momentum;      // MSGD beta
  float beta1, beta2;  // Adam
  float one_minus_beta1, one_minus_beta2;  // fl(1 - beta)
  float c1, c2;        // Adam bias corrections fl(1 - beta^T)
  float eps, weight_decay;
  float fN;            // number of nodes
};

// x (and m, v) updated from G over every coordinate.  vec: 16-byte aligned
// arrays and d % 4 == 0; cap: the device has the MI355X's 160 KB of LDS per
// compute unit, used to cap the vectorised launch's occupancy.
hipError_t launch_optimizer(bool vec, bool cap, const OptimizerArgs& o, const float* G, float* x,
                            float* m, float* v, int64_t d, hipStream_t stream);

// ---- host projection (arc_projection.cpp) ----
// V_t (n x r, row-major) for the shared seed and step t.
void generate_projection(uint64_t seed, int64_t t, int64_t n, int32_t r,
                         float* V);
// Rows [j0, j1) of the same V_t, written at V[j*r + k].
void generate_projection_rows(uint64_t seed, int64_t t, int64_t n, int32_t r, int64_t j0,
                              int64_t j1, float* V);

// One width's V_t inside a staging buffer: `width` rows of r floats at
// float offset `offset`.
struct ProjectionBlock {
  int64_t width;
  int64_t offset;
};

// Host threads that fill a staging buffer with every width's V_t, so that
// one step's projection can be generated while the device runs the previous
// step.  start() returns at once (after any job still running has ended);
// wait() returns when the last started job is complete.  The blocks and the
// destination must stay valid until then.  One caller at a time.
class ProjectionPool {
 public:
  explicit ProjectionPool(int threads);
  ~ProjectionPool();
  ProjectionPool(const ProjectionPool&) = delete;
  ProjectionPool& operator=(const ProjectionPool&) = delete;
  void start(uint64_t seed, int64_t t, int32_t r, const std::vector<ProjectionBlock>* blocks,
             float* dst);
  void wait();

 private:
  void run(int id, int nthreads);
  std::vector<std::thread> threads_;
  std::mutex mu_;
  std::condition_variable cv_job_, cv_done_;
  uint64_t job_ = 0;
  int remaining_ = 0;
  bool quit_ = false;
  uint64_t seed_ = 0;
  int64_t t_ = 0, total_rows_ = 0;
  int32_t r_ = 0;
  const std::vector<ProjectionBlock>* blocks_ = nullptr;
  float* dst_ = nullptr;
};

}  // namespace arc
