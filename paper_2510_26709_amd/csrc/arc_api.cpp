// libarctopk C ABI: configuration checks, device workspace, and the per-step
// enqueue of the ARC-Top-K + EF21M pipeline on the caller's HIP stream.
//
// Both layouts the library accepts -- one m x n view of the whole vector
// (Eq. (3)) and one natural 2-D view per tensor -- are lowered at create time
// to the same tables: row groups of up to 64 rows for the sketch kernels,
// selection buckets for the arg-top-K, and (per-tensor mode) gather buckets
// for the variable-width payload.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <map>
#include <memory>
#include <new>
#include <stdexcept>
#include <thread>
#include <string>
#include <vector>

#include "arc_context.h"

namespace {
thread_local std::string g_last_error;
}  // namespace

namespace arc {

arc_status fail(arc_status s, const std::string& why) {
  g_last_error = why;
  return s;
}

arc_status fail_hip(hipError_t e, const char* where) {
  g_last_error = std::string(where) + ": " + hipGetErrorString(e);
  return e == hipErrorOutOfMemory ? ARC_ERR_NOMEM : ARC_ERR_DEVICE;
}

}  // namespace arc

namespace {

using arc::fail;
using arc::fail_hip;

constexpr int64_t kGroupRows = 64;  // rows of one row group (one wave's rows)
constexpr int32_t kMaxTensors = 1 << 24;

bool ranges_overlap(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t pa = reinterpret_cast<uintptr_t>(a);
  const uintptr_t pb = reinterpret_cast<uintptr_t>(b);
  return pa < pb + nb && pb < pa + na;
}

bool aligned16(const void* p) {
  return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}

// r values the vectorised sketch kernels are instantiated for.
bool vector_r(int32_t r) { return r == 1 || r == 2 || r == 4 || r == 8; }

// Rows per group of the vectorised sketch kernels for a view of width cols,
// or 0 when the width needs the general kernel (not a multiple of 4, or a
// group too large for 32-bit byte offsets).  Fewer rows per group give more,
// shorter waves whose rows are read in longer runs (the chunk widens
// instead): the first size whose chunk divides the width, else the one with
// the widest chunk that fits in a row (each row's last chunk is then
// partial).  Measured on one MI355X against a 16-row minimum: ResNet-18
// 0.38 -> 0.35 ms, per-tensor ResNet-18 0.54 -> 0.51 ms, GPT-2 small
// 3.06 -> 3.00 ms (per tensor 3.23 -> 3.17), TinyLlama 11.87 -> 11.60 ms
// (per tensor 12.02 -> 11.70).
// The exception: power-of-two widths from 1024 to 4096 take 16-row groups,
// which with the launch shapes and row spacing below stream 4-9% faster
// than 8-row groups do with theirs (step ms for 1.1·10⁹ bf16 elements, 4
// workers: 1024 values 2.39 vs 2.57, 2048 2.44 vs 2.67, 4096 2.51 vs 2.60);
// at 8192 the two tie and at 16384 8-row groups are 17% faster.
constexpr int32_t kGroupSizes[] = {8, 16, 32, 64};
bool power_of_two(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }
int32_t vector_group_rows(int64_t cols) {
  if (cols > (int64_t{1} << 22) || cols % 4 != 0) return 0;
  if (power_of_two(cols) && cols >= 1024 && cols <= 4096) return 16;
  for (int32_t gr : kGroupSizes)
    if (cols % arc::vector_chunk_cols(gr) == 0) return gr;
  for (int32_t gr : kGroupSizes)
    if (cols >= arc::vector_chunk_cols(gr)) return gr;
  return 64;
}

}  // namespace


namespace {

// Per-tensor checks; m_out receives the total number of rows.
arc_status check_tensors(const arc_config* cfg, int64_t* m_out) {
  if (cfg->num_tensors > kMaxTensors) return fail(ARC_ERR_INVALID, "num_tensors exceeds 2^24");
  if (cfg->tensors == nullptr) return fail(ARC_ERR_INVALID, "tensors is NULL");
  if (cfg->n != 0 || cfg->K != 0 || cfg->num_buckets != 0)
    return fail(ARC_ERR_INVALID, "per-tensor mode needs n == 0, K == 0 and num_buckets == 0");
  int64_t covered = 0, m = 0;
  for (int32_t b = 0; b < cfg->num_tensors; ++b) {
    const arc_tensor& t = cfg->tensors[b];
    if (t.rows < 1 || t.cols < 1 || t.K < 0)
      return fail(ARC_ERR_INVALID, "tensor rows and cols must be >= 1 and K >= 0");
    if (t.cols > INT32_MAX) return fail(ARC_ERR_INVALID, "tensor cols must be < 2^31");
    if (t.rows > (cfg->d - covered) / t.cols)
      return fail(ARC_ERR_INVALID, "tensors cover more than d coordinates");
    covered += t.rows * t.cols;
    m += t.rows;
  }
  if (covered != cfg->d) return fail(ARC_ERR_INVALID, "tensors must cover exactly d coordinates");
  if (m > INT32_MAX) return fail(ARC_ERR_INVALID, "total rows exceed 2^31-1");
  *m_out = m;
  return ARC_OK;
}

}  // namespace

namespace arc {

namespace {

// The checks of everything but the compressor's own bounds.
arc_status check_problem(const arc_config* cfg, int64_t* m_out) {
  if (cfg == nullptr) return fail(ARC_ERR_INVALID, "cfg is NULL");
  if (cfg->d <= 0) return fail(ARC_ERR_INVALID, "d must be > 0");
  if (cfg->N <= 0 || cfg->N > 65535) return fail(ARC_ERR_INVALID, "N must be in 1..65535");
  if (cfg->r <= 0 || cfg->r > ARC_MAX_R) return fail(ARC_ERR_INVALID, "r must be in 1..ARC_MAX_R");
  if (cfg->grad_dtype != ARC_DTYPE_F32 && cfg->grad_dtype != ARC_DTYPE_BF16)
    return fail(ARC_ERR_INVALID, "grad_dtype must be ARC_DTYPE_F32 or ARC_DTYPE_BF16");
  if (!(cfg->eta >= 0.0f && cfg->eta <= 1.0f)) return fail(ARC_ERR_INVALID, "eta must be in [0, 1]");
  if (cfg->reserved != 0) return fail(ARC_ERR_INVALID, "reserved must be 0");
  if (cfg->compressor < ARC_COMP_ARC || cfg->compressor > ARC_COMP_TOPK)
    return fail(ARC_ERR_INVALID, "compressor must be ARC_COMP_ARC, ARC_COMP_RANDK or ARC_COMP_TOPK");
  if (cfg->d > INT64_MAX / cfg->N) return fail(ARC_ERR_INVALID, "N*d overflows");
  if (cfg->num_tensors < 0) return fail(ARC_ERR_INVALID, "num_tensors must be >= 0");
  if (cfg->num_tensors > 0) return check_tensors(cfg, m_out);
  if (cfg->n <= 0) return fail(ARC_ERR_INVALID, "n must be > 0");
  if (cfg->n > INT32_MAX) return fail(ARC_ERR_INVALID, "n must be < 2^31");
  const int64_t m = cfg->d / cfg->n + (cfg->d % cfg->n != 0);
  if (m > INT32_MAX) return fail(ARC_ERR_INVALID, "m = ceil(d/n) exceeds 2^31-1");
  if (cfg->num_buckets < 0) return fail(ARC_ERR_INVALID, "num_buckets must be >= 0");
  if (cfg->num_buckets == 0) {
    if (cfg->K < 0) return fail(ARC_ERR_INVALID, "K must be >= 0");
  } else {
    if (cfg->bucket_row_begin == nullptr || cfg->bucket_K == nullptr)
      return fail(ARC_ERR_INVALID, "bucket arrays are NULL");
    if (cfg->bucket_row_begin[0] != 0 || cfg->bucket_row_begin[cfg->num_buckets] != m)
      return fail(ARC_ERR_INVALID, "buckets must cover rows [0, m)");
    for (int32_t b = 0; b < cfg->num_buckets; ++b) {
      if (cfg->bucket_row_begin[b + 1] <= cfg->bucket_row_begin[b])
        return fail(ARC_ERR_INVALID, "bucket_row_begin must be strictly increasing");
      if (cfg->bucket_K[b] < 0) return fail(ARC_ERR_INVALID, "bucket_K must be >= 0");
    }
  }
  *m_out = m;
  return ARC_OK;
}

}  // namespace

// Configuration checks shared by the entry points; no HIP call is made here.
arc_status check_config(const arc_config* cfg, int64_t* m_out) {
  const arc_status st = check_problem(cfg, m_out);
  if (st != ARC_OK) return st;
  if (cfg->compressor == ARC_COMP_TOPK && *m_out > INT32_MAX / cfg->N)
    return fail(ARC_ERR_INVALID, "Top-K: N * m must be below 2^31");
  return ARC_OK;
}

}  // namespace arc

namespace {

// Selection buckets from row boundaries begin[0..nb] and requested K's.
// Fat blocks (few blocks per bucket keep the per-bin atomics and the
// block-prefix sums short), at most kMaxBlocksPerBucket of them per bucket.
void build_selection_plan(const std::vector<int64_t>& begin, const std::vector<int64_t>& want,
                          arc_ctx* c) {
  int64_t out = 0;
  for (size_t b = 0; b < want.size(); ++b) {
    arc::BucketDesc bd{};
    bd.lo = begin[b];
    bd.hi = begin[b + 1];
    const int64_t rows = bd.hi - bd.lo;
    bd.k = want[b] < rows ? want[b] : rows;
    bd.out_off = out;
    bd.mode = bd.k == 0 ? arc::kSelectNone : bd.k == rows ? arc::kSelectAll : arc::kSelectRadix;
    const int64_t per_block_cap = (int64_t)arc::kSelectThreads * arc::kMaxBlocksPerBucket;
    int64_t rpt = (rows + per_block_cap - 1) / per_block_cap;
    if (rpt < arc::kMinRowsPerThread) rpt = arc::kMinRowsPerThread;
    const int64_t rows_per_block = rpt * arc::kSelectThreads;
    bd.rows_per_thread = rpt;
    bd.first_blk = static_cast<int32_t>(c->blocks.size());
    for (int64_t lo = bd.lo; lo < bd.hi; lo += rows_per_block) {
      arc::BlockDesc blk{};
      blk.lo = lo;
      blk.hi = lo + rows_per_block < bd.hi ? lo + rows_per_block : bd.hi;
      blk.bucket = static_cast<int32_t>(b);
      c->blocks.push_back(blk);
    }
    bd.nblk = static_cast<int32_t>(c->blocks.size()) - bd.first_blk;
    out += bd.k;
    c->buckets.push_back(bd);
  }
  c->K_total = out;
}

struct GroupLists {
  std::vector<arc::RowGroup> vec[4], general;  // vec: 64, 32, 16, 8 rows
};

int size_slot(int32_t group_rows) {
  return group_rows == 64 ? 0 : group_rows == 32 ? 1 : group_rows == 16 ? 2 : 3;
}

// Occupancy of one vectorised sketch launch from its groups' mean number of
// chunks per row (weighted by coordinates).  A wave streams one chunk while
// its chains run over the previous one; fewer waves per compute unit keep
// fewer DRAM rows open at once, which the stage gains from as long as each
// wave has enough chunks to keep its loads ahead of its chains.  Measured on
// one MI355X (step ms, 4-wave workgroups at 3 per CU / 4 waves per CU /
// 2 waves per CU): 2048-wide rows in 16-row groups (16 chunks) 11.37 / 10.69
// / 10.09; 4096-wide in 8-row groups (16 chunks) 33.97 / 32.03 / 31.15;
// 768-wide in 8-row groups (3 chunks) 2.88 / 2.76 / 2.93; 512-wide (2
// chunks) 0.350 / 0.345 / 0.370; 256-wide (one chunk, a 50 MB working set)
// 0.047 / 0.049 / 0.053.  16-row groups, whose chunks are half as wide,
// gain from 2 waves from 6 chunks on (768 values: 2.73 vs 2.78 ms; 1024:
// 2.42 vs 2.49 ms at 1.1·10⁹ elements), 8-row groups from 9 (2048 values:
// 10.67 vs 10.39 ms on the 1.1B workload, 2304: 2.82 vs 2.89 ms).
int32_t two_wave_chunks(int32_t group_rows) { return group_rows == 16 ? 6 : 9; }
constexpr double kChunkSlack = 0.01;
arc::SketchOccupancy sketch_occupancy(const std::vector<arc::RowGroup>& groups,
                                      int32_t group_rows) {
  double elems = 0.0, weighted = 0.0;
  const int64_t cw = arc::vector_chunk_cols(group_rows);
  for (const arc::RowGroup& grp : groups) {
    const double e = static_cast<double>(grp.rows) * grp.cols;
    elems += e;
    weighted += e * static_cast<double>((grp.cols + cw - 1) / cw);
  }
  // A short tail row (a view's last, ragged row) must not pull a layout of
  // whole rows below a threshold: ResNet-18's 22,832 rows of 512 values end
  // with one of 40, which put the mean at 1.99998 chunks and the launch at
  // the hardware's occupancy (stage 0.290 ms, 0.286 ms with one workgroup
  // per compute unit).
  const double chunks = (elems > 0.0 ? weighted / elems : 0.0) + kChunkSlack;
  if (chunks >= two_wave_chunks(group_rows)) return {2, 1};
  if (chunks >= 2.0) return {4, 1};
  return {4, 0};
}

// Rows between the local rows of a full vectorised group.  A wave streams
// its rows a chunk at a time, one short run per row; with its rows S apart,
// the runs of the S groups of a block (next to each other in the launch)
// interleave in memory.  Power-of-two widths do best with a group's rows
// 32 KiB apart (S = 8192 / width, 1 from 8192 on: step ms for 1.1·10⁹ bf16
// elements, 4 workers, rows 1 / 2 / 4 / 8 apart: 1024 values 2.60 / 2.48 /
// 2.42 / 2.39; 2048 2.54 / 2.47 / 2.44 / -; 4096 2.55 / 2.51 / 2.89 / 2.87;
// 8192 with 8-row groups 2.51 / 2.55 / 2.79 / 2.80).  Other widths take rows
// 4 apart (3072 values 2.77 vs 2.70 ms; 2304 and 5632 unchanged).  Rows of
// too few chunks for two waves stay consecutive (768 values: equal; 512: 1-2%
// slower apart).  Strided groups span at most 2^30 bytes.
constexpr int64_t kPowerOfTwoRowBytes = 32 * 1024;
constexpr int32_t kRowInterleave = 4;
int32_t row_interleave(int64_t cols, int32_t group_rows) {
  const int64_t cw = arc::vector_chunk_cols(group_rows);
  if ((cols + cw - 1) / cw < two_wave_chunks(group_rows)) return 1;
  int64_t S = kRowInterleave;
  if (power_of_two(cols)) S = std::max<int64_t>(1, kPowerOfTwoRowBytes / (cols * 4));
  const int64_t span = ((group_rows - 1) * S + 1) * cols * 4;
  return span <= (int64_t{1} << 30) ? static_cast<int32_t>(S) : 1;
}

// Row groups over `rows` rows of width `cols` that start at coordinate
// elem_off and global row row0; the last row holds last_len <= cols values.
// group_rows > 0: vectorisable groups of that many rows (the view has no
// ragged row); 0: general groups of 64 rows.
// Vectorised groups take every S-th row of a block of S*G consecutive rows
// (S groups per block), the rest consecutive rows.
void add_groups(int64_t elem_off, int64_t row0, int64_t rows, int64_t cols, int64_t last_len,
                int64_t v_off, int32_t group_rows, GroupLists* out) {
  const int64_t step = group_rows > 0 ? group_rows : kGroupRows;
  auto push = [&](int64_t p, int64_t nrows, int32_t stride) {
    arc::RowGroup grp{};
    grp.elem_off = elem_off + p * cols;
    grp.row0 = row0 + p;
    grp.v_off = v_off;
    grp.rows = static_cast<int32_t>(nrows);
    grp.cols = static_cast<int32_t>(cols);
    grp.last_len = static_cast<int32_t>(p + (nrows - 1) * stride == rows - 1 ? last_len : cols);
    grp.stride = stride;
    (group_rows > 0 ? out->vec[size_slot(group_rows)] : out->general).push_back(grp);
  };
  int64_t p = 0;
  const int32_t S = group_rows > 0 ? row_interleave(cols, group_rows) : 1;
  if (S > 1)
    for (; p + S * step <= rows; p += S * step)
      for (int32_t ph = 0; ph < S; ++ph) push(p + ph, step, S);
  for (; p < rows; p += step) push(p, rows - p < step ? rows - p : step, 1);
}


// Selection buckets of one node's view (begin[0..nb], want[0..nb)).  Top-K
// selects for every node separately over the N*m norms: node i's copies of
// the buckets are offset by i*m rows.
void build_node_selection(const std::vector<int64_t>& begin, const std::vector<int64_t>& want,
                          arc_ctx* c) {
  if (c->compressor != ARC_COMP_TOPK) {
    build_selection_plan(begin, want, c);
    c->K_node = c->K_total;
    return;
  }
  std::vector<int64_t> all_begin{0}, all_want;
  for (int32_t i = 0; i < c->N; ++i)
    for (size_t b = 0; b + 1 < begin.size(); ++b) {
      all_begin.push_back(static_cast<int64_t>(i) * c->m + begin[b + 1]);
      all_want.push_back(want[b]);
    }
  build_selection_plan(all_begin, all_want, c);
  c->K_node = c->K_total / c->N;
}

// Lowers the configuration to the kernels' tables (host side only).
void build_plan(const arc_config* cfg, arc_ctx* c) {
  GroupLists lists;
  std::vector<int64_t> begin{0}, want;
  // r in {1,2,4,8} for the vectorised sketch; the other compressors use no V.
  const bool r_ok = c->compressor != ARC_COMP_ARC || vector_r(c->r);
  if (!c->tensor_mode) {
    // One m x n view (Eq. (3)); rows [0, m_full) are whole, row m_full (if
    // any) holds the d - m_full*n remaining coordinates.
    c->widths.push_back(c->n);
    c->v_off[c->n] = 0;
    c->v_floats = c->n * c->r;
    const int64_t m_full = c->d / c->n;
    const int32_t gr = c->d % 4 == 0 && r_ok ? vector_group_rows(c->n) : 0;
    if (gr > 0) {
      add_groups(0, 0, m_full, c->n, c->n, 0, gr, &lists);
      // The ragged row (a multiple of 4 values, as d and n are) is a
      // one-row group as wide as its values.
      const int64_t tail = c->d - m_full * c->n;
      if (tail > 0) add_groups(m_full * c->n, m_full, 1, tail, tail, 0, gr, &lists);
    } else {
      add_groups(0, 0, c->m, c->n, c->d - (c->m - 1) * c->n, 0, 0, &lists);
    }
    if (cfg->num_buckets == 0) {
      begin.push_back(c->m);
      want.push_back(cfg->K);
    } else {
      for (int32_t b = 0; b < cfg->num_buckets; ++b) {
        begin.push_back(cfg->bucket_row_begin[b + 1]);
        want.push_back(cfg->bucket_K[b]);
      }
    }
    build_node_selection(begin, want, c);
    c->payload_node = c->K_node * c->n;
    // Top-K gathers each node's rows through bucket tables (both layouts).
    int64_t work = 0;
    for (size_t b = 0; b + 1 < begin.size(); ++b) {
      const arc::BucketDesc& bd = c->buckets[b];
      arc::GatherBucket gb{};
      gb.row0 = bd.lo;
      gb.elem_off = bd.lo * c->n;
      gb.out_off = bd.out_off;
      gb.agg_off = bd.out_off * c->n;
      gb.work_off = work;
      gb.rows = bd.hi - bd.lo;
      gb.cols = static_cast<int32_t>(c->n);
      gb.k = static_cast<int32_t>(bd.k);
      gb.vec = c->n % 4 == 0 && c->d % 4 == 0;
      if (c->compressor == ARC_COMP_TOPK) c->gather.push_back(gb);
      work += bd.k * ((c->n + 3) / 4);
    }
    c->gather_work = c->compressor == ARC_COMP_TOPK ? work : 0;
  } else {
    // One view per tensor; tensors of equal width share one V_t.
    for (int32_t b = 0; b < cfg->num_tensors; ++b) {
      const int64_t w = cfg->tensors[b].cols;
      if (c->v_off.emplace(w, c->v_floats).second) {
        c->widths.push_back(w);
        c->v_floats += w * c->r;
      }
    }
    int64_t off = 0, row0 = 0;
    for (int32_t b = 0; b < cfg->num_tensors; ++b) {
      const arc_tensor& t = cfg->tensors[b];
      const int32_t gr = off % 4 == 0 && c->d % 4 == 0 && r_ok ? vector_group_rows(t.cols) : 0;
      add_groups(off, row0, t.rows, t.cols, t.cols, c->v_off[t.cols], gr, &lists);
      off += t.rows * t.cols;
      row0 += t.rows;
      begin.push_back(row0);
      want.push_back(t.K);
    }
    build_node_selection(begin, want, c);
    int64_t agg_off = 0, work = 0;
    off = 0;
    for (int32_t b = 0; b < cfg->num_tensors; ++b) {
      const arc_tensor& t = cfg->tensors[b];
      const arc::BucketDesc& bd = c->buckets[b];
      arc::GatherBucket gb{};
      gb.row0 = bd.lo;
      gb.elem_off = off;
      gb.out_off = bd.out_off;
      gb.agg_off = agg_off;
      gb.work_off = work;
      gb.rows = t.rows;
      gb.cols = static_cast<int32_t>(t.cols);
      gb.k = static_cast<int32_t>(bd.k);
      gb.vec = t.cols % 4 == 0 && off % 4 == 0 && agg_off % 4 == 0 && c->d % 4 == 0;
      c->gather.push_back(gb);
      agg_off += bd.k * t.cols;
      work += bd.k * ((t.cols + 3) / 4);
      off += t.rows * t.cols;
    }
    c->payload_node = agg_off;
    c->gather_work = work;
  }
  const int64_t nodes = c->compressor == ARC_COMP_TOPK ? c->N : 1;
  c->payload = nodes * c->payload_node;
  c->groups.clear();
  for (int sz = 0; sz < 4; ++sz) {
    c->vec_count[sz] = static_cast<int64_t>(lists.vec[sz].size());
    c->vec_occ[sz] = sketch_occupancy(lists.vec[sz], 64 >> sz);
    for (const arc::RowGroup& grp : lists.vec[sz])
      c->stage_elems[sz] += (grp.rows - 1) * static_cast<int64_t>(grp.cols) + grp.last_len;
    c->groups.insert(c->groups.end(), lists.vec[sz].begin(), lists.vec[sz].end());
  }
  c->nvec_groups = static_cast<int64_t>(c->groups.size());
  c->groups.insert(c->groups.end(), lists.general.begin(), lists.general.end());
  for (const arc::RowGroup& grp : lists.general)
    c->stage_elems[4] += (grp.rows - 1) * static_cast<int64_t>(grp.cols) + grp.last_len;
}

template <typename T>
arc_status dev_alloc(T** p, size_t count, const char* what) {
  if (count == 0) count = 1;
  const hipError_t e = hipMalloc(reinterpret_cast<void**>(p), count * sizeof(T));
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    return fail_hip(e, what);
  }
  return ARC_OK;
}

template <typename T>
hipError_t upload(T* dst, const std::vector<T>& src) {
  if (src.empty()) return hipSuccess;
  return hipMemcpy(dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice);
}

arc_status record(arc_ctx* c, size_t slot, int which) {
  if (!c->timing) return ARC_OK;
  ARC_HIP(hipEventRecord(c->ev_pool[slot][which], c->stream), "hipEventRecord");
  return ARC_OK;
}

// Host threads for the projection: one per 8K values (a few hundred
// microseconds of Box-Muller each, well under a step of the device), at most
// 8 and at most half the cores.
int projection_threads(int64_t v_floats) {
  const int64_t by_size = 1 + v_floats / 8192;
  const int64_t cores = static_cast<int64_t>(std::thread::hardware_concurrency());
  const int64_t cap = std::max<int64_t>(1, std::min<int64_t>(8, cores / 2));
  return static_cast<int>(std::min(by_size, cap));
}

// Waits until the device has read pinned slot s (its last staging kernel is
// done).
arc_status release_slot(arc_ctx* c, int s) {
  if (c->V_pending[s]) {
    ARC_HIP(hipEventSynchronize(c->V_done[s]), "hipEventSynchronize(projection)");
    c->V_pending[s] = false;
  }
  return ARC_OK;
}

// Pinned staging of this step's projections and the kernel that moves them
// into V on the stream.  Once that is queued, the pool starts on V_{t+1} in
// the next slot of the ring, so that a caller stepping t, t+1, ... finds the
// next projection ready; any other t is generated on the spot.  A slot is
// refilled only after the staging kernel that last read it
// (kProjectionSlots - 1 calls earlier) has completed.
arc_status upload_projection(arc_ctx* c, int64_t t) {
  const int s = c->V_slot;
  const int next = (s + 1) % arc::kProjectionSlots;
  c->V_slot = next;
  c->V_pool->wait();
  const bool ready = !c->use_override && c->V_prefetch_t == t;
  c->V_prefetch_t = -1;
  arc_status st;
  if (!ready) {
    if ((st = release_slot(c, s))) return st;
    if (c->use_override) {
      std::memcpy(c->V_pinned[s], c->V_override.data(), c->V_override.size() * sizeof(float));
    } else {
      c->V_pool->start(c->seed, t, c->r, &c->V_blocks, c->V_pinned[s]);
      c->V_pool->wait();
    }
  }
  // A kernel reads the pinned buffer through its device mapping: with the
  // host queueing steps ahead, the runtime's copy of a pinned buffer stalled
  // the calling thread for 11-12 ms every eighth or ninth step (per-tensor
  // ResNet-18, four buffers in the ring), which this does not.
  ARC_HIP(arc::launch_stage_projection(c->V_pinned_dev[s], c->V_dev, c->v_floats, c->stream),
          "projection staging launch");
  ARC_HIP(hipEventRecord(c->V_done[s], c->stream), "hipEventRecord(projection)");
  c->V_pending[s] = true;
  if (!c->use_override && t < INT64_MAX) {
    if ((st = release_slot(c, next))) return st;
    c->V_pool->start(c->seed, t + 1, c->r, &c->V_blocks, c->V_pinned[next]);
    c->V_prefetch_t = t + 1;
  }
  return ARC_OK;
}

}  // namespace

extern "C" {

const char* arc_status_str(arc_status s) {
  switch (s) {
    case ARC_OK: return "ARC_OK";
    case ARC_ERR_INVALID: return "ARC_ERR_INVALID";
    case ARC_ERR_NOMEM: return "ARC_ERR_NOMEM";
    case ARC_ERR_DEVICE: return "ARC_ERR_DEVICE";
    case ARC_ERR_UNSUPPORTED: return "ARC_ERR_UNSUPPORTED";
  }
  return "ARC_ERR_UNKNOWN";
}

const char* arc_last_error(void) { return g_last_error.c_str(); }

arc_status arc_projection(uint64_t seed, int64_t t, int64_t n, int32_t r, float* V) {
  if (V == nullptr) return fail(ARC_ERR_INVALID, "V is NULL");
  if (t < 0) return fail(ARC_ERR_INVALID, "t must be >= 0");
  if (n < 1) return fail(ARC_ERR_INVALID, "n must be >= 1");
  if (r < 1 || r > ARC_MAX_R) return fail(ARC_ERR_INVALID, "r must be in 1..ARC_MAX_R");
  arc::generate_projection(seed, t, n, r, V);
  return ARC_OK;
}

arc_status arc_create(const arc_config* cfg, void* hip_stream, arc_ctx** out) {
  if (out == nullptr) return fail(ARC_ERR_INVALID, "out is NULL");
  *out = nullptr;
  int64_t m = 0;
  arc_status st = arc::check_config(cfg, &m);
  if (st != ARC_OK) return st;

  arc_ctx* c = new (std::nothrow) arc_ctx();
  if (c == nullptr) return fail(ARC_ERR_NOMEM, "host allocation failed");
  st = arc::plan_context(cfg, m, hip_stream, c);
  if (st != ARC_OK) {
    delete c;
    return st;
  }

  auto bail = [&](arc_status s) {
    c->release();
    delete c;
    return s;
  };
  if ((st = arc::bind_device(c)) != ARC_OK) return bail(st);
  hipError_t e;

  const size_t nb = c->buckets.size(), nblk = c->blocks.size();
  if ((st = dev_alloc(&c->V_dev, static_cast<size_t>(c->v_floats), "hipMalloc(V)")) ||
      (st = dev_alloc(&c->S_dev, static_cast<size_t>(c->N) * c->m * c->r, "hipMalloc(S)")) ||
      (st = dev_alloc(&c->sigma_dev, static_cast<size_t>(c->m), "hipMalloc(sigma)")) ||
      (st = dev_alloc(&c->groups_dev, c->groups.size(), "hipMalloc(groups)")) ||
      (st = dev_alloc(&c->gather_dev, c->gather.size(), "hipMalloc(gather)")) ||
      (st = dev_alloc(&c->buckets_dev, nb, "hipMalloc(buckets)")) ||
      (st = dev_alloc(&c->blocks_dev, nblk, "hipMalloc(blocks)")) ||
      (st = dev_alloc(&c->state_dev, arc::kRadixPasses * nb, "hipMalloc(state)")) ||
      (st = dev_alloc(&c->hist_dev, arc::kRadixPasses * nb * arc::kRadixBins,
                      "hipMalloc(hist)")) ||
      (st = dev_alloc(&c->blockcnt_dev, 2 * nblk, "hipMalloc(blockcnt)")) ||
      (st = dev_alloc(&c->sel_dev, c->compressor == ARC_COMP_TOPK ? c->K_total : 0,
                      "hipMalloc(selection)")) ||
      (st = dev_alloc(&c->mark_dev,
                      c->compressor == ARC_COMP_TOPK ? static_cast<size_t>(c->N) * c->m : 0,
                      "hipMalloc(merge tags)")))
    return bail(st);
  for (int s = 0; s < arc::kProjectionSlots; ++s) {
    // Coherent and mapped: the staging kernel reads it from the device, and
    // every step rewrites it, so the device must not keep stale copies.
    e = hipHostMalloc(reinterpret_cast<void**>(&c->V_pinned[s]),
                      static_cast<size_t>(std::max<int64_t>(c->v_floats, 1)) * sizeof(float),
                      hipHostMallocMapped | hipHostMallocCoherent);
    if (e != hipSuccess) {
      c->V_pinned[s] = nullptr;
      return bail(fail_hip(e, "hipHostMalloc(projection)"));
    }
    e = hipHostGetDevicePointer(reinterpret_cast<void**>(&c->V_pinned_dev[s]), c->V_pinned[s], 0);
    if (e != hipSuccess) return bail(fail_hip(e, "hipHostGetDevicePointer(projection)"));
    e = hipEventCreateWithFlags(&c->V_done[s], hipEventDisableTiming);
    if (e != hipSuccess) {
      c->V_done[s] = nullptr;
      return bail(fail_hip(e, "hipEventCreate"));
    }
  }
  if (c->compressor == ARC_COMP_ARC) {
    for (int64_t w : c->widths) c->V_blocks.push_back({w, c->v_off[w]});
    try {
      c->V_pool.reset(new arc::ProjectionPool(projection_threads(c->v_floats)));
    } catch (const std::exception&) {
      return bail(fail(ARC_ERR_NOMEM, "cannot start the projection threads"));
    }
  }
  {
    int launches = c->stage_elems[4] > 0 ? 1 : 0;
    for (int sz = 0; sz < 4; ++sz) launches += c->vec_count[sz] > 0;
    if (launches > 1) {
      e = hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking);
      for (int k = 0; k < arc::kProjectionSlots && e == hipSuccess; ++k) {
        e = hipEventCreateWithFlags(&c->fork_ev[k], hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&c->join_ev[k], hipEventDisableTiming);
      }
      if (e != hipSuccess) return bail(fail_hip(e, "hipStreamCreate(side)"));
    }
  }
  // Constant tables, and zeroed radix scratch (kept zero between uses by the
  // kernels themselves).
  e = upload(c->buckets_dev, c->buckets);
  if (e == hipSuccess) e = upload(c->blocks_dev, c->blocks);
  if (e == hipSuccess) e = upload(c->groups_dev, c->groups);
  if (e == hipSuccess) e = upload(c->gather_dev, c->gather);
  if (e == hipSuccess)
    e = hipMemset(c->hist_dev, 0, arc::kRadixPasses * nb * arc::kRadixBins * sizeof(uint32_t));
  if (e == hipSuccess && c->compressor == ARC_COMP_TOPK)
    e = hipMemset(c->mark_dev, 0, static_cast<size_t>(c->N) * c->m * sizeof(uint64_t));
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) return bail(fail_hip(e, "workspace initialisation"));
  *out = c;
  return ARC_OK;
}

arc_status arc_destroy(arc_ctx* ctx) {
  if (ctx == nullptr) return ARC_OK;
  ctx->release();
  delete ctx;
  return ARC_OK;
}

int64_t arc_num_rows(const arc_ctx* ctx) { return ctx ? ctx->m : -1; }

int64_t arc_selected_rows(const arc_ctx* ctx) { return ctx ? ctx->K_total : -1; }

int64_t arc_payload_elems(const arc_ctx* ctx) { return ctx ? ctx->payload : -1; }

}  // extern "C"

namespace arc {

// need_outputs: the call writes out_idx / out_agg (every compressed step).
arc_status check_step_args(const arc_ctx* c, int64_t t, const void* grad, const float* h,
                           const float* g, const int32_t* out_idx, const float* out_agg,
                           bool need_outputs) {
  if (c == nullptr) return fail(ARC_ERR_INVALID, "ctx is NULL");
  if (t < 0) return fail(ARC_ERR_INVALID, "t must be >= 0");
  if (grad == nullptr || h == nullptr || g == nullptr)
    return fail(ARC_ERR_INVALID, "grad, h and g must be non-NULL");
  if (need_outputs && c->K_total > 0 && (out_idx == nullptr || out_agg == nullptr))
    return fail(ARC_ERR_INVALID, "out_idx and out_agg must be non-NULL");
  const size_t elems = static_cast<size_t>(c->N) * static_cast<size_t>(c->d);
  const size_t grad_bytes = elems * (c->grad_bf16 ? 2 : 4), state_bytes = elems * 4;
  if (ranges_overlap(grad, grad_bytes, h, state_bytes) ||
      ranges_overlap(grad, grad_bytes, g, state_bytes) ||
      ranges_overlap(h, state_bytes, g, state_bytes))
    return fail(ARC_ERR_INVALID, "grad, h and g must not overlap");
  if (need_outputs && c->K_total > 0) {
    // The gather writes out_agg while it reads h and g of other rows, and
    // out_idx is read back after the selection wrote it: an alias would
    // corrupt the state or the payload without an error.
    const size_t idx_bytes = static_cast<size_t>(c->K_total) * sizeof(int32_t);
    const size_t agg_bytes = static_cast<size_t>(c->payload) * sizeof(float);
    if (ranges_overlap(out_idx, idx_bytes, out_agg, agg_bytes))
      return fail(ARC_ERR_INVALID, "out_idx and out_agg must not overlap");
    const void* in[3] = {grad, h, g};
    const size_t in_bytes[3] = {grad_bytes, state_bytes, state_bytes};
    for (int k = 0; k < 3; ++k)
      if (ranges_overlap(out_idx, idx_bytes, in[k], in_bytes[k]) ||
          ranges_overlap(out_agg, agg_bytes, in[k], in_bytes[k]))
        return fail(ARC_ERR_INVALID, "out_idx and out_agg must not overlap grad, h or g");
  }
  return ARC_OK;
}

}  // namespace arc

namespace {

// The streaming stage (S1-S3; norm: Top-K's row norms): one launch per
// row-group size present and one for the general groups.  When there are several, the one over the most coordinates runs on
// the caller's stream and the others on the second stream, forked after
// everything queued before and joined before anything queued after, so that
// they overlap it instead of following it.
arc_status launch_streaming_stage(arc_ctx* c, const void* grad, float* h, const float* g,
                                  int64_t nvec, int64_t ngroups, bool norm) {
  int which[5], nl = 0, big = 0;
  for (int sz = 0; sz < 4; ++sz)
    if (nvec > 0 && c->vec_count[sz] > 0) which[nl++] = sz;
  if (ngroups > nvec) which[nl++] = 4;
  // With misaligned pointers every group is general: one launch.
  const auto elems = [&](int w) {
    if (w < 4) return c->stage_elems[w];
    return nvec > 0 ? c->stage_elems[4] : c->m;  // m stands in for "all of them"
  };
  for (int l = 1; l < nl; ++l)
    if (elems(which[l]) > elems(which[big])) big = l;
  const bool fork = nl > 1 && c->side != nullptr;
  if (fork) {
    c->fork_slot = (c->fork_slot + 1) % arc::kProjectionSlots;
    ARC_HIP(hipEventRecord(c->fork_ev[c->fork_slot], c->stream), "hipEventRecord(fork)");
    ARC_HIP(hipStreamWaitEvent(c->side, c->fork_ev[c->fork_slot], 0), "hipStreamWaitEvent(fork)");
  }
  // The smaller launches go first, so that they start while the largest
  // fills the rest of the device.
  for (int pass = 0; pass < 2; ++pass) {
    for (int l = 0; l < nl; ++l) {
      if ((l == big) != (pass == 1)) continue;
      hipStream_t s = fork && l != big ? c->side : c->stream;
      const int w = which[l];
      if (w == 4) {
        ARC_HIP(arc::launch_sketch_general(grad, c->grad_bf16, h, g, c->V_dev,
                                           c->groups_dev + nvec, ngroups - nvec, c->S_dev, c->d,
                                           c->m, c->N, norm ? 1 : c->r, c->eta, c->a, norm, s),
                norm ? "row norm launch (general rows)" : "sketch launch (general rows)");
        continue;
      }
      int64_t first = 0;
      for (int sz = 0; sz < w; ++sz) first += c->vec_count[sz];
      const int32_t gr = 64 >> w;
      const arc::RowGroup* grp = c->groups_dev + first;
      if (norm) {
        ARC_HIP(arc::launch_row_norms(gr, grad, c->grad_bf16, h, g, c->V_dev, grp,
                                      c->vec_count[w], c->S_dev, c->d, c->m, c->N, c->eta, c->a,
                                      c->vec_occ[w], s),
                "row norm launch");
      } else {
        ARC_HIP(arc::launch_sketch_per_worker(gr, grad, c->grad_bf16, h, g, c->V_dev, grp,
                                              c->vec_count[w], c->S_dev, c->d, c->m, c->N,
                                              c->r, c->eta, c->a, c->vec_occ[w], s),
                "sketch launch");
      }
    }
  }
  if (fork) {
    ARC_HIP(hipEventRecord(c->join_ev[c->fork_slot], c->side), "hipEventRecord(join)");
    ARC_HIP(hipStreamWaitEvent(c->stream, c->join_ev[c->fork_slot], 0), "hipStreamWaitEvent(join)");
  }
  return ARC_OK;
}

}  // namespace

namespace arc {

// The compressor step (arguments already checked); with a non-null G the
// payload is also added into G at the selected coordinates.
arc_status enqueue_step(arc_ctx* c, int64_t t, const void* grad, float* h, float* g,
                        int32_t* out_idx, float* out_agg, float* G) {
  // Vectorisable groups take the 16-byte kernels only when the three streams
  // are 16-byte aligned; otherwise every group takes the general kernel.
  const int64_t ngroups = static_cast<int64_t>(c->groups.size());
  const int64_t nvec = aligned16(grad) && aligned16(h) && aligned16(g) ? c->nvec_groups : 0;

  size_t slot = 0;
  if (c->timing) {
    if (c->ev_used == c->ev_pool.size()) {
      std::array<hipEvent_t, arc::kEventsPerStep> evs{};
      for (auto& e : evs) ARC_HIP(hipEventCreate(&e), "hipEventCreate");
      c->ev_pool.push_back(evs);
    }
    slot = c->ev_used++;
  }
  arc_status st;
  if ((st = record(c, slot, 0))) return st;
  if (c->compressor == ARC_COMP_ARC && !c->V_staged && (st = upload_projection(c, t)))
    return st;
  if ((st = record(c, slot, 1))) return st;
  const arc::SelectWorkspace ws = c->select_ws();
  if (c->compressor == ARC_COMP_RANDK) {
    // Stage 0: Eq. (11a) alone (the residual is needed at the kept rows only).
    const bool vec = (c->N * c->d) % 4 == 0 && aligned16(grad) && aligned16(h);
    ARC_HIP(arc::launch_momentum(vec, grad, c->grad_bf16, h, c->N * c->d, c->eta, c->a,
                                 c->stream),
            "momentum launch");
    if ((st = record(c, slot, 2))) return st;
    // Stage 1: the shared random keys; stage 2: their per-bucket top-K.
    ARC_HIP(arc::launch_randk_keys(c->seed, t, c->m, c->sigma_dev, c->stream), "keys launch");
    if ((st = record(c, slot, 3))) return st;
    ARC_HIP(arc::launch_select(c->sigma_dev, ws, out_idx, c->stream), "select launch");
    if ((st = record(c, slot, 4))) return st;
  } else if (c->compressor == ARC_COMP_TOPK) {
    // Stage 0: Eq. (11a) with every node's squared row norms of Delta.
    if ((st = launch_streaming_stage(c, grad, h, g, nvec, ngroups, true))) return st;
    if ((st = record(c, slot, 2))) return st;
    if ((st = record(c, slot, 3))) return st;
    // Stage 2: every node's own top-K over its norms.
    ARC_HIP(arc::launch_select(c->S_dev, ws, c->sel_dev, c->stream), "select launch");
    if ((st = record(c, slot, 4))) return st;
    // Stage 3: every node's rows, unsummed (the All-Gather payload); in the
    // model step, tagged per node for the merge that follows.
    const bool vec = c->d % 4 == 0 && c->payload_node % 4 == 0 && aligned16(h) &&
                     aligned16(g) && aligned16(out_agg);
    const bool merge = G != nullptr && c->mark_dev != nullptr;
    if (merge && ++c->mark_stamp == 0) {
      // After 2^32 merges the stamps wrap: clear the old tags first.
      ARC_HIP(arc::launch_zero_u64(c->mark_dev, static_cast<int64_t>(c->N) * c->m, c->stream),
              "tag clear launch");
      c->mark_stamp = 1;
    }
    ARC_HIP(arc::launch_topk_gather(h, g, c->sel_dev, out_idx, out_agg, c->gather_dev,
                                    static_cast<int32_t>(c->gather.size()), c->gather_work,
                                    c->K_node, c->payload_node, c->d, c->m, c->N, vec,
                                    merge ? c->mark_dev : nullptr, c->mark_stamp, c->stream),
            "gather launch");
    if (merge)
      ARC_HIP(arc::launch_topk_merge(out_agg, c->sel_dev, c->mark_dev, c->mark_stamp,
                                     c->gather_dev, static_cast<int32_t>(c->gather.size()),
                                     c->gather_work, c->K_node, c->payload_node, c->d, c->m,
                                     c->N, G, vec && aligned16(G), c->stream),
              "merge launch");
    return record(c, slot, 5);
  } else {
    // Stage 0: momentum + residual + per-worker sketch in one HBM stream.
    // Measured on one MI355X, this order (one worker's row groups per block,
    // then the reduce kernel) is as fast as or faster than streaming the N
    // workers' copies of a group in one block and summing them in LDS, for
    // every worker count: 7B with 2 workers 33.5-34.0 vs 34.4-34.7 ms, 1.1B
    // with 1 worker 2.94 vs 3.00 ms, with 2 equal.
    if ((st = launch_streaming_stage(c, grad, h, g, nvec, ngroups, false))) return st;
    if ((st = record(c, slot, 2))) return st;
    // Stage 1: worker sum + importance of every row.
    ARC_HIP(arc::launch_reduce_rows(c->S_dev, c->sigma_dev, c->m, c->N, c->r, c->stream),
            "reduce launch");
    if ((st = record(c, slot, 3))) return st;
    // Stage 2: per-bucket top-K.
    ARC_HIP(arc::launch_select(c->sigma_dev, ws, out_idx, c->stream), "select launch");
    if ((st = record(c, slot, 4))) return st;
  }
  // Stage 3: gather + worker sum + error-feedback update.
  const bool G_ok = G == nullptr || aligned16(G);
  if (c->tensor_mode) {
    const bool vec_ok = aligned16(h) && aligned16(g) && aligned16(out_agg) && G_ok;
    ARC_HIP(arc::launch_gather_update_tensors(h, g, out_idx, out_agg, G, c->gather_dev,
                                              static_cast<int32_t>(c->gather.size()),
                                              c->gather_work, c->d, c->N, vec_ok, c->stream),
            "gather launch");
  } else {
    const bool fast_gather = c->n % 4 == 0 && c->d % 4 == 0 && aligned16(h) && aligned16(g) &&
                             aligned16(out_agg) && G_ok;
    ARC_HIP(arc::launch_gather_update(fast_gather, h, g, out_idx, out_agg, G, c->K_total, c->d,
                                      c->n, c->m, c->N, c->stream),
            "gather launch");
  }
  if ((st = record(c, slot, 5))) return st;
  return ARC_OK;
}

}  // namespace arc

namespace {

bool finite(float v) { return std::isfinite(v); }

}  // namespace

extern "C" {

arc_status arc_step(arc_ctx* c, int64_t t, const void* grad, float* h, float* g,
                    int32_t* out_idx, float* out_agg) {
  const arc_status st = arc::check_step_args(c, t, grad, h, g, out_idx, out_agg, true);
  if (st != ARC_OK) return st;
  return arc::enqueue_step(c, t, grad, h, g, out_idx, out_agg, nullptr);
}

arc_status arc_model_step(arc_ctx* c, const arc_model_config* mc, int64_t t, const void* grad,
                          float* h, float* g, float* G, float* x, float* opt_m, float* opt_v,
                          int32_t* out_idx, float* out_agg) {
  if (mc == nullptr) return fail(ARC_ERR_INVALID, "model config is NULL");
  // A dense iteration writes no payload, so out_idx / out_agg may be NULL.
  const bool dense = t < mc->dense_steps;
  arc_status st = arc::check_step_args(c, t, grad, h, g, out_idx, out_agg, !dense);
  if (st != ARC_OK) return st;
  if (mc->optimizer < ARC_OPT_SGD || mc->optimizer > ARC_OPT_ADAM)
    return fail(ARC_ERR_INVALID, "optimizer must be ARC_OPT_SGD, ARC_OPT_MSGD or ARC_OPT_ADAM");
  if (mc->dense_steps < 0) return fail(ARC_ERR_INVALID, "dense_steps must be >= 0");
  if (!finite(mc->lr) || !finite(mc->weight_decay))
    return fail(ARC_ERR_INVALID, "lr and weight_decay must be finite");
  if (!(mc->momentum >= 0.0f && mc->momentum < 1.0f) ||
      !(mc->beta1 >= 0.0f && mc->beta1 < 1.0f) || !(mc->beta2 >= 0.0f && mc->beta2 < 1.0f) ||
      !(mc->eps >= 0.0f) || !finite(mc->eps))
    return fail(ARC_ERR_INVALID, "momentum, beta1, beta2 must be in [0, 1), eps >= 0");
  if (G == nullptr || x == nullptr) return fail(ARC_ERR_INVALID, "G and x must be non-NULL");
  if (mc->optimizer >= ARC_OPT_MSGD && opt_m == nullptr)
    return fail(ARC_ERR_INVALID, "opt_m must be non-NULL for MSGD and Adam");
  if (mc->optimizer == ARC_OPT_ADAM && opt_v == nullptr)
    return fail(ARC_ERR_INVALID, "opt_v must be non-NULL for Adam");
  {
    const size_t elems = static_cast<size_t>(c->N) * static_cast<size_t>(c->d);
    const size_t vb = static_cast<size_t>(c->d) * 4;
    const void* big[3] = {grad, h, g};
    const size_t big_bytes[3] = {elems * (c->grad_bf16 ? 2 : 4), elems * 4, elems * 4};
    const void* vecs[4] = {G, x, mc->optimizer >= ARC_OPT_MSGD ? opt_m : nullptr,
                           mc->optimizer == ARC_OPT_ADAM ? opt_v : nullptr};
    for (int a = 0; a < 4; ++a) {
      if (vecs[a] == nullptr) continue;
      for (int b = a + 1; b < 4; ++b)
        if (vecs[b] != nullptr && ranges_overlap(vecs[a], vb, vecs[b], vb))
          return fail(ARC_ERR_INVALID, "G, x, opt_m and opt_v must not overlap");
      for (int b = 0; b < 3; ++b)
        if (ranges_overlap(vecs[a], vb, big[b], big_bytes[b]))
          return fail(ARC_ERR_INVALID, "G, x, opt_m, opt_v must not overlap grad, h or g");
      if (!dense && c->K_total > 0 &&
          (ranges_overlap(vecs[a], vb, out_idx, static_cast<size_t>(c->K_total) * 4) ||
           ranges_overlap(vecs[a], vb, out_agg, static_cast<size_t>(c->payload) * 4)))
        return fail(ARC_ERR_INVALID, "G, x, opt_m, opt_v must not overlap out_idx or out_agg");
    }
  }

  if (dense) {
    const bool vec = c->d % 4 == 0 && aligned16(grad) && aligned16(h) && aligned16(g) &&
                     aligned16(G);
    ARC_HIP(arc::launch_dense_step(vec, grad, c->grad_bf16, h, g, G, c->d, c->N, c->eta, c->a,
                                   c->stream),
            "dense step launch");
  } else {
    st = arc::enqueue_step(c, t, grad, h, g, out_idx, out_agg, G);
    if (st != ARC_OK) return st;
  }

  arc::OptimizerArgs o{};
  o.kind = mc->optimizer;
  o.neg_lr = -mc->lr;
  o.momentum = mc->momentum;
  o.beta1 = mc->beta1;
  o.beta2 = mc->beta2;
  o.one_minus_beta1 = 1.0f - mc->beta1;
  o.one_minus_beta2 = 1.0f - mc->beta2;
  double p1 = 1.0, p2 = 1.0;
  if (mc->optimizer == ARC_OPT_ADAM)
    for (int64_t k = 0; k <= t; ++k) {  // beta^T with T = t + 1
      p1 *= static_cast<double>(mc->beta1);
      p2 *= static_cast<double>(mc->beta2);
    }
  o.c1 = static_cast<float>(1.0 - p1);
  o.c2 = static_cast<float>(1.0 - p2);
  o.eps = mc->eps;
  o.weight_decay = mc->weight_decay;
  o.fN = static_cast<float>(c->N);
  const bool vec = c->d % 4 == 0 && aligned16(G) && aligned16(x) &&
                   (o.kind < 1 || aligned16(opt_m)) && (o.kind < 2 || aligned16(opt_v));
  ARC_HIP(arc::launch_optimizer(vec, c->lds_per_cu == arc::kLdsPerCu, o, G, x, opt_m, opt_v,
                                c->d, c->stream),
          "optimizer launch");
  return ARC_OK;
}

arc_status arc_describe(const arc_ctx* c, char* buf, int64_t len) {
  if (c == nullptr || buf == nullptr || len <= 0) return fail(ARC_ERR_INVALID, "NULL argument");
  const int64_t ngroups = static_cast<int64_t>(c->groups.size());
  const char* comp = c->compressor == ARC_COMP_RANDK  ? "randk"
                     : c->compressor == ARC_COMP_TOPK ? "topk"
                                                      : "arc";
  const char* sketch = c->compressor == ARC_COMP_RANDK ? "none"
                       : c->nvec_groups == 0           ? "general"
                       : c->compressor == ARC_COMP_TOPK ? "row_norms"
                                                       : "per_worker+reduce";
  int radix = 0;
  for (const auto& b : c->buckets) radix += b.mode == arc::kSelectRadix;
  long long strided = 0;
  for (const auto& grp : c->groups) strided += grp.stride > 1;
  std::snprintf(buf, static_cast<size_t>(len),
                "compressor=%s mode=%s sketch=%s widths=%zu row_groups=%lld vector_groups=%lld "
                "(64:%lld 32:%lld 16:%lld 8:%lld rows) workgroup_waves=(%d%s %d%s %d%s %d%s) "
                "interleaved_groups=%lld general_groups=%lld "
                "lds_limit=%zu buckets=%zu radix_buckets=%d select=%s%s K_total=%lld "
                "payload=%lld",
                comp, c->tensor_mode ? "tensors" : "single_view", sketch, c->widths.size(),
                static_cast<long long>(ngroups), static_cast<long long>(c->nvec_groups),
                static_cast<long long>(c->vec_count[0]), static_cast<long long>(c->vec_count[1]),
                static_cast<long long>(c->vec_count[2]), static_cast<long long>(c->vec_count[3]),
                c->vec_occ[0].waves, c->vec_occ[0].one_per_cu ? "/cu" : "",
                c->vec_occ[1].waves, c->vec_occ[1].one_per_cu ? "/cu" : "",
                c->vec_occ[2].waves, c->vec_occ[2].one_per_cu ? "/cu" : "",
                c->vec_occ[3].waves, c->vec_occ[3].one_per_cu ? "/cu" : "", strided,
                static_cast<long long>(ngroups - c->nvec_groups),
                c->max_lds_per_block, c->buckets.size(),
                radix, c->select_ws().small ? "one_workgroup_per_bucket" : "blocks:",
                c->select_ws().small ? "" : std::to_string(c->blocks.size()).c_str(),
                static_cast<long long>(c->K_total),
                static_cast<long long>(c->payload));
  return ARC_OK;
}

arc_status arc_debug_sigma(arc_ctx* c, float* out_sigma) {
  if (c == nullptr || out_sigma == nullptr) return fail(ARC_ERR_INVALID, "NULL argument");
  ARC_HIP(hipMemcpyAsync(out_sigma, c->sigma_dev, static_cast<size_t>(c->m) * sizeof(float),
                         hipMemcpyDeviceToDevice, c->stream),
          "hipMemcpyAsync(sigma)");
  return ARC_OK;
}

arc_status arc_debug_sketch(arc_ctx* c, float* out_S) {
  if (c == nullptr || out_S == nullptr) return fail(ARC_ERR_INVALID, "NULL argument");
  ARC_HIP(hipMemcpyAsync(out_S, c->S_dev,
                         static_cast<size_t>(c->N) * c->m * c->r * sizeof(float),
                         hipMemcpyDeviceToDevice, c->stream),
          "hipMemcpyAsync(S)");
  return ARC_OK;
}

arc_status arc_debug_projection(arc_ctx* c, int64_t t, float* out_V) {
  if (c == nullptr || out_V == nullptr) return fail(ARC_ERR_INVALID, "NULL argument");
  if (t < 0) return fail(ARC_ERR_INVALID, "t must be >= 0");
  if (c->tensor_mode)
    return fail(ARC_ERR_UNSUPPORTED, "per-tensor mode: use arc_projection with the width");
  if (c->use_override)
    std::memcpy(out_V, c->V_override.data(), c->V_override.size() * sizeof(float));
  else
    arc::generate_projection(c->seed, t, c->n, c->r, out_V);
  return ARC_OK;
}

arc_status arc_set_projection(arc_ctx* c, const float* V) {
  if (c == nullptr) return fail(ARC_ERR_INVALID, "ctx is NULL");
  if (c->tensor_mode) return fail(ARC_ERR_UNSUPPORTED, "arc_set_projection: per-tensor mode");
  if (V == nullptr) {
    c->use_override = false;
    c->V_override.clear();
    return ARC_OK;
  }
  try {
    c->V_override.assign(V, V + static_cast<size_t>(c->n) * c->r);
  } catch (...) {
    return fail(ARC_ERR_NOMEM, "host allocation failed");
  }
  c->use_override = true;
  return ARC_OK;
}

arc_status arc_timing_enable(arc_ctx* c, int32_t on) {
  if (c == nullptr) return fail(ARC_ERR_INVALID, "ctx is NULL");
  c->timing = on != 0;
  return ARC_OK;
}

arc_status arc_timing_read(arc_ctx* c, double* ms, int64_t* steps) {
  if (c == nullptr || ms == nullptr || steps == nullptr)
    return fail(ARC_ERR_INVALID, "NULL argument");
  for (int k = 0; k < ARC_NUM_STAGES; ++k) ms[k] = 0.0;
  for (size_t s = 0; s < c->ev_used; ++s) {
    auto& ev = c->ev_pool[s];
    ARC_HIP(hipEventSynchronize(ev[arc::kEventsPerStep - 1]), "hipEventSynchronize");
    float x = 0.f;
    const int pairs[ARC_NUM_STAGES][2] = {{1, 2}, {2, 3}, {3, 4}, {4, 5}, {0, 5}};
    for (int k = 0; k < ARC_NUM_STAGES; ++k) {
      ARC_HIP(hipEventElapsedTime(&x, ev[pairs[k][0]], ev[pairs[k][1]]),
              "hipEventElapsedTime");
      ms[k] += x;
    }
  }
  *steps = static_cast<int64_t>(c->ev_used);
  c->ev_used = 0;
  return ARC_OK;
}

}  // extern "C"

namespace arc {

arc_status plan_context(const arc_config* cfg, int64_t m, void* stream, arc_ctx* c) {
  try {
    c->d = cfg->d;
    c->tensor_mode = cfg->num_tensors > 0;
    c->compressor = cfg->compressor;
    c->n = c->tensor_mode ? 0 : cfg->n;
    c->m = m;
    c->N = cfg->N;
    c->r = cfg->r;
    c->grad_bf16 = cfg->grad_dtype == ARC_DTYPE_BF16;
    c->eta = cfg->eta;
    c->a = 1.0f - cfg->eta;
    c->seed = cfg->seed;
    c->stream = static_cast<hipStream_t>(stream);
    build_plan(cfg, c);
  } catch (...) {
    return fail(ARC_ERR_NOMEM, "host allocation failed");
  }
  return ARC_OK;
}

arc_status bind_device(arc_ctx* c) {
  ARC_HIP(hipGetDevice(&c->device), "hipGetDevice");
  int lds_limit = 0;
  ARC_HIP(hipDeviceGetAttribute(&lds_limit, hipDeviceAttributeMaxSharedMemoryPerBlock, c->device),
          "hipDeviceGetAttribute");
  c->max_lds_per_block = static_cast<size_t>(lds_limit);
  // One workgroup per compute unit is reached through the LDS reservation,
  // which assumes the gfx950 figure; on any other, launches go uncapped.
  int lds_cu = 0;
  ARC_HIP(hipDeviceGetAttribute(&lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor,
                                c->device),
          "hipDeviceGetAttribute");
  c->lds_per_cu = lds_cu;
  if (lds_cu != kLdsPerCu || lds_limit < kLdsPerCu / 2 + 1024)
    for (auto& o : c->vec_occ) o.one_per_cu = 0;
  return ARC_OK;
}

}  // namespace arc
