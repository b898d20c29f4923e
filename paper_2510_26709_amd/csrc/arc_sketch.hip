// Streaming stage of the compressor step: EF21M momentum (11a), residual
// Delta = h_t - g_{t-1} and per-worker sketch P^(i) = G^(i) V (Alg. 1) in one
// pass over HBM; then the worker sum and row importance Sigma = diag(P P^T)
// (Eq. (4)) in a small kernel over the sketches.
//
// Numerics follow the contract in libarctopk.h: binary32; the dot product of
// a row with column k of V is a fused multiply-add chain in ascending column
// order from +0; the worker sum is a chain of plain additions in ascending
// worker order; Sigma is a fused multiply-add chain of squares in ascending k.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "arc_device.h"
#include "arc_internal.h"

namespace arc {
namespace {

// Row groups of G in {64, 32, 16, 8} rows.  One 16-byte load instruction of
// a wave covers G/8 rows of LPR = 512/G lanes each, so eight instructions
// cover the group's G rows over a chunk of CW = 4*LPR columns (32 to 256).  The
// LDS tile holds G rows of Delta with LPR float4 per row plus one float4 of
// padding (at most 576 float4 for every G), so that consecutive lanes reading
// consecutive rows hit distinct 16-byte bank groups.
template <int G>
struct GroupShape {
  static_assert(G == 64 || G == 32 || G == 16 || G == 8, "row group of 64 to 8 rows");
  static constexpr int kLanesPerRow = 512 / G;
  static constexpr int kRowsPerLoad = kWave / kLanesPerRow;
  static constexpr int kChunkCols = 4 * kLanesPerRow;
  static constexpr int kRowF4 = kLanesPerRow + 1;
};
constexpr int kTileF4 = 576;  // >= G * (512 / G + 1) for every G
// Rows of fewer chunks than this keep unshifted windows where the shift onto
// whole lines would add a chunk (see sketch_rows).
constexpr uint32_t kShiftMinChunks = 3;

// (row, k) lanes: when G * R <= 64, lane l runs only the chain of row l % G
// against column (l / G) % R of V, and the R results of a row are collected
// from their lanes at the end.  Otherwise every lane runs all R chains of
// row l % G.
template <int R, int G, bool NORM>
constexpr bool k_split() { return !NORM && G * R <= kWave; }

// After its tile, a wave's LDS holds the projection rows of the current
// chunk (CW x R binary32), so that the chains read V from LDS: wave-uniform
// scalar loads of V would share the lgkm counter with the tile reads, and a
// wait for one would be a wait for both.  With (row, k) lanes the slice is
// transposed, [k][column] with a pitch of CW + 4 floats (each lane reads its
// column of V as float4s, and the R columns fall in distinct banks).
template <int R, int G, bool NORM>
constexpr int slice_src_f4() { return NORM ? 0 : GroupShape<G>::kChunkCols * R / 4; }
template <int R, int G, bool NORM>
constexpr int slice_f4() {
  return k_split<R, G, NORM>() ? R * (GroupShape<G>::kChunkCols + 4) / 4
                               : slice_src_f4<R, G, NORM>();
}
template <int R, int G, bool NORM>
constexpr int wave_lds_f4() { return kTileF4 + slice_f4<R, G, NORM>(); }
// Offset whose access the hardware drops: a group spans at most 2^30 bytes
// (64 consecutive rows of at most 2^22 binary32 values; the host keeps
// groups of rows further apart within the same span), so 2^31, and the 2^30
// it becomes for the bf16 stream's halved offsets, lie beyond every
// resource here.
constexpr uint32_t kDropOffset = 0x80000000u;

// One wave's pass over the rows of one row group of worker i: loads the
// grad/h/g tile of each chunk with coalesced 16-byte accesses, applies (11a),
// writes h back, parks Delta in LDS, then runs this lane's r chains over its
// row.  Local row l of the group starts at coordinate elem_off + l*stride*n;
// n is a multiple of 4 but need not be one of the chunk width, in which case
// each row's last chunk is partial: its lanes past the row's end load and
// store nothing, and the chains stop at the row's end.  Rows that start off
// a 128-byte line take chunks shifted onto whole lines (below), with a
// partial first chunk as well.  The three streams are
// read through buffer resources that end at the group's last row, so in a
// group of fewer than G rows (always consecutive rows, stride 1) the missing
// rows read as zero and are not stored.
// Lanes G..63 repeat the chains of lanes 0..G-1; the caller keeps only lanes
// below the group's row count.  NORM (R = 1): the chain is the row's squared
// norm, fmaf(Delta, Delta, s), and V is unused.
template <int R, bool BF16, int G, bool NORM = false>
__device__ __forceinline__ void sketch_rows(
    const void* __restrict__ grad, float* __restrict__ h,
    const float* __restrict__ g, const float* __restrict__ V, int64_t d,
    const RowGroup& grp, int32_t i, float eta, float a, float4* tile,
    float (&s)[R]) {
  using Shape = GroupShape<G>;
  constexpr bool kSplit = k_split<R, G, NORM>();
  constexpr int kSliceF4 = slice_src_f4<R, G, NORM>();  // float4 of V per chunk
  constexpr int kSliceRegs = (kSliceF4 + kWave - 1) / kWave;
  constexpr int kLPR = Shape::kLanesPerRow;
  constexpr int kRPL = Shape::kRowsPerLoad;
  constexpr int kCW = Shape::kChunkCols;
  constexpr int kPitch = Shape::kRowF4;
  const int lane = threadIdx.x & (kWave - 1);
  const int sub = lane / kLPR;   // row within one load's rows
  const int quad = lane % kLPR;  // 16-byte column group within the chunk
  const uint32_t n = (uint32_t)grp.cols;
  const int32_t rows = grp.rows;
  const uint32_t rstride = (uint32_t)grp.stride;
  const int64_t wbase = (int64_t)i * d + grp.elem_off;
  const uint32_t bytes = ((uint32_t)(rows - 1) * rstride + 1u) * n * 4u;
  const buffer_rsrc rh = make_buffer(h + wbase, bytes);
  const buffer_rsrc rg = make_buffer(g + wbase, bytes);
  const buffer_rsrc rx =
      BF16 ? make_buffer(static_cast<const uint16_t*>(grad) + wbase, bytes / 2)
           : make_buffer(static_cast<const float*>(grad) + wbase, bytes);
  V += grp.v_off;
  // Column windows on whole 128-byte lines.  Where every row of the group
  // starts the same number of bytes past a line of h (one row, or a row
  // pitch that is a multiple of 128 bytes), chunk c covers the columns
  // [c*kCW - shift, (c+1)*kCW - shift) rather than [c*kCW, (c+1)*kCW), with
  // shift the rows' offset from the line in binary32 values (a multiple of
  // 4, as h is 16-byte aligned): each load instruction then covers whole
  // lines instead of straddling one more.  The chains still take a row's
  // columns in ascending order, so the results do not change.  A row can
  // gain a chunk, which rows of one or two chunks cannot afford.  Stage ms,
  // 8 binary32 workers of about 1.2e7 values each, d = 8 mod 32 (each
  // worker's base 32 bytes further past a line than the previous one's),
  // without / with the shift: 512-wide rows (2 chunks)
  // 0.289 / 0.314, 768 (3) 0.305 / 0.297, 1024 (8, 16-row groups) 0.309 /
  // 0.264, 1536 (6) 0.312 / 0.289, 2304 (9) 0.330 / 0.311, 4608 (18) 0.351
  // / 0.322; at 6e7 values each alike.
  uint32_t shift = 0;
  if constexpr (G <= 16) {
    if (rows == 1 || (rstride * n) % 32u == 0u)
      shift = (uint32_t)(reinterpret_cast<uintptr_t>(h + wbase) & 127u) / 4u;
    const uint32_t plain = (n + kCW - 1) / kCW;
    if ((n + shift + kCW - 1) / kCW > plain && plain < kShiftMinChunks) shift = 0;
  }
  // byte offset of this lane's 16 bytes of binary32 in row u*kRPL + sub, in
  // chunk 0 (wrapped below zero for the lanes before a shifted row's start,
  // whose accesses in chunk 0 are dropped)
  uint32_t off[8];
#pragma unroll
  for (int u = 0; u < 8; ++u)
    off[u] = ((uint32_t)(u * kRPL + sub) * rstride * n + quad * 4 - shift) * 4u;
#pragma unroll
  for (int k = 0; k < R; ++k) s[k] = 0.0f;
  float s_own = 0.0f;  // (row, k) lanes: this lane's chain

  const uint32_t nchunks = (n + shift + kCW - 1) / kCW;
  // Window positions of the last chunk: kCW unless the shifted width is not
  // a multiple of it.  Every bound here is a multiple of 4.
  const uint32_t tail = n + shift - (nchunks - 1) * kCW;
  const bool in_tail = (uint32_t)quad * 4 < tail;
  const bool in_head = (uint32_t)quad * 4 >= shift;
  // Offset o of this lane's access in chunk c, or kDropOffset (the hardware
  // drops the access) where the lane is before a shifted row's start or
  // past the end of a partial last chunk.
  auto col_off = [&](uint32_t o, uint32_t c) {
    return (c > 0 || in_head) && (c + 1 < nchunks || in_tail) ? o : kDropOffset;
  };
  uint2 x_next[8];  // bf16, 64-row groups: this lane's grad of the next chunk
  // Loads of chunk c into xv, hv, gv (off[] at chunk c).  The loop issues
  // the next chunk's loads as soon as this chunk's momentum has consumed the
  // registers, so they are in flight while this chunk's chains run.  bf16
  // gradients stay packed in xv.x, xv.y until used.
  float4 xv[8], hv[8], gv[8];
  using VRegs = float __attribute__((ext_vector_type(4 * (kSliceRegs > 0 ? kSliceRegs : 1))));
  VRegs vreg;  // this lane's share of chunk c's V rows
  float4* vslice = tile + kTileF4;
  // Float4 of chunk c's slice that this lane moves for register r4; lanes
  // past the slice's end (shorter in a partial last chunk, whose V rows end
  // with the width's) repeat its last float4 (same value, same address), so
  // that neither the load nor the store needs a branch.
  auto slice_at = [&](int r4, uint32_t c) {
    const int last = c + 1 < nchunks ? kSliceF4 - 1 : (int)(tail * R / 4) - 1;
    return min(lane + r4 * kWave, last);
  };
  auto issue_loads = [&](uint32_t c) __attribute__((always_inline)) {
    const bool even = (c & 1) == 0;
    if constexpr (kSliceF4 > 0) {
      // Chunk c's V rows start at column c*kCW - shift; the positions before
      // a shifted row's start (no chain reads them) take V's first float4.
      const float4* src = reinterpret_cast<const float4*>(V);
      const int first = ((int)(c * kCW) - (int)shift) * R / 4;
#pragma unroll
      for (int r4 = 0; r4 < kSliceRegs; ++r4)
      {
        const float4 t = src[max(first + slice_at(r4, c), 0)];
        vreg[4 * r4] = t.x;
        vreg[4 * r4 + 1] = t.y;
        vreg[4 * r4 + 2] = t.z;
        vreg[4 * r4 + 3] = t.w;
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint32_t o = col_off(off[u], c);
      if constexpr (BF16 && G == 64) {
        // A row's bf16 grad for two consecutive 32-column chunks is one
        // 128-byte line; both 8-byte halves are requested together on even
        // chunks, so the line is fetched once rather than once per chunk.
        uint2 w;
        if (even) {
          w = buffer_load_u2<kCacheDefault>(rx, o / 2);
          if (c + 1 < nchunks)
            x_next[u] = buffer_load_u2<kCacheDefault>(rx, col_off(off[u] + kCW * 4, c + 1) / 2);
        } else {
          w = x_next[u];
        }
        xv[u] = make_float4(__uint_as_float(w.x), __uint_as_float(w.y), 0.f, 0.f);
      } else if constexpr (BF16) {
        // 32 or more lanes per row: each load already covers whole lines.
        const uint2 w = buffer_load_u2<kCacheDefault>(rx, o / 2);
        xv[u] = make_float4(__uint_as_float(w.x), __uint_as_float(w.y), 0.f, 0.f);
      } else {
        xv[u] = buffer_load_f4<kCacheNonTemporal>(rx, o);
      }
      hv[u] = buffer_load_f4<kCacheNonTemporal>(rh, o);
      gv[u] = buffer_load_f4<kCacheNonTemporal>(rg, o);
    }
  };
  if (nchunks > 0) issue_loads(0);
  for (uint32_t c = 0; c < nchunks; ++c) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      float4 x4 = xv[u];
      if constexpr (BF16) {
        const uint32_t w0 = __float_as_uint(xv[u].x), w1 = __float_as_uint(xv[u].y);
        x4 = make_float4(bf16_lo(w0), bf16_hi(w0), bf16_lo(w1), bf16_hi(w1));
      }
      float4 hn;
      hn.x = fmaf(eta, x4.x, a * hv[u].x);
      hn.y = fmaf(eta, x4.y, a * hv[u].y);
      hn.z = fmaf(eta, x4.z, a * hv[u].z);
      hn.w = fmaf(eta, x4.w, a * hv[u].w);
      // Rows past the group's end get an offset far outside the resource, so
      // the hardware drops their store: a select rather than a branch, which
      // would make the compiler's wait counts for the loads in flight
      // conservative on every path.
      buffer_store_f4<kCacheStreamDevice>(
          rh, u * kRPL + sub < rows ? col_off(off[u], c) : kDropOffset, hn);
      float4 dl;
      dl.x = hn.x - gv[u].x;
      dl.y = hn.y - gv[u].y;
      dl.z = hn.z - gv[u].z;
      dl.w = hn.w - gv[u].w;
      tile[(u * kRPL + sub) * kPitch + quad] = dl;
      off[u] += kCW * 4;
    }
    if constexpr (kSliceF4 > 0 && kSplit) {
      float* vt = reinterpret_cast<float*>(vslice);
#pragma unroll
      for (int r4 = 0; r4 < kSliceRegs; ++r4) {
        const int f = slice_at(r4, c);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int idx = 4 * f + e;  // V[idx / R][idx % R] of the chunk
          vt[(idx % R) * (kCW + 4) + idx / R] = vreg[4 * r4 + e];
        }
      }
    } else if constexpr (kSliceF4 > 0) {
#pragma unroll
      for (int r4 = 0; r4 < kSliceRegs; ++r4)
        vslice[slice_at(r4, c)] =
            make_float4(vreg[4 * r4], vreg[4 * r4 + 1], vreg[4 * r4 + 2], vreg[4 * r4 + 3]);
    }
    // The next chunk's loads go out before this chunk's chains run.
    if (c + 1 < nchunks) issue_loads(c + 1);
    __builtin_amdgcn_sched_barrier(0);
    wave_lds_fence();
    const float* Vc = reinterpret_cast<const float*>(vslice);
    const float4* my_row = tile + (lane & (G - 1)) * kPitch;
    // The chains take window positions [4*q0, 4*q1): from a shifted row's
    // first column in chunk 0, to its last in the last chunk.
    const int q0 = c == 0 ? (int)shift / 4 : 0;
    const int q1 = c + 1 < nchunks ? kLPR : (int)tail / 4;
    auto chain4 = [&](int q) __attribute__((always_inline)) {
      const float4 dv = my_row[q];
      if constexpr (kSplit) {
        const float4 v4 =
            *reinterpret_cast<const float4*>(Vc + ((lane / G) % R) * (kCW + 4) + q * 4);
        s_own = fmaf(dv.x, v4.x, s_own);
        s_own = fmaf(dv.y, v4.y, s_own);
        s_own = fmaf(dv.z, v4.z, s_own);
        s_own = fmaf(dv.w, v4.w, s_own);
      } else {
        const float e4[4] = {dv.x, dv.y, dv.z, dv.w};
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          if constexpr (NORM) {
            s[0] = fmaf(e4[jj], e4[jj], s[0]);
          } else {
#pragma unroll
            for (int k = 0; k < R; ++k)
              s[k] = fmaf(e4[jj], Vc[(q * 4 + jj) * R + k], s[k]);
          }
        }
      }
    };
    if (q0 == 0 && q1 == kLPR) {
#pragma unroll
      for (int q = 0; q < kLPR; ++q) chain4(q);
    } else {
      for (int q = q0; q < q1; ++q) chain4(q);
    }
    wave_lds_fence();
  }
  if constexpr (kSplit) {
    // Row l % G's R results, from lanes l % G + k * G.
#pragma unroll
    for (int k = 0; k < R; ++k) s[k] = __shfl(s_own, (lane & (G - 1)) + k * G, kWave);
  }
}

// ---------------------------------------------------------------------------
// One wave per (row group, worker), WAVES groups of one worker per workgroup;
// the sketch goes to S for the reduce kernel (4r bytes per row and worker).
// HBM traffic per element and worker: grad (4 or 2 B) + h read and write
// (8 B) + g read (4 B).  Delta never leaves the chip.
// ---------------------------------------------------------------------------
template <int R, bool BF16, int G, int WAVES, bool NORM = false>
__global__ void __launch_bounds__(WAVES * kWave)
sketch_per_worker_kernel(const void* __restrict__ grad, float* __restrict__ h,
                         const float* __restrict__ g, const float* __restrict__ V,
                         const RowGroup* __restrict__ groups, int64_t ngroups,
                         float* __restrict__ S, int64_t d, int64_t m, float eta,
                         float a, int32_t flat) {
  __shared__ float4 tiles[WAVES][wave_lds_f4<R, G, NORM>()];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  int32_t i;   // worker
  int64_t gb;  // block of row groups within the worker's list
  if (flat) {
    const int64_t nbx = (ngroups + WAVES - 1) / WAVES;
    const int64_t f = xcd_contiguous_block(blockIdx.x, gridDim.x);
    i = (int32_t)(f / nbx);
    gb = f - (int64_t)i * nbx;
  } else {
    i = blockIdx.y;
    gb = xcd_contiguous_block(blockIdx.x, gridDim.x);
  }
  const int64_t gi = gb * WAVES + wave;
  if (gi >= ngroups) return;  // whole wave; no block barrier follows
  const RowGroup grp = groups[gi];
  float s[R];
  sketch_rows<R, BF16, G, NORM>(grad, h, g, V, d, grp, i, eta, a, tiles[wave], s);
  if (lane < grp.rows) {
    float* out = S + ((int64_t)i * m + grp.row0 + (int64_t)lane * grp.stride) * R;
#pragma unroll
    for (int k = 0; k < R; ++k) out[k] = s[k];
  }
}

// Launch over ngroups row groups and N workers.  With one_per_cu the launch
// asks for dynamic LDS beyond the kernel's own tiles so that a workgroup holds
// more than half of a compute unit's LDS: then at most one workgroup (of this
// or any other such launch) runs per compute unit.  Fewer waves streaming at
// once keep fewer DRAM rows open at a time; on the 1.1B-parameter workload
// two waves per compute unit moved the stage from 5.5 to 6.1 TB/s.
template <int R, bool BF16, int G, bool NORM, int WAVES>
void launch_per_worker_waves(bool one_per_cu, const void* grad, float* h, const float* g,
                             const float* V, const RowGroup* groups, int64_t ngroups, float* S,
                             int64_t d, int64_t m, int32_t N, float eta, float a,
                             hipStream_t stream) {
  constexpr size_t kStatic = (size_t)WAVES * wave_lds_f4<R, G, NORM>() * sizeof(float4);
  constexpr size_t kHalf = kLdsPerCu / 2 + 1024;  // a margin past one half
  static_assert(kStatic < kHalf, "the reservation below assumes tiles under half the LDS");
  const size_t reserve = one_per_cu ? kHalf - kStatic : 0;
  // With N a multiple of 8 the grid is one-dimensional over (worker, block)
  // and each XCD's contiguous eighth is whole workers, so every XCD streams
  // the same bytes whatever the layout's spread of row widths (per-tensor
  // GPT-2 small 2.91 -> 2.81 ms, ResNet-18 and GPT-2 small single views,
  // per-tensor ResNet-18 and tiny within 0.5%, interleaved runs on one
  // box).  With 4 workers an eighth is half a worker, and the 1.1B workload
  // read 10.2-10.3 ms against 9.5-10.0 ms with a grid row per worker, which
  // other worker counts therefore keep (as does a grid too large for one
  // dimension).
  const unsigned nbx = blocks_for(ngroups, WAVES);
  const bool flat = N % 8 == 0 && (int64_t)nbx * N <= INT32_MAX;
  hipLaunchKernelGGL((sketch_per_worker_kernel<R, BF16, G, WAVES, NORM>),
                     flat ? dim3(nbx * (unsigned)N) : dim3(nbx, (unsigned)N), dim3(WAVES * kWave),
                     reserve, stream, grad, h, g, V, groups, ngroups, S, d, m, eta, a,
                     flat ? 1 : 0);
}

template <int R, bool BF16, int G, bool NORM>
void launch_per_worker(const SketchOccupancy& occ, const void* grad, float* h, const float* g,
                       const float* V, const RowGroup* groups, int64_t ngroups, float* S,
                       int64_t d, int64_t m, int32_t N, float eta, float a, hipStream_t stream) {
  if (occ.waves == 2)
    launch_per_worker_waves<R, BF16, G, NORM, 2>(occ.one_per_cu != 0, grad, h, g, V, groups,
                                                 ngroups, S, d, m, N, eta, a, stream);
  else
    launch_per_worker_waves<R, BF16, G, NORM, 4>(occ.one_per_cu != 0, grad, h, g, V, groups,
                                                 ngroups, S, d, m, N, eta, a, stream);
}

// Worker sum P = S^(0) + S^(1) + ... (ascending worker order) and importance
// sum_k P_k^2 (fma chain in ascending k) of row p.
__device__ __forceinline__ void reduce_row(const float* __restrict__ S, float* __restrict__ sigma,
                                           int64_t p, int64_t m, int32_t N, int32_t r) {
  float acc = 0.0f;
  if (r == 4) {
    float4 P = *reinterpret_cast<const float4*>(S + p * 4);
    for (int32_t i = 1; i < N; ++i) {
      const float4 q = *reinterpret_cast<const float4*>(S + ((int64_t)i * m + p) * 4);
      P.x = P.x + q.x;
      P.y = P.y + q.y;
      P.z = P.z + q.z;
      P.w = P.w + q.w;
    }
    acc = fmaf(P.x, P.x, acc);
    acc = fmaf(P.y, P.y, acc);
    acc = fmaf(P.z, P.z, acc);
    acc = fmaf(P.w, P.w, acc);
  } else {
    for (int32_t k = 0; k < r; ++k) {
      float P = S[p * r + k];
      for (int32_t i = 1; i < N; ++i) P = P + S[((int64_t)i * m + p) * r + k];
      acc = fmaf(P, P, acc);
    }
  }
  sigma[p] = acc;
}

// For every row: one thread per row.
__global__ void __launch_bounds__(256)
reduce_rows_kernel(const float* __restrict__ S, float* __restrict__ sigma, int64_t m, int32_t N,
                   int32_t r) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p < m) reduce_row(S, sigma, p, m, N, r);
}

template <int R, bool BF16, int G>
struct PerWorkerLaunch {
  static void run(const SketchOccupancy& occ, const void* grad, float* h, const float* g,
                  const float* V, const RowGroup* groups, int64_t ngroups, float* S, int64_t d,
                  int64_t m, int32_t N, float eta, float a, hipStream_t stream) {
    launch_per_worker<R, BF16, G, false>(occ, grad, h, g, V, groups, ngroups, S, d, m, N, eta,
                                         a, stream);
  }
};

template <template <int, bool, int> class Launch, int R, bool BF16, typename... Args>
bool dispatch_g(int32_t group_rows, Args... args) {
  switch (group_rows) {
    case 64: Launch<R, BF16, 64>::run(args...); return true;
    case 32: Launch<R, BF16, 32>::run(args...); return true;
    case 16: Launch<R, BF16, 16>::run(args...); return true;
    case 8: Launch<R, BF16, 8>::run(args...); return true;
    default: return false;
  }
}

// Launch<r, dtype, group_rows>::run(args...) for the instantiated values;
// false for any other r or group size.
template <template <int, bool, int> class Launch, typename... Args>
bool dispatch(int32_t r, bool bf16, int32_t group_rows, Args... args) {
  switch (r) {
    case 1: return bf16 ? dispatch_g<Launch, 1, true>(group_rows, args...)
                        : dispatch_g<Launch, 1, false>(group_rows, args...);
    case 2: return bf16 ? dispatch_g<Launch, 2, true>(group_rows, args...)
                        : dispatch_g<Launch, 2, false>(group_rows, args...);
    case 4: return bf16 ? dispatch_g<Launch, 4, true>(group_rows, args...)
                        : dispatch_g<Launch, 4, false>(group_rows, args...);
    case 8: return bf16 ? dispatch_g<Launch, 8, true>(group_rows, args...)
                        : dispatch_g<Launch, 8, false>(group_rows, args...);
    default: return false;
  }
}

}  // namespace

hipError_t launch_sketch_per_worker(int32_t group_rows, const void* grad, int32_t grad_bf16,
                                    float* h, const float* g, const float* V,
                                    const RowGroup* groups, int64_t ngroups, float* S,
                                    int64_t d, int64_t m, int32_t N, int32_t r, float eta,
                                    float a, SketchOccupancy occ, hipStream_t stream) {
  if (ngroups <= 0) return hipSuccess;
  if (!dispatch<PerWorkerLaunch>(r, grad_bf16 != 0, group_rows, occ, grad, h, g, V, groups,
                                 ngroups, S, d, m, N, eta, a, stream))
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_row_norms(int32_t group_rows, const void* grad, int32_t grad_bf16, float* h,
                            const float* g, const float* V, const RowGroup* groups, int64_t ngroups,
                            float* norms, int64_t d, int64_t m, int32_t N, float eta, float a,
                            SketchOccupancy occ, hipStream_t stream) {
  if (ngroups <= 0) return hipSuccess;
#define ARC_NORM_CASE(GG)                                                                    \
  case GG:                                                                                   \
    if (grad_bf16)                                                                           \
      launch_per_worker<1, true, GG, true>(occ, grad, h, g, V, groups, ngroups, norms, d, m, \
                                           N, eta, a, stream);                               \
    else                                                                                     \
      launch_per_worker<1, false, GG, true>(occ, grad, h, g, V, groups, ngroups, norms, d,   \
                                            m, N, eta, a, stream);                           \
    break;
  switch (group_rows) {
    ARC_NORM_CASE(64)
    ARC_NORM_CASE(32)
    ARC_NORM_CASE(16)
    ARC_NORM_CASE(8)
    default:
      return hipErrorInvalidValue;
  }
#undef ARC_NORM_CASE
  return hipGetLastError();
}

hipError_t launch_reduce_rows(const float* S, float* sigma, int64_t m, int32_t N, int32_t r,
                              hipStream_t stream) {
  if (m <= 0) return hipSuccess;
  hipLaunchKernelGGL(reduce_rows_kernel, dim3(blocks_for(m, 256)), dim3(256), 0, stream, S,
                     sigma, m, N, r);
  return hipGetLastError();
}

}  // namespace arc
