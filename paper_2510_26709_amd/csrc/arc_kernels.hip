// HIP kernels of the ARC-Top-K + EF21M compressor step for gfx950 (MI355X).
//
// Numerics follow the contract in libarctopk.h: binary32, sums in ascending
// index order, fused multiply-add chains for the dot products and squares,
// plain additions across workers.  Build with -ffp-contract=off so that no
// other operation is fused.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "arc_internal.h"

namespace arc {
namespace {

constexpr int kWave = 64;

// Order this wave's LDS accesses: everything issued before has completed
// before anything after is issued.  Waves of a block never share LDS rows in
// the sketch kernel, so no block barrier is needed.
__device__ __forceinline__ void wave_lds_fence() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

__device__ __forceinline__ float bf16_lo(uint32_t w) {
  return __uint_as_float(w << 16);
}
__device__ __forceinline__ float bf16_hi(uint32_t w) {
  return __uint_as_float(w & 0xFFFF0000u);
}

// ---------------------------------------------------------------------------
// Streaming sketch, vectorised path.
//
// One wave owns 64 consecutive rows of one worker; lane L owns row p0 + L for
// the dot products.  Rows are walked in chunks of 32 columns.  For a chunk,
// the wave loads the 64 x 32 tile of grad, h and g with 16-byte accesses in a
// coalesced layout (8 lanes per row, 8 rows per instruction), applies the
// EF21M momentum (11a) and writes h back in place, forms the residual
// Delta = h_new - g and parks it in LDS.  Each lane then reads its own row of
// Delta from LDS and continues its r fused multiply-add chains in ascending
// column order, with V[j][0..r) read as wave-uniform scalars.  Delta never
// goes back to HBM.
//
// HBM traffic per element and worker: grad (4 or 2 B) + h read and write (8 B)
// + g read (4 B).
// ---------------------------------------------------------------------------
constexpr int kChunk = 32;          // columns per chunk
constexpr int kLdsRowF4 = 9;        // 8 float4 of data + 1 of padding per row
constexpr int kSketchWaves = 4;

template <int R, bool BF16>
__global__ void __launch_bounds__(kSketchWaves * kWave)
sketch_fast_kernel(const void* __restrict__ grad, float* __restrict__ h,
                   const float* __restrict__ g, const float* __restrict__ V,
                   float* __restrict__ S, int64_t d, int64_t n, int64_t m,
                   int64_t row_lo, int64_t row_hi, float eta, float a) {
  __shared__ float4 lds[kSketchWaves][kWave * kLdsRowF4];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int i = blockIdx.y;
  const int64_t p0 = row_lo + ((int64_t)blockIdx.x * kSketchWaves + wave) * kWave;
  if (p0 >= row_hi) return;
  const int sub = lane >> 3;   // row within an 8-row slab
  const int quad = lane & 7;   // 16-byte column group within the chunk
  const int64_t wbase = (int64_t)i * d;
  float4* tile = lds[wave];

  float s[R];
#pragma unroll
  for (int k = 0; k < R; ++k) s[k] = 0.0f;

  const int64_t nchunks = n / kChunk;
  for (int64_t c = 0; c < nchunks; ++c) {
    const int64_t col = c * kChunk + quad * 4;
    float4 xv[8], hv[8], gv[8];
    bool ok[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int64_t p = p0 + u * 8 + sub;
      ok[u] = p < row_hi;
      const int64_t e = wbase + p * n + col;
      if (ok[u]) {
        if constexpr (BF16) {
          const uint2 w = *reinterpret_cast<const uint2*>(
              static_cast<const uint16_t*>(grad) + e);
          xv[u] = make_float4(bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y));
        } else {
          xv[u] = *reinterpret_cast<const float4*>(static_cast<const float*>(grad) + e);
        }
        hv[u] = *reinterpret_cast<const float4*>(h + e);
        gv[u] = *reinterpret_cast<const float4*>(g + e);
      } else {
        xv[u] = hv[u] = gv[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      float4 hn;
      hn.x = fmaf(eta, xv[u].x, a * hv[u].x);
      hn.y = fmaf(eta, xv[u].y, a * hv[u].y);
      hn.z = fmaf(eta, xv[u].z, a * hv[u].z);
      hn.w = fmaf(eta, xv[u].w, a * hv[u].w);
      if (ok[u]) {
        const int64_t p = p0 + u * 8 + sub;
        *reinterpret_cast<float4*>(h + wbase + p * n + col) = hn;
      }
      float4 dl;
      dl.x = hn.x - gv[u].x;
      dl.y = hn.y - gv[u].y;
      dl.z = hn.z - gv[u].z;
      dl.w = hn.w - gv[u].w;
      tile[(u * 8 + sub) * kLdsRowF4 + quad] = dl;
    }
    wave_lds_fence();
    const float* Vc = V + c * kChunk * R;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const float4 dv = tile[lane * kLdsRowF4 + q];
      const float e4[4] = {dv.x, dv.y, dv.z, dv.w};
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
#pragma unroll
        for (int k = 0; k < R; ++k)
          s[k] = fmaf(e4[jj], Vc[(q * 4 + jj) * R + k], s[k]);
      }
    }
    wave_lds_fence();
  }
  const int64_t p = p0 + lane;
  if (p < row_hi) {
    float* out = S + ((int64_t)i * m + p) * R;
#pragma unroll
    for (int k = 0; k < R; ++k) out[k] = s[k];
  }
}

// ---------------------------------------------------------------------------
// Streaming sketch, general path: one thread per (row, worker).  Any n, d, r
// and alignment.  First pass updates h over the row; then, for each k, one
// pass re-reads h (new) and g and runs that column's chain.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256)
sketch_generic_kernel(const void* __restrict__ grad, int32_t grad_bf16,
                      float* __restrict__ h, const float* __restrict__ g,
                      const float* __restrict__ V, float* __restrict__ S,
                      int64_t d, int64_t n, int64_t m, int32_t N, int32_t r,
                      int64_t row_lo, int64_t row_hi, float eta, float a) {
  const int64_t rows = row_hi - row_lo;
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tid >= rows * N) return;
  const int32_t i = (int32_t)(tid / rows);
  const int64_t p = row_lo + tid % rows;
  const int64_t base = (int64_t)i * d;
  const int64_t e0 = p * n;
  const int64_t len = (e0 + n <= d) ? n : d - e0;
  for (int64_t j = 0; j < len; ++j) {
    const int64_t e = base + e0 + j;
    float x;
    if (grad_bf16)
      x = __uint_as_float((uint32_t)static_cast<const uint16_t*>(grad)[e] << 16);
    else
      x = static_cast<const float*>(grad)[e];
    h[e] = fmaf(eta, x, a * h[e]);
  }
  for (int32_t k = 0; k < r; ++k) {
    float s = 0.0f;
    for (int64_t j = 0; j < len; ++j) {
      const int64_t e = base + e0 + j;
      const float dl = h[e] - g[e];
      s = fmaf(dl, V[j * r + k], s);
    }
    S[((int64_t)i * m + p) * r + k] = s;
  }
}

// ---------------------------------------------------------------------------
// Worker sum (the sketch All-Reduce of Alg. 1) and row importance (Eq. (4)):
// P[p][k] = S[0][p][k] + S[1][p][k] + ... (ascending worker order),
// sigma[p] = fma chain of P[p][k]^2 over ascending k.  Thread per row.
// Threads p < nb also reset bucket p's radix state for this step.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256)
reduce_importance_kernel(const float* __restrict__ S, float* __restrict__ sigma,
                         int64_t m, int32_t N, int32_t r,
                         const BucketDesc* __restrict__ buckets,
                         BucketState* __restrict__ state, int32_t nb) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p < nb) {
    BucketState st;
    st.prefix = 0u;
    st.mask = 0u;
    st.kleft = buckets[p].k;
    state[p] = st;
  }
  if (p >= m) return;
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

// ---------------------------------------------------------------------------
// Top-K selection (Eq. (4)) by radix select on the binary32 bit patterns of
// sigma >= +0 (unsigned order equals numeric order), per bucket.
//
//  1. Three histogram passes over the digits [31:21], [20:10], [9:0] of the
//     keys that share the digits found so far.  Each block histograms its
//     rows in LDS (integer atomics) and adds the non-zero bins to the bucket's
//     global histogram; the last block to finish walks every bucket's
//     histogram from the top bin down, fixes the next digit of the threshold
//     key and the number of rows still to take among equal keys, and clears
//     the histogram for the next pass.
//  2. Count: per block, rows above the threshold and rows equal to it; the
//     last block turns these into per-bucket exclusive prefixes.
//  3. Write: each block re-derives its flags, ranks the ties by row (the
//     lower row wins) and writes the selected rows in ascending order with
//     block-wide prefix sums.
// Integer atomics only; the result does not depend on scheduling.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t key_of(const float* sigma, int64_t p) {
  return __float_as_uint(sigma[p]);
}

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t v) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const uint32_t o = __shfl_up(v, off, kWave);
    if (lane >= off) v += o;
  }
  return v;
}

// Exclusive prefix sum over the block (blockDim.x == kSelectThreads); also
// returns the block total.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v,
                                                         uint32_t* total) {
  __shared__ uint32_t wsum[kSelectThreads / kWave];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const uint32_t incl = wave_inclusive_scan(v);
  if (lane == kWave - 1) wsum[wave] = incl;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kSelectThreads / kWave; ++w) {
    if (w < wave) before += wsum[w];
    all += wsum[w];
  }
  __syncthreads();
  *total = all;
  return before + incl - v;
}

__device__ __forceinline__ bool elect_last_block(uint32_t* counter) {
  __shared__ bool last;
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0)
    last = atomicAdd(counter, 1u) == gridDim.x - 1;
  __syncthreads();
  if (last) __threadfence();
  return last;
}

__device__ __forceinline__ uint32_t load_relaxed(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int PASS>
__global__ void __launch_bounds__(kSelectThreads)
radix_hist_kernel(const float* __restrict__ sigma, SelectWorkspace ws) {
  constexpr int kShift = PASS == 0 ? 21 : (PASS == 1 ? 10 : 0);
  constexpr int kBits = PASS == 2 ? 10 : 11;
  constexpr uint32_t kDigitMask = (1u << kBits) - 1u;
  constexpr int kBins = 1 << kBits;
  __shared__ uint32_t hist[kRadixBins];
  for (int b = threadIdx.x; b < kBins; b += kSelectThreads) hist[b] = 0u;
  __syncthreads();

  const BlockDesc bd = ws.blocks[blockIdx.x];
  const BucketDesc bk = ws.buckets[bd.bucket];
  if (bk.mode == kSelectRadix) {
    const BucketState st = ws.state[bd.bucket];
    const int64_t r0 = bd.lo + (int64_t)threadIdx.x * kRowsPerThread;
#pragma unroll
    for (int u = 0; u < kRowsPerThread; ++u) {
      const int64_t p = r0 + u;
      if (p < bd.hi) {
        const uint32_t key = key_of(sigma, p);
        if ((key & st.mask) == st.prefix)
          atomicAdd(&hist[(key >> kShift) & kDigitMask], 1u);
      }
    }
  }
  __syncthreads();
  if (bk.mode == kSelectRadix) {
    uint32_t* gh = ws.ghist + (int64_t)bd.bucket * kRadixBins;
    for (int b = threadIdx.x; b < kBins; b += kSelectThreads) {
      const uint32_t c = hist[b];
      if (c != 0u) atomicAdd(&gh[b], c);
    }
  }
  if (!elect_last_block(ws.counter)) return;

  // Last block: fix one digit per bucket, one wave per bucket.
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  constexpr int kPerLane = kBins / kWave;
  for (int32_t b = wave; b < ws.nb; b += kSelectThreads / kWave) {
    if (ws.buckets[b].mode != kSelectRadix) continue;
    uint32_t* gh = ws.ghist + (int64_t)b * kRadixBins;
    BucketState st = ws.state[b];
    // lane 0 owns the top kPerLane bins, lane 1 the next ones, ...
    const int top = kBins - 1 - lane * kPerLane;
    uint32_t cnt[kPerLane];
    uint32_t lane_sum = 0;
#pragma unroll
    for (int u = 0; u < kPerLane; ++u) {
      cnt[u] = load_relaxed(&gh[top - u]);
      lane_sum += cnt[u];
    }
    const uint32_t incl = wave_inclusive_scan(lane_sum);
    const uint32_t excl = incl - lane_sum;
    const uint64_t kleft = (uint64_t)st.kleft;
    const bool mine = (uint64_t)excl < kleft && kleft <= (uint64_t)incl;
    const uint64_t who = __ballot(mine);
    const int src = who ? __ffsll((unsigned long long)who) - 1 : 0;
    uint32_t digit = 0, above = 0;
    if (mine) {
      uint32_t cum = excl;
#pragma unroll
      for (int u = 0; u < kPerLane; ++u) {
        if ((uint64_t)cum + cnt[u] >= kleft) {
          digit = (uint32_t)(top - u);
          above = cum;
          break;
        }
        cum += cnt[u];
      }
    }
    digit = __shfl(digit, src, kWave);
    above = __shfl(above, src, kWave);
#pragma unroll
    for (int u = 0; u < kPerLane; ++u) gh[top - u] = 0u;
    if (lane == 0) {
      st.prefix |= digit << kShift;
      st.mask |= kDigitMask << kShift;
      st.kleft = (int64_t)(kleft - above);
      ws.state[b] = st;
    }
  }
  if (threadIdx.x == 0) *ws.counter = 0u;
}

__global__ void __launch_bounds__(kSelectThreads)
select_count_kernel(const float* __restrict__ sigma, SelectWorkspace ws) {
  const BlockDesc bd = ws.blocks[blockIdx.x];
  const BucketDesc bk = ws.buckets[bd.bucket];
  uint32_t gt = 0, eq = 0;
  if (bk.mode == kSelectRadix) {
    const uint32_t T = ws.state[bd.bucket].prefix;
    const int64_t r0 = bd.lo + (int64_t)threadIdx.x * kRowsPerThread;
#pragma unroll
    for (int u = 0; u < kRowsPerThread; ++u) {
      const int64_t p = r0 + u;
      if (p < bd.hi) {
        const uint32_t key = key_of(sigma, p);
        gt += key > T;
        eq += key == T;
      }
    }
  }
  uint32_t tgt, teq;
  block_exclusive_scan(gt, &tgt);
  block_exclusive_scan(eq, &teq);
  if (threadIdx.x == 0) {
    ws.blockcnt[2 * blockIdx.x] = tgt;
    ws.blockcnt[2 * blockIdx.x + 1] = teq;
  }
  if (!elect_last_block(ws.counter)) return;

  // Last block: exclusive prefix of the block counts within each bucket.
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  for (int32_t b = wave; b < ws.nb; b += kSelectThreads / kWave) {
    const BucketDesc bb = ws.buckets[b];
    uint32_t run_gt = 0, run_eq = 0;
    for (int32_t base = 0; base < bb.nblk; base += kWave) {
      const int32_t blk = bb.first_blk + base + lane;
      const bool in = base + lane < bb.nblk;
      const uint32_t cg = in ? load_relaxed(&ws.blockcnt[2 * blk]) : 0u;
      const uint32_t ce = in ? load_relaxed(&ws.blockcnt[2 * blk + 1]) : 0u;
      const uint32_t ig = wave_inclusive_scan(cg);
      const uint32_t ie = wave_inclusive_scan(ce);
      if (in) {
        ws.blockbase[2 * blk] = run_gt + ig - cg;
        ws.blockbase[2 * blk + 1] = run_eq + ie - ce;
      }
      run_gt += __shfl(ig, kWave - 1, kWave);
      run_eq += __shfl(ie, kWave - 1, kWave);
    }
  }
  if (threadIdx.x == 0) *ws.counter = 0u;
}

__global__ void __launch_bounds__(kSelectThreads)
select_write_kernel(const float* __restrict__ sigma, SelectWorkspace ws,
                    int32_t* __restrict__ out_idx) {
  const BlockDesc bd = ws.blocks[blockIdx.x];
  const BucketDesc bk = ws.buckets[bd.bucket];
  const int64_t r0 = bd.lo + (int64_t)threadIdx.x * kRowsPerThread;
  if (bk.mode == kSelectNone) return;
  if (bk.mode == kSelectAll) {
    for (int u = 0; u < kRowsPerThread; ++u) {
      const int64_t p = r0 + u;
      if (p < bd.hi) out_idx[bk.out_off + (p - bk.lo)] = (int32_t)p;
    }
    return;
  }
  const BucketState st = ws.state[bd.bucket];
  const uint32_t T = st.prefix;
  const uint64_t kleft = (uint64_t)st.kleft;
  uint32_t keys[kRowsPerThread];
  uint32_t n_eq = 0;
#pragma unroll
  for (int u = 0; u < kRowsPerThread; ++u) {
    const int64_t p = r0 + u;
    keys[u] = p < bd.hi ? key_of(sigma, p) : 0u;
    n_eq += (p < bd.hi) && keys[u] == T;
  }
  uint32_t tot;
  const uint32_t eq_before =
      ws.blockbase[2 * blockIdx.x + 1] + block_exclusive_scan(n_eq, &tot);
  // selected rows of this thread, in row order
  uint32_t n_sel = 0;
  {
    uint32_t rank = eq_before;
#pragma unroll
    for (int u = 0; u < kRowsPerThread; ++u) {
      const int64_t p = r0 + u;
      if (p < bd.hi) {
        if (keys[u] > T) {
          ++n_sel;
        } else if (keys[u] == T) {
          n_sel += (uint64_t)rank < kleft;
          ++rank;
        }
      }
    }
  }
  const uint32_t gt_base = ws.blockbase[2 * blockIdx.x];
  const uint32_t eq_base = ws.blockbase[2 * blockIdx.x + 1];
  const uint64_t taken_ties = (uint64_t)eq_base < kleft ? eq_base : kleft;
  int64_t pos = bk.out_off + (int64_t)gt_base + (int64_t)taken_ties +
                block_exclusive_scan(n_sel, &tot);
  uint32_t rank = eq_before;
#pragma unroll
  for (int u = 0; u < kRowsPerThread; ++u) {
    const int64_t p = r0 + u;
    if (p < bd.hi) {
      bool sel = false;
      if (keys[u] > T) {
        sel = true;
      } else if (keys[u] == T) {
        sel = (uint64_t)rank < kleft;
        ++rank;
      }
      // pos stays below the bucket's end by construction; the bound keeps a
      // broken invariant from writing outside out_idx.
      if (sel && pos < bk.out_off + bk.k) out_idx[pos++] = (int32_t)p;
    }
  }
}

// ---------------------------------------------------------------------------
// Gather + worker sum + error-feedback update (Eq. (5), Alg. 1's payload
// All-Reduce, Eq. (11b)).  Thread per (selected row, 4 columns) on the
// vectorised path: for each worker in ascending order Delta = h - g,
// agg += Delta, g = g + Delta.  Rows are contiguous, so every access is a
// coalesced 16-byte access.  Columns past d give agg = +0.
// ---------------------------------------------------------------------------
constexpr int kMaxUnrolledWorkers = 8;

__global__ void __launch_bounds__(256)
gather_update_fast_kernel(const float* __restrict__ h, float* __restrict__ g,
                          const int32_t* __restrict__ idx,
                          float* __restrict__ agg, int64_t K_total, int64_t d,
                          int64_t n, int64_t m, int32_t N) {
  const int64_t per_row = n / 4;
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tid >= K_total * per_row) return;
  const int64_t q = tid / per_row;
  const int64_t col = (tid - q * per_row) * 4;
  const int64_t p = idx[q];
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  if (p < 0 || p >= m) {  // not a row: leave the state alone
    *reinterpret_cast<float4*>(agg + q * n + col) = acc;
    return;
  }
  const int64_t e = p * n + col;
  if (e + 4 <= d) {
    for (int32_t i0 = 0; i0 < N; i0 += kMaxUnrolledWorkers) {
      const int32_t cnt = N - i0 < kMaxUnrolledWorkers ? N - i0 : kMaxUnrolledWorkers;
      float4 hv[kMaxUnrolledWorkers], gv[kMaxUnrolledWorkers];
#pragma unroll
      for (int u = 0; u < kMaxUnrolledWorkers; ++u) {
        if (u < cnt) {
          const int64_t at = (int64_t)(i0 + u) * d + e;
          hv[u] = *reinterpret_cast<const float4*>(h + at);
          gv[u] = *reinterpret_cast<const float4*>(g + at);
        }
      }
#pragma unroll
      for (int u = 0; u < kMaxUnrolledWorkers; ++u) {
        if (u < cnt) {
          float4 dl;
          dl.x = hv[u].x - gv[u].x;
          dl.y = hv[u].y - gv[u].y;
          dl.z = hv[u].z - gv[u].z;
          dl.w = hv[u].w - gv[u].w;
          if (i0 + u == 0) {
            acc = dl;
          } else {
            acc.x = acc.x + dl.x;
            acc.y = acc.y + dl.y;
            acc.z = acc.z + dl.z;
            acc.w = acc.w + dl.w;
          }
          float4 gn;
          gn.x = gv[u].x + dl.x;
          gn.y = gv[u].y + dl.y;
          gn.z = gv[u].z + dl.z;
          gn.w = gv[u].w + dl.w;
          *reinterpret_cast<float4*>(g + (int64_t)(i0 + u) * d + e) = gn;
        }
      }
    }
  } else {
    float a4[4] = {0.f, 0.f, 0.f, 0.f};
    for (int jj = 0; jj < 4; ++jj) {
      if (e + jj >= d) break;
      for (int32_t i = 0; i < N; ++i) {
        const int64_t at = (int64_t)i * d + e + jj;
        const float dl = h[at] - g[at];
        a4[jj] = (i == 0) ? dl : a4[jj] + dl;
        g[at] = g[at] + dl;
      }
    }
    acc = make_float4(a4[0], a4[1], a4[2], a4[3]);
  }
  *reinterpret_cast<float4*>(agg + q * n + col) = acc;
}

__global__ void __launch_bounds__(256)
gather_update_generic_kernel(const float* __restrict__ h, float* __restrict__ g,
                             const int32_t* __restrict__ idx,
                             float* __restrict__ agg, int64_t K_total,
                             int64_t d, int64_t n, int64_t m, int32_t N) {
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tid >= K_total * n) return;
  const int64_t q = tid / n;
  const int64_t j = tid - q * n;
  const int64_t p = idx[q];
  const int64_t e = p * n + j;
  float acc = 0.0f;
  if (p >= 0 && p < m && e < d) {
    for (int32_t i = 0; i < N; ++i) {
      const int64_t at = (int64_t)i * d + e;
      const float dl = h[at] - g[at];
      acc = (i == 0) ? dl : acc + dl;
      g[at] = g[at] + dl;
    }
  }
  agg[tid] = acc;
}

inline unsigned blocks_for(int64_t work, int threads) {
  return (unsigned)((work + threads - 1) / threads);
}

}  // namespace

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
hipError_t launch_sketch(bool fast, const void* grad, int32_t grad_bf16,
                         float* h, const float* g, const float* V, float* S,
                         int64_t d, int64_t n, int64_t m, int32_t N, int32_t r,
                         int64_t row_lo, int64_t row_hi, float eta, float a,
                         hipStream_t stream) {
  const int64_t rows = row_hi - row_lo;
  if (rows <= 0) return hipSuccess;
  if (fast) {
    const int64_t rows_per_block = (int64_t)kSketchWaves * kWave;
    const dim3 grid(blocks_for(rows, (int)rows_per_block), (unsigned)N);
    const dim3 block(kSketchWaves * kWave);
#define ARC_SKETCH_CASE(RR)                                                      \
  case RR:                                                                       \
    if (grad_bf16)                                                               \
      hipLaunchKernelGGL((sketch_fast_kernel<RR, true>), grid, block, 0, stream,  \
                         grad, h, g, V, S, d, n, m, row_lo, row_hi, eta, a);     \
    else                                                                         \
      hipLaunchKernelGGL((sketch_fast_kernel<RR, false>), grid, block, 0, stream, \
                         grad, h, g, V, S, d, n, m, row_lo, row_hi, eta, a);     \
    break;
    switch (r) {
      ARC_SKETCH_CASE(1)
      ARC_SKETCH_CASE(2)
      ARC_SKETCH_CASE(4)
      ARC_SKETCH_CASE(8)
      default:
        return hipErrorInvalidValue;
    }
#undef ARC_SKETCH_CASE
  } else {
    hipLaunchKernelGGL(sketch_generic_kernel, dim3(blocks_for(rows * N, 256)),
                       dim3(256), 0, stream, grad, grad_bf16, h, g, V, S, d, n,
                       m, N, r, row_lo, row_hi, eta, a);
  }
  return hipGetLastError();
}

hipError_t launch_reduce_importance(const float* S, float* sigma, int64_t m,
                                    int32_t N, int32_t r,
                                    const SelectWorkspace& ws,
                                    hipStream_t stream) {
  hipLaunchKernelGGL(reduce_importance_kernel, dim3(blocks_for(m, 256)),
                     dim3(256), 0, stream, S, sigma, m, N, r, ws.buckets,
                     ws.state, ws.nb);
  return hipGetLastError();
}

hipError_t launch_select(const float* sigma, const SelectWorkspace& ws,
                         int32_t* out_idx, hipStream_t stream) {
  const dim3 grid((unsigned)ws.nblk), block(kSelectThreads);
  hipLaunchKernelGGL(radix_hist_kernel<0>, grid, block, 0, stream, sigma, ws);
  hipLaunchKernelGGL(radix_hist_kernel<1>, grid, block, 0, stream, sigma, ws);
  hipLaunchKernelGGL(radix_hist_kernel<2>, grid, block, 0, stream, sigma, ws);
  hipLaunchKernelGGL(select_count_kernel, grid, block, 0, stream, sigma, ws);
  hipLaunchKernelGGL(select_write_kernel, grid, block, 0, stream, sigma, ws,
                     out_idx);
  return hipGetLastError();
}

hipError_t launch_gather_update(bool fast, const float* h, float* g,
                                const int32_t* idx, float* agg, int64_t K_total,
                                int64_t d, int64_t n, int64_t m, int32_t N,
                                hipStream_t stream) {
  if (K_total <= 0) return hipSuccess;
  if (fast) {
    hipLaunchKernelGGL(gather_update_fast_kernel,
                       dim3(blocks_for(K_total * (n / 4), 256)), dim3(256), 0,
                       stream, h, g, idx, agg, K_total, d, n, m, N);
  } else {
    hipLaunchKernelGGL(gather_update_generic_kernel,
                       dim3(blocks_for(K_total * n, 256)), dim3(256), 0, stream,
                       h, g, idx, agg, K_total, d, n, m, N);
  }
  return hipGetLastError();
}

}  // namespace arc
