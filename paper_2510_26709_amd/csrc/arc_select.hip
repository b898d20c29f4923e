// Top-K row selection of the compressor step (Eq. (4): I = arg top_K(Sigma)),
// independently per bucket, with ties going to the lower row and the rows of
// each bucket returned in ascending order.
//
// Radix select on the binary32 bit patterns of Sigma >= +0 (their unsigned
// order is the numeric order), digits [31:21], [20:10], [9:0]:
//   pass 0..2  each block histograms, in LDS, the digit of the keys that share
//              the digits already fixed and adds its non-zero bins to the
//              bucket's global histogram of that pass (integer atomics);
//   pass p > 0 first fixes digit p-1: every block of the bucket reads the
//              radix state after digit p-2 (slot p-2, written by the previous
//              kernel) and walks the previous histogram from the top bin down
//              to the bin holding the kleft-th largest remaining key (all
//              blocks reach the same answer); the bucket's first block records
//              the new state in slot p-1, which no block of the same launch
//              reads;
//   count      fixes the last digit (the threshold key T and how many keys
//              equal to T are kept) and counts, per block, keys above and equal
//              to T;
//   write      each block adds up the counts of the blocks before it, ranks
//              its ties by row, writes the selected rows in order with
//              block-wide prefix sums, and clears the histograms for the next
//              step.
// No kernel waits on another block: there are no grid-wide counters, every
// global location a kernel reads was written by an earlier launch on the
// stream (the state slots are per pass for this reason), and the result does
// not depend on scheduling.
// The selection is a chain of short launches, so latency rather than
// bandwidth bounds it: every kernel reads its keys in coalesced tiles whose
// loads are all in flight together, the first tile requested before the
// radix state's dependent reads, and the write kernel stages each tile in
// LDS so that every thread walks its own contiguous rows there.
//
// When every bucket has at most kSmallBucketRows rows, one launch of
// select_small_kernel does all of this instead, one 1024-thread workgroup per
// bucket, with the bucket's keys, the histograms, the radix state and the
// counts in LDS.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "arc_device.h"
#include "arc_internal.h"

namespace arc {
namespace {

template <int PASS>
struct RadixDigit {
  static constexpr int kShift = PASS == 0 ? 21 : (PASS == 1 ? 10 : 0);
  static constexpr int kBits = PASS == 2 ? 10 : 11;
  static constexpr uint32_t kMask = (1u << kBits) - 1u;
  static constexpr int kBins = 1 << kBits;
};

// The multi-block kernels take a block's rows in tiles of kTileRows: thread t
// holds key u of a tile (row tile + u * kSelectThreads + t) in a register, so
// that a tile's loads are coalesced and all in flight together.
constexpr int kTileKeys = 32;
constexpr int64_t kTileRows = (int64_t)kSelectThreads * kTileKeys;
static_assert(kTileRows < (1 << 16), "a tile's key counts fit 16 bits");

__device__ __forceinline__ void load_tile(const float* __restrict__ sigma, int64_t lo, int64_t hi,
                                          uint32_t (&keys)[kTileKeys]) {
#pragma unroll
  for (int u = 0; u < kTileKeys; ++u) {
    const int64_t p = lo + (int64_t)u * kSelectThreads + threadIdx.x;
    keys[u] = p < hi ? __float_as_uint(sigma[p]) : 0u;
  }
}

__device__ __forceinline__ const uint32_t* hist_of(const SelectWorkspace& ws,
                                                   int pass, int32_t b) {
  return ws.hist + ((int64_t)pass * ws.nb + b) * kRadixBins;
}
__device__ __forceinline__ uint32_t* hist_of_mut(const SelectWorkspace& ws,
                                                 int pass, int32_t b) {
  return ws.hist + ((int64_t)pass * ws.nb + b) * kRadixBins;
}

// Executed by one full wave: append digit PASS to st using the bucket's
// histogram of that pass.
template <int PASS>
__device__ BucketState fix_digit(const uint32_t* gh, BucketState st) {
  using D = RadixDigit<PASS>;
  constexpr int kPerLane = D::kBins / kWave;
  const int lane = threadIdx.x & (kWave - 1);
  // lane 0 owns the top kPerLane bins, lane 1 the next ones, ...
  const int top = D::kBins - 1 - lane * kPerLane;
  uint32_t cnt[kPerLane];
  uint32_t lane_sum = 0;
#pragma unroll
  for (int u = 0; u < kPerLane; ++u) {
    cnt[u] = gh[top - u];
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
  st.prefix |= digit << D::kShift;
  st.mask |= D::kMask << D::kShift;
  st.kleft = (int64_t)(kleft - above);
  return st;
}

// Radix state of bucket b after digits 0..q (slot q of the per-pass states).
__device__ __forceinline__ BucketState* state_slot(const SelectWorkspace& ws, int q, int32_t b) {
  return ws.state + (int64_t)q * ws.nb + b;
}

// Radix state entering pass PASS (digits 0..PASS-1 fixed), computed by wave 0
// and shared with the block.  It starts from slot PASS-2, written by the
// previous kernel, and the bucket's first block stores the result in slot
// PASS-1 for the next kernel: no slot is both read and written in a launch.
template <int PASS>
__device__ BucketState state_before_pass(const SelectWorkspace& ws,
                                         const BucketDesc& bk, int32_t b) {
  __shared__ BucketState sh;
  if (threadIdx.x < kWave) {
    BucketState st;
    if constexpr (PASS <= 1) {
      st.prefix = 0u;
      st.mask = 0u;
      st.kleft = bk.k;
    } else {
      st = *state_slot(ws, PASS - 2, b);
    }
    if constexpr (PASS >= 1) st = fix_digit<PASS - 1>(hist_of(ws, PASS - 1, b), st);
    if (threadIdx.x == 0) {
      sh = st;
      if (PASS >= 1 && (int32_t)blockIdx.x == bk.first_blk) *state_slot(ws, PASS - 1, b) = st;
    }
  }
  __syncthreads();
  return sh;
}

template <int PASS>
__global__ void __launch_bounds__(kSelectThreads)
radix_pass_kernel(const float* __restrict__ sigma, SelectWorkspace ws) {
  using D = RadixDigit<PASS>;
  __shared__ uint32_t lhist[kRadixBins];
  const BlockDesc bd = ws.blocks[blockIdx.x];
  const BucketDesc bk = ws.buckets[bd.bucket];
  if (bk.mode != kSelectRadix) return;  // whole block
  for (int b = threadIdx.x; b < D::kBins; b += kSelectThreads) lhist[b] = 0u;
  // The first tile's keys are requested before the radix state, whose
  // dependent reads then overlap them.
  uint32_t keys[kTileKeys];
  load_tile(sigma, bd.lo, bd.hi, keys);
  const BucketState st = state_before_pass<PASS>(ws, bk, bd.bucket);  // syncs
  for (int64_t tile = bd.lo; tile < bd.hi; tile += kTileRows) {
#pragma unroll
    for (int u = 0; u < kTileKeys; ++u) {
      const int64_t p = tile + (int64_t)u * kSelectThreads + threadIdx.x;
      if (p < bd.hi && (keys[u] & st.mask) == st.prefix)
        atomicAdd(&lhist[(keys[u] >> D::kShift) & D::kMask], 1u);
    }
    if (tile + kTileRows < bd.hi) load_tile(sigma, tile + kTileRows, bd.hi, keys);
  }
  __syncthreads();
  uint32_t* gh = hist_of_mut(ws, PASS, bd.bucket);
  for (int b = threadIdx.x; b < D::kBins; b += kSelectThreads) {
    const uint32_t c = lhist[b];
    if (c != 0u) atomicAdd(&gh[b], c);
  }
}

__global__ void __launch_bounds__(kSelectThreads)
select_count_kernel(const float* __restrict__ sigma, SelectWorkspace ws) {
  __shared__ uint32_t part[2][kSelectThreads / kWave];
  const BlockDesc bd = ws.blocks[blockIdx.x];
  const BucketDesc bk = ws.buckets[bd.bucket];
  if (bk.mode != kSelectRadix) return;  // whole block
  uint32_t keys[kTileKeys];
  load_tile(sigma, bd.lo, bd.hi, keys);
  const BucketState st = state_before_pass<3>(ws, bk, bd.bucket);  // syncs
  const uint32_t T = st.prefix;
  uint32_t gt = 0, eq = 0;
  for (int64_t tile = bd.lo; tile < bd.hi; tile += kTileRows) {
#pragma unroll
    for (int u = 0; u < kTileKeys; ++u) {
      const bool valid = tile + (int64_t)u * kSelectThreads + threadIdx.x < bd.hi;
      gt += valid && keys[u] > T;
      eq += valid && keys[u] == T;
    }
    if (tile + kTileRows < bd.hi) load_tile(sigma, tile + kTileRows, bd.hi, keys);
  }
  gt = wave_sum(gt);
  eq = wave_sum(eq);
  const int wave = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) {
    part[0][wave] = gt;
    part[1][wave] = eq;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t tg = 0, te = 0;
    for (int w = 0; w < kSelectThreads / kWave; ++w) {
      tg += part[0][w];
      te += part[1][w];
    }
    ws.blockcnt[2 * blockIdx.x] = tg;
    ws.blockcnt[2 * blockIdx.x + 1] = te;
  }
}

// Exclusive prefix sum over the block (blockDim.x == THREADS); *total gets
// the block's sum.
template <int THREADS = kSelectThreads>
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* total = nullptr) {
  __shared__ uint32_t wsum[THREADS / kWave];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const uint32_t incl = wave_inclusive_scan(v);
  if (lane == kWave - 1) wsum[wave] = incl;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < THREADS / kWave; ++w) {
    if (w < wave) before += wsum[w];
    all += wsum[w];
  }
  __syncthreads();
  if (total != nullptr) *total = all;
  return before + incl - v;
}

// LDS words per thread of a staged tile: its kTileKeys contiguous rows plus
// one word of padding, so that the lanes of a wave, each reading its own
// rows, hit distinct banks.
constexpr int kTilePitch = kTileKeys + 1;

__global__ void __launch_bounds__(kSelectThreads)
select_write_kernel(const float* __restrict__ sigma, SelectWorkspace ws,
                    int32_t* __restrict__ out_idx) {
  __shared__ uint32_t staged[kSelectThreads * kTilePitch];
  __shared__ uint32_t sh_before[2];
  const BlockDesc bd = ws.blocks[blockIdx.x];
  const BucketDesc bk = ws.buckets[bd.bucket];
  if (bk.mode == kSelectNone) return;  // whole block
  if (bk.mode == kSelectAll) {
    for (int64_t p = bd.lo + threadIdx.x; p < bd.hi; p += kSelectThreads)
      out_idx[bk.out_off + (p - bk.lo)] = (int32_t)p;
    return;
  }
  // The first tile's keys are requested before the state and counts below.
  uint32_t keys[kTileKeys];
  load_tile(sigma, bd.lo, bd.hi, keys);
  const BucketState st = *state_slot(ws, kRadixPasses - 1, bd.bucket);
  const uint32_t T = st.prefix;
  const uint64_t kleft = (uint64_t)st.kleft;
  // Keys above / equal to T in the bucket's earlier blocks.
  if (threadIdx.x < kWave) {
    uint32_t g_before = 0, e_before = 0;
    for (int32_t j = bk.first_blk + (int32_t)threadIdx.x; j < (int32_t)blockIdx.x; j += kWave) {
      g_before += ws.blockcnt[2 * j];
      e_before += ws.blockcnt[2 * j + 1];
    }
    g_before = wave_sum(g_before);
    e_before = wave_sum(e_before);
    if (threadIdx.x == 0) {
      sh_before[0] = g_before;
      sh_before[1] = e_before;
    }
  }
  // This block's share of clearing the bucket's three histograms.
  {
    const int32_t jb = (int32_t)blockIdx.x - bk.first_blk;
    const int64_t total = (int64_t)kRadixPasses * kRadixBins;
    for (int64_t e = (int64_t)jb * kSelectThreads + threadIdx.x; e < total;
         e += (int64_t)bk.nblk * kSelectThreads)
      hist_of_mut(ws, (int)(e / kRadixBins), bd.bucket)[e % kRadixBins] = 0u;
  }
  __syncthreads();
  // Keys above / equal to T before the current tile: earlier blocks, then
  // this block's earlier tiles.
  uint32_t gt_before = sh_before[0], eq_before = sh_before[1];
  const int64_t end = bk.out_off + bk.k;
  for (int64_t tile = bd.lo; tile < bd.hi; tile += kTileRows) {
    // Row tile + r goes to word (r / kTileKeys) * kTilePitch + r % kTileKeys:
    // after the barrier, thread t reads rows tile + t*kTileKeys onwards, in
    // order, so thread order is row order.
#pragma unroll
    for (int u = 0; u < kTileKeys; ++u) {
      const int r = u * kSelectThreads + (int)threadIdx.x;
      staged[(r / kTileKeys) * kTilePitch + r % kTileKeys] = keys[u];
    }
    __syncthreads();
    const int64_t next = tile + kTileRows;
    if (next < bd.hi) load_tile(sigma, next, bd.hi, keys);
    const int64_t r0 = tile + (int64_t)threadIdx.x * kTileKeys;
    const int nr = r0 >= bd.hi ? 0 : (bd.hi - r0 < kTileKeys ? (int)(bd.hi - r0) : kTileKeys);
    const uint32_t* mine = staged + threadIdx.x * kTilePitch;
    uint32_t n_gt = 0, n_eq = 0;
#pragma unroll
    for (int u = 0; u < kTileKeys; ++u) {
      const uint32_t key = mine[u];
      n_gt += u < nr && key > T;
      n_eq += u < nr && key == T;
    }
    // One scan for both counts: at most kTileRows < 2^16 keys a tile, so the
    // two 16-bit halves never carry into each other.
    uint32_t tile_both = 0;
    const uint32_t both_excl = block_exclusive_scan(n_gt | (n_eq << 16), &tile_both);
    const uint64_t eq_rank0 = (uint64_t)eq_before + (both_excl >> 16);
    // ties this thread keeps: ranks eq_rank0 .. eq_rank0 + n_eq - 1 below kleft
    const uint64_t ties_kept =
        eq_rank0 >= kleft ? 0 : ((kleft - eq_rank0) < n_eq ? (kleft - eq_rank0) : n_eq);
    const uint32_t n_sel = n_gt + (uint32_t)ties_kept;
    const uint64_t taken_before = (uint64_t)eq_before < kleft ? eq_before : kleft;
    int64_t pos = bk.out_off + (int64_t)gt_before + (int64_t)taken_before +
                  block_exclusive_scan(n_sel);
    uint64_t rank = eq_rank0;
#pragma unroll
    for (int u = 0; u < kTileKeys; ++u) {
      const uint32_t key = mine[u];
      bool sel = false;
      if (u < nr) {
        if (key > T) {
          sel = true;
        } else if (key == T) {
          sel = rank < kleft;
          ++rank;
        }
      }
      // pos stays below the bucket's end by construction; the bound keeps a
      // broken invariant from writing outside out_idx.
      if (sel && pos < end) out_idx[pos++] = (int32_t)(r0 + u);
    }
    gt_before += tile_both & 0xffffu;
    eq_before += tile_both >> 16;
    __syncthreads();  // this tile's reads of `staged` before the next tile's writes
  }
}

// Word of key p in the small kernel's LDS copy of a bucket: one word of
// padding after every 32 keys, so that both the passes (lane l reads key
// u * kSmallSelectThreads + l) and the write (thread t reads its rpt
// consecutive keys) spread a wave's reads over the banks.
__device__ __forceinline__ int32_t small_word(int32_t p) { return p + (p >> 5); }

// Histogram of digit PASS of the bucket's keys that match st, into the
// block's LDS histogram (cleared here), then the digit fixed from it.  The
// bucket's `rows` keys are in LDS.
template <int PASS>
__device__ BucketState small_pass(const uint32_t* keys, int32_t rows, BucketState st,
                                  uint32_t* lhist, BucketState* sh) {
  using D = RadixDigit<PASS>;
  for (int b = threadIdx.x; b < D::kBins; b += kSmallSelectThreads) lhist[b] = 0u;
  __syncthreads();
  for (int32_t p = (int32_t)threadIdx.x; p < rows; p += kSmallSelectThreads) {
    const uint32_t key = keys[small_word(p)];
    if ((key & st.mask) == st.prefix) atomicAdd(&lhist[(key >> D::kShift) & D::kMask], 1u);
  }
  __syncthreads();
  if (threadIdx.x < kWave) {
    const BucketState next = fix_digit<PASS>(lhist, st);
    if (threadIdx.x == 0) *sh = next;
  }
  __syncthreads();
  return *sh;
}

// One workgroup per bucket: the bucket's keys are read once into LDS (the
// launch's dynamic LDS holds small_key_words(ws.small_rows) words), then the
// three radix passes and the write of the kept rows in ascending order, ties
// to the lower row (as the multi-block kernels, with the block's threads in
// the roles of the blocks), run from there.
// KEYS: keys per thread of the largest bucket (8 up to 8192 rows, else
// kSmallKeysPerThread), so that short buckets issue no masked-off loads.
template <int KEYS>
__global__ void __launch_bounds__(kSmallSelectThreads)
select_small_kernel(const float* __restrict__ sigma, SelectWorkspace ws,
                    int32_t* __restrict__ out_idx) {
  static_assert(KEYS <= kSmallKeysPerThread, "keys per thread");
  __shared__ uint32_t lhist[kRadixBins];
  __shared__ BucketState sh;
  extern __shared__ uint32_t keys[];
  const BucketDesc bk = ws.buckets[blockIdx.x];
  if (bk.mode == kSelectNone) return;  // whole block
  if (bk.mode == kSelectAll) {
    for (int64_t p = bk.lo + threadIdx.x; p < bk.hi; p += kSmallSelectThreads)
      out_idx[bk.out_off + (p - bk.lo)] = (int32_t)p;
    return;
  }
  // The host takes this kernel only when every bucket has at most
  // kSmallBucketRows rows and sizes the LDS for the largest; the bound keeps
  // a broken invariant inside LDS.
  const int64_t all = bk.hi - bk.lo;
  const int32_t cap = ws.small_rows < KEYS * kSmallSelectThreads ? ws.small_rows
                                                                 : KEYS * kSmallSelectThreads;
  const int32_t rows = (int32_t)(all < cap ? all : cap);
  {
    // All of a thread's loads are in flight before the first store.
    uint32_t k[KEYS];
#pragma unroll
    for (int u = 0; u < KEYS; ++u) {
      const int32_t p = u * kSmallSelectThreads + (int32_t)threadIdx.x;
      k[u] = p < rows ? __float_as_uint(sigma[bk.lo + p]) : 0u;
    }
#pragma unroll
    for (int u = 0; u < KEYS; ++u) {
      const int32_t p = u * kSmallSelectThreads + (int32_t)threadIdx.x;
      if (p < rows) keys[small_word(p)] = k[u];
    }
  }
  // (small_pass's first barrier orders these stores before any read.)
  BucketState st;
  st.prefix = 0u;
  st.mask = 0u;
  st.kleft = bk.k;
  st = small_pass<0>(keys, rows, st, lhist, &sh);
  st = small_pass<1>(keys, rows, st, lhist, &sh);
  st = small_pass<2>(keys, rows, st, lhist, &sh);
  const uint32_t T = st.prefix;
  const uint64_t kleft = (uint64_t)st.kleft;
  // Thread t owns rows [r0, r1), contiguous, so thread order is row order.
  const int32_t rpt = (rows + kSmallSelectThreads - 1) / kSmallSelectThreads;
  const int32_t r0 = (int32_t)threadIdx.x * rpt;
  const int32_t r1 = r0 + rpt < rows ? r0 + rpt : rows;
  uint32_t n_eq = 0, n_gt = 0;
  for (int32_t p = r0; p < r1; ++p) {
    const uint32_t key = keys[small_word(p)];
    n_gt += key > T;
    n_eq += key == T;
  }
  const uint64_t eq_rank0 = block_exclusive_scan<kSmallSelectThreads>(n_eq);
  const uint64_t ties_kept =
      eq_rank0 >= kleft ? 0 : ((kleft - eq_rank0) < n_eq ? (kleft - eq_rank0) : n_eq);
  int64_t pos = bk.out_off +
                block_exclusive_scan<kSmallSelectThreads>(n_gt + (uint32_t)ties_kept);
  const int64_t end = bk.out_off + bk.k;
  uint64_t rank = eq_rank0;
  for (int32_t p = r0; p < r1; ++p) {
    const uint32_t key = keys[small_word(p)];
    bool sel = key > T;
    if (key == T) {
      sel = rank < kleft;
      ++rank;
    }
    // pos stays below the bucket's end by construction; the bound keeps a
    // broken invariant from writing outside out_idx.
    if (sel && pos < end) out_idx[pos++] = (int32_t)(bk.lo + p);
  }
}

}  // namespace

hipError_t launch_select(const float* sigma, const SelectWorkspace& ws,
                         int32_t* out_idx, hipStream_t stream) {
  if (ws.small) {
    if (ws.any_output) {
      const size_t lds = (size_t)small_key_words(ws.small_rows) * sizeof(uint32_t);
      if (ws.small_rows <= 8 * kSmallSelectThreads)
        hipLaunchKernelGGL(select_small_kernel<8>, dim3((unsigned)ws.nb),
                           dim3(kSmallSelectThreads), lds, stream, sigma, ws, out_idx);
      else
        hipLaunchKernelGGL(select_small_kernel<kSmallKeysPerThread>, dim3((unsigned)ws.nb),
                           dim3(kSmallSelectThreads), lds, stream, sigma, ws, out_idx);
    }
    return hipGetLastError();
  }
  const dim3 grid((unsigned)ws.nblk), block(kSelectThreads);
  if (ws.any_radix) {
    hipLaunchKernelGGL(radix_pass_kernel<0>, grid, block, 0, stream, sigma, ws);
    hipLaunchKernelGGL(radix_pass_kernel<1>, grid, block, 0, stream, sigma, ws);
    hipLaunchKernelGGL(radix_pass_kernel<2>, grid, block, 0, stream, sigma, ws);
    hipLaunchKernelGGL(select_count_kernel, grid, block, 0, stream, sigma, ws);
  }
  if (ws.any_output)
    hipLaunchKernelGGL(select_write_kernel, grid, block, 0, stream, sigma, ws, out_idx);
  return hipGetLastError();
}

}  // namespace arc
