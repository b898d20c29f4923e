// Comparison compressors of Table I inside the same EF21M step: the kernels
// Rand-K and Top-K need beyond the ARC-Top-K pipeline (the row selection and
// the summed gather are shared with it).
//   Rand-K: Eq. (11a) over all coordinates, a uniform random key per row from
//   the shared seed, the arg-top-K of the keys, the summed gather.
//   Top-K: Eq. (11a) with every node's squared row norms of Delta (the sketch
//   kernels in norm mode), one selection per node, and a gather that returns
//   each node's own rows unsummed (the All-Gather payload).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "arc_device.h"
#include "arc_internal.h"

namespace arc {
namespace {

// h = fmaf(eta, grad, fl(a * h)), element-wise over the [N][d] batch.
template <bool BF16>
__global__ void __launch_bounds__(256)
momentum_vec_kernel(const void* __restrict__ grad, float* __restrict__ h, int64_t count,
                    float eta, float a) {
  const int64_t e = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (e >= count) return;
  float4 x;
  if constexpr (BF16) {
    const uint2 w = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(grad) + e);
    x = make_float4(bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y));
  } else {
    x = stream_load(reinterpret_cast<const float4*>(static_cast<const float*>(grad) + e));
  }
  float4 hv = stream_load(reinterpret_cast<const float4*>(h + e));
  hv.x = fmaf(eta, x.x, a * hv.x);
  hv.y = fmaf(eta, x.y, a * hv.y);
  hv.z = fmaf(eta, x.z, a * hv.z);
  hv.w = fmaf(eta, x.w, a * hv.w);
  stream_store(reinterpret_cast<float4*>(h + e), hv);
}

__global__ void __launch_bounds__(256)
momentum_scalar_kernel(const void* __restrict__ grad, int32_t grad_bf16, float* __restrict__ h,
                       int64_t count, float eta, float a) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= count) return;
  const float x =
      grad_bf16 ? __uint_as_float((uint32_t)static_cast<const uint16_t*>(grad)[e] << 16)
                : static_cast<const float*>(grad)[e];
  h[e] = fmaf(eta, x, a * h[e]);
}

// SplitMix64 (Steele, Lea & Flood, OOPSLA 2014): output number c of the
// stream seeded with `seed` is the variant-13 mix of seed + (c + 1) * gamma.
__device__ __forceinline__ uint64_t splitmix64_output(uint64_t seed, uint64_t c) {
  uint64_t z = seed + (c + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__global__ void __launch_bounds__(256)
randk_keys_kernel(uint64_t seed, int64_t t, int64_t m, float* __restrict__ keys) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= m) return;
  const uint64_t x = splitmix64_output(seed, (uint64_t)(t * m + p));
  keys[p] = (float)(uint32_t)(x >> 40);  // an integer below 2^24: exact
}

// Work item w of node i (one selected row x 4 columns): its bucket, the
// row's position q within the bucket's list, and the first column.
struct TopkItem {
  GatherBucket bk;
  int64_t q, col;
};

__device__ __forceinline__ TopkItem topk_item(const GatherBucket* __restrict__ buckets,
                                              int32_t nb, int64_t w) {
  int32_t lo = 0, hi = nb;  // last bucket whose work_off <= w
  while (hi - lo > 1) {
    const int32_t mid = (lo + hi) >> 1;
    if (buckets[mid].work_off <= w) lo = mid; else hi = mid;
  }
  TopkItem it;
  it.bk = buckets[lo];
  const int64_t per_row = (it.bk.cols + 3) / 4;
  const int64_t item = w - it.bk.work_off;
  it.q = item / per_row;
  it.col = (item - it.q * per_row) * 4;
  return it;
}

// One work item = one selected row x 4 columns of one node (see the
// launcher).  Each node's rows are its own; nothing is summed.  With `mark`
// (the model step), node i's row p is tagged mark[i*m + p] = stamp << 32 | q
// for the merge that follows.
__global__ void __launch_bounds__(256)
topk_gather_kernel(const float* __restrict__ h, float* __restrict__ g,
                   const int32_t* __restrict__ sel, int32_t* __restrict__ out_idx,
                   float* __restrict__ agg, const GatherBucket* __restrict__ buckets,
                   int32_t nb, int64_t work, int64_t K_total, int64_t payload, int64_t d,
                   int64_t m, int32_t N, int32_t vec, uint64_t* __restrict__ mark,
                   uint32_t stamp) {
  const int64_t w_all = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (w_all >= (int64_t)N * work) return;
  const int64_t i = w_all / work, w = w_all - i * work;
  const TopkItem it = topk_item(buckets, nb, w);
  const GatherBucket& bk = it.bk;
  const int64_t q = it.q, col = it.col;
  const int64_t pos = i * K_total + bk.out_off + q;
  const int64_t p = (int64_t)sel[pos] - i * m;  // row of the view
  const int64_t pr = p - bk.row0;               // row within the bucket
  // Only this node's rows of this bucket; the bounds keep a broken index from
  // touching memory outside the vectors.
  if (q >= bk.k || pr < 0 || pr >= bk.rows) return;
  if (col == 0) {
    out_idx[pos] = (int32_t)p;
    if (mark != nullptr) mark[i * m + p] = ((uint64_t)stamp << 32) | (uint64_t)q;
  }
  float* out = agg + i * payload + bk.agg_off + q * bk.cols + col;
  const int64_t e = bk.elem_off + pr * bk.cols + col;
  const int64_t ncols = bk.cols - col < 4 ? bk.cols - col : 4;
  const int64_t at = i * d + e;
  if (vec && bk.vec && e + 4 <= d) {
    const float4 hv = *reinterpret_cast<const float4*>(h + at);
    const float4 gv = *reinterpret_cast<const float4*>(g + at);
    const float4 dl = make_float4(hv.x - gv.x, hv.y - gv.y, hv.z - gv.z, hv.w - gv.w);
    *reinterpret_cast<float4*>(g + at) =
        make_float4(gv.x + dl.x, gv.y + dl.y, gv.z + dl.z, gv.w + dl.w);
    *reinterpret_cast<float4*>(out) = dl;
  } else {
    for (int64_t jj = 0; jj < ncols; ++jj) {
      if (e + jj >= d) {  // past d in a ragged last row
        out[jj] = 0.0f;
        continue;
      }
      const float dl = h[at + jj] - g[at + jj];
      g[at + jj] = g[at + jj] + dl;
      out[jj] = dl;
    }
  }
}

// Top-K's merge into G = sum_i g^(i) (Sec. III): every coordinate of a row
// some node kept gets the kept values of the nodes that kept it, summed in
// ascending node order (the first as it is, then plain additions), added to
// G.  Work items as in the gather; the item of the lowest node that kept a
// row does that row's columns, the others return.  mark holds this step's
// tags from the gather (older steps' tags carry another stamp).
__global__ void __launch_bounds__(256)
topk_merge_kernel(const float* __restrict__ agg, const int32_t* __restrict__ sel,
                  const uint64_t* __restrict__ mark, uint32_t stamp,
                  const GatherBucket* __restrict__ buckets, int32_t nb, int64_t work,
                  int64_t K_total, int64_t payload, int64_t d, int64_t m, int32_t N,
                  float* __restrict__ G, int32_t vec) {
  const int64_t w_all = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (w_all >= (int64_t)N * work) return;
  const int64_t i = w_all / work, w = w_all - i * work;
  const TopkItem it = topk_item(buckets, nb, w);
  const GatherBucket& bk = it.bk;
  const int64_t q = it.q, col = it.col;
  const int64_t p = (int64_t)sel[i * K_total + bk.out_off + q] - i * m;
  const int64_t pr = p - bk.row0;
  if (q >= bk.k || pr < 0 || pr >= bk.rows) return;
  for (int64_t j = 0; j < i; ++j)
    if ((uint32_t)(mark[j * m + p] >> 32) == stamp) return;  // a lower node owns the row
  const int64_t e = bk.elem_off + pr * bk.cols + col;
  const int64_t ncols = bk.cols - col < 4 ? bk.cols - col : 4;
  if (vec && bk.vec && e + 4 <= d) {
    // four columns as one 16-byte access each (rows, payload slots and G
    // 16-byte aligned)
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    bool have = false;
    for (int64_t j = i; j < N; ++j) {
      const uint64_t mv = mark[j * m + p];
      if ((uint32_t)(mv >> 32) != stamp) continue;
      const int64_t qj = (int64_t)(uint32_t)mv;
      if (qj >= bk.k) continue;  // a broken tag touches nothing
      const float4 v = *reinterpret_cast<const float4*>(agg + j * payload + bk.agg_off +
                                                        qj * bk.cols + col);
      if (have) {
        acc.x = acc.x + v.x;
        acc.y = acc.y + v.y;
        acc.z = acc.z + v.z;
        acc.w = acc.w + v.w;
      } else {
        acc = v;
      }
      have = true;
    }
    if (!have) return;
    float4 Gv = *reinterpret_cast<const float4*>(G + e);
    Gv.x = Gv.x + acc.x;
    Gv.y = Gv.y + acc.y;
    Gv.z = Gv.z + acc.z;
    Gv.w = Gv.w + acc.w;
    *reinterpret_cast<float4*>(G + e) = Gv;
    return;
  }
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  bool have = false;
  for (int64_t j = i; j < N; ++j) {
    const uint64_t mv = mark[j * m + p];
    if ((uint32_t)(mv >> 32) != stamp) continue;
    const int64_t qj = (int64_t)(uint32_t)mv;
    if (qj >= bk.k) continue;  // a broken tag touches nothing
    const float* src = agg + j * payload + bk.agg_off + qj * bk.cols + col;
    for (int64_t jj = 0; jj < ncols; ++jj) acc[jj] = have ? acc[jj] + src[jj] : src[jj];
    have = true;
  }
  if (!have) return;
  for (int64_t jj = 0; jj < ncols; ++jj)
    if (e + jj < d) G[e + jj] = G[e + jj] + acc[jj];
}

__global__ void __launch_bounds__(256) zero_u64_kernel(uint64_t* __restrict__ p, int64_t n) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < n) p[e] = 0u;
}

}  // namespace

hipError_t launch_momentum(bool vec, const void* grad, int32_t grad_bf16, float* h,
                           int64_t count, float eta, float a, hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  if (vec) {
    const dim3 grid(blocks_for((count + 3) / 4, 256));
    if (grad_bf16)
      hipLaunchKernelGGL(momentum_vec_kernel<true>, grid, dim3(256), 0, stream, grad, h, count,
                         eta, a);
    else
      hipLaunchKernelGGL(momentum_vec_kernel<false>, grid, dim3(256), 0, stream, grad, h, count,
                         eta, a);
  } else {
    hipLaunchKernelGGL(momentum_scalar_kernel, dim3(blocks_for(count, 256)), dim3(256), 0, stream,
                       grad, grad_bf16, h, count, eta, a);
  }
  return hipGetLastError();
}

hipError_t launch_randk_keys(uint64_t seed, int64_t t, int64_t m, float* keys,
                             hipStream_t stream) {
  if (m <= 0) return hipSuccess;
  hipLaunchKernelGGL(randk_keys_kernel, dim3(blocks_for(m, 256)), dim3(256), 0, stream, seed, t,
                     m, keys);
  return hipGetLastError();
}

hipError_t launch_topk_gather(const float* h, float* g, const int32_t* sel, int32_t* out_idx,
                              float* agg, const GatherBucket* buckets, int32_t nb,
                              int64_t work, int64_t K_total, int64_t payload, int64_t d,
                              int64_t m, int32_t N, bool vec, uint64_t* mark, uint32_t stamp,
                              hipStream_t stream) {
  if (work <= 0) return hipSuccess;
  hipLaunchKernelGGL(topk_gather_kernel, dim3(blocks_for((int64_t)N * work, 256)), dim3(256), 0,
                     stream, h, g, sel, out_idx, agg, buckets, nb, work, K_total, payload, d, m,
                     N, vec ? 1 : 0, mark, stamp);
  return hipGetLastError();
}

hipError_t launch_topk_merge(const float* agg, const int32_t* sel, const uint64_t* mark,
                             uint32_t stamp, const GatherBucket* buckets, int32_t nb,
                             int64_t work, int64_t K_total, int64_t payload, int64_t d,
                             int64_t m, int32_t N, float* G, bool vec, hipStream_t stream) {
  if (work <= 0) return hipSuccess;
  hipLaunchKernelGGL(topk_merge_kernel, dim3(blocks_for((int64_t)N * work, 256)), dim3(256), 0,
                     stream, agg, sel, mark, stamp, buckets, nb, work, K_total, payload, d, m, N,
                     G, vec ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_zero_u64(uint64_t* p, int64_t n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_u64_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, stream, p, n);
  return hipGetLastError();
}

}  // namespace arc
