// Gather + worker sum + error-feedback update of the compressor step (Eq. (5),
// Alg. 1's payload All-Reduce, Eq. (11b)).  With a non-null G the summed
// payload is also added into the node-summed tracker, G = fl(G + agg), at the
// same coordinates (the model step's view of the payload, Eq. (11c)).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "arc_device.h"
#include "arc_internal.h"

namespace arc {
namespace {

// ---------------------------------------------------------------------------
// Thread per (selected row, 4 columns) on the vectorised path: for each worker
// in ascending order Delta = h - g, agg += Delta, g = g + Delta.  Rows are
// contiguous, so every access is a coalesced 16-byte access.  Columns past d
// give agg = +0.
// ---------------------------------------------------------------------------
constexpr int kMaxUnrolledWorkers = 8;

__global__ void __launch_bounds__(256)
gather_update_fast_kernel(const float* __restrict__ h, float* __restrict__ g,
                          const int32_t* __restrict__ idx,
                          float* __restrict__ agg, float* __restrict__ G, int64_t K_total,
                          int64_t d, int64_t n, int64_t m, int32_t N) {
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
    if (G) {
      float4 Gv = *reinterpret_cast<const float4*>(G + e);
      Gv.x = Gv.x + acc.x;
      Gv.y = Gv.y + acc.y;
      Gv.z = Gv.z + acc.z;
      Gv.w = Gv.w + acc.w;
      *reinterpret_cast<float4*>(G + e) = Gv;
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
      if (G) G[e + jj] = G[e + jj] + a4[jj];
    }
    acc = make_float4(a4[0], a4[1], a4[2], a4[3]);
  }
  *reinterpret_cast<float4*>(agg + q * n + col) = acc;
}

__global__ void __launch_bounds__(256)
gather_update_generic_kernel(const float* __restrict__ h, float* __restrict__ g,
                             const int32_t* __restrict__ idx,
                             float* __restrict__ agg, float* __restrict__ G, int64_t K_total,
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
    if (G) G[e] = G[e] + acc;
  }
  agg[tid] = acc;
}

// ---------------------------------------------------------------------------
// Per-tensor mode: one work item = one selected row x 4 columns of a tensor.
// Items are numbered tensor after tensor (GatherBucket::work_off); a thread
// finds its tensor by binary search.  Same arithmetic as above: for each
// worker in ascending order Delta = h - g, agg += Delta, g = g + Delta.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256)
gather_update_tensors_kernel(const float* __restrict__ h, float* __restrict__ g,
                             const int32_t* __restrict__ idx,
                             float* __restrict__ agg, float* __restrict__ G,
                             const GatherBucket* __restrict__ buckets,
                             int32_t nb, int64_t total_work, int64_t d,
                             int32_t N, int32_t allow_vec) {
  const int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (w >= total_work) return;
  int32_t lo = 0, hi = nb;  // last bucket whose work_off <= w
  while (hi - lo > 1) {
    const int32_t mid = (lo + hi) >> 1;
    if (buckets[mid].work_off <= w) lo = mid; else hi = mid;
  }
  const GatherBucket bk = buckets[lo];
  const int64_t per_row = (bk.cols + 3) / 4;
  const int64_t item = w - bk.work_off;
  const int64_t q = item / per_row;
  const int64_t col = (item - q * per_row) * 4;
  const int64_t p = (int64_t)idx[bk.out_off + q] - bk.row0;
  float* out = agg + bk.agg_off + q * bk.cols + col;
  const int64_t ncols = bk.cols - col < 4 ? bk.cols - col : 4;
  const int64_t e = bk.elem_off + p * bk.cols + col;
  // Only rows of this tensor; the bounds keep a broken index from touching
  // memory outside the vectors.
  if (p < 0 || p >= bk.rows || q >= bk.k || e + ncols > d) return;
  if (bk.vec && allow_vec) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int32_t i = 0; i < N; ++i) {
      const int64_t at = (int64_t)i * d + e;
      const float4 hv = *reinterpret_cast<const float4*>(h + at);
      const float4 gv = *reinterpret_cast<const float4*>(g + at);
      float4 dl;
      dl.x = hv.x - gv.x;
      dl.y = hv.y - gv.y;
      dl.z = hv.z - gv.z;
      dl.w = hv.w - gv.w;
      if (i == 0) {
        acc = dl;
      } else {
        acc.x = acc.x + dl.x;
        acc.y = acc.y + dl.y;
        acc.z = acc.z + dl.z;
        acc.w = acc.w + dl.w;
      }
      float4 gn;
      gn.x = gv.x + dl.x;
      gn.y = gv.y + dl.y;
      gn.z = gv.z + dl.z;
      gn.w = gv.w + dl.w;
      *reinterpret_cast<float4*>(g + at) = gn;
    }
    if (G) {
      float4 Gv = *reinterpret_cast<const float4*>(G + e);
      Gv.x = Gv.x + acc.x;
      Gv.y = Gv.y + acc.y;
      Gv.z = Gv.z + acc.z;
      Gv.w = Gv.w + acc.w;
      *reinterpret_cast<float4*>(G + e) = Gv;
    }
    *reinterpret_cast<float4*>(out) = acc;
  } else {
    for (int64_t jj = 0; jj < ncols; ++jj) {
      float acc = 0.0f;
      for (int32_t i = 0; i < N; ++i) {
        const int64_t at = (int64_t)i * d + e + jj;
        const float dl = h[at] - g[at];
        acc = (i == 0) ? dl : acc + dl;
        g[at] = g[at] + dl;
      }
      if (G) G[e + jj] = G[e + jj] + acc;
      out[jj] = acc;
    }
  }
}

}  // namespace

hipError_t launch_gather_update(bool fast, const float* h, float* g,
                                const int32_t* idx, float* agg, float* G, int64_t K_total,
                                int64_t d, int64_t n, int64_t m, int32_t N,
                                hipStream_t stream) {
  if (K_total <= 0) return hipSuccess;
  if (fast) {
    hipLaunchKernelGGL(gather_update_fast_kernel,
                       dim3(blocks_for(K_total * (n / 4), 256)), dim3(256), 0,
                       stream, h, g, idx, agg, G, K_total, d, n, m, N);
  } else {
    hipLaunchKernelGGL(gather_update_generic_kernel,
                       dim3(blocks_for(K_total * n, 256)), dim3(256), 0, stream,
                       h, g, idx, agg, G, K_total, d, n, m, N);
  }
  return hipGetLastError();
}

hipError_t launch_gather_update_tensors(const float* h, float* g,
                                        const int32_t* idx, float* agg, float* G,
                                        const GatherBucket* buckets, int32_t nb,
                                        int64_t total_work, int64_t d, int32_t N,
                                        bool allow_vec, hipStream_t stream) {
  if (total_work <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_update_tensors_kernel, dim3(blocks_for(total_work, 256)),
                     dim3(256), 0, stream, h, g, idx, agg, G, buckets, nb, total_work, d, N,
                     allow_vec ? 1 : 0);
  return hipGetLastError();
}

}  // namespace arc
