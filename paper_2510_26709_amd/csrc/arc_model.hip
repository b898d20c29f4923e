// Model step around the compressor: the dense (identity-compressor) step of
// the warm-up iterations, and the x update of Eq. (11c) with the optimisers of
// the experiments (SGD, heavy-ball momentum SGD, Adam).
//
// The nodes keep G = sum_i g^(i) by adding each step's summed payload (the
// gather kernels do that at the selected coordinates; the dense step here at
// all of them).  Every operation is binary32 and correctly rounded, in the
// order documented in libarctopk.h, so that the result is bit-exact against a
// sequential evaluation.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "arc_device.h"
#include "arc_internal.h"

namespace arc {
namespace {

// ---------------------------------------------------------------------------
// Dense step, per coordinate e: for each worker in ascending order
//   h_i = fmaf(eta, grad_i, fl(a * h_i)),  Delta_i = h_i - g_i,
//   acc = Delta_0 + Delta_1 + ...,  g_i = g_i + Delta_i;
// then G = G + acc.  HBM per coordinate: N * (b_g + 16) + 8 bytes.
// ---------------------------------------------------------------------------
template <bool BF16>
__device__ __forceinline__ float4 load_grad4(const void* grad, int64_t at) {
  if constexpr (BF16) {
    const uint2 w = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(grad) + at);
    return make_float4(bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y));
  } else {
    return stream_load(reinterpret_cast<const float4*>(static_cast<const float*>(grad) + at));
  }
}

template <bool BF16>
__global__ void __launch_bounds__(256)
dense_step_vec_kernel(const void* __restrict__ grad, float* __restrict__ h,
                      float* __restrict__ g, float* __restrict__ G, int64_t d, int32_t N,
                      float eta, float a) {
  const int64_t e = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (e >= d) return;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int32_t i = 0; i < N; ++i) {
    const int64_t at = (int64_t)i * d + e;
    const float4 x = load_grad4<BF16>(grad, at);
    float4 hv = stream_load(reinterpret_cast<const float4*>(h + at));
    const float4 gv = stream_load(reinterpret_cast<const float4*>(g + at));
    hv.x = fmaf(eta, x.x, a * hv.x);
    hv.y = fmaf(eta, x.y, a * hv.y);
    hv.z = fmaf(eta, x.z, a * hv.z);
    hv.w = fmaf(eta, x.w, a * hv.w);
    const float4 dl = make_float4(hv.x - gv.x, hv.y - gv.y, hv.z - gv.z, hv.w - gv.w);
    if (i == 0) {
      acc = dl;
    } else {
      acc.x = acc.x + dl.x;
      acc.y = acc.y + dl.y;
      acc.z = acc.z + dl.z;
      acc.w = acc.w + dl.w;
    }
    stream_store(reinterpret_cast<float4*>(h + at), hv);
    stream_store(reinterpret_cast<float4*>(g + at),
                 make_float4(gv.x + dl.x, gv.y + dl.y, gv.z + dl.z, gv.w + dl.w));
  }
  float4 Gv = stream_load(reinterpret_cast<const float4*>(G + e));
  Gv.x = Gv.x + acc.x;
  Gv.y = Gv.y + acc.y;
  Gv.z = Gv.z + acc.z;
  Gv.w = Gv.w + acc.w;
  stream_store(reinterpret_cast<float4*>(G + e), Gv);
}

__global__ void __launch_bounds__(256)
dense_step_scalar_kernel(const void* __restrict__ grad, int32_t grad_bf16,
                         float* __restrict__ h, float* __restrict__ g, float* __restrict__ G,
                         int64_t d, int32_t N, float eta, float a) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= d) return;
  float acc = 0.0f;
  for (int32_t i = 0; i < N; ++i) {
    const int64_t at = (int64_t)i * d + e;
    const float x =
        grad_bf16 ? __uint_as_float((uint32_t)static_cast<const uint16_t*>(grad)[at] << 16)
                  : static_cast<const float*>(grad)[at];
    const float hn = fmaf(eta, x, a * h[at]);
    const float dl = hn - g[at];
    acc = (i == 0) ? dl : acc + dl;
    h[at] = hn;
    g[at] = g[at] + dl;
  }
  G[e] = G[e] + acc;
}

// ---------------------------------------------------------------------------
// x update of one coordinate (division and sqrtf correctly rounded: the
// library is built with -fhip-fp32-correctly-rounded-divide-sqrt; the
// __fdiv_rn / __fsqrt_rn intrinsics are not used, as __fsqrt_rn maps to the
// native approximate square root): dir = fmaf(wd, x, G / N), then
//   SGD:  x = fmaf(-lr, dir, x)
//   MSGD: m = fmaf(beta, m, dir);  x = fmaf(-lr, m, x)
//   Adam: m = fmaf(beta1, m, fl((1-beta1) dir));  v = fmaf(beta2, v, fl((1-beta2) fl(dir dir)));
//         x = fmaf(-lr, fl(fl(m / c1) / fl(sqrt(fl(v / c2)) + eps)), x)
// HBM per coordinate: SGD 12 bytes, MSGD 20, Adam 28.
// ---------------------------------------------------------------------------
template <int KIND>
__device__ __forceinline__ void update_one(const OptimizerArgs& o, float Gi, float& x, float& m,
                                           float& v) {
  const float dir = fmaf(o.weight_decay, x, Gi / o.fN);
  if constexpr (KIND == 0) {
    x = fmaf(o.neg_lr, dir, x);
  } else if constexpr (KIND == 1) {
    m = fmaf(o.momentum, m, dir);
    x = fmaf(o.neg_lr, m, x);
  } else {
    m = fmaf(o.beta1, m, o.one_minus_beta1 * dir);
    v = fmaf(o.beta2, v, o.one_minus_beta2 * (dir * dir));
    const float mh = m / o.c1, vh = v / o.c2;
    const float step = mh / (sqrtf(vh) + o.eps);
    x = fmaf(o.neg_lr, step, x);
  }
}

// Vectorised x update: one workgroup of 256 threads per tile of kOptTile
// coordinates, each thread kOptUnroll float4 of every array (all loads of a
// thread in flight together), through buffer resources that end at d: the
// hardware returns zero for loads past the end and drops those stores, so the
// last, partial tile needs no branch.  Loads are non-temporal (every value is
// read once), stores non-temporal at device scope (read again only by later
// launches).  Adam over 1.1e9 coordinates (28 bytes each), three MI355X
// boxes, every variant in one process per box: one float4 per thread
// through plain pointers 5.66 / 4.91-4.93 / 5.37-5.39 ms; this tile (four
// float4 per thread, at most four workgroups per compute unit through the
// launch's LDS reservation) - / 4.83 / 5.44-5.46 ms; two float4 per thread
// through buffer resources 5.49 / 4.87 / 5.61-5.63 ms.  The spread between
// boxes (up to 12%) is larger than between shapes on one box (2-3%).
// Default-policy stores were 3-4% slower, default-policy loads 3-7%, and
// grid-stride loops over tiles 7-30%.
constexpr int kOptUnroll = 4;
constexpr int kOptTile = 256 * 4 * kOptUnroll;

template <int KIND>
__global__ void __launch_bounds__(256)
optimizer_vec_kernel(OptimizerArgs o, const float* __restrict__ G, float* __restrict__ x,
                     float* __restrict__ m, float* __restrict__ v, int64_t d) {
  const int64_t b0 = (int64_t)blockIdx.x * kOptTile;
  const int64_t left = d - b0;
  const uint32_t bytes = (uint32_t)(left < kOptTile ? left : kOptTile) * 4u;
  const buffer_rsrc rG = make_buffer(G + b0, bytes);
  const buffer_rsrc rx = make_buffer(x + b0, bytes);
  const buffer_rsrc rm = make_buffer(KIND >= 1 ? m + b0 : x + b0, bytes);
  const buffer_rsrc rv = make_buffer(KIND == 2 ? v + b0 : x + b0, bytes);
  float4 Gv[kOptUnroll], xv[kOptUnroll], mv[kOptUnroll], vv[kOptUnroll];
#pragma unroll
  for (int u = 0; u < kOptUnroll; ++u) {
    const uint32_t off = (uint32_t)(u * 1024 + threadIdx.x * 4) * 4u;
    Gv[u] = buffer_load_f4<kCacheNonTemporal>(rG, off);
    xv[u] = buffer_load_f4<kCacheNonTemporal>(rx, off);
    mv[u] = vv[u] = make_float4(0.f, 0.f, 0.f, 0.f);
    if constexpr (KIND >= 1) mv[u] = buffer_load_f4<kCacheNonTemporal>(rm, off);
    if constexpr (KIND == 2) vv[u] = buffer_load_f4<kCacheNonTemporal>(rv, off);
  }
#pragma unroll
  for (int u = 0; u < kOptUnroll; ++u) {
    const uint32_t off = (uint32_t)(u * 1024 + threadIdx.x * 4) * 4u;
    update_one<KIND>(o, Gv[u].x, xv[u].x, mv[u].x, vv[u].x);
    update_one<KIND>(o, Gv[u].y, xv[u].y, mv[u].y, vv[u].y);
    update_one<KIND>(o, Gv[u].z, xv[u].z, mv[u].z, vv[u].z);
    update_one<KIND>(o, Gv[u].w, xv[u].w, mv[u].w, vv[u].w);
    buffer_store_f4<kCacheStreamDevice>(rx, off, xv[u]);
    if constexpr (KIND >= 1) buffer_store_f4<kCacheStreamDevice>(rm, off, mv[u]);
    if constexpr (KIND == 2) buffer_store_f4<kCacheStreamDevice>(rv, off, vv[u]);
  }
}

template <int KIND>
__global__ void __launch_bounds__(256)
optimizer_scalar_kernel(OptimizerArgs o, const float* __restrict__ G, float* __restrict__ x,
                        float* __restrict__ m, float* __restrict__ v, int64_t d) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= d) return;
  float xe = x[e], me = 0.0f, ve = 0.0f;
  if constexpr (KIND >= 1) me = m[e];
  if constexpr (KIND == 2) ve = v[e];
  update_one<KIND>(o, G[e], xe, me, ve);
  x[e] = xe;
  if constexpr (KIND >= 1) m[e] = me;
  if constexpr (KIND == 2) v[e] = ve;
}

// Dynamic LDS that caps the vectorised update at four workgroups per compute
// unit (of the MI355X's 160 KB).
constexpr size_t kOptLdsCap = 36 * 1024;

template <int KIND>
void launch_optimizer_kind(bool vec, bool cap, const OptimizerArgs& o, const float* G, float* x,
                           float* m, float* v, int64_t d, hipStream_t stream) {
  if (vec)
    hipLaunchKernelGGL(optimizer_vec_kernel<KIND>, dim3(blocks_for(d, kOptTile)), dim3(256),
                       cap ? kOptLdsCap : 0, stream, o, G, x, m, v, d);
  else
    hipLaunchKernelGGL(optimizer_scalar_kernel<KIND>, dim3(blocks_for(d, 256)), dim3(256), 0,
                       stream, o, G, x, m, v, d);
}

}  // namespace

hipError_t launch_dense_step(bool vec, const void* grad, int32_t grad_bf16, float* h, float* g,
                             float* G, int64_t d, int32_t N, float eta, float a,
                             hipStream_t stream) {
  if (d <= 0) return hipSuccess;
  if (vec) {
    const dim3 grid(blocks_for((d + 3) / 4, 256));
    if (grad_bf16)
      hipLaunchKernelGGL(dense_step_vec_kernel<true>, grid, dim3(256), 0, stream, grad, h, g, G,
                         d, N, eta, a);
    else
      hipLaunchKernelGGL(dense_step_vec_kernel<false>, grid, dim3(256), 0, stream, grad, h, g,
                         G, d, N, eta, a);
  } else {
    hipLaunchKernelGGL(dense_step_scalar_kernel, dim3(blocks_for(d, 256)), dim3(256), 0, stream,
                       grad, grad_bf16, h, g, G, d, N, eta, a);
  }
  return hipGetLastError();
}

hipError_t launch_optimizer(bool vec, bool cap, const OptimizerArgs& o, const float* G, float* x,
                            float* m, float* v, int64_t d, hipStream_t stream) {
  if (d <= 0) return hipSuccess;
  if (vec && d > INT64_MAX - kOptTile) return hipErrorInvalidValue;
  switch (o.kind) {
    case 0: launch_optimizer_kind<0>(vec, cap, o, G, x, m, v, d, stream); break;
    case 1: launch_optimizer_kind<1>(vec, cap, o, G, x, m, v, d, stream); break;
    case 2: launch_optimizer_kind<2>(vec, cap, o, G, x, m, v, d, stream); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace arc
