// arc_step_static: one compressor step from a configuration, for callers that
// cannot allocate device memory.  Every device buffer the step needs beyond
// the caller's inputs and outputs (the kernels' tables, V_t, the per-worker
// sketch, the importance, the selection's radix state, histograms and block
// counts) lives in one file-scope device array, `scratch`, of
// ARC_STATIC_SCRATCH_BYTES.  Each device the library runs on holds its own
// copy of it until the process ends.  The step runs exactly the kernels and
// tables of arc_step, so its results are the same bits.
//
// Host code never uses the array's name as an address: at the first call on
// a device, with that device current, hipGetSymbolAddress gives that
// device's copy, which is kept per device and passed to the kernels.
#include <hip/hip_runtime.h>

#include <cstring>
#include <mutex>
#include <vector>

#include "arc_context.h"
#include "arc_device.h"

static __device__ __align__(256) unsigned char scratch[ARC_STATIC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
constexpr size_t kAlign = 256;

struct DeviceScratch {
  bool ready = false;
  unsigned char* ptr = nullptr;  // this device's copy of `scratch`
  // The upload of the last call's tables and V_t reads `staging`; `copied`
  // is recorded after it, so the next call refills staging only once the
  // device has read it.
  hipEvent_t copied = nullptr;
  bool pending = false;
  std::vector<unsigned char> staging;
};

std::mutex g_mu;
DeviceScratch g_dev[kMaxDevices];

// Set-up of device `dev` (current): its address of `scratch` and the upload
// event, once per device.
arc_status setup_device(int dev, DeviceScratch** out) {
  DeviceScratch& ds = g_dev[dev];
  if (!ds.ready) {
    void* p = nullptr;
    ARC_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (p == nullptr)
      return arc::fail(ARC_ERR_DEVICE, "hipGetSymbolAddress(scratch) gave a NULL address");
    if (ds.copied == nullptr)
      ARC_HIP(hipEventCreateWithFlags(&ds.copied, hipEventDisableTiming), "hipEventCreate");
    ds.ptr = static_cast<unsigned char*>(p);
    ds.ready = true;
  }
  *out = &ds;
  return ARC_OK;
}

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Byte offsets in the scratch array.  [0, upload_end) is copied from the
// host every call (tables, then V_t); the rest is written by the kernels.
struct Layout {
  size_t groups, gather, buckets, blocks, V, upload_end;
  size_t S, sigma, sel, state, hist, blockcnt, total;
};

Layout layout_of(const arc_ctx& c) {
  Layout L{};
  size_t at = 0;
  auto take = [&](size_t bytes) {
    const size_t off = at;
    at = align_up(at + bytes);
    return off;
  };
  const size_t nb = c.buckets.size(), nblk = c.blocks.size();
  L.groups = take(c.groups.size() * sizeof(arc::RowGroup));
  L.gather = take(c.gather.size() * sizeof(arc::GatherBucket));
  L.buckets = take(nb * sizeof(arc::BucketDesc));
  L.blocks = take(nblk * sizeof(arc::BlockDesc));
  L.V = take(static_cast<size_t>(c.v_floats) * sizeof(float));
  L.upload_end = at;
  L.S = take(static_cast<size_t>(c.N) * static_cast<size_t>(c.m) * c.r * sizeof(float));
  L.sigma = take(static_cast<size_t>(c.m) * sizeof(float));
  L.sel = take(c.compressor == ARC_COMP_TOPK ? static_cast<size_t>(c.K_total) * 4 : 0);
  L.state = take(arc::kRadixPasses * nb * sizeof(arc::BucketState));
  L.hist = take(arc::kRadixPasses * nb * arc::kRadixBins * sizeof(uint32_t));
  L.blockcnt = take(2 * nblk * sizeof(uint32_t));
  L.total = at;
  return L;
}

template <typename T>
void put(std::vector<unsigned char>& dst, size_t off, const std::vector<T>& src) {
  if (!src.empty()) std::memcpy(dst.data() + off, src.data(), src.size() * sizeof(T));
}

// The radix histograms start every step at zero (a kernel, not a memset, so
// that the call stays a plain sequence of kernels and one copy).
__global__ void __launch_bounds__(256) zero_words_kernel(uint32_t* __restrict__ p, int64_t n) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < n) p[e] = 0u;
}

}  // namespace

extern "C" arc_status arc_step_static(const arc_config* cfg, void* hip_stream, int64_t t,
                                      const void* grad, float* h, float* g, int32_t* out_idx,
                                      float* out_agg) {
  int64_t m = 0;
  arc_status st = arc::check_config(cfg, &m);
  if (st != ARC_OK) return st;
  // Host tables only: its device pointers are set into the scratch array
  // below, and it is never released.
  arc_ctx c;
  if ((st = arc::plan_context(cfg, m, hip_stream, &c)) != ARC_OK) return st;
  const Layout L = layout_of(c);
  if (L.total > ARC_STATIC_SCRATCH_BYTES)
    return arc::fail(ARC_ERR_INVALID,
                     "arc_step_static: this configuration needs " + std::to_string(L.total) +
                         " bytes of device scratch, more than the static " +
                         std::to_string(static_cast<size_t>(ARC_STATIC_SCRATCH_BYTES)) +
                         " (use arc_create / arc_step)");
  if ((st = arc::check_step_args(&c, t, grad, h, g, out_idx, out_agg, true)) != ARC_OK)
    return st;
  if ((st = arc::bind_device(&c)) != ARC_OK) return st;
  if (c.device < 0 || c.device >= kMaxDevices)
    return arc::fail(ARC_ERR_UNSUPPORTED, "arc_step_static: device index beyond 63");

  std::lock_guard<std::mutex> lock(g_mu);
  DeviceScratch* ds = nullptr;
  if ((st = setup_device(c.device, &ds)) != ARC_OK) return st;
  if (ds->pending) {
    ARC_HIP(hipEventSynchronize(ds->copied), "hipEventSynchronize(static upload)");
    ds->pending = false;
  }
  try {
    ds->staging.assign(L.upload_end, 0);
  } catch (...) {
    return arc::fail(ARC_ERR_NOMEM, "host allocation failed");
  }
  put(ds->staging, L.groups, c.groups);
  put(ds->staging, L.gather, c.gather);
  put(ds->staging, L.buckets, c.buckets);
  put(ds->staging, L.blocks, c.blocks);
  if (c.compressor == ARC_COMP_ARC)
    for (const int64_t w : c.widths)
      arc::generate_projection(c.seed, t, w, c.r,
                               reinterpret_cast<float*>(ds->staging.data() + L.V) + c.v_off[w]);

  unsigned char* base = ds->ptr;
  if (L.upload_end > 0) {
    ARC_HIP(hipMemcpyAsync(base, ds->staging.data(), L.upload_end, hipMemcpyHostToDevice,
                           c.stream),
            "hipMemcpyAsync(static tables)");
    ARC_HIP(hipEventRecord(ds->copied, c.stream), "hipEventRecord(static upload)");
    ds->pending = true;
  }
  c.groups_dev = reinterpret_cast<arc::RowGroup*>(base + L.groups);
  c.gather_dev = reinterpret_cast<arc::GatherBucket*>(base + L.gather);
  c.buckets_dev = reinterpret_cast<arc::BucketDesc*>(base + L.buckets);
  c.blocks_dev = reinterpret_cast<arc::BlockDesc*>(base + L.blocks);
  c.V_dev = reinterpret_cast<float*>(base + L.V);
  c.S_dev = reinterpret_cast<float*>(base + L.S);
  c.sigma_dev = reinterpret_cast<float*>(base + L.sigma);
  c.sel_dev = reinterpret_cast<int32_t*>(base + L.sel);
  c.state_dev = reinterpret_cast<arc::BucketState*>(base + L.state);
  c.hist_dev = reinterpret_cast<uint32_t*>(base + L.hist);
  c.blockcnt_dev = reinterpret_cast<uint32_t*>(base + L.blockcnt);
  c.V_staged = true;
  const arc::SelectWorkspace ws = c.select_ws();
  if (ws.any_radix && !ws.small) {
    const int64_t words =
        static_cast<int64_t>(arc::kRadixPasses) * ws.nb * arc::kRadixBins;
    hipLaunchKernelGGL(zero_words_kernel, dim3(arc::blocks_for(words, 256)), dim3(256), 0,
                       c.stream, c.hist_dev, words);
    ARC_HIP(hipGetLastError(), "histogram clear launch");
  }
  return arc::enqueue_step(&c, t, grad, h, g, out_idx, out_agg, nullptr);
}
