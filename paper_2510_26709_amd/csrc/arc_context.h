// The context behind the C ABI and the host-side steps shared by the entry
// points of libarctopk: configuration checks, the lowering of a configuration
// to the kernels' tables, the per-call argument checks and the enqueue of one
// compressor step on the context's stream.
#pragma once

#include <array>
#include <map>
#include <memory>
#include <string>
#include <vector>

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "arc_internal.h"
#include "libarctopk.h"

namespace arc {

// HIP events recorded per step when stage timing is on.
constexpr int kEventsPerStep = 6;

// Pinned host buffers staging V_t, used in turn: a step refills a buffer only
// once the device has read it (the staging kernel of the step that last used
// it), so the host can queue this many steps minus one ahead of the device
// before it waits.
constexpr int kProjectionSlots = 4;

// Record `why` as the calling thread's last error and return s.
arc_status fail(arc_status s, const std::string& why);
// The same for a HIP error at `where` (ARC_ERR_NOMEM for out-of-memory).
arc_status fail_hip(hipError_t e, const char* where);

}  // namespace arc

#define ARC_HIP(call, where)                                       \
  do {                                                             \
    const hipError_t arc_e_ = (call);                              \
    if (arc_e_ != hipSuccess) return arc::fail_hip(arc_e_, where); \
  } while (0)

struct arc_ctx {
  // problem
  int64_t d = 0, n = 0, m = 0;
  int32_t N = 0, r = 0, grad_bf16 = 0;
  float eta = 0.f, a = 0.f;
  uint64_t seed = 0;
  bool tensor_mode = false;
  int32_t compressor = ARC_COMP_ARC;
  // Rows kept and payload floats per step, over all nodes (Top-K returns
  // every node's rows; the others one shared list), and for one node.
  int64_t K_total = 0, payload = 0, K_node = 0, payload_node = 0;
  std::vector<arc::BucketDesc> buckets;
  std::vector<arc::BlockDesc> blocks;
  // projection: one V_t per distinct row width, concatenated in first-use order
  std::vector<int64_t> widths;
  std::map<int64_t, int64_t> v_off;
  int64_t v_floats = 0;
  // row groups: the vectorisable ones by group size (64, 32, 16, 8 rows),
  // then the general ones
  std::vector<arc::RowGroup> groups;
  int64_t nvec_groups = 0;
  std::array<int64_t, 4> vec_count{};  // groups of 64, 32, 16 and 8 rows
  std::array<int64_t, 5> stage_elems{};  // coordinates per launch: those sizes, general
  std::array<arc::SketchOccupancy, 4> vec_occ{};  // launch shape per group size
  // per-tensor gather
  std::vector<arc::GatherBucket> gather;
  int64_t gather_work = 0;
  // device
  hipStream_t stream = nullptr;
  // second stream for the smaller launches of the streaming stage, forked
  // from and joined back into `stream` (only when there are several)
  hipStream_t side = nullptr;
  // a pair of events per step in flight, used in turn (an event is
  // re-recorded only after kProjectionSlots further steps)
  hipEvent_t fork_ev[arc::kProjectionSlots] = {}, join_ev[arc::kProjectionSlots] = {};
  int fork_slot = 0;
  int device = 0;
  size_t max_lds_per_block = 0;
  int lds_per_cu = 0;
  float* V_dev = nullptr;
  float* S_dev = nullptr;
  float* sigma_dev = nullptr;
  arc::RowGroup* groups_dev = nullptr;
  int32_t* sel_dev = nullptr;  // Top-K: selection over the N*m norms
  // Top-K in the model step: [N*m] tags of the rows each node kept, for the
  // merge into G; a tag carries the stamp of its step (0 = never tagged)
  uint64_t* mark_dev = nullptr;
  uint32_t mark_stamp = 0;
  arc::GatherBucket* gather_dev = nullptr;
  arc::BucketDesc* buckets_dev = nullptr;
  arc::BlockDesc* blocks_dev = nullptr;
  arc::BucketState* state_dev = nullptr;
  uint32_t* hist_dev = nullptr;
  uint32_t* blockcnt_dev = nullptr;
  // projection staging: a ring of pinned buffers; the pool fills the next
  // step's buffer while the device runs this step
  float* V_pinned[arc::kProjectionSlots] = {};
  float* V_pinned_dev[arc::kProjectionSlots] = {};  // the same buffers, device-mapped
  hipEvent_t V_done[arc::kProjectionSlots] = {};
  bool V_pending[arc::kProjectionSlots] = {};
  int V_slot = 0;
  std::vector<float> V_override;
  bool use_override = false;
  // V_t is already on the device for this step (put there by the entry
  // point that owns no staging buffers); enqueue_step then skips the upload
  bool V_staged = false;
  std::vector<arc::ProjectionBlock> V_blocks;
  std::unique_ptr<arc::ProjectionPool> V_pool;
  int64_t V_prefetch_t = -1;  // step whose V_t the pool put in V_pinned[V_slot]
  // stage timing
  bool timing = false;
  std::vector<std::array<hipEvent_t, arc::kEventsPerStep>> ev_pool;
  size_t ev_used = 0;

  arc::SelectWorkspace select_ws() const {
    arc::SelectWorkspace ws;
    ws.buckets = buckets_dev;
    ws.blocks = blocks_dev;
    ws.state = state_dev;
    ws.hist = hist_dev;
    ws.blockcnt = blockcnt_dev;
    ws.nb = static_cast<int32_t>(buckets.size());
    ws.nblk = static_cast<int32_t>(blocks.size());
    ws.any_radix = 0;
    ws.any_output = 0;
    ws.small = 1;
    ws.small_rows = 0;
    for (const auto& b : buckets) {
      ws.any_radix |= b.mode == arc::kSelectRadix;
      ws.any_output |= b.mode != arc::kSelectNone;
      ws.small &= b.hi - b.lo <= arc::kSmallBucketRows;
      if (b.mode == arc::kSelectRadix && b.hi - b.lo > ws.small_rows)
        ws.small_rows = static_cast<int32_t>(
            b.hi - b.lo < arc::kSmallBucketRows ? b.hi - b.lo : arc::kSmallBucketRows);
    }
    return ws;
  }

  void release() {
    V_pool.reset();  // joins the threads before their buffers go
    (void)hipStreamSynchronize(stream);
    if (side) {
      (void)hipStreamSynchronize(side);
      (void)hipStreamDestroy(side);
    }
    for (int k = 0; k < arc::kProjectionSlots; ++k)
      for (hipEvent_t e : {fork_ev[k], join_ev[k]})
        if (e) (void)hipEventDestroy(e);
    for (void* p : {static_cast<void*>(V_dev), static_cast<void*>(S_dev),
                    static_cast<void*>(sigma_dev), static_cast<void*>(groups_dev),
                    static_cast<void*>(sel_dev), static_cast<void*>(mark_dev),
                    static_cast<void*>(gather_dev), static_cast<void*>(buckets_dev),
                    static_cast<void*>(blocks_dev), static_cast<void*>(state_dev),
                    static_cast<void*>(hist_dev), static_cast<void*>(blockcnt_dev)})
      if (p) (void)hipFree(p);
    for (int s = 0; s < arc::kProjectionSlots; ++s) {
      if (V_done[s]) (void)hipEventDestroy(V_done[s]);
      if (V_pinned[s]) (void)hipHostFree(V_pinned[s]);
    }
    for (auto& evs : ev_pool)
      for (hipEvent_t e : evs)
        if (e) (void)hipEventDestroy(e);
    ev_pool.clear();
  }
};

namespace arc {

// Checks cfg (no HIP call); on success *m_out is the number of rows.
arc_status check_config(const arc_config* cfg, int64_t* m_out);

// Fills the context's problem fields and lowers cfg (already checked, m
// rows) to the kernels' host tables; binds the context to `stream`.  Host
// work only.
arc_status plan_context(const arc_config* cfg, int64_t m, void* stream, arc_ctx* c);

// The current device, its LDS limit and the launch shapes that depend on
// it (no allocation).
arc_status bind_device(arc_ctx* c);

// Checks the arguments of one step (no HIP call).  need_outputs: the call
// writes out_idx / out_agg.
arc_status check_step_args(const arc_ctx* c, int64_t t, const void* grad, const float* h,
                           const float* g, const int32_t* out_idx, const float* out_agg,
                           bool need_outputs);

// Enqueues one compressor step (arguments already checked) on c->stream;
// with a non-null G the payload is also added into G at the selected
// coordinates.
arc_status enqueue_step(arc_ctx* c, int64_t t, const void* grad, float* h, float* g,
                        int32_t* out_idx, float* out_agg, float* G);

}  // namespace arc
