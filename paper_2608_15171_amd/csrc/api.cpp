// extern "C" entry points of libppas.so (declared in include/ppas.h).
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "plan.h"
#include "ppas.h"

namespace ppas {

hipError_t launch_attn_step(const uint16_t* q, uint16_t* out, const uint16_t* kp, const uint16_t* vp,
                            const int32_t* bt, int32_t bt_stride, int32_t hq, int32_t hkv, float scale,
                            const WorkItem* items, int n_items, const CombineItem* comb, int n_comb,
                            float2* part_ml, float* part_acc, int tile_pos, hipStream_t stream,
                            hipEvent_t ev_start, hipEvent_t ev_stop);
hipError_t launch_kv_append(uint16_t* kp, uint16_t* vp, const uint16_t* kn, const uint16_t* vn,
                            const ppas_seq* seqs, int32_t n_seqs, const int32_t* bt, int32_t bt_stride,
                            int32_t hkv, hipStream_t stream, hipEvent_t ev_start, hipEvent_t ev_stop);
hipError_t launch_rope_append(uint16_t* q, uint16_t* kp, uint16_t* vp, const uint16_t* kn, const uint16_t* vn,
                              const ppas_seq* seqs, int32_t n_seqs, const int32_t* bt, int32_t bt_stride,
                              int32_t hq, int32_t hkv, double theta, hipStream_t stream, hipEvent_t ev_start,
                              hipEvent_t ev_stop);

namespace {

struct DeviceInfo {
  bool known = false;
  bool gfx950 = false;
  int cus = 256;
};

std::mutex g_mu;
std::vector<DeviceInfo> g_dev;
std::atomic<void*> g_ev_start{nullptr};
std::atomic<void*> g_ev_stop{nullptr};

// Compute-unit count and architecture of the current device (cached). Without a
// usable device, reports 256 CUs and not-gfx950.
DeviceInfo current_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return DeviceInfo{};
  }
  std::lock_guard<std::mutex> lk(g_mu);
  if (dev >= int(g_dev.size())) g_dev.resize(size_t(dev) + 1);
  DeviceInfo& d = g_dev[size_t(dev)];
  if (!d.known) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) == hipSuccess) {
      d.gfx950 = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
      d.cus = prop.multiProcessorCount > 0 ? prop.multiProcessorCount : 256;
    } else {
      (void)hipGetLastError();
    }
    d.known = true;
  }
  return d;
}

// Work-item counts and partial-slot offsets travel as int32 (and the item count
// sets the launch grid): a step too large for that is refused.
bool plan_fits(const Plan& plan) {
  return plan.items.size() <= size_t(INT32_MAX) && plan.combine.size() <= size_t(INT32_MAX) &&
         plan.part_slots <= int64_t(INT32_MAX) - 64 * kGroup;
}

// Pinned host staging for the work list, one ring per device (a slot's
// completion event belongs to the device it was created on). The kernels read
// their items straight from the slot's pinned memory: each workgroup reads its
// 32-byte item once, which costs less than a host-to-device copy on a separate
// engine and the two cross-engine waits around it. A slot is refilled only after
// the event recorded behind the last kernel that reads it has completed, so
// callers wait on the device only when kSlots launches are still in flight.
constexpr int kSlots = 8;
struct Slot {
  void* host = nullptr;
  char* dev = nullptr;      // the same memory as the device addresses it
  size_t cap = 0;
  hipEvent_t done = nullptr;
  bool pending = false;
};
struct Ring {
  Slot slots[kSlots];
  int next = 0;
};
std::vector<Ring> g_rings;
std::mutex g_stage_mu;     // held from taking a slot until its event is recorded

// The next slot of the current device's ring, with room for `bytes`. Caller holds g_stage_mu.
ppas_status take_slot(size_t bytes, Slot*& out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return PPAS_EHIP;
  if (dev >= int(g_rings.size())) g_rings.resize(size_t(dev) + 1);
  Ring& ring = g_rings[size_t(dev)];
  Slot& s = ring.slots[ring.next];
  ring.next = (ring.next + 1) % kSlots;
  if (s.pending) {
    if (hipEventSynchronize(s.done) != hipSuccess) return PPAS_EHIP;
    s.pending = false;
  }
  if (!s.done && hipEventCreateWithFlags(&s.done, hipEventDisableTiming) != hipSuccess) return PPAS_EHIP;
  if (s.cap < bytes) {
    if (s.host) (void)hipHostFree(s.host);
    s.host = nullptr;
    s.dev = nullptr;
    s.cap = 0;
    size_t cap = 1 << 16;
    while (cap < bytes) cap <<= 1;
    if (hipHostMalloc(&s.host, cap, hipHostMallocDefault) != hipSuccess) return PPAS_EHIP;
    void* d = nullptr;
    if (hipHostGetDevicePointer(&d, s.host, 0) != hipSuccess) {
      (void)hipHostFree(s.host);
      s.host = nullptr;
      return PPAS_EHIP;
    }
    s.dev = static_cast<char*>(d);
    s.cap = cap;
  }
  out = &s;
  return PPAS_OK;
}

}  // namespace
}  // namespace ppas

using namespace ppas;

extern "C" {

const char* ppas_status_string(ppas_status status) {
  switch (status) {
    case PPAS_OK: return "PPAS_OK";
    case PPAS_EINVAL: return "PPAS_EINVAL: invalid argument or step description";
    case PPAS_ERANGE: return "PPAS_ERANGE: block-table entry, length or step size out of range";
    case PPAS_ENOSPACE: return "PPAS_ENOSPACE: workspace too small";
    case PPAS_EHIP: return "PPAS_EHIP: HIP runtime error";
    case PPAS_EUNSUPPORTED: return "PPAS_EUNSUPPORTED: shape or device outside the compiled set";
  }
  return "PPAS: unknown status";
}

ppas_status ppas_validate_step(const ppas_shape* shape, const ppas_seq* seqs, int32_t n_seqs,
                               const int32_t* block_table_host, int32_t bt_stride) {
  try {
    return validate(shape, seqs, n_seqs, block_table_host, bt_stride, true);
  } catch (...) {
    return PPAS_EINVAL;
  }
}

ppas_status ppas_set_profile_events(void* start_event, void* stop_event) {
  if ((start_event == nullptr) != (stop_event == nullptr)) return PPAS_EINVAL;
  g_ev_start.store(start_event);
  g_ev_stop.store(stop_event);
  return PPAS_OK;
}

ppas_status ppas_set_split_keys(int32_t prefill_split, int32_t decode_split) {
  if (prefill_split < 0 || decode_split < 0) return PPAS_EINVAL;
  set_split_keys(prefill_split, decode_split);
  return PPAS_OK;
}

ppas_status ppas_set_tile_positions(int32_t tile_positions) {
  if (tile_positions != 0 && tile_positions != kTilePosSmall && tile_positions != kTilePosLarge) return PPAS_EINVAL;
  set_tile_positions(tile_positions);
  return PPAS_OK;
}

int32_t ppas_plan_items(const ppas_shape* shape, const ppas_seq* seqs, int32_t n_seqs, int32_t num_cus,
                        int32_t* items_out, int32_t capacity) {
  try {
    const ppas_status st = validate(shape, seqs, n_seqs, nullptr, INT32_MAX, false);
    if (st != PPAS_OK) return st;
    Plan plan;
    make_plan(*shape, seqs, n_seqs, num_cus, plan);
    if (!plan_fits(plan)) return PPAS_ERANGE;
    const int32_t n = int32_t(plan.items.size());
    if (items_out) {
      for (int32_t i = 0; i < n && i < capacity; ++i) {
        const WorkItem& w = plan.items[size_t(i)];
        int32_t* o = items_out + 8 * size_t(i);
        o[0] = w.npos_kind >> 16;
        o[1] = w.seq;
        o[2] = w.kvh;
        o[3] = w.row0;
        o[4] = w.pos0;
        o[5] = w.npos_kind & 0xffff;
        o[6] = w.key_lo;
        o[7] = w.key_hi;
      }
    }
    return n;
  } catch (...) {
    return PPAS_EINVAL;
  }
}

size_t ppas_attn_workspace_bytes(const ppas_shape* shape, const ppas_seq* seqs, int32_t n_seqs) {
  try {
    if (validate(shape, seqs, n_seqs, nullptr, INT32_MAX, false) != PPAS_OK) return 0;
    Plan plan;
    make_plan(*shape, seqs, n_seqs, current_device().cus, plan);
    return plan_fits(plan) ? plan.total : 0;
  } catch (...) {
    return 0;
  }
}

ppas_status ppas_kv_append(const ppas_shape* shape, void* k_pages, void* v_pages, const void* k_new,
                           const void* v_new, const ppas_seq* seqs, int32_t n_seqs,
                           const int32_t* block_table_dev, int32_t bt_stride,
                           const int32_t* block_table_host, void* hip_stream) {
  try {
    ppas_status st = validate(shape, seqs, n_seqs, block_table_host, bt_stride, true);
    if (st != PPAS_OK) return st;
    if (n_seqs == 0) return PPAS_OK;
    if (!k_pages || !v_pages || !k_new || !v_new || !block_table_dev) return PPAS_EINVAL;
    if (!current_device().gfx950) return PPAS_EUNSUPPORTED;
    const hipError_t e = launch_kv_append(static_cast<uint16_t*>(k_pages), static_cast<uint16_t*>(v_pages),
                                          static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new),
                                          seqs, n_seqs, block_table_dev, bt_stride, shape->n_kv_heads,
                                          static_cast<hipStream_t>(hip_stream),
                                          static_cast<hipEvent_t>(g_ev_start.load()),
                                          static_cast<hipEvent_t>(g_ev_stop.load()));
    return e == hipSuccess ? PPAS_OK : PPAS_EHIP;
  } catch (...) {
    return PPAS_EINVAL;
  }
}

ppas_status ppas_rope_kv_append(const ppas_shape* shape, float rope_theta, void* q, void* k_pages, void* v_pages,
                                const void* k_new, const void* v_new, const ppas_seq* seqs, int32_t n_seqs,
                                const int32_t* block_table_dev, int32_t bt_stride,
                                const int32_t* block_table_host, void* hip_stream) {
  try {
    if (!std::isfinite(rope_theta) || !(rope_theta > 0.f)) return PPAS_EINVAL;
    ppas_status st = validate(shape, seqs, n_seqs, block_table_host, bt_stride, true);
    if (st != PPAS_OK) return st;
    if (n_seqs == 0) return PPAS_OK;
    if (!q || !k_pages || !v_pages || !k_new || !v_new || !block_table_dev) return PPAS_EINVAL;
    if (!current_device().gfx950) return PPAS_EUNSUPPORTED;
    const hipError_t e = launch_rope_append(static_cast<uint16_t*>(q), static_cast<uint16_t*>(k_pages),
                                            static_cast<uint16_t*>(v_pages), static_cast<const uint16_t*>(k_new),
                                            static_cast<const uint16_t*>(v_new), seqs, n_seqs, block_table_dev,
                                            bt_stride, shape->n_q_heads, shape->n_kv_heads, double(rope_theta),
                                            static_cast<hipStream_t>(hip_stream),
                                            static_cast<hipEvent_t>(g_ev_start.load()),
                                            static_cast<hipEvent_t>(g_ev_stop.load()));
    return e == hipSuccess ? PPAS_OK : PPAS_EHIP;
  } catch (...) {
    return PPAS_EINVAL;
  }
}

ppas_status ppas_attn_step(const ppas_shape* shape, void* out, const void* q, const void* k_pages,
                           const void* v_pages, const ppas_seq* seqs, int32_t n_seqs,
                           const int32_t* block_table_dev, int32_t bt_stride, const int32_t* block_table_host,
                           void* workspace, size_t workspace_bytes, void* hip_stream) {
  try {
    ppas_status st = validate(shape, seqs, n_seqs, block_table_host, bt_stride, false);
    if (st != PPAS_OK) return st;
    if (n_seqs == 0) return PPAS_OK;
    if (!out || !q || !k_pages || !v_pages || !block_table_dev || !workspace) return PPAS_EINVAL;
    const DeviceInfo dev = current_device();
    if (!dev.gfx950) return PPAS_EUNSUPPORTED;
    Plan plan;
    make_plan(*shape, seqs, n_seqs, dev.cus, plan);
    if (!plan_fits(plan)) return PPAS_ERANGE;
    if (workspace_bytes < plan.total) return PPAS_ENOSPACE;
    hipStream_t stream = static_cast<hipStream_t>(hip_stream);
    char* ws = static_cast<char*>(workspace);
    // The work list (items, then combine items at their aligned offset) goes into a
    // pinned staging slot that the kernels read directly; the workspace holds the
    // split partials.
    std::lock_guard<std::mutex> lk(g_stage_mu);
    Slot* slot = nullptr;
    st = take_slot(plan.list_bytes, slot);
    if (st != PPAS_OK) return st;
    char* host = static_cast<char*>(slot->host);
    std::memcpy(host, plan.items.data(), plan.items.size() * sizeof(WorkItem));
    if (!plan.combine.empty())
      std::memcpy(host + plan.off_combine, plan.combine.data(), plan.combine.size() * sizeof(CombineItem));
    const hipError_t e = launch_attn_step(
        static_cast<const uint16_t*>(q), static_cast<uint16_t*>(out), static_cast<const uint16_t*>(k_pages),
        static_cast<const uint16_t*>(v_pages), block_table_dev, bt_stride, shape->n_q_heads, shape->n_kv_heads,
        shape->scale, reinterpret_cast<const WorkItem*>(slot->dev), int(plan.items.size()),
        reinterpret_cast<const CombineItem*>(slot->dev + plan.off_combine), int(plan.combine.size()),
        reinterpret_cast<float2*>(ws + plan.off_ml), reinterpret_cast<float*>(ws + plan.off_acc), plan.tile_pos, stream,
        static_cast<hipEvent_t>(g_ev_start.load()), static_cast<hipEvent_t>(g_ev_stop.load()));
    // the slot is free again once the last kernel that reads it has finished (also
    // after a failed launch: a kernel that did start may still read it)
    const bool recorded = hipEventRecord(slot->done, stream) == hipSuccess;
    slot->pending = recorded;
    // without the event, drain the stream before the slot can be refilled
    if (!recorded) (void)hipStreamSynchronize(stream);
    return (e == hipSuccess && recorded) ? PPAS_OK : PPAS_EHIP;
  } catch (...) {
    return PPAS_EINVAL;
  }
}

}  // extern "C"
