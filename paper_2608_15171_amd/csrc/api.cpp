// extern "C" entry points of libppas.so (declared in include/ppas.h).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <utility>
#include <vector>

#include "device.h"
#include "plan.h"
#include "ppas.h"

namespace ppas {

hipError_t launch_kv_append(uint16_t* kp, uint16_t* vp, const uint16_t* kn, const uint16_t* vn,
                            const AppendItem* items, int32_t n_items, const int32_t* bt, int32_t bt_stride,
                            int32_t hkv, hipStream_t stream, hipEvent_t ev_start, hipEvent_t ev_stop);
hipError_t launch_rope_append(uint16_t* q, uint16_t* kp, uint16_t* vp, const uint16_t* kn, const uint16_t* vn,
                              const AppendItem* items, int32_t n_items, const int32_t* bt, int32_t bt_stride,
                              int32_t hq, int32_t hkv, double theta, hipStream_t stream, hipEvent_t ev_start,
                              hipEvent_t ev_stop);

namespace {

std::mutex g_dev_mu;
std::vector<DeviceInfo> g_dev;

}  // namespace

// Compute-unit count and architecture of the current device (cached). Without a
// usable device, reports 256 CUs and not-gfx950.
DeviceInfo current_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return DeviceInfo{};
  }
  std::lock_guard<std::mutex> lk(g_dev_mu);
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

namespace {

// Work-item counts and partial-slot offsets travel as int32 (and the item count
// sets the launch grid): a step too large for that is refused.
bool plan_fits(const Plan& plan, size_t n_append) {
  return plan.items.size() <= size_t(INT32_MAX) && plan.combine.size() <= size_t(INT32_MAX) &&
         n_append <= size_t(INT32_MAX) && plan.part_slots <= int64_t(INT32_MAX) - 64 * kGroup;
}

ppas_status check_opts(const ppas_plan_opts* o) {
  if (!o) return PPAS_OK;
  if (o->prefill_split < 0 || o->decode_split < 0 || o->num_cus < 0) return PPAS_EINVAL;
  if (o->tile_positions != 0 && o->tile_positions != kTilePosSmall && o->tile_positions != kTilePosLarge)
    return PPAS_EINVAL;
  return PPAS_OK;
}

PlanOpts to_opts(const ppas_plan_opts* o) {
  PlanOpts p;
  if (o) {
    p.prefill_split = o->prefill_split;
    p.decode_split = o->decode_split;
    p.tile_pos = o->tile_positions;
  }
  return p;
}

ppas_status check_events(const ppas_events* ev) {
  if (!ev) return PPAS_OK;
  if ((ev->start == nullptr) != (ev->stop == nullptr)) return PPAS_EINVAL;
  if ((ev->merge_start == nullptr) != (ev->merge_stop == nullptr)) return PPAS_EINVAL;
  return PPAS_OK;
}

hipEvent_t ev_of(const ppas_events* ev, int which) {
  if (!ev) return nullptr;
  void* const e[4] = {ev->start, ev->stop, ev->merge_start, ev->merge_stop};
  return static_cast<hipEvent_t>(e[which]);
}

// ---------------------------------------------------------------------------
// Pinned host buffers holding work lists. The kernels read their items straight
// from this memory: each workgroup reads its 32-byte item once, which costs less
// than a host-to-device copy on a separate engine and the two cross-engine
// waits around it. A buffer in use belongs to one plan; once released it is
// handed out again only after every launch that read it has completed (an event
// is recorded behind those launches, one per stream).
// ---------------------------------------------------------------------------
struct Pinned {
  void* host = nullptr;
  char* dev = nullptr;      // the same memory as the device addresses it
  size_t cap = 0;
  bool in_use = false;
  bool settled = true;      // every recorded use is known to have completed
  std::vector<std::pair<hipStream_t, hipEvent_t>> uses;
};

constexpr size_t kPoolMax = 64;   // buffers kept; beyond that a call reuses a released one
std::mutex g_pool_mu;
std::vector<Pinned*> g_pool;

bool idle(Pinned& b) {
  if (b.settled) return true;
  for (const auto& u : b.uses) {
    const hipError_t e = hipEventQuery(u.second);
    if (e == hipErrorNotReady) return false;
    if (e != hipSuccess) (void)hipGetLastError();
  }
  b.settled = true;
  return true;
}

void drop_events(Pinned& b) {
  for (auto& u : b.uses) (void)hipEventDestroy(u.second);
  b.uses.clear();
}

ppas_status grow(Pinned& b, size_t bytes) {
  if (b.cap >= bytes) return PPAS_OK;
  if (b.host) (void)hipHostFree(b.host);
  b.host = nullptr;
  b.dev = nullptr;
  b.cap = 0;
  size_t cap = size_t(1) << 16;
  while (cap < bytes) cap <<= 1;
  if (hipHostMalloc(&b.host, cap, hipHostMallocDefault) != hipSuccess) {
    b.host = nullptr;
    return PPAS_EHIP;
  }
  void* d = nullptr;
  if (hipHostGetDevicePointer(&d, b.host, 0) != hipSuccess) {
    (void)hipHostFree(b.host);
    b.host = nullptr;
    return PPAS_EHIP;
  }
  b.dev = static_cast<char*>(d);
  b.cap = cap;
  return PPAS_OK;
}

// A buffer of at least `bytes`, marked in use.
ppas_status acquire(size_t bytes, Pinned*& out) {
  std::lock_guard<std::mutex> lk(g_pool_mu);
  Pinned* pick = nullptr;
  for (Pinned* b : g_pool)   // the smallest idle buffer that fits
    if (!b->in_use && b->cap >= bytes && idle(*b) && (!pick || b->cap < pick->cap)) pick = b;
  if (!pick && g_pool.size() < kPoolMax) {
    pick = new (std::nothrow) Pinned;
    if (!pick) return PPAS_EHIP;
    g_pool.push_back(pick);
  }
  if (!pick)   // the pool is full: an idle buffer that is too small, grown
    for (Pinned* b : g_pool)
      if (!b->in_use && idle(*b)) pick = b;
  if (!pick) {  // else wait for a released buffer whose launches are still running
    for (Pinned* b : g_pool)
      if (!b->in_use) pick = b;
    if (pick) {
      for (auto& u : pick->uses)
        if (hipEventSynchronize(u.second) != hipSuccess) return PPAS_EHIP;
      pick->settled = true;
    }
  }
  if (!pick) {  // every buffer belongs to a live plan: the pool grows past its cap
    pick = new (std::nothrow) Pinned;
    if (!pick) return PPAS_EHIP;
    g_pool.push_back(pick);
  }
  if (pick->uses.size() > 8) drop_events(*pick);
  const ppas_status st = grow(*pick, bytes);
  if (st != PPAS_OK) return st;
  pick->in_use = true;
  out = pick;
  return PPAS_OK;
}

// Records, behind the work just enqueued on `stream`, that the buffer was read.
// Without the event the stream is drained, so the buffer is never reused early.
bool note_use(Pinned* b, hipStream_t stream) {
  std::lock_guard<std::mutex> lk(g_pool_mu);
  hipEvent_t ev = nullptr;
  for (auto& u : b->uses)
    if (u.first == stream) ev = u.second;
  if (!ev) {
    if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) {
      (void)hipStreamSynchronize(stream);
      return false;
    }
    b->uses.emplace_back(stream, ev);
  }
  if (hipEventRecord(ev, stream) != hipSuccess) {
    (void)hipStreamSynchronize(stream);
    return false;
  }
  b->settled = false;
  return true;
}

void release(Pinned* b) {
  if (!b) return;
  std::lock_guard<std::mutex> lk(g_pool_mu);
  b->in_use = false;
}

}  // namespace
}  // namespace ppas

using namespace ppas;

// The plan of one step: validated descriptors, the attention work list and the
// page-write list, staged in one pinned buffer.
struct ppas_step_plan {
  ppas_shape shape{};
  int32_t bt_stride = 0;
  int32_t n_seqs = 0;
  Plan plan;
  int32_t n_append = 0;
  size_t off_append = 0;
  Pinned* buf = nullptr;
};

namespace {

enum : int { kWantAttn = 1, kWantAppend = 2 };

// Validate, plan and stage. On success p.buf holds the lists (nullptr for an empty step).
ppas_status build_plan(ppas_step_plan& p, const ppas_shape* shape, const ppas_seq* seqs, int32_t n_seqs,
                       const int32_t* bt_host, int32_t bt_stride, const ppas_plan_opts* opts, int want,
                       bool check_overlap) {
  ppas_status st = check_opts(opts);
  if (st != PPAS_OK) return st;
  st = validate(shape, seqs, n_seqs, bt_host, bt_stride, check_overlap);
  if (st != PPAS_OK) return st;
  p.shape = *shape;
  p.bt_stride = bt_stride;
  p.n_seqs = n_seqs;
  if (n_seqs == 0) return PPAS_OK;
  const DeviceInfo dev = current_device();
  if (!dev.gfx950) return PPAS_EUNSUPPORTED;
  std::vector<AppendItem> app;
  if (want & kWantAttn)
    make_plan(*shape, seqs, n_seqs, (opts && opts->num_cus > 0) ? opts->num_cus : dev.cus, to_opts(opts), p.plan);
  if (want & kWantAppend) make_append_items(seqs, n_seqs, app);
  if (!plan_fits(p.plan, app.size())) return PPAS_ERANGE;
  p.n_append = int32_t(app.size());
  const size_t list = (want & kWantAttn) ? p.plan.list_bytes : 0;
  p.off_append = (list + 255) / 256 * 256;
  const size_t bytes = p.off_append + app.size() * sizeof(AppendItem);
  st = acquire(std::max<size_t>(bytes, 256), p.buf);
  if (st != PPAS_OK) return st;
  char* host = static_cast<char*>(p.buf->host);
  if (!p.plan.items.empty()) std::memcpy(host, p.plan.items.data(), p.plan.items.size() * sizeof(WorkItem));
  if (!p.plan.combine.empty())
    std::memcpy(host + p.plan.off_combine, p.plan.combine.data(), p.plan.combine.size() * sizeof(CombineItem));
  if (!app.empty()) std::memcpy(host + p.off_append, app.data(), app.size() * sizeof(AppendItem));
  return PPAS_OK;
}

ppas_status run_append(const ppas_step_plan& p, bool rope, float theta, void* q, void* k_pages, void* v_pages,
                       const void* k_new, const void* v_new, const int32_t* bt_dev, const ppas_events* ev,
                       void* hip_stream) {
  if (p.n_seqs == 0) return PPAS_OK;
  if (!k_pages || !v_pages || !k_new || !v_new || !bt_dev || (rope && !q)) return PPAS_EINVAL;
  if (!p.buf || p.n_append == 0) return PPAS_EINVAL;   // a plan made without the page-write list
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  const AppendItem* items = reinterpret_cast<const AppendItem*>(p.buf->dev + p.off_append);
  hipError_t e;
  if (rope)
    e = launch_rope_append(static_cast<uint16_t*>(q), static_cast<uint16_t*>(k_pages), static_cast<uint16_t*>(v_pages),
                           static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new), items, p.n_append,
                           bt_dev, p.bt_stride, p.shape.n_q_heads, p.shape.n_kv_heads, double(theta), stream,
                           ev_of(ev, 0), ev_of(ev, 1));
  else
    e = launch_kv_append(static_cast<uint16_t*>(k_pages), static_cast<uint16_t*>(v_pages),
                         static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new), items, p.n_append,
                         bt_dev, p.bt_stride, p.shape.n_kv_heads, stream, ev_of(ev, 0), ev_of(ev, 1));
  // the buffer is free again once the kernel that reads it has finished (also
  // after a failed launch: a kernel that did start may still read it)
  const bool noted = note_use(p.buf, stream);
  return (e == hipSuccess && noted) ? PPAS_OK : PPAS_EHIP;
}

ppas_status run_attn(const ppas_step_plan& p, void* out, const void* q, const void* k_pages, const void* v_pages,
                     const int32_t* bt_dev, void* workspace, size_t workspace_bytes, const ppas_events* ev,
                     void* hip_stream) {
  if (p.n_seqs == 0) return PPAS_OK;
  if (!out || !q || !k_pages || !v_pages || !bt_dev || !workspace) return PPAS_EINVAL;
  if (!p.buf || p.plan.items.empty()) return PPAS_EINVAL;   // a plan made without the attention list
  if (workspace_bytes < p.plan.total) return PPAS_ENOSPACE;
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  char* ws = static_cast<char*>(workspace);
  const Plan& plan = p.plan;
  const hipError_t e = launch_attn_step(
      static_cast<const uint16_t*>(q), static_cast<uint16_t*>(out), static_cast<const uint16_t*>(k_pages),
      static_cast<const uint16_t*>(v_pages), bt_dev, p.bt_stride, p.shape.n_q_heads, p.shape.n_kv_heads,
      p.shape.scale, reinterpret_cast<const WorkItem*>(p.buf->dev), int(plan.items.size()),
      reinterpret_cast<const CombineItem*>(p.buf->dev + plan.off_combine), int(plan.combine.size()),
      reinterpret_cast<float2*>(ws + plan.off_ml), reinterpret_cast<float*>(ws + plan.off_acc), plan.tile_pos,
      stream, ev_of(ev, 0), ev_of(ev, 1), ev_of(ev, 2), ev_of(ev, 3));
  const bool noted = note_use(p.buf, stream);
  return (e == hipSuccess && noted) ? PPAS_OK : PPAS_EHIP;
}

}  // namespace

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

int32_t ppas_plan_items(const ppas_shape* shape, const ppas_seq* seqs, int32_t n_seqs, const ppas_plan_opts* opts,
                        int32_t* items_out, int32_t capacity) {
  try {
    ppas_status st = check_opts(opts);
    if (st != PPAS_OK) return st;
    st = validate(shape, seqs, n_seqs, nullptr, INT32_MAX, false);
    if (st != PPAS_OK) return st;
    Plan plan;
    make_plan(*shape, seqs, n_seqs, (opts && opts->num_cus > 0) ? opts->num_cus : 256, to_opts(opts), plan);
    if (!plan_fits(plan, 0)) return PPAS_ERANGE;
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
    make_plan(*shape, seqs, n_seqs, current_device().cus, PlanOpts{}, plan);
    return plan_fits(plan, 0) ? plan.total : 0;
  } catch (...) {
    return 0;
  }
}

ppas_status ppas_step_plan_create(const ppas_shape* shape, const ppas_seq* seqs, int32_t n_seqs,
                                  const int32_t* block_table_host, int32_t bt_stride, const ppas_plan_opts* opts,
                                  ppas_step_plan** plan) {
  if (!plan) return PPAS_EINVAL;
  *plan = nullptr;
  ppas_step_plan* p = nullptr;
  try {
    p = new ppas_step_plan;
    const ppas_status st =
        build_plan(*p, shape, seqs, n_seqs, block_table_host, bt_stride, opts, kWantAttn | kWantAppend, true);
    if (st != PPAS_OK) {
      release(p->buf);
      delete p;
      return st;
    }
    *plan = p;
    return PPAS_OK;
  } catch (...) {
    if (p) {
      release(p->buf);
      delete p;
    }
    return PPAS_EINVAL;
  }
}

ppas_status ppas_step_plan_info(const ppas_step_plan* plan, ppas_plan_info* info) {
  if (!plan || !info) return PPAS_EINVAL;
  info->n_items = int32_t(plan->plan.items.size());
  info->n_merge = int32_t(plan->plan.combine.size());
  info->tile_positions = plan->plan.tile_pos;
  info->n_append = plan->n_append;
  info->workspace_bytes = plan->n_seqs ? uint64_t(plan->plan.total) : 256;
  return PPAS_OK;
}

void ppas_step_plan_destroy(ppas_step_plan* plan) {
  if (!plan) return;
  release(plan->buf);
  delete plan;
}

ppas_status ppas_kv_append_planned(const ppas_step_plan* plan, void* k_pages, void* v_pages, const void* k_new,
                                   const void* v_new, const int32_t* block_table_dev, const ppas_events* events,
                                   void* hip_stream) {
  if (!plan) return PPAS_EINVAL;
  const ppas_status st = check_events(events);
  if (st != PPAS_OK) return st;
  try {
    return run_append(*plan, false, 0.f, nullptr, k_pages, v_pages, k_new, v_new, block_table_dev, events,
                      hip_stream);
  } catch (...) {
    return PPAS_EINVAL;
  }
}

ppas_status ppas_rope_kv_append_planned(const ppas_step_plan* plan, float rope_theta, void* q, void* k_pages,
                                        void* v_pages, const void* k_new, const void* v_new,
                                        const int32_t* block_table_dev, const ppas_events* events,
                                        void* hip_stream) {
  if (!plan) return PPAS_EINVAL;
  if (!std::isfinite(rope_theta) || !(rope_theta > 0.f)) return PPAS_EINVAL;
  const ppas_status st = check_events(events);
  if (st != PPAS_OK) return st;
  try {
    return run_append(*plan, true, rope_theta, q, k_pages, v_pages, k_new, v_new, block_table_dev, events,
                      hip_stream);
  } catch (...) {
    return PPAS_EINVAL;
  }
}

ppas_status ppas_attn_step_planned(const ppas_step_plan* plan, void* out, const void* q, const void* k_pages,
                                   const void* v_pages, const int32_t* block_table_dev, void* workspace,
                                   size_t workspace_bytes, const ppas_events* events, void* hip_stream) {
  if (!plan) return PPAS_EINVAL;
  const ppas_status st = check_events(events);
  if (st != PPAS_OK) return st;
  try {
    return run_attn(*plan, out, q, k_pages, v_pages, block_table_dev, workspace, workspace_bytes, events,
                    hip_stream);
  } catch (...) {
    return PPAS_EINVAL;
  }
}

namespace {

ppas_status check_gateup(int32_t n_tokens, int32_t hidden, int32_t n_out) {
  if (n_tokens < 0 || hidden <= 0 || n_out <= 0) return PPAS_EINVAL;
  if (hidden % 64 != 0) return PPAS_EUNSUPPORTED;
  // tile origins and edges stay inside int32, and the grid inside its limit
  if (n_tokens > INT32_MAX - 512 || n_out > INT32_MAX - 512) return PPAS_ERANGE;
  if (gateup_tiles(n_tokens, n_out) > INT32_MAX) return PPAS_ERANGE;
  return PPAS_OK;
}

}  // namespace

size_t ppas_gateup_workspace_bytes(int32_t n_tokens, int32_t hidden, int32_t n_out) {
  try {
    if (check_gateup(n_tokens, hidden, n_out) != PPAS_OK || n_tokens == 0) return 0;
    return gateup_workspace_bytes(n_tokens, n_out, gateup_splits(n_tokens, hidden, n_out, current_device().cus));
  } catch (...) {
    return 0;
  }
}

namespace {

// Both projection entry points: n_out weight rows; with `act` the output holds the
// gated activation of the two halves (n_out / 2 columns).
ppas_status gateup_call(const void* x, const void* w, void* y, int32_t n_tokens, int32_t hidden, int32_t n_out,
                        bool act, void* workspace, size_t workspace_bytes, const ppas_events* events,
                        void* hip_stream) {
  ppas_status st = check_gateup(n_tokens, hidden, n_out);
  if (st != PPAS_OK) return st;
  st = check_events(events);
  if (st != PPAS_OK) return st;
  if (n_tokens == 0) return PPAS_OK;
  if (!x || !w || !y || (workspace_bytes > 0 && !workspace)) return PPAS_EINVAL;
  const DeviceInfo dev = current_device();
  if (!dev.gfx950) return PPAS_EUNSUPPORTED;
  // the automatic split, reduced to what the workspace holds (no split needs none)
  int splits = gateup_splits(n_tokens, hidden, n_out, dev.cus);
  while (splits > 1 && gateup_workspace_bytes(n_tokens, n_out, splits) > workspace_bytes) --splits;
  if (gateup_tiles(n_tokens, n_out) * splits > INT32_MAX) splits = 1;
  const hipError_t e = launch_gateup(static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w),
                                     static_cast<uint16_t*>(y), n_tokens, hidden, n_out, act, splits,
                                     static_cast<float*>(workspace), dev.cus, static_cast<hipStream_t>(hip_stream),
                                     ev_of(events, 0), ev_of(events, 1));
  return e == hipSuccess ? PPAS_OK : PPAS_EHIP;
}

// weight rows of the activated projection (two per intermediate feature), or -1
int32_t act_rows(int32_t n_inter) { return (n_inter <= 0 || n_inter > (INT32_MAX - 512) / 2) ? -1 : 2 * n_inter; }

}  // namespace

ppas_status ppas_gateup_proj(const void* x, const void* w, void* y, int32_t n_tokens, int32_t hidden, int32_t n_out,
                             void* workspace, size_t workspace_bytes, const ppas_events* events, void* hip_stream) {
  try {
    return gateup_call(x, w, y, n_tokens, hidden, n_out, false, workspace, workspace_bytes, events, hip_stream);
  } catch (...) {
    return PPAS_EINVAL;
  }
}

size_t ppas_gateup_act_workspace_bytes(int32_t n_tokens, int32_t hidden, int32_t n_inter) {
  const int32_t n_out = act_rows(n_inter);
  return n_out < 0 ? 0 : ppas_gateup_workspace_bytes(n_tokens, hidden, n_out);
}

ppas_status ppas_gateup_act(const void* x, const void* w, void* y, int32_t n_tokens, int32_t hidden, int32_t n_inter,
                            void* workspace, size_t workspace_bytes, const ppas_events* events, void* hip_stream) {
  try {
    if (n_inter > (INT32_MAX - 512) / 2) return PPAS_ERANGE;
    const int32_t n_out = act_rows(n_inter);
    if (n_out < 0) return PPAS_EINVAL;
    return gateup_call(x, w, y, n_tokens, hidden, n_out, true, workspace, workspace_bytes, events, hip_stream);
  } catch (...) {
    return PPAS_EINVAL;
  }
}

ppas_status ppas_stream_read(const void* buf, size_t bytes, void* sink, const ppas_events* events,
                             void* hip_stream) {
  try {
    const ppas_status st = check_events(events);
    if (st != PPAS_OK) return st;
    if (!buf || !sink || bytes % 16 != 0 || reinterpret_cast<uintptr_t>(buf) % 16 != 0 ||
        reinterpret_cast<uintptr_t>(sink) % 4 != 0)
      return PPAS_EINVAL;
    if (bytes == 0) return PPAS_OK;
    const DeviceInfo dev = current_device();
    if (!dev.gfx950) return PPAS_EUNSUPPORTED;
    const hipError_t e = launch_stream_read(buf, bytes, static_cast<uint32_t*>(sink), dev.cus,
                                            static_cast<hipStream_t>(hip_stream), ev_of(events, 0),
                                            ev_of(events, 1));
    return e == hipSuccess ? PPAS_OK : PPAS_EHIP;
  } catch (...) {
    return PPAS_EINVAL;
  }
}

ppas_status ppas_kv_append(const ppas_shape* shape, void* k_pages, void* v_pages, const void* k_new,
                           const void* v_new, const ppas_seq* seqs, int32_t n_seqs,
                           const int32_t* block_table_dev, int32_t bt_stride,
                           const int32_t* block_table_host, void* hip_stream) {
  ppas_step_plan p;
  try {
    ppas_status st = validate(shape, seqs, n_seqs, block_table_host, bt_stride, true);
    if (st != PPAS_OK) return st;
    if (n_seqs == 0) return PPAS_OK;
    if (!k_pages || !v_pages || !k_new || !v_new || !block_table_dev) return PPAS_EINVAL;
    // validated above; build only the page-write list
    st = build_plan(p, shape, seqs, n_seqs, nullptr, bt_stride, nullptr, kWantAppend, false);
    if (st == PPAS_OK) st = run_append(p, false, 0.f, nullptr, k_pages, v_pages, k_new, v_new, block_table_dev,
                                       nullptr, hip_stream);
    release(p.buf);
    return st;
  } catch (...) {
    release(p.buf);
    return PPAS_EINVAL;
  }
}

ppas_status ppas_rope_kv_append(const ppas_shape* shape, float rope_theta, void* q, void* k_pages, void* v_pages,
                                const void* k_new, const void* v_new, const ppas_seq* seqs, int32_t n_seqs,
                                const int32_t* block_table_dev, int32_t bt_stride,
                                const int32_t* block_table_host, void* hip_stream) {
  ppas_step_plan p;
  try {
    if (!std::isfinite(rope_theta) || !(rope_theta > 0.f)) return PPAS_EINVAL;
    ppas_status st = validate(shape, seqs, n_seqs, block_table_host, bt_stride, true);
    if (st != PPAS_OK) return st;
    if (n_seqs == 0) return PPAS_OK;
    if (!q || !k_pages || !v_pages || !k_new || !v_new || !block_table_dev) return PPAS_EINVAL;
    st = build_plan(p, shape, seqs, n_seqs, nullptr, bt_stride, nullptr, kWantAppend, false);
    if (st == PPAS_OK) st = run_append(p, true, rope_theta, q, k_pages, v_pages, k_new, v_new, block_table_dev,
                                       nullptr, hip_stream);
    release(p.buf);
    return st;
  } catch (...) {
    release(p.buf);
    return PPAS_EINVAL;
  }
}

ppas_status ppas_attn_step(const ppas_shape* shape, void* out, const void* q, const void* k_pages,
                           const void* v_pages, const ppas_seq* seqs, int32_t n_seqs,
                           const int32_t* block_table_dev, int32_t bt_stride, const int32_t* block_table_host,
                           void* workspace, size_t workspace_bytes, void* hip_stream) {
  ppas_step_plan p;
  try {
    ppas_status st = validate(shape, seqs, n_seqs, block_table_host, bt_stride, false);
    if (st != PPAS_OK) return st;
    if (n_seqs == 0) return PPAS_OK;
    if (!out || !q || !k_pages || !v_pages || !block_table_dev || !workspace) return PPAS_EINVAL;
    st = build_plan(p, shape, seqs, n_seqs, nullptr, bt_stride, nullptr, kWantAttn, false);
    if (st == PPAS_OK)
      st = run_attn(p, out, q, k_pages, v_pages, block_table_dev, workspace, workspace_bytes, nullptr, hip_stream);
    release(p.buf);
    return st;
  } catch (...) {
    release(p.buf);
    return PPAS_EINVAL;
  }
}

}  // extern "C"
