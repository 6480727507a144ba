// ppas_attn_step_noalloc: the attention step of ppas_attn_step for callers
// that cannot allocate memory. The work list and the split partials live in a
// fixed-size file-scope device array instead of a caller workspace and the
// library's pinned host pool; the kernels are the same.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <mutex>
#include <vector>

#include "device.h"
#include "plan.h"
#include "ppas.h"

namespace ppas {
namespace {

// Each device the library runs on holds its own copy until the process ends.
// In host code this name is only a handle for hipGetSymbolAddress: the device
// address of the current device's copy is what the kernels and copies take.
static __device__ __align__(256) char scratch[PPAS_NOALLOC_SCRATCH_BYTES];

std::mutex g_scratch_mu;
std::vector<char*> g_scratch_ptr;   // per device id; nullptr until resolved

// Device address of the current device's scratch array, resolved once per
// device with that device current.
ppas_status scratch_of_current_device(char** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return PPAS_EHIP;
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (dev >= int(g_scratch_ptr.size())) g_scratch_ptr.resize(size_t(dev) + 1, nullptr);
  if (!g_scratch_ptr[size_t(dev)]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
      (void)hipGetLastError();
      return PPAS_EHIP;
    }
    g_scratch_ptr[size_t(dev)] = static_cast<char*>(ptr);
  }
  *out = g_scratch_ptr[size_t(dev)];
  return PPAS_OK;
}

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

ppas_status run(const ppas_shape* shape, void* out, const void* q, const void* k_pages, const void* v_pages,
                const ppas_seq* seqs, int32_t n_seqs, const int32_t* bt_dev, int32_t bt_stride,
                const int32_t* bt_host, void* hip_stream) {
  ppas_status st = validate(shape, seqs, n_seqs, bt_host, bt_stride, false);
  if (st != PPAS_OK) return st;
  if (n_seqs == 0) return PPAS_OK;
  if (!out || !q || !k_pages || !v_pages || !bt_dev) return PPAS_EINVAL;
  const DeviceInfo dev = current_device();
  Plan plan;
  make_plan(*shape, seqs, n_seqs, dev.cus, PlanOpts{}, plan);
  if (plan.items.size() > size_t(INT32_MAX) || plan.combine.size() > size_t(INT32_MAX)) return PPAS_ERANGE;
  // scratch layout: the work list (items, then merge items) from offset 0, the
  // split partials after it
  const size_t off_part = align256(plan.list_bytes);
  if (off_part > PPAS_NOALLOC_SCRATCH_BYTES || plan.total > PPAS_NOALLOC_SCRATCH_BYTES - off_part)
    return PPAS_ENOSPACE;
  if (!dev.gfx950) return PPAS_EUNSUPPORTED;
  char* base = nullptr;
  st = scratch_of_current_device(&base);
  if (st != PPAS_OK) return st;

  std::vector<char> list(plan.list_bytes, 0);
  std::memcpy(list.data(), plan.items.data(), plan.items.size() * sizeof(WorkItem));
  if (!plan.combine.empty())
    std::memcpy(list.data() + plan.off_combine, plan.combine.data(), plan.combine.size() * sizeof(CombineItem));
  hipStream_t stream = static_cast<hipStream_t>(hip_stream);
  // From pageable host memory: the source has been consumed when the call returns.
  if (hipMemcpyAsync(base, list.data(), list.size(), hipMemcpyHostToDevice, stream) != hipSuccess) {
    (void)hipGetLastError();
    return PPAS_EHIP;
  }
  char* part = base + off_part;
  const hipError_t e = launch_attn_step(
      static_cast<const uint16_t*>(q), static_cast<uint16_t*>(out), static_cast<const uint16_t*>(k_pages),
      static_cast<const uint16_t*>(v_pages), bt_dev, bt_stride, shape->n_q_heads, shape->n_kv_heads, shape->scale,
      reinterpret_cast<const WorkItem*>(base), int(plan.items.size()),
      reinterpret_cast<const CombineItem*>(base + plan.off_combine), int(plan.combine.size()),
      reinterpret_cast<float2*>(part + plan.off_ml), reinterpret_cast<float*>(part + plan.off_acc), plan.tile_pos,
      stream, nullptr, nullptr, nullptr, nullptr);
  return e == hipSuccess ? PPAS_OK : PPAS_EHIP;
}

}  // namespace
}  // namespace ppas

extern "C" ppas_status ppas_attn_step_noalloc(const ppas_shape* shape, void* out, const void* q,
                                              const void* k_pages, const void* v_pages, const ppas_seq* seqs,
                                              int32_t n_seqs, const int32_t* block_table_dev, int32_t bt_stride,
                                              const int32_t* block_table_host, void* hip_stream) {
  try {
    return ppas::run(shape, out, q, k_pages, v_pages, seqs, n_seqs, block_table_dev, bt_stride, block_table_host,
                     hip_stream);
  } catch (...) {
    return PPAS_EINVAL;
  }
}
