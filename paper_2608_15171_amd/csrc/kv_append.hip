// Scatter a step's new K/V rows into the paged cache (bit copies).
//
// One workgroup per (request, touched page, KV head); the (request, page) pairs
// come from a list the host builds, so one launch covers any number of requests. The K page of one head is
// 16 chunks of 8 features, each holding the 16 slots' 16-byte pieces: thread t
// copies the piece (chunk t/16, slot t%16) when that slot is one of the step's
// positions, so a workgroup's K stores are one contiguous 4 KB run. The V page
// of one head is 128 feature rows of 16 tokens: thread t owns the chunk
// (feature t/2, slots 8(t%2)..+7), gathers those slots from the new rows, and
// stores the whole chunk when all 8 slots are new, else only the new elements.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>

#include "plan.h"

namespace ppas {

struct AppendArgs {
  uint16_t* kp;
  uint16_t* vp;
  const uint16_t* kn;
  const uint16_t* vn;
  const int32_t* bt;
  const AppendItem* items;   // one per workgroup (x): request and logical page
  int32_t bt_stride, hkv;
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void kv_append_kernel(AppendArgs a) {
  const AppendItem it = a.items[blockIdx.x];
  const int g = blockIdx.y, tid = threadIdx.x;
  const int c = it.cached_len, nq = it.n_query, qs = it.query_start;
  const int lpage = it.lpage;
  const int pos_lo = lpage * kPage;                       // position of slot 0 of this page
  const int32_t page = a.bt[size_t(it.seq) * a.bt_stride + lpage];
  const size_t base = (size_t(page) * a.hkv + g) * kPage * kHeadDim;
  const size_t row_stride = size_t(a.hkv) * kHeadDim;     // elements between new rows

  // K: chunk tid/16 (features 8*(tid/16)..+7), slot tid%16
  {
    const int chunk = tid >> 4, slot = tid & 15;
    const int pos = pos_lo + slot;
    if (pos >= c && pos < c + nq) {
      const uint16_t* src = a.kn + size_t(qs + pos - c) * row_stride + g * kHeadDim + 8 * chunk;
      *reinterpret_cast<u32x4*>(a.kp + base + 8 * tid) = *reinterpret_cast<const u32x4*>(src);
    }
  }
  // V: feature tid/2, slots 8*(tid%2)..+7
  {
    const int d = tid >> 1;
    const int s0 = 8 * (tid & 1);
    uint16_t* dst = a.vp + base + d * kPage + s0;
    uint16_t vals[8];
    int cnt = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int pos = pos_lo + s0 + e;
      const bool mine = pos >= c && pos < c + nq;
      vals[e] = mine ? a.vn[size_t(qs + pos - c) * row_stride + g * kHeadDim + d] : uint16_t(0);
      cnt += mine;
    }
    if (cnt == 8) {
      u32x4 v;
#pragma unroll
      for (int w = 0; w < 4; ++w) v[w] = uint32_t(vals[2 * w]) | (uint32_t(vals[2 * w + 1]) << 16);
      *reinterpret_cast<u32x4*>(dst) = v;
    } else if (cnt > 0) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int pos = pos_lo + s0 + e;
        if (pos >= c && pos < c + nq) dst[e] = vals[e];
      }
    }
  }
}

hipError_t launch_kv_append(uint16_t* kp, uint16_t* vp, const uint16_t* kn, const uint16_t* vn,
                            const AppendItem* items, int32_t n_items, const int32_t* bt, int32_t bt_stride,
                            int32_t hkv, hipStream_t stream, hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (n_items <= 0) return hipSuccess;
  AppendArgs a;
  a.kp = kp;
  a.vp = vp;
  a.kn = kn;
  a.vn = vn;
  a.bt = bt;
  a.items = items;
  a.bt_stride = bt_stride;
  a.hkv = hkv;
  hipExtLaunchKernelGGL(kv_append_kernel, dim3(n_items, hkv), dim3(256), 0, stream, ev_start, ev_stop, 0, a);
  return hipGetLastError();
}

}  // namespace ppas
