// Rotary position embedding of a step's new query and key rows, fused with the
// page write of the new keys and values.
//
// Positional rotation is not described by the paper; the operation is the
// standard rotate-half rotary embedding over the whole head: at position p,
// feature pairs (i, i + 64) of every query and key head turn by the angle
// p * theta^(-2i/128). Query rows are rotated in place; rotated keys go to the
// pages exactly where the plain append puts keys; values are copied unrotated.
//
// One workgroup per (request, touched page), from a list the host builds: it covers up to 16 consecutive
// positions of one request and all heads of those rows, so the cos/sin pairs of
// its positions are computed once (16 x 64 entries in LDS) and shared by the 16
// query heads and the KV heads. Angles are reduced in fp64 (whole turns
// removed), then cos and sin are taken in fp32; the rotation itself is fp32 and
// results are rounded to bf16 nearest-even. Memory access: a query head row is
// 8 threads, each reading and writing 16 bytes from each half (the two halves
// pair up), so a wave covers 2 KB of contiguous rows; key pieces are stored in
// the page's chunk-major order, 16 consecutive slots per chunk.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "plan.h"

namespace ppas {

constexpr int kRopePairs = kHeadDim / 2;

struct RopeArgs {
  uint16_t* q;
  uint16_t* kp;
  uint16_t* vp;
  const uint16_t* kn;
  const uint16_t* vn;
  const int32_t* bt;
  const AppendItem* items;               // one per workgroup: request and logical page
  int32_t bt_stride, hq, hkv;
  double turns[kRopePairs];              // turns per position of pair i: theta^(-2i/128) / (2 pi)
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float lo_f(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_f(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  const f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// x holds features f..f+7 of the first half, y features f+64..f+71; cs[e] = (cos, sin)
// of pair f+e.
__device__ __forceinline__ void rotate8(u32x4& x, u32x4& y, const float2* cs) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float2 c0 = cs[2 * w], c1 = cs[2 * w + 1];
    const float x0 = lo_f(x[w]), x1 = hi_f(x[w]), y0 = lo_f(y[w]), y1 = hi_f(y[w]);
    x[w] = pack2(fmaf(x0, c0.x, -(y0 * c0.y)), fmaf(x1, c1.x, -(y1 * c1.y)));
    y[w] = pack2(fmaf(y0, c0.x, x0 * c0.y), fmaf(y1, c1.x, x1 * c1.y));
  }
}

__global__ __launch_bounds__(256) void rope_append_kernel(RopeArgs a) {
  __shared__ float2 cs[kPage][kRopePairs];
  const AppendItem it = a.items[blockIdx.x];
  const int tid = threadIdx.x;
  const int c = it.cached_len, nq = it.n_query, qs = it.query_start;
  const int lpage = it.lpage;
  const int pos_lo = lpage * kPage;                                   // position of slot 0
  const int slot_lo = max(c - pos_lo, 0), slot_hi = min(c + nq - pos_lo, kPage);
  const int32_t page = a.bt[size_t(it.seq) * a.bt_stride + lpage];

  for (int e = tid; e < kPage * kRopePairs; e += blockDim.x) {
    const int slot = e / kRopePairs, i = e % kRopePairs;
    if (slot < slot_lo || slot >= slot_hi) continue;
    const double t = double(pos_lo + slot) * a.turns[i];
    const float ang = float((t - rint(t)) * (2.0 * M_PI));             // in [-pi, pi]
    float sn, cn;
    sincosf(ang, &sn, &cn);
    cs[slot][i] = make_float2(cn, sn);
  }
  __syncthreads();

  // Query rows, in place: task (slot, head, chunk j), j fastest.
  const int q_tasks = (slot_hi - slot_lo) * a.hq * 8;
  for (int t = tid; t < q_tasks; t += blockDim.x) {
    const int j = t & 7, hs = t >> 3;
    const int h = hs % a.hq, slot = slot_lo + hs / a.hq;
    uint16_t* p = a.q + (size_t(qs + pos_lo + slot - c) * a.hq + h) * kHeadDim + 8 * j;
    u32x4 x = *reinterpret_cast<const u32x4*>(p);
    u32x4 y = *reinterpret_cast<const u32x4*>(p + kRopePairs);
    rotate8(x, y, &cs[slot][8 * j]);
    *reinterpret_cast<u32x4*>(p) = x;
    *reinterpret_cast<u32x4*>(p + kRopePairs) = y;
  }

  const size_t row_stride = size_t(a.hkv) * kHeadDim;                // elements between new rows
  // Keys: task (head g, chunk j, slot), slot fastest; chunks j and j + 8 of the page.
  for (int t = tid; t < a.hkv * 8 * kPage; t += blockDim.x) {
    const int slot = t & 15, j = (t >> 4) & 7, g = t >> 7;
    if (slot < slot_lo || slot >= slot_hi) continue;
    const uint16_t* src = a.kn + size_t(qs + pos_lo + slot - c) * row_stride + g * kHeadDim + 8 * j;
    u32x4 x = *reinterpret_cast<const u32x4*>(src);
    u32x4 y = *reinterpret_cast<const u32x4*>(src + kRopePairs);
    rotate8(x, y, &cs[slot][8 * j]);
    uint16_t* dst = a.kp + (size_t(page) * a.hkv + g) * kPage * kHeadDim;
    *reinterpret_cast<u32x4*>(dst + (j * kPage + slot) * 8) = x;
    *reinterpret_cast<u32x4*>(dst + ((j + 8) * kPage + slot) * 8) = y;
  }

  // Values, unrotated: task (head g, feature d, half), owning slots 8 half .. +7 of
  // feature d's 16-slot run; whole 16-byte stores when all 8 slots are new.
  for (int t = tid; t < a.hkv * kHeadDim * 2; t += blockDim.x) {
    const int g = t / (2 * kHeadDim), d = (t >> 1) % kHeadDim, s0 = 8 * (t & 1);
    uint16_t* dst = a.vp + (size_t(page) * a.hkv + g) * kPage * kHeadDim + d * kPage + s0;
    uint16_t vals[8];
    int cnt = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const bool mine = s0 + e >= slot_lo && s0 + e < slot_hi;
      vals[e] = mine ? a.vn[size_t(qs + pos_lo + s0 + e - c) * row_stride + g * kHeadDim + d] : uint16_t(0);
      cnt += mine;
    }
    if (cnt == 8) {
      u32x4 v;
#pragma unroll
      for (int w = 0; w < 4; ++w) v[w] = uint32_t(vals[2 * w]) | (uint32_t(vals[2 * w + 1]) << 16);
      *reinterpret_cast<u32x4*>(dst) = v;
    } else if (cnt > 0) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (s0 + e >= slot_lo && s0 + e < slot_hi) dst[e] = vals[e];
    }
  }
}

hipError_t launch_rope_append(uint16_t* q, uint16_t* kp, uint16_t* vp, const uint16_t* kn, const uint16_t* vn,
                              const AppendItem* items, int32_t n_items, const int32_t* bt, int32_t bt_stride,
                              int32_t hq, int32_t hkv, double theta, hipStream_t stream, hipEvent_t ev_start,
                              hipEvent_t ev_stop) {
  if (n_items <= 0) return hipSuccess;
  RopeArgs a;
  for (int i = 0; i < kRopePairs; ++i) a.turns[i] = std::pow(theta, -2.0 * i / kHeadDim) / (2.0 * M_PI);
  a.q = q;
  a.kp = kp;
  a.vp = vp;
  a.kn = kn;
  a.vn = vn;
  a.bt = bt;
  a.items = items;
  a.bt_stride = bt_stride;
  a.hq = hq;
  a.hkv = hkv;
  hipExtLaunchKernelGGL(rope_append_kernel, dim3(n_items), dim3(256), 0, stream, ev_start, ev_stop, 0, a);
  return hipGetLastError();
}

}  // namespace ppas
