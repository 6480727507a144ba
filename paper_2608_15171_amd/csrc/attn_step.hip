// Packed mixed-step attention for gfx950 (CDNA4): one launch whose workgroups
// are either prefill tiles (MFMA bf16, K/V pages staged in LDS, the 8 query
// heads of a KV head packed into the tile's rows) or split-K decode items (K/V
// streamed from HBM straight into MFMA operands), followed by a small launch
// that merges rows whose keys were split across workgroups.
//
// Math per row (position p) and query head: softmax over keys 0..p of
// scale * q.k, applied to V; computed online over key blocks in the base-2
// domain (running max m, running sum l, unnormalised accumulator), fp32
// accumulation, probabilities rounded to bf16 for the PV product.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "plan.h"

namespace ppas {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

struct StepArgs {
  const uint16_t* q;
  uint16_t* out;
  const uint16_t* kp;
  const uint16_t* vp;
  const int32_t* bt;
  const WorkItem* items;
  float2* part_ml;
  float* part_acc;
  int32_t bt_stride;
  int32_t hq, hkv;
  float scale_log2;     // softmax scale * log2(e)
};

constexpr int kThreads = 256;
constexpr int kStageBytes = 32768;   // one 64-key block: 16 KB of K + 16 KB of V
constexpr float kNegInf = -__builtin_inff();

__device__ __forceinline__ u32x4 ldg16(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return uint32_t(__builtin_bit_cast(uint16_t, (__bf16)a)) |
         (uint32_t(__builtin_bit_cast(uint16_t, (__bf16)b)) << 16);
}

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __builtin_bit_cast(float, u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __builtin_bit_cast(float, u & 0xffff0000u); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Zero the bf16 elements of an 8-element chunk whose index (first + e) is >= lim.
__device__ __forceinline__ u32x4 keep_first(u32x4 v, int first, int lim) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t m = 0;
    if (first + 2 * w < lim) m |= 0x0000ffffu;
    if (first + 2 * w + 1 < lim) m |= 0xffff0000u;
    v[w] &= m;
  }
  return v;
}

// ---------------------------------------------------------------------------
// Prefill tile: 16 positions x 8 query heads = 128 rows; wave w owns positions
// 4w..4w+3 (32 rows, one per lane column n = lane & 31; lanes n and n+32 share
// a row). S^T = K Q^T and O^T += V^T P^T on 32x32x16 MFMAs, so every softmax
// reduction stays inside a lane plus one exchange across the two half-waves.
//
// LDS per stage: K block [64 keys][128 d] with the 16-byte chunk index of key k
// XOR-ed by (k & 15); V block [4 pages][128 d][16 keys] with the 16-byte half of
// feature row d XOR-ed by bit 2 ^ bit 3 of d. Both keep MFMA operand reads free
// of bank conflicts.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void prefill_tile(const StepArgs& a, const WorkItem& it, char* smem) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  const int npos = it.npos_kind & 0xffff;
  const int pl = 4 * w + (n >> 3);
  const int hl = n & 7;
  const bool rvalid = pl < npos;
  const int p = it.pos0 + pl;
  const int qhead = it.kvh * kGroup + hl;

  // Q^T operand: k-step j covers features 16j..16j+15; this lane holds 8h..8h+7 of them.
  bf16x8 qf[8];
  {
    const uint16_t* qrow = a.q + (size_t(it.row0 + (rvalid ? pl : 0)) * a.hq + qhead) * kHeadDim + 8 * h;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      u32x4 v = rvalid ? ldg16(qrow + 16 * j) : u32x4{0, 0, 0, 0};
      qf[j] = as_bf16x8(v);
    }
  }

  // MFMA row m of a 32-key tile reads key pi(m): swaps the middle two groups of 4
  // in each 16 so that half-wave h ends up holding keys 16s+8h..16s+8h+7 of P^T.
  int key_of_row[2];
  {
    const int grp = (n >> 2) & 3;
    const int base = (grp == 0) ? 0 : (grp == 1) ? 8 : (grp == 2) ? 4 : 12;
    const int km = (n & 16) | base | (n & 3);
    key_of_row[0] = km;
    key_of_row[1] = 32 + km;
  }

  const int32_t* btrow = a.bt + size_t(it.seq) * a.bt_stride;
  const size_t head_off = size_t(it.kvh) * kPage * kHeadDim;
  const size_t page_stride = size_t(a.hkv) * kPage * kHeadDim;
  const int kend = it.key_hi;
  const int nblk = (kend - it.key_lo + kPrefillBlock - 1) / kPrefillBlock;

  u32x4 sk[4], sv[4];
  auto gload = [&](int kb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key0 = kb + 16 * i;
      if (key0 < kend) {
        const size_t pg = size_t(btrow[key0 >> 4]) * page_stride + head_off;
        sk[i] = ldg16(a.kp + pg + tid * 8);
        sv[i] = ldg16(a.vp + pg + tid * 8);
        const int lim = kend - key0;          // valid slots of this page
        if (lim < 16) {
          if ((tid >> 4) >= lim) sk[i] = u32x4{0, 0, 0, 0};
          sv[i] = keep_first(sv[i], 8 * (tid & 1), lim);
        }
      } else {
        sk[i] = u32x4{0, 0, 0, 0};
        sv[i] = u32x4{0, 0, 0, 0};
      }
    }
  };
  auto swrite = [&](char* buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = 16 * i + (tid >> 4);
      *reinterpret_cast<u32x4*>(buf + key * 256 + (((tid & 15) ^ (key & 15)) << 4)) = sk[i];
      const int d = tid >> 1;
      const int sw = ((d >> 2) ^ (d >> 3)) & 1;
      *reinterpret_cast<u32x4*>(buf + 16384 + i * 4096 + d * 32 + (((tid & 1) ^ sw) << 4)) = sv[i];
    }
  };

  f32x16 oacc[4];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[t][r] = 0.f;
  float m_run = kNegInf, l_run = 0.f;

  const int wave_pmin = it.pos0 + 4 * w;
  const int wave_pmax = it.pos0 + min(4 * w + 3, npos - 1);

  gload(it.key_lo);
  swrite(smem);
  __syncthreads();

  for (int b = 0; b < nblk; ++b) {
    char* cur = smem + (b & 1) * kStageBytes;
    const int kb = it.key_lo + b * kPrefillBlock;
    const bool has_next = b + 1 < nblk;
    if (has_next) gload(kb + kPrefillBlock);

    if (kb <= wave_pmax) {
      // S^T = K Q^T: two 32-key tiles, 8 k-steps over the 128 features
      f32x16 sacc[2];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[t][r] = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const int key = key_of_row[t];
          const u32x4 kv = *reinterpret_cast<const u32x4*>(cur + key * 256 + (((2 * j + h) ^ (key & 15)) << 4));
          sacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kv), qf[j], sacc[t], 0, 0, 0);
        }
      }
      // causal mask: key (tile t, reg r) = kb + 32t + 16(r/8) + 8h + r%8, visible iff <= p
      if (kb + kPrefillBlock - 1 > wave_pmin) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = kb + 32 * t + 16 * (r >> 3) + 8 * h + (r & 7);
            if (key > p) sacc[t][r] = kNegInf;
          }
      }
      float mx = kNegInf;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[t][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx * a.scale_log2);
      const float m_use = (m_new == kNegInf) ? 0.f : m_new;
      const float alpha = fast_exp2(m_run - m_use);
      m_run = m_new;

      // P^T operand for k-step s (keys 16s..16s+15): tile s/2, registers 8(s%2)..8(s%2)+7
      u32x4 pk[4];
      float lsum = 0.f;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float x0 = fast_exp2(sacc[s >> 1][8 * (s & 1) + 2 * e] * a.scale_log2 - m_use);
          const float x1 = fast_exp2(sacc[s >> 1][8 * (s & 1) + 2 * e + 1] * a.scale_log2 - m_use);
          const uint32_t pr = pack_bf16x2(x0, x1);
          pk[s][e] = pr;
          lsum += bf16_lo(pr) + bf16_hi(pr);
        }
      }
      l_run = l_run * alpha + lsum;
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[t][r] *= alpha;

      // O^T += V^T P^T: 4 feature tiles of 32, 4 k-steps of 16 keys (one page each)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int d = 32 * t + n;
        const int sw = ((d >> 2) ^ (d >> 3)) & 1;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const u32x4 vv = *reinterpret_cast<const u32x4*>(cur + 16384 + s * 4096 + d * 32 + ((h ^ sw) << 4));
          oacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vv), as_bf16x8(pk[s]), oacc[t], 0, 0, 0);
        }
      }
    }

    if (has_next) swrite(smem + ((b + 1) & 1) * kStageBytes);
    __syncthreads();
  }

  // Epilogue. O^T register r of feature tile t holds feature 32t + 8(r/4) + 4h + r%4.
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!rvalid) return;
  if (it.part < 0) {
    const float inv = 1.f / l_tot;
    uint16_t* orow = a.out + (size_t(it.row0 + pl) * a.hq + qhead) * kHeadDim;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d = 32 * t + 8 * g + 4 * h;
        u32x2 v;
        v[0] = pack_bf16x2(oacc[t][4 * g] * inv, oacc[t][4 * g + 1] * inv);
        v[1] = pack_bf16x2(oacc[t][4 * g + 2] * inv, oacc[t][4 * g + 3] * inv);
        *reinterpret_cast<u32x2*>(orow + d) = v;
      }
  } else {
    const int slot = it.part + 32 * w + n;
    float* acc = a.part_acc + size_t(slot) * kHeadDim;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d = 32 * t + 8 * g + 4 * h;
        *reinterpret_cast<f32x4*>(acc + d) =
            f32x4{oacc[t][4 * g], oacc[t][4 * g + 1], oacc[t][4 * g + 2], oacc[t][4 * g + 3]};
      }
    if (h == 0) a.part_ml[slot] = make_float2(m_run, l_tot);
  }
}

// ---------------------------------------------------------------------------
// Decode item: one query row (8 heads) of one KV head over keys [key_lo, key_hi).
// The four waves take interleaved 32-key blocks and stream K/V from HBM straight
// into 16x16x32 MFMA operands (heads in the N dimension, padded 8 -> 16), then
// merge their running (m, l, acc) through LDS.
// Lane (n = lane & 15, q = lane >> 4): K rows of tile t are keys 8*(m/4) + 4t + m%4,
// so after S^T lane q holds keys 8q..8q+7 of the block, which is exactly the k
// range of its P^T operand slot; its V^T operand is the 16 contiguous bytes of
// feature d holding keys 8q..8q+7.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void decode_row(const StepArgs& a, const WorkItem& it, char* smem) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int n = lane & 15, q = lane >> 4;
  const bool hvalid = n < kGroup;

  // Q^T operand: k-step j holds features 32q + 8j .. 32q + 8j + 7 (the same
  // feature permutation is used for the K operand).
  bf16x8 qf[4];
  {
    const uint16_t* qrow = a.q + (size_t(it.row0) * a.hq + it.kvh * kGroup + (hvalid ? n : 0)) * kHeadDim + 32 * q;
#pragma unroll
    for (int j = 0; j < 4; ++j) qf[j] = as_bf16x8(hvalid ? ldg16(qrow + 8 * j) : u32x4{0, 0, 0, 0});
  }

  const int32_t* btrow = a.bt + size_t(it.seq) * a.bt_stride;
  const size_t head_off = size_t(it.kvh) * kPage * kHeadDim;
  const size_t page_stride = size_t(a.hkv) * kPage * kHeadDim;
  const int kend = it.key_hi;
  const int nblk = (kend - it.key_lo + kDecodeBlock - 1) / kDecodeBlock;

  const int krow = 8 * (n >> 2) + (n & 3);   // + 4t for tile t

  u32x4 kr[2][4], vr[8];
  auto gload = [&](int kb) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int key = kb + krow + 4 * t;
      if (key < kend) {
        const uint16_t* src = a.kp + size_t(btrow[key >> 4]) * page_stride + head_off + (key & 15) * kHeadDim + 32 * q;
#pragma unroll
        for (int j = 0; j < 4; ++j) kr[t][j] = ldg16(src + 8 * j);
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) kr[t][j] = u32x4{0, 0, 0, 0};
      }
    }
    const int key0 = kb + 8 * q;
    if (key0 < kend) {
      const uint16_t* src = a.vp + size_t(btrow[key0 >> 4]) * page_stride + head_off + (key0 & 15) + n * kPage;
      const int lim = kend - key0;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        vr[t] = ldg16(src + 16 * t * kPage);
        if (lim < 8) vr[t] = keep_first(vr[t], 0, lim);
      }
    } else {
#pragma unroll
      for (int t = 0; t < 8; ++t) vr[t] = u32x4{0, 0, 0, 0};
    }
  };

  f32x4 oacc[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) oacc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = kNegInf, l_run = 0.f;

  int b = w;
  if (b < nblk) gload(it.key_lo + b * kDecodeBlock);
  for (; b < nblk; b += 4) {
    const int kb = it.key_lo + b * kDecodeBlock;
    u32x4 kc[2][4], vc[8];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int j = 0; j < 4; ++j) kc[t][j] = kr[t][j];
#pragma unroll
    for (int t = 0; t < 8; ++t) vc[t] = vr[t];
    if (b + 4 < nblk) gload(kb + 4 * kDecodeBlock);

    f32x4 sacc[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      sacc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < 4; ++j)
        sacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kc[t][j]), qf[j], sacc[t], 0, 0, 0);
    }
    // S^T register r of tile t: key kb + 8q + 4t + r
    if (kb + kDecodeBlock > kend) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (kb + 8 * q + 4 * t + r >= kend) sacc[t][r] = kNegInf;
    }
    float mx = kNegInf;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) mx = fmaxf(mx, sacc[t][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx * a.scale_log2);
    const float m_use = (m_new == kNegInf) ? 0.f : m_new;
    const float alpha = fast_exp2(m_run - m_use);
    m_run = m_new;
    u32x4 pb;
    float lsum = 0.f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const uint32_t pr = pack_bf16x2(fast_exp2(sacc[t][2 * e] * a.scale_log2 - m_use),
                                        fast_exp2(sacc[t][2 * e + 1] * a.scale_log2 - m_use));
        pb[2 * t + e] = pr;
        lsum += bf16_lo(pr) + bf16_hi(pr);
      }
    l_run = l_run * alpha + lsum;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      oacc[t] *= alpha;
      oacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vc[t]), as_bf16x8(pb), oacc[t], 0, 0, 0);
    }
  }

  // Merge the four waves. O^T register r of feature tile t holds feature 16t + 4q + r.
  float l_w = l_run + __shfl_xor(l_run, 16);
  l_w += __shfl_xor(l_w, 32);
  float* wo = reinterpret_cast<float*>(smem);                 // [4][8][128]
  float* wm = wo + 4 * kGroup * kHeadDim;                      // [4][8]
  float* wl = wm + 4 * kGroup;                                 // [4][8]
  if (hvalid) {
#pragma unroll
    for (int t = 0; t < 8; ++t)
      *reinterpret_cast<f32x4*>(wo + (w * kGroup + n) * kHeadDim + 16 * t + 4 * q) = oacc[t];
    if (q == 0) {
      wm[w * kGroup + n] = m_run;
      wl[w * kGroup + n] = l_w;
    }
  }
  __syncthreads();
  const int head = tid >> 5;            // 0..7
  const int d0 = (tid & 31) * 4;
  float M = kNegInf;
#pragma unroll
  for (int v = 0; v < 4; ++v) M = fmaxf(M, wm[v * kGroup + head]);
  const float M_use = (M == kNegInf) ? 0.f : M;
  float L = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const float f = fast_exp2(wm[v * kGroup + head] - M_use);
    L += f * wl[v * kGroup + head];
    acc += f * *reinterpret_cast<const f32x4*>(wo + (v * kGroup + head) * kHeadDim + d0);
  }
  if (it.part < 0) {
    const float inv = 1.f / L;
    uint16_t* orow = a.out + (size_t(it.row0) * a.hq + it.kvh * kGroup + head) * kHeadDim + d0;
    u32x2 v;
    v[0] = pack_bf16x2(acc[0] * inv, acc[1] * inv);
    v[1] = pack_bf16x2(acc[2] * inv, acc[3] * inv);
    *reinterpret_cast<u32x2*>(orow) = v;
  } else {
    const int slot = it.part + head;
    *reinterpret_cast<f32x4*>(a.part_acc + size_t(slot) * kHeadDim + d0) = acc;
    if ((tid & 31) == 0) a.part_ml[slot] = make_float2(M, L);
  }
}

__global__ __launch_bounds__(kThreads, 2) void attn_step_kernel(StepArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[2 * kStageBytes];
  const WorkItem it = a.items[blockIdx.x];
  if ((it.npos_kind >> 16) == kKindDecode)
    decode_row(a, it, smem);
  else
    prefill_tile(a, it, smem);
}

// Merge split partials: for local row r of a combine item with partials
// (m_s, l_s, acc_s), M = max m_s, out = sum 2^(m_s-M) acc_s / sum 2^(m_s-M) l_s.
// One wave per row, two features per lane.
__global__ __launch_bounds__(kThreads) void combine_kernel(const CombineItem* items, const float2* part_ml,
                                                           const float* part_acc, uint16_t* out, int hq) {
  const CombineItem ci = items[blockIdx.x];
  const int rows = ci.npos * kGroup;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int r = w; r < rows; r += kThreads / 64) {
    float M = kNegInf;
    for (int s = 0; s < ci.nsplit; ++s) M = fmaxf(M, part_ml[ci.part + s * rows + r].x);
    const float M_use = (M == kNegInf) ? 0.f : M;
    float L = 0.f, x0 = 0.f, x1 = 0.f;
    for (int s = 0; s < ci.nsplit; ++s) {
      const int slot = ci.part + s * rows + r;
      const float2 ml = part_ml[slot];
      const float f = fast_exp2(ml.x - M_use);
      L += f * ml.y;
      const float2 v = *reinterpret_cast<const float2*>(part_acc + size_t(slot) * kHeadDim + 2 * lane);
      x0 += f * v.x;
      x1 += f * v.y;
    }
    const float inv = 1.f / L;
    uint16_t* orow = out + (size_t(ci.row0 + r / kGroup) * hq + ci.kvh * kGroup + r % kGroup) * kHeadDim;
    *reinterpret_cast<uint32_t*>(orow + 2 * lane) = pack_bf16x2(x0 * inv, x1 * inv);
  }
}

hipError_t launch_attn_step(const uint16_t* q, uint16_t* out, const uint16_t* kp, const uint16_t* vp,
                            const int32_t* bt, int32_t bt_stride, int32_t hq, int32_t hkv, float scale,
                            const WorkItem* items, int n_items, const CombineItem* comb, int n_comb,
                            float2* part_ml, float* part_acc, hipStream_t stream,
                            hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (n_items > 0) {
    StepArgs a;
    a.q = q;
    a.out = out;
    a.kp = kp;
    a.vp = vp;
    a.bt = bt;
    a.items = items;
    a.part_ml = part_ml;
    a.part_acc = part_acc;
    a.bt_stride = bt_stride;
    a.hq = hq;
    a.hkv = hkv;
    a.scale_log2 = scale * 1.4426950408889634f;
    if (ev_start && hipEventRecord(ev_start, stream) != hipSuccess) return hipGetLastError();
    hipLaunchKernelGGL(attn_step_kernel, dim3(n_items), dim3(kThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (ev_stop && hipEventRecord(ev_stop, stream) != hipSuccess) return hipGetLastError();
  }
  if (n_comb > 0) {
    hipLaunchKernelGGL(combine_kernel, dim3(n_comb), dim3(kThreads), 0, stream, comb, part_ml, part_acc, out, hq);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace ppas
