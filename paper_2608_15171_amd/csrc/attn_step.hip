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
//
// Page layouts: K pages are chunk-major, [16 chunks of 8 features][16 slots][8];
// V pages are feature-major, [128 features][16 slots].
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>

#include "plan.h"

namespace ppas {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void global_cvoid;
// The block table is read-only during a launch: reading it through the constant
// address space lets uniform page-id loads use the scalar unit.
typedef __attribute__((address_space(4))) const int32_t const_i32;

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

// The kernel comes in two shapes, by waves per workgroup W: W = 4 (prefill tiles
// of 16 positions, two workgroups per CU) and W = 8 (tiles of 32 positions, one
// workgroup per CU; each staged K/V byte then serves 256 rows). The planner
// picks one per step.
template <int kW>
constexpr int threads_of() { return 64 * kW; }
constexpr int kRegion = 1024;              // one wave's 64 x 16-byte LDS transfer
constexpr int kBlockBytes = 16 * kRegion;  // K (or V) of one 64-key block
constexpr float kNegInf = -__builtin_inff();
constexpr int kPageElems = kPage * kHeadDim;
constexpr int kChunkElems = kPage * 8;     // one 8-feature chunk of a K page

__device__ __forceinline__ u32x4 ldg16(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }
// Streaming load that bypasses cache retention (decode K/V are read exactly once).
__device__ __forceinline__ u32x4 ldg16_nt(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ u32x4 lds16(const char* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// One v_cvt_pk_bf16_f32: two floats to a packed bf16 pair, nearest-even.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// acc + lo + hi of a packed bf16 pair, exactly, in one dot instruction.
__device__ __forceinline__ float sum_bf16x2(uint32_t pr, float acc) {
  const bf16x2 one = {(__bf16)1.f, (__bf16)1.f};
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pr), one, acc, false);
}

// 16 bytes from global memory into LDS: lane L of the wave lands at lds + 16 L.
__device__ __forceinline__ void dma16(const uint16_t* g, char* lds) {
  __builtin_amdgcn_global_load_lds((global_cvoid*)g, (lds_void*)lds, 16, 0, 0);
}

// Wait for this wave's outstanding global loads (including LDS transfers).
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Online-softmax bookkeeping with a lazy maximum: a row's running max m (base-2
// logits) is only raised when the block's max exceeds it by more than kSlack, so
// the accumulator rescale is skipped on almost every block. Probabilities are
// then bounded by 2^kSlack, which fp32 sums and bf16 operands hold exactly as
// well as values <= 1. Exact: every term and the final sum share the same m.
constexpr float kSlack = 8.f;
template <int N, typename Acc>
__device__ __forceinline__ void rescale_if_grown(float block_max, float& m_run, float& l_run, Acc (&acc)[N]) {
  const bool grow = block_max > m_run + kSlack;
  if (__any(grow)) {
    const float m_new = grow ? block_max : m_run;
    const float alpha = grow ? fast_exp2(m_run - m_new) : 1.f;
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int t = 0; t < N; ++t) acc[t] *= alpha;
  }
}

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
// Prefill tile: 4W positions x 8 query heads = 32W rows; wave w owns positions
// 4w..4w+3 (32 rows, one per lane column n = lane & 31; lanes n and n+32 share
// a row). All W waves read the same staged K/V blocks. S^T = K Q^T and O^T += V^T P^T on 32x32x16 MFMAs, so every softmax
// reduction stays inside a lane plus one exchange across the two half-waves.
//
// MFMA row m of a 32-key tile reads key pi(m), which swaps the middle two groups
// of 4 in each 16, so that half-wave h ends up holding keys 16s+8h..16s+8h+7 of
// the P^T operand of k-step s.
//
// LDS holds each 64-key block in MFMA operand order, written straight from
// global memory by 16-byte LDS transfers (16 regions of K and 16 of V per block,
// 16/W of each per wave): K region (t, j) = 8t + j holds, at
// 16 L, lane L's A chunk for key tile t and k-step j (key 32t + pi(L & 31),
// features 16j + 8(L >> 5) .. +7); V region (tt, s) = 4tt + s holds lane L's V^T
// chunk (feature 32tt + (L & 31), keys 16s + 8(L >> 5) .. +7). Every operand
// read is then base + 16 L + constant, free of bank conflicts, and each
// transfer reads whole 32-byte runs of a page.
//
// Pipeline: iteration b issues the transfers of K(b+2) and V(b+1), runs the
// QK^T MFMAs of block b+1 while it exponentiates block b, then the PV MFMAs of
// block b while it reduces the max of block b+1. Blocks wholly below the tile's
// first position need no mask and run the branch-free main loop; the last
// blocks (diagonal, ragged tail) run the general iteration.
// ---------------------------------------------------------------------------
struct PrefillCtx {
  const StepArgs* a;
  const_i32* btrow;
  size_t page_stride;
  int key_lo, kend, last_page;
  int lane, w, n, h, pi_n;
  uint32_t k_lane_off, v_lane_off;   // per-lane element offsets inside a page (head included)
};

struct PageIds {
  int p[4];
};

__device__ __forceinline__ PageIds page_ids(const PrefillCtx& c, int blk) {
  PageIds r;
  const int first = (c.key_lo >> 4) + 4 * blk;
#pragma unroll
  for (int i = 0; i < 4; ++i) r.p[i] = c.btrow[min(first + i, c.last_page)];
  return r;
}

// This wave's K transfers of a block: regions R w .. R w + R-1 (R = 16/W), all in
// key tile t = R w / 8 (pages 2t and 2t+1 of the block), k-steps (R w mod 8) + i.
template <int kW>
__device__ __forceinline__ void dma_k(const PrefillCtx& c, const PageIds& pg, char* kbuf) {
  constexpr int R = 16 / kW;
  const bool t1 = (R * c.w) >> 3;
  const int lo = t1 ? pg.p[2] : pg.p[0];
  const int hi = t1 ? pg.p[3] : pg.p[1];
  const uint16_t* lo_base = c.a->kp + size_t(lo) * c.page_stride;
  const uint16_t* hi_base = c.a->kp + size_t(hi) * c.page_stride;
  const uint16_t* base = ((c.pi_n >> 4) ? hi_base : lo_base) + c.k_lane_off;
#pragma unroll
  for (int i = 0; i < R; ++i) dma16(base + 2 * i * kChunkElems, kbuf + (R * c.w + i) * kRegion);
}

// This wave's V transfers of a block: regions R w .. R w + R-1, all in feature
// tile tt = R w / 4, over pages s = (R w mod 4) + i of the block.
template <int kW>
__device__ __forceinline__ void dma_v(const PrefillCtx& c, const PageIds& pg, char* vbuf) {
  constexpr int R = 16 / kW;
  if constexpr (R == 4) {
#pragma unroll
    for (int s = 0; s < 4; ++s)
      dma16(c.a->vp + size_t(pg.p[s]) * c.page_stride + c.v_lane_off, vbuf + (4 * c.w + s) * kRegion);
  } else {
    static_assert(R == 2, "four or eight waves");
    const int p0 = (c.w & 1) ? pg.p[2] : pg.p[0];
    const int p1 = (c.w & 1) ? pg.p[3] : pg.p[1];
    dma16(c.a->vp + size_t(p0) * c.page_stride + c.v_lane_off, vbuf + (2 * c.w) * kRegion);
    dma16(c.a->vp + size_t(p1) * c.page_stride + c.v_lane_off, vbuf + (2 * c.w + 1) * kRegion);
  }
}

__device__ __forceinline__ void qk_block(const char* kbuf, int lane, const bf16x8 (&qf)[8], f32x16 (&S)[2]) {
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) S[t][r] = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const u32x4 kv = lds16(kbuf + (8 * t + j) * kRegion + 16 * lane);
      S[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kv), qf[j], S[t], 0, 0, 0);
    }
}

__device__ __forceinline__ float block_max(const f32x16 (&S)[2]) {
  float mx = kNegInf;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, S[t][r]);
  return fmaxf(mx, __shfl_xor(mx, 32));
}

// P^T operand of k-step s (keys 16s..16s+15) from tile s/2, registers 8(s%2)..;
// returns the sum of the bf16-rounded probabilities (numerator and denominator
// use the same weights).
__device__ __forceinline__ float probs(const f32x16 (&S)[2], float scale_log2, float m_use, u32x4 (&pk)[4]) {
  float lsum = 0.f;
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float x0 = fast_exp2(S[s >> 1][8 * (s & 1) + 2 * e] * scale_log2 - m_use);
      const float x1 = fast_exp2(S[s >> 1][8 * (s & 1) + 2 * e + 1] * scale_log2 - m_use);
      const uint32_t pr = pack_bf16x2(x0, x1);
      pk[s][e] = pr;
      lsum = sum_bf16x2(pr, lsum);
    }
  return lsum;
}

// O^T += V^T P^T. With the tail limit, keys >= kend contribute zero V (their
// probabilities are already zero; this keeps unwritten slots out of the sum).
template <bool kTail>
__device__ __forceinline__ void pv_block(const char* vbuf, int lane, int h, const u32x4 (&pk)[4], f32x16 (&O)[4],
                                         int kb, int kend) {
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) {   // four independent accumulators in turn
      u32x4 vv = lds16(vbuf + (4 * tt + s) * kRegion + 16 * lane);
      if (kTail) vv = keep_first(vv, 0, kend - (kb + 16 * s + 8 * h));
      O[tt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vv), as_bf16x8(pk[s]), O[tt], 0, 0, 0);
    }
}

template <int kW>
__device__ __forceinline__ void prefill_tile(const StepArgs& a, const WorkItem& it, char* smem) {
  constexpr int R = 16 / kW;   // transfers of K (and of V) per wave per block
  const int tid = threadIdx.x;
  PrefillCtx c;
  c.a = &a;
  c.lane = tid & 63;
  // In the eight-wave shape the wave index is declared wave-uniform, so the page
  // selects and page bases of the LDS transfers stay on the scalar unit (16 % fewer
  // vector instructions in the main loop, ~1 % faster); the four-wave shape measured
  // ~1 % slower that way and keeps the per-lane form.
  c.w = kW == 8 ? int(__builtin_amdgcn_readfirstlane(tid >> 6)) : tid >> 6;
  c.n = c.lane & 31;
  c.h = c.lane >> 5;
  {
    const int grp = (c.n >> 2) & 3;
    const int base = (grp == 0) ? 0 : (grp == 1) ? 8 : (grp == 2) ? 4 : 12;
    c.pi_n = (c.n & 16) | base | (c.n & 3);
  }
  c.btrow = (const_i32*)(a.bt) + size_t(it.seq) * a.bt_stride;
  c.page_stride = size_t(a.hkv) * kPageElems;
  {
    const uint32_t head_off = uint32_t(it.kvh) * kPageElems;
    // K: chunk 2j + h of k-step j = (R w mod 8) + i, slot pi(n) & 15
    c.k_lane_off = head_off + (2 * ((R * c.w) & 7) + c.h) * kChunkElems + (c.pi_n & 15) * 8;
    // V: feature 32 tt + n with tt = R w / 4, slots 8h..8h+7
    c.v_lane_off = head_off + (32 * ((R * c.w) >> 2) + c.n) * kPage + 8 * c.h;
  }
  c.key_lo = it.key_lo;
  c.kend = it.key_hi;
  c.last_page = (it.key_hi - 1) >> 4;

  const int npos = it.npos_kind & 0xffff;
  const int pl = 4 * c.w + (c.n >> 3);
  const int hl = c.n & 7;
  const bool rvalid = pl < npos;
  const int p = it.pos0 + pl;
  const int qhead = it.kvh * kGroup + hl;
  const float sl2 = a.scale_log2;

  // Q^T operand: k-step j covers features 16j..16j+15; this lane holds 8h..8h+7 of them.
  bf16x8 qf[8];
  {
    const uint16_t* qrow = a.q + (size_t(it.row0 + (rvalid ? pl : 0)) * a.hq + qhead) * kHeadDim + 8 * c.h;
#pragma unroll
    for (int j = 0; j < 8; ++j) qf[j] = as_bf16x8(rvalid ? ldg16(qrow + 16 * j) : u32x4{0, 0, 0, 0});
  }

  // K buffers at smem + {0, 1} * kBlockBytes, V buffers after them
  auto kbuf = [&](int i) { return smem + (i & 1) * kBlockBytes; };
  auto vbuf = [&](int i) { return smem + (2 + (i & 1)) * kBlockBytes; };
  const int nblk = (c.kend - c.key_lo + kPrefillBlock - 1) / kPrefillBlock;
  // blocks 0..nfull-1 lie wholly at or below the tile's first position
  const int nfull = min(nblk, (it.pos0 + 1 - c.key_lo) >> 6);

  f32x16 O[4];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) O[t][r] = 0.f;
  float m_run = kNegInf, l_run = 0.f;

  // prologue: K(0), K(1), V(0) in flight; page ids of blocks 1 and 2 kept for the loop
  const PageIds pg0 = page_ids(c, 0);
  PageIds pg1 = page_ids(c, 1), pg2 = page_ids(c, 2);
  dma_k<kW>(c, pg0, kbuf(0));
  dma_k<kW>(c, pg1, kbuf(1));
  dma_v<kW>(c, pg0, vbuf(0));
  wait_vmem();
  __syncthreads();

  f32x16 SA[2], SB[2];
  qk_block(kbuf(0), c.lane, qf, SA);
  if (nfull >= 1) rescale_if_grown(block_max(SA) * sl2, m_run, l_run, O);

  // Main loop: blocks b and b + 1 both unmasked.
  auto main_iter = [&](int b, f32x16 (&Scur)[2], f32x16 (&Snext)[2]) {
    dma_k<kW>(c, pg2, kbuf(b));
    dma_v<kW>(c, pg1, vbuf(b + 1));
    pg1 = pg2;
    pg2 = page_ids(c, b + 3);
    const float m_use = (m_run == kNegInf) ? 0.f : m_run;
    u32x4 pk[4];
    qk_block(kbuf(b + 1), c.lane, qf, Snext);
    l_run += probs(Scur, sl2, m_use, pk);
    pv_block<false>(vbuf(b), c.lane, c.h, pk, O, 0, 0);
    const float mx = block_max(Snext) * sl2;
    wait_vmem();
    __syncthreads();
    rescale_if_grown(mx, m_run, l_run, O);
  };
  int b = 0;
  for (; b + 2 < nfull; b += 2) {
    main_iter(b, SA, SB);
    main_iter(b + 1, SB, SA);
  }
  if (b + 1 < nfull) {
    main_iter(b, SA, SB);
    ++b;
#pragma unroll
    for (int t = 0; t < 2; ++t) SA[t] = SB[t];
  }

  // General iterations: the last unmasked block (its max is already folded in)
  // and the blocks that need the causal mask or the ragged-tail limit.
  for (; b < nblk; ++b) {
    const int kb = c.key_lo + b * kPrefillBlock;
    if (b >= nfull) {
      // key (tile t, reg r) = kb + 32t + 16(r/8) + 8h + r%8, visible iff <= p
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kb + 32 * t + 16 * (r >> 3) + 8 * c.h + (r & 7);
          if (key > p) SA[t][r] = kNegInf;
        }
      rescale_if_grown(block_max(SA) * sl2, m_run, l_run, O);
    }
    if (b + 2 < nblk) dma_k<kW>(c, pg2, kbuf(b));
    if (b + 1 < nblk) dma_v<kW>(c, pg1, vbuf(b + 1));
    pg1 = pg2;
    pg2 = page_ids(c, b + 3);
    const float m_use = (m_run == kNegInf) ? 0.f : m_run;
    u32x4 pk[4];
    if (b + 1 < nblk) qk_block(kbuf(b + 1), c.lane, qf, SB);
    l_run += probs(SA, sl2, m_use, pk);
    if (kb + kPrefillBlock > c.kend)
      pv_block<true>(vbuf(b), c.lane, c.h, pk, O, kb, c.kend);
    else
      pv_block<false>(vbuf(b), c.lane, c.h, pk, O, kb, c.kend);
    wait_vmem();
    __syncthreads();
#pragma unroll
    for (int t = 0; t < 2; ++t) SA[t] = SB[t];
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
        const int d = 32 * t + 8 * g + 4 * c.h;
        u32x2 v;
        v[0] = pack_bf16x2(O[t][4 * g] * inv, O[t][4 * g + 1] * inv);
        v[1] = pack_bf16x2(O[t][4 * g + 2] * inv, O[t][4 * g + 3] * inv);
        *reinterpret_cast<u32x2*>(orow + d) = v;
      }
  } else {
    const int slot = it.part + 32 * c.w + c.n;
    float* acc = a.part_acc + size_t(slot) * kHeadDim;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d = 32 * t + 8 * g + 4 * c.h;
        *reinterpret_cast<f32x4*>(acc + d) = f32x4{O[t][4 * g], O[t][4 * g + 1], O[t][4 * g + 2], O[t][4 * g + 3]};
      }
    if (c.h == 0) a.part_ml[slot] = make_float2(m_run, l_tot);
  }
}

// ---------------------------------------------------------------------------
// Decode item: one query row (8 heads) of one KV head over keys [key_lo, key_hi).
// The W waves take interleaved 32-key blocks and stream K/V from HBM straight
// into 16x16x32 MFMA operands (heads in the N dimension, padded 8 -> 16), then
// merge their running (m, l, acc) through LDS.
// Lane (n = lane & 15, q = lane >> 4): S^T tile t is the block's page t (row m =
// key 16t + m), so one K load reads whole 256-byte chunk runs of a page, and
// after S^T lane q holds keys 4q..4q+3 of each page. The PV product takes its k
// elements in key order (lane q: keys 8q..8q+7), so that lane q's V^T operand
// is the 16 contiguous bytes of feature d holding those keys; the bf16
// probabilities are regrouped into that order through a 1 KB LDS slot of the
// wave. The QK^T reduction runs over features in the order 32q + 8j + i (k-step
// j) for both the Q and K operands, so lane q's K operand is chunks 4q..4q+3 of
// its key.
// ---------------------------------------------------------------------------
template <int kW>
__device__ __forceinline__ void decode_row(const StepArgs& a, const WorkItem& it, char* smem) {
  constexpr int kWaves = kW;
  constexpr int kThreads = threads_of<kW>();
  const int tid = threadIdx.x;
  // the wave index is uniform; saying so keeps per-wave control flow scalar
  const int lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 15, q = lane >> 4;
  const bool hvalid = n < kGroup;

  bf16x8 qf[4];
  {
    const uint16_t* qrow = a.q + (size_t(it.row0) * a.hq + it.kvh * kGroup + (hvalid ? n : 0)) * kHeadDim + 32 * q;
#pragma unroll
    for (int j = 0; j < 4; ++j) qf[j] = as_bf16x8(hvalid ? ldg16(qrow + 8 * j) : u32x4{0, 0, 0, 0});
  }

  const int32_t* btrow = a.bt + size_t(it.seq) * a.bt_stride;
  const size_t head_off = size_t(it.kvh) * kPageElems;
  const size_t page_stride = size_t(a.hkv) * kPageElems;
  const int kend = it.key_hi;
  const int nblk = (kend - it.key_lo + kDecodeBlock - 1) / kDecodeBlock;
  const int nmine = nblk > w ? (nblk - w + kWaves - 1) / kWaves : 0;   // blocks w, w+W, ... of this wave

  // Page ids. Item key ranges start on 32-key boundaries, so block b covers
  // pages first + 2b and first + 2b + 1. This wave's i-th block is b = w + Wi;
  // lane L of page-id register r holds page 2(w + W(32r + L/2)) + (L & 1), so one
  // register serves 32 blocks and the ids of a block come out with two lane
  // reads, with no load on the loop's critical path. Ids past the item's last
  // page are clamped to it, so every block's loads stay inside the item's pages.
  const int first_page = it.key_lo >> 4;
  const int last_page = (kend - 1) >> 4;
  constexpr int kPidRegs = kDecodeMaxKeys / (kWaves * 32 * kDecodeBlock);
  static_assert(kPidRegs * kWaves * 32 * kDecodeBlock == kDecodeMaxKeys, "whole page-id registers");
  int pid[kPidRegs];
#pragma unroll
  for (int r = 0; r < kPidRegs; ++r) {
    const int blk = w + kWaves * (32 * r + (lane >> 1));
    pid[r] = btrow[min(first_page + 2 * blk + (lane & 1), last_page)];
  }
  // Complete the page-id loads here, once (the Q loads stay in flight), so the
  // loop never waits on them.
#pragma unroll
  for (int r = 0; r < kPidRegs; ++r) asm volatile("" ::"v"(pid[r]));

  // One 32-key block of this lane's MFMA operands: K rows for the two S^T tiles
  // and V^T chunks for the eight feature tiles. Two sets alternate so that the
  // next block's loads are in flight while the current one is consumed.
  struct Blk {
    u32x4 k[2][4];
    u32x4 v[8];
  };
  // K: chunk 4q + j, slot n of page t; V: feature 16tt + n, slots 8(q & 1)..+7 of page q >> 1
  const uint32_t k_lane = uint32_t(head_off) + 4 * q * kChunkElems + 8 * n;
  const uint32_t v_lane = uint32_t(head_off) + n * kPage + 8 * (q & 1);
  // Every load() issues exactly the same 16 loads, with no branch around
  // any of them (a ragged last block reads clamped pages and is masked where it
  // is consumed). The count of loads in flight is then the same on every path
  // into consume(), so each of its waits lets the next block's loads stay
  // outstanding.
  auto load = [&](Blk& B, int i) {
    // lane reads from every register, then a scalar choice (a register chosen by
    // a runtime index would be moved to memory)
    const int r = i >> 5, l0 = 2 * (i & 31);
    int p0 = __builtin_amdgcn_readlane(pid[0], l0);
    int p1 = __builtin_amdgcn_readlane(pid[0], l0 + 1);
#pragma unroll
    for (int k = 1; k < kPidRegs; ++k) {
      const int c0 = __builtin_amdgcn_readlane(pid[k], l0);
      const int c1 = __builtin_amdgcn_readlane(pid[k], l0 + 1);
      p0 = (r == k) ? c0 : p0;
      p1 = (r == k) ? c1 : p1;
    }
    const uint16_t* k0 = a.kp + size_t(p0) * page_stride + k_lane;
    const uint16_t* k1 = a.kp + size_t(p1) * page_stride + k_lane;
    const uint16_t* vb = a.vp + size_t(q >= 2 ? p1 : p0) * page_stride + v_lane;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      B.k[0][j] = ldg16_nt(k0 + j * kChunkElems);
      B.k[1][j] = ldg16_nt(k1 + j * kChunkElems);
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) B.v[t] = ldg16_nt(vb + 16 * t * kPage);
  };

  f32x4 oacc[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) oacc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = kNegInf, l_run = 0.f;
  // this wave's probability-regrouping slot, past the region the final merge uses
  char* pslot = smem + 3 * kBlockBytes + w * 1024;
  static_assert(kWaves * 1024 <= kBlockBytes, "regrouping slots fit in the last ring block");

  // Block at keys kb..kb+31. In a ragged last block, keys >= kend get logit
  // -inf and zero V, whatever their (clamped) pages hold.
  auto consume = [&](const Blk& B, int kb) {
    const bool tail = kb + kDecodeBlock > kend;
    f32x4 sacc[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      sacc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < 4; ++j)
        sacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(B.k[t][j]), qf[j], sacc[t], 0, 0, 0);
    }
    // S^T register r of tile t: key kb + 16t + 4q + r
    if (tail) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (kb + 16 * t + 4 * q + r >= kend) sacc[t][r] = kNegInf;
    }
    float mx = kNegInf;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) mx = fmaxf(mx, sacc[t][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    rescale_if_grown(mx * a.scale_log2, m_run, l_run, oacc);
    const float m_use = (m_run == kNegInf) ? 0.f : m_run;
    u32x4 pb;
    float lsum = 0.f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const uint32_t pr = pack_bf16x2(fast_exp2(sacc[t][2 * e] * a.scale_log2 - m_use),
                                        fast_exp2(sacc[t][2 * e + 1] * a.scale_log2 - m_use));
        pb[2 * t + e] = pr;
        lsum = sum_bf16x2(pr, lsum);
      }
    l_run += lsum;
    // Regroup: the 8 bytes of (page t, keys 4q..4q+3) go to slot (n, t, q); lane q
    // then reads keys 8q..8q+7 = (page q >> 1, quads 2(q & 1), 2(q & 1) + 1) as one
    // 16-byte run.
    *reinterpret_cast<u32x2*>(pslot + ((2 * n) * 4 + q) * 8) = u32x2{pb[0], pb[1]};
    *reinterpret_cast<u32x2*>(pslot + ((2 * n + 1) * 4 + q) * 8) = u32x2{pb[2], pb[3]};
    pb = lds16(pslot + ((2 * n + (q >> 1)) * 4 + 2 * (q & 1)) * 8);
    // V^T chunk: keys kb + 8q .. +7
    const int vlim = kend - (kb + 8 * q);
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const u32x4 vv = tail ? keep_first(B.v[t], 0, vlim) : B.v[t];
      oacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vv), as_bf16x8(pb), oacc[t], 0, 0, 0);
    }
  };

  // wave w takes blocks w, w+W, w+2W, ... (wave-block i = block w + W i). The
  // block after the last one is loaded as a (clamped, unused) copy of the last,
  // so the loop body always issues its loads.
  if (nmine > 0) {
    Blk A, B;
    const int last = nmine - 1;
    auto kb_of = [&](int i) { return it.key_lo + (w + kWaves * i) * kDecodeBlock; };
    // the scheduling barriers keep each block's loads ahead of the previous
    // block's arithmetic, so two blocks are in flight while one is consumed
    load(A, 0);
    for (int i = 0;; i += 2) {
      load(B, min(i + 1, last));
      __builtin_amdgcn_sched_barrier(0);
      consume(A, kb_of(i));
      if (i + 1 > last) break;
      load(A, min(i + 2, last));
      __builtin_amdgcn_sched_barrier(0);
      consume(B, kb_of(i + 1));
      if (i + 2 > last) break;
    }
    wait_vmem();
  }

  // Merge the waves. O^T register r of feature tile t holds feature 16t + 4q + r.
  float l_w = l_run + __shfl_xor(l_run, 16);
  l_w += __shfl_xor(l_w, 32);
  float* wo = reinterpret_cast<float*>(smem);                 // [W][8][128]
  float* wm = wo + kWaves * kGroup * kHeadDim;                 // [W][8]
  float* wl = wm + kWaves * kGroup;                            // [W][8]
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
  // thread t finishes head t / (kThreads/8), kF consecutive features
  constexpr int kTPH = kThreads / kGroup;   // threads per head
  constexpr int kF = kHeadDim / kTPH;       // features per thread: 4 or 2
  const int head = tid / kTPH;
  const int d0 = (tid % kTPH) * kF;
  float M = kNegInf;
#pragma unroll
  for (int v = 0; v < kWaves; ++v) M = fmaxf(M, wm[v * kGroup + head]);
  const float M_use = (M == kNegInf) ? 0.f : M;
  float L = 0.f;
  float acc[kF] = {};
#pragma unroll
  for (int v = 0; v < kWaves; ++v) {
    const float f = fast_exp2(wm[v * kGroup + head] - M_use);
    L += f * wl[v * kGroup + head];
    const float* src = wo + (v * kGroup + head) * kHeadDim + d0;
#pragma unroll
    for (int e = 0; e < kF; ++e) acc[e] += f * src[e];
  }
  if (it.part < 0) {
    const float inv = 1.f / L;
    uint16_t* orow = a.out + (size_t(it.row0) * a.hq + it.kvh * kGroup + head) * kHeadDim + d0;
#pragma unroll
    for (int e = 0; e < kF; e += 2)
      *reinterpret_cast<uint32_t*>(orow + e) = pack_bf16x2(acc[e] * inv, acc[e + 1] * inv);
  } else {
    const int slot = it.part + head;
    float* dst = a.part_acc + size_t(slot) * kHeadDim + d0;
#pragma unroll
    for (int e = 0; e < kF; ++e) dst[e] = acc[e];
    if ((tid % kTPH) == 0) a.part_ml[slot] = make_float2(M, L);
  }
}

template <int kW>
__global__ __launch_bounds__(threads_of<kW>(), kW == 4 ? 2 : 1) void attn_step_kernel(StepArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem[4 * kBlockBytes];
  const WorkItem it = a.items[blockIdx.x];
  if ((it.npos_kind >> 16) == kKindDecode)
    decode_row<kW>(a, it, smem);
  else
    prefill_tile<kW>(a, it, smem);
}

// Merge split partials: for local row r of a combine item with partials
// (m_s, l_s, acc_s), M = max m_s, out = sum 2^(m_s-M) acc_s / sum 2^(m_s-M) l_s.
// Block (item, y) handles rows 8y..8y+7 of the item; 32 lanes per row, 4
// features per lane.
constexpr int kCombineRowsPerBlock = 8;
constexpr int kMergeBatch = 4;            // splits whose loads a merge thread issues together
constexpr int kCombineThreads = 32 * kCombineRowsPerBlock;
__global__ __launch_bounds__(kCombineThreads) void combine_kernel(const CombineItem* items, const float2* part_ml,
                                                           const float* part_acc, uint16_t* out, int hq) {
  const CombineItem ci = items[blockIdx.x];
  const int rows = ci.npos * kGroup;
  const int r = blockIdx.y * kCombineRowsPerBlock + (threadIdx.x >> 5);
  if (r >= rows) return;
  const int d0 = (threadIdx.x & 31) * 4;
  // Splits are merged in batches of kMergeBatch whose (m, l) and accumulator loads
  // are all issued before any is used (one memory round trip per batch); a later
  // batch rescales what is merged so far to its larger maximum. Absent splits of a
  // batch enter with m = -inf and weigh 0. Every split gives each of its rows at
  // least one key, so a real split's m is finite.
  float M = kNegInf, L = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < ci.nsplit; s0 += kMergeBatch) {
    float2 ml[kMergeBatch];
    f32x4 pa[kMergeBatch];
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i) {
      const int slot = ci.part + min(s0 + i, ci.nsplit - 1) * rows + r;
      ml[i] = part_ml[slot];
      pa[i] = *reinterpret_cast<const f32x4*>(part_acc + size_t(slot) * kHeadDim + d0);
      if (s0 + i >= ci.nsplit) ml[i].x = kNegInf;
    }
    float Mb = M;
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i) Mb = fmaxf(Mb, ml[i].x);
    const float sc = fast_exp2(M - Mb);      // 0 while nothing is merged (M = -inf)
    L *= sc;
    acc *= sc;
#pragma unroll
    for (int i = 0; i < kMergeBatch; ++i) {
      const float f = fast_exp2(ml[i].x - Mb);
      L += f * ml[i].y;
      acc += f * pa[i];
    }
    M = Mb;
  }
  const float inv = 1.f / L;
  uint16_t* orow = out + (size_t(ci.row0 + r / kGroup) * hq + ci.kvh * kGroup + r % kGroup) * kHeadDim + d0;
  u32x2 v;
  v[0] = pack_bf16x2(acc[0] * inv, acc[1] * inv);
  v[1] = pack_bf16x2(acc[2] * inv, acc[3] * inv);
  *reinterpret_cast<u32x2*>(orow) = v;
}

hipError_t launch_attn_step(const uint16_t* q, uint16_t* out, const uint16_t* kp, const uint16_t* vp,
                            const int32_t* bt, int32_t bt_stride, int32_t hq, int32_t hkv, float scale,
                            const WorkItem* items, int n_items, const CombineItem* comb, int n_comb,
                            float2* part_ml, float* part_acc, int tile_pos, hipStream_t stream,
                            hipEvent_t ev_start, hipEvent_t ev_stop, hipEvent_t ev_merge_start,
                            hipEvent_t ev_merge_stop) {
  if (tile_pos != kTilePosSmall && tile_pos != kTilePosLarge) return hipErrorInvalidValue;
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
    // With profiling events, the launch itself records them at the dispatch's
    // start and end (events recorded as separate commands would also time the
    // gap between those commands and the dispatch).
    if (tile_pos == kTilePosLarge)
      hipExtLaunchKernelGGL(attn_step_kernel<8>, dim3(n_items), dim3(threads_of<8>()), 0, stream, ev_start, ev_stop,
                            0, a);
    else
      hipExtLaunchKernelGGL(attn_step_kernel<4>, dim3(n_items), dim3(threads_of<4>()), 0, stream, ev_start, ev_stop,
                            0, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (n_comb > 0) {
    const int ymax = tile_pos * kGroup / kCombineRowsPerBlock;
    hipExtLaunchKernelGGL(combine_kernel, dim3(n_comb, ymax), dim3(kCombineThreads), 0, stream, ev_merge_start,
                          ev_merge_stop, 0, comb, part_ml, part_acc, out, hq);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace ppas
