// Fused gate-up projection of a decoder block's MLP on gfx950 (CDNA4):
//   Y[T][N2] = X[T][H] * W[N2][H]^T
// bf16 inputs, fp32 accumulation on 32x32x16 MFMAs, output rounded to bf16
// (nearest even). W stacks the gate rows over the up rows, so one launch
// computes both projections of a prefill chunk.
//
// Tiling. A workgroup of eight waves (two per SIMD) computes a 256 x 256
// output tile; wave (wn, wm) owns 128 output columns x 64 token rows as 4 x 2
// MFMA tiles (128 fp32 accumulators per lane), so that while one wave of a SIMD
// waits (its transfers' issue, an LDS read) the other keeps the matrix core
// busy. (Four waves of 128 x 128, one per SIMD with 256 accumulators each,
// read half as many LDS bytes per MFMA but measured 5 % slower.) The reduction
// advances 64 features per stage: a stage's W rows and X rows (32 KB each) are
// copied into LDS by 16-byte global-to-LDS transfers, each covering eight whole
// 128-byte row runs (one cache line per row), into a two-slot ring. In LDS a
// row keeps its eight 16-byte chunks in an XOR-swizzled order, so each operand
// fragment read (row tile, k-step: 32 rows x 32 bytes) is one bank-conflict-free
// ds_read_b128. The next stage's transfers are issued in the first two of the
// stage's four k-steps, and the next k-step's fragments are read in two groups
// while the current k-step's MFMAs run. (Transfers of 32-byte row pieces
// straight into operand order, and rings of four or five 32-feature stages,
// measured 33 %, 6-13 % and 2-12 % slower; transfers spread over all four
// k-steps 4-7 % slower, issued in one k-step 2-8 % slower, or interleaved one by
// one with the MFMAs no faster.)
//
// The MFMA's first operand is W (rows = output columns), its second X (rows =
// tokens): lane L of a 32 x 32 result then holds token row L % 32 and, in
// registers 4g..4g+3, four consecutive output columns 8g + 4(L / 32) + 0..3,
// which the epilogue packs into 8-byte LDS writes; the wave's block then leaves
// LDS as 256-byte row runs of 16-byte stores, eight LDS reads ahead of their
// stores.
//
// Tile order. The grid holds one workgroup per compute unit, each looping over
// its tiles. Workgroup b runs on XCD b % 8; each XCD takes a contiguous range
// of tiles, and tiles are numbered in groups of 8 token-row tiles that share a
// weight tile, so the workgroups resident on one XCD share operand tiles in
// that XCD's L2.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>
#include <cstddef>
#include <cstdint>

namespace ppas {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void global_cvoid;

#ifndef PPAS_GATEUP_BK
#define PPAS_GATEUP_BK 64
#endif
#ifndef PPAS_GATEUP_RING
#define PPAS_GATEUP_RING 2
#endif
#ifndef PPAS_GATEUP_SPREAD
#define PPAS_GATEUP_SPREAD 2
#endif
#ifndef PPAS_GATEUP_WAVES
#define PPAS_GATEUP_WAVES 8
#endif
constexpr int kWaves = PPAS_GATEUP_WAVES;  // waves per workgroup: one or two per SIMD
static_assert(kWaves == 4 || kWaves == 8, "four or eight waves");
constexpr int kThreads = 64 * kWaves;
constexpr int kBM = 256;                 // token rows per tile
constexpr int kBMTail = 64;              // token rows per tile of the last T % 256 rows
constexpr int kBN = 256;                 // output columns per tile
constexpr int kBK = PPAS_GATEUP_BK;     // features per stage
constexpr int kKSteps = kBK / 16;        // MFMA k-steps per stage
constexpr int kRing = PPAS_GATEUP_RING;  // stages in the LDS ring; transfers run kRing - 1 stages ahead
constexpr int kCPR = kBK / 8;            // 16-byte chunks of a row per stage
constexpr int kRowBytes = 16 * kCPR;
constexpr int kRowsPerDma = 64 / kCPR;   // whole rows covered by one 64-lane 16-byte transfer
constexpr int kPart = 256 * kRowBytes;   // the 256 W (or X) rows of one stage
constexpr int kStage = 2 * kPart;
static_assert(kBK == 32 || kBK == 64, "stages of 32 or 64 features");
static_assert(kRing >= 2 && kRing <= 5, "a ring of two to five stages");
constexpr int kSpread = PPAS_GATEUP_SPREAD < kKSteps ? PPAS_GATEUP_SPREAD : kKSteps;   // k-steps that issue the next stage
constexpr int kPitch = 128 * 2 + 16;     // epilogue LDS row pitch in bytes (16-byte aligned, padded)
constexpr int kEpiWave = (kBM * 2 / kWaves) * kPitch;   // one wave's output block of a full tile (<= 128 columns)
constexpr int kSmem = (kRing * kStage > kWaves * kEpiWave) ? kRing * kStage : kWaves * kEpiWave;
static_assert(kSmem <= 160 * 1024, "the LDS of one compute unit");
constexpr int kGroupM = 8;               // token-row tiles per tile-order group
#ifndef PPAS_GATEUP_PERSIST
#define PPAS_GATEUP_PERSIST 1
#endif
constexpr bool kPersist = PPAS_GATEUP_PERSIST;   // a workgroup per compute unit, looping over tiles


struct GemmArgs {
  const uint16_t* x;
  const uint16_t* w;
  uint16_t* y;
  float* part;            // splits > 1: fp32 partial sums [splits][T][N2]
  int32_t T, H, N2;
  int32_t tiles_m, tiles_n;   // full 256-row tiles, 256-column tiles
  int32_t tail_m;             // 64-row tiles of the last T % 256 rows
  int32_t splits;             // reduction split over this many workgroups per tile
  int32_t I;                  // with the gated activation: N2 / 2 intermediate features
};

__device__ __forceinline__ u32x4 lds16(const char* p) { return *reinterpret_cast<const u32x4*>(p); }

// LDS row layout of a stage: row R's 16-byte chunk c sits at position
// c ^ swizzle(R). Sixteen consecutive rows span 256 bytes' worth of banks in
// kRowBytes-sized rows, and the swizzle gives each of them a different position
// for the same chunk, so the 16 lanes an operand read serves per cycle hit 16
// different 16-byte bank groups.
__device__ __forceinline__ int swizzle(int R) { return (R / (16 / kCPR)) % kCPR; }
__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// silu(g) = g / (1 + e^-g) in fp32 (e^-g through the hardware base-2 exponential;
// +inf for large negative g, which gives -0).
__device__ __forceinline__ float silu_f32(float g) {
  return g / (1.f + __builtin_amdgcn_exp2f(-g * 1.4426950408889634f));
}

// 16 bytes from global memory into LDS: lane L of the wave lands at lds + 16 L.
__device__ __forceinline__ void dma16(const uint16_t* g, char* lds) {
  __builtin_amdgcn_global_load_lds((global_cvoid*)g, (lds_void*)lds, 16, 0, 0);
}

__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Wait until at most `later` stages of PER transfers each are still in flight
// (vmcnt: bits 3:0 and 15:14 of the s_waitcnt immediate).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}
template <int PER>
__device__ __forceinline__ void wait_stages(int later) {
  static_assert((kRing - 2) * PER < 64, "the transfers in flight fit the vmcnt counter");
  if (later >= 3)
    wait_vmcnt<(kRing >= 5 ? 3 * PER : 0)>();
  else if (later == 2)
    wait_vmcnt<2 * PER>();
  else if (later == 1)
    wait_vmcnt<PER>();
  else
    wait_vmcnt<0>();
}

// Workgroup barrier without a memory fence (the fence of __syncthreads would also
// wait for the transfers still in flight for later stages). The LDS data it
// guards is written only by the transfers, whose completion each wave waits for
// explicitly; the empty asm keeps the compiler from moving memory accesses
// across it.
__device__ __forceinline__ void bare_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::: "memory");
}

// One output tile of BM token rows x 256 columns over stages k_lo .. k_hi - 1.
// BM = 256 (full tiles) or 64 (the ragged last rows of the tokens, and calls of
// fewer than 256 tokens). Wave (wn, wm) owns a WN x WM block of it (columns x
// token rows) as kNT x kMT MFMA tiles of 32 x 32:
//   four waves:  128 x 128 (full), 128 x 32 (tail)
//   eight waves: 128 x 64 (full),   64 x 32 (tail)
// The W part of a stage is always 256 rows, the X part BM rows; the first half
// of the waves copy the W part, the second half the X part, in equal shares.
template <int BM, bool kAct>
__device__ __forceinline__ void tile_body(const GemmArgs& a, char* smem, int m0, int n0, int split, int k_lo,
                                          int k_hi) {
  constexpr int WN = (BM == kBM || kWaves == 4) ? 128 : 64;   // columns per wave
  constexpr int NG = kBN / WN;                                // column groups
  constexpr int WM = BM / (kWaves / NG);                      // token rows per wave
  constexpr int kNT = WN / 32, kMT = WM / 32;                 // MFMA tiles per wave
  static_assert(NG * (BM / WM) == kWaves && WM % 32 == 0, "wave blocks tile the output tile");
  constexpr int kHalf = kWaves / 2;                  // waves per operand part
  constexpr int kDmaX = (BM / kHalf) / kRowsPerDma;  // transfers per X wave per stage
  constexpr int kDmaMax = (kBN / kHalf) / kRowsPerDma;   // a W wave's count (the larger)
  static_assert(kDmaX >= 1, "every X wave copies whole transfers");
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

  // Transfers: wave w copies its share of one part of every stage: W rows (the
  // first half of the waves) or X rows (the second half). One transfer covers
  // kRowsPerDma whole rows (the row's 16-byte chunks spread over kCPR consecutive
  // lanes); lane L lands at 16 L, i.e. at row position L % kCPR of its row, and
  // fetches the chunk stored there under the swizzle.
  const bool is_x = w >= kHalf;
  const int half = w % kHalf;
  const int rows_half = is_x ? BM / kHalf : kBN / kHalf;
  const uint16_t* gptr[kDmaMax];
  {
    const uint16_t* base = is_x ? a.x : a.w;
    const int r0 = (is_x ? m0 : n0) + rows_half * half;
    const int rmax = (is_x ? a.T : a.N2) - 1;
#pragma unroll
    for (int i = 0; i < kDmaMax; ++i) {
      const int R = rows_half * half + i * kRowsPerDma + lane / kCPR;   // row within the part
      const int c = (lane % kCPR) ^ swizzle(R);
      int r = min(r0 + i * kRowsPerDma + lane / kCPR, rmax);           // rows past the edge read the last row
      if (kAct && !is_x) {
        // with the gated activation the tile covers features n0 / 2 .. + 127: the
        // rows of wave column group R / WN are gate rows of WN / 2 features, then
        // the up rows of the same features (features past the end read the last)
        const int rr = R % WN;
        const int f = min(n0 / 2 + (WN / 2) * (R / WN) + rr % (WN / 2), a.I - 1);
        r = rr < WN / 2 ? f : a.I + f;
      }
      gptr[i] = base + size_t(r) * a.H + 8 * c;
    }
  }
  const int dst0 = (is_x ? kPart : 0) + rows_half * half * kRowBytes;
  // this wave's transfers i0 .. i0 + n - 1 of stage s (n a compile-time count)
  auto issue = [&](int s, int i0, auto n) {
    char* stage = smem + (s % kRing) * kStage + dst0;
#pragma unroll
    for (int i = 0; i < decltype(n)::value; ++i)
      dma16(gptr[i0 + i] + s * kBK, stage + (i0 + i) * kRowsPerDma * kRowBytes);
  };
  auto issue_all = [&](int s) {
    if (is_x)
      issue(s, 0, std::integral_constant<int, kDmaX>{});
    else
      issue(s, 0, std::integral_constant<int, kDmaMax>{});
  };
  // transfer i of this wave for stage sd into ring slot `slot` (in tail tiles
  // the X waves have fewer transfers than the W waves)
  auto dma_one = [&](int sd, int slot, int i) {
    if (kDmaX == kDmaMax || !is_x || i < kDmaX)
      dma16(gptr[i] + sd * kBK, smem + slot * kStage + dst0 + i * kRowsPerDma * kRowBytes);
  };
  constexpr int kDmaStep = kDmaMax / kSpread;   // transfers per k-step in the first kSpread k-steps
  static_assert(kDmaMax % kSpread == 0 && (kDmaX % kDmaStep == 0 || kDmaX < kDmaStep),
                "transfers split evenly over the k-steps");

  const int wn = w % NG, wm = w / NG;
  f32x16 acc[kNT][kMT];
#pragma unroll
  for (int i = 0; i < kNT; ++i)
#pragma unroll
    for (int j = 0; j < kMT; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Operand fragment (row tile q, k-step j) of lane L: row 32 q + L % 32 of the
  // wave's rows, chunk 2 j + L / 32; the swizzle term depends on the lane only.
  int roff[kKSteps];
#pragma unroll
  for (int j = 0; j < kKSteps; ++j)
    roff[j] = (lane & 31) * kRowBytes + 16 * ((2 * j + (lane >> 5)) ^ swizzle(lane & 31));

#pragma unroll
  for (int s = 0; s < kRing - 1; ++s)
    if (k_lo + s < k_hi) issue_all(k_lo + s);

  // Entering stage s: this wave's transfers of stage s are done once at most
  // those of the stages after it are still in flight; the barrier then makes
  // every wave's part visible and tells that stage s - 1, whose ring slot the
  // next transfers overwrite, has been read by all waves.
  auto enter = [&](int s) {
    const int later = min(k_hi - 1 - s, kRing - 2);
    if (is_x)
      wait_stages<kDmaX>(later);
    else
      wait_stages<kDmaMax>(later);
    bare_barrier();
  };
  // Operand fragments, double-buffered over k-steps. A k-step's eight reads go
  // out in two groups, (W 0, W 1, X 0 .. kMT-1) and (W 2, W 3), the first ahead
  // of the previous k-step's MFMAs and the second halfway through them, so that
  // at most 14 reads are outstanding (the LDS wait counter holds 15; with more
  // in flight every wait would have to drain them all).
  bf16x8 fa[2][kNT], fb[2][kMT];
  auto stage_ptrs = [&](int s, const char*& wf, const char*& xf) {
    const char* cur = smem + (s % kRing) * kStage;
    wf = cur + WN * wn * kRowBytes;
    xf = cur + kPart + WM * wm * kRowBytes;
  };
  auto read_a = [&](int s, int j, int f) {
    const char *wf, *xf;
    stage_ptrs(s, wf, xf);
#pragma unroll
    for (int q = 0; q < kNT / 2; ++q) fa[f][q] = as_bf16x8(lds16(wf + 32 * q * kRowBytes + roff[j]));
#pragma unroll
    for (int q = 0; q < kMT; ++q) fb[f][q] = as_bf16x8(lds16(xf + 32 * q * kRowBytes + roff[j]));
  };
  auto read_b = [&](int s, int j, int f) {
    const char *wf, *xf;
    stage_ptrs(s, wf, xf);
#pragma unroll
    for (int q = kNT / 2; q < kNT; ++q) fa[f][q] = as_bf16x8(lds16(wf + 32 * q * kRowBytes + roff[j]));
  };
  constexpr int kN = kNT * kMT;   // MFMAs per k-step: W row tile idx / kMT, X row tile idx % kMT
  static_assert(kKSteps % 2 == 0, "k-steps alternate the two fragment buffers");

  if (k_lo < k_hi) {
    enter(k_lo);
    read_a(k_lo, 0, 0);
    read_b(k_lo, 0, 0);
  }
  for (int s = k_lo; s < k_hi; ++s) {
    // The transfers of stage s + kRing - 1 go into the slot of stage s - 1, which
    // every wave has finished reading (the barrier of entering s). Past the last
    // stage they repeat stage k_hi - 1 into that free slot, which keeps the loop
    // free of branches around them; the waits count them as stages in flight.
    const int sd = min(s + kRing - 1, k_hi - 1);
    const int slot = (s + kRing - 1) % kRing;
#pragma unroll
    for (int j = 0; j < kKSteps; ++j) {
      const int f = j & 1;
      const bool last = j + 1 == kKSteps;
      if (!last) read_a(s, j + 1, f ^ 1);
      // this k-step's share of the next stage's transfers, behind the operand
      // reads so that the matrix cores start without waiting for them
      if (j < kSpread) {
#pragma unroll
        for (int d = 0; d < kDmaStep; ++d) dma_one(sd, slot, j * kDmaStep + d);
      }
      __builtin_amdgcn_sched_barrier(0);
      // the MFMAs, with the second read group halfway
#pragma unroll
      for (int idx = 0; idx < kN; ++idx) {
        const int ti = idx / kMT, tj = idx % kMT;
        acc[ti][tj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[f][ti], fb[f][tj], acc[ti][tj], 0, 0, 0);
        if (!last && idx == kN / 2 - 1) {
          __builtin_amdgcn_sched_barrier(0);
          read_b(s, j + 1, f ^ 1);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      if (last) {
        if (s + 1 < k_hi) {
          enter(s + 1);
          read_a(s + 1, 0, 0);
          read_b(s + 1, 0, 0);
        }
        // (outside the condition: a scheduling barrier inside it made the
        // register allocator spill)
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  wait_vmem();   // the repeated transfers of the last stages have landed
  __syncthreads();   // every wave is done with the ring before it holds the output

  // Result register r of MFMA tile (ti, tj): token row 32 tj + L % 32 of the
  // wave's rows, column 32 ti + 8(r / 4) + 4(L / 32) + r % 4 of its columns.
  const int mw = m0 + WM * wm, nw = n0 + WN * wn;
  if (a.splits > 1) {
    // fp32 partial sums of this split, straight from the accumulators: four
    // consecutive columns of one token row per (ti, tj, g)
    float* pb = a.part + size_t(split) * a.T * a.N2;
#pragma unroll
    for (int ti = 0; ti < kNT; ++ti)
#pragma unroll
      for (int tj = 0; tj < kMT; ++tj) {
        const int m = mw + 32 * tj + (lane & 31);
        if (m >= a.T) continue;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          // columns n .. n + 3, valid below `lim`
          int n = nw + 32 * ti + 8 * g + 4 * (lane >> 5);
          int lim = a.N2;
          bool vec = (a.N2 & 3) == 0;
          if (kAct) {
            // partials keep the weight-row order: gate feature f at column f,
            // its up row at I + f (features from I on belong to neither)
            const int f = n0 / 2 + (WN / 2) * wn + 32 * (ti % (kNT / 2)) + 8 * g + 4 * (lane >> 5);
            if (f >= a.I) continue;
            n = ti < kNT / 2 ? f : a.I + f;
            lim = ti < kNT / 2 ? a.I : a.N2;
            vec = (a.I & 3) == 0;
          }
          float* dst = pb + size_t(m) * a.N2 + n;
          if (n + 4 <= lim && vec) {
            *reinterpret_cast<f32x4*>(dst) =
                f32x4{acc[ti][tj][4 * g], acc[ti][tj][4 * g + 1], acc[ti][tj][4 * g + 2], acc[ti][tj][4 * g + 3]};
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (n + e < lim) dst[e] = acc[ti][tj][4 * g + e];
          }
        }
      }
    return;
  }

  if constexpr (kAct) {
    // silu(gate) * up: MFMA tiles ti and ti + kNT / 2 hold the gate and the up
    // value of the same (token row, feature) in the same register; the wave's
    // WN / 2 features x WM rows go to LDS, then out in WN-byte row runs.
    char* eb = smem + w * kEpiWave;
#pragma unroll
    for (int ti = 0; ti < kNT / 2; ++ti)
#pragma unroll
      for (int tj = 0; tj < kMT; ++tj)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int row = 32 * tj + (lane & 31);
          const int col = 32 * ti + 8 * g + 4 * (lane >> 5);
          float z[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) z[e] = silu_f32(acc[ti][tj][4 * g + e]) * acc[ti + kNT / 2][tj][4 * g + e];
          u32x2 v;
          v[0] = pack_bf16x2(z[0], z[1]);
          v[1] = pack_bf16x2(z[2], z[3]);
          *reinterpret_cast<u32x2*>(eb + row * kPitch + col * 2) = v;
        }
    __syncthreads();
    constexpr int WF = WN / 2;                       // features per wave
    constexpr int kLPR = WF / 8, kRPI = 64 / kLPR, kIters = WM / kRPI;
    const int fw = n0 / 2 + WF * wn;
    const int fb = fw + 8 * (lane % kLPR);
    if (mw + WM <= a.T && fw + WF <= a.I) {
      constexpr int kB = kIters < 8 ? kIters : 8;
#pragma unroll
      for (int s0 = 0; s0 < kIters; s0 += kB) {
        u32x4 v[kB];
#pragma unroll
        for (int i = 0; i < kB; ++i)
          v[i] = lds16(eb + (kRPI * (s0 + i) + lane / kLPR) * kPitch + 16 * (lane % kLPR));
#pragma unroll
        for (int i = 0; i < kB; ++i)
          *reinterpret_cast<u32x4*>(a.y + size_t(mw + kRPI * (s0 + i) + lane / kLPR) * a.I + fb) = v[i];
      }
      return;
    }
#pragma unroll 4
    for (int s = 0; s < kIters; ++s) {
      const int row = kRPI * s + lane / kLPR;
      const int m = mw + row;
      if (m >= a.T) break;
      const u32x4 v = lds16(eb + row * kPitch + 16 * (lane % kLPR));
      uint16_t* dst = a.y + size_t(m) * a.I + fb;
      if (fb + 8 <= a.I) {
        *reinterpret_cast<u32x4*>(dst) = v;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (fb + e < a.I) dst[e] = uint16_t(v[e >> 1] >> (16 * (e & 1)));
      }
    }
    return;
  }

  // bf16: the wave's block to LDS (token-row major), then out in WN * 2-byte row
  // runs (kLPR lanes per row, kRPI rows per store instruction).
  char* eb = smem + w * kEpiWave;
#pragma unroll
  for (int ti = 0; ti < kNT; ++ti)
#pragma unroll
    for (int tj = 0; tj < kMT; ++tj)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int row = 32 * tj + (lane & 31);
        const int col = 32 * ti + 8 * g + 4 * (lane >> 5);
        u32x2 v;
        v[0] = pack_bf16x2(acc[ti][tj][4 * g], acc[ti][tj][4 * g + 1]);
        v[1] = pack_bf16x2(acc[ti][tj][4 * g + 2], acc[ti][tj][4 * g + 3]);
        *reinterpret_cast<u32x2*>(eb + row * kPitch + col * 2) = v;
      }
  __syncthreads();
  constexpr int kLPR = WN / 8, kRPI = 64 / kLPR, kIters = WM / kRPI;
  const int nb = nw + 8 * (lane % kLPR);
  if (mw + WM <= a.T && nw + WN <= a.N2) {
    // interior block: up to eight LDS reads in flight, then their stores
    constexpr int kB = kIters < 8 ? kIters : 8;
#pragma unroll
    for (int s0 = 0; s0 < kIters; s0 += kB) {
      u32x4 v[kB];
#pragma unroll
      for (int i = 0; i < kB; ++i)
        v[i] = lds16(eb + (kRPI * (s0 + i) + lane / kLPR) * kPitch + 16 * (lane % kLPR));
#pragma unroll
      for (int i = 0; i < kB; ++i)
        *reinterpret_cast<u32x4*>(a.y + size_t(mw + kRPI * (s0 + i) + lane / kLPR) * a.N2 + nb) = v[i];
    }
    return;
  }
#pragma unroll 4
  for (int s = 0; s < kIters; ++s) {
    const int row = kRPI * s + lane / kLPR;
    const int m = mw + row;
    if (m >= a.T) break;
    const u32x4 v = lds16(eb + row * kPitch + 16 * (lane % kLPR));
    uint16_t* dst = a.y + size_t(m) * a.N2 + nb;
    if (nb + 8 <= a.N2) {
      *reinterpret_cast<u32x4*>(dst) = v;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (nb + e < a.N2) dst[e] = uint16_t(v[e >> 1] >> (16 * (e & 1)));
    }
  }
}

template <bool kAct>
__global__ __launch_bounds__(kThreads, 1) void gateup_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem[kSmem];

  // Work item q -> (tile, split): the first 8 * (items / 8) items give XCD q % 8
  // the contiguous range xcd * (items / 8) + q / 8 (workgroup b runs on XCD b % 8,
  // and the grid is a multiple of 8 whenever it is smaller than the item count);
  // the remainder runs in order. Item u is tile u % tiles of reduction split
  // u / tiles, so the workgroups next to each other on an XCD work on
  // neighbouring tiles of the same split. Tiles 0 .. full - 1 are the 256-row
  // tiles (in groups of 8 that share a weight tile), the rest the 64-row tiles of
  // the last T % 256 rows. A workgroup takes items blockIdx.x, + gridDim.x, ...
  const int full = a.tiles_m * a.tiles_n;
  const int ntiles = full + a.tail_m * a.tiles_n;
  const int nitems = ntiles * a.splits;
  const int per_xcd = nitems / 8;
  const int nk_all = a.H / kBK;
  for (int q = blockIdx.x; q < nitems; q += gridDim.x) {
    const int u = (q < 8 * per_xcd) ? (q % 8) * per_xcd + q / 8 : q;
    const int t = u % ntiles;
    const int split = u / ntiles;
    const int k_lo = int(int64_t(split) * nk_all / a.splits);
    const int k_hi = int(int64_t(split + 1) * nk_all / a.splits);
    if (t < full) {
      const int grp = t / (kGroupM * a.tiles_n);
      const int first_m = grp * kGroupM;
      const int gm = min(kGroupM, a.tiles_m - first_m);
      const int in_grp = t - grp * kGroupM * a.tiles_n;
      tile_body<kBM, kAct>(a, smem, (first_m + in_grp % gm) * kBM, (in_grp / gm) * kBN, split, k_lo, k_hi);
    } else {
      const int tt = t - full;
      tile_body<kBMTail, kAct>(a, smem, a.tiles_m * kBM + (tt % a.tail_m) * kBMTail, (tt / a.tail_m) * kBN,
                               split, k_lo, k_hi);
    }
    // the next item's transfers overwrite the LDS this item's epilogue has read;
    // its stores may still be in flight
    __builtin_amdgcn_s_waitcnt(0xC07F);
    bare_barrier();
  }
}

// y = bf16(sum over splits of the partials), the splits summed in order; thread i
// covers elements 4i .. 4i + 3 of the flattened [T][N2] output.
__global__ __launch_bounds__(256) void gateup_reduce_kernel(const float* part, uint16_t* y, int64_t total,
                                                            int32_t splits) {
  const int64_t e0 = (int64_t(blockIdx.x) * 256 + threadIdx.x) * 4;
  if (e0 >= total) return;
  if (e0 + 4 <= total) {
    f32x4 s = *reinterpret_cast<const f32x4*>(part + e0);
    for (int k = 1; k < splits; ++k) s += *reinterpret_cast<const f32x4*>(part + size_t(k) * total + e0);
    u32x2 v;
    v[0] = pack_bf16x2(s[0], s[1]);
    v[1] = pack_bf16x2(s[2], s[3]);
    *reinterpret_cast<u32x2*>(y + e0) = v;
  } else {
    for (int64_t e = e0; e < total; ++e) {
      float s = part[e];
      for (int k = 1; k < splits; ++k) s += part[size_t(k) * total + e];
      y[e] = uint16_t(pack_bf16x2(s, 0.f) & 0xffff);
    }
  }
}

// The gated activation from split partials: z[m][f] = bf16(silu(g) * u), g and u
// the in-order sums over splits of partial columns f and I + f of row m. Thread i
// covers elements 4i .. 4i + 3 of the flattened [T][I] output.
__global__ __launch_bounds__(256) void gateup_act_reduce_kernel(const float* part, uint16_t* y, int32_t T,
                                                                int32_t I, int32_t splits) {
  const int64_t total = int64_t(T) * I;
  const int64_t e0 = (int64_t(blockIdx.x) * 256 + threadIdx.x) * 4;
  if (e0 >= total) return;
  const int64_t plane = int64_t(T) * 2 * I;   // one split's [T][2I] partials
  auto one = [&](int64_t e) {
    const int64_t m = e / I, f = e % I;
    const float* pg = part + m * 2 * I + f;
    float g = pg[0], u = pg[I];
    for (int k = 1; k < splits; ++k) {
      g += pg[size_t(k) * plane];
      u += pg[size_t(k) * plane + I];
    }
    return silu_f32(g) * u;
  };
  if ((I & 3) == 0 && e0 + 4 <= total) {
    const int64_t m = e0 / I, f = e0 % I;
    const float* pg = part + m * 2 * I + f;
    f32x4 g = *reinterpret_cast<const f32x4*>(pg), u = *reinterpret_cast<const f32x4*>(pg + I);
    for (int k = 1; k < splits; ++k) {
      g += *reinterpret_cast<const f32x4*>(pg + size_t(k) * plane);
      u += *reinterpret_cast<const f32x4*>(pg + size_t(k) * plane + I);
    }
    u32x2 v;
    v[0] = pack_bf16x2(silu_f32(g[0]) * u[0], silu_f32(g[1]) * u[1]);
    v[1] = pack_bf16x2(silu_f32(g[2]) * u[2], silu_f32(g[3]) * u[3]);
    *reinterpret_cast<u32x2*>(y + e0) = v;
  } else {
    for (int64_t e = e0; e < e0 + 4 && e < total; ++e) y[e] = uint16_t(pack_bf16x2(one(e), 0.f) & 0xffff);
  }
}

}  // namespace

int64_t gateup_tiles(int32_t T, int32_t N2) {
  return (int64_t(T / kBM) + (T % kBM + kBMTail - 1) / kBMTail) * ((N2 + kBN - 1) / kBN);
}

int gateup_splits(int32_t T, int32_t H, int32_t N2, int cus) {
  const int64_t tiles = gateup_tiles(T, N2);
  const int nk = H / kBK;
  if (tiles <= 0 || tiles >= cus) return 1;
  // about one workgroup per compute unit, each with at least four stages
  return int(std::max<int64_t>(1, std::min<int64_t>(cus / tiles, nk / 4)));
}

size_t gateup_workspace_bytes(int32_t T, int32_t N2, int splits) {
  return splits > 1 ? size_t(splits) * size_t(T) * size_t(N2) * sizeof(float) : 0;
}

hipError_t launch_gateup(const uint16_t* x, const uint16_t* w, uint16_t* y, int32_t T, int32_t H, int32_t N2,
                         bool act, int splits, float* part, int cus, hipStream_t stream, hipEvent_t ev_start,
                         hipEvent_t ev_stop) {
  GemmArgs a;
  a.x = x;
  a.w = w;
  a.y = y;
  a.part = part;
  a.T = T;
  a.H = H;
  a.N2 = N2;
  a.tiles_m = T / kBM;
  a.tail_m = (T % kBM + kBMTail - 1) / kBMTail;
  a.tiles_n = (N2 + kBN - 1) / kBN;
  a.splits = splits;
  a.I = N2 / 2;
  const int64_t n = gateup_tiles(T, N2) * splits;
  if (n <= 0) return hipSuccess;
  if (n > INT32_MAX || splits < 1 || splits > H / kBK || (splits > 1 && !part) || (act && N2 % 2 != 0))
    return hipErrorInvalidValue;
  // one workgroup per compute unit, each looping over its items (a multiple of 8
  // workgroups, so that every workgroup stays on one XCD's share of the items)
  const int64_t slots = kPersist ? std::max(8, cus / 8 * 8) : n;
  const int64_t grid = std::min<int64_t>(n, slots);
  if (act)
    hipExtLaunchKernelGGL(gateup_kernel<true>, dim3(unsigned(grid)), dim3(kThreads), 0, stream, ev_start,
                          splits > 1 ? nullptr : ev_stop, 0, a);
  else
    hipExtLaunchKernelGGL(gateup_kernel<false>, dim3(unsigned(grid)), dim3(kThreads), 0, stream, ev_start,
                          splits > 1 ? nullptr : ev_stop, 0, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  const int64_t total = act ? int64_t(T) * (N2 / 2) : int64_t(T) * N2;
  const int64_t blocks = (total + 1023) / 1024;
  if (blocks > INT32_MAX) return hipErrorInvalidValue;
  if (act)
    hipExtLaunchKernelGGL(gateup_act_reduce_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream, nullptr, ev_stop,
                          0, static_cast<const float*>(part), y, T, N2 / 2, splits);
  else
    hipExtLaunchKernelGGL(gateup_reduce_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream, nullptr, ev_stop, 0,
                          static_cast<const float*>(part), y, total, splits);
  return hipGetLastError();
}

}  // namespace ppas
