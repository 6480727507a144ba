// Fused gate-up projection of a decoder block's MLP on gfx950 (CDNA4):
//   Y[T][N2] = X[T][H] * W[N2][H]^T
// bf16 inputs, fp32 accumulation on 32x32x16 MFMAs, output rounded to bf16
// (nearest even). W stacks the gate rows over the up rows, so one launch
// computes both projections of a prefill chunk.
//
// Tiling. A workgroup of four waves (one per SIMD) computes a 256 x 256 output
// tile; wave (wn, wm) owns its 128 output columns x 128 token rows as 4 x 4
// MFMA tiles (256 fp32 accumulators per lane, held in the accumulation
// registers). The reduction advances 64 features per stage: a stage's W rows
// and X rows (32 KB each) are copied into LDS by 16-byte global-to-LDS
// transfers, each covering eight whole 128-byte row runs (one cache line per
// row), into a two-slot ring. In LDS a row keeps its eight 16-byte chunks in
// an XOR-swizzled order, so each operand fragment read (row tile, k-step: 32
// rows x 32 bytes) is one bank-conflict-free ds_read_b128, and each fragment
// feeds four MFMAs. The next stage's transfers are issued a quarter per k-step
// behind the operand reads, and the next k-step's fragments are read while the
// current k-step's 16 MFMAs run. (Transfers of 32-byte row pieces straight into
// operand order, and rings of four 32-feature stages, measured 33 % and 6 %
// slower.)
//
// The MFMA's first operand is W (rows = output columns), its second X (rows =
// tokens): lane L of a 32 x 32 result then holds token row L % 32 and, in
// registers 4g..4g+3, four consecutive output columns 8g + 4(L / 32) + 0..3,
// which the epilogue packs into 8-byte LDS writes; the tile then leaves LDS as
// 256-byte row runs of 16-byte stores.
//
// Tile order. Workgroup b runs on XCD b % 8; each XCD takes a contiguous range
// of tiles, and tiles are numbered in groups of 8 token-row tiles that share a
// weight tile, so the workgroups resident on one XCD share operand tiles in
// that XCD's L2.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>

namespace ppas {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
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
constexpr int kThreads = 256;
constexpr int kBM = 256;                 // token rows per tile
constexpr int kBN = 256;                 // output columns per tile
constexpr int kBK = PPAS_GATEUP_BK;     // features per stage
constexpr int kKSteps = kBK / 16;        // MFMA k-steps per stage
constexpr int kRing = PPAS_GATEUP_RING;  // stages in the LDS ring; transfers run kRing - 1 stages ahead
constexpr int kCPR = kBK / 8;            // 16-byte chunks of a row per stage
constexpr int kRowBytes = 16 * kCPR;
constexpr int kRowsPerDma = 64 / kCPR;   // whole rows covered by one 64-lane 16-byte transfer
constexpr int kPart = 256 * kRowBytes;   // the 256 W (or X) rows of one stage
constexpr int kStage = 2 * kPart;
constexpr int kDmaPerStage = 128 / kRowsPerDma;   // transfers per wave per stage (two waves per part)
static_assert(kBK == 32 || kBK == 64, "stages of 32 or 64 features");
static_assert(kRing >= 2 && kRing <= 4, "a ring of two to four stages");
constexpr int kPitch = 128 * 2 + 16;     // epilogue LDS row pitch in bytes (16-byte aligned, padded)
constexpr int kEpiWave = 128 * kPitch;   // one wave's 128 x 128 bf16 output block
constexpr int kSmem = (kRing * kStage > 4 * kEpiWave) ? kRing * kStage : 4 * kEpiWave;
constexpr int kGroupM = 8;               // token-row tiles per tile-order group

struct GemmArgs {
  const uint16_t* x;
  const uint16_t* w;
  uint16_t* y;
  int32_t T, H, N2;
  int32_t tiles_m, tiles_n;
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

// 16 bytes from global memory into LDS: lane L of the wave lands at lds + 16 L.
__device__ __forceinline__ void dma16(const uint16_t* g, char* lds) {
  __builtin_amdgcn_global_load_lds((global_cvoid*)g, (lds_void*)lds, 16, 0, 0);
}

__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

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

__global__ __launch_bounds__(kThreads, 1) void gateup_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem[kSmem];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);

  // blockIdx -> tile: the first 8 * (tiles / 8) workgroups give XCD b % 8 the
  // contiguous range of tiles xcd * (tiles / 8) + ...; the remainder runs in order.
  const int ntiles = a.tiles_m * a.tiles_n;
  const int per_xcd = ntiles / 8;
  const int b = blockIdx.x;
  const int t = (b < 8 * per_xcd) ? (b % 8) * per_xcd + b / 8 : b;
  const int grp = t / (kGroupM * a.tiles_n);
  const int first_m = grp * kGroupM;
  const int gm = min(kGroupM, a.tiles_m - first_m);
  const int in_grp = t - grp * kGroupM * a.tiles_n;
  const int m0 = (first_m + in_grp % gm) * kBM;
  const int n0 = (in_grp / gm) * kBN;

  // Transfers: wave w copies half of one part of every stage: W rows (waves 0, 1)
  // or X rows (waves 2, 3), rows 128(w & 1) .. 128(w & 1) + 127 of the tile. One
  // transfer covers kRowsPerDma whole rows (the row's 16-byte chunks spread over
  // kCPR consecutive lanes); lane L lands at 16 L, i.e. at row position L % kCPR
  // of its row, and fetches the chunk stored there under the swizzle.
  const bool is_x = w >= 2;
  const int half = w & 1;
  const uint16_t* gptr[kDmaPerStage];
  {
    const uint16_t* base = is_x ? a.x : a.w;
    const int r0 = (is_x ? m0 : n0) + 128 * half;
    const int rmax = (is_x ? a.T : a.N2) - 1;
#pragma unroll
    for (int i = 0; i < kDmaPerStage; ++i) {
      const int R = 128 * half + i * kRowsPerDma + lane / kCPR;      // row within the part
      const int c = (lane % kCPR) ^ swizzle(R);
      const int r = min(r0 + i * kRowsPerDma + lane / kCPR, rmax);   // rows past the edge read the last row
      gptr[i] = base + size_t(r) * a.H + 8 * c;
    }
  }
  const int dst0 = (is_x ? kPart : 0) + 128 * half * kRowBytes;
  // transfers i0 .. i0 + n - 1 of stage s
  auto issue = [&](int s, int i0, int n) {
    char* stage = smem + (s % kRing) * kStage + dst0;
#pragma unroll
    for (int i = i0; i < i0 + n; ++i) dma16(gptr[i] + s * kBK, stage + i * kRowsPerDma * kRowBytes);
  };

  const int wn = w >> 1, wm = w & 1;
  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // Operand fragment (row tile q, k-step j) of lane L: row 32 q + L % 32 of the
  // wave's half, chunk 2 j + L / 32; the swizzle term depends on the lane only.
  int roff[kKSteps];
#pragma unroll
  for (int j = 0; j < kKSteps; ++j)
    roff[j] = (lane & 31) * kRowBytes + 16 * ((2 * j + (lane >> 5)) ^ swizzle(lane & 31));

  const int nk = a.H / kBK;
#pragma unroll
  for (int s = 0; s < kRing - 1; ++s)
    if (s < nk) issue(s, 0, kDmaPerStage);
  for (int s = 0; s < nk; ++s) {
    // this wave's transfers of stage s are done once at most those of the stages
    // after it (up to two) are still in flight; the barrier then makes every
    // wave's part visible and tells that stage s - 1, whose ring slot the next
    // transfers overwrite, has been read by all waves
    const int later = min(nk - 1 - s, kRing - 2);
    if (later >= 2)
      __builtin_amdgcn_s_waitcnt(0x0F70 | ((2 * kDmaPerStage) & 15) | (((2 * kDmaPerStage) >> 4) << 14));
    else if (later == 1)
      __builtin_amdgcn_s_waitcnt(0x0F70 | (kDmaPerStage & 15) | ((kDmaPerStage >> 4) << 14));
    else
      wait_vmem();
    bare_barrier();
    const bool more = s + kRing - 1 < nk;
    const char* cur = smem + (s % kRing) * kStage;
    const char* wf = cur + 128 * wn * kRowBytes;
    const char* xf = cur + kPart + 128 * wm * kRowBytes;
    // The eight fragments of k-step j + 1 are read while the 16 MFMAs of k-step j
    // run (the scheduling barriers keep the reads ahead of those MFMAs).
    bf16x8 fa[2][4], fb[2][4];
    auto read = [&](int j, bf16x8 (&ra)[4], bf16x8 (&rb)[4]) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        ra[q] = as_bf16x8(lds16(wf + 32 * q * kRowBytes + roff[j]));
        rb[q] = as_bf16x8(lds16(xf + 32 * q * kRowBytes + roff[j]));
      }
    };
    read(0, fa[0], fb[0]);
#pragma unroll
    for (int j = 0; j < kKSteps; ++j) {
      if (j + 1 < kKSteps) read(j + 1, fa[(j + 1) & 1], fb[(j + 1) & 1]);
      // the next stage's transfers, a quarter per k-step, issued behind this
      // k-step's operand reads so that the matrix cores start without waiting
      // for the whole batch of transfers
      if (more) issue(s + kRing - 1, j * (kDmaPerStage / kKSteps), kDmaPerStage / kKSteps);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int ti = 0; ti < 4; ++ti)
#pragma unroll
        for (int tj = 0; tj < 4; ++tj)
          acc[ti][tj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[j & 1][ti], fb[j & 1][tj], acc[ti][tj], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  __syncthreads();   // every wave is done with the ring before it holds the output

  // Epilogue: this wave's 128 x 128 block to LDS (token-row major), then out in
  // 256-byte row runs. Result register r of MFMA tile (ti, tj): token row
  // 32 tj + L % 32, column 32 ti + 8(r / 4) + 4(L / 32) + r % 4.
  char* eb = smem + w * kEpiWave;
#pragma unroll
  for (int ti = 0; ti < 4; ++ti)
#pragma unroll
    for (int tj = 0; tj < 4; ++tj)
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
  const int mb = m0 + 128 * wm, nb = n0 + 128 * wn + 8 * (lane & 15);
#pragma unroll 4
  for (int s = 0; s < 32; ++s) {
    const int row = 4 * s + (lane >> 4);
    const int m = mb + row;
    if (m >= a.T) break;
    const u32x4 v = lds16(eb + row * kPitch + 16 * (lane & 15));
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

}  // namespace

hipError_t launch_gateup(const uint16_t* x, const uint16_t* w, uint16_t* y, int32_t T, int32_t H, int32_t N2,
                         hipStream_t stream, hipEvent_t ev_start, hipEvent_t ev_stop) {
  GemmArgs a;
  a.x = x;
  a.w = w;
  a.y = y;
  a.T = T;
  a.H = H;
  a.N2 = N2;
  a.tiles_m = (T + kBM - 1) / kBM;
  a.tiles_n = (N2 + kBN - 1) / kBN;
  const int64_t n = int64_t(a.tiles_m) * a.tiles_n;
  if (n <= 0) return hipSuccess;
  if (n > INT32_MAX) return hipErrorInvalidValue;
  hipExtLaunchKernelGGL(gateup_kernel, dim3(unsigned(n)), dim3(kThreads), 0, stream, ev_start, ev_stop, 0, a);
  return hipGetLastError();
}

}  // namespace ppas
