// A plain streaming read of one device buffer: the attainable HBM read rate of
// the device, against which the library's memory-bound kernels (the decode
// items of the attention step, the page writes) are measured. Not a step of the
// method. Each wave reads contiguous 8 KB runs of the buffer (eight 1 KB loads in
// flight, nontemporal: the words are read once), the grid's waves a run apart,
// with one 256-thread workgroup per compute unit (on an MI355X this reads ~7 TB/s
// where a grid stride per thread, or more workgroups, read 5.6-6.5), and folds
// the 16-byte words by XOR; each wave folds its lanes and one lane XORs the
// wave's word into the 16-byte sink, so the output is exactly the XOR of all words
// of the buffer (XORed into what the sink held) and the loads cannot be elided.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "device.h"

namespace ppas {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kRun = 8;  // 1 KB loads per wave per run

__global__ __launch_bounds__(kThreads) void stream_read_kernel(const u32x4* __restrict__ buf, size_t n,
                                                               uint32_t* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  const size_t waves = size_t(gridDim.x) * (kThreads / 64);
  const size_t runs = n / (64 * kRun);
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (size_t r = size_t(blockIdx.x) * (kThreads / 64) + (threadIdx.x >> 6); r < runs; r += waves) {
    const u32x4* p = buf + r * (64 * kRun) + lane;
    u32x4 v[kRun];
#pragma unroll
    for (int k = 0; k < kRun; ++k) v[k] = __builtin_nontemporal_load(p + 64 * k);
#pragma unroll
    for (int k = 0; k < kRun; ++k) acc ^= v[k];
  }
  // the words after the last whole run, one per thread of the grid
  for (size_t i = runs * (64 * kRun) + size_t(blockIdx.x) * kThreads + threadIdx.x; i < n;
       i += size_t(gridDim.x) * kThreads)
    acc ^= __builtin_nontemporal_load(buf + i);
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    acc.x ^= __shfl_xor(acc.x, o);
    acc.y ^= __shfl_xor(acc.y, o);
    acc.z ^= __shfl_xor(acc.z, o);
    acc.w ^= __shfl_xor(acc.w, o);
  }
  if ((threadIdx.x & 63) == 0 && (acc.x | acc.y | acc.z | acc.w) != 0u) {
    atomicXor(sink + 0, acc.x);
    atomicXor(sink + 1, acc.y);
    atomicXor(sink + 2, acc.z);
    atomicXor(sink + 3, acc.w);
  }
}

}  // namespace

hipError_t launch_stream_read(const void* buf, size_t bytes, uint32_t* sink, int cus, hipStream_t stream,
                              hipEvent_t ev_start, hipEvent_t ev_stop) {
  const size_t n = bytes / 16;
  const size_t runs = n / (64 * kRun);
  // one workgroup per compute unit, fewer when the buffer has fewer runs
  const size_t need = (runs + kThreads / 64 - 1) / (kThreads / 64);
  const size_t grid = need < 1 ? 1 : (need < size_t(cus) ? need : size_t(cus));
  hipExtLaunchKernelGGL(stream_read_kernel, dim3(unsigned(grid)), dim3(kThreads), 0, stream, ev_start, ev_stop, 0,
                        static_cast<const u32x4*>(buf), n, sink);
  return hipGetLastError();
}

}  // namespace ppas
