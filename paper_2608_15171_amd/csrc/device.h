// Host-side helpers shared by the entry points: kernel launchers and the
// current device's properties.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "plan.h"

namespace ppas {

struct DeviceInfo {
  bool known = false;
  bool gfx950 = false;
  int cus = 256;
};

// Compute-unit count and architecture of the current device (cached per device).
// Without a usable device: 256 CUs, not gfx950.
DeviceInfo current_device();

// The packed attention launch and, when n_comb > 0, the split-merge launch.
hipError_t launch_attn_step(const uint16_t* q, uint16_t* out, const uint16_t* kp, const uint16_t* vp,
                            const int32_t* bt, int32_t bt_stride, int32_t hq, int32_t hkv, float scale,
                            const WorkItem* items, int n_items, const CombineItem* comb, int n_comb,
                            float2* part_ml, float* part_acc, int tile_pos, hipStream_t stream,
                            hipEvent_t ev_start, hipEvent_t ev_stop, hipEvent_t ev_merge_start,
                            hipEvent_t ev_merge_stop);

// The gate-up projection: y = x w^T (hidden a multiple of 64), or with `act` the
// gated activation of its two halves, y[t][f] = silu(s[t][f]) s[t][N2/2 + f]
// (N2 even, y [T][N2/2]). With splits > 1 the reduction is split over that many
// workgroups per output tile, whose fp32 partial sums (gateup_workspace_bytes of
// `part`, columns in weight-row order) a second launch adds in order. `cus` is
// the device's compute-unit count (the grid holds one workgroup per unit).
hipError_t launch_gateup(const uint16_t* x, const uint16_t* w, uint16_t* y, int32_t T, int32_t H, int32_t N2,
                         bool act, int splits, float* part, int cus, hipStream_t stream, hipEvent_t ev_start,
                         hipEvent_t ev_stop);
// Output tiles of a call: 256 x 256, plus 64 x 256 for the last T % 256 token rows.
int64_t gateup_tiles(int32_t T, int32_t N2);
// Reduction splits chosen for a device with `cus` compute units (1: no split).
int gateup_splits(int32_t T, int32_t H, int32_t N2, int cus);
size_t gateup_workspace_bytes(int32_t T, int32_t N2, int splits);

// XOR of every 16-byte word of buf (bytes a multiple of 16) into sink[0..3],
// read once by a streaming grid of up to `cus` workgroups.
hipError_t launch_stream_read(const void* buf, size_t bytes, uint32_t* sink, int cus, hipStream_t stream,
                              hipEvent_t ev_start, hipEvent_t ev_stop);

}  // namespace ppas
