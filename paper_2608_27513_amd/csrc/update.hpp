// Parameters shared by the decode-step update kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace damp {

struct UpdateParams {
  uint8_t* layer_base;
  uint64_t slot_stride;
  uint64_t tile_stride;
  const int32_t* slot_idx;
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* g;
  const uint16_t* beta;
  const uint8_t* perm;
  void* o;
  float scale;
  int32_t num_slots;
  int32_t HK;
  int32_t HV;
  int32_t k_hi;
  int32_t o_bf16;
  int32_t had;  // block-32 Hadamard on the low tier (paper tiers only)
};

// The streaming kernel for d = 128 mixed tiles with k_hi <= 32 (update_stream.hip)
// in the default tiers (fmt = kMixed) or another format of App. A.1's table
// (kPaper, kInt4, kFp8, kNvfp4). Returns false if it did not launch (the occupancy
// query or the launch failed).
bool launch_stream128(bool kda, int fmt, const UpdateParams& p, int B, hipStream_t stream);

// The FP32-state update at d = 128 (update_fp32.hip): one workgroup per tile,
// grid (HV, B), every access whole 128-byte lines.
void launch_fp32_128(bool kda, const UpdateParams& p, int B, hipStream_t stream);

}  // namespace damp
