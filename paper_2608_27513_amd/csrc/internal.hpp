// Library-internal declarations shared by the translation units of libdamp.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "damp.h"

namespace damp {

// Byte geometry of one packed tile (the format is documented in damp.h).
struct TileGeom {
  int32_t dk, dv, k_hi, kind;
  size_t hi_bytes;    // k_hi * dv * 2 (mixed) or dk * dv * 4 (fp32)
  size_t code_bytes;  // (dk - k_hi) * dv
  size_t meta_bytes;  // (dk - k_hi) * metadata bytes per row
  size_t tail_bytes;  // 4 (the E2M1 global scale) or 0
  size_t bytes;       // sum of the regions
  size_t stride;      // bytes rounded up to 128
};

// Fills g from a layout; returns false (and records why) if the layout is
// not one the layout math accepts.
bool tile_geom(const damp_layout* layout, TileGeom* g);

// Kernel codec of a layout (the KIND template argument of the kernels):
// the FP32 state, the default tiers, the paper's INT8 tiers, or the other
// rows of App. A.1's format table; kCodecNone if no kernel encodes it.
enum Codec {
  kCodecFp32 = 0,
  kCodecDefault = 1,
  kCodecPaper = 2,
  kCodecInt4 = 3,
  kCodecFp8 = 4,
  kCodecNvfp4 = 5,
  kCodecNone = -1
};
int layout_codec(const damp_layout* layout);

// True for the paper's tiers (App. A.1, Eq. (17)): FP16 high tier, groups
// of 32 with FP16 (s, z), UINT8 codes, with or without the block-32
// Hadamard transform.
bool layout_is_paper(const damp_layout* layout);

// True for the default tiers: BF16 high tier, one fp32 (s, z) pair per row,
// no transform.
bool layout_is_default(const damp_layout* layout);

// True if the layout has kernels: d_k == d_v in {16, 32, 64, 128} with the
// FP32 state or the default tiers, or d_k == d_v in {32, 64, 128} with the
// paper's tiers or another format of App. A.1's table.
bool layout_has_kernels(const damp_layout* layout);

// Validates a pool descriptor (non-null, consistent strides and counts).
damp_status check_pool(const damp_pool* pool);

// With the environment variable DAMP_CHECK_SLOTS set (and not "0"): copies
// the device slot ids to the host on `stream` (synchronising it) and fails
// with DAMP_ERR_INVALID_ARG if a slot inside the pool occurs twice. Without
// it: DAMP_OK at once. Called by every entry point that writes tiles.
damp_status debug_check_slots(const damp_pool* pool, const int32_t* slot_idx, int32_t B,
                              hipStream_t stream, const char* name);

// Thread-local error message.
damp_status fail(damp_status st, const char* fmt, ...);
void clear_error();

inline uint8_t* layer_base(const damp_pool* pool, int32_t layer) {
  return static_cast<uint8_t*>(pool->base) +
         static_cast<size_t>(layer) * static_cast<size_t>(pool->num_slots) *
             static_cast<size_t>(pool->num_v_heads) * pool->tile_stride;
}

inline hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

// Returns DAMP_ERR_HIP with a message if the last launch failed.
damp_status check_launch(const char* what);

// Enqueues the prefill kernel for input tokens [t0, t0 + T) of arrays that
// hold t_pitch tokens per request; o ([B, T, HV, d_v]) may be NULL. The
// caller has validated the pool, the layer, the sizes and the pointers.
void prefill_window(bool kda, const damp_pool* pool, int32_t layer, const int32_t* slot_idx,
                    int32_t B, int32_t t0, int32_t T, int32_t t_pitch, int32_t num_k_heads,
                    const uint16_t* q, const uint16_t* k, const uint16_t* v, const uint16_t* g,
                    const uint16_t* beta, const uint8_t* perm, float scale, void* o,
                    bool o_bf16, hipStream_t stream);

// Enqueues || Q_lo(x) - x ||^2 in double for `rows` independent fp32 rows of
// dv values (row i at states + i * dv) with Q_lo the paper's UINT8 group tier
// (groups of 32, FP16 (s, z), optionally after the block-32 transform);
// dv <= 128 and a multiple of 32. Row i's sum goes to err[i].
void launch_row_errors_group(const float* states, int64_t rows, int dv, bool had, double* err,
                             hipStream_t stream);

}  // namespace damp
