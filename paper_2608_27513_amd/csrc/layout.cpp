// Layout arithmetic, pool descriptors and error reporting of libdamp.
//
// Tile format: section 5.2 and App. A.5 (Eq. (17)) of the DAMP paper, with
// one (s, z) pair per low-tier row; storage cost: Eq. (7) and Eq. (12).
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "internal.hpp"

namespace damp {

namespace {
thread_local char g_error[512] = "";

int dtype_bits(int32_t dt) {
  switch (dt) {
    case DAMP_DT_FP32: return 32;
    case DAMP_DT_BF16: return 16;
    case DAMP_DT_FP16: return 16;
    case DAMP_DT_E4M3: return 8;
    default: return -1;
  }
}
}  // namespace

damp_status fail(damp_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_error, sizeof g_error, fmt, ap);
  va_end(ap);
  return st;
}

void clear_error() { g_error[0] = '\0'; }

damp_status check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(DAMP_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return DAMP_OK;
}

bool tile_geom(const damp_layout* L, TileGeom* g) {
  if (!L) {
    fail(DAMP_ERR_INVALID_ARG, "layout is NULL");
    return false;
  }
  if (L->d_k <= 0 || L->d_v <= 0 || L->d_k > 256 || L->d_v > 4096) {
    fail(DAMP_ERR_INVALID_ARG, "d_k = %d, d_v = %d out of range (d_k <= 256)", L->d_k, L->d_v);
    return false;
  }
  if (L->kind != DAMP_STATE_FP32 && L->kind != DAMP_STATE_MIXED) {
    fail(DAMP_ERR_INVALID_ARG, "unknown state kind %d", L->kind);
    return false;
  }
  g->dk = L->d_k;
  g->dv = L->d_v;
  g->kind = L->kind;
  const size_t dk = static_cast<size_t>(L->d_k), dv = static_cast<size_t>(L->d_v);
  g->tail_bytes = 0;
  if (L->kind == DAMP_STATE_FP32) {
    g->k_hi = 0;
    g->hi_bytes = dk * dv * 4;
    g->code_bytes = g->meta_bytes = 0;
  } else {
    if (L->k_hi < 0 || L->k_hi > L->d_k) {
      fail(DAMP_ERR_INVALID_ARG, "k_hi = %d outside [0, d_k = %d]", L->k_hi, L->d_k);
      return false;
    }
    const int hb = dtype_bits(L->hi_dtype), mb = dtype_bits(L->meta_dtype);
    if (hb < 0 || hb == 8 || mb < 0) {
      fail(DAMP_ERR_INVALID_ARG, "unknown high-tier or metadata dtype");
      return false;
    }
    if (L->group <= 0 || L->d_v % L->group != 0) {
      fail(DAMP_ERR_INVALID_ARG, "group = %d does not divide d_v = %d", L->group, L->d_v);
      return false;
    }
    // metadata per group: (s, z) for the integer codes, one fp32 scale for
    // E4M3, one E4M3 block scale for E2M1 (plus the tile's fp32 global scale)
    const int cd = L->code_dtype;
    const bool ok = (cd == DAMP_DT_U8 && (mb == 32 || mb == 16)) ||
                    (cd == DAMP_DT_U4 && L->meta_dtype == DAMP_DT_FP16) ||
                    (cd == DAMP_DT_E4M3 && L->meta_dtype == DAMP_DT_FP32) ||
                    (cd == DAMP_DT_E2M1 && L->meta_dtype == DAMP_DT_E4M3);
    if (!ok) {
      fail(DAMP_ERR_INVALID_ARG, "code dtype %d with metadata dtype %d is not a format", cd,
           L->meta_dtype);
      return false;
    }
    const bool nibble = cd == DAMP_DT_U4 || cd == DAMP_DT_E2M1;
    if (nibble && L->d_v % 2 != 0) {
      fail(DAMP_ERR_INVALID_ARG, "4-bit codes need an even d_v");
      return false;
    }
    const size_t lo_rows = dk - static_cast<size_t>(L->k_hi);
    const size_t groups = dv / static_cast<size_t>(L->group);
    g->k_hi = L->k_hi;
    g->hi_bytes = static_cast<size_t>(L->k_hi) * dv * static_cast<size_t>(hb / 8);
    g->code_bytes = lo_rows * (nibble ? dv / 2 : dv);
    const size_t words = (cd == DAMP_DT_U8 || cd == DAMP_DT_U4) ? 2 : 1;
    g->meta_bytes = lo_rows * groups * words * static_cast<size_t>(mb / 8);
    g->tail_bytes = cd == DAMP_DT_E2M1 ? 4 : 0;
  }
  g->bytes = g->hi_bytes + g->code_bytes + g->meta_bytes + g->tail_bytes;
  g->stride = (g->bytes + 127) / 128 * 128;
  return true;
}

bool layout_is_paper(const damp_layout* L) {
  return layout_codec(L) == kCodecPaper;
}

bool layout_is_default(const damp_layout* L) {
  return L->kind == DAMP_STATE_MIXED && L->hi_dtype == DAMP_DT_BF16 &&
         L->meta_dtype == DAMP_DT_FP32 && L->group == L->d_v && L->hadamard == 0 &&
         L->code_dtype == DAMP_DT_U8;
}

int layout_codec(const damp_layout* L) {
  if (L->kind == DAMP_STATE_FP32) return kCodecFp32;
  if (L->kind != DAMP_STATE_MIXED) return kCodecNone;
  if (layout_is_default(L)) return kCodecDefault;
  if (L->hi_dtype != DAMP_DT_FP16) return kCodecNone;
  const bool had01 = L->hadamard == 0 || L->hadamard == 1;
  if (L->code_dtype == DAMP_DT_U8 && L->meta_dtype == DAMP_DT_FP16 && L->group == 32 && had01)
    return kCodecPaper;
  if (L->code_dtype == DAMP_DT_U4 && L->meta_dtype == DAMP_DT_FP16 && L->group == 32 && had01)
    return kCodecInt4;
  if (L->code_dtype == DAMP_DT_E4M3 && L->meta_dtype == DAMP_DT_FP32 && L->group == 32 &&
      L->hadamard == 0)
    return kCodecFp8;
  if (L->code_dtype == DAMP_DT_E2M1 && L->meta_dtype == DAMP_DT_E4M3 && L->group == 16 &&
      L->hadamard == 0)
    return kCodecNvfp4;
  return kCodecNone;
}

bool layout_has_kernels(const damp_layout* L) {
  if (L->d_k != L->d_v) return false;
  if (L->d_k != 16 && L->d_k != 32 && L->d_k != 64 && L->d_k != 128) return false;
  const int c = layout_codec(L);
  if (c == kCodecFp32 || c == kCodecDefault) return true;
  return c != kCodecNone && L->d_k >= 32;
}

damp_status check_pool(const damp_pool* pool) {
  if (!pool) return fail(DAMP_ERR_INVALID_ARG, "pool is NULL");
  TileGeom g;
  if (!tile_geom(&pool->layout, &g)) return DAMP_ERR_INVALID_ARG;
  if (!pool->base) return fail(DAMP_ERR_INVALID_ARG, "pool base is NULL");
  if (pool->num_layers <= 0 || pool->num_slots <= 0 || pool->num_v_heads <= 0)
    return fail(DAMP_ERR_INVALID_ARG, "pool counts must be positive");
  if (pool->tile_stride != g.stride)
    return fail(DAMP_ERR_INVALID_ARG, "pool tile_stride %zu != layout stride %zu",
                pool->tile_stride, g.stride);
  const size_t need = g.stride * static_cast<size_t>(pool->num_layers) *
                      static_cast<size_t>(pool->num_slots) *
                      static_cast<size_t>(pool->num_v_heads);
  if (pool->bytes < need)
    return fail(DAMP_ERR_INVALID_ARG, "pool spans %zu bytes, needs %zu", pool->bytes, need);
  return DAMP_OK;
}

namespace {

// The first slot in [0, num_slots) that occurs twice among ids[0..B), or -1.
int32_t first_repeat(const int32_t* ids, int32_t B, int32_t num_slots) {
  std::vector<int32_t> v;
  v.reserve(static_cast<size_t>(B));
  for (int32_t i = 0; i < B; ++i)
    if (ids[i] >= 0 && ids[i] < num_slots) v.push_back(ids[i]);
  std::sort(v.begin(), v.end());
  const auto it = std::adjacent_find(v.begin(), v.end());
  return it == v.end() ? -1 : *it;
}

damp_status check_slots(const damp_pool* pool, const int32_t* slot_idx, int32_t B,
                        bool on_device, hipStream_t stream, const char* name) {
  if (B <= 0) return DAMP_OK;
  const int32_t* ids = slot_idx;
  std::vector<int32_t> host;
  if (on_device) {
    host.resize(static_cast<size_t>(B));
    hipError_t e = hipMemcpyAsync(host.data(), slot_idx, sizeof(int32_t) * host.size(),
                                  hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return fail(DAMP_ERR_HIP, "%s: slot ids: %s", name, hipGetErrorString(e));
    ids = host.data();
  }
  const int32_t rep = first_repeat(ids, B, pool->num_slots);
  if (rep >= 0)
    return fail(DAMP_ERR_INVALID_ARG, "%s: slot %d appears more than once in the batch", name,
                rep);
  return DAMP_OK;
}

}  // namespace

damp_status debug_check_slots(const damp_pool* pool, const int32_t* slot_idx, int32_t B,
                              hipStream_t stream, const char* name) {
  const char* env = std::getenv("DAMP_CHECK_SLOTS");
  if (!env || env[0] == '\0' || env[0] == '0') return DAMP_OK;
  return check_slots(pool, slot_idx, B, true, stream, name);
}

}  // namespace damp

using namespace damp;

extern "C" {

const char* damp_last_error(void) { return g_error; }

damp_status damp_layout_init(damp_layout* out, int32_t d_k, int32_t d_v, int32_t k_hi,
                             int32_t kind) {
  clear_error();
  if (!out) return fail(DAMP_ERR_INVALID_ARG, "out is NULL");
  damp_layout L;
  std::memset(&L, 0, sizeof L);
  L.d_k = d_k;
  L.d_v = d_v;
  L.k_hi = kind == DAMP_STATE_FP32 ? 0 : k_hi;
  L.kind = kind;
  L.hi_dtype = DAMP_DT_BF16;
  L.group = d_v;
  L.meta_dtype = DAMP_DT_FP32;
  L.hadamard = 0;
  L.code_dtype = DAMP_DT_U8;
  TileGeom g;
  if (!tile_geom(&L, &g)) return DAMP_ERR_INVALID_ARG;
  *out = L;
  return DAMP_OK;
}

size_t damp_tile_bytes(const damp_layout* layout) {
  TileGeom g;
  return tile_geom(layout, &g) ? g.bytes : 0;
}

size_t damp_tile_stride(const damp_layout* layout) {
  TileGeom g;
  return tile_geom(layout, &g) ? g.stride : 0;
}

double damp_bits_per_value(const damp_layout* layout) {
  TileGeom g;
  if (!tile_geom(layout, &g)) return -1.0;
  if (layout->kind == DAMP_STATE_FP32) return 32.0;
  // Eq. (7): b = b_lo + (k_hi / d_k) (b_hi - b_lo), with b_lo = code bits plus
  // the metadata words of a group (the per-tile global scale of E2M1 is left
  // out, as App. A.1 does).
  const int cd = layout->code_dtype;
  const double meta_bits = static_cast<double>(dtype_bits(layout->meta_dtype));
  const double words = (cd == DAMP_DT_U8 || cd == DAMP_DT_U4) ? 2.0 : 1.0;
  const double code_bits = (cd == DAMP_DT_U4 || cd == DAMP_DT_E2M1) ? 4.0 : 8.0;
  const double b_lo = code_bits + words * meta_bits / static_cast<double>(layout->group);
  const double b_hi = layout->hi_dtype == DAMP_DT_FP32 ? 32.0 : 16.0;
  return b_lo + (static_cast<double>(layout->k_hi) / layout->d_k) * (b_hi - b_lo);
}

size_t damp_pool_required_bytes(const damp_layout* layout, int32_t num_layers,
                                int32_t num_slots, int32_t num_v_heads) {
  TileGeom g;
  if (!tile_geom(layout, &g) || num_layers <= 0 || num_slots <= 0 || num_v_heads <= 0) return 0;
  return g.stride * static_cast<size_t>(num_layers) * static_cast<size_t>(num_slots) *
         static_cast<size_t>(num_v_heads);
}

damp_status damp_check_slots(const damp_pool* pool, const int32_t* slot_idx, int32_t B,
                             int32_t on_device, void* stream) {
  clear_error();
  damp_status st = check_pool(pool);
  if (st != DAMP_OK) return st;
  if (B < 0) return fail(DAMP_ERR_INVALID_ARG, "damp_check_slots: B = %d is negative", B);
  if (B > 0 && !slot_idx) return fail(DAMP_ERR_INVALID_ARG, "damp_check_slots: slot_idx is NULL");
  return check_slots(pool, slot_idx, B, on_device != 0, as_stream(stream), "damp_check_slots");
}

damp_status damp_pool_init(damp_pool* pool, const damp_layout* layout, int32_t num_layers,
                           int32_t num_slots, int32_t num_v_heads, void* base, size_t bytes) {
  clear_error();
  if (!pool) return fail(DAMP_ERR_INVALID_ARG, "pool is NULL");
  TileGeom g;
  if (!tile_geom(layout, &g)) return DAMP_ERR_INVALID_ARG;
  if (!base) return fail(DAMP_ERR_INVALID_ARG, "base is NULL");
  if (reinterpret_cast<uintptr_t>(base) % 256 != 0)
    return fail(DAMP_ERR_INVALID_ARG, "base is not 256-byte aligned");
  const size_t need = damp_pool_required_bytes(layout, num_layers, num_slots, num_v_heads);
  if (need == 0) return fail(DAMP_ERR_INVALID_ARG, "pool counts must be positive");
  if (bytes < need)
    return fail(DAMP_ERR_INVALID_ARG, "%zu bytes given, pool needs %zu", bytes, need);
  std::memset(pool, 0, sizeof *pool);
  pool->layout = *layout;
  pool->num_layers = num_layers;
  pool->num_slots = num_slots;
  pool->num_v_heads = num_v_heads;
  pool->base = base;
  pool->tile_stride = g.stride;
  pool->bytes = need;
  return DAMP_OK;
}

}  // extern "C"
