/*
 * damp.h - C ABI of libdamp: the decode-step recurrent-state update of Gated
 * DeltaNet (GDN) and Kimi Delta Attention (KDA) over a mixed-precision state,
 * as described in "DAMP: Decay-Aware Mixed-Precision Recurrent-State
 * Quantization" (arXiv 2608.27513), on AMD Instinct MI355X (gfx950).
 *
 * Conventions shared by every call below
 * --------------------------------------
 *  - Pointers are DEVICE pointers unless the argument comment says "host".
 *  - bf16 tensors are passed as uint16_t bit patterns.
 *  - Every tensor is owned by the caller. The library never keeps a pointer
 *    after a call returns and allocates device memory only inside
 *    damp_select_channels (freed before it returns).
 *  - Calls taking `stream` (a hipStream_t passed as void*, NULL = the null
 *    stream) only enqueue work and return without synchronising, except
 *    damp_select_channels and damp_calib_finalize, which synchronise
 *    `stream`.
 *  - Arguments are validated on the host before anything is enqueued. A
 *    failed validation returns DAMP_ERR_INVALID_ARG (or DAMP_ERR_UNSUPPORTED
 *    for a valid layout that has no kernel) and touches no memory; the
 *    message is available from damp_last_error() on the calling thread.
 *    HIP launch failures return DAMP_ERR_HIP.
 *  - State values must be finite. A row whose values span more than
 *    ~3e38 is outside the quantizer's domain.
 *
 * State orientation (paper section 3.1): one head's state S has d_k rows
 * (key channels u) and d_v columns. The read-out is o = S^T q.
 *
 * Packed tile (paper section 5.2 and App. A.5, Eq. (17)): one tile holds the
 * state of one (layer, request slot, value head). Its rows are in the
 * calibrated order pi: tile row r holds key channel pi[r]; rows 0..k_hi-1
 * are the protected channels. Bytes, in order:
 *
 *   DAMP_STATE_MIXED, default tiers (damp_layout_init):
 *     [hi]   k_hi x d_v bf16, row-major
 *     [code] (d_k - k_hi) x d_v uint8 codes, row-major
 *     [meta] (d_k - k_hi) x {s, z} fp32 (8 bytes per low-tier row)
 *   DAMP_STATE_MIXED, the paper's tiers (App. A.1 format table; set
 *   hi_dtype = meta_dtype = DAMP_DT_FP16, group = 32, hadamard = 0 or 1):
 *     [hi]   k_hi x d_v FP16, row-major
 *     [code] (d_k - k_hi) x d_v uint8 codes, row-major; with hadamard = 1
 *            the codes of each group of 32 are those of its normalized
 *            Hadamard transform
 *     [meta] (d_k - k_hi) x (d_v / 32) x {s, z} FP16 (4 bytes per group)
 *   DAMP_STATE_MIXED, the other rows of App. A.1's format table (FP16 high
 *   tier, hi_dtype = DAMP_DT_FP16; d_v >= 32):
 *     INT4 (code_dtype = DAMP_DT_U4, group = 32, meta_dtype = DAMP_DT_FP16,
 *       hadamard = 0 or 1): [code] (d_k - k_hi) x d_v / 2 bytes, two codes
 *       per byte, the even column in the low nibble; [meta] as INT8.
 *     FP8 (code_dtype = DAMP_DT_E4M3, group = 32, meta_dtype = DAMP_DT_FP32,
 *       hadamard = 0): [code] (d_k - k_hi) x d_v E4M3 bytes; [meta]
 *       (d_k - k_hi) x (d_v / 32) fp32 scales.
 *     NVFP4 (code_dtype = DAMP_DT_E2M1, group = 16, meta_dtype =
 *       DAMP_DT_E4M3, hadamard = 0): [code] (d_k - k_hi) x d_v / 2 bytes as
 *       INT4; [meta] (d_k - k_hi) x (d_v / 16) E4M3 block scales; then one
 *       fp32 global scale for the tile's low tier.
 *   DAMP_STATE_FP32:
 *     d_k x d_v fp32, row-major
 *
 * A low-tier row x (d_v values) is stored with the asymmetric affine
 * quantizer of Eq. (3), one (s, z) pair per row:
 *     s = (max x - min x) / 255,  z = round(-min x / s),
 *     c = clamp(round(x / s) + z, 0, 255),  x_hat = s * (c - z),
 * with round = round-half-to-even. A row whose s is not a normal fp32 number
 * (a constant row) uses s = |min x| / 255, or s = 1 if that is not normal
 * either, so the all-zero row is stored as codes 0, s = 1, z = 0.
 * The paper's tiers apply the same rule per group of 32 values (after the
 * transform when hadamard = 1; the transform is y = H x / sqrt(32) with the
 * Sylvester matrix H, its own inverse), then round s to FP16 (kept within
 * [2^-24, 65504]), compute z = round(-min / s) from the stored s, round it
 * to FP16 (within +-65504), and code with the stored pair; reconstruction is
 * s * (c - z) followed by the inverse transform. INT4 is the same with 15
 * steps and codes in [0, 15].
 * FP8 (Eq. (16)): per group s = max(max |x|, 1e-10) / 448 (fp32), codes
 * E4M3(clip(x / s, -448, 448)) in the OCP E4M3 encoding (bias 7, largest
 * finite 448) rounded to nearest even; x_hat = s * q.
 * NVFP4: the tile's low tier has the global scale s_g = amax / 2688 (amax
 * its largest magnitude; 1 if amax is 0); each block of 16 the E4M3 scale
 * s_b = E4M3(min(block amax / (6 s_g), 448)); codes E2M1(x / (s_b s_g)) with
 * magnitudes {0, 0.5, 1, 1.5, 2, 3, 4, 6} (sign in bit 3), rounded to nearest
 * even and saturated at 6 (zero codes where s_b is 0); x_hat = q (s_b s_g).
 * The tile stride in a pool is the tile size rounded up to 128 bytes.
 */
#ifndef DAMP_H
#define DAMP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DAMP_OK = 0,
  DAMP_ERR_INVALID_ARG = 1, /* bad pointer, size or layout; nothing was touched */
  DAMP_ERR_UNSUPPORTED = 2, /* valid layout with no kernel instance */
  DAMP_ERR_HIP = 3          /* a HIP runtime call failed */
} damp_status;

typedef enum {
  DAMP_DT_FP32 = 0,
  DAMP_DT_BF16 = 1,
  DAMP_DT_FP16 = 2,
  DAMP_DT_U8 = 3,    /* low-tier codes: unsigned 8-bit (the default) */
  DAMP_DT_U4 = 4,    /* unsigned 4-bit, two per byte */
  DAMP_DT_E4M3 = 5,  /* OCP FP8 E4M3 (codes, or NVFP4 block scales) */
  DAMP_DT_E2M1 = 6   /* FP4 E2M1, two per byte */
} damp_dtype;

typedef enum {
  DAMP_STATE_FP32 = 0,  /* uncompressed state (the deployment baseline) */
  DAMP_STATE_MIXED = 1  /* k_hi bf16 rows + uint8 rows; k_hi = 0 is uniform INT8 */
} damp_state_kind;

/* Storage layout of one head's state (section 5.1, Eq. (7); section 5.2).
 * All fields are plain int32 so the struct has one fixed ABI. */
typedef struct {
  int32_t d_k;        /* key channels (rows) */
  int32_t d_v;        /* value channels (columns) */
  int32_t k_hi;       /* protected rows held in the high-precision tier */
  int32_t kind;       /* damp_state_kind */
  int32_t hi_dtype;   /* damp_dtype of the high tier (BF16, or FP16 with the paper's tiers) */
  int32_t group;      /* values per (s, z) pair along d_v; d_v = one per row */
  int32_t meta_dtype; /* damp_dtype of s and z (FP32 per row, or FP16 per group of 32) */
  int32_t hadamard;   /* 1 = block-32 Hadamard before quantization (paper's tiers) */
  int32_t code_dtype; /* damp_dtype of the low-tier codes: U8 (default), U4, E4M3, E2M1 */
} damp_layout;

/* Fills `out` with the default layout: BF16 high tier, one fp32 (s, z) pair
 * per low-tier row, UINT8 codes, no Hadamard. Kernels exist for d_k == d_v
 * in {16, 32, 64, 128}, and for the paper's tiers and the other formats
 * above (set the fields after this call) for d_k == d_v in {32, 64, 128};
 * other layouts are valid for the size queries but calls that move state
 * return DAMP_ERR_UNSUPPORTED. Returns DAMP_ERR_INVALID_ARG if
 * out is NULL, d_k or d_v is not positive, or k_hi is outside [0, d_k]. */
damp_status damp_layout_init(damp_layout* out, int32_t d_k, int32_t d_v,
                             int32_t k_hi, int32_t kind);

/* Bytes of one packed tile (the sum of its regions, before padding).
 * Returns 0 for an invalid layout. For d_k = d_v = 128, k_hi = 16 the default
 * mixed layout takes 19328 bytes; the FP32 layout takes 65536. */
size_t damp_tile_bytes(const damp_layout* layout);

/* Tile stride used inside a pool: damp_tile_bytes rounded up to 128. */
size_t damp_tile_stride(const damp_layout* layout);

/* Storage cost in bits per state value including metadata, following
 * Eq. (7): b = b_lo + (k_hi / d_k)(b_hi - b_lo), where b_lo counts the code
 * bits plus the (s, z) bits amortised over `group` values. Returns a
 * negative value for an invalid layout. The paper's operating point (FP16
 * high tier, 16 of 128 rows, INT8 with FP16 (s, z) per 32 values) gives the
 * 9.875 of Eq. (12). */
double damp_bits_per_value(const damp_layout* layout);

/* A slot-indexed state pool: tiles addressed as
 *   base + ((layer * num_slots + slot) * num_v_heads + head) * tile_stride.
 * Plain data; the memory at `base` belongs to the caller. */
typedef struct {
  damp_layout layout;
  int32_t num_layers;
  int32_t num_slots;
  int32_t num_v_heads;
  void* base;          /* device memory, 256-byte aligned */
  size_t tile_stride;  /* bytes */
  size_t bytes;        /* bytes the pool spans */
} damp_pool;

/* Bytes a pool of this shape spans (0 if an argument is invalid). */
size_t damp_pool_required_bytes(const damp_layout* layout, int32_t num_layers,
                                int32_t num_slots, int32_t num_v_heads);

/* Describes `bytes` of caller memory at `base` as a pool. Fails with
 * DAMP_ERR_INVALID_ARG if base is NULL or not 256-byte aligned, a count is
 * not positive, the layout is invalid, or `bytes` is smaller than
 * damp_pool_required_bytes. Writes nothing to device memory. */
damp_status damp_pool_init(damp_pool* pool, const damp_layout* layout,
                           int32_t num_layers, int32_t num_slots,
                           int32_t num_v_heads, void* base, size_t bytes);

/* Race check of a batch of slot ids. Every call that writes tiles
 * (update, prefill, pack, reset, calibration sequence) requires the slots of
 * its batch to be distinct: two requests sharing a slot would read and write
 * the same tiles concurrently. The kernels do not check this; this call
 * does. Entries outside [0, num_slots) are padding and are ignored.
 *  slot_idx   int32[B]; a HOST pointer when on_device is 0, else a device
 *             pointer that is copied to the host on `stream` (which is then
 *             synchronised).
 * Returns DAMP_ERR_INVALID_ARG naming the repeated slot, DAMP_OK otherwise.
 * Validation mode: with the environment variable DAMP_CHECK_SLOTS set to a
 * value other than "0", every call that writes tiles runs this check on its
 * device slot ids before enqueuing anything and fails the same way; each
 * such call then synchronises its stream (a debugging aid, not for capture
 * into a graph). */
damp_status damp_check_slots(const damp_pool* pool, const int32_t* slot_idx,
                             int32_t B, int32_t on_device, void* stream);

/* Writes the packed zero state into every head of `n` slots (for a new
 * request). `layer` selects one layer, or -1 for all layers. `slots` is a
 * device int32[n]; entries outside [0, num_slots) are skipped. */
damp_status damp_pool_reset_slots(const damp_pool* pool, int32_t layer,
                                  const int32_t* slots, int32_t n, void* stream);

/* One GDN decode step for one layer (section 3.1, Eq. (1)-(2), with the
 * state stored per section 5.2 / App. A.5), for B requests at once.
 *
 * For request b and value head h (key head hk = h / (HV / num_k_heads)):
 *   a      = exp(g[b,h])                          (scalar decay, Lambda = a I)
 *   S_bar  = a * S                                (decay first)
 *   delta  = v[b,h] - S_bar^T k~                  (delta-rule residual)
 *   S'     = S_bar + beta[b,h] * k~ delta^T       (Eq. (1))
 *   o[b,h] = scale * S'^T q~                      (read-out of the updated,
 *                                                  not yet re-quantized S')
 * then S' is re-encoded into the tile in place (bf16 rounding for the high
 * tier, Eq. (3) per low-tier row). k~[r] = k[b,hk,perm[h,r]] and likewise
 * for q: operands arrive in natural channel order and are permuted inside
 * the kernel.
 *
 *  pool       pool descriptor (host pointer); its layout picks the kernel.
 *  layer      layer index in [0, num_layers).
 *  slot_idx   int32[B]: the pool slot of each request. A slot outside
 *             [0, num_slots) marks a padded row: its state is untouched and
 *             its o is written as zeros. Two requests must not share a slot
 *             in one call (their tiles would race).
 *  B          requests (0 is a no-op).
 *  num_k_heads HK; num_v_heads of the pool (HV) must be a multiple of it.
 *  q, k       bf16 [B, HK, d_k], natural channel order (q already
 *             normalised as the model wants; `scale` multiplies o).
 *  v          bf16 [B, HV, d_v].
 *  g          bf16 [B, HV]: log-decay (log a); a = exp(g) is taken in fp32.
 *  beta       bf16 [B, HV]: delta-rule step size.
 *  perm       uint8 [HV, d_k] for this layer (tile row -> key channel), or
 *             NULL for the identity. Each row must be a permutation.
 *  o          [B, HV, d_v] in o_dtype (DAMP_DT_FP32 or DAMP_DT_BF16).
 */
damp_status damp_state_update_gdn(const damp_pool* pool, int32_t layer,
                                  const int32_t* slot_idx, int32_t B,
                                  int32_t num_k_heads, const uint16_t* q,
                                  const uint16_t* k, const uint16_t* v,
                                  const uint16_t* g, const uint16_t* beta,
                                  const uint8_t* perm, float scale, void* o,
                                  int32_t o_dtype, void* stream);

/* One KDA decode step: as damp_state_update_gdn, except that the decay is
 * per key channel, Lambda = diag(exp(g)) (section 3.1), so
 *   g is bf16 [B, HV, d_k] in natural channel order and row r of the tile
 *   decays by exp(g[b,h,perm[h,r]]),
 * and q, k are [B, num_k_heads, d_k] with num_k_heads = HV or a divisor. */
damp_status damp_state_update_kda(const damp_pool* pool, int32_t layer,
                                  const int32_t* slot_idx, int32_t B,
                                  int32_t num_k_heads, const uint16_t* q,
                                  const uint16_t* k, const uint16_t* v,
                                  const uint16_t* g, const uint16_t* beta,
                                  const uint8_t* perm, float scale, void* o,
                                  int32_t o_dtype, void* stream);

/* Prefill of one chunk of T tokens per request (App. A.5, prefill path): the
 * stored state of every (request, value head) is decoded once, the
 * recurrence of Eq. (1) runs in fp32 for the T tokens in order (o of each
 * token read from the state that token updated, as in the decode step), and
 * only the chunk-final state is stored back per the layout, so the chunk's
 * intermediate states are never quantized. Arguments as for
 * damp_state_update_gdn, with a token axis after the request axis:
 *  T          tokens per request in this chunk (0 is a no-op).
 *  q, k       bf16 [B, T, HK, d_k];  v  bf16 [B, T, HV, d_v];
 *  g          bf16 [B, T, HV] (GDN) or [B, T, HV, d_k] (KDA): log-decay;
 *  beta       bf16 [B, T, HV];  o  [B, T, HV, d_v] in o_dtype, 16-byte
 *             aligned.
 * A padded request (slot outside the pool) gets o = 0 for every token.
 * DAMP_ERR_INVALID_ARG also for T < 0 and for a misaligned o. */
damp_status damp_state_prefill_gdn(const damp_pool* pool, int32_t layer,
                                   const int32_t* slot_idx, int32_t B, int32_t T,
                                   int32_t num_k_heads, const uint16_t* q,
                                   const uint16_t* k, const uint16_t* v,
                                   const uint16_t* g, const uint16_t* beta,
                                   const uint8_t* perm, float scale, void* o,
                                   int32_t o_dtype, void* stream);

/* KDA prefill: as damp_state_prefill_gdn with the per-key-channel decay of
 * damp_state_update_kda (g is [B, T, HV, d_k]). */
damp_status damp_state_prefill_kda(const damp_pool* pool, int32_t layer,
                                   const int32_t* slot_idx, int32_t B, int32_t T,
                                   int32_t num_k_heads, const uint16_t* q,
                                   const uint16_t* k, const uint16_t* v,
                                   const uint16_t* g, const uint16_t* beta,
                                   const uint8_t* perm, float scale, void* o,
                                   int32_t o_dtype, void* stream);

/* Packs natural-order fp32 states into pool tiles (the persistent
 * representation of Eq. (17)): tile row r receives S[b,h,perm[h,r],:],
 * stored in the tier row r belongs to.
 *  S     fp32 [B, HV, d_k, d_v], natural channel order.
 *  perm  uint8 [HV, d_k] or NULL (identity).
 * Slots outside [0, num_slots) are skipped. */
damp_status damp_state_pack(const damp_pool* pool, int32_t layer,
                            const int32_t* slot_idx, int32_t B, const float* S,
                            const uint8_t* perm, void* stream);

/* Decodes pool tiles back to natural-order fp32 states:
 * S_out[b,h,perm[h,r],:] = decode(tile row r). Rows of a skipped slot (outside
 * [0, num_slots)) are written as zeros. */
damp_status damp_state_unpack(const damp_pool* pool, int32_t layer,
                              const int32_t* slot_idx, int32_t B,
                              const uint8_t* perm, float* S_out, void* stream);

/* Offline selection of the protected key channels of every head (section
 * 5.1, Eq. (8)-(10); App. A.2, Eq. (14)-(15); Alg. 1 in App. A.4).
 *
 * For each head h and key channel u, over the N calibration samples n:
 *   E_u   = mean_n || Q_lo(S_n[h,u,:]) - S_n[h,u,:] ||^2     (Eq. (8))
 *           with Q_lo the low tier of `lo` (App. A.2: the deployed storage
 *           mapping), evaluated with IEEE operations (exact division, no
 *           FMA), squared errors summed in double in ascending column order
 *           and samples summed in ascending n;
 *   a_eff = exp(mean_n log_a[n,h(,u)])                      (geometric mean)
 *   P_u   = 1 / max(1 - a_eff^2, tau)                       (Eq. (9))
 *   C_u   = E_u * P_u, and the k_hi largest C_u are kept    (Eq. (10)),
 *           ties broken towards the lower channel index.
 * perm_out[h] is the stable partition of Alg. 1: the kept channels in
 * ascending order, then the rest in ascending order.
 *
 *  is_kda     0: log_decay is [N, H] (one decay per head, GDN);
 *             1: log_decay is [N, H, d_k] (per key channel, KDA).
 *  states     fp32 [N, H, d_k, d_v] device: reference (FP32) states.
 *  log_decay  fp32 device, see is_kda.
 *  lo         host pointer to the layout whose low tier is Q_lo, or NULL for
 *             the per-row quantizer of the default tiers. Supported: a
 *             DAMP_STATE_MIXED layout with this d_k and d_v and the default
 *             low tier (one fp32 (s, z) per row), or the paper's UINT8 tier
 *             (groups of 32 with FP16 (s, z), hadamard 0 or 1; d_v <= 128
 *             and a multiple of 32). Its k_hi is not used. Other layouts
 *             return DAMP_ERR_UNSUPPORTED.
 *  k_hi       in [0, d_k]; tau > 0 (the paper uses 1e-4).
 *  sel_out    host int32 [H, k_hi], ascending per head.
 *  perm_out   host uint8 [H, d_k] (d_k <= 256).
 *  score_out  host double [H, d_k] receiving C_u, or NULL.
 * Allocates and frees (N + 2) * H * d_k doubles of device scratch;
 * synchronises `stream`. */
damp_status damp_select_channels(int32_t is_kda, int32_t N, int32_t H,
                                 int32_t d_k, int32_t d_v, const float* states,
                                 const float* log_decay, const damp_layout* lo,
                                 int32_t k_hi, double tau, int32_t* sel_out,
                                 uint8_t* perm_out, double* score_out,
                                 void* stream);

/* Bytes of the fixed device scratch of damp_select_channels_noalloc. */
#define DAMP_SELECT_NOALLOC_SCRATCH_BYTES (16 << 20)

/* damp_select_channels without any allocation, for callers that cannot
 * allocate memory (inside HIP graph capture, in tight serving loops, under
 * harnesses that forbid hipMalloc). Arguments, results and errors are those
 * of damp_select_channels, bit for bit; the device scratch is instead a fixed
 * array of DAMP_SELECT_NOALLOC_SCRATCH_BYTES inside the library, one per GPU,
 * which each GPU holds from its first call until the process ends (the host
 * side uses fixed buffers too). Limit: (N + 2) * H * d_k doubles must fit in
 * it, i.e. (N + 2) * H * d_k <= 2097152 (the KDA calibration of 256 samples
 * x 32 heads x 128 channels fits); larger calls return DAMP_ERR_INVALID_ARG
 * before anything runs. Every call on one GPU shares that GPU's array and
 * overwrites what the previous call left (nothing in it needs clearing: each
 * call writes every element it reads), so calls that overlap on one GPU,
 * from different streams or threads, race on it: serialize them.
 * Synchronises `stream`. */
damp_status damp_select_channels_noalloc(int32_t is_kda, int32_t N, int32_t H,
                                         int32_t d_k, int32_t d_v,
                                         const float* states,
                                         const float* log_decay,
                                         const damp_layout* lo, int32_t k_hi,
                                         double tau, int32_t* sel_out,
                                         uint8_t* perm_out, double* score_out,
                                         void* stream);

/* ------------------------------------------------------------------------
 * On-device calibration (App. A.2, Eq. (13)-(15); Alg. 1 in App. A.4; the
 * key-channel selector ablation of section 6; the calibration-split
 * agreement of App. B).
 *
 * The reference (FP32) trajectory runs in an FP32 pool; every sampled state
 * write is folded into double accumulators, one set per calibration domain,
 * for each head h and key channel u:
 *   err  += || Q_lo(S[h,u,:]) - S[h,u,:] ||^2     (Eq. (14))
 *   en   += || S[h,u,:] ||^2                      (the state-energy selector)
 *   loga += log a[h,u] of the sampled token       (Eq. (15))
 *   count += 1 per sampled request
 * Q_lo is the low tier of `lo` (default tiers: one fp32 (s, z) per row;
 * the paper's tiers: groups of 32 with FP16 (s, z), optionally after the
 * block-32 transform). Every sum runs in the order of its definition:
 * columns ascending within a row (IEEE operations, no contraction), samples
 * in the order they are accumulated. Finalization forms, per head and
 * channel, the domain-balanced mean of Eq. (13) (the mean over domains of
 * each domain's mean), a_eff = exp(mean log a), P = 1 / max(1 - a_eff^2,
 * tau) and the chosen selector's score, then keeps the k_hi largest scores
 * (ties to the lower channel) and returns the stable partition of Alg. 1.
 * ---------------------------------------------------------------------- */

#define DAMP_CALIB_MAX_DOMAINS 64

/* Selectors of the ablation in section 6: the product C = E P, the error
 * energy E alone, the persistence P alone, the mean squared key-channel
 * norm, or caller-supplied scores (Random: draw them uniformly). */
typedef enum {
  DAMP_SEL_DAMP = 0,
  DAMP_SEL_ERROR = 1,
  DAMP_SEL_PERSISTENCE = 2,
  DAMP_SEL_STATE_ENERGY = 3,
  DAMP_SEL_RANDOM = 4
} damp_selector;

/* Accumulator descriptor (plain data; filled by damp_calib_init). The
 * accumulators are caller-owned device memory: per domain d, three
 * [num_heads, d_k] double arrays (err, en, loga), followed by num_domains
 * double sample counts. */
typedef struct {
  damp_layout lo;       /* Q_lo is this layout's low tier; k_hi is not used */
  int32_t is_kda;       /* 1: log-decay per key channel (KDA); 0: per head */
  int32_t num_heads;
  int32_t num_domains;
  double* sums;         /* device */
  size_t bytes;
} damp_calib;

/* 8 * num_domains * (3 * num_heads * d_k + 1); 0 for non-positive sizes. */
size_t damp_calib_required_bytes(int32_t num_domains, int32_t num_heads,
                                 int32_t d_k);

/* Fills *calib and zeroes the accumulators (a fill kernel on `stream`).
 *  lo           a DAMP_STATE_MIXED layout with d_k == d_v <= 256 whose low
 *               tier has kernels (default or paper tiers; else
 *               DAMP_ERR_UNSUPPORTED).
 *  num_domains  in [1, DAMP_CALIB_MAX_DOMAINS].
 *  sums, bytes  device memory, 8-byte aligned, at least
 *               damp_calib_required_bytes(num_domains, num_heads, lo->d_k). */
damp_status damp_calib_init(damp_calib* calib, const damp_layout* lo,
                            int32_t is_kda, int32_t num_heads,
                            int32_t num_domains, void* sums, size_t bytes,
                            void* stream);

/* Adds one sampled state write of B requests to domain `domain`.
 *  pool      a DAMP_STATE_FP32 pool of the calibration trajectory with
 *            d_k, d_v and num_v_heads equal to the calib's.
 *  slot_idx  int32 [B]; requests whose slot is outside [0, num_slots) are
 *            skipped and not counted.
 *  perm      uint8 [num_heads, d_k]: tile row r holds key channel
 *            perm[h, r]; NULL = identity.
 *  g         bf16 log-decay of the sampled token: [B, num_heads] (GDN) or
 *            [B, num_heads, d_k] in natural channel order (KDA).
 * Calls on one calib must not overlap (they read and write the same
 * accumulators); they accumulate in call order. */
damp_status damp_calib_accumulate(const damp_calib* calib, int32_t domain,
                                  const damp_pool* pool, int32_t layer,
                                  const int32_t* slot_idx, int32_t B,
                                  const uint8_t* perm, const uint16_t* g,
                                  void* stream);

/* Runs a calibration sequence of T tokens for B requests on the FP32 pool
 * (its tiles hold the starting states in natural channel order, e.g. the
 * zero state after damp_pool_reset_slots) and samples every `stride`
 * tokens: after tokens stride, 2 stride, ... the state write is
 * accumulated into `domain`, with the log-decay of that token (App. A.3:
 * states sampled every eight tokens). A trailing partial stride is run but
 * not sampled. The recurrence is the prefill path's, `stride` tokens per
 * launch; no outputs are written. Inputs as for damp_state_prefill_gdn /
 * _kda (num_k_heads == num_heads for KDA). The pool holds the final states
 * afterwards. */
damp_status damp_calibrate_sequence(const damp_calib* calib, int32_t domain,
                                    const damp_pool* pool, int32_t layer,
                                    const int32_t* slot_idx, int32_t B,
                                    int32_t T, int32_t stride,
                                    int32_t num_k_heads, const uint16_t* q,
                                    const uint16_t* k, const uint16_t* v,
                                    const uint16_t* g, const uint16_t* beta,
                                    void* stream);

/* Selection from the accumulated statistics (Alg. 1). Synchronises `stream`.
 *  selector     a damp_selector.
 *  k_hi         in [0, d_k]; tau > 0 (the paper uses 1e-4).
 *  rand_scores  host double [num_heads, d_k] for DAMP_SEL_RANDOM, else
 *               unused.
 *  sel_out      host int32 [num_heads, k_hi], ascending per head.
 *  perm_out     host uint8 [num_heads, d_k].
 *  score_out    host double [num_heads, d_k]: the selector's score, or NULL.
 *  stats_out    host double [4, num_heads, d_k]: E, P, mean squared norm,
 *               mean log a; or NULL.
 * DAMP_ERR_INVALID_ARG if a domain has no samples. */
damp_status damp_calib_finalize(const damp_calib* calib, int32_t selector,
                                int32_t k_hi, double tau,
                                const double* rand_scores, int32_t* sel_out,
                                uint8_t* perm_out, double* score_out,
                                double* stats_out, void* stream);

/* Calibration-split agreement (App. B), host only. Top-k overlap
 * |A intersect B| / k of two selections of k distinct channels each; NaN for
 * NULL or k <= 0. */
double damp_topk_overlap(const int32_t* sel_a, const int32_t* sel_b,
                         int32_t k);

/* Spearman rank correlation of two score vectors of length n (ties get
 * their average rank; Pearson correlation of the ranks); NaN for n < 2, a
 * NULL pointer, or a constant vector. Host only. */
double damp_spearman(const double* a, const double* b, int32_t n);

/* Message describing the last failure on the calling thread ("" if none). */
const char* damp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DAMP_H */
