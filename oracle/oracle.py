"""CPU oracle of DAMP's decode-step state update (arXiv 2608.27513).

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import this module; the product path
(``paper_2608_27513_amd``) never does, and this module imports nothing from
it. The arithmetic lives in ``damp_oracle.c`` (plain fp32 C, see its header
for the precision and the readings taken); this file builds it with gcc and
marshals numpy arrays. It also keeps its own description of the packed pool
(tile offsets, stride), written independently of the library's.

Every function cites the passage it follows:
  update      section 3.1 Eq. (1)-(2); section 3.2; App. A.5 (fused executor)
  prefill     App. A.5 (prefill path); section 3.1 Eq. (1)
  quant_row   section 3.2 Eq. (3); App. A.1 (integer formats)
  pack/unpack section 5.2; App. A.5 Eq. (17); App. A.1 (storage formats)
  select      section 5.1 Eq. (8)-(10); App. A.2 Eq. (13)-(15); Alg. 1
  bits        section 5.1 Eq. (7); App. A.1 Eq. (12) and the format table
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "damp_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

KIND_FP32 = 0
KIND_MIXED = 1

# Storage formats (high-tier type, values per metadata group, metadata type,
# Hadamard[, code type]): types 1 = BF16, 2 = FP16, 0 = FP32, 5 = E4M3; code
# types 3 = UINT8 (the default when omitted), 4 = UINT4, 5 = E4M3, 6 = E2M1.
# None is the default format: BF16 high tier, one fp32 (s, z) pair per row,
# no transform. The others are rows of App. A.1's format table, each with an
# FP16 high tier.
FMT_PAPER = (2, 32, 2, 1)        # INT8 + H32, FP16 (s, z) per 32 (the paper's layout)
FMT_PAPER_PLAIN = (2, 32, 2, 0)  # INT8, FP16 (s, z) per 32
FMT_INT4_H32 = (2, 32, 2, 1, 4)  # INT4 + H32, FP16 (s, z) per 32
FMT_INT4 = (2, 32, 2, 0, 4)      # INT4, FP16 (s, z) per 32
FMT_FP8 = (2, 32, 0, 0, 5)       # E4M3 codes, one fp32 scale per 32 (Eq. (16))
FMT_NVFP4 = (2, 16, 5, 0, 6)     # E2M1 codes, E4M3 scale per 16, fp32 scale per tile
CODE_U8, CODE_U4, CODE_E4M3, CODE_E2M1 = 3, 4, 5, 6

_lib = None


def build(force: bool = False) -> str:
    """Compile damp_oracle.c into liboracle.so (gcc, fp32, no contraction)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp"
        cmd = ["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC",
               "-shared", "-std=c11", SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB)
    return LIB


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = ctypes.CDLL(LIB)
        vp, i32, i64, f32, f64 = (ctypes.c_void_p, ctypes.c_int, ctypes.c_int64,
                                  ctypes.c_float, ctypes.c_double)
        L.orc_max_threads.restype = i32
        L.orc_bf16_round.argtypes = [vp, vp, i64]
        L.orc_bf16_widen.argtypes = [vp, vp, i64]
        L.orc_fp16_round.argtypes = [vp, vp, i64]
        L.orc_fp16_widen.argtypes = [vp, vp, i64]
        L.orc_hadamard32.argtypes = [vp, vp]
        L.orc_quant_group_fp16.argtypes = [vp, i32, vp, vp, vp]
        L.orc_quant_group_fp16_u4.argtypes = [vp, i32, vp, vp, vp]
        L.orc_quant_group_e4m3.argtypes = [vp, i32, vp, vp]
        L.orc_quant_block_e2m1.argtypes = [vp, i32, f32, vp]
        L.orc_quant_block_e2m1.restype = ctypes.c_uint8
        L.orc_nvfp4_global.argtypes = [f32]
        L.orc_nvfp4_global.restype = f32
        for nm in ("orc_e4m3_round", "orc_e4m3_widen", "orc_e2m1_round", "orc_e2m1_widen"):
            getattr(L, nm).argtypes = [vp, vp, i64]
        L.orc_quant_params.argtypes = [vp, i32, vp, vp]
        L.orc_quant_row.argtypes = [vp, i32, vp, vp, vp]
        L.orc_dequant_row.argtypes = [vp, i32, f32, f32, vp]
        L.orc_tile_bytes.argtypes = [i32, vp, i32, i32, i32]
        L.orc_tile_bytes.restype = i64
        L.orc_bits_per_value.argtypes = [i32, i32, i32, i32, i32, i32]
        L.orc_bits_per_value.restype = f64
        L.orc_pack.argtypes = [i32, vp, i32, i32, i32, vp, i64, i64, i32, vp, i32, i32, vp, vp]
        L.orc_unpack.argtypes = [i32, vp, i32, i32, i32, vp, i64, i64, i32, vp, i32, i32, vp, vp]
        L.orc_update.argtypes = [i32, i32, vp, i32, i32, i32, vp, i64, i64, i32, vp, i32, i32,
                                 i32, vp, vp, vp, vp, vp, vp, f32, vp, vp]
        L.orc_reset.argtypes = [i32, vp, i32, i32, i32, vp, i64, i64, i32, vp, i32, i32]
        L.orc_prefill.argtypes = [i32, i32, vp, i32, i32, i32, vp, i64, i64, i32, vp, i32, i32,
                                  i32, i32, vp, vp, vp, vp, vp, vp, f32, vp]
        L.orc_select.argtypes = [i32, i32, i32, i32, i32, vp, vp, i32, f64, vp, vp, vp, vp, vp]
        L.orc_select.restype = i32
        L.orc_calib_accumulate.argtypes = [i32, vp, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp]
        L.orc_calib_finalize.argtypes = [i32, i32, i32, vp, vp, i32, i32, f64, vp, vp, vp, vp, vp]
        L.orc_calib_finalize.restype = i32
        _lib = L
    return _lib


def max_threads() -> int:
    """Threads the oracle's OpenMP loops use."""
    return int(lib().orc_max_threads())


# ------------------------------------------------------------------ formats

def bf16_round(x) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round-to-nearest-even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, np.uint16)
    lib().orc_bf16_round(_p(x), _p(out), x.size)
    return out


def bf16_widen(u) -> np.ndarray:
    u = np.ascontiguousarray(u, dtype=np.uint16)
    out = np.empty(u.shape, np.float32)
    lib().orc_bf16_widen(_p(u), _p(out), u.size)
    return out


def fp16_round(x) -> np.ndarray:
    """fp32 -> IEEE binary16 bit patterns, round-to-nearest-even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, np.uint16)
    lib().orc_fp16_round(_p(x), _p(out), x.size)
    return out


def fp16_widen(u) -> np.ndarray:
    u = np.ascontiguousarray(u, dtype=np.uint16)
    out = np.empty(u.shape, np.float32)
    lib().orc_fp16_widen(_p(u), _p(out), u.size)
    return out


def hadamard32(x) -> np.ndarray:
    """Normalized block-32 Hadamard transform of one group (App. A.1)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    assert x.shape == (32,)
    y = np.empty(32, np.float32)
    lib().orc_hadamard32(_p(x), _p(y))
    return y


def quant_group_fp16(x):
    """Eq. (3) on one group with FP16 metadata (App. A.1): (codes, s, z), with
    s and z the stored FP16 values widened to fp32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    codes = np.empty(x.shape, np.uint8)
    s = ctypes.c_float()
    z = ctypes.c_float()
    lib().orc_quant_group_fp16(_p(x), x.size, _p(codes), ctypes.byref(s), ctypes.byref(z))
    return codes, np.float32(s.value), np.float32(z.value)


def fmt5(fmt):
    """The five-field form of a format (code type UINT8 when omitted)."""
    return None if fmt is None else (tuple(fmt) + (CODE_U8,))[:5]


def _fmt_arr(fmt):
    if fmt is None:
        return None
    hi, group, meta, had, code = fmt5(fmt)
    assert hi in (1, 2) and group > 0
    assert (code, meta, group) in ((CODE_U8, 0, group), (CODE_U8, 2, group), (CODE_U4, 2, 32),
                                   (CODE_E4M3, 0, 32), (CODE_E2M1, 5, 16))
    assert not had or (group == 32 and code in (CODE_U8, CODE_U4))
    return np.ascontiguousarray(fmt5(fmt), dtype=np.int32)


def e4m3_round(x) -> np.ndarray:
    """fp32 -> OCP E4M3 (FN) codes, round to nearest even, saturating."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, np.uint8)
    lib().orc_e4m3_round(_p(x), _p(out), x.size)
    return out


def e4m3_widen(c) -> np.ndarray:
    c = np.ascontiguousarray(c, dtype=np.uint8)
    out = np.empty(c.shape, np.float32)
    lib().orc_e4m3_widen(_p(c), _p(out), c.size)
    return out


def e2m1_round(x) -> np.ndarray:
    """fp32 -> E2M1 codes (sign in bit 3), round to nearest even, saturating."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, np.uint8)
    lib().orc_e2m1_round(_p(x), _p(out), x.size)
    return out


def e2m1_widen(c) -> np.ndarray:
    c = np.ascontiguousarray(c, dtype=np.uint8)
    out = np.empty(c.shape, np.float32)
    lib().orc_e2m1_widen(_p(c), _p(out), c.size)
    return out


def quant_group_fp16_u4(x):
    """INT4 (App. A.1) on one group with FP16 (s, z): (codes, s, z)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    codes = np.empty(x.shape, np.uint8)
    s, z = ctypes.c_float(), ctypes.c_float()
    lib().orc_quant_group_fp16_u4(_p(x), x.size, _p(codes), ctypes.byref(s), ctypes.byref(z))
    return codes, np.float32(s.value), np.float32(z.value)


def quant_group_e4m3(x):
    """FP8 of Eq. (16) on one group: (E4M3 codes, fp32 s)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    codes = np.empty(x.shape, np.uint8)
    s = ctypes.c_float()
    lib().orc_quant_group_e4m3(_p(x), x.size, _p(codes), ctypes.byref(s))
    return codes, np.float32(s.value)


def nvfp4_global(amax: float) -> np.float32:
    return np.float32(lib().orc_nvfp4_global(ctypes.c_float(amax)))


def quant_block_e2m1(x, s_g):
    """One NVFP4 block: (E2M1 codes, E4M3 block-scale code)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    codes = np.empty(x.shape, np.uint8)
    sb = lib().orc_quant_block_e2m1(_p(x), x.size, ctypes.c_float(s_g), _p(codes))
    return codes, np.uint8(sb)


def quant_row(x):
    """Eq. (3) on one row: returns (codes uint8, s, z)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    codes = np.empty(x.shape, np.uint8)
    s = ctypes.c_float()
    z = ctypes.c_float()
    lib().orc_quant_row(_p(x), x.size, _p(codes), ctypes.byref(s), ctypes.byref(z))
    return codes, np.float32(s.value), np.float32(z.value)


def dequant_row(codes, s, z) -> np.ndarray:
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    out = np.empty(codes.shape, np.float32)
    lib().orc_dequant_row(_p(codes), codes.size, float(s), float(z), _p(out))
    return out


def qdq_row(x) -> np.ndarray:
    """Q(x) = dequant(quant(x)) for one row."""
    c, s, z = quant_row(x)
    return dequant_row(c, s, z)


# ------------------------------------------------------------------- layout

def tile_bytes(kind: int, dk: int, dv: int, k_hi: int, fmt=None) -> int:
    f = _fmt_arr(fmt)
    if f is not None:
        assert dv % fmt[1] == 0
    return int(lib().orc_tile_bytes(kind, _p(f), dk, dv, k_hi))


def tile_stride(kind: int, dk: int, dv: int, k_hi: int, fmt=None) -> int:
    tb = tile_bytes(kind, dk, dv, k_hi, fmt)
    return (tb + 127) // 128 * 128


def bits_per_value(dk: int, k_hi: int, hi_bits: int = 16, code_bits: int = 8,
                   group: int = 32, meta_bits: int = 16) -> float:
    return float(lib().orc_bits_per_value(dk, k_hi, hi_bits, code_bits, group, meta_bits))


class Pool:
    """Host byte image of a slot-indexed pool, laid out as the library's."""

    def __init__(self, kind: int, dk: int, dv: int, k_hi: int, num_layers: int,
                 num_slots: int, num_v_heads: int, fmt=None):
        self.kind, self.dk, self.dv, self.k_hi = kind, dk, dv, k_hi
        self.num_layers, self.num_slots, self.hv = num_layers, num_slots, num_v_heads
        self.fmt = None if kind == KIND_FP32 else fmt
        self._fmt = _fmt_arr(self.fmt)
        self.tile_stride = tile_stride(kind, dk, dv, k_hi, self.fmt)
        self.slot_stride = self.tile_stride * num_v_heads
        self.layer_stride = self.slot_stride * num_slots
        self.buf = np.zeros(self.layer_stride * num_layers, np.uint8)

    def layer_ptr(self, layer: int):
        return ctypes.c_void_p(self.buf.ctypes.data + layer * self.layer_stride)

    def tile(self, layer: int, slot: int, head: int) -> np.ndarray:
        o = layer * self.layer_stride + slot * self.slot_stride + head * self.tile_stride
        return self.buf[o:o + tile_bytes(self.kind, self.dk, self.dv, self.k_hi, self.fmt)]

    def copy(self) -> "Pool":
        c = Pool.__new__(Pool)
        c.__dict__.update(self.__dict__)
        c.buf = self.buf.copy()
        return c


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def pack(pool: Pool, layer: int, slot_idx, S, perm=None) -> None:
    """Natural-order fp32 states [B, HV, dk, dv] -> tiles (Eq. (17))."""
    slot_idx = _i32(slot_idx)
    S = np.ascontiguousarray(S, dtype=np.float32)
    perm = None if perm is None else np.ascontiguousarray(perm, dtype=np.uint8)
    B = slot_idx.size
    assert S.shape == (B, pool.hv, pool.dk, pool.dv)
    lib().orc_pack(pool.kind, _p(pool._fmt), pool.dk, pool.dv, pool.k_hi, pool.layer_ptr(layer),
                   pool.slot_stride, pool.tile_stride, pool.num_slots, _p(slot_idx), B,
                   pool.hv, _p(S), _p(perm))


def unpack(pool: Pool, layer: int, slot_idx, perm=None) -> np.ndarray:
    slot_idx = _i32(slot_idx)
    perm = None if perm is None else np.ascontiguousarray(perm, dtype=np.uint8)
    B = slot_idx.size
    S = np.empty((B, pool.hv, pool.dk, pool.dv), np.float32)
    lib().orc_unpack(pool.kind, _p(pool._fmt), pool.dk, pool.dv, pool.k_hi, pool.layer_ptr(layer),
                     pool.slot_stride, pool.tile_stride, pool.num_slots, _p(slot_idx), B,
                     pool.hv, _p(perm), _p(S))
    return S


def reset(pool: Pool, layer: int, slots) -> None:
    slots = _i32(slots)
    layers = range(pool.num_layers) if layer < 0 else [layer]
    for l in layers:
        lib().orc_reset(pool.kind, _p(pool._fmt), pool.dk, pool.dv, pool.k_hi, pool.layer_ptr(l),
                        pool.slot_stride, pool.tile_stride, pool.num_slots, _p(slots),
                        slots.size, pool.hv)


def update(pool: Pool, layer: int, slot_idx, *, kda: bool, q, k, v, g, beta, perm=None,
           scale: float = 1.0, want_pre: bool = False):
    """One decode step (Eq. (1)) on every listed slot, in place.

    q, k: bf16 bits [B, HK, dk]; v: [B, HV, dv]; g: [B, HV] (GDN) or
    [B, HV, dk] (KDA); beta: [B, HV]. Returns o fp32 [B, HV, dv] (and the
    pre-quantization state in tile-row order if want_pre)."""
    slot_idx = _i32(slot_idx)
    B = slot_idx.size
    u16 = lambda a: np.ascontiguousarray(a, dtype=np.uint16)
    q, k, v, g, beta = u16(q), u16(k), u16(v), u16(g), u16(beta)
    HK = q.shape[1]
    assert q.shape == (B, HK, pool.dk) and k.shape == q.shape
    assert v.shape == (B, pool.hv, pool.dv) and beta.shape == (B, pool.hv)
    assert g.shape == ((B, pool.hv, pool.dk) if kda else (B, pool.hv))
    assert pool.hv % HK == 0
    perm = None if perm is None else np.ascontiguousarray(perm, dtype=np.uint8)
    o = np.empty((B, pool.hv, pool.dv), np.float32)
    pre = np.empty((B, pool.hv, pool.dk, pool.dv), np.float32) if want_pre else None
    lib().orc_update(int(kda), pool.kind, _p(pool._fmt), pool.dk, pool.dv, pool.k_hi,
                     pool.layer_ptr(layer),
                     pool.slot_stride, pool.tile_stride, pool.num_slots, _p(slot_idx), B, HK,
                     pool.hv, _p(q), _p(k), _p(v), _p(g), _p(beta), _p(perm), float(scale),
                     _p(o), _p(pre))
    return (o, pre) if want_pre else o


def prefill(pool: Pool, layer: int, slot_idx, *, kda: bool, q, k, v, g, beta, perm=None,
            scale: float = 1.0):
    """One chunk of T tokens per request (App. A.5, prefill path), in place:
    decode once, T fp32 steps of Eq. (1), encode once. q, k: bf16 bits
    [B, T, HK, dk]; v: [B, T, HV, dv]; g: [B, T, HV] (GDN) or [B, T, HV, dk]
    (KDA); beta: [B, T, HV]. Returns o fp32 [B, T, HV, dv]."""
    slot_idx = _i32(slot_idx)
    B = slot_idx.size
    u16 = lambda a: np.ascontiguousarray(a, dtype=np.uint16)
    q, k, v, g, beta = u16(q), u16(k), u16(v), u16(g), u16(beta)
    T, HK = q.shape[1], q.shape[2]
    assert q.shape == (B, T, HK, pool.dk) and k.shape == q.shape
    assert v.shape == (B, T, pool.hv, pool.dv) and beta.shape == (B, T, pool.hv)
    assert g.shape == ((B, T, pool.hv, pool.dk) if kda else (B, T, pool.hv))
    assert pool.hv % HK == 0
    perm = None if perm is None else np.ascontiguousarray(perm, dtype=np.uint8)
    o = np.empty((B, T, pool.hv, pool.dv), np.float32)
    lib().orc_prefill(int(kda), pool.kind, _p(pool._fmt), pool.dk, pool.dv, pool.k_hi,
                      pool.layer_ptr(layer), pool.slot_stride, pool.tile_stride, pool.num_slots,
                      _p(slot_idx), B, T, HK, pool.hv, _p(q), _p(k), _p(v), _p(g), _p(beta),
                      _p(perm), float(scale), _p(o))
    return o


def select(*, kda: bool, states, log_decay, k_hi: int, tau: float = 1e-4) -> dict:
    """Alg. 1 with App. A.2's estimates. states fp32 [N, H, dk, dv]."""
    states = np.ascontiguousarray(states, dtype=np.float32)
    log_decay = np.ascontiguousarray(log_decay, dtype=np.float32)
    N, H, dk, dv = states.shape
    assert log_decay.shape == ((N, H, dk) if kda else (N, H))
    sel = np.zeros((H, k_hi), np.int32)
    perm = np.zeros((H, dk), np.uint8)
    E = np.zeros((H, dk))
    P = np.zeros((H, dk))
    C = np.zeros((H, dk))
    rc = lib().orc_select(int(kda), N, H, dk, dv, _p(states), _p(log_decay), k_hi,
                          float(tau), _p(sel), _p(perm), _p(E), _p(P), _p(C))
    if rc != 0:
        raise ValueError("orc_select rejected its arguments")
    return dict(sel=sel, perm=perm, E=E, P=P, C=C)


def run_fp32(S0, *, kda: bool, q, k, v, g, beta, scale: float = 1.0, sample_every: int = 0):
    """FP32-state reference trajectory (natural channel order) over T steps.

    S0: fp32 [B, HV, dk, dv]; step inputs carry a leading T axis. Returns the
    final state, the outputs [T, B, HV, dv] and, if sample_every > 0, the
    states after steps sample_every, 2*sample_every, ... (the calibration
    state writes of App. A.2)."""
    T = q.shape[0]
    B, HV, dk, dv = S0.shape
    pool = Pool(KIND_FP32, dk, dv, 0, 1, B, HV)
    slots = np.arange(B, dtype=np.int32)
    pool.buf.view(np.float32)[:] = np.ascontiguousarray(S0, np.float32).reshape(-1)
    outs, samples = [], []
    for t in range(T):
        outs.append(update(pool, 0, slots, kda=kda, q=q[t], k=k[t], v=v[t], g=g[t],
                           beta=beta[t], scale=scale))
        if sample_every and (t + 1) % sample_every == 0:
            samples.append(pool.buf.view(np.float32).reshape(B, HV, dk, dv).copy())
    S = pool.buf.view(np.float32).reshape(B, HV, dk, dv).copy()
    return S, np.stack(outs), (np.stack(samples) if samples else None)


# ------------------------------------------------------------- calibration

SEL_DAMP, SEL_ERROR, SEL_PERSISTENCE, SEL_STATE_ENERGY, SEL_RANDOM = 0, 1, 2, 3, 4


class Calib:
    """Accumulators of App. A.2 over sampled state writes, one set per
    calibration domain: err, en, loga [D, H, dk] (Eq. (14), the state-energy
    selector's squared row norms, Eq. (15)) and sample counts [D]. fmt names
    Q_lo's low tier as for Pool (None: one fp32 (s, z) per row)."""

    def __init__(self, *, kda: bool, H: int, dk: int, dv: int, num_domains: int = 1, fmt=None):
        if fmt is not None and fmt5(fmt)[4] != CODE_U8:
            raise ValueError("calibration takes the UINT8 low tiers")
        self.kda, self.H, self.dk, self.dv, self.fmt = kda, H, dk, dv, fmt
        self.sums = np.zeros((num_domains, 3, H, dk))
        self.counts = np.zeros(num_domains)

    def accumulate(self, domain: int, states, g) -> None:
        """states fp32 [B, H, dk, dv] in natural channel order; g bf16 bits of
        the sampled token's log-decay, [B, H] (GDN) or [B, H, dk] (KDA)."""
        states = np.ascontiguousarray(states, dtype=np.float32)
        g = np.ascontiguousarray(g, dtype=np.uint16)
        B = states.shape[0]
        assert states.shape == (B, self.H, self.dk, self.dv)
        assert g.shape == ((B, self.H, self.dk) if self.kda else (B, self.H))
        s = self.sums[domain]
        err, en, loga = (np.ascontiguousarray(s[i]) for i in range(3))
        cnt = np.array([self.counts[domain]])
        lib().orc_calib_accumulate(int(self.kda), _p(_fmt_arr(self.fmt)), B, self.H, self.dk,
                                   self.dv, _p(states), _p(g), _p(err), _p(en), _p(loga),
                                   _p(cnt))
        s[0], s[1], s[2] = err, en, loga
        self.counts[domain] = cnt[0]

    def finalize(self, k_hi: int, selector: int = SEL_DAMP, tau: float = 1e-4,
                 rand_scores=None) -> dict:
        """Alg. 1 from the domain-balanced estimates (Eq. (13)-(15))."""
        D, H, dk = self.sums.shape[0], self.H, self.dk
        sums = np.ascontiguousarray(self.sums)
        counts = np.ascontiguousarray(self.counts)
        rs = None if rand_scores is None else np.ascontiguousarray(rand_scores, np.float64)
        sel = np.zeros((H, k_hi), np.int32)
        perm = np.zeros((H, dk), np.uint8)
        score = np.zeros((H, dk))
        stats = np.zeros((4, H, dk))
        rc = lib().orc_calib_finalize(D, H, dk, _p(sums), _p(counts), selector, k_hi, float(tau),
                                      _p(rs), _p(sel), _p(perm), _p(score), _p(stats))
        if rc != 0:
            raise ValueError("orc_calib_finalize rejected its arguments")
        return dict(sel=sel, perm=perm, score=score, E=stats[0], P=stats[1], energy=stats[2],
                    mean_log_a=stats[3])


def calibrate_sequence(calib: Calib, domain: int, S0, *, stride: int, q, k, v, g, beta):
    """The FP32 reference trajectory from S0 (natural order, [B, H, dk, dv])
    over step-major inputs [T, B, ...], with the state write after every
    `stride` tokens accumulated (App. A.3). Returns the final state."""
    S, _, samples = run_fp32(S0, kda=calib.kda, q=q, k=k, v=v, g=g, beta=beta,
                             sample_every=stride)
    if samples is not None:
        for n in range(samples.shape[0]):
            calib.accumulate(domain, samples[n], g[(n + 1) * stride - 1])
    return S


def topk_overlap(sel_a, sel_b) -> float:
    """|A intersect B| / k (App. B, calibration-split agreement)."""
    a, b = np.asarray(sel_a).ravel(), np.asarray(sel_b).ravel()
    return len(set(a.tolist()) & set(b.tolist())) / float(len(a))


def spearman(a, b) -> float:
    """Spearman rank correlation: Pearson correlation of the average ranks."""
    def ranks(x):
        x = np.asarray(x, dtype=np.float64)
        order = np.argsort(x, kind="stable")
        r = np.empty(len(x))
        i = 0
        while i < len(x):
            j = i
            while j + 1 < len(x) and x[order[j + 1]] == x[order[i]]:
                j += 1
            r[order[i:j + 1]] = (i + j) / 2.0 + 1.0
            i = j + 1
        return r
    ra, rb = ranks(a), ranks(b)
    ra -= ra.mean()
    rb -= rb.mean()
    den = np.sqrt((ra * ra).sum() * (rb * rb).sum())
    return float((ra * rb).sum() / den) if den > 0 else float("nan")
