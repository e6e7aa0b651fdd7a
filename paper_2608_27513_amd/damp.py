"""Thin Python binding of libdamp (include/damp.h).

Argument marshalling only: every function checks tensor placement, dtype and
shape, passes raw device pointers and the current HIP stream to the C ABI of
the same name, and raises DampError on a non-zero status. All compute runs in
the HIP kernels of libdamp.so. There is no fallback: if the library is not
built, loading it raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdamp.so")

DAMP_OK, DAMP_ERR_INVALID_ARG, DAMP_ERR_UNSUPPORTED, DAMP_ERR_HIP = 0, 1, 2, 3
DAMP_DT_FP32, DAMP_DT_BF16, DAMP_DT_FP16 = 0, 1, 2
DAMP_DT_U8, DAMP_DT_U4, DAMP_DT_E4M3, DAMP_DT_E2M1 = 3, 4, 5, 6
DAMP_STATE_FP32, DAMP_STATE_MIXED = 0, 1
DAMP_SEL_DAMP, DAMP_SEL_ERROR, DAMP_SEL_PERSISTENCE, DAMP_SEL_STATE_ENERGY, DAMP_SEL_RANDOM = \
    0, 1, 2, 3, 4
DAMP_CALIB_MAX_DOMAINS = 64


class DampError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"damp status {status}: {message}")
        self.status = status


class damp_layout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("d_k", "d_v", "k_hi", "kind", "hi_dtype", "group", "meta_dtype", "hadamard",
                 "code_dtype")]


class damp_calib(ctypes.Structure):
    _fields_ = [("lo", damp_layout), ("is_kda", ctypes.c_int32), ("num_heads", ctypes.c_int32),
                ("num_domains", ctypes.c_int32), ("sums", ctypes.c_void_p),
                ("bytes", ctypes.c_size_t)]


class damp_pool(ctypes.Structure):
    _fields_ = [("layout", damp_layout), ("num_layers", ctypes.c_int32),
                ("num_slots", ctypes.c_int32), ("num_v_heads", ctypes.c_int32),
                ("base", ctypes.c_void_p),
                ("tile_stride", ctypes.c_size_t), ("bytes", ctypes.c_size_t)]


EXPORTS = ("damp_layout_init", "damp_tile_bytes", "damp_tile_stride", "damp_bits_per_value",
           "damp_pool_required_bytes", "damp_pool_init", "damp_check_slots", "damp_pool_reset_slots",
           "damp_state_update_gdn", "damp_state_update_kda", "damp_state_prefill_gdn",
           "damp_state_prefill_kda", "damp_state_pack", "damp_state_unpack",
           "damp_select_channels", "damp_select_channels_noalloc", "damp_calib_required_bytes", "damp_calib_init",
           "damp_calib_accumulate", "damp_calibrate_sequence", "damp_calib_finalize",
           "damp_topk_overlap", "damp_spearman", "damp_last_error")

_lib = None


def lib() -> ctypes.CDLL:
    """Loads libdamp.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2608_27513_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    P, i32, sz, f32, f64, st = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t,
                                ctypes.c_float, ctypes.c_double, ctypes.c_int)
    LP, PP = ctypes.POINTER(damp_layout), ctypes.POINTER(damp_pool)
    CP = ctypes.POINTER(damp_calib)
    sig = {
        "damp_layout_init": (st, [LP, i32, i32, i32, i32]),
        "damp_tile_bytes": (sz, [LP]),
        "damp_tile_stride": (sz, [LP]),
        "damp_bits_per_value": (f64, [LP]),
        "damp_pool_required_bytes": (sz, [LP, i32, i32, i32]),
        "damp_pool_init": (st, [PP, LP, i32, i32, i32, P, sz]),
        "damp_check_slots": (st, [PP, P, i32, i32, P]),
        "damp_pool_reset_slots": (st, [PP, i32, P, i32, P]),
        "damp_state_update_gdn": (st, [PP, i32, P, i32, i32, P, P, P, P, P, P, f32, P, i32, P]),
        "damp_state_update_kda": (st, [PP, i32, P, i32, i32, P, P, P, P, P, P, f32, P, i32, P]),
        "damp_state_prefill_gdn": (st, [PP, i32, P, i32, i32, i32, P, P, P, P, P, P, f32, P, i32,
                                        P]),
        "damp_state_prefill_kda": (st, [PP, i32, P, i32, i32, i32, P, P, P, P, P, P, f32, P, i32,
                                        P]),
        "damp_state_pack": (st, [PP, i32, P, i32, P, P, P]),
        "damp_state_unpack": (st, [PP, i32, P, i32, P, P, P]),
        "damp_select_channels": (st, [i32, i32, i32, i32, i32, P, P, LP, i32, f64, P, P, P, P]),
        "damp_select_channels_noalloc": (st, [i32, i32, i32, i32, i32, P, P, LP, i32, f64, P, P,
                                              P, P]),
        "damp_calib_required_bytes": (sz, [i32, i32, i32]),
        "damp_calib_init": (st, [CP, LP, i32, i32, i32, P, sz, P]),
        "damp_calib_accumulate": (st, [CP, i32, PP, i32, P, i32, P, P, P]),
        "damp_calibrate_sequence": (st, [CP, i32, PP, i32, P, i32, i32, i32, i32, P, P, P, P, P,
                                         P]),
        "damp_calib_finalize": (st, [CP, i32, i32, f64, P, P, P, P, P, P]),
        "damp_topk_overlap": (f64, [P, P, i32]),
        "damp_spearman": (f64, [P, P, i32]),
        "damp_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def _check(status: int) -> None:
    if status != DAMP_OK:
        raise DampError(status, lib().damp_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(t: torch.Tensor, dtype, name: str, shape=None) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t


# ------------------------------------------------------------------ layout

def damp_layout_init(d_k: int, d_v: int, k_hi: int, kind: int = DAMP_STATE_MIXED) -> damp_layout:
    L = damp_layout()
    _check(lib().damp_layout_init(ctypes.byref(L), d_k, d_v, k_hi, kind))
    return L


def damp_tile_bytes(layout: damp_layout) -> int:
    return int(lib().damp_tile_bytes(ctypes.byref(layout)))


def damp_tile_stride(layout: damp_layout) -> int:
    return int(lib().damp_tile_stride(ctypes.byref(layout)))


def damp_bits_per_value(layout: damp_layout) -> float:
    return float(lib().damp_bits_per_value(ctypes.byref(layout)))


def damp_pool_required_bytes(layout: damp_layout, num_layers: int, num_slots: int,
                             num_v_heads: int) -> int:
    return int(lib().damp_pool_required_bytes(ctypes.byref(layout), num_layers, num_slots,
                                              num_v_heads))


class Pool:
    """A slot-indexed state pool: a torch uint8 buffer on the GPU plus its
    damp_pool descriptor (keeps the buffer alive)."""

    def __init__(self, layout: damp_layout, num_layers: int, num_slots: int, num_v_heads: int,
                 device="cuda", buffer: torch.Tensor | None = None):
        need = damp_pool_required_bytes(layout, num_layers, num_slots, num_v_heads)
        if need == 0:
            raise ValueError("invalid pool shape")
        if buffer is None:
            buffer = torch.empty(need, dtype=torch.uint8, device=device)
        self.buffer = _dev(buffer, torch.uint8, "buffer")
        self.desc = damp_pool()
        _check(lib().damp_pool_init(ctypes.byref(self.desc), ctypes.byref(layout), num_layers,
                                    num_slots, num_v_heads, _ptr(self.buffer),
                                    self.buffer.numel()))
        self.layout = layout
        self.num_layers, self.num_slots, self.num_v_heads = num_layers, num_slots, num_v_heads
        self.tile_stride = int(self.desc.tile_stride)

    @property
    def d(self) -> int:
        return self.layout.d_k


def damp_pool_init(layout: damp_layout, num_layers: int, num_slots: int, num_v_heads: int,
                   buffer: torch.Tensor) -> Pool:
    return Pool(layout, num_layers, num_slots, num_v_heads, buffer=buffer)


def damp_check_slots(pool: Pool, slot_idx, stream=None) -> None:
    """Raises DampError (DAMP_ERR_INVALID_ARG) if a slot of the pool occurs
    twice in slot_idx (a device int32 tensor, or host ids)."""
    if isinstance(slot_idx, torch.Tensor) and slot_idx.device.type == "cuda":
        slot_idx = _dev(slot_idx, torch.int32, "slot_idx")
        _check(lib().damp_check_slots(ctypes.byref(pool.desc), _ptr(slot_idx), slot_idx.numel(), 1,
                                      _stream(stream)))
        return
    ids = (ctypes.c_int32 * len(slot_idx))(*[int(x) for x in slot_idx])
    _check(lib().damp_check_slots(ctypes.byref(pool.desc), ids, len(slot_idx), 0, None))


def damp_pool_reset_slots(pool: Pool, layer: int, slots: torch.Tensor, stream=None) -> None:
    slots = _dev(slots, torch.int32, "slots")
    _check(lib().damp_pool_reset_slots(ctypes.byref(pool.desc), layer, _ptr(slots),
                                       slots.numel(), _stream(stream)))


# ------------------------------------------------------------------ update

def _update_args(kda: bool, pool: Pool, layer: int, slot_idx, q, k, v, g, beta, perm, scale,
                 o, stream):
    """Checks the operands and returns (C function, argument tuple)."""
    d = pool.d
    HV = pool.num_v_heads
    slot_idx = _dev(slot_idx, torch.int32, "slot_idx")
    B = slot_idx.numel()
    HK = q.shape[1] if q.dim() == 3 else -1
    _dev(q, torch.bfloat16, "q", (B, HK, d))
    _dev(k, torch.bfloat16, "k", (B, HK, d))
    _dev(v, torch.bfloat16, "v", (B, HV, d))
    _dev(g, torch.bfloat16, "g", (B, HV, d) if kda else (B, HV))
    _dev(beta, torch.bfloat16, "beta", (B, HV))
    if perm is not None:
        _dev(perm, torch.uint8, "perm", (HV, d))
    if o.dtype == torch.float32:
        o_dt = DAMP_DT_FP32
    elif o.dtype == torch.bfloat16:
        o_dt = DAMP_DT_BF16
    else:
        raise ValueError("o must be float32 or bfloat16")
    _dev(o, o.dtype, "o", (B, HV, d))
    fn = lib().damp_state_update_kda if kda else lib().damp_state_update_gdn
    args = (ctypes.byref(pool.desc), layer, _ptr(slot_idx), B, HK, _ptr(q), _ptr(k), _ptr(v),
            _ptr(g), _ptr(beta), _ptr(perm), float(scale), _ptr(o), o_dt, _stream(stream))
    return fn, args


def _update(kda: bool, pool: Pool, layer: int, slot_idx, q, k, v, g, beta, perm, scale, o,
            stream):
    fn, args = _update_args(kda, pool, layer, slot_idx, q, k, v, g, beta, perm, scale, o, stream)
    _check(fn(*args))
    return o


def damp_state_update_gdn(pool: Pool, layer: int, slot_idx, q, k, v, g, beta, perm=None,
                          scale: float = 1.0, o=None, stream=None):
    """One GDN decode step in place on the pool; returns o [B, HV, d]."""
    if o is None:
        o = torch.empty((slot_idx.numel(), pool.num_v_heads, pool.d), dtype=torch.float32,
                        device=pool.buffer.device)
    return _update(False, pool, layer, slot_idx, q, k, v, g, beta, perm, scale, o, stream)


def damp_state_update_kda(pool: Pool, layer: int, slot_idx, q, k, v, g, beta, perm=None,
                          scale: float = 1.0, o=None, stream=None):
    """One KDA decode step in place on the pool; returns o [B, HV, d]."""
    if o is None:
        o = torch.empty((slot_idx.numel(), pool.num_v_heads, pool.d), dtype=torch.float32,
                        device=pool.buffer.device)
    return _update(True, pool, layer, slot_idx, q, k, v, g, beta, perm, scale, o, stream)


def _prefill(kda: bool, pool: Pool, layer: int, slot_idx, q, k, v, g, beta, perm, scale, o,
             stream):
    d = pool.d
    HV = pool.num_v_heads
    slot_idx = _dev(slot_idx, torch.int32, "slot_idx")
    B = slot_idx.numel()
    if q.dim() != 4:
        raise ValueError("q must be [B, T, HK, d]")
    T, HK = q.shape[1], q.shape[2]
    _dev(q, torch.bfloat16, "q", (B, T, HK, d))
    _dev(k, torch.bfloat16, "k", (B, T, HK, d))
    _dev(v, torch.bfloat16, "v", (B, T, HV, d))
    _dev(g, torch.bfloat16, "g", (B, T, HV, d) if kda else (B, T, HV))
    _dev(beta, torch.bfloat16, "beta", (B, T, HV))
    if perm is not None:
        _dev(perm, torch.uint8, "perm", (HV, d))
    if o is None:
        o = torch.empty((B, T, HV, d), dtype=torch.float32, device=pool.buffer.device)
    if o.dtype == torch.float32:
        o_dt = DAMP_DT_FP32
    elif o.dtype == torch.bfloat16:
        o_dt = DAMP_DT_BF16
    else:
        raise ValueError("o must be float32 or bfloat16")
    _dev(o, o.dtype, "o", (B, T, HV, d))
    fn = lib().damp_state_prefill_kda if kda else lib().damp_state_prefill_gdn
    _check(fn(ctypes.byref(pool.desc), layer, _ptr(slot_idx), B, T, HK, _ptr(q), _ptr(k), _ptr(v),
              _ptr(g), _ptr(beta), _ptr(perm), float(scale), _ptr(o), o_dt, _stream(stream)))
    return o


def damp_state_prefill_gdn(pool: Pool, layer: int, slot_idx, q, k, v, g, beta, perm=None,
                           scale: float = 1.0, o=None, stream=None):
    """One GDN prefill chunk in place on the pool (inputs [B, T, ...]);
    returns o [B, T, HV, d]."""
    return _prefill(False, pool, layer, slot_idx, q, k, v, g, beta, perm, scale, o, stream)


def damp_state_prefill_kda(pool: Pool, layer: int, slot_idx, q, k, v, g, beta, perm=None,
                           scale: float = 1.0, o=None, stream=None):
    """One KDA prefill chunk in place on the pool (inputs [B, T, ...]);
    returns o [B, T, HV, d]."""
    return _prefill(True, pool, layer, slot_idx, q, k, v, g, beta, perm, scale, o, stream)


# ----------------------------------------------------------- pack / unpack

def damp_state_pack(pool: Pool, layer: int, slot_idx, S, perm=None, stream=None) -> None:
    slot_idx = _dev(slot_idx, torch.int32, "slot_idx")
    d = pool.d
    _dev(S, torch.float32, "S", (slot_idx.numel(), pool.num_v_heads, d, d))
    if perm is not None:
        _dev(perm, torch.uint8, "perm", (pool.num_v_heads, d))
    _check(lib().damp_state_pack(ctypes.byref(pool.desc), layer, _ptr(slot_idx),
                                 slot_idx.numel(), _ptr(S), _ptr(perm), _stream(stream)))


def damp_state_unpack(pool: Pool, layer: int, slot_idx, perm=None, S_out=None, stream=None):
    slot_idx = _dev(slot_idx, torch.int32, "slot_idx")
    d = pool.d
    shape = (slot_idx.numel(), pool.num_v_heads, d, d)
    if S_out is None:
        S_out = torch.empty(shape, dtype=torch.float32, device=pool.buffer.device)
    _dev(S_out, torch.float32, "S_out", shape)
    if perm is not None:
        _dev(perm, torch.uint8, "perm", (pool.num_v_heads, d))
    _check(lib().damp_state_unpack(ctypes.byref(pool.desc), layer, _ptr(slot_idx),
                                   slot_idx.numel(), _ptr(perm), _ptr(S_out), _stream(stream)))
    return S_out


# --------------------------------------------------------------- selection

def _select(fn, states, log_decay, k_hi, kda, lo, tau, stream):
    states = _dev(states, torch.float32, "states")
    if states.dim() != 4:
        raise ValueError("states must be [N, H, d_k, d_v]")
    N, H, dk, dv = states.shape
    _dev(log_decay, torch.float32, "log_decay", (N, H, dk) if kda else (N, H))
    sel = torch.zeros((H, k_hi), dtype=torch.int32)
    perm = torch.zeros((H, dk), dtype=torch.uint8)
    score = torch.zeros((H, dk), dtype=torch.float64)
    _check(fn(int(kda), N, H, dk, dv, _ptr(states), _ptr(log_decay),
              None if lo is None else ctypes.byref(lo), k_hi, float(tau), _ptr(sel), _ptr(perm),
              _ptr(score), _stream(stream)))
    return sel, perm, score


def damp_select_channels(states, log_decay, k_hi: int, *, kda: bool, lo: damp_layout = None,
                         tau: float = 1e-4, stream=None):
    """Alg. 1 on device-resident calibration samples, with E measured under
    the low tier of `lo` (None: the per-row quantizer); returns host tensors
    (sel int32 [H, k_hi], perm uint8 [H, d_k], score float64 [H, d_k])."""
    return _select(lib().damp_select_channels, states, log_decay, k_hi, kda, lo, tau, stream)


def damp_select_channels_noalloc(states, log_decay, k_hi: int, *, kda: bool,
                                 lo: damp_layout = None, tau: float = 1e-4, stream=None):
    """As damp_select_channels, with the library's fixed device scratch
    instead of an allocation per call ((N + 2) * H * d_k <= 2^21)."""
    return _select(lib().damp_select_channels_noalloc, states, log_decay, k_hi, kda, lo, tau,
                   stream)


# ------------------------------------------------------------- calibration

class Calib:
    """Calibration accumulators (a torch float64 buffer on the GPU) and their
    damp_calib descriptor (keeps the buffer alive)."""

    def __init__(self, lo: damp_layout, *, kda: bool, num_heads: int, num_domains: int = 1,
                 device="cuda", stream=None):
        need = lib().damp_calib_required_bytes(num_domains, num_heads, lo.d_k)
        if need == 0:
            raise ValueError("invalid calibration shape")
        self.buffer = torch.empty(need // 8, dtype=torch.float64, device=device)
        self.desc = damp_calib()
        _check(lib().damp_calib_init(ctypes.byref(self.desc), ctypes.byref(lo), int(kda),
                                     num_heads, num_domains, _ptr(self.buffer), need,
                                     _stream(stream)))
        self.lo, self.kda = lo, kda
        self.num_heads, self.num_domains = num_heads, num_domains


def damp_calib_accumulate(calib: Calib, domain: int, pool: Pool, layer: int, slot_idx, g,
                          perm=None, stream=None) -> None:
    """One sampled state write of the FP32 pool's slots (g: bf16 log-decay of
    the sampled token, [B, H] or [B, H, d_k])."""
    slot_idx = _dev(slot_idx, torch.int32, "slot_idx")
    B, H, d = slot_idx.numel(), calib.num_heads, calib.lo.d_k
    _dev(g, torch.bfloat16, "g", (B, H, d) if calib.kda else (B, H))
    if perm is not None:
        _dev(perm, torch.uint8, "perm", (H, d))
    _check(lib().damp_calib_accumulate(ctypes.byref(calib.desc), domain, ctypes.byref(pool.desc),
                                       layer, _ptr(slot_idx), B, _ptr(perm), _ptr(g),
                                       _stream(stream)))


def damp_calibrate_sequence(calib: Calib, domain: int, pool: Pool, layer: int, slot_idx, q, k, v,
                            g, beta, stride: int = 8, stream=None) -> None:
    """Runs T tokens ([B, T, ...] inputs) of the FP32 recurrence on the pool,
    accumulating the state write after every `stride` tokens."""
    slot_idx = _dev(slot_idx, torch.int32, "slot_idx")
    B, H, d = slot_idx.numel(), calib.num_heads, calib.lo.d_k
    if q.dim() != 4:
        raise ValueError("q must be [B, T, HK, d]")
    T, HK = q.shape[1], q.shape[2]
    _dev(q, torch.bfloat16, "q", (B, T, HK, d))
    _dev(k, torch.bfloat16, "k", (B, T, HK, d))
    _dev(v, torch.bfloat16, "v", (B, T, H, d))
    _dev(g, torch.bfloat16, "g", (B, T, H, d) if calib.kda else (B, T, H))
    _dev(beta, torch.bfloat16, "beta", (B, T, H))
    _check(lib().damp_calibrate_sequence(ctypes.byref(calib.desc), domain, ctypes.byref(pool.desc),
                                         layer, _ptr(slot_idx), B, T, stride, HK, _ptr(q), _ptr(k),
                                         _ptr(v), _ptr(g), _ptr(beta), _stream(stream)))


def damp_calib_finalize(calib: Calib, k_hi: int, selector: int = DAMP_SEL_DAMP,
                        tau: float = 1e-4, rand_scores=None, stream=None) -> dict:
    """Selection from the accumulated statistics; host tensors sel int32
    [H, k_hi], perm uint8 [H, d_k], score and E, P, energy, mean log a
    (float64 [H, d_k])."""
    H, d = calib.num_heads, calib.lo.d_k
    sel = torch.zeros((H, k_hi), dtype=torch.int32)
    perm = torch.zeros((H, d), dtype=torch.uint8)
    score = torch.zeros((H, d), dtype=torch.float64)
    stats = torch.zeros((4, H, d), dtype=torch.float64)
    rs = None
    if rand_scores is not None:
        rs = torch.as_tensor(rand_scores, dtype=torch.float64).contiguous()
        if tuple(rs.shape) != (H, d) or rs.device.type != "cpu":
            raise ValueError("rand_scores must be a host float64 [H, d_k] tensor")
    _check(lib().damp_calib_finalize(ctypes.byref(calib.desc), selector, k_hi, float(tau),
                                     _ptr(rs), _ptr(sel), _ptr(perm), _ptr(score), _ptr(stats),
                                     _stream(stream)))
    return dict(sel=sel, perm=perm, score=score, E=stats[0], P=stats[1], energy=stats[2],
                mean_log_a=stats[3])


def damp_topk_overlap(sel_a, sel_b) -> float:
    """|A intersect B| / k of two [k] int32 host selections."""
    a = torch.as_tensor(sel_a, dtype=torch.int32).contiguous()
    b = torch.as_tensor(sel_b, dtype=torch.int32).contiguous()
    if a.numel() != b.numel() or a.device.type != "cpu" or b.device.type != "cpu":
        raise ValueError("two host selections of equal size")
    return lib().damp_topk_overlap(_ptr(a), _ptr(b), a.numel())


def damp_spearman(a, b) -> float:
    """Spearman rank correlation of two host score vectors."""
    x = torch.as_tensor(a, dtype=torch.float64).contiguous()
    y = torch.as_tensor(b, dtype=torch.float64).contiguous()
    if x.numel() != y.numel() or x.device.type != "cpu" or y.device.type != "cpu":
        raise ValueError("two host score vectors of equal size")
    return lib().damp_spearman(_ptr(x), _ptr(y), x.numel())


class PreparedUpdate:
    """A decode-step call with its arguments checked and marshalled once, for
    loops that re-issue the same buffers (the benchmark's timed region, a
    serving step). Calling it enqueues the kernel on the stream captured at
    construction; it raises DampError on a non-zero status."""

    def __init__(self, kda: bool, pool: Pool, layer: int, slot_idx, q, k, v, g, beta, perm,
                 scale: float, o, stream=None):
        self._fn, self._args = _update_args(kda, pool, layer, slot_idx, q, k, v, g, beta, perm,
                                            scale, o, stream)
        self._keep = (pool, slot_idx, q, k, v, g, beta, perm, o)

    def __call__(self) -> None:
        st = self._fn(*self._args)
        if st != DAMP_OK:
            _check(st)
