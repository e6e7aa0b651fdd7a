"""Helpers of the GPU parity tests: moving seeded inputs to the device and
comparing packed tiles from the HIP path with the oracle's, field by field.

Tolerances (the acceptance bar of the DAMP state update):
  - FP32-state path: state and o within 1e-5 relative L2;
  - mixed path: o within 2e-3 relative L2, low-tier codes within 1 LSB on at
    least 99.9% of entries, high-tier bf16 / FP16 values within 1 ulp on
    99.9%; fp32 scales within 1e-5 relative, FP16 scales equal on 99.9% and
    within one FP16 step everywhere;
  - channel selection and unpack: bit-exact.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import oracle as orc

O_TOL_MIXED = 2e-3
FP32_TOL = 1e-5
CODE_FRAC = 0.999


def dev_bf16(u16: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).view(torch.bfloat16).cuda()


def dev_inputs(step_inp: dict) -> dict:
    return {k: dev_bf16(v) for k, v in step_inp.items()}


def dev_i32(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def dev_u8(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).cuda()


def rel_l2(x, y) -> float:
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    return float(np.linalg.norm(x - y) / max(np.linalg.norm(y), 1e-300))


def _bf16_order(u: np.ndarray) -> np.ndarray:
    """Monotone integer key of bf16 bit patterns (adjacent values differ by 1)."""
    u = u.astype(np.int32)
    return np.where(u & 0x8000, -(u & 0x7FFF), u)


def split_tiles(buf: np.ndarray, pool: "orc.Pool"):
    """(hi 16-bit [T, k_hi*dv], codes uint8 [T, nl*dv], s [T, nl*groups],
    z [T, nl*groups]) or the fp32 state [T, dk*dv] for every tile slot of the
    pool; s and z are widened to fp32 for the paper's FP16 metadata."""
    tb = orc.tile_bytes(pool.kind, pool.dk, pool.dv, pool.k_hi, pool.fmt)
    tiles = np.ascontiguousarray(buf.reshape(-1, pool.tile_stride)[:, :tb])
    if pool.kind == orc.KIND_FP32:
        return tiles.view(np.float32)
    hb = pool.k_hi * pool.dv * 2
    nl = pool.dk - pool.k_hi
    hi = np.ascontiguousarray(tiles[:, :hb]).view(np.uint16)
    codes = tiles[:, hb:hb + nl * pool.dv]
    raw = np.ascontiguousarray(tiles[:, hb + nl * pool.dv:])
    if pool.fmt is None:
        meta = raw.view(np.float32).reshape(tiles.shape[0], nl, 2)
    else:
        meta = raw.view(np.float16).astype(np.float32).reshape(tiles.shape[0], -1, 2)
    return hi, codes, meta[..., 0], meta[..., 1]


def _sm_order(c: np.ndarray, sign_bit: int) -> np.ndarray:
    """Monotone integer key of sign-magnitude codes (E4M3, E2M1)."""
    c = c.astype(np.int32)
    return np.where(c & sign_bit, -(c & (sign_bit - 1)), c)


def split_tiles_table(buf: np.ndarray, pool: "orc.Pool") -> dict:
    """Fields of the other formats of App. A.1's table for every tile slot:
    FP16 high rows, codes (one byte per value), and the metadata (FP16 s and
    z for INT4, fp32 s for FP8, E4M3 block-scale codes and the fp32 global
    scale for NVFP4)."""
    _, group, _, _, code = orc.fmt5(pool.fmt)
    tb = orc.tile_bytes(pool.kind, pool.dk, pool.dv, pool.k_hi, pool.fmt)
    t = np.ascontiguousarray(buf.reshape(-1, pool.tile_stride)[:, :tb])
    n, dv, nl = t.shape[0], pool.dv, pool.dk - pool.k_hi
    hb = pool.k_hi * dv * 2
    nib = code in (orc.CODE_U4, orc.CODE_E2M1)
    cb = nl * (dv // 2 if nib else dv)
    raw = t[:, hb:hb + cb]
    codes = np.stack([raw & 0xF, raw >> 4], -1).reshape(n, -1) if nib else raw
    meta = np.ascontiguousarray(t[:, hb + cb:])
    out = dict(hi=np.ascontiguousarray(t[:, :hb]).view(np.uint16), codes=codes, code=code)
    if code == orc.CODE_U4:
        sz = meta.view(np.float16).astype(np.float32).reshape(n, -1, 2)
        out.update(s=sz[..., 0], z=sz[..., 1])
    elif code == orc.CODE_E4M3:
        out.update(s=meta.view(np.float32))
    else:
        out.update(sb=meta[:, :nl * (dv // group)], g=np.ascontiguousarray(meta[:, -4:]).view(np.float32))
    return out


def compare_tiles_table(gpu_buf: np.ndarray, ref: "orc.Pool", label: str = "",
                        s16_exact_min: float = CODE_FRAC) -> dict:
    """The bar of compare_tiles for the INT4, FP8 and NVFP4 formats: codes
    (as ordered values for the floating-point codes) and NVFP4 block scales
    within one step on 99.9%, FP16 high rows within 1 ulp on 99.9%, INT4's
    FP16 (s, z) as the paper's, FP8 and NVFP4 fp32 scales within 1e-5."""
    a, b = split_tiles_table(gpu_buf, ref), split_tiles_table(ref.buf, ref)
    stats = {}
    if a["hi"].size:
        dh = np.abs(_bf16_order(a["hi"]) - _bf16_order(b["hi"]))
        stats["hi_le1ulp"] = float((dh <= 1).mean())
        assert stats["hi_le1ulp"] >= CODE_FRAC, f"{label}: hi tier {stats}"
    code = a["code"]
    if code == orc.CODE_U4:
        ka, kb = a["codes"].astype(np.int32), b["codes"].astype(np.int32)
    else:
        sign = 0x80 if code == orc.CODE_E4M3 else 0x8
        ka, kb = _sm_order(a["codes"], sign), _sm_order(b["codes"], sign)
    dc = np.abs(ka - kb)
    stats["code_exact"] = float((dc == 0).mean())
    stats["code_le1"] = float((dc <= 1).mean())
    assert stats["code_le1"] >= CODE_FRAC, f"{label}: codes {stats}"
    if code == orc.CODE_U4:
        live = b["s"] != 0
        rel = np.abs(a["s"][live].astype(np.float64) - b["s"][live]) / np.abs(b["s"][live])
        stats["s_rel_max"] = float(rel.max()) if rel.size else 0.0
        stats["s_exact"] = float((a["s"][live] == b["s"][live]).mean()) if rel.size else 1.0
        stats["z_le1"] = float((np.abs(a["z"] - b["z"]) <= 1).mean())
        assert stats["s_rel_max"] <= 2.0 ** -10 * 1.0001, f"{label}: scales {stats}"
        assert stats["s_exact"] >= s16_exact_min and stats["z_le1"] >= CODE_FRAC, f"{label}: {stats}"
    elif code == orc.CODE_E4M3:
        live = b["s"] != 0
        rel = np.abs(a["s"][live].astype(np.float64) - b["s"][live]) / np.abs(b["s"][live])
        stats["s_rel_max"] = float(rel.max()) if rel.size else 0.0
        assert stats["s_rel_max"] <= 1e-5, f"{label}: scales {stats}"
    else:
        dsb = np.abs(_sm_order(a["sb"], 0x80) - _sm_order(b["sb"], 0x80))
        stats["sb_le1"] = float((dsb <= 1).mean())
        live = b["g"] != 0
        rel = np.abs(a["g"][live].astype(np.float64) - b["g"][live]) / np.abs(b["g"][live])
        stats["g_rel_max"] = float(rel.max()) if rel.size else 0.0
        assert stats["sb_le1"] >= CODE_FRAC and stats["g_rel_max"] <= 1e-5, f"{label}: {stats}"
    return stats


def compare_tiles(gpu_buf: np.ndarray, ref: "orc.Pool", label: str = "",
                  s16_exact_min: float = CODE_FRAC) -> dict:
    """Field-by-field comparison; asserts the acceptance bar and returns stats.
    s16_exact_min: fraction of FP16 scales that must match exactly (the rest
    within one FP16 step); lower after several fp32 steps, whose rounding
    differences move more scales across an FP16 rounding boundary."""
    if ref.fmt is not None and orc.fmt5(ref.fmt)[4] != orc.CODE_U8:
        return compare_tiles_table(gpu_buf, ref, label, s16_exact_min)
    if ref.kind == orc.KIND_FP32:
        a = split_tiles(gpu_buf, ref)
        b = split_tiles(ref.buf, ref)
        err = rel_l2(a, b)
        assert err <= FP32_TOL, f"{label}: fp32 state rel-L2 {err:.3e}"
        return dict(state_rel=err)
    ha, ca, sa, za = split_tiles(gpu_buf, ref)
    hb, cb, sb, zb = split_tiles(ref.buf, ref)
    stats = {}
    if ha.size:
        dh = np.abs(_bf16_order(ha) - _bf16_order(hb))
        stats["hi_exact"] = float((dh == 0).mean())
        stats["hi_le1ulp"] = float((dh <= 1).mean())
        assert stats["hi_le1ulp"] >= CODE_FRAC, f"{label}: hi tier {stats}"
    if ca.size:
        dc = np.abs(ca.astype(np.int32) - cb.astype(np.int32))
        stats["code_exact"] = float((dc == 0).mean())
        stats["code_le1"] = float((dc <= 1).mean())
        stats["code_maxdiff"] = int(dc.max())
        stats["z_le1"] = float((np.abs(za - zb) <= 1).mean())
        live = sb != 0  # tiles never written hold zero bytes on both sides
        assert np.array_equal(sa[~live], sb[~live]), f"{label}: unwritten tiles differ"
        rel = np.abs(sa[live].astype(np.float64) - sb[live]) / np.abs(sb[live])
        stats["s_rel_max"] = float(rel.max()) if rel.size else 0.0
        assert stats["code_le1"] >= CODE_FRAC, f"{label}: codes {stats}"
        assert stats["z_le1"] >= CODE_FRAC, f"{label}: zero points {stats}"
        if ref.fmt is None:
            assert stats["s_rel_max"] <= 1e-5, f"{label}: scales {stats}"
        else:
            # FP16 scales: a last-bit difference of the fp32 scale can flip
            # its FP16 rounding, by one FP16 step (2^-10 relative)
            stats["s_exact"] = float((sa[live] == sb[live]).mean()) if rel.size else 1.0
            assert stats["s_rel_max"] <= 2.0 ** -10 * 1.0001, f"{label}: scales {stats}"
            assert stats["s_exact"] >= s16_exact_min, f"{label}: scales {stats}"
    return stats


def gpu_pool_from(ref: "orc.Pool", damp_mod, layout=None):
    """A device pool holding exactly the bytes of an oracle pool."""
    kind = ref.kind
    if layout is None:
        layout = damp_mod.damp_layout_init(ref.dk, ref.dv, ref.k_hi, kind)
        if ref.fmt is not None:
            (layout.hi_dtype, layout.group, layout.meta_dtype, layout.hadamard,
             layout.code_dtype) = orc.fmt5(ref.fmt)
    buf = torch.from_numpy(ref.buf.copy()).cuda()
    return damp_mod.Pool(layout, ref.num_layers, ref.num_slots, ref.hv, buffer=buf)
