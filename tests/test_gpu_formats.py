"""GPU parity of the other low-tier formats of App. A.1's format table (INT4
with and without H32, FP8 E4M3 per Eq. (16), NVFP4) against the oracle:
pack, unpack, reset, one decode step and one prefill chunk. Both sides start
from identical bytes packed by the oracle (see parity_util for the bar).
"""
import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_2608_27513_amd import damp as D
from paper_2608_27513_amd import inputs
from parity_util import (O_TOL_MIXED, compare_tiles, dev_i32, dev_inputs, dev_u8, gpu_pool_from,
                         rel_l2)

pytestmark = pytest.mark.gpu

FORMATS = {"int4": orc.FMT_INT4, "int4_h32": orc.FMT_INT4_H32, "fp8": orc.FMT_FP8,
           "nvfp4": orc.FMT_NVFP4}


def _say(*a):
    print(*a, flush=True)


def _states(seed, B, HV, d):
    S = inputs.synthetic_states(seed, B, HV, d)
    inputs.scale_channels(S, inputs.outlier_channels(seed, HV, d, min(8, d // 4)), 10.0)
    return S


@pytest.mark.parametrize("name", list(FORMATS))
@pytest.mark.parametrize("d,k_hi", [(32, 8), (64, 0), (128, 16)])
def test_pack_parity(name, d, k_hi):
    fmt = FORMATS[name]
    _say(f"format pack {name} d={d} k_hi={k_hi}")
    B, HV = 3, 4
    seed = 1000 + d + k_hi
    S = _states(seed, B, HV, d)
    perm = inputs.random_perms(seed, HV, d)
    slots = inputs.slot_order(seed, B + 2, B)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B + 2, HV, fmt=fmt)
    gpool = gpu_pool_from(ref, D)
    orc.pack(ref, 0, slots, S, perm)
    D.damp_state_pack(gpool, 0, dev_i32(slots), torch.from_numpy(S).cuda(), dev_u8(perm))
    torch.cuda.synchronize()
    _say(f"  {compare_tiles(gpool.buffer.cpu().numpy(), ref, f'pack {name} d={d}')}")


@pytest.mark.parametrize("name", list(FORMATS))
def test_unpack_parity(name):
    """Unpack of oracle-packed bytes: one product per value for FP8 and
    NVFP4 and s (c - z) for INT4 are exact; with the transform, equal up to
    its summation order."""
    fmt = FORMATS[name]
    d, k_hi, B, HV = 64, 16, 3, 2
    _say(f"format unpack {name}")
    S = _states(1100, B, HV, d)
    perm = inputs.random_perms(1100, HV, d)
    slots = np.arange(B, dtype=np.int32)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B, HV, fmt=fmt)
    orc.pack(ref, 0, slots, S, perm)
    gpool = gpu_pool_from(ref, D)
    out = D.damp_state_unpack(gpool, 0, dev_i32(slots), dev_u8(perm))
    torch.cuda.synchronize()
    got, want = out.cpu().numpy(), orc.unpack(ref, 0, slots, perm)
    if orc.fmt5(fmt)[3]:
        assert np.abs(got - want).max() <= 2e-6 * np.abs(want).max()
    else:
        assert np.array_equal(got, want)


@pytest.mark.parametrize("name", list(FORMATS))
def test_reset_matches_oracle_bytes(name):
    d, k_hi, HV = 64, 8, 3
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 2, 4, HV, fmt=FORMATS[name])
    ref.buf[:] = 0x5A
    gpool = gpu_pool_from(ref, D)
    slots = np.array([2, 0], np.int32)
    orc.reset(ref, -1, slots)
    D.damp_pool_reset_slots(gpool, -1, dev_i32(slots))
    torch.cuda.synchronize()
    assert np.array_equal(gpool.buffer.cpu().numpy(), ref.buf)


@pytest.mark.parametrize("name", list(FORMATS))
@pytest.mark.parametrize("kda,d,HK,HV,B,k_hi", [(False, 128, 2, 4, 3, 16), (True, 64, 2, 2, 2, 8),
                                                (False, 32, 1, 2, 2, 0),
                                                (True, 128, 2, 2, 2, 40)])  # K_hi > 32: generic kernel
def test_single_step_parity(name, kda, d, HK, HV, B, k_hi):
    fmt = FORMATS[name]
    _say(f"format step {name} kda={kda} d={d} HK={HK} HV={HV} B={B} k_hi={k_hi}")
    seed = 1200 + d + B + k_hi + 7 * kda
    slots = inputs.slot_order(seed, B + 2, B)
    perm = inputs.random_perms(seed, HV, d)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B + 2, HV, fmt=fmt)
    orc.pack(ref, 0, slots, _states(seed, B, HV, d), perm)
    gpool = gpu_pool_from(ref, D)
    inp = inputs.step(inputs.decode_inputs(seed, 1, B, HK, HV, d, kda=kda), 0)
    x = dev_inputs(inp)
    o = torch.empty((B, HV, d), dtype=torch.float32, device="cuda")
    fn = D.damp_state_update_kda if kda else D.damp_state_update_gdn
    fn(gpool, 0, dev_i32(slots), x["q"], x["k"], x["v"], x["g"], x["beta"], perm=dev_u8(perm),
       scale=0.5, o=o)
    o_ref = orc.update(ref, 0, slots, kda=kda, perm=perm, scale=0.5, **inp)
    torch.cuda.synchronize()
    err = rel_l2(o.cpu().numpy(), o_ref)
    stats = compare_tiles(gpool.buffer.cpu().numpy(), ref, f"step {name} d={d}")
    _say(f"  o rel-L2 {err:.2e}  {stats}")
    assert err <= O_TOL_MIXED and err <= 1e-4  # identical starting bytes


@pytest.mark.parametrize("name", list(FORMATS))
def test_prefill_parity(name):
    fmt = FORMATS[name]
    d, HK, HV, B, T, k_hi = 64, 2, 4, 2, 6, 16
    _say(f"format prefill {name}")
    seed = 1300
    slots = inputs.slot_order(seed, B + 1, B)
    perm = inputs.random_perms(seed, HV, d)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B + 1, HV, fmt=fmt)
    orc.pack(ref, 0, slots, _states(seed, B, HV, d), perm)
    gpool = gpu_pool_from(ref, D)
    inp = inputs.as_prefill(inputs.decode_inputs(seed, T, B, HK, HV, d))
    x = dev_inputs(inp)
    o = torch.empty((B, T, HV, d), dtype=torch.float32, device="cuda")
    D.damp_state_prefill_gdn(gpool, 0, dev_i32(slots), x["q"], x["k"], x["v"], x["g"], x["beta"],
                             perm=dev_u8(perm), o=o)
    o_ref = orc.prefill(ref, 0, slots, kda=False, perm=perm, **inp)
    torch.cuda.synchronize()
    err = rel_l2(o.cpu().numpy(), o_ref)
    stats = compare_tiles(gpool.buffer.cpu().numpy(), ref, f"prefill {name}", s16_exact_min=0.99)
    _say(f"  o rel-L2 {err:.2e}  {stats}")
    assert err <= 1e-4


STREAM_FORMATS = ["int4", "int4_h32", "fp8", "nvfp4"]


@pytest.mark.parametrize("name", STREAM_FORMATS)
@pytest.mark.parametrize("kda,k_hi", [(False, 16), (True, 12), (False, 0), (True, 32),
                                      (False, 8)])
def test_many_tiles_per_workgroup(name, kda, k_hi):
    """d = 128 (the persistent streaming kernel) with more requests than
    resident workgroups, so each workgroup streams several tiles; slots in
    random order, some padded or out of range (o = 0, their tiles untouched).
    k_hi = 12 puts 16-bit and code rows in one wave, 0 and 32 leave only one
    kind of row in slot 0."""
    fmt = FORMATS[name]
    d, HV, B = 128, 4, 300
    HK = HV if kda else 2
    _say(f"format many tiles {name} kda={kda} k_hi={k_hi}")
    seed = 1400 + 3 * kda + k_hi
    n_slots = B + 40
    slots = inputs.slot_order(seed, n_slots, B)
    slots[::37] = -1
    slots[5] = n_slots  # out of range
    perm = inputs.random_perms(seed, HV, d)
    S = _states(seed, B, HV, d)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, n_slots, HV, fmt=fmt)
    live = (slots >= 0) & (slots < n_slots)
    orc.pack(ref, 0, slots[live], S[live], perm)
    gpool = gpu_pool_from(ref, D)
    inp = inputs.step(inputs.decode_inputs(seed, 1, B, HK, HV, d, kda=kda), 0)
    x = dev_inputs(inp)
    o = torch.empty((B, HV, d), dtype=torch.float32, device="cuda")
    fn = D.damp_state_update_kda if kda else D.damp_state_update_gdn
    fn(gpool, 0, dev_i32(slots), x["q"], x["k"], x["v"], x["g"], x["beta"], perm=dev_u8(perm),
       o=o)
    o_ref = orc.update(ref, 0, slots, kda=kda, perm=perm, **inp)
    torch.cuda.synchronize()
    o_gpu = o.cpu().numpy()
    assert np.all(o_gpu[~live] == 0) and np.all(o_ref[~live] == 0)
    err = rel_l2(o_gpu, o_ref)
    stats = compare_tiles(gpool.buffer.cpu().numpy(), ref, f"many tiles {name}")
    _say(f"  o rel-L2 {err:.2e}  {stats}")
    assert err <= 1e-4


@pytest.mark.parametrize("name", STREAM_FORMATS)
@pytest.mark.parametrize("kda", [False, True])
def test_full_size_step(name, kda):
    """The decode workload (B = 256, 32 value heads, d = 128, 16 FP16 rows)
    in these formats, in the launch configuration of the benchmark; the
    oracle runs the whole step, so every output and stored byte is compared."""
    fmt = FORMATS[name]
    B, HV, d, k_hi = 256, 32, 128, 16
    HK = HV if kda else 16
    seed = 1500 + kda
    _say(f"format full-size {name} kda={kda}")
    S = _states(seed, B, HV, d)
    perm = inputs.random_perms(seed, HV, d)
    slots = inputs.slot_order(seed, B, B)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B, HV, fmt=fmt)
    orc.pack(ref, 0, slots, S, perm)
    del S
    gpool = gpu_pool_from(ref, D)
    inp = inputs.step(inputs.decode_inputs(seed, 1, B, HK, HV, d, kda=kda), 0)
    x = dev_inputs(inp)
    o = torch.empty((B, HV, d), dtype=torch.float32, device="cuda")
    fn = D.damp_state_update_kda if kda else D.damp_state_update_gdn
    fn(gpool, 0, dev_i32(slots), x["q"], x["k"], x["v"], x["g"], x["beta"], perm=dev_u8(perm),
       o=o)
    torch.cuda.synchronize()
    _say("  gpu step done; running the oracle")
    o_ref = orc.update(ref, 0, slots, kda=kda, perm=perm, **inp)
    err = rel_l2(o.cpu().numpy(), o_ref)
    stats = compare_tiles(gpool.buffer.cpu().numpy(), ref, f"full-size {name}")
    _say(f"  o rel-L2 {err:.2e}  {stats}")
    assert err <= O_TOL_MIXED and err <= 1e-4


@pytest.mark.parametrize("name", ["default", "int8_h32", "int8_g32"] + STREAM_FORMATS)
@pytest.mark.parametrize("zeroed", ["some", "low_tier"])
def test_degenerate_rows_from_zero_state(name, zeroed):
    """d = 128 (the pipelined kernel) from the reset state with key channels
    set to zero: their rows stay exactly zero, so the quantizers take their
    constant-row rules (R9; the FP16 group rules; FP8's floor on the scale;
    NVFP4's zero block scale). With every low-tier channel zeroed (identity
    permutation), NVFP4's tile maximum is 0 and its global scale 1."""
    fmt = {"default": None, "int8_h32": orc.FMT_PAPER, "int8_g32": orc.FMT_PAPER_PLAIN,
           **FORMATS}[name]
    d, HK, HV, B, k_hi = 128, 2, 4, 3, 16
    seed = 1600 + (zeroed == "low_tier")
    _say(f"degenerate rows {name} zeroed={zeroed}")
    slots = inputs.slot_order(seed, B + 2, B)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B + 2, HV, fmt=fmt)
    ref.buf[:] = 0x5A
    orc.reset(ref, 0, slots)
    gpool = gpu_pool_from(ref, D)
    inp = inputs.step(inputs.decode_inputs(seed, 1, B, HK, HV, d), 0)
    if zeroed == "some":
        perm = inputs.random_perms(seed, HV, d)
        chans = np.random.default_rng(seed).choice(d, size=40, replace=False)
    else:
        perm = None
        chans = np.arange(k_hi, d)
    inp["k"] = inp["k"].copy()
    inp["k"][..., chans] = 0
    x = dev_inputs(inp)
    o = torch.empty((B, HV, d), dtype=torch.float32, device="cuda")
    D.damp_state_update_gdn(gpool, 0, dev_i32(slots), x["q"], x["k"], x["v"], x["g"], x["beta"],
                            perm=None if perm is None else dev_u8(perm), o=o)
    o_ref = orc.update(ref, 0, slots, kda=False, perm=perm, **inp)
    torch.cuda.synchronize()
    err = rel_l2(o.cpu().numpy(), o_ref)
    stats = compare_tiles(gpool.buffer.cpu().numpy(), ref, f"degenerate {name}")
    _say(f"  o rel-L2 {err:.2e}  {stats}")
    assert err <= 1e-4
