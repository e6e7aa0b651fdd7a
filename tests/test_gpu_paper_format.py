"""GPU parity of the paper's storage tiers (App. A.1 format table, Eq. (17)):
FP16 high rows, groups of 32 with FP16 (s, z), with and without the
normalized block-32 Hadamard transform. Both sides start from identical
bytes packed by the oracle (see parity_util for the bar).
"""
import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_2608_27513_amd import damp as D
from paper_2608_27513_amd import inputs
from parity_util import O_TOL_MIXED, compare_tiles, dev_i32, dev_inputs, dev_u8, gpu_pool_from, rel_l2

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)


def _fmt(had):
    return orc.FMT_PAPER if had else orc.FMT_PAPER_PLAIN


@pytest.mark.parametrize("d,k_hi,had", [(32, 8, 1), (64, 0, 1), (64, 16, 0), (128, 16, 1),
                                        (128, 16, 0), (128, 32, 1), (128, 128, 1)])
def test_pack_parity(d, k_hi, had):
    _say(f"paper pack d={d} k_hi={k_hi} had={had}")
    B, HV = 3, 4
    seed = 300 + d + k_hi + had
    S = inputs.synthetic_states(seed, B, HV, d)
    inputs.scale_channels(S, inputs.outlier_channels(seed, HV, d, min(8, d // 4)), 10.0)
    perm = inputs.random_perms(seed, HV, d)
    slots = inputs.slot_order(seed, B + 2, B)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B + 2, HV, fmt=_fmt(had))
    gpool = gpu_pool_from(ref, D)
    orc.pack(ref, 0, slots, S, perm)
    D.damp_state_pack(gpool, 0, dev_i32(slots), torch.from_numpy(S).cuda(), dev_u8(perm))
    torch.cuda.synchronize()
    stats = compare_tiles(gpool.buffer.cpu().numpy(), ref, f"pack d={d}")
    _say(f"  {stats}")


@pytest.mark.parametrize("d,k_hi,had", [(32, 8, 1), (64, 16, 0), (128, 16, 1), (128, 16, 0)])
def test_unpack_parity(d, k_hi, had):
    """Unpack of oracle-packed bytes: bit-exact without the transform (s (c - z)
    and the FP16 rows are exact); with it, equal up to the summation order of
    the transform."""
    _say(f"paper unpack d={d} k_hi={k_hi} had={had}")
    B, HV = 3, 2
    seed = 400 + d + had
    S = inputs.synthetic_states(seed, B, HV, d)
    perm = inputs.random_perms(seed, HV, d)
    slots = np.arange(B, dtype=np.int32)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B, HV, fmt=_fmt(had))
    orc.pack(ref, 0, slots, S, perm)
    gpool = gpu_pool_from(ref, D)
    out = torch.empty((B, HV, d, d), dtype=torch.float32, device="cuda")
    D.damp_state_unpack(gpool, 0, dev_i32(slots), dev_u8(perm), out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    want = orc.unpack(ref, 0, slots, perm)
    if had:
        assert np.abs(got - want).max() <= 2e-6 * np.abs(want).max()
    else:
        assert np.array_equal(got, want)


def test_reset_matches_oracle_bytes():
    d, k_hi, HV = 64, 8, 3
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 2, 4, HV, fmt=orc.FMT_PAPER)
    ref.buf[:] = 0x5A
    gpool = gpu_pool_from(ref, D)
    slots = np.array([2, 0], np.int32)
    orc.reset(ref, -1, slots)
    D.damp_pool_reset_slots(gpool, -1, dev_i32(slots))
    torch.cuda.synchronize()
    assert np.array_equal(gpool.buffer.cpu().numpy(), ref.buf)


CASES = [
    # (d, kda, HK, HV, B, k_hi, had)
    (32, False, 1, 2, 3, 8, 1),
    (32, True, 2, 2, 2, 0, 0),
    (64, False, 2, 4, 3, 16, 1),
    (64, True, 4, 4, 2, 8, 1),
    (128, False, 2, 4, 3, 16, 1),
    (128, True, 4, 4, 3, 16, 1),
    (128, False, 4, 8, 2, 16, 0),
    (128, True, 2, 2, 2, 32, 0),
]


def _step(kda, ref, gpool, slots, inp, perm, scale=1.0):
    d_inp = dev_inputs(inp)
    B, HV, d = len(slots), ref.hv, ref.dv
    o = torch.empty((B, HV, d), dtype=torch.float32, device="cuda")
    fn = D.damp_state_update_kda if kda else D.damp_state_update_gdn
    fn(gpool, 0, dev_i32(slots), d_inp["q"], d_inp["k"], d_inp["v"], d_inp["g"], d_inp["beta"],
       perm=None if perm is None else dev_u8(perm), scale=scale, o=o)
    o_ref = orc.update(ref, 0, slots, kda=kda, perm=perm, scale=scale, **inp)
    torch.cuda.synchronize()
    return o.cpu().numpy(), o_ref


@pytest.mark.parametrize("d,kda,HK,HV,B,k_hi,had", CASES)
def test_single_step_parity(d, kda, HK, HV, B, k_hi, had):
    _say(f"paper step d={d} kda={kda} HK={HK} HV={HV} B={B} k_hi={k_hi} had={had}")
    seed = 500 + d + B + k_hi + 7 * kda + had
    slots = inputs.slot_order(seed, B + 2, B)
    perm = inputs.random_perms(seed, HV, d)
    S = inputs.synthetic_states(seed, B, HV, d)
    inputs.scale_channels(S, inputs.outlier_channels(seed, HV, d, min(8, d // 4)), 10.0)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B + 2, HV, fmt=_fmt(had))
    orc.pack(ref, 0, slots, S, perm)
    gpool = gpu_pool_from(ref, D)
    inp = inputs.step(inputs.decode_inputs(seed, 1, B, HK, HV, d, kda=kda), 0)
    o_gpu, o_ref = _step(kda, ref, gpool, slots, inp, perm, scale=0.5)
    err = rel_l2(o_gpu, o_ref)
    stats = compare_tiles(gpool.buffer.cpu().numpy(), ref, f"paper d={d} kda={kda}")
    _say(f"  o rel-L2 {err:.2e}  {stats}")
    assert err <= O_TOL_MIXED
    assert err <= 1e-4  # identical starting bytes: only fp32 rounding order differs


def test_trajectory_from_the_zero_state():
    """Eight GDN steps from the packed zero state on both sides, each side on
    its own state: o within the mixed-path bar at every step."""
    d, HK, HV, B, k_hi = 64, 2, 4, 2, 8
    slots = np.array([1, 0], np.int32)
    perm = inputs.random_perms(600, HV, d)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, 2, HV, fmt=orc.FMT_PAPER)
    orc.reset(ref, 0, slots)
    gpool = gpu_pool_from(ref, D)
    inp = inputs.decode_inputs(601, 8, B, HK, HV, d)
    for t in range(8):
        o_gpu, o_ref = _step(False, ref, gpool, slots, inputs.step(inp, t), perm)
        err = rel_l2(o_gpu, o_ref)
        _say(f"  step {t}: o rel-L2 {err:.2e}")
        assert err <= O_TOL_MIXED
    compare_tiles(gpool.buffer.cpu().numpy(), ref, "paper trajectory")


@pytest.mark.parametrize("kda,had,k_hi", [(False, 1, 16), (True, 1, 16), (False, 0, 32),
                                          (True, 0, 8)])
def test_many_tiles_per_workgroup(kda, had, k_hi):
    """d = 128 with more requests than resident workgroups, so each
    workgroup streams several tiles; slots in random order, some padded or
    out of range (o = 0, their tiles untouched)."""
    d, HV, B = 128, 4, 300
    HK = HV if kda else 2
    _say(f"paper many tiles kda={kda} had={had} k_hi={k_hi}")
    seed = 900 + 3 * kda + had + k_hi
    n_slots = B + 40
    slots = inputs.slot_order(seed, n_slots, B)
    slots[::37] = -1
    slots[5] = n_slots  # out of range
    perm = inputs.random_perms(seed, HV, d)
    S = inputs.synthetic_states(seed, B, HV, d)
    inputs.scale_channels(S, inputs.outlier_channels(seed, HV, d, 8), 10.0)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, n_slots, HV, fmt=_fmt(had))
    live = (slots >= 0) & (slots < n_slots)
    orc.pack(ref, 0, slots[live], S[live], perm)
    gpool = gpu_pool_from(ref, D)
    inp = inputs.step(inputs.decode_inputs(seed, 1, B, HK, HV, d, kda=kda), 0)
    o_gpu, o_ref = _step(kda, ref, gpool, slots, inp, perm, scale=1.0)
    assert np.all(o_gpu[~live] == 0) and np.all(o_ref[~live] == 0)
    err = rel_l2(o_gpu, o_ref)
    stats = compare_tiles(gpool.buffer.cpu().numpy(), ref, f"paper many tiles kda={kda}")
    _say(f"  o rel-L2 {err:.2e}  {stats}")
    assert err <= 1e-4
