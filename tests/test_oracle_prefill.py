"""Pins of the oracle's prefill path (App. A.5): a chunk of T tokens runs the
recurrence of Eq. (1) in fp32 and stores only the chunk-final state (CPU only).

References: the float64 brute force of oracle/brute.py, and the quantizer's
reconstruction bound for the single re-encoding at the end of the chunk.
"""
import numpy as np
import pytest

from oracle import brute
from oracle import oracle as orc
from paper_2608_27513_amd import inputs


def _rows_to_natural(tile_order, perm_h):
    out = np.empty_like(tile_order)
    out[perm_h] = tile_order
    return out


@pytest.mark.parametrize("kda,HK,HV", [(False, 1, 2), (True, 2, 2), (False, 2, 4)])
def test_fp32_prefill_matches_the_float64_recurrence(kda, HK, HV):
    """FP32 state: every o_t and the final state equal Eq. (1) in float64."""
    d, B, T = 32, 2, 12
    S0 = inputs.synthetic_states(40 + kda, B, HV, d)
    perm = inputs.random_perms(41, HV, d)
    inp = inputs.decode_inputs(42 + HV, T, B, HK, HV, d, kda=kda)
    pool = orc.Pool(orc.KIND_FP32, d, d, 0, 1, B, HV)
    slots = np.arange(B, dtype=np.int32)
    orc.pack(pool, 0, slots, S0, perm)
    o = orc.prefill(pool, 0, slots, kda=kda, perm=perm, scale=0.5, **inputs.as_prefill(inp))
    S = orc.unpack(pool, 0, slots, perm)
    for b in range(B):
        for h in range(HV):
            states, outs = brute.trajectory(S0[b, h], inp, b, h, HK, HV, kda, scale=0.5)
            ref_o = np.stack(outs)
            assert np.linalg.norm(o[b, :, h] - ref_o) <= 1e-5 * np.linalg.norm(ref_o)
            assert np.linalg.norm(S[b, h] - states[-1]) <= 1e-5 * np.linalg.norm(states[-1])


@pytest.mark.parametrize("fmt", [None, orc.FMT_PAPER])
def test_mixed_prefill_quantizes_once_per_chunk(fmt):
    """Mixed state: the chunk starts from the stored state, runs T tokens
    without re-quantizing (o_t and the state follow the exact recurrence from
    the dequantized start), and the stored result is one re-encoding of the
    exact final state."""
    d, B, HK, HV, T, k_hi = 64, 2, 2, 2, 16, 8
    S0 = inputs.synthetic_states(43, B, HV, d)
    perm = inputs.random_perms(44, HV, d)
    inp = inputs.decode_inputs(45, T, B, HK, HV, d, kda=True)
    pool = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B, HV, fmt=fmt)
    slots = np.arange(B, dtype=np.int32)
    orc.pack(pool, 0, slots, S0, perm)
    start = orc.unpack(pool, 0, slots, perm)
    o = orc.prefill(pool, 0, slots, kda=True, perm=perm, **inputs.as_prefill(inp))
    end = orc.unpack(pool, 0, slots, perm)
    # the exact final state, stored once with the same format
    exact = np.empty_like(start)
    for b in range(B):
        for h in range(HV):
            states, outs = brute.trajectory(start[b, h], inp, b, h, HK, HV, True)
            ref_o = np.stack(outs)
            assert np.linalg.norm(o[b, :, h] - ref_o) <= 1e-5 * np.linalg.norm(ref_o)
            exact[b, h] = states[-1]
    once = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B, HV, fmt=fmt)
    orc.pack(once, 0, slots, exact.astype(np.float32), perm)
    # the codes agree but for rounding flips of the fp32 recurrence
    hb = k_hi * d * 2
    tiles_a = once.buf.reshape(-1, once.tile_stride)[:, hb:hb + (d - k_hi) * d].astype(np.int32)
    tiles_b = pool.buf.reshape(-1, pool.tile_stride)[:, hb:hb + (d - k_hi) * d].astype(np.int32)
    assert np.abs(tiles_a - tiles_b).max() <= 1
    assert (tiles_a != tiles_b).mean() <= 1e-3
    err = np.linalg.norm(end - exact) / np.linalg.norm(exact)
    err_once = np.linalg.norm(orc.unpack(once, 0, slots, perm) - exact) / np.linalg.norm(exact)
    assert err <= 1.05 * err_once + 1e-6


def test_prefill_of_one_token_is_the_decode_step():
    d, B, HK, HV, k_hi = 32, 2, 1, 2, 4
    S0 = inputs.synthetic_states(46, B, HV, d)
    inp = inputs.decode_inputs(47, 1, B, HK, HV, d)
    a = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B, HV)
    slots = np.arange(B, dtype=np.int32)
    orc.pack(a, 0, slots, S0)
    b = a.copy()
    o1 = orc.prefill(a, 0, slots, kda=False, **inputs.as_prefill(inp))
    o2 = orc.update(b, 0, slots, kda=False, **inputs.step(inp, 0))
    assert np.array_equal(o1[:, 0], o2) and np.array_equal(a.buf, b.buf)


def test_prefill_skips_padded_requests():
    d, HV, T = 32, 2, 3
    pool = orc.Pool(orc.KIND_MIXED, d, d, 4, 1, 2, HV)
    orc.pack(pool, 0, [0, 1], inputs.synthetic_states(48, 2, HV, d))
    before = pool.buf.copy()
    inp = inputs.as_prefill(inputs.decode_inputs(49, T, 2, HV, HV, d))
    o = orc.prefill(pool, 0, np.array([-1, 5], np.int32), kda=False, **inp)
    assert np.all(o == 0) and np.array_equal(pool.buf, before)
