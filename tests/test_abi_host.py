"""Host-side checks of libdamp: exports, layout arithmetic, argument validation.

No GPU needed: every call here either is pure host arithmetic or fails
validation before anything is enqueued.
"""
import ctypes
import json
import os
import re

import numpy as np
import pytest
import scipy.stats

from oracle import oracle as orc
from paper_2608_27513_amd import damp as D

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "damp.h")
GOLDEN = os.path.join(ROOT, "tests", "golden", "paper_numbers.json")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(D.LIB_PATH):
        from paper_2608_27513_amd import build
        build.build()
    return D.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(damp_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert len(names) == 24
    for n in names:
        assert hasattr(L, n), n
    assert sorted(D.EXPORTS) == names


@pytest.mark.parametrize("d", [16, 32, 64, 128])
def test_tile_geometry_matches_oracle(L, d):
    for kind in (D.DAMP_STATE_FP32, D.DAMP_STATE_MIXED):
        for k_hi in sorted({0, 1, 4, 8, d // 8, d // 4, d}):
            lay = D.damp_layout_init(d, d, k_hi, kind)
            ok = k_hi if kind == D.DAMP_STATE_MIXED else 0
            assert D.damp_tile_bytes(lay) == orc.tile_bytes(kind, d, d, ok)
            assert D.damp_tile_stride(lay) == orc.tile_stride(kind, d, d, ok)
            bits = D.damp_bits_per_value(lay)
            assert bits == orc.tile_bytes(kind, d, d, ok) * 8 / (d * d)
    if d >= 32:  # the paper's tiers: groups of 32 along d_v
        for k_hi in sorted({0, 8, d // 4, d}):
            lay = D.damp_layout_init(d, d, k_hi, D.DAMP_STATE_MIXED)
            lay.hi_dtype, lay.group, lay.meta_dtype, lay.hadamard = orc.FMT_PAPER
            assert D.damp_tile_bytes(lay) == orc.tile_bytes(D.DAMP_STATE_MIXED, d, d, k_hi,
                                                            orc.FMT_PAPER)
            assert D.damp_tile_stride(lay) == orc.tile_stride(D.DAMP_STATE_MIXED, d, d, k_hi,
                                                              orc.FMT_PAPER)


@pytest.mark.parametrize("fmt,bits", [(orc.FMT_INT4, 5.0), (orc.FMT_INT4_H32, 5.0),
                                      (orc.FMT_FP8, 9.0), (orc.FMT_NVFP4, 4.5)])
def test_table_format_geometry(L, fmt, bits):
    """The other rows of App. A.1's format table: tile bytes equal the
    oracle's and the low tier costs the table's bits per value."""
    for d in (32, 64, 128):
        for k_hi in sorted({0, 8, d // 4, d}):
            lay = D.damp_layout_init(d, d, k_hi, D.DAMP_STATE_MIXED)
            lay.hi_dtype, lay.group, lay.meta_dtype, lay.hadamard, lay.code_dtype = fmt
            assert D.damp_tile_bytes(lay) == orc.tile_bytes(D.DAMP_STATE_MIXED, d, d, k_hi, fmt)
            assert D.damp_tile_stride(lay) == orc.tile_stride(D.DAMP_STATE_MIXED, d, d, k_hi, fmt)
            if k_hi == 0:
                assert D.damp_bits_per_value(lay) == bits
    lay = D.damp_layout_init(16, 16, 4, D.DAMP_STATE_MIXED)
    lay.hi_dtype, lay.group, lay.meta_dtype, lay.hadamard, lay.code_dtype = fmt
    if fmt[1] > 16:  # a group wider than d_v: not a layout
        assert L.damp_tile_bytes(ctypes.byref(lay)) == 0
    else:            # a layout, but the kernels need d_v >= 32
        pool = _fake_pool(L, lay)
        p = ctypes.c_void_p(0x7f0000100000)
        assert L.damp_state_pack(ctypes.byref(pool), 0, p, 4, p, None, None) == \
            D.DAMP_ERR_UNSUPPORTED
    bad = D.damp_layout_init(64, 64, 8, D.DAMP_STATE_MIXED)
    bad.code_dtype = D.DAMP_DT_E2M1  # E2M1 codes with fp32 (s, z) pairs: not a format
    assert L.damp_tile_bytes(ctypes.byref(bad)) == 0


def test_bits_per_value_of_the_paper_layout(L):
    gold = json.load(open(GOLDEN))["damp_bits_per_value"]
    lay = D.damp_layout_init(128, 128, 16, D.DAMP_STATE_MIXED)
    lay.hi_dtype = D.DAMP_DT_FP16
    lay.group = 32
    lay.meta_dtype = D.DAMP_DT_FP16
    lay.hadamard = 1
    assert D.damp_bits_per_value(lay) == gold["value"]
    # 16 fp16 rows + 112 code rows + 112 * 4 groups * 2 fp16 words
    assert D.damp_tile_bytes(lay) == 16 * 256 + 112 * 128 + 112 * 4 * 4 == 20224


def test_default_layout_numbers(L):
    lay = D.damp_layout_init(128, 128, 16)
    assert D.damp_tile_bytes(lay) == 19328 and D.damp_tile_stride(lay) == 19328
    assert D.damp_bits_per_value(lay) == 9.4375
    assert D.damp_pool_required_bytes(lay, 48, 512, 32) == 48 * 512 * 32 * 19328
    fp = D.damp_layout_init(128, 128, 0, D.DAMP_STATE_FP32)
    assert D.damp_pool_required_bytes(fp, 30, 256, 32) == 15 * 2 ** 30


def _status(fn, *args):
    st = fn(*args)
    return st, D.lib().damp_last_error().decode()


def test_layout_validation(L):
    lay = D.damp_layout()
    st, msg = _status(L.damp_layout_init, ctypes.byref(lay), 128, 128, 129, 1)
    assert st == D.DAMP_ERR_INVALID_ARG and "k_hi" in msg
    st, msg = _status(L.damp_layout_init, ctypes.byref(lay), 0, 128, 0, 1)
    assert st == D.DAMP_ERR_INVALID_ARG
    st, msg = _status(L.damp_layout_init, ctypes.byref(lay), 128, 128, 0, 7)
    assert st == D.DAMP_ERR_INVALID_ARG and "kind" in msg
    assert L.damp_tile_bytes(None) == 0 and L.damp_bits_per_value(None) < 0


def test_pool_validation(L):
    lay = D.damp_layout_init(128, 128, 16)
    pool = D.damp_pool()
    need = D.damp_pool_required_bytes(lay, 2, 4, 8)
    fake = ctypes.c_void_p(0x7f0000000000)  # never dereferenced: every call below fails first
    st, msg = _status(L.damp_pool_init, ctypes.byref(pool), ctypes.byref(lay), 2, 4, 8, None, need)
    assert st == D.DAMP_ERR_INVALID_ARG and "NULL" in msg
    st, msg = _status(L.damp_pool_init, ctypes.byref(pool), ctypes.byref(lay), 2, 4, 8,
                      ctypes.c_void_p(0x7f0000000010), need)
    assert st == D.DAMP_ERR_INVALID_ARG and "aligned" in msg
    st, msg = _status(L.damp_pool_init, ctypes.byref(pool), ctypes.byref(lay), 2, 4, 8, fake,
                      need - 1)
    assert st == D.DAMP_ERR_INVALID_ARG and "needs" in msg
    st, _ = _status(L.damp_pool_init, ctypes.byref(pool), ctypes.byref(lay), 0, 4, 8, fake, need)
    assert st == D.DAMP_ERR_INVALID_ARG
    st, _ = _status(L.damp_pool_init, ctypes.byref(pool), ctypes.byref(lay), 2, 4, 8, fake, need)
    assert st == D.DAMP_OK and pool.tile_stride == 19328 and pool.bytes == need


def _fake_pool(L, layout, layers=2, slots=4, hv=8):
    pool = D.damp_pool()
    need = D.damp_pool_required_bytes(layout, layers, slots, hv)
    assert L.damp_pool_init(ctypes.byref(pool), ctypes.byref(layout), layers, slots, hv,
                            ctypes.c_void_p(0x7f0000000000), need) == 0
    return pool


def test_update_validation_fails_before_launch(L):
    lay = D.damp_layout_init(128, 128, 16)
    pool = _fake_pool(L, lay)
    p = ctypes.c_void_p(0x7f0000100000)  # never dereferenced
    for fn in (L.damp_state_update_gdn, L.damp_state_update_kda):
        args = [ctypes.byref(pool), 0, p, 4, 4, p, p, p, p, p, p, 1.0, p, D.DAMP_DT_FP32, None]
        bad = dict(layer=(1, 2), B=(3, -1), hk=(4, 3), odt=(13, 7))
        for name, (i, val) in bad.items():
            a = list(args)
            a[i] = val
            st, msg = _status(fn, *a)
            assert st == D.DAMP_ERR_INVALID_ARG, name
            assert msg
        a = list(args)
        a[3] = 0  # B = 0 is a no-op
        assert fn(*a) == D.DAMP_OK
        a = list(args)
        a[5] = None  # q
        assert fn(*a) == D.DAMP_ERR_INVALID_ARG
        assert fn(None, *args[1:]) == D.DAMP_ERR_INVALID_ARG


def test_prefill_validation_fails_before_launch(L):
    lay = D.damp_layout_init(64, 64, 8)
    pool = _fake_pool(L, lay)
    p = ctypes.c_void_p(0x7f0000100000)  # never dereferenced
    for fn in (L.damp_state_prefill_gdn, L.damp_state_prefill_kda):
        args = [ctypes.byref(pool), 0, p, 4, 3, 4, p, p, p, p, p, p, 1.0, p, D.DAMP_DT_FP32, None]
        bad = dict(layer=(1, 2), B=(3, -1), T=(4, -2), hk=(5, 3), odt=(14, 7))
        for name, (i, val) in bad.items():
            a = list(args)
            a[i] = val
            st, msg = _status(fn, *a)
            assert st == D.DAMP_ERR_INVALID_ARG, name
            assert msg
        for i in (3, 4):  # B = 0 or T = 0 is a no-op
            a = list(args)
            a[i] = 0
            assert fn(*a) == D.DAMP_OK
        a = list(args)
        a[10] = None  # beta
        assert fn(*a) == D.DAMP_ERR_INVALID_ARG
        a = list(args)
        a[13] = ctypes.c_void_p(0x7f0000100008)  # o must be 16-byte aligned
        st, msg = _status(fn, *a)
        assert st == D.DAMP_ERR_INVALID_ARG and "aligned" in msg


def test_layouts_without_kernels_are_reported(L):
    lay = D.damp_layout_init(128, 128, 16)
    lay.group = 32  # groups of 32 with a BF16 tier and fp32 metadata: no kernel
    pool = _fake_pool(L, lay)
    p = ctypes.c_void_p(0x7f0000100000)
    st, msg = _status(L.damp_state_update_gdn, ctypes.byref(pool), 0, p, 4, 4, p, p, p, p, p,
                      None, 1.0, p, 0, None)
    assert st == D.DAMP_ERR_UNSUPPORTED and "no kernel" in msg
    st, _ = _status(L.damp_state_pack, ctypes.byref(pool), 0, p, 4, p, None, None)
    assert st == D.DAMP_ERR_UNSUPPORTED
    lay = D.damp_layout_init(96, 96, 16)  # valid layout, no kernel width
    pool = _fake_pool(L, lay)
    st, _ = _status(L.damp_state_unpack, ctypes.byref(pool), 0, p, 4, None, p, None)
    assert st == D.DAMP_ERR_UNSUPPORTED
    lay = D.damp_layout_init(16, 16, 4)  # the paper's tiers need d_v >= 32
    lay.hi_dtype, lay.group, lay.meta_dtype, lay.hadamard = (D.DAMP_DT_FP16, 16, D.DAMP_DT_FP16, 0)
    pool = _fake_pool(L, lay)
    st, _ = _status(L.damp_state_pack, ctypes.byref(pool), 0, p, 4, p, None, None)
    assert st == D.DAMP_ERR_UNSUPPORTED


def test_pack_reset_validation(L):
    lay = D.damp_layout_init(64, 64, 8)
    pool = _fake_pool(L, lay)
    p = ctypes.c_void_p(0x7f0000100000)
    assert L.damp_state_pack(ctypes.byref(pool), 2, p, 4, p, None, None) == D.DAMP_ERR_INVALID_ARG
    assert L.damp_state_pack(ctypes.byref(pool), 0, None, 4, p, None, None) == D.DAMP_ERR_INVALID_ARG
    assert L.damp_state_unpack(ctypes.byref(pool), 0, p, 4, None, None, None) == \
        D.DAMP_ERR_INVALID_ARG
    assert L.damp_pool_reset_slots(ctypes.byref(pool), 5, p, 1, None) == D.DAMP_ERR_INVALID_ARG
    assert L.damp_pool_reset_slots(ctypes.byref(pool), -1, p, 0, None) == D.DAMP_OK


def test_duplicate_slots_are_rejected(L):
    """Two requests of one batch sharing a slot would race on its tiles
    (every tile is read and written in place): damp_check_slots finds the
    repeat among host slot ids; padded and out-of-range entries are not
    slots of the pool and may repeat."""
    pool = _fake_pool(L, D.damp_layout_init(128, 128, 16), slots=64)

    def check(ids):
        arr = (ctypes.c_int32 * max(1, len(ids)))(*ids)
        return _status(L.damp_check_slots, ctypes.byref(pool), arr, len(ids), 0, None)

    assert check([3, 1, 2, 0])[0] == D.DAMP_OK
    assert check([])[0] == D.DAMP_OK
    assert check([-1, 5, -1, 64, 64, 70, -7])[0] == D.DAMP_OK  # padding only repeats
    st, msg = check([4, 9, 63, 2, 9])
    assert st == D.DAMP_ERR_INVALID_ARG and "slot 9" in msg
    st, msg = check([0, 1, 2, 3, 4, 5, 6, 7, 0])
    assert st == D.DAMP_ERR_INVALID_ARG and "slot 0" in msg
    rng = np.random.default_rng(3)
    ids = rng.permutation(64).astype(np.int32).tolist()
    assert check(ids)[0] == D.DAMP_OK
    ids[40] = ids[7]
    st, msg = check(ids)
    assert st == D.DAMP_ERR_INVALID_ARG and f"slot {ids[7]}" in msg
    assert L.damp_check_slots(ctypes.byref(pool), None, 4, 0, None) == D.DAMP_ERR_INVALID_ARG
    assert L.damp_check_slots(ctypes.byref(pool), None, 0, 0, None) == D.DAMP_OK
    assert L.damp_check_slots(None, None, 0, 0, None) == D.DAMP_ERR_INVALID_ARG


def test_select_validation(L):
    p = ctypes.c_void_p(0x7f0000100000)
    f = L.damp_select_channels
    assert f(0, 4, 2, 128, 128, p, p, None, 129, 1e-4, p, p, None, None) == D.DAMP_ERR_INVALID_ARG
    assert f(0, 4, 2, 128, 128, p, p, None, 16, 0.0, p, p, None, None) == D.DAMP_ERR_INVALID_ARG
    assert f(0, 0, 2, 128, 128, p, p, None, 16, 1e-4, p, p, None, None) == D.DAMP_ERR_INVALID_ARG
    assert f(0, 4, 2, 300, 128, p, p, None, 16, 1e-4, p, p, None, None) == D.DAMP_ERR_INVALID_ARG
    assert f(0, 4, 2, 128, 128, None, p, None, 16, 1e-4, p, p, None, None) == \
        D.DAMP_ERR_INVALID_ARG


def test_select_noalloc_refuses_calls_beyond_its_scratch(L):
    """The no-allocation selection keeps (N + 2) * H * d_k doubles in a fixed
    16 MiB array: larger calls fail before anything runs, with the limit in
    the message; its argument checks are those of damp_select_channels."""
    p = ctypes.c_void_p(0x7f0000100000)  # never dereferenced
    f = L.damp_select_channels_noalloc
    assert (254 + 2) * 64 * 128 == 2 ** 21  # the largest N at H = 64, d_k = 128
    st, msg = _status(f, 1, 255, 64, 128, 128, p, p, None, 16, 1e-4, p, p, None, None)
    assert st == D.DAMP_ERR_INVALID_ARG and "scratch" in msg and "2097152" in msg
    st, msg = _status(f, 0, 100000, 32, 128, 128, p, p, None, 16, 1e-4, p, p, None, None)
    assert st == D.DAMP_ERR_INVALID_ARG and "scratch" in msg
    assert f(0, 4, 2, 128, 128, p, p, None, 129, 1e-4, p, p, None, None) == D.DAMP_ERR_INVALID_ARG
    assert f(0, 4, 2, 128, 128, None, p, None, 16, 1e-4, p, p, None, None) == \
        D.DAMP_ERR_INVALID_ARG


def test_select_low_tier_argument(L):
    """Q_lo of the selection is the low tier of `lo` (App. A.2): the per-row
    tier or the paper's UINT8 group tier; other formats, another shape or an
    FP32 layout are refused before anything runs."""
    p = ctypes.c_void_p(0x7f0000100000)  # never dereferenced
    f = L.damp_select_channels

    def tier(d, fmt):
        lo = D.damp_layout_init(d, d, 0)
        if fmt is not None:
            lo.hi_dtype, lo.group, lo.meta_dtype, lo.hadamard, lo.code_dtype = fmt
        return lo

    paper = (D.DAMP_DT_FP16, 32, D.DAMP_DT_FP16, 1, D.DAMP_DT_U8)
    int4 = (D.DAMP_DT_FP16, 32, D.DAMP_DT_FP16, 0, D.DAMP_DT_U4)
    fp8 = (D.DAMP_DT_FP16, 32, D.DAMP_DT_FP32, 0, D.DAMP_DT_E4M3)
    for lo in (tier(128, int4), tier(128, fp8), tier(64, paper),
               D.damp_layout_init(128, 128, 0, D.DAMP_STATE_FP32)):
        st, msg = _status(f, 0, 4, 2, 128, 128, p, p, ctypes.byref(lo), 16, 1e-4, p, p, None, None)
        assert st == D.DAMP_ERR_UNSUPPORTED and "Q_lo" in msg
    big = tier(256, paper)  # groups of 32 are evaluated by one wave per row: d_v <= 128
    assert f(0, 4, 2, 256, 256, p, p, ctypes.byref(big), 16, 1e-4, p, p, None, None) == \
        D.DAMP_ERR_UNSUPPORTED
    # invalid sizes are reported before the layout is looked at
    assert f(0, 0, 2, 128, 128, p, p, ctypes.byref(tier(128, int4)), 16, 1e-4, p, p, None,
             None) == D.DAMP_ERR_INVALID_ARG


def test_split_agreement_functions_match_scipy(L):
    """damp_spearman / damp_topk_overlap (host code of the library) against
    scipy's Spearman correlation and a set intersection."""
    rng = np.random.default_rng(5)
    for n in (2, 9, 128):
        a = rng.standard_normal(n)
        b = 0.5 * a + rng.standard_normal(n)
        assert abs(D.damp_spearman(a, b) - scipy.stats.spearmanr(a, b).statistic) <= 1e-12
    a = np.array([3.0, 1.0, 1.0, 2.0, 2.0, 2.0, 8.0])
    b = np.array([1.0, 1.0, 4.0, 4.0, 0.5, 9.0, 9.0])
    assert abs(D.damp_spearman(a, b) - scipy.stats.spearmanr(a, b).statistic) <= 1e-12
    assert np.isnan(D.damp_spearman(np.ones(5), a[:5]))
    for k in (1, 4, 16):
        x = rng.permutation(128)[:k].astype(np.int32)
        y = rng.permutation(128)[:k].astype(np.int32)
        assert D.damp_topk_overlap(x, y) == len(set(x) & set(y)) / k
    assert np.isnan(L.damp_topk_overlap(None, None, 4))


def test_calib_validation_fails_before_launch(L):
    lo = D.damp_layout_init(128, 128, 16)
    cal = D.damp_calib()
    p = ctypes.c_void_p(0x7f0000100000)  # never dereferenced
    need = L.damp_calib_required_bytes(2, 32, 128)
    assert need == 8 * 2 * (3 * 32 * 128 + 1)
    assert L.damp_calib_required_bytes(0, 32, 128) == 0
    st, msg = _status(L.damp_calib_init, ctypes.byref(cal), ctypes.byref(lo), 0, 32, 2, p, need - 8,
                      None)
    assert st == D.DAMP_ERR_INVALID_ARG and "need" in msg
    st, _ = _status(L.damp_calib_init, ctypes.byref(cal), ctypes.byref(lo), 0, 32, 65, p, need, None)
    assert st == D.DAMP_ERR_INVALID_ARG
    fp = D.damp_layout_init(128, 128, 0, D.DAMP_STATE_FP32)
    st, _ = _status(L.damp_calib_init, ctypes.byref(cal), ctypes.byref(fp), 0, 32, 2, p, need, None)
    assert st == D.DAMP_ERR_INVALID_ARG
    odd = D.damp_layout_init(128, 128, 16)
    odd.group = 32  # grouped with fp32 metadata: no kernel
    st, _ = _status(L.damp_calib_init, ctypes.byref(cal), ctypes.byref(odd), 0, 32, 2, p, need, None)
    assert st == D.DAMP_ERR_UNSUPPORTED
    # a descriptor filled by hand, as damp_calib_init would (no launch below)
    cal.lo, cal.is_kda, cal.num_heads, cal.num_domains = lo, 0, 32, 2
    cal.sums, cal.bytes = p, need
    pool = _fake_pool(L, D.damp_layout_init(128, 128, 0, D.DAMP_STATE_FP32), hv=32)
    mixed = _fake_pool(L, lo, hv=32)
    acc = L.damp_calib_accumulate
    assert acc(ctypes.byref(cal), 2, ctypes.byref(pool), 0, p, 4, None, p, None) == \
        D.DAMP_ERR_INVALID_ARG  # domain out of range
    st, msg = _status(acc, ctypes.byref(cal), 0, ctypes.byref(mixed), 0, p, 4, None, p, None)
    assert st == D.DAMP_ERR_INVALID_ARG and "FP32" in msg
    assert acc(ctypes.byref(cal), 0, ctypes.byref(pool), 0, None, 4, None, p, None) == \
        D.DAMP_ERR_INVALID_ARG
    assert acc(ctypes.byref(cal), 0, ctypes.byref(pool), 0, p, 0, None, p, None) == D.DAMP_OK
    seq = L.damp_calibrate_sequence
    args = [ctypes.byref(cal), 0, ctypes.byref(pool), 0, p, 4, 64, 8, 16, p, p, p, p, p, None]
    for i, val in ((6, -1), (7, 0), (8, 5)):  # T, stride, num_k_heads
        a = list(args)
        a[i] = val
        assert seq(*a) == D.DAMP_ERR_INVALID_ARG, i
    a = list(args)
    a[6] = 0
    assert seq(*a) == D.DAMP_OK
    sel = (ctypes.c_int32 * (32 * 16))()
    perm = (ctypes.c_uint8 * (32 * 128))()
    fin = L.damp_calib_finalize
    assert fin(ctypes.byref(cal), 7, 16, 1e-4, None, sel, perm, None, None, None) == \
        D.DAMP_ERR_INVALID_ARG
    assert fin(ctypes.byref(cal), 0, 129, 1e-4, None, sel, perm, None, None, None) == \
        D.DAMP_ERR_INVALID_ARG
    assert fin(ctypes.byref(cal), 0, 16, 0.0, None, sel, perm, None, None, None) == \
        D.DAMP_ERR_INVALID_ARG
    assert fin(ctypes.byref(cal), D.DAMP_SEL_RANDOM, 16, 1e-4, None, sel, perm, None, None,
               None) == D.DAMP_ERR_INVALID_ARG
