"""Pins of the oracle's other low-tier formats of App. A.1's format table:
INT4 (with and without H32), FP8 E4M3 with one fp32 scale per 32 values
(Eq. (16)), and NVFP4 (E2M1 in blocks of 16 with an E4M3 block scale and an
fp32 global scale), each with an FP16 high tier (CPU only).

Independent references: torch's float8_e4m3fn cast, a brute-force search of
the E2M1 grid, the quantizers' reconstruction bounds, the table's bits per
value, and the error recurrence of Eq. (5).
"""
import numpy as np
import pytest
import torch

from oracle import brute
from oracle import oracle as orc
from paper_2608_27513_amd import inputs

E2M1_GRID = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def _ties_e4m3(rng, n):
    """Exact midpoints between neighbouring positive E4M3 values."""
    codes = rng.integers(1, 0x7E, n).astype(np.uint8)
    lo = torch.from_numpy(codes).view(torch.float8_e4m3fn).float().numpy().astype(np.float64)
    hi = torch.from_numpy(codes + 1).view(torch.float8_e4m3fn).float().numpy().astype(np.float64)
    return ((lo + hi) / 2).astype(np.float32)


def test_e4m3_matches_torch():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal(200000) * 10.0 ** rng.uniform(-4, 2.6, 200000)).astype(np.float32)
    x = np.clip(x, -448, 448)
    t = _ties_e4m3(rng, 20000)
    x = np.concatenate([x, t, -t, np.float32([0.0, -0.0, 448.0, -448.0, 2.0 ** -9, 2.0 ** -10,
                                              3 * 2.0 ** -11, 2.0 ** -6, 1e-30])])
    want = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(orc.e4m3_round(x), want)
    back = torch.from_numpy(want).view(torch.float8_e4m3fn).float().numpy()
    assert np.array_equal(orc.e4m3_widen(want), back)
    assert np.all(orc.e4m3_round(np.float32([460.0, 1e6, -500.0])) == [0x7E, 0x7E, 0xFE])


def test_e2m1_is_the_nearest_grid_value_ties_to_even():
    rng = np.random.default_rng(2)
    mid = (E2M1_GRID[1:] + E2M1_GRID[:-1]) / 2
    x = np.concatenate([rng.uniform(-7, 7, 50000), mid, -mid, [0.0, 6.0, 6.5, 100.0]])
    x = x.astype(np.float32)
    c = orc.e2m1_round(x)
    got = orc.e2m1_widen(c)
    a = np.minimum(np.abs(x.astype(np.float64)), 6.0)
    d = np.abs(a[:, None] - E2M1_GRID[None, :])
    best = d.min(1, keepdims=True)
    cand = d == best
    # ties go to the even mantissa: grid positions 0, 2, 4, 6 (0, 1, 2, 4)
    even = cand & (np.arange(8)[None, :] % 2 == 0)
    idx = np.where(cand.sum(1) > 1, even.argmax(1), cand.argmax(1))
    want = np.copysign(E2M1_GRID[idx], x)
    assert np.array_equal(np.abs(got), np.abs(want).astype(np.float32))
    assert np.all((c & 0x7) == idx)
    assert np.all(np.signbit(got[got != 0]) == np.signbit(x[got != 0]))


def _groups(seed, n, size=32):
    rng = np.random.default_rng(seed)
    g = rng.standard_normal((n, size)) * 10.0 ** rng.uniform(-3, 2, (n, 1))
    g += rng.standard_normal((n, 1)) * 0.3 * np.abs(g).max(1, keepdims=True)
    return g.astype(np.float32)


def test_int4_group_quantizer():
    """Eq. (3) with b = 4: FP16 (s, z), codes in [0, 15], the minimum on code
    0, every unsaturated entry within s/2."""
    for x in _groups(3, 2000):
        c, s, z = orc.quant_group_fp16_u4(x)
        assert np.float32(np.float16(s)) == s and np.float32(np.float16(z)) == z
        assert c.max() <= 15
        xr = s * (c.astype(np.float32) - z)
        inside = (c > 0) & (c < 15)
        err = np.abs(xr.astype(np.float64) - x)
        assert np.all(err[inside] <= 0.5 * s * (1 + 1e-5) + 2 * np.spacing(np.abs(x[inside])))
        if abs(z) <= 2048:
            assert c[np.argmin(x)] == 0


def test_fp8_group_quantizer():
    """Eq. (16): s = max|x| / 448, the largest magnitude lands on +-448, and
    every entry reconstructs within half an E4M3 step of x / s."""
    for x in _groups(4, 2000):
        c, s = orc.quant_group_e4m3(x)
        assert s == np.float32(max(np.abs(x).max(), np.float32(1e-10)) / np.float32(448.0))
        q = orc.e4m3_widen(c)
        assert np.abs(q[np.argmax(np.abs(x))]) == 448.0
        y = (x / s).astype(np.float64)
        half = np.where(np.abs(y) >= 2.0 ** -6, np.abs(y) * 2.0 ** -4, 2.0 ** -10)
        assert np.all(np.abs(q - y) <= half * (1 + 1e-6) + 1e-12)
    c, s = orc.quant_group_e4m3(np.zeros(32, np.float32))
    assert np.all(c == 0) and s == np.float32(1e-10) / np.float32(448.0)


def test_nvfp4_block_quantizer():
    """The block scale is E4M3(max|x| / (6 s_g)) and every code is the E2M1
    rounding of x / (s_b s_g); a zero block scale gives zero codes."""
    rng = np.random.default_rng(5)
    for x in _groups(6, 1000, 16):
        s_g = orc.nvfp4_global(float(np.abs(x).max()) * float(rng.uniform(1, 30)))
        c, sb = orc.quant_block_e2m1(x, s_g)
        t = min(np.float32(np.abs(x).max()) / (np.float32(6.0) * s_g), np.float32(448.0))
        assert sb == orc.e4m3_round(np.float32([t]))[0]
        scale = orc.e4m3_widen(np.uint8([sb]))[0] * s_g
        if scale > 0:
            assert np.array_equal(c, orc.e2m1_round((x / scale).astype(np.float32)))
        else:
            assert np.all(c == 0)
    assert orc.nvfp4_global(0.0) == 1.0
    assert orc.nvfp4_global(2688.0) == 1.0


def test_bits_per_value_of_the_format_table():
    """App. A.1's table: INT4 5.0, FP8 9.0, NVFP4 4.5 bits per low value
    (NVFP4's per-tile global scale adds 32 bits per tile)."""
    d, k_hi = 128, 16
    hi = k_hi * d * 2
    lo_vals = (d - k_hi) * d
    for fmt, bits, tail in ((orc.FMT_INT4, 5.0, 0), (orc.FMT_INT4_H32, 5.0, 0),
                            (orc.FMT_FP8, 9.0, 0), (orc.FMT_NVFP4, 4.5, 4),
                            (orc.FMT_PAPER, 9.0, 0)):
        tb = orc.tile_bytes(orc.KIND_MIXED, d, d, k_hi, fmt)
        assert (tb - hi - tail) * 8 / lo_vals == bits, fmt
    assert orc.tile_bytes(orc.KIND_MIXED, d, d, k_hi, orc.FMT_INT4) == 13056
    assert orc.tile_bytes(orc.KIND_MIXED, d, d, k_hi, orc.FMT_FP8) == 20224
    assert orc.tile_bytes(orc.KIND_MIXED, d, d, k_hi, orc.FMT_NVFP4) == 12164


NEW = [orc.FMT_INT4, orc.FMT_INT4_H32, orc.FMT_FP8, orc.FMT_NVFP4]


@pytest.mark.parametrize("fmt", NEW)
def test_pack_layout(fmt):
    """Byte layout: FP16 high rows, 4-bit codes two per byte (even column in
    the low nibble) or one byte per code, per-row metadata group by group,
    then NVFP4's global scale; every group decodes as its quantizer says."""
    d, k_hi, B, HV = 64, 8, 2, 2
    _, group, _, had, code = orc.fmt5(fmt)
    S = inputs.synthetic_states(30, B, HV, d)
    inputs.scale_channels(S, inputs.outlier_channels(30, HV, d, 4), 10.0)
    perm = inputs.random_perms(31, HV, d)
    pool = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B, HV, fmt=fmt)
    slots = np.arange(B, dtype=np.int32)
    orc.pack(pool, 0, slots, S, perm)
    R = orc.unpack(pool, 0, slots, perm)
    nib = code in (orc.CODE_U4, orc.CODE_E2M1)
    crow = d // 2 if nib else d
    mrow = {orc.CODE_U4: d // 32 * 4, orc.CODE_E4M3: d // 32 * 4, orc.CODE_E2M1: d // 16}[code]
    for b in range(B):
        for h in range(HV):
            tile = pool.tile(0, b, h)
            codes = tile[k_hi * d * 2:k_hi * d * 2 + (d - k_hi) * crow].reshape(d - k_hi, crow)
            meta = tile[k_hi * d * 2 + (d - k_hi) * crow:][:(d - k_hi) * mrow].reshape(d - k_hi, mrow)
            lo_rows = S[b, h][perm[h][k_hi:]]
            s_g = None
            if code == orc.CODE_E2M1:
                s_g = orc.nvfp4_global(float(np.abs(lo_rows).max()))
                assert tile[-4:].view(np.float32)[0] == s_g
            for r in range(k_hi, d):
                u = perm[h, r]
                x = S[b, h, u]
                cr = codes[r - k_hi]
                c_all = np.stack([cr & 0xF, cr >> 4], 1).ravel() if nib else cr
                for g in range(d // group):
                    xg = x[group * g:group * (g + 1)]
                    cg = c_all[group * g:group * (g + 1)]
                    rec = R[b, h, u, group * g:group * (g + 1)]
                    if code == orc.CODE_U4:
                        yg = orc.hadamard32(xg) if had else xg
                        c, s, z = orc.quant_group_fp16_u4(yg)
                        assert np.array_equal(cg, c)
                        assert np.array_equal(meta[r - k_hi, 4 * g:4 * g + 4].view(np.uint16),
                                              np.float16([s, z]).view(np.uint16))
                        want = s * (c.astype(np.float32) - z)
                        if had:
                            want = orc.hadamard32(want)
                        assert np.array_equal(rec, want)
                    elif code == orc.CODE_E4M3:
                        c, s = orc.quant_group_e4m3(xg)
                        assert np.array_equal(cg, c)
                        assert meta[r - k_hi, 4 * g:4 * g + 4].view(np.float32)[0] == s
                        assert np.array_equal(rec, s * orc.e4m3_widen(c))
                    else:
                        c, sb = orc.quant_block_e2m1(xg, s_g)
                        assert np.array_equal(cg, c) and meta[r - k_hi, g] == sb
                        scale = orc.e4m3_widen(np.uint8([sb]))[0] * s_g
                        assert np.array_equal(rec, orc.e2m1_widen(c) * scale)


@pytest.mark.parametrize("fmt", NEW)
@pytest.mark.parametrize("kda", [False, True])
def test_error_recurrence_with_each_format(fmt, kda):
    """Section 3.3 Eq. (5) for every low tier: with R_t = Q(x_t) - x_t,
    Delta S_t = A_t Delta S_{t-1} + R_t along the oracle's trajectory."""
    d, T, k_hi = 64, 12, 8
    inp = inputs.decode_inputs(32 + kda, T, 1, 1, 1, d, kda=kda)
    perm = inputs.random_perms(34, 1, d)
    pool = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, 1, 1, fmt=fmt)
    orc.reset(pool, 0, [0])
    assert np.all(orc.unpack(pool, 0, [0], perm) == 0)
    inv = np.argsort(perm[0])
    S_ref = np.zeros((d, d))
    dS_prev = np.zeros((d, d))
    for t in range(T):
        st = inputs.step(inp, t)
        _, pre = orc.update(pool, 0, [0], kda=kda, perm=perm, want_pre=True, **st)
        Sq = orc.unpack(pool, 0, [0], perm)[0, 0].astype(np.float64)
        R = Sq - pre[0, 0][inv].astype(np.float64)
        q, k, v, lam, beta = brute.head_inputs(inp, t, 0, 0, 1, 1, kda)
        A = brute.transition(k, lam, beta)
        S_ref = A @ S_ref + beta * np.outer(k, v)
        dS = Sq - S_ref
        assert np.linalg.norm(dS - (A @ dS_prev + R)) <= 1e-3 * np.linalg.norm(dS)
        dS_prev = dS


def _nvfp4_tile(S, k_hi):
    """Packs one natural-order tile [d, d] in NVFP4 and returns the low tier's
    codes (one E2M1 code per value, [d - k_hi, d]), its E4M3 block-scale
    bytes ([d - k_hi, d / 16]), the fp32 global scale and the reconstruction."""
    d = S.shape[0]
    pool = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, 1, 1, fmt=orc.FMT_NVFP4)
    orc.pack(pool, 0, [0], S[None, None])
    nl = d - k_hi
    t = pool.buf
    c0 = k_hi * d * 2
    packed = t[c0:c0 + nl * d // 2].reshape(nl, d // 2)
    codes = np.empty((nl, d), np.uint8)
    codes[:, 0::2] = packed & 0x0F  # the even column in the low nibble
    codes[:, 1::2] = packed >> 4
    m0 = c0 + nl * d // 2
    sb = t[m0:m0 + nl * d // 16].reshape(nl, d // 16)
    sg = t[m0 + nl * d // 16:m0 + nl * d // 16 + 4].copy().view(np.float32)[0]
    rec = orc.unpack(pool, 0, [0])[0, 0]
    return codes, sb, sg, rec


def _wide_tiles(seed, n, d):
    """Tiles whose rows span many octaves, with a few large outliers."""
    rng = np.random.default_rng(seed)
    for _ in range(n):
        S = rng.standard_normal((d, d)).astype(np.float32)
        S *= np.exp2(rng.uniform(-12, 12, size=(d, 1))).astype(np.float32)
        idx = rng.integers(0, d, size=(3, 2))
        S[idx[:, 0], idx[:, 1]] *= np.float32(rng.uniform(20, 200))
        yield S


def test_nvfp4_scale_rule_properties():
    """Properties of NVFP4's two-level scale that fix its constants without
    restating them (App. A.1's format table: E2M1 values whose largest
    magnitude is 6, E4M3 block scales whose largest finite value is 448, one
    fp32 global scale): the tile's largest magnitude uses the whole range of
    both, so its block scale is 448, its code is +-6 and it reconstructs to
    itself; every block's largest magnitude is coded +-6; every block scale
    is a finite E4M3 value; every value
    reconstructs within one E2M1 step (at most 1 in units of its block's
    scale) of itself, saturation included; and scaling a tile by a power of
    two scales only the global scale."""
    d, k_hi = 64, 8
    for S in _wide_tiles(41, 12, d):
        codes, sb, sg, rec = _nvfp4_tile(S, k_hi)
        lo, rec_lo = S[k_hi:], rec[k_hi:]
        i, j = np.unravel_index(np.argmax(np.abs(lo)), lo.shape)
        amax = np.abs(lo[i, j])
        assert orc.e4m3_widen(sb[i, j // 16:j // 16 + 1])[0] == 448.0
        assert codes[i, j] & 0x7 == 0x7 and (codes[i, j] >> 3) == (lo[i, j] < 0)
        assert abs(abs(rec_lo[i, j]) - amax) <= 4 * np.spacing(amax)
        assert orc.e4m3_widen(sb).max() == 448.0
        assert np.all((sb & 0x7F) != 0x7F)  # no E4M3 NaN
        block = np.repeat(orc.e4m3_widen(sb).astype(np.float64) * sg, 16, axis=1)
        err = np.abs(rec_lo.astype(np.float64) - lo)
        normal = block >= 2.0 ** -6 * sg  # E4M3 normal block scales
        assert np.all(err[normal] <= block[normal] * (1 + 1e-6))
        # each block's scale spans the E2M1 range: its largest magnitude is
        # coded +-6 (within E4M3's rounding of the scale, 6 / (1 +- 2^-4)
        # still rounds to 6), wherever that scale is a normal E4M3 value
        blocks = np.abs(lo).reshape(d - k_hi, d // 16, 16)
        top = np.argmax(blocks, axis=2)
        top_codes = np.take_along_axis(codes.reshape(d - k_hi, d // 16, 16), top[..., None],
                                       axis=2)[..., 0]
        sbv = orc.e4m3_widen(sb)
        live = (sbv >= 2.0 ** -6) & (blocks.max(axis=2) > 0)
        assert live.sum() >= 32
        assert np.all(top_codes[live] & 0x7 == 0x7)
        for k in (-7, 5):
            codes2, sb2, sg2, _ = _nvfp4_tile(S * np.float32(2.0 ** k), k_hi)
            assert np.array_equal(codes2, codes) and np.array_equal(sb2, sb)
            assert sg2 == sg * np.float32(2.0 ** k)
