"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Every case starts the HIP kernel and the oracle from identical packed bytes
(packed by the oracle) and identical bf16 inputs, runs both, and compares
element by element (see parity_util for the bar).
"""
import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_2608_27513_amd import damp as D
from paper_2608_27513_amd import inputs
import parity_util as pu
from parity_util import (FP32_TOL, O_TOL_MIXED, compare_tiles, dev_i32, dev_inputs, dev_u8,
                         gpu_pool_from, rel_l2)

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)


def _run_step(kda, ref, gpool, layer, slots, inp, perm, scale=1.0, o_dtype=torch.float32):
    """One step on both sides; returns (o_gpu, o_ref)."""
    d_inp = dev_inputs(inp)
    d_slots = dev_i32(slots)
    d_perm = None if perm is None else dev_u8(perm)
    B, HV, d = len(slots), ref.hv, ref.dv
    o = torch.empty((B, HV, d), dtype=o_dtype, device="cuda")
    fn = D.damp_state_update_kda if kda else D.damp_state_update_gdn
    fn(gpool, layer, d_slots, d_inp["q"], d_inp["k"], d_inp["v"], d_inp["g"], d_inp["beta"],
       perm=d_perm, scale=scale, o=o)
    o_ref = orc.update(ref, layer, slots, kda=kda, perm=perm, scale=scale, **inp)
    torch.cuda.synchronize()
    return o.float().cpu().numpy(), o_ref


CASES = [
    # (d, kda, HK, HV, B, k_hi, kind)
    (16, False, 2, 2, 1, 4, orc.KIND_MIXED),
    (16, True, 2, 2, 3, 4, orc.KIND_MIXED),
    (32, False, 1, 4, 5, 8, orc.KIND_MIXED),
    (32, True, 4, 4, 2, 0, orc.KIND_MIXED),
    (64, False, 2, 4, 3, 12, orc.KIND_MIXED),
    (64, True, 4, 4, 4, 64, orc.KIND_MIXED),
    (128, False, 2, 4, 3, 16, orc.KIND_MIXED),
    (128, True, 4, 4, 3, 16, orc.KIND_MIXED),
    (128, False, 4, 8, 2, 0, orc.KIND_MIXED),
    (128, True, 2, 2, 2, 32, orc.KIND_MIXED),
    (128, False, 2, 2, 2, 128, orc.KIND_MIXED),
    (16, False, 1, 2, 2, 0, orc.KIND_FP32),
    (64, True, 2, 2, 3, 0, orc.KIND_FP32),
    (128, False, 2, 4, 3, 0, orc.KIND_FP32),
    (128, True, 4, 4, 2, 0, orc.KIND_FP32),
]


@pytest.mark.parametrize("d,kda,HK,HV,B,k_hi,kind", CASES)
def test_single_step_parity(d, kda, HK, HV, B, k_hi, kind):
    _say(f"case d={d} kda={kda} HK={HK} HV={HV} B={B} k_hi={k_hi} kind={kind}")
    num_slots, layers = B + 3, 2
    seed = d * 7 + B + k_hi + 100 * kda
    slots = inputs.slot_order(seed, num_slots, B)
    perm = inputs.random_perms(seed, HV, d)
    S = inputs.synthetic_states(seed, B, HV, d)
    inputs.scale_channels(S, inputs.outlier_channels(seed, HV, d, min(8, d // 4)), 10.0)
    ref = orc.Pool(kind, d, d, k_hi, layers, num_slots, HV)
    orc.pack(ref, 1, slots, S, perm)
    gpool = gpu_pool_from(ref, D)
    inp = inputs.step(inputs.decode_inputs(seed, 1, B, HK, HV, d, kda=kda), 0)
    o_gpu, o_ref = _run_step(kda, ref, gpool, 1, slots, inp, perm, scale=0.75)
    err = rel_l2(o_gpu, o_ref)
    stats = compare_tiles(gpool.buffer.cpu().numpy(), ref, f"d={d} kda={kda}")
    _say(f"  o rel-L2 {err:.2e}  {stats}")
    assert err <= (FP32_TOL if kind == orc.KIND_FP32 else O_TOL_MIXED)
    assert err <= 1e-4  # identical starting bytes: only fp32 rounding order differs


def test_padded_and_out_of_range_slots_leave_memory_untouched():
    d, HV, HK, B = 128, 4, 2, 4
    ref = orc.Pool(orc.KIND_MIXED, d, d, 16, 1, 6, HV)
    S = inputs.synthetic_states(3, 6, HV, d)
    orc.pack(ref, 0, np.arange(6), S)
    # canary bytes around the pool
    pad = 4096
    raw = torch.full((ref.buf.size + 2 * pad,), 0xA5, dtype=torch.uint8, device="cuda")
    raw[pad:pad + ref.buf.size] = torch.from_numpy(ref.buf).cuda()
    gpool = D.Pool(D.damp_layout_init(d, d, 16), 1, 6, HV, buffer=raw[pad:pad + ref.buf.size])
    slots = np.array([4, -1, 6, 1], np.int32)  # -1 padded, 6 == num_slots out of range
    inp = inputs.step(inputs.decode_inputs(4, 1, B, HK, HV, d), 0)
    o_gpu, o_ref = _run_step(False, ref, gpool, 0, slots, inp, None)
    assert (o_gpu[1] == 0).all() and (o_gpu[2] == 0).all()
    assert rel_l2(o_gpu, o_ref) <= 1e-4
    host = raw.cpu().numpy()
    assert (host[:pad] == 0xA5).all() and (host[-pad:] == 0xA5).all()
    compare_tiles(host[pad:-pad], ref, "padded")
    st = ref.slot_stride
    for s in (0, 2, 3, 5):
        assert np.array_equal(host[pad + s * st:pad + (s + 1) * st], ref.buf[s * st:(s + 1) * st])


def test_bf16_output():
    d, HV, HK, B = 128, 4, 2, 3
    ref = orc.Pool(orc.KIND_MIXED, d, d, 16, 1, B, HV)
    orc.pack(ref, 0, np.arange(B), inputs.synthetic_states(5, B, HV, d))
    gpool = gpu_pool_from(ref, D)
    inp = inputs.step(inputs.decode_inputs(6, 1, B, HK, HV, d), 0)
    o_gpu, o_ref = _run_step(False, ref, gpool, 0, np.arange(B), inp, None, o_dtype=torch.bfloat16)
    want = torch.from_numpy(o_ref).to(torch.bfloat16).float().numpy()
    ulp = np.abs(o_gpu - want) <= np.spacing(np.abs(want).astype(np.float32)) * 256
    assert ulp.mean() >= 0.999


@pytest.mark.parametrize("kind,k_hi", [(orc.KIND_MIXED, 16), (orc.KIND_MIXED, 0),
                                       (orc.KIND_FP32, 0)])
@pytest.mark.parametrize("d", [16, 64, 128])
def test_pack_parity_and_unpack_bit_exact(kind, k_hi, d):
    k_hi = min(k_hi, d)
    HV, B = 4, 3
    _say(f"pack d={d} kind={kind} k_hi={k_hi}")
    S = inputs.synthetic_states(7 + d, B, HV, d)
    inputs.scale_channels(S, inputs.outlier_channels(8, HV, d, 4), 10.0)
    perm = inputs.random_perms(9, HV, d)
    slots = np.array([2, 0, 4], np.int32)
    ref = orc.Pool(kind, d, d, k_hi, 1, 5, HV)
    orc.pack(ref, 0, slots, S, perm)
    gpool = D.Pool(D.damp_layout_init(d, d, k_hi, kind), 1, 5, HV)
    gpool.buffer.zero_()
    D.damp_state_pack(gpool, 0, dev_i32(slots), torch.from_numpy(S).cuda(), dev_u8(perm))
    torch.cuda.synchronize()
    compare_tiles(gpool.buffer.cpu().numpy(), ref, "pack")
    # unpack the oracle's bytes on the GPU: bit-exact decode
    gref = gpu_pool_from(ref, D)
    U = D.damp_state_unpack(gref, 0, dev_i32(np.array([0, 2, -1, 4], np.int32)), dev_u8(perm))
    want = orc.unpack(ref, 0, np.array([0, 2, -1, 4], np.int32), perm)
    assert np.array_equal(U.cpu().numpy(), want)


@pytest.mark.parametrize("kind,k_hi,d", [(orc.KIND_MIXED, 16, 128), (orc.KIND_MIXED, 4, 16),
                                         (orc.KIND_FP32, 0, 64)])
def test_reset_writes_the_packed_zero_state(kind, k_hi, d):
    HV = 3
    ref = orc.Pool(kind, d, d, k_hi, 2, 4, HV)
    ref.buf[:] = 0x5C
    orc.reset(ref, -1, [3, 1])
    gpool = D.Pool(D.damp_layout_init(d, d, k_hi, kind), 2, 4, HV)
    gpool.buffer.fill_(0x5C)
    D.damp_pool_reset_slots(gpool, -1, dev_i32([3, 1, -1, 9]))
    torch.cuda.synchronize()
    got = gpool.buffer.cpu().numpy()
    if kind == orc.KIND_FP32:
        assert np.array_equal(got, ref.buf)
    else:  # zero points are +0 or -0: compare as floats
        a, b = ref.copy(), ref.copy()
        a.buf = got
        ha, ca, sa, za = pu.split_tiles(a.buf, a)
        hb, cb, sb, zb = pu.split_tiles(b.buf, b)
        assert np.array_equal(ha, hb) and np.array_equal(ca, cb)
        assert np.array_equal(sa, sb) and np.array_equal(za, zb)
    S = D.damp_state_unpack(gpool, 1, dev_i32([3, 1]))
    assert (S.cpu().numpy() == 0).all()


def test_beta0_decay1_is_a_fixed_point_on_gpu():
    """beta = 0, g = 0 on a state the quantizer produced twice: the HIP path
    leaves every code, zero point and high-tier value unchanged."""
    d, HV, B = 128, 8, 4
    S = inputs.synthetic_states(10, B, HV, d)
    perm = inputs.random_perms(11, HV, d)
    ref = orc.Pool(orc.KIND_MIXED, d, d, 16, 1, B, HV)
    slots = np.arange(B, dtype=np.int32)
    orc.pack(ref, 0, slots, S, perm)
    orc.pack(ref, 0, slots, orc.unpack(ref, 0, slots, perm), perm)
    gpool = gpu_pool_from(ref, D)
    inp = inputs.step(inputs.decode_inputs(12, 1, B, HV, HV, d), 0)
    inp["beta"][:] = 0
    inp["g"][:] = 0
    _run_step(False, ref, gpool, 0, slots, inp, perm)
    ha, ca, sa, za = pu.split_tiles(gpool.buffer.cpu().numpy(), ref)
    hb, cb, sb, zb = pu.split_tiles(ref.buf, ref)
    assert np.array_equal(ha, hb)
    assert (ca != cb).mean() <= 1e-5 and np.array_equal(za, zb)


def test_slot_validation_mode_rejects_repeated_slots(monkeypatch):
    """With DAMP_CHECK_SLOTS=1 every call that writes tiles copies its slot ids
    to the host first and refuses a batch in which a pool slot repeats (the
    two requests would race on its tiles), touching nothing; distinct slots,
    padding and the mode switched off run as usual."""
    d, HK, HV, B, k_hi = 64, 2, 4, 3, 8
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, 6, HV)
    orc.pack(ref, 0, np.arange(6), inputs.synthetic_states(41, 6, HV, d))
    gpool = gpu_pool_from(ref, D)
    inp = inputs.step(inputs.decode_inputs(42, 1, B, HK, HV, d), 0)
    x = dev_inputs(inp)
    before = gpool.buffer.clone()
    monkeypatch.setenv("DAMP_CHECK_SLOTS", "1")
    dup = dev_i32([4, 1, 4])
    with pytest.raises(D.DampError) as e:
        D.damp_state_update_gdn(gpool, 0, dup, x["q"], x["k"], x["v"], x["g"], x["beta"])
    assert e.value.status == D.DAMP_ERR_INVALID_ARG and "slot 4" in str(e.value)
    with pytest.raises(D.DampError):
        D.damp_state_pack(gpool, 0, dup, torch.zeros((B, HV, d, d), device="cuda"))
    with pytest.raises(D.DampError):
        D.damp_pool_reset_slots(gpool, 0, dup)
    with pytest.raises(D.DampError):
        D.damp_check_slots(gpool, dup)
    torch.cuda.synchronize()
    assert torch.equal(gpool.buffer, before)
    ok = dev_i32([4, -1, 2])
    D.damp_state_update_gdn(gpool, 0, ok, x["q"], x["k"], x["v"], x["g"], x["beta"])
    D.damp_check_slots(gpool, dev_i32([-1, -1, 7, 7, 5]))  # padding may repeat
    monkeypatch.setenv("DAMP_CHECK_SLOTS", "0")
    D.damp_check_slots(gpool, [0, 1, 2])
    torch.cuda.synchronize()


# ------------------------------------------------------------- selection

@pytest.mark.parametrize("kda", [False, True])
def test_selection_bit_exact(kda):
    N, H, d, k_hi = 24, 8, 128, 16
    states = inputs.synthetic_states(13, N, H, d)
    inputs.scale_channels(states, inputs.outlier_channels(14, H, d, 8), 10.0)
    rng = np.random.default_rng(15)
    logs = (-np.abs(rng.normal(0, 1, (N, H, d) if kda else (N, H)))).astype(np.float32)
    r = orc.select(kda=kda, states=states, log_decay=logs, k_hi=k_hi)
    sel, perm, score = D.damp_select_channels(torch.from_numpy(states).cuda(),
                                              torch.from_numpy(logs).cuda(), k_hi, kda=kda)
    assert np.array_equal(sel.numpy(), r["sel"])
    assert np.array_equal(perm.numpy(), r["perm"])
    assert np.array_equal(score.numpy(), r["C"])


@pytest.mark.parametrize("kda,fmt,d", [(True, orc.FMT_PAPER, 128), (False, orc.FMT_PAPER, 64),
                                       (True, orc.FMT_PAPER_PLAIN, 128), (False, None, 32)])
def test_selection_under_the_deployed_low_tier(kda, fmt, d):
    """E measured with the deployed Q_lo (App. A.2): the selection with the
    paper's tier as `lo` equals the calibration oracle fed the same samples
    (one domain), bit for bit: kept channels, pi and C."""
    N, H, k_hi = 20, 4, 16
    _say(f"select lo={fmt} kda={kda} d={d}")
    states = inputs.synthetic_states(31 + d, N, H, d)
    inputs.scale_channels(states, inputs.outlier_channels(32, H, d, 8), 10.0)
    rng = np.random.default_rng(33)
    g = inputs.to_bf16_bits(-np.abs(rng.normal(0, 1, (N, H, d) if kda else (N, H))))
    cal = orc.Calib(kda=kda, H=H, dk=d, dv=d, fmt=fmt)
    for n in range(N):  # sample n is a batch of one request
        cal.accumulate(0, states[n:n + 1], g[n:n + 1])
    want = cal.finalize(k_hi)
    lo = D.damp_layout_init(d, d, 0)
    if fmt is not None:
        lo.hi_dtype, lo.group, lo.meta_dtype, lo.hadamard = fmt
    sel, perm, score = D.damp_select_channels(torch.from_numpy(states).cuda(),
                                              torch.from_numpy(orc.bf16_widen(g)).cuda(), k_hi,
                                              kda=kda, lo=lo)
    assert np.array_equal(score.numpy(), want["score"])
    assert np.array_equal(sel.numpy(), want["sel"])
    assert np.array_equal(perm.numpy(), want["perm"])
    if fmt is not None:  # a different Q_lo measures different errors
        _, _, s_row = D.damp_select_channels(torch.from_numpy(states).cuda(),
                                             torch.from_numpy(orc.bf16_widen(g)).cuda(), k_hi,
                                             kda=kda)
        assert not np.array_equal(s_row.numpy(), score.numpy())


# ------------------------------------------------- multi-step trajectory

def test_config1_tiny_gdn_trajectory():
    """Tiny GDN decode: B=1, 2 heads, d=16, 4 BF16 rows, 32 FP32 warm-up tokens,
    channels selected from stride-8 samples, then 8 mixed decode steps run
    independently on each side."""
    d, B, HK, HV, k_hi, T_w, T = 16, 1, 2, 2, 4, 32, 8
    inp = inputs.decode_inputs(0, T_w + T, B, HK, HV, d)
    warm = {k: v[:T_w] for k, v in inp.items()}
    S0 = np.zeros((B, HV, d, d), np.float32)
    S_w, _, samples = orc.run_fp32(S0, kda=False, sample_every=8, **warm)
    N = samples.shape[0]
    states = samples[:, 0]                                  # request 0: [N, HV, d, d]
    logs = orc.bf16_widen(warm["g"][7::8, 0])               # decay at the sampled steps
    r = orc.select(kda=False, states=states, log_decay=logs, k_hi=k_hi)
    sel, perm_g, _ = D.damp_select_channels(torch.from_numpy(states).cuda(),
                                            torch.from_numpy(logs).cuda(), k_hi, kda=False)
    assert np.array_equal(perm_g.numpy(), r["perm"]) and N == 4
    perm = r["perm"]
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B, HV)
    orc.pack(ref, 0, [0], S_w, perm)
    gpool = gpu_pool_from(ref, D)
    for t in range(T):
        st = inputs.step(inp, T_w + t)
        o_gpu, o_ref = _run_step(False, ref, gpool, 0, np.zeros(1, np.int32), st, perm)
        err = rel_l2(o_gpu, o_ref)
        _say(f"  step {t}: o rel-L2 {err:.2e}")
        assert err <= O_TOL_MIXED
        compare_tiles(gpool.buffer.cpu().numpy(), ref, f"step {t}")
        # each side continues from its own state


def test_graph_replay_matches_eager_launches():
    """The update captured in a HIP graph and replayed three times, with eager
    work and synchronisation between replays, gives byte-identical pools and
    outputs to the same steps launched eagerly."""
    d, HV, HK, B, k_hi = 128, 8, 4, 40, 16
    S = inputs.synthetic_states(50, B, HV, d)
    perm = inputs.random_perms(51, HV, d)
    slots = inputs.slot_order(52, B + 8, B)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B + 8, HV)
    orc.pack(ref, 0, slots, S, perm)
    eager, graphed = gpu_pool_from(ref, D), gpu_pool_from(ref, D)
    d_slots, d_perm = dev_i32(slots), dev_u8(perm)
    x = dev_inputs(inputs.step(inputs.decode_inputs(53, 1, B, HK, HV, d), 0))
    o_e = torch.empty((B, HV, d), dtype=torch.float32, device="cuda")
    o_g = torch.empty_like(o_e)

    def run(pool, o):
        D.damp_state_update_gdn(pool, 0, d_slots, x["q"], x["k"], x["v"], x["g"], x["beta"],
                                perm=d_perm, o=o)

    run(graphed, o_g)  # warm-up step on both sides keeps them in lockstep
    run(eager, o_e)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run(graphed, o_g)
    for _ in range(3):
        g.replay()
        run(eager, o_e)
        torch.cuda.synchronize()
        junk = torch.randn(1 << 20, device="cuda").sum()  # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(graphed.buffer, eager.buffer)
        assert torch.equal(o_g, o_e)
    del junk
