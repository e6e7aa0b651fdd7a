"""GPU parity of on-device calibration (App. A.2 Eq. (13)-(15), Alg. 1,
section 6's selectors) against the oracle.

Accumulation from identical FP32 states is bit-exact (both sides follow the
definitions' summation order with IEEE operations), so the selection is too.
A whole calibration sequence runs each side's own FP32 trajectory, whose
rounding differs; there the statistics agree to a relative tolerance and the
selection must be a valid top-k of the oracle's scores up to that tolerance.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_2608_27513_amd import damp as D
from paper_2608_27513_amd import inputs
from parity_util import dev_i32, dev_u8

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)


def _layout(d, fmt):
    lo = D.damp_layout_init(d, d, 0)
    if fmt is not None:
        lo.hi_dtype, lo.group, lo.meta_dtype, lo.hadamard = fmt
    return lo


def _fp32_pool(S, perm, slots, num_slots):
    """A device FP32 pool whose bytes the oracle wrote: S natural [B, H, d, d]
    stored with rows permuted by perm into the given slots."""
    B, H, d, _ = S.shape
    ref = orc.Pool(orc.KIND_FP32, d, d, 0, 1, num_slots, H)
    orc.pack(ref, 0, slots, S, perm)
    buf = torch.from_numpy(ref.buf.copy()).cuda()
    return D.Pool(D.damp_layout_init(d, d, 0, D.DAMP_STATE_FP32), 1, num_slots, H, buffer=buf)


def _device_sums(cal):
    D_, H, d = cal.num_domains, cal.num_heads, cal.lo.d_k
    h = cal.buffer.cpu().numpy()
    return h[:D_ * 3 * H * d].reshape(D_, 3, H, d), h[D_ * 3 * H * d:]


@pytest.mark.parametrize("kda,fmt,d", [(False, None, 64), (True, None, 64), (False, orc.FMT_PAPER, 64),
                                       (True, orc.FMT_PAPER, 64), (True, orc.FMT_PAPER_PLAIN, 64),
                                       (False, None, 128), (True, orc.FMT_PAPER, 128),
                                       (False, orc.FMT_PAPER_PLAIN, 32), (True, None, 16)])
def test_accumulate_and_finalize_are_bit_exact(kda, fmt, d):
    H, B = 4, 5
    _say(f"calib accumulate kda={kda} fmt={fmt} d={d}")
    seed = 800 + 3 * kda + (0 if fmt is None else fmt[3] + 1) + d
    cal = D.Calib(_layout(d, fmt), kda=kda, num_heads=H, num_domains=2)
    ref = orc.Calib(kda=kda, H=H, dk=d, dv=d, num_domains=2, fmt=fmt)
    rng = np.random.default_rng(seed)
    for call, domain in enumerate((0, 1, 0)):
        S = inputs.synthetic_states(seed + call, B, H, d)
        inputs.scale_channels(S, inputs.outlier_channels(seed + call, H, d, 6), 10.0)
        perm = inputs.random_perms(seed + call, H, d)
        slots = rng.permutation(B + 3)[:B].astype(np.int32)
        gpool = _fp32_pool(S, perm, slots, B + 3)
        shape = (B, H, d) if kda else (B, H)
        g = inputs.to_bf16_bits(-np.log1p(np.exp(rng.standard_normal(shape).astype(np.float32))))
        slots_dev = slots.copy()
        slots_dev[1] = -1  # a padded request: skipped on both sides
        D.damp_calib_accumulate(cal, domain, gpool, 0, dev_i32(slots_dev),
                                torch.from_numpy(g.view(np.int16)).cuda().view(torch.bfloat16),
                                perm=dev_u8(perm))
        keep = np.arange(B) != 1
        ref.accumulate(domain, S[keep], g[keep])
    torch.cuda.synchronize()
    sums, counts = _device_sums(cal)
    assert np.array_equal(counts, ref.counts)
    assert np.array_equal(sums, ref.sums)
    rand = np.random.default_rng(seed).random((H, d))
    for sel in (D.DAMP_SEL_DAMP, D.DAMP_SEL_ERROR, D.DAMP_SEL_PERSISTENCE,
                D.DAMP_SEL_STATE_ENERGY, D.DAMP_SEL_RANDOM):
        got = D.damp_calib_finalize(cal, 12, selector=sel, rand_scores=torch.from_numpy(rand))
        want = ref.finalize(12, selector=sel, rand_scores=rand)
        assert np.array_equal(got["sel"].numpy(), want["sel"]), sel
        assert np.array_equal(got["perm"].numpy(), want["perm"]), sel
        assert np.array_equal(got["score"].numpy(), want["score"]), sel
        for name in ("E", "P", "energy", "mean_log_a"):
            assert np.array_equal(got[name].numpy(), want[name]), (sel, name)


def _valid_topk(sel, score, k, rtol):
    """sel (per head) is a top-k of score up to rtol: every kept channel
    scores at least the k-th largest score less rtol of it."""
    for h in range(score.shape[0]):
        kth = np.sort(score[h])[::-1][k - 1]
        assert np.all(score[h][sel[h]] >= kth * (1.0 - rtol)), h


@pytest.mark.parametrize("kda,fmt,HK,H,B,T", [(False, None, 2, 4, 3, 44), (True, orc.FMT_PAPER, 2, 2, 2, 40),
                                          (True, None, 3, 3, 2, 32)])
def test_calibrate_sequence_matches_the_oracle_trajectory(kda, fmt, HK, H, B, T):
    """Each side runs its own FP32 trajectory from the zero state and samples
    every 8 tokens; the counts agree exactly and the statistics to the fp32
    rounding of the trajectory."""
    d = 32
    _say(f"calib sequence kda={kda} fmt={fmt} H={H} B={B} T={T}")
    inp = inputs.decode_inputs(900 + T, T, B, HK, H, d, kda=kda)
    ref = orc.Calib(kda=kda, H=H, dk=d, dv=d, fmt=fmt)
    S_ref = orc.calibrate_sequence(ref, 0, np.zeros((B, H, d, d), np.float32), stride=8, **inp)
    pool = D.Pool(D.damp_layout_init(d, d, 0, D.DAMP_STATE_FP32), 1, B + 1, H)
    slots = torch.arange(1, B + 1, dtype=torch.int32, device="cuda")
    D.damp_pool_reset_slots(pool, 0, slots)
    cal = D.Calib(_layout(d, fmt), kda=kda, num_heads=H)
    x = {n: torch.from_numpy(np.ascontiguousarray(np.swapaxes(a, 0, 1)).view(np.int16)).cuda()
         .view(torch.bfloat16) for n, a in inp.items()}
    D.damp_calibrate_sequence(cal, 0, pool, 0, slots, x["q"], x["k"], x["v"], x["g"], x["beta"])
    S_gpu = D.damp_state_unpack(pool, 0, slots).cpu().numpy()
    torch.cuda.synchronize()
    assert np.linalg.norm(S_gpu - S_ref) <= 1e-5 * np.linalg.norm(S_ref)
    sums, counts = _device_sums(cal)
    assert np.array_equal(counts, ref.counts) and counts[0] == (T // 8) * B
    assert np.array_equal(sums[0, 2], ref.sums[0, 2])  # log a: the same inputs
    np.testing.assert_allclose(sums[0, 1], ref.sums[0, 1], rtol=1e-5)
    np.testing.assert_allclose(sums[0, 0], ref.sums[0, 0], rtol=2e-3)
    got = D.damp_calib_finalize(cal, 8)
    want = ref.finalize(8)
    _valid_topk(got["sel"].numpy(), want["score"], 8, 2e-3)


def test_kda_workload_calibration():
    """The KDA workload's calibration: one 2048-token sequence, 32 heads,
    d = 128, samples every 8 tokens (256 per head), the paper's low tier as
    Q_lo; the selection against the oracle's own run."""
    d, H, T = 128, 32, 2048
    _say("calib KDA workload: 2048 tokens, 32 heads, d=128")
    inp = inputs.decode_inputs(1, T, 1, H, H, d, kda=True)
    ref = orc.Calib(kda=True, H=H, dk=d, dv=d, fmt=orc.FMT_PAPER)
    orc.calibrate_sequence(ref, 0, np.zeros((1, H, d, d), np.float32), stride=8, **inp)
    pool = D.Pool(D.damp_layout_init(d, d, 0, D.DAMP_STATE_FP32), 1, 1, H)
    slots = torch.zeros(1, dtype=torch.int32, device="cuda")
    D.damp_pool_reset_slots(pool, 0, slots)
    cal = D.Calib(_layout(d, orc.FMT_PAPER), kda=True, num_heads=H)
    x = {n: torch.from_numpy(np.ascontiguousarray(np.swapaxes(a, 0, 1)).view(np.int16)).cuda()
         .view(torch.bfloat16) for n, a in inp.items()}
    D.damp_calibrate_sequence(cal, 0, pool, 0, slots, x["q"], x["k"], x["v"], x["g"], x["beta"])
    got = D.damp_calib_finalize(cal, 16)
    want = ref.finalize(16)
    assert ref.counts[0] == 256
    _valid_topk(got["sel"].numpy(), want["score"], 16, 5e-3)
    overlap = np.mean([orc.topk_overlap(got["sel"][h].numpy(), want["sel"][h]) for h in range(H)])
    _say(f"  overlap with the oracle's selection {overlap:.4f}")
    assert overlap >= 0.97
