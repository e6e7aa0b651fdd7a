"""damp_select_channels_noalloc (the selection with the library's fixed device
scratch) against damp_select_channels on the same inputs: bit-identical kept
channels, pi and scores, on two calls in a row, the second with a smaller
input, so stale contents of the shared array from the first call must not
leak into the second."""
import numpy as np
import pytest
import torch

from paper_2608_27513_amd import damp as D
from paper_2608_27513_amd import inputs

pytestmark = pytest.mark.gpu


def _samples(seed, N, H, d, kda):
    S = inputs.synthetic_states(seed, N, H, d)
    inputs.scale_channels(S, inputs.outlier_channels(seed, H, d, 8), 10.0)
    rng = np.random.default_rng(seed)
    logs = (-np.abs(rng.normal(0, 1, (N, H, d) if kda else (N, H)))).astype(np.float32)
    return torch.from_numpy(S).cuda(), torch.from_numpy(logs).cuda()


def _paper_lo(d):
    lo = D.damp_layout_init(d, d, 0)
    lo.hi_dtype, lo.group, lo.meta_dtype, lo.hadamard = D.DAMP_DT_FP16, 32, D.DAMP_DT_FP16, 1
    return lo


@pytest.mark.parametrize("kda", [False, True])
def test_noalloc_selection_matches_the_allocating_one(kda):
    print(f"select noalloc kda={kda}", flush=True)
    calls = [  # (seed, N, H, d, lo): the second call is smaller than the first
        (61, 48, 16, 128, None),
        (62, 9, 4, 64, _paper_lo(64)),
    ]
    for seed, N, H, d, lo in calls:
        S, logs = _samples(seed, N, H, d, kda)
        want = D.damp_select_channels(S, logs, 16, kda=kda, lo=lo)
        got = D.damp_select_channels_noalloc(S, logs, 16, kda=kda, lo=lo)
        for a, b in zip(got, want):
            assert torch.equal(a, b)
    torch.cuda.synchronize()


def test_noalloc_selection_at_the_kda_calibration_size():
    """256 samples x 32 heads x 128 channels: the KDA workload's calibration,
    (N + 2) H d_k = 1 056 768 doubles, within the fixed scratch; then a
    smaller call on the same array."""
    print("select noalloc N=256 H=32 d=128", flush=True)
    for seed, N, H in ((71, 256, 32), (72, 5, 3)):
        S, logs = _samples(seed, N, H, 128, True)
        want = D.damp_select_channels(S, logs, 16, kda=True)
        got = D.damp_select_channels_noalloc(S, logs, 16, kda=True)
        for a, b in zip(got, want):
            assert torch.equal(a, b)
        del S, logs
    torch.cuda.synchronize()
