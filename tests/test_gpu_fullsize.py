"""Full-size GPU parity in the launch configuration the benchmark times.

The GDN workload (B=256, 16 key / 32 value heads, d=128, 16 BF16 rows, 8
outlier channels per head at 10x) and the KDA workload (B=256, 32 heads, per-channel
decay with ~10% persistent channels, 16 channels chosen by the selection).
The oracle packs every tile and runs the whole step, so every output and
every stored byte is compared; the same for the paper's tiers. Also the
largest batch a launch takes, the empty batch, and the prefill of a 64-token
chunk for the whole batch, checked on sampled requests.
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


@pytest.mark.parametrize("kda", [False, True])
def test_full_size_step(kda):
    B, HV, d, k_hi = 256, 32, 128, 16
    HK = HV if kda else 16
    seed = 2 if not kda else 3
    _say(f"full-size {'KDA' if kda else 'GDN'}: B={B} HK={HK} HV={HV} d={d} k_hi={k_hi}")
    S = inputs.synthetic_states(seed, B, HV, d)
    mu = inputs.kda_mu(seed, HV, d) if kda else None
    if not kda:
        inputs.scale_channels(S, inputs.outlier_channels(seed, HV, d, 8), 10.0)
    # channel selection from 64 calibration samples of the same distribution
    cal = S[:64]
    if kda:
        logs = -np.logaddexp(0.0, mu[None] + np.random.default_rng(seed).standard_normal(
            (64, HV, d))).astype(np.float32)
    else:
        logs = np.full((64, HV), -0.5, np.float32)
    perm = orc.select(kda=kda, states=cal, log_decay=logs, k_hi=k_hi)["perm"]
    slots = inputs.slot_order(seed, B, B)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B, HV)
    orc.pack(ref, 0, slots, S, perm)
    del S, cal
    gpool = gpu_pool_from(ref, D)
    inp = inputs.step(inputs.decode_inputs(seed, 1, B, HK, HV, d, kda=kda, mu=mu), 0)
    di = dev_inputs(inp)
    o = torch.empty((B, HV, d), dtype=torch.float32, device="cuda")
    fn = D.damp_state_update_kda if kda else D.damp_state_update_gdn
    fn(gpool, 0, dev_i32(slots), di["q"], di["k"], di["v"], di["g"], di["beta"],
       perm=dev_u8(perm), o=o)
    torch.cuda.synchronize()
    _say("  gpu step done; running the oracle")
    o_ref = orc.update(ref, 0, slots, kda=kda, perm=perm, **inp)
    err = rel_l2(o.cpu().numpy(), o_ref)
    stats = compare_tiles(gpool.buffer.cpu().numpy(), ref, "full-size")
    _say(f"  o rel-L2 {err:.2e}  {stats}")
    assert err <= O_TOL_MIXED and err <= 1e-4


@pytest.mark.parametrize("kda,B,HK,HV", [(False, 256, 2, 4), (True, 256, 4, 4), (False, 32, 16, 32),
                                         (False, 16, 16, 32), (True, 64, 32, 32), (True, 1, 32, 32)])
def test_small_batch_launch_shapes(kda, B, HK, HV):
    """The small-batch launches the benchmark times: one GPU's share of an
    8-way tensor-parallel step (B = 256 with 4 value heads: 1024 tiles, two
    per workgroup), B = 32 (two per workgroup), B = 16, B = 64 (three rounds)
    and B = 1, at scattered slots of a larger pool; every output and every
    stored byte against the oracle."""
    d, k_hi = 128, 16
    seed = 60 + B + HV + kda
    num_slots = B + 37
    _say(f"small batch: kda={kda} B={B} HK={HK} HV={HV}")
    S = inputs.synthetic_states(seed, num_slots, HV, d)
    mu = inputs.kda_mu(seed, HV, d) if kda else None
    perm = inputs.random_perms(seed, HV, d)
    slots = inputs.slot_order(seed, num_slots, B)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, num_slots, HV)
    orc.pack(ref, 0, np.arange(num_slots, dtype=np.int32), S, perm)
    gpool = gpu_pool_from(ref, D)
    inp = inputs.step(inputs.decode_inputs(seed, 1, B, HK, HV, d, kda=kda, mu=mu), 0)
    di = dev_inputs(inp)
    o = torch.empty((B, HV, d), dtype=torch.float32, device="cuda")
    fn = D.damp_state_update_kda if kda else D.damp_state_update_gdn
    fn(gpool, 0, dev_i32(slots), di["q"], di["k"], di["v"], di["g"], di["beta"],
       perm=dev_u8(perm), o=o)
    torch.cuda.synchronize()
    o_ref = orc.update(ref, 0, slots, kda=kda, perm=perm, **inp)
    err = rel_l2(o.cpu().numpy(), o_ref)
    stats = compare_tiles(gpool.buffer.cpu().numpy(), ref, "small batch")
    _say(f"  o rel-L2 {err:.2e}  {stats}")
    assert err <= O_TOL_MIXED and err <= 1e-4


def test_largest_batch_and_empty_batch():
    B, HV, d, k_hi = 65535, 1, 16, 4
    _say(f"max batch: B={B} HV={HV} d={d}")
    S = inputs.synthetic_states(4, B, HV, d)
    slots = np.arange(B, dtype=np.int32)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B, HV)
    orc.pack(ref, 0, slots, S)
    gpool = gpu_pool_from(ref, D)
    inp = inputs.step(inputs.decode_inputs(5, 1, B, 1, HV, d), 0)
    di = dev_inputs(inp)
    o = torch.empty((B, HV, d), dtype=torch.float32, device="cuda")
    D.damp_state_update_gdn(gpool, 0, dev_i32(slots), di["q"], di["k"], di["v"], di["g"],
                            di["beta"], o=o)
    torch.cuda.synchronize()
    o_ref = orc.update(ref, 0, slots, kda=False, **inp)
    assert rel_l2(o.cpu().numpy(), o_ref) <= 1e-4
    compare_tiles(gpool.buffer.cpu().numpy(), ref, "max batch")
    # an empty batch is a no-op
    before = gpool.buffer.clone()
    e = torch.empty(0, dtype=torch.int32, device="cuda")
    z = torch.empty((0, 1, d), dtype=torch.bfloat16, device="cuda")
    D.damp_state_update_gdn(gpool, 0, e, z, z, z, torch.empty((0, 1), dtype=torch.bfloat16,
                            device="cuda"), torch.empty((0, 1), dtype=torch.bfloat16,
                            device="cuda"), o=torch.empty((0, 1, d), device="cuda"))
    torch.cuda.synchronize()
    assert torch.equal(before, gpool.buffer)


@pytest.mark.parametrize("kda,k_hi,o_bf16", [(False, 16, False), (True, 8, True), (False, 0, False),
                                              (True, 32, False), (False, 12, False)])
def test_many_tiles_per_workgroup_with_padding(kda, k_hi, o_bf16):
    """B = 600 requests in a 700-slot pool (several tiles per resident
    workgroup), with padded (-1) and out-of-range slots scattered through the
    batch: padded requests leave their memory untouched and output zeros."""
    B, HV, d, num_slots = 600, 32, 128, 700
    HK = HV if kda else 8
    seed = 40 + k_hi + kda
    _say(f"padded batch: kda={kda} k_hi={k_hi} o_bf16={o_bf16}")
    slots = inputs.slot_order(seed, num_slots, B).copy()
    rng = np.random.default_rng(seed)
    pad = rng.choice(B, size=37, replace=False)
    slots[pad[:30]] = -1
    slots[pad[30:]] = num_slots + rng.integers(0, 5, 7)
    S = inputs.synthetic_states(seed, num_slots, HV, d)
    perm = inputs.random_perms(seed, HV, d)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 2, num_slots, HV)
    orc.pack(ref, 1, np.arange(num_slots), S, perm)
    del S
    gpool = gpu_pool_from(ref, D)
    inp = inputs.step(inputs.decode_inputs(seed, 1, B, HK, HV, d, kda=kda), 0)
    di = dev_inputs(inp)
    o = torch.empty((B, HV, d), dtype=torch.bfloat16 if o_bf16 else torch.float32,
                    device="cuda")
    fn = D.damp_state_update_kda if kda else D.damp_state_update_gdn
    fn(gpool, 1, dev_i32(slots), di["q"], di["k"], di["v"], di["g"], di["beta"],
       perm=dev_u8(perm), scale=0.5, o=o)
    torch.cuda.synchronize()
    o_ref = orc.update(ref, 1, slots, kda=kda, perm=perm, scale=0.5, **inp)
    o_gpu = o.float().cpu().numpy()
    assert (o_gpu[pad] == 0).all()
    tol = 1e-2 if o_bf16 else 1e-4
    assert rel_l2(o_gpu, o_ref) <= tol
    stats = compare_tiles(gpool.buffer.cpu().numpy(), ref, "padded batch")
    _say(f"  o rel-L2 {rel_l2(o_gpu, o_ref):.2e} {stats}")


@pytest.mark.parametrize("fmt", [orc.FMT_PAPER, orc.FMT_PAPER_PLAIN])
@pytest.mark.parametrize("kda", [False, True])
def test_full_size_step_paper_tiers(kda, fmt):
    """The decode workload in the paper's tiers (FP16 rows, groups of 32 with
    FP16 (s, z), with and without the block-32 transform), every output and
    stored byte compared."""
    B, HV, d, k_hi = 256, 32, 128, 16
    HK = HV if kda else 16
    seed = 20 + kda + 2 * fmt[3]
    _say(f"full-size paper tiers kda={kda} had={fmt[3]}")
    S = inputs.synthetic_states(seed, B, HV, d)
    inputs.scale_channels(S, inputs.outlier_channels(seed, HV, d, 8), 10.0)
    perm = inputs.random_perms(seed, HV, d)
    slots = inputs.slot_order(seed, B, B)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B, HV, fmt=fmt)
    orc.pack(ref, 0, slots, S, perm)
    del S
    gpool = gpu_pool_from(ref, D)
    inp = inputs.step(inputs.decode_inputs(seed, 1, B, HK, HV, d, kda=kda), 0)
    di = dev_inputs(inp)
    o = torch.empty((B, HV, d), dtype=torch.float32, device="cuda")
    fn = D.damp_state_update_kda if kda else D.damp_state_update_gdn
    fn(gpool, 0, dev_i32(slots), di["q"], di["k"], di["v"], di["g"], di["beta"],
       perm=dev_u8(perm), o=o)
    torch.cuda.synchronize()
    _say("  gpu step done; running the oracle")
    o_ref = orc.update(ref, 0, slots, kda=kda, perm=perm, **inp)
    err = rel_l2(o.cpu().numpy(), o_ref)
    stats = compare_tiles(gpool.buffer.cpu().numpy(), ref, "full-size paper tiers")
    _say(f"  o rel-L2 {err:.2e}  {stats}")
    assert err <= O_TOL_MIXED and err <= 1e-4


@pytest.mark.parametrize("kda", [False, True])
def test_full_size_prefill_sampled(kda):
    """The prefill in the benchmark's launch configuration (B = 256, 16 or 32
    key and 32 value heads, d = 128, 16 BF16 rows, one 64-token chunk per
    request): the GPU runs every request; the oracle runs four sampled
    requests from the same starting bytes, and their outputs and stored
    tiles are compared."""
    B, HV, d, k_hi, T = 256, 32, 128, 16, 64
    HK = HV if kda else 16
    seed = 30 + kda
    _say(f"full-size prefill kda={kda}: B={B} HK={HK} HV={HV} d={d} T={T}")
    S = inputs.synthetic_states(seed, B, HV, d)
    perm = inputs.random_perms(seed, HV, d)
    slots = inputs.slot_order(seed, B, B)
    full = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B, HV)
    orc.pack(full, 0, slots, S, perm)
    gpool = gpu_pool_from(full, D)
    inp = inputs.as_prefill(inputs.decode_inputs(seed, T, B, HK, HV, d, kda=kda))
    di = dev_inputs(inp)
    o = torch.empty((B, T, HV, d), dtype=torch.float32, device="cuda")
    fn = D.damp_state_prefill_kda if kda else D.damp_state_prefill_gdn
    fn(gpool, 0, dev_i32(slots), di["q"], di["k"], di["v"], di["g"], di["beta"],
       perm=dev_u8(perm), o=o)
    torch.cuda.synchronize()
    _say("  gpu chunk done; running the oracle on the sampled requests")
    pick = np.array([0, 77, 150, 255])
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, len(pick), HV)
    orc.pack(ref, 0, np.arange(len(pick)), S[pick], perm)
    del S
    o_ref = orc.prefill(ref, 0, np.arange(len(pick)), kda=kda, perm=perm,
                        **{n: a[pick] for n, a in inp.items()})
    err = rel_l2(o.cpu().numpy()[pick], o_ref)
    got = gpool.buffer.cpu().numpy().reshape(B, -1)[slots[pick]].reshape(-1)
    stats = compare_tiles(got, ref, "full-size prefill", s16_exact_min=0.99)
    _say(f"  o rel-L2 {err:.2e}  {stats}")
    assert err <= 1e-4


def test_multilayer_pool_at_its_last_layer():
    """The 48-layer decode workload's pool: 48 GDN layers x 512 request slots x
    32 value heads of 19 328-byte tiles (15.2 GB), 384 requests active in
    random non-contiguous slots. One decode step of layer 47, whose tiles sit
    past 14.9 GB into the pool, in the launch configuration the 48-layer
    benchmark replays; the oracle runs the same step on a pool holding only
    the active slots' tiles. Every output, every stored byte of the 384 active
    slots of that layer, and the untouched rest of the layer (filled with a
    canary) are compared."""
    L, num_slots, B, HK, HV, d, k_hi = 48, 512, 384, 16, 32, 128, 16
    layer = L - 1
    seed = 48
    _say(f"48-layer pool: layer {layer}, {B} of {num_slots} slots, {HV} heads, d={d}")
    active = inputs.slot_order(seed, num_slots, B)
    perm = inputs.random_perms(seed, HV, d)
    ref = orc.Pool(orc.KIND_MIXED, d, d, k_hi, 1, B, HV)  # host slot i <-> pool slot active[i]
    S = inputs.synthetic_states(seed, B, HV, d)
    orc.pack(ref, 0, np.arange(B), S, perm)
    del S
    lay = D.damp_layout_init(d, d, k_hi)
    need = D.damp_pool_required_bytes(lay, L, num_slots, HV)
    assert need == 15_200_157_696
    buf = torch.full((need,), 0xA5, dtype=torch.uint8, device="cuda")
    gpool = D.Pool(lay, L, num_slots, HV, buffer=buf)
    slot_bytes = HV * ref.tile_stride
    rows = buf.view(L * num_slots, slot_bytes)
    idx = torch.from_numpy(layer * num_slots + active.astype(np.int64)).cuda()
    rows[idx] = torch.from_numpy(ref.buf.reshape(B, slot_bytes)).cuda()
    inp = inputs.step(inputs.decode_inputs(seed, 1, B, HK, HV, d), 0)
    di = dev_inputs(inp)
    o = torch.empty((B, HV, d), dtype=torch.float32, device="cuda")
    D.damp_state_update_gdn(gpool, layer, dev_i32(active), di["q"], di["k"], di["v"], di["g"],
                            di["beta"], perm=dev_u8(perm), o=o)
    torch.cuda.synchronize()
    _say("  gpu step done; running the oracle")
    o_ref = orc.update(ref, 0, np.arange(B), kda=False, perm=perm, **inp)
    err = rel_l2(o.cpu().numpy(), o_ref)
    stats = compare_tiles(rows[idx].cpu().numpy().reshape(-1), ref, "48-layer pool, layer 47")
    _say(f"  o rel-L2 {err:.2e}  {stats}")
    assert err <= O_TOL_MIXED and err <= 1e-4
    # nothing else of layer 47, and nothing of its neighbouring layer, was written
    keep = torch.ones(num_slots, dtype=torch.bool, device="cuda")
    keep[torch.from_numpy(active.astype(np.int64)).cuda()] = False
    lay47 = rows[layer * num_slots:(layer + 1) * num_slots]
    assert bool((lay47[keep] == 0xA5).all())
    assert bool((rows[(layer - 1) * num_slots:layer * num_slots] == 0xA5).all())
    del buf, rows, lay47
    torch.cuda.empty_cache()
