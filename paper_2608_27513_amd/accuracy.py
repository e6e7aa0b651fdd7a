"""Held-out trajectory accuracy of a stored state against the FP32 state.

App. E measures a stored-state layout by the relative RMS error of its
trajectory against the FP32-state trajectory over held-out decode steps,

    RRMSE(Y) = ( sum_t ||Y^_t - Y_t||_F^2 / sum_t ||Y_t||_F^2 )^(1/2),

for the recurrent state (Y_t = S_t) and for the output (Y_t = o_t). This
module runs those trajectories through libdamp's kernels: every decode step of
every layout is a damp_state_update_* launch on its own pool, and the states
are read back with damp_state_unpack into natural channel order. Only the
error sums (torch reductions over the unpacked states and outputs) and the
input draws happen outside the library.

Protocol, per workload (GDN or KDA decode, B requests, HV value heads, d = 128):
  1. warm state: the FP32 recurrence over `warm` tokens from the zero state;
  2. calibration: a separate FP32 sequence of `calib_tokens` tokens (one
     request, another seed) sampled every 8 tokens and accumulated on the
     device under the deployed low tier (App. A.2), then the selectors of
     section 6: C = E P (DAMP), E alone, and random scores;
  3. held-out trajectory: every layout starts from the warm state packed
     into it (one quantization), then `steps` decode steps on identical
     inputs, as does the FP32 state. Uniform INT8 is the same low tier with
     no protected rows.
"""
from __future__ import annotations

import numpy as np
import torch

from . import damp as D
from . import inputs

PAPER_TIER = (D.DAMP_DT_FP16, 32, D.DAMP_DT_FP16, 1)  # INT8 + H32, FP16 (s, z), FP16 rows


def layout_for(d: int, k_hi: int, tier=None) -> D.damp_layout:
    """The default tiers (tier None) or the paper's (PAPER_TIER) with k_hi rows."""
    lay = D.damp_layout_init(d, d, k_hi)
    if tier is not None:
        lay.hi_dtype, lay.group, lay.meta_dtype, lay.hadamard = tier
    return lay


def warm_states(*, kda: bool, B: int, HK: int, HV: int, d: int, tokens: int, gen, mu=None,
                key_scale=None):
    """FP32 states after `tokens` decode steps from zero, natural order
    [B, HV, d, d] (the library's FP32-state update)."""
    pool = D.Pool(D.damp_layout_init(d, d, 0, D.DAMP_STATE_FP32), 1, B, HV)
    slots = torch.arange(B, dtype=torch.int32, device="cuda")
    D.damp_pool_reset_slots(pool, 0, slots)
    o = torch.empty((B, HV, d), dtype=torch.float32, device="cuda")
    fn = D.damp_state_update_kda if kda else D.damp_state_update_gdn
    for _ in range(tokens):
        x = inputs.decode_inputs_device(gen, B, HK, HV, d, kda=kda, mu=mu, key_scale=key_scale)
        fn(pool, 0, slots, x["q"], x["k"], x["v"], x["g"], x["beta"], o=o)
    return D.damp_state_unpack(pool, 0, slots)


def calibrate(*, kda: bool, HK: int, HV: int, d: int, lo: D.damp_layout, tokens: int, gen,
              mu=None, key_scale=None, stride: int = 8) -> D.Calib:
    """On-device calibration of one FP32 sequence from the zero state under
    the low tier of `lo` (App. A.2-A.3)."""
    steps = [inputs.decode_inputs_device(gen, 1, HK, HV, d, kda=kda, mu=mu, key_scale=key_scale)
             for _ in range(tokens)]
    x = {n: torch.stack([s[n] for s in steps], dim=1).contiguous() for n in steps[0]}
    del steps
    pool = D.Pool(D.damp_layout_init(d, d, 0, D.DAMP_STATE_FP32), 1, 1, HV)
    slots = torch.zeros(1, dtype=torch.int32, device="cuda")
    D.damp_pool_reset_slots(pool, 0, slots)
    cal = D.Calib(lo, kda=kda, num_heads=HV)
    D.damp_calibrate_sequence(cal, 0, pool, 0, slots, x["q"], x["k"], x["v"], x["g"], x["beta"],
                              stride=stride)
    return cal


def selections(cal: D.Calib, k_hi: int, seed: int) -> dict:
    """Permutations (device uint8 [HV, d]) of the DAMP, E-only and random
    selectors from one calibration."""
    H, d = cal.num_heads, cal.lo.d_k
    rand = np.random.default_rng([seed, 0x726e]).random((H, d))
    out = {}
    for name, sel in (("damp", D.DAMP_SEL_DAMP), ("error_only", D.DAMP_SEL_ERROR),
                      ("random", D.DAMP_SEL_RANDOM)):
        r = D.damp_calib_finalize(cal, k_hi, selector=sel,
                                  rand_scores=torch.from_numpy(rand) if sel == D.DAMP_SEL_RANDOM
                                  else None)
        out[name] = r["perm"].cuda()
    return out


def trajectory_rrmse(*, kda: bool, HK: int, S0: torch.Tensor, variants: dict, step_inputs,
                     o_dtype=torch.float32) -> dict:
    """State and output RRMSE of each stored layout against the FP32 state.

    S0: natural-order fp32 [B, HV, d, d] start state. variants: name ->
    (layout, perm or None). step_inputs: an iterable of decode inputs (dicts
    of device bf16 tensors). Each layout's pool gets S0 packed once; then
    every step runs the same inputs on every pool and on an FP32 pool."""
    B, HV, d, _ = S0.shape
    slots = torch.arange(B, dtype=torch.int32, device="cuda")
    fn = D.damp_state_update_kda if kda else D.damp_state_update_gdn
    ref = D.Pool(D.damp_layout_init(d, d, 0, D.DAMP_STATE_FP32), 1, B, HV)
    D.damp_state_pack(ref, 0, slots, S0)
    pools = {}
    for name, (lay, perm) in variants.items():
        pool = D.Pool(lay, 1, B, HV)
        D.damp_state_pack(pool, 0, slots, S0, perm)
        pools[name] = (pool, perm)
    o_ref = torch.empty((B, HV, d), dtype=torch.float32, device="cuda")
    o_hat = torch.empty((B, HV, d), dtype=o_dtype, device="cuda")
    S_hat = torch.empty_like(S0)
    acc = {name: torch.zeros(4, dtype=torch.float64, device="cuda") for name in pools}
    n_steps = 0
    for x in step_inputs:
        fn(ref, 0, slots, x["q"], x["k"], x["v"], x["g"], x["beta"], o=o_ref)
        S_ref = D.damp_state_unpack(ref, 0, slots)
        s_den = torch.sum(S_ref.square(), dtype=torch.float64)
        o_den = torch.sum(o_ref.square(), dtype=torch.float64)
        for name, (pool, perm) in pools.items():
            fn(pool, 0, slots, x["q"], x["k"], x["v"], x["g"], x["beta"], perm=perm, o=o_hat)
            D.damp_state_unpack(pool, 0, slots, perm, S_out=S_hat)
            a = acc[name]
            a[0] += torch.sum(S_hat.sub_(S_ref).square_(), dtype=torch.float64)
            a[1] += s_den
            a[2] += torch.sum((o_hat.float() - o_ref).square_(), dtype=torch.float64)
            a[3] += o_den
        n_steps += 1
    out = {}
    for name, a in acc.items():
        a = a.cpu().numpy()
        out[name] = dict(state_rrmse=float(np.sqrt(a[0] / a[1])),
                         output_rrmse=float(np.sqrt(a[2] / a[3])),
                         bits_per_value=D.damp_bits_per_value(variants[name][0]))
    out["steps"] = n_steps
    return out


def study(*, kda: bool, B: int = 64, HK: int = None, HV: int = 32, d: int = 128, k_hi: int = 16,
          warm: int = 512, calib_tokens: int = 2048, steps: int = 256, seed: int = 0,
          key_channels: int = 0, key_factor: float = 4.0,
          tiers=(("default", None), ("int8_h32", PAPER_TIER)), log=None) -> dict:
    """The held-out accuracy of uniform INT8 and of the random, E-only and
    DAMP selections, for each tier, on one decode workload (the synthetic
    distributions of the benchmark: GDN 16 key / 32 value heads with a
    scalar decay, KDA 32 heads with per-channel decays). key_channels > 0
    draws keys whose energy concentrates in that many seeded channels per key
    head (key_factor times the others before normalization), in warm-up,
    calibration and held-out steps alike."""
    if HK is None:
        HK = HV if kda else HV // 2
    mu = torch.from_numpy(inputs.kda_mu(seed, HV, d)).cuda() if kda else None
    ks = None
    if key_channels > 0:
        ks = torch.from_numpy(inputs.key_channel_scale(seed, HK, d, key_channels, key_factor)).cuda()
    g_warm = torch.Generator(device="cuda")
    g_warm.manual_seed(1000 + seed)
    S0 = warm_states(kda=kda, B=B, HK=HK, HV=HV, d=d, tokens=warm, gen=g_warm, mu=mu, key_scale=ks)
    variants = {}
    for tname, tier in tiers:
        g_cal = torch.Generator(device="cuda")
        g_cal.manual_seed(2000 + seed)
        cal = calibrate(kda=kda, HK=HK, HV=HV, d=d, lo=layout_for(d, 0, tier),
                        tokens=calib_tokens, gen=g_cal, mu=mu, key_scale=ks)
        sel = selections(cal, k_hi, seed)
        variants[f"{tname}/uniform_int8"] = (layout_for(d, 0, tier), None)
        for sname, perm in sel.items():
            variants[f"{tname}/{sname}"] = (layout_for(d, k_hi, tier), perm)
        del cal
    g_run = torch.Generator(device="cuda")
    g_run.manual_seed(3000 + seed)

    def held_out():
        for _ in range(steps):
            yield inputs.decode_inputs_device(g_run, B, HK, HV, d, kda=kda, mu=mu, key_scale=ks)

    res = trajectory_rrmse(kda=kda, HK=HK, S0=S0, variants=variants, step_inputs=held_out())
    res["config"] = dict(model="KDA" if kda else "GDN", B=B, HK=HK, HV=HV, d=d, k_hi=k_hi,
                         warm_tokens=warm, calib_tokens=calib_tokens, held_out_steps=steps,
                         key_channels=key_channels, key_factor=key_factor if key_channels else None)
    if log:
        tag = res["config"]["model"] + (f" ({key_channels} key channels x{key_factor})" if key_channels else "")
        for name, r in res.items():
            if isinstance(r, dict) and "state_rrmse" in r:
                log(f"  {tag} {name}: state RRMSE {r['state_rrmse']:.3e}, "
                    f"output RRMSE {r['output_rrmse']:.3e}")
    return res
