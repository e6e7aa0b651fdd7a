"""Seeded synthetic decode workloads for the DAMP state update.

This module only draws inputs: it holds none of the update's arithmetic,
so that the HIP path and the CPU oracle can be fed identical bytes without
sharing any code. Distributions follow the decode workloads the library is
benchmarked on (GDN/KDA heads of width 128, batch up to 1024):

  q, k   ~ N(0, 1), L2-normalised per head            (section 3.1 operands)
  v      ~ N(0, 1)
  beta   = sigmoid(N(0, 1))                           (delta-rule step size)
  g(GDN) = -softplus(N(0, 1)), one per (request, value head)
  g(KDA) = -softplus(N(mu[h, u], 1)) per key channel, with a fixed
           mu[h, u] ~ N(-2, 2^2) per (head, channel), so that ~10% of the
           channels are persistent (median decay exp(g) > 0.99)

Every array is rounded once to bf16 (torch's round-to-nearest-even cast) and
returned as uint16 bit patterns; both sides consume exactly those bits.
"""
from __future__ import annotations

import numpy as np


def to_bf16_bits(x) -> np.ndarray:
    """fp32 values -> bf16 bit patterns (uint16), via torch's CPU cast."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def _softplus(x):
    return np.logaddexp(np.float32(0.0), x).astype(np.float32)


def _sigmoid(x):
    return (1.0 / (1.0 + np.exp(-x))).astype(np.float32)


def _unit(x):
    n = np.sqrt(np.sum(x.astype(np.float64) ** 2, axis=-1, keepdims=True))
    return (x / np.maximum(n, 1e-12)).astype(np.float32)


def kda_mu(seed: int, hv: int, d: int) -> np.ndarray:
    """Per-(head, channel) mean of the KDA decay logits."""
    rng = np.random.default_rng([seed, 0x6d75])
    return rng.normal(-2.0, 2.0, size=(hv, d)).astype(np.float32)


def decode_inputs(seed: int, steps: int, B: int, HK: int, HV: int, d: int, *,
                  kda: bool = False, mu: np.ndarray | None = None) -> dict:
    """Inputs of `steps` decode steps as bf16 bits with a leading step axis:
    q, k [T, B, HK, d]; v [T, B, HV, d]; g [T, B, HV] (GDN) or [T, B, HV, d]
    (KDA); beta [T, B, HV]."""
    rng = np.random.default_rng(seed)
    f = np.float32
    q = _unit(rng.standard_normal((steps, B, HK, d), dtype=f))
    k = _unit(rng.standard_normal((steps, B, HK, d), dtype=f))
    v = rng.standard_normal((steps, B, HV, d), dtype=f)
    if kda:
        if mu is None:
            mu = kda_mu(seed, HV, d)
        g = -_softplus(mu[None, None] + rng.standard_normal((steps, B, HV, d), dtype=f))
    else:
        g = -_softplus(rng.standard_normal((steps, B, HV), dtype=f))
    beta = _sigmoid(rng.standard_normal((steps, B, HV), dtype=f))
    return {name: to_bf16_bits(a) for name, a in
            dict(q=q, k=k, v=v, g=g, beta=beta).items()}


def step(inp: dict, t: int) -> dict:
    """The inputs of step t (drops the leading step axis)."""
    return {name: np.ascontiguousarray(a[t]) for name, a in inp.items()}


def as_prefill(inp: dict) -> dict:
    """Step-major inputs [T, B, ...] as one prefill chunk per request
    [B, T, ...] (the same values)."""
    return {name: np.ascontiguousarray(np.swapaxes(a, 0, 1)) for name, a in inp.items()}


def outlier_channels(seed: int, hv: int, d: int, n: int = 8) -> np.ndarray:
    """n distinct key channels per head, int32 [hv, n], ascending."""
    rng = np.random.default_rng([seed, 0x6f75])
    return np.sort(np.stack([rng.choice(d, size=n, replace=False) for _ in range(hv)]),
                   axis=1).astype(np.int32)


def scale_channels(S: np.ndarray, channels: np.ndarray, factor: float = 10.0) -> np.ndarray:
    """Multiplies key-channel rows of states [..., HV, d_k, d_v] in place:
    channels[h] lists the rows of head h (outlier injection)."""
    for h in range(channels.shape[0]):
        S[..., h, channels[h], :] *= np.float32(factor)
    return S


def random_perms(seed: int, hv: int, d: int) -> np.ndarray:
    """A random permutation of the d key channels per head, uint8 [hv, d]."""
    rng = np.random.default_rng([seed, 0x7065])
    return np.stack([rng.permutation(d) for _ in range(hv)]).astype(np.uint8)


def slot_order(seed: int, num_slots: int, n_active: int) -> np.ndarray:
    """n_active distinct pool slots in random (non-contiguous) order."""
    rng = np.random.default_rng([seed, 0x736c])
    return rng.choice(num_slots, size=n_active, replace=False).astype(np.int32)


def synthetic_states(seed: int, B: int, HV: int, d: int, rank: int = 16) -> np.ndarray:
    """Warm-looking fp32 states [B, HV, d, d] without running any recurrence:
    a sum of `rank` random outer products k_i v_i^T with geometrically
    decaying weights plus small noise (a stand-in for a state that has
    absorbed many tokens)."""
    rng = np.random.default_rng([seed, 0x7374])
    f = np.float32
    K = _unit(rng.standard_normal((B * HV, rank, d), dtype=f))
    V = rng.standard_normal((B * HV, rank, d), dtype=f)
    w = (0.8 ** np.arange(rank, dtype=f)) * 0.5
    S = np.matmul(np.swapaxes(K * w[None, :, None], 1, 2), V)
    S += f(0.01) * rng.standard_normal(S.shape, dtype=f)
    return S.reshape(B, HV, d, d).astype(f)


def key_channel_scale(seed: int, hk: int, d: int, n: int = 8, factor: float = 4.0) -> np.ndarray:
    """fp32 [hk, d]: 1 everywhere except n seeded channels per key head, which
    get `factor` (an anisotropic key distribution whose energy concentrates
    in a few key channels, applied before the L2 normalization)."""
    s = np.ones((hk, d), np.float32)
    ch = outlier_channels(seed, hk, d, n)
    for h in range(hk):
        s[h, ch[h]] = np.float32(factor)
    return s


def decode_inputs_device(gen, B: int, HK: int, HV: int, d: int, *, kda: bool = False,
                         mu=None, key_scale=None, device="cuda") -> dict:
    """One decode step of the same distributions drawn on the GPU with a seeded
    torch.Generator (used for long warm-up and calibration runs, where moving
    host arrays would dominate). key_scale (device fp32 [HK, d], optional)
    multiplies k before its normalization. Returns bf16 device tensors
    q, k [B, HK, d]; v [B, HV, d]; g [B, HV] or [B, HV, d]; beta [B, HV]."""
    import torch

    f = torch.float32
    q = torch.randn((B, HK, d), generator=gen, device=device, dtype=f)
    k = torch.randn((B, HK, d), generator=gen, device=device, dtype=f)
    if key_scale is not None:
        k = k * key_scale
    q = q / q.norm(dim=-1, keepdim=True).clamp_min(1e-12)
    k = k / k.norm(dim=-1, keepdim=True).clamp_min(1e-12)
    v = torch.randn((B, HV, d), generator=gen, device=device, dtype=f)
    if kda:
        x = torch.randn((B, HV, d), generator=gen, device=device, dtype=f) + mu
    else:
        x = torch.randn((B, HV), generator=gen, device=device, dtype=f)
    g = -torch.nn.functional.softplus(x)
    beta = torch.sigmoid(torch.randn((B, HV), generator=gen, device=device, dtype=f))
    bf = torch.bfloat16
    return dict(q=q.to(bf), k=k.to(bf), v=v.to(bf), g=g.to(bf), beta=beta.to(bf))
