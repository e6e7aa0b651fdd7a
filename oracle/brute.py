"""fp64 brute force of the GDN / KDA recurrence - TEST INFRASTRUCTURE ONLY.

Used to pin the fp32 C oracle (damp_oracle.c) to the paper's equations by a
route that shares nothing with it: explicit d_k x d_k transition matrices,
matrix products in float64, no permutation, no packing.

  delta_step  section 3.1 Eq. (1): S_bar = Lambda S, delta = v - S_bar^T k,
              S = S_bar + beta k delta^T, o = S^T q.
  transition  section 3.1 Eq. (2): A_t = (I - beta_t k_t k_t^T) Lambda_t.
  unrolled    Eq. (2) unrolled from S_0:
              S_T = (A_T ... A_1) S_0 + sum_i (A_T ... A_{i+1}) beta_i k_i v_i^T.
GDN is the case Lambda_t = exp(g_t) I, KDA the case diag(exp(g_t)).
Only tests may import this module.
"""
from __future__ import annotations

import numpy as np


def widen_bf16(u) -> np.ndarray:
    """bf16 bit patterns -> float64 (exact)."""
    u = np.asarray(u, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def decay_vector(g, dk: int) -> np.ndarray:
    """Diagonal of Lambda: exp(g) per channel (g scalar for GDN)."""
    g = np.asarray(g, dtype=np.float64)
    return np.exp(np.broadcast_to(g, (dk,)) if g.ndim == 0 else g)


def transition(k, lam, beta) -> np.ndarray:
    dk = k.shape[0]
    return (np.eye(dk) - beta * np.outer(k, k)) @ np.diag(lam)


def delta_step(S, q, k, v, lam, beta, scale=1.0):
    """Eq. (1) in float64; returns (S_t, o_t)."""
    S_bar = lam[:, None] * S
    delta = v - S_bar.T @ k
    S_new = S_bar + beta * np.outer(k, delta)
    return S_new, scale * (S_new.T @ q)


def unrolled(S0, ks, vs, lams, betas) -> np.ndarray:
    """S_T from the closed form of Eq. (2), built with explicit products."""
    T = len(ks)
    dk = S0.shape[0]
    A = [transition(ks[t], lams[t], betas[t]) for t in range(T)]
    prod = np.eye(dk)
    for t in range(T):          # A_T ... A_1
        prod = A[t] @ prod
    S = prod @ S0
    for i in range(T):
        tail = np.eye(dk)
        for t in range(i + 1, T):  # A_T ... A_{i+1}
            tail = A[t] @ tail
        S = S + tail @ (betas[i] * np.outer(ks[i], vs[i]))
    return S


def head_inputs(inp: dict, t: int, b: int, h: int, HK: int, HV: int, kda: bool):
    """float64 operands of one (step, request, value head) from bf16 bits.
    Value head h reads key head h // (HV // HK)."""
    hk = h // (HV // HK)
    q = widen_bf16(inp["q"][t, b, hk])
    k = widen_bf16(inp["k"][t, b, hk])
    v = widen_bf16(inp["v"][t, b, h])
    g = widen_bf16(inp["g"][t, b, h])
    beta = float(widen_bf16(inp["beta"][t, b, h]))
    return q, k, v, decay_vector(g, q.shape[0]), beta


def trajectory(S0, inp: dict, b: int, h: int, HK: int, HV: int, kda: bool, scale=1.0):
    """Eq. (1) step by step in float64 for one (request, head); returns the
    list of states and outputs after every step."""
    S = np.asarray(S0, dtype=np.float64)
    states, outs = [], []
    for t in range(inp["q"].shape[0]):
        q, k, v, lam, beta = head_inputs(inp, t, b, h, HK, HV, kda)
        S, o = delta_step(S, q, k, v, lam, beta, scale)
        states.append(S)
        outs.append(o)
    return states, outs
