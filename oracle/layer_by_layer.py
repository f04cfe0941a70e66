"""Layer-by-layer (unfused) attention with bfloat16 intermediates, float64 arithmetic.

TEST INFRASTRUCTURE ONLY (see the package docstring). This is the oracle of the unfused GPU
baseline. It follows the paper's diagnostic baseline mapping (Sec. "Diagnostic Baseline: Unfused
Layer-by-Layer Attention"): attention as separate operators run one after another, each taking its
input from device memory and leaving its result there. Table 3 lists what that mapping spills (Q, K,
V, the score matrix QK^T, the probability matrix G and the row scale), all in bfloat16. For one head,
with visible keys as in Eq. (1) plus the causal mask:

1. score operator:  S~ = bf16(scale * Q K^T), every entry (the score operator is a plain product);
2. mask + softmax:  LSE_i = log sum_{j visible} exp(S~_ij);
                    G_ij = bf16(exp(S~_ij - LSE_i)) for visible j, and 0 for masked j;
3. value operator:  O = bf16(G V).

Readings where the paper is silent (each listed in the design notes): the scale is applied inside the
score operator, before rounding; the softmax output is normalised before it is rounded (it is the
probability matrix itself, so the value operator is a plain product); the row statistic that
travels with it is the natural-log LSE in fp32. Everything between the roundings is float64.
"""

from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

# Largest finite bfloat16, (2 - 2^-7) * 2^127.
BF16_MAX = float.fromhex("0x1.fep127")


def round_bf16(x) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value, ties to even (returned as float64).

    bfloat16 keeps 8 significant bits and the binary32 exponent range. For |x| in [2^(e-1), 2^e)
    consecutive bfloat16 values are 2^(e-8) apart; below the smallest normal (2^-126) the spacing
    stays 2^-133. Scaling by a power of two is exact in float64, so one call of numpy's
    round-half-to-even on x / spacing is the correctly rounded result, with a single rounding (not
    via binary32, which could round twice). Magnitudes that round to 2^128 or above overflow to
    infinity; infinities and NaN pass through.
    """
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    q = np.maximum(e.astype(np.int64) - 8, -133)
    y = np.ldexp(np.round(np.ldexp(x, -q)), q)
    finite = np.isfinite(x)
    y = np.where(finite & (np.abs(y) >= 2.0 ** 128), np.copysign(np.inf, x), y)
    return np.where(finite, y, x)


def _visible(n: int, sk: int, causal: bool, q_pos: Optional[Sequence[int]], sq: Optional[int]) -> np.ndarray:
    """[n, sk] mask of visible keys: all keys, or key j <= i + (Sk - Sq) for query position i."""
    if not causal:
        return np.ones((n, sk), dtype=bool)
    pos = np.arange(n) if q_pos is None else np.asarray(q_pos, dtype=np.int64)
    sq = n if sq is None else int(sq)
    return np.arange(sk)[None, :] <= (pos[:, None] + (sk - sq))


def lbl_scores_head(q, k, scale: float) -> np.ndarray:
    """Score operator for one head: S~ = bf16(scale * Q K^T), q: [n, dqk], k: [Sk, dqk] -> [n, Sk]."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    return round_bf16(scale * (q @ k.T))


def lbl_softmax_head(s, causal: bool, q_pos: Optional[Sequence[int]] = None, sq: Optional[int] = None):
    """Mask + softmax operator for one head on the spilled scores s: [n, Sk] (bf16 values).

    Returns (G [n, Sk], LSE [n]): G = bf16(exp(s - LSE)) on visible keys and 0 on masked ones; a row
    that sees no key gets G = 0 and LSE = -inf.
    """
    s = np.asarray(s, dtype=np.float64)
    n, sk = s.shape
    vis = _visible(n, sk, causal, q_pos, sq)
    t = np.where(vis, s, -np.inf)
    m = t.max(axis=1) if sk > 0 else np.full(n, -np.inf)
    empty = np.isneginf(m)
    m_ref = np.where(empty, 0.0, m)
    l = np.exp(t - m_ref[:, None]).sum(axis=1)
    lse = np.where(empty, -np.inf, m_ref + np.log(np.where(empty, 1.0, l)))
    lse_ref = np.where(empty, 0.0, lse)
    g = np.where(vis & ~empty[:, None], round_bf16(np.exp(t - lse_ref[:, None])), 0.0)
    return g, lse


def lbl_pv_head(g, v) -> np.ndarray:
    """Value operator for one head: O = bf16(G V), g: [n, Sk], v: [Sk, dv] -> [n, dv]."""
    g = np.asarray(g, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    if g.shape[1] == 0:
        return np.zeros((g.shape[0], v.shape[1]))
    return round_bf16(g @ v)


def layer_by_layer_attention(q, k, v, scale: float, causal: bool, return_intermediates: bool = False):
    """The three operators over contiguous BHSD arrays; query head h reads key/value head
    h // (Hq // Hkv). Returns O [B, Hq, Sq, dv] and LSE [B, Hq, Sq]; with ``return_intermediates``
    also S~ and G [B, Hq, Sq, Sk]."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, Hq, Sq, _ = q.shape
    Hkv, Sk, dv = k.shape[1], k.shape[2], v.shape[3]
    if Hkv == 0 or Hq % Hkv:
        raise ValueError("Hq must be a positive multiple of Hkv")
    group = Hq // Hkv
    o = np.zeros((B, Hq, Sq, dv))
    lse = np.zeros((B, Hq, Sq))
    s_all = np.zeros((B, Hq, Sq, Sk)) if return_intermediates else None
    g_all = np.zeros((B, Hq, Sq, Sk)) if return_intermediates else None
    for b in range(B):
        for h in range(Hq):
            kv = h // group
            s = lbl_scores_head(q[b, h], k[b, kv], scale)
            g, lse[b, h] = lbl_softmax_head(s, causal)
            o[b, h] = lbl_pv_head(g, v[b, kv])
            if return_intermediates:
                s_all[b, h], g_all[b, h] = s, g
    if return_intermediates:
        return o, lse, s_all, g_all
    return o, lse


def lbl_error_bound(max_abs_score, max_abs_v):
    """Bound on |O_lbl - O| per output row, from the three bf16 roundings (unit roundoff u = 2^-8).

    With M the row's largest visible |exact score|: each spilled score moves by at most u*M, so each
    log-probability moves by at most 2*u*M (the score and the LSE, which is 1-Lipschitz in the max
    norm); rounding G multiplies each probability by at most (1 + u) and rounding O adds u*|O|.
    Since the probabilities sum to 1: |O_lbl - O| <= max|V| * ((1 + u)^2 * exp(2*u*M) - 1).
    """
    u = 2.0 ** -8
    m = np.asarray(max_abs_score, dtype=np.float64)
    return np.asarray(max_abs_v, dtype=np.float64) * ((1 + u) ** 2 * np.exp(2 * u * m) - 1)
