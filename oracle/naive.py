"""Naive three-stage attention in float64 -- the oracle the GPU path is checked against.

TEST INFRASTRUCTURE ONLY (see the package docstring). Follows the paper's statement of scaled
dot-product attention, Eq. (1) in Sec. 2.1: for one head, O = softmax(scale * Q K^T) V with
Q in R^{lq x dk}, K in R^{lk x dk}, V in R^{lk x dv}, replicated over heads. The score matrix is
materialised in full; this is the quadratic-memory formulation that FlashAttention reorders
without changing its result (Sec. 2.1, the paragraph after Alg. 2).

Readings where the paper is silent (each listed in the design notes):

* scale is a caller argument (Eq. 1 uses 1/sqrt(dk)); it multiplies the fp64 scores.
* causal masking is bottom-right aligned: key j is visible to query i iff j <= i + (Sk - Sq),
  which is the usual j <= i when Sq == Sk. Rows that see no key give O = 0 and LSE = -inf.
* grouped-query attention: query head h reads key/value head h // (Hq // Hkv).
* LSE is the natural-log log-sum-exp of the visible scaled scores of each query row.
"""

from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import numpy as np


def bf16_bits_to_f64(bits) -> np.ndarray:
    """Decode bfloat16 bit patterns (any integer array) to float64, exactly.

    A bfloat16 is the upper 16 bits of an IEEE binary32; widening to binary32 by appending 16 zero
    bits and then to binary64 is exact.
    """
    b = np.asarray(bits).astype(np.uint32) & 0xFFFF
    return (b << 16).astype(np.uint32).view(np.float32).astype(np.float64)


def attention_head(q, k, v, scale: float, causal: bool, q_pos: Optional[Sequence[int]] = None,
                   sq: Optional[int] = None, return_p: bool = False):
    """Attention for one head (Eq. 1), materialising the full score matrix.

    q: [n, dqk] query rows at absolute positions ``q_pos`` (default 0..n-1) of a query sequence of
    length ``sq`` (default n); k: [Sk, dqk]; v: [Sk, dv]. Returns (O [n, dv], LSE [n]) and, with
    ``return_p``, the probability matrix P [n, Sk].
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    n, sk, dv = q.shape[0], k.shape[0], v.shape[1]
    q_pos = np.arange(n) if q_pos is None else np.asarray(q_pos, dtype=np.int64)
    sq = n if sq is None else int(sq)

    # Stage 1: the score matrix S = scale * Q K^T.
    s = scale * (q @ k.T)
    # Causal mask: hide keys j > i + (Sk - Sq).
    if causal:
        visible = np.arange(sk)[None, :] <= (q_pos[:, None] + (sk - sq))
        s = np.where(visible, s, -np.inf)
    # Stage 2: row-wise softmax, with the row max subtracted before exponentiation.
    m = s.max(axis=1) if sk > 0 else np.full(n, -np.inf)
    empty = np.isneginf(m)
    m_ref = np.where(empty, 0.0, m)
    e = np.exp(s - m_ref[:, None])
    l = e.sum(axis=1)
    l_safe = np.where(empty, 1.0, l)
    p = e / l_safe[:, None]
    # Stage 3: the weighted sum of value rows.
    o = p @ v if sk > 0 else np.zeros((n, dv))
    o[empty] = 0.0
    lse = np.where(empty, -np.inf, m_ref + np.log(l_safe))
    if return_p:
        return o, lse, p
    return o, lse


def _kv_head(h: int, hq: int, hkv: int) -> int:
    return h // (hq // hkv)


def naive_attention(q, k, v, scale: float, causal: bool, return_p: bool = False):
    """Batched multi-head attention over contiguous BHSD arrays.

    q: [B, Hq, Sq, dqk], k: [B, Hkv, Sk, dqk], v: [B, Hkv, Sk, dv] (any real dtype, used as float64).
    Returns O [B, Hq, Sq, dv] and LSE [B, Hq, Sq] (and P [B, Hq, Sq, Sk] with ``return_p``).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, Hq, Sq, _ = q.shape
    Hkv, Sk, dv = k.shape[1], k.shape[2], v.shape[3]
    if Hkv == 0 or Hq % Hkv:
        raise ValueError("Hq must be a positive multiple of Hkv")
    o = np.zeros((B, Hq, Sq, dv))
    lse = np.zeros((B, Hq, Sq))
    ps = np.zeros((B, Hq, Sq, Sk)) if return_p else None
    for b in range(B):
        for h in range(Hq):
            g = _kv_head(h, Hq, Hkv)
            res = attention_head(q[b, h], k[b, g], v[b, g], scale, causal, return_p=return_p)
            o[b, h], lse[b, h] = res[0], res[1]
            if return_p:
                ps[b, h] = res[2]
    return (o, lse, ps) if return_p else (o, lse)


def naive_attention_rows(q_rows_fn, k_head_fn, v_head_fn, B: int, Hq: int, Hkv: int, Sq: int,
                         scale: float, causal: bool, rows: List[np.ndarray]
                         ) -> List[Tuple[np.ndarray, np.ndarray]]:
    """Attention for a subset of query rows of every (batch, query head), head by head.

    The callables return float64 arrays on demand so that only one key/value head is widened at a
    time: ``q_rows_fn(b, h, rows) -> [len(rows), dqk]``, ``k_head_fn(b, g) -> [Sk, dqk]``,
    ``v_head_fn(b, g) -> [Sk, dv]``. ``rows[b * Hq + h]`` lists the absolute query positions.
    Returns one (O_rows, LSE_rows) pair per (b, h), in that order.
    """
    out = []
    cache_key, kh, vh = None, None, None
    for b in range(B):
        for h in range(Hq):
            g = _kv_head(h, Hq, Hkv)
            if cache_key != (b, g):
                kh, vh, cache_key = k_head_fn(b, g), v_head_fn(b, g), (b, g)
            r = rows[b * Hq + h]
            out.append(attention_head(q_rows_fn(b, h, r), kh, vh, scale, causal, q_pos=r, sq=Sq))
    return out
