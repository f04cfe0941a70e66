"""Online-softmax attention in float64, written from the paper's two algorithms.

TEST INFRASTRUCTURE ONLY. This is an independent second route to the same result as
:mod:`oracle.naive`; the tests require the two to agree to 1e-12.

* :func:`flash_tile` follows Alg. 1 ("Per-tile FlashAttention"): scale the query block, stream the
  key/value rows in chunks of ``bn``, keep the running row max u and row sum s, rescale the
  unnormalised accumulator G' by r = exp(u_old - u_new) and add P V. It returns the unnormalised
  triple (G', u, s).
* :func:`spatial_flash_attention` follows Alg. 2 ("Tile-to-tile FlashAttention"): query blocks of
  ``bm`` rows, the key range split into C contiguous parts, one Alg. 1 run per part, then a merge.

Readings of the printed algorithms (each listed in the design notes):

* The causal mask of Alg. 1 is an additive 0/-inf matrix that initialises G before the score
  product is added; without causal masking G starts at 0.
* No divisibility of lq, lk by the block sizes is required; the last block is short.
* The merge in Alg. 2 is read as the log-sum-exp combination: u = max(u_a, u_b), both partial
  accumulators and sums are rescaled by exp(u_part - u) before adding. The printed merge rescales
  only the running side, by the previous part's max, which is not the same unless the maxima agree.
* When a row has seen no visible key yet (u = -inf), its probabilities are 0 and the rescale
  factor is taken as 1 (nothing has been accumulated).
* No bfloat16 conversion of P: the oracle stays in float64 throughout.
"""

from __future__ import annotations

from typing import Tuple

import numpy as np


def flash_tile(q_blk, k, v, scale: float, causal: bool, bn: int, q_pos, k_off: int, sk_total: int,
               sq_total: int) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Alg. 1 for one query block against the key/value rows ``k``, ``v``.

    ``q_pos`` are the absolute positions of the query rows; ``k_off`` is the absolute position of
    ``k[0]`` in a key sequence of length ``sk_total``; ``sq_total`` is the full query length (they
    set the causal alignment). Returns (G' [n, dv], u [n], s [n]).
    """
    A = np.asarray(q_blk, dtype=np.float64) * scale
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    n, dv = A.shape[0], v.shape[1]
    q_pos = np.asarray(q_pos, dtype=np.int64)
    G_acc = np.zeros((n, dv))
    u_prev = np.full(n, -np.inf)
    s_prev = np.zeros(n)
    for j0 in range(0, k.shape[0], bn):
        Kj = k[j0:j0 + bn]
        Vj = v[j0:j0 + bn]
        G = np.zeros((n, Kj.shape[0]))
        if causal:
            key_pos = k_off + j0 + np.arange(Kj.shape[0])
            G = np.where(key_pos[None, :] <= q_pos[:, None] + (sk_total - sq_total), 0.0, -np.inf)
        G = A @ Kj.T + G
        u = np.maximum(u_prev, G.max(axis=1))
        seen = ~np.isneginf(u)
        u_ref = np.where(seen, u, 0.0)
        P = np.exp(G - u_ref[:, None])
        r = np.where(seen, np.exp(u_prev - u_ref), 1.0)
        G_acc = P @ Vj + G_acc * r[:, None]
        s = P.sum(axis=1) + s_prev * r
        u_prev, s_prev = u, s
    return G_acc, u_prev, s_prev


def _merge(a, b):
    """Combine two partial summaries (G', u, s) of disjoint key ranges (log-sum-exp merge)."""
    Ga, ua, sa = a
    Gb, ub, sb = b
    u = np.maximum(ua, ub)
    seen = ~np.isneginf(u)
    u_ref = np.where(seen, u, 0.0)
    ra = np.exp(ua - u_ref)
    rb = np.exp(ub - u_ref)
    return Ga * ra[:, None] + Gb * rb[:, None], u, sa * ra + sb * rb


def spatial_flash_attention(q, k, v, scale: float, causal: bool, bm: int, bn: int, C: int = 1):
    """Alg. 2 over one head: q [Sq, dqk], k [Sk, dqk], v [Sk, dv]. Returns (O [Sq, dv], LSE [Sq])."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    sq, sk, dv = q.shape[0], k.shape[0], v.shape[1]
    o = np.zeros((sq, dv))
    lse = np.full(sq, -np.inf)
    bounds = [(c * sk) // C for c in range(C + 1)]
    for i0 in range(0, sq, bm):
        q_pos = np.arange(i0, min(i0 + bm, sq))
        Qb = q[i0:i0 + bm]
        parts = [flash_tile(Qb, k[bounds[c]:bounds[c + 1]], v[bounds[c]:bounds[c + 1]], scale, causal,
                            bn, q_pos, bounds[c], sk, sq) for c in range(C)]
        acc = parts[0]
        for c in range(1, C):
            acc = _merge(acc, parts[c])
        G, u, s = acc
        ok = s > 0
        o[i0:i0 + bm] = np.where(ok[:, None], G / np.where(ok, s, 1.0)[:, None], 0.0)
        lse[i0:i0 + bm] = np.where(ok, u + np.log(np.where(ok, s, 1.0)), -np.inf)
    return o, lse
