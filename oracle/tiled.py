"""Streaming (online-softmax) attention in float64: a second route to the result of Eq. (1).

TEST INFRASTRUCTURE ONLY. This is an independent second route to the same result as
:mod:`oracle.naive`; the tests require the two to agree to 1e-12.

The method of the paper's two algorithms (Alg. 1, per-tile; Alg. 2, tile-to-tile; Sec. 2.1) rests on
one fact: softmax attention over a union of disjoint key sets can be assembled from the attention
over each set, provided each set also reports how much probability mass it carries. For a query
row and a key set J write

    Z(J) = log sum_{j in J} exp(s_j)            (the set's log-sum-exp, -inf for no visible key)
    A(J) = sum_{j in J} exp(s_j - Z(J)) v_j     (attention restricted to J, 0 when Z(J) = -inf)

Then for disjoint J1, J2, with Z = log(exp Z(J1) + exp Z(J2)):

    Z(J1 u J2) = Z,    A(J1 u J2) = exp(Z(J1) - Z) A(J1) + exp(Z(J2) - Z) A(J2).

This module keeps exactly that pair (A, Z) per query row and folds it over key chunks:

* :func:`flash_tile` -- Alg. 1's job for one block of query rows: the keys arrive in chunks of ``bn``
  rows, each chunk's (A, Z) is computed directly and folded into the running pair. The result for
  the block is the pair over all the keys it was given.
* :func:`spatial_flash_attention` -- Alg. 2's job: query blocks of ``bm`` rows, the key range cut
  into C contiguous parts, one :func:`flash_tile` per part, then the parts folded together with the
  same combination.

The paper's algorithms carry the unnormalised form of the same state (a running maximum, a running
sum of exponentials relative to it, and the unnormalised product with V); normalising at every fold,
as here, is mathematically identical and keeps this code structurally apart from the kernel, which
uses the unnormalised form. Readings (each listed in the design notes): the causal mask is a
0 / -inf addition to the scores, absent in non-causal mode; no divisibility of the sequence lengths
by the block sizes is required; the merge of parts is the combination above (the log-sum-exp merge;
the printed Alg. 2 rescales with the previous part's maximum, which agrees only when the maxima
do); a row with no visible key so far carries Z = -inf and A = 0 and contributes nothing to a fold.
No bfloat16 rounding anywhere: float64 throughout.
"""

from __future__ import annotations

from typing import Tuple

import numpy as np


def _chunk_pair(z):
    """(A-weights, Z) of one key chunk for every row: the chunk's log-sum-exp Z (-inf for a row with
    no visible key in the chunk) and the chunk-local softmax weights (0 for such a row)."""
    peak = z.max(axis=1) if z.shape[1] else np.full(z.shape[0], -np.inf)
    live = np.isfinite(peak)
    shift = np.where(live, peak, 0.0)
    e = np.exp(z - shift[:, None])
    mass = e.sum(axis=1)
    lse = np.where(live, shift + np.log(np.where(live, mass, 1.0)), -np.inf)
    weights = np.where(live[:, None], e / np.where(live, mass, 1.0)[:, None], 0.0)
    return weights, lse


def _fold(a1, z1, a2, z2):
    """Combine the (A, Z) pairs of two disjoint key sets (rows of A are output vectors)."""
    z = np.logaddexp(z1, z2)
    live = np.isfinite(z)
    zs = np.where(live, z, 0.0)
    w1 = np.where(live, np.exp(z1 - zs), 0.0)
    w2 = np.where(live, np.exp(z2 - zs), 0.0)
    return w1[:, None] * a1 + w2[:, None] * a2, z


def flash_tile(q_blk, k, v, scale: float, causal: bool, bn: int, q_pos, k_off: int, sk_total: int,
               sq_total: int) -> Tuple[np.ndarray, np.ndarray]:
    """Attention of one block of query rows over the keys ``k``, ``v``, streamed ``bn`` keys at a time.

    ``q_pos`` are the absolute positions of the query rows in a query sequence of length
    ``sq_total``; ``k_off`` is the absolute position of ``k[0]`` in a key sequence of length
    ``sk_total`` (together they set the bottom-right causal alignment: key j is visible to query i
    iff j <= i + sk_total - sq_total). Returns (A [n, dv], Z [n]) over all the given keys.
    """
    qb = np.asarray(q_blk, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    q_pos = np.asarray(q_pos, dtype=np.int64)
    rows, dv = qb.shape[0], v.shape[1]
    acc = np.zeros((rows, dv))
    z_acc = np.full(rows, -np.inf)
    limit = q_pos + (sk_total - sq_total)  # last visible key of each row
    for c0 in range(0, k.shape[0], bn):
        kc, vc = k[c0:c0 + bn], v[c0:c0 + bn]
        z = scale * (qb @ kc.T)
        if causal:
            pos = k_off + c0 + np.arange(kc.shape[0])
            z = z + np.where(pos[None, :] <= limit[:, None], 0.0, -np.inf)
        weights, z_c = _chunk_pair(z)
        acc, z_acc = _fold(acc, z_acc, weights @ vc, z_c)
    return acc, z_acc


def spatial_flash_attention(q, k, v, scale: float, causal: bool, bm: int, bn: int, C: int = 1):
    """Alg. 2's two-level decomposition over one head: q [Sq, dqk], k [Sk, dqk], v [Sk, dv]; query
    blocks of ``bm`` rows, the keys cut into C contiguous parts of about Sk / C keys, each part
    streamed in chunks of ``bn``. Returns (O [Sq, dv], LSE [Sq]); rows with no visible key get O = 0,
    LSE = -inf."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    sq, sk, dv = q.shape[0], k.shape[0], v.shape[1]
    o = np.zeros((sq, dv))
    lse = np.full(sq, -np.inf)
    cuts = [(c * sk) // C for c in range(C + 1)]
    for r0 in range(0, sq, bm):
        pos = np.arange(r0, min(r0 + bm, sq))
        acc, z_acc = np.zeros((len(pos), dv)), np.full(len(pos), -np.inf)
        for c in range(C):
            a_c, z_c = flash_tile(q[pos], k[cuts[c]:cuts[c + 1]], v[cuts[c]:cuts[c + 1]], scale, causal, bn, pos,
                                  cuts[c], sk, sq)
            acc, z_acc = _fold(acc, z_acc, a_c, z_c)
        o[pos], lse[pos] = acc, z_acc
    return o, lse
