"""Pins for the fp64 oracle: facts that hold independently of the oracle's own code.

Each test checks the oracle against something it cannot agree with by construction: torch's float64
CPU attention routine, closed forms, invariances of softmax attention, a brute force over Python
floats, and the paper's printed throughput table for the FLOP formula. A dropped term, a wrong sign
or index, a transposed operand or a wrong mask alignment fails at least one of them.
"""

import csv
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import workloads as W
from oracle import (attention_head, bf16_bits_to_f64, brute_attention, naive_attention,
                    naive_attention_rows, spatial_flash_attention)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
RNG = np.random.default_rng(12345)


def rnd(*shape, scale=1.0):
    return RNG.standard_normal(shape) * scale


def sdpa64(q, k, v, scale, causal):
    """torch's CPU scaled_dot_product_attention in float64, bottom-right causal via an explicit mask."""
    B, Hq, Sq, _ = q.shape
    Hkv, Sk = k.shape[1], k.shape[2]
    qt, kt, vt = (torch.from_numpy(np.ascontiguousarray(x)) for x in (q, k, v))
    if Hq != Hkv:
        kt = kt.repeat_interleave(Hq // Hkv, dim=1)
        vt = vt.repeat_interleave(Hq // Hkv, dim=1)
    mask = None
    if causal:
        mask = torch.ones(Sq, Sk, dtype=torch.bool).tril(diagonal=Sk - Sq)
    return F.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=scale).numpy()


# ---------------------------------------------------------------------------------------------
# bfloat16 decoding
# ---------------------------------------------------------------------------------------------

def test_bf16_decode_known_patterns():
    bits = np.array([0x0000, 0x8000, 0x3F80, 0xC000, 0x7F80, 0xFF80, 0x3E00, 0x0001, 0x7F7F])
    got = bf16_bits_to_f64(bits)
    want = [0.0, -0.0, 1.0, -2.0, math.inf, -math.inf, 0.125, 2.0 ** -133, 3.3895313892515355e38]
    assert np.array_equal(got, np.array(want))
    assert math.copysign(1.0, got[1]) == -1.0


def test_bf16_decode_matches_torch_widening():
    x = torch.randn(4096, generator=torch.Generator().manual_seed(3)).to(torch.bfloat16)
    bits = x.view(torch.int16).numpy()
    assert np.array_equal(bf16_bits_to_f64(bits), x.to(torch.float64).numpy())


# ---------------------------------------------------------------------------------------------
# library routine: torch float64 SDPA
# ---------------------------------------------------------------------------------------------

@pytest.mark.parametrize("B,Hq,Hkv,Sq,Sk,dqk,dv,causal", [
    (1, 1, 1, 17, 17, 8, 8, False),
    (2, 4, 2, 33, 33, 16, 8, True),
    (1, 6, 3, 9, 23, 12, 5, False),
    (1, 2, 1, 5, 31, 4, 4, True),     # Sq < Sk, bottom-right alignment
    (2, 3, 3, 40, 40, 7, 11, True),
])
def test_naive_matches_torch_sdpa_f64(B, Hq, Hkv, Sq, Sk, dqk, dv, causal):
    q, k, v = rnd(B, Hq, Sq, dqk), rnd(B, Hkv, Sk, dqk), rnd(B, Hkv, Sk, dv)
    scale = 0.37
    o, lse = naive_attention(q, k, v, scale, causal)
    ref = sdpa64(q, k, v, scale, causal)
    assert np.max(np.abs(o - ref)) < 1e-12
    # LSE against an independent log-sum-exp of torch's float64 score matrix.
    kk = np.repeat(k, Hq // Hkv, axis=1)
    s = torch.from_numpy(scale * np.einsum("bhid,bhjd->bhij", q, kk))
    if causal:
        s = s.masked_fill(~torch.ones(Sq, Sk, dtype=torch.bool).tril(diagonal=Sk - Sq), -math.inf)
    assert np.max(np.abs(lse - torch.logsumexp(s, dim=-1).numpy())) < 1e-12


# ---------------------------------------------------------------------------------------------
# softmax and weighted-sum properties
# ---------------------------------------------------------------------------------------------

@pytest.mark.parametrize("causal", [False, True])
def test_probabilities_are_a_distribution(causal):
    q, k, v = rnd(1, 2, 30, 8), rnd(1, 2, 30, 8), rnd(1, 2, 30, 6)
    _, _, p = naive_attention(q, k, v, 0.5, causal, return_p=True)
    assert np.all(p >= 0)
    assert np.max(np.abs(p.sum(-1) - 1.0)) < 1e-12
    if causal:
        upper = np.triu(np.ones((30, 30), dtype=bool), k=1)
        assert np.all(p[..., upper] == 0.0)


@pytest.mark.parametrize("causal", [False, True])
def test_constant_values_return_the_constant(causal):
    q, k = rnd(1, 3, 21, 8, scale=3.0), rnd(1, 3, 21, 8, scale=3.0)
    c = np.array([1.5, -2.25, 0.0, 7.0])
    v = np.broadcast_to(c, (1, 3, 21, 4)).copy()
    o, _ = naive_attention(q, k, v, 0.9, causal)
    assert np.max(np.abs(o - c)) < 1e-12


def test_two_keys_closed_form():
    # d = 1, two keys: softmax of two logits is a logistic sigmoid.
    q, k, v = np.array([[0.7]]), np.array([[1.3], [-0.4]]), np.array([[2.0], [-3.0]])
    scale = 1.1
    s0, s1 = scale * 0.7 * 1.3, scale * 0.7 * -0.4
    sig = lambda x: 1.0 / (1.0 + math.exp(-x))
    want = sig(s0 - s1) * 2.0 + sig(s1 - s0) * -3.0
    o, lse = attention_head(q, k, v, scale, False)
    assert abs(o[0, 0] - want) < 1e-14
    assert abs(lse[0] - math.log(math.exp(s0) + math.exp(s1))) < 1e-14


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("zero", ["q", "scale"])
def test_uniform_weights_give_prefix_mean(causal, zero):
    Sq = Sk = 25
    q, k, v = rnd(1, 1, Sq, 8), rnd(1, 1, Sk, 8), rnd(1, 1, Sk, 5)
    scale = 0.7
    if zero == "q":
        q[:] = 0.0
    else:
        scale = 0.0
    o, lse = naive_attention(q, k, v, scale, causal)
    for i in range(Sq):
        n = i + 1 if causal else Sk
        assert np.max(np.abs(o[0, 0, i] - v[0, 0, :n].mean(axis=0))) < 1e-12
        assert abs(lse[0, 0, i] - math.log(n)) < 1e-13


def test_causal_first_row_is_first_value():
    q, k, v = rnd(1, 2, 12, 8), rnd(1, 2, 12, 8), rnd(1, 2, 12, 8)
    o, lse = naive_attention(q, k, v, 0.3, True)
    assert np.array_equal(o[:, :, 0], v[:, :, 0])
    assert np.allclose(lse[:, :, 0], 0.3 * np.einsum("bhd,bhd->bh", q[:, :, 0], k[:, :, 0]), atol=1e-14)


def test_key_shift_invariance():
    q, k, v = rnd(1, 2, 14, 6), rnd(1, 2, 19, 6), rnd(1, 2, 19, 3)
    w = rnd(6)
    scale = 0.45
    o1, l1 = naive_attention(q, k, v, scale, False)
    o2, l2 = naive_attention(q, k + w, v, scale, False)
    assert np.max(np.abs(o1 - o2)) < 1e-12
    assert np.max(np.abs((l2 - l1) - scale * (q @ w))) < 1e-12


def test_permutation_equivariance():
    q, k, v = rnd(1, 1, 16, 6), rnd(1, 1, 22, 6), rnd(1, 1, 22, 4)
    perm_k, perm_q = RNG.permutation(22), RNG.permutation(16)
    o, lse = naive_attention(q, k, v, 0.8, False)
    o_k, _ = naive_attention(q, k[:, :, perm_k], v[:, :, perm_k], 0.8, False)
    o_q, lse_q = naive_attention(q[:, :, perm_q], k, v, 0.8, False)
    assert np.max(np.abs(o - o_k)) < 1e-12
    assert np.max(np.abs(o[:, :, perm_q] - o_q)) < 1e-12
    assert np.max(np.abs(lse[:, :, perm_q] - lse_q)) < 1e-12


def test_gqa_equals_repeated_kv_heads():
    q, k, v = rnd(2, 8, 13, 6), rnd(2, 2, 13, 6), rnd(2, 2, 13, 5)
    o1, l1 = naive_attention(q, k, v, 0.6, True)
    o2, l2 = naive_attention(q, np.repeat(k, 4, axis=1), np.repeat(v, 4, axis=1), 0.6, True)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)
    # heads 0..3 read kv head 0, heads 4..7 read kv head 1 (contiguous groups)
    o3, _ = naive_attention(q[:, 4:8], k[:, 1:2], v[:, 1:2], 0.6, True)
    assert np.array_equal(o1[:, 4:8], o3)


def test_rows_with_no_visible_key():
    # Sq > Sk under bottom-right causal alignment: the first Sq - Sk rows see nothing.
    q, k, v = rnd(1, 1, 10, 4), rnd(1, 1, 6, 4), rnd(1, 1, 6, 3)
    o, lse = naive_attention(q, k, v, 1.0, True)
    assert np.all(o[0, 0, :4] == 0.0) and np.all(np.isneginf(lse[0, 0, :4]))
    assert np.array_equal(o[0, 0, 4], v[0, 0, 0])
    o0, lse0 = naive_attention(q, k[:, :, :0], v[:, :, :0], 1.0, False)
    assert np.all(o0 == 0.0) and np.all(np.isneginf(lse0))


# ---------------------------------------------------------------------------------------------
# independent routes: tiled online softmax (Alg. 1 / Alg. 2) and scalar brute force
# ---------------------------------------------------------------------------------------------

@pytest.mark.parametrize("bm", [1, 3, 16])
@pytest.mark.parametrize("bn", [1, 3, 16])
@pytest.mark.parametrize("C", [1, 2, 3])
@pytest.mark.parametrize("causal", [False, True])
def test_tiled_matches_naive(bm, bn, C, causal):
    Sq, Sk = (37, 53) if not causal else (41, 41)
    q, k, v = rnd(Sq, 9, scale=2.0), rnd(Sk, 9, scale=2.0), rnd(Sk, 7)
    o1, l1 = attention_head(q, k, v, 0.55, causal)
    o2, l2 = spatial_flash_attention(q, k, v, 0.55, causal, bm, bn, C)
    assert np.max(np.abs(o1 - o2)) < 1e-12
    assert np.max(np.abs(l1 - l2)) < 1e-12


def test_tiled_matches_naive_with_empty_rows_and_parts():
    q, k, v = rnd(12, 4), rnd(7, 4), rnd(7, 3)
    o1, l1 = attention_head(q, k, v, 1.0, True)
    o2, l2 = spatial_flash_attention(q, k, v, 1.0, True, bm=5, bn=2, C=3)
    assert np.max(np.abs(o1 - o2)) < 1e-12
    assert np.array_equal(np.isneginf(l1), np.isneginf(l2))
    fin = np.isfinite(l1)
    assert np.max(np.abs(l1[fin] - l2[fin])) < 1e-12


def _planted_folds():
    """Plausible mistakes in the streaming oracle's fold of two (A, Z) pairs."""
    def no_rescale_running(a1, z1, a2, z2):  # forgets to rescale the running pair
        z = np.logaddexp(z1, z2)
        w2 = np.where(np.isfinite(z), np.exp(z2 - np.where(np.isfinite(z), z, 0.0)), 0.0)
        return a1 + w2[:, None] * a2, z

    def max_not_lse(a1, z1, a2, z2):  # keeps the larger log-sum-exp instead of their sum
        z = np.maximum(z1, z2)
        live = np.isfinite(z)
        zs = np.where(live, z, 0.0)
        return (np.where(live, np.exp(z1 - zs), 0.0)[:, None] * a1
                + np.where(live, np.exp(z2 - zs), 0.0)[:, None] * a2), z

    def swapped_weights(a1, z1, a2, z2):  # each side weighted by the other side's mass
        z = np.logaddexp(z1, z2)
        live = np.isfinite(z)
        zs = np.where(live, z, 0.0)
        return (np.where(live, np.exp(z2 - zs), 0.0)[:, None] * a1
                + np.where(live, np.exp(z1 - zs), 0.0)[:, None] * a2), z
    return [no_rescale_running, max_not_lse, swapped_weights]


@pytest.mark.parametrize("bad", _planted_folds(), ids=lambda f: f.__name__)
def test_tiled_pin_catches_planted_fold_mistakes(bad, monkeypatch):
    """The tiled-vs-naive pin is not vacuous: each planted mistake in the fold makes it fail."""
    import oracle.tiled as tiled

    q, k, v = rnd(37, 9, scale=2.0), rnd(53, 9, scale=2.0), rnd(53, 7)
    o1, l1 = attention_head(q, k, v, 0.55, False)
    monkeypatch.setattr(tiled, "_fold", bad)
    o2, l2 = tiled.spatial_flash_attention(q, k, v, 0.55, False, 16, 3, 2)
    assert max(np.max(np.abs(o1 - o2)), np.max(np.abs(l1 - l2))) > 1e-6


@pytest.mark.parametrize("Sq,Sk,causal", [(1, 1, False), (2, 3, False), (4, 4, True), (3, 2, True),
                                          (4, 2, False), (1, 4, True)])
def test_brute_force_matches_naive(Sq, Sk, causal):
    q, k, v = rnd(Sq, 3), rnd(Sk, 3), rnd(Sk, 2)
    ob, lb = brute_attention(q.tolist(), k.tolist(), v.tolist(), 0.9, causal)
    on, ln = attention_head(q, k, v, 0.9, causal)
    assert np.max(np.abs(np.array(ob) - on)) < 1e-13
    lb = np.array(lb)
    assert np.array_equal(np.isneginf(lb), np.isneginf(ln))
    assert np.max(np.abs(lb[np.isfinite(lb)] - ln[np.isfinite(ln)]), initial=0.0) < 1e-13


def test_row_subset_matches_full():
    w = W.small("rows", B=2, Hq=4, Hkv=2, Sq=40, Sk=40, dqk=8, dv=8, causal=True)
    q, k, v = (x.to(torch.float64).numpy() for x in W.make_inputs(w))
    o, lse = naive_attention(q, k, v, w.scale, True)
    rows = W.sample_rows(w, n=7)
    res = naive_attention_rows(lambda b, h, r: q[b, h, r], lambda b, g: k[b, g], lambda b, g: v[b, g],
                               w.B, w.Hq, w.Hkv, w.Sq, w.scale, True, rows)
    for idx, (orow, lrow) in enumerate(res):
        b, h = divmod(idx, w.Hq)
        assert np.max(np.abs(orow - o[b, h, rows[idx]])) < 1e-13
        assert np.max(np.abs(lrow - lse[b, h, rows[idx]])) < 1e-13


# ---------------------------------------------------------------------------------------------
# measurement formulas, pinned to the paper's printed throughput
# ---------------------------------------------------------------------------------------------

def _read(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return list(csv.DictReader(line for line in f if not line.startswith("#")))


def test_paper_flop_formula_reproduces_table6():
    rows = _read("table6_fused_xdna2.csv")
    assert len(rows) == 12
    for r in rows:
        H, dk, S = int(r["H"]), int(r["dk"]), int(r["seq_len"])
        gflops = W.paper_flops(H, S, S, dk, dk) / (float(r["latency_us"]) * 1e-6) / 1e9
        assert abs(gflops / float(r["gflops"]) - 1.0) < 1e-4, r["model"]


def test_paper_flop_formula_reproduces_table5_long_rows():
    for r in _read("table5_fused_xdna2.csv"):
        S = int(r["seq_len"])
        gflops = W.paper_flops(12, S, S, 64, 64) / (float(r["latency_ms"]) * 1e-3) / 1e9
        assert abs(gflops / float(r["gflops"]) - 1.0) < 0.03


def test_metric_flops_halves_causal_exactly():
    w = W.CONFIGS[3]
    assert W.metric_flops(w) == 0.5 * W.paper_flops(w.Hq, w.Sq, w.Sk, w.dqk, w.dv)
    w2 = W.CONFIGS[2]
    assert W.metric_flops(w2) == W.paper_flops(w2.Hq, w2.Sq, w2.Sk, w2.dqk, w2.dv, B=w2.B)
    assert W.metric_flops(w2) == 4 * 512 * 512 * 64 * 8 * 12


def test_workload_inputs_are_seeded_bf16():
    w = W.CONFIGS[1]
    a = W.make_inputs(w)
    b = W.make_inputs(w)
    assert all(x.dtype == torch.bfloat16 and x.is_contiguous() for x in a)
    assert all(torch.equal(x, y) for x, y in zip(a, b))
    assert a[0].shape == (1, 1, 256, 64)
    assert W.algorithmic_bytes(w) == 132096
