"""GPU parity of both instances of the fused kernel.

Problems with at most 1024 (d = 64) or 256 (d = 128) query blocks of fa_block_rows() rows
(B * Hq * ceil(Sq / rows)) at (d_qk, d_v) = (64, 64) or (128, 128) run the short instance (half as
many rows per workgroup, two workgroups per CU); every other problem runs the long instance. The
small edge cases of test_gpu_parity.py have few blocks and so exercise the short instance; here the
same cases are widened past the switch (more heads, same per-head shape and GQA ratio, seeded afresh)
so that the long instance meets them too, and every output element is compared with the fp64 oracle.
"""

import numpy as np
import pytest
import torch

import paper_2609_21264_amd as fa
import workloads as W
from oracle import naive_attention
from parity import check_full, compare, run_gpu, to_f64
from test_gpu_parity import SMALL_CASES

pytestmark = pytest.mark.gpu

SHORT_MAX = {64: 1024, 128: 256}  # largest block count that runs the short instance, by head dim


def blocks(w):
    bm = fa.fa_block_rows(w.dqk, w.dv, w.causal)
    return w.B * w.Hq * -(-w.Sq // bm)


def short(w):
    return w.dqk == w.dv and w.dqk in SHORT_MAX and blocks(w) <= SHORT_MAX[w.dqk]


def widened(w):
    """The same per-head problem with enough heads for the long instance."""
    m = -(-(SHORT_MAX[w.dqk] + 1) // blocks(w))
    v = w.with_(name=w.name + f" x{m} heads", Hq=w.Hq * m, Hkv=w.Hkv * m, seed=w.seed + 500)
    assert not short(v)
    return v


CASES = [w for w in SMALL_CASES if (w.dqk, w.dv) != (192, 128)]


def test_small_cases_run_the_short_instance():
    # the premise of this file: the edge cases of test_gpu_parity.py have few blocks
    assert CASES and all(short(w) for w in CASES)


@pytest.mark.parametrize("w", CASES, ids=[c.name for c in CASES])
def test_long_instance_small_shapes_match_oracle(w):
    v = widened(w)
    print(f"\n[case] {v}", flush=True)
    check_full(v)


@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
@pytest.mark.parametrize("heads", [2, 2 * 43], ids=["short", "long"])
def test_rising_maxima_rebase_both_instances(causal, heads):
    """Keys whose scores jump far above everything before them in the second key tile, two middle
    tiles and the last one, so that tiles are redone from their exact maximum at each position."""
    w = W.small("spikes", dqk=128, dv=128, Hq=heads, Hkv=heads // 2, Sq=640, Sk=640, causal=causal, seed=181)
    assert short(w) == (heads == 2)
    q, k, v = W.make_inputs(w)
    for key, factor in ((70, 4.0), (300, 8.0), (520, 16.0), (600, 32.0)):
        k[:, :, key] *= factor
    print(f"\n[case] {w}", flush=True)
    o, lse = run_gpu(q, k, v, w)
    o_ref, lse_ref = naive_attention(to_f64(q), to_f64(k), to_f64(v), w.scale, causal)
    assert np.nanmax(lse_ref) > 20.0
    compare(to_f64(o), lse.cpu().double().numpy(), o_ref, lse_ref, w.name)


@pytest.mark.parametrize("mult", [1, 0], ids=["short", "long"])
@pytest.mark.parametrize("d", [64, 128])
def test_causal_first_row_bitwise_both_instances(mult, d):
    heads = 4 if mult else 2 * (SHORT_MAX[d] // 4 + 1)  # 300 rows: 2 blocks per head
    w = W.small("row0", dqk=d, dv=d, Hq=heads, Hkv=heads // 2, Sq=300, Sk=300, causal=True, seed=151)
    assert short(w) == bool(mult)
    q, k, v = W.make_inputs(w)
    o, _ = run_gpu(q, k, v, w)
    o = o.cpu()
    for h in range(heads):
        assert torch.equal(o[0, h, 0], v[0, h // 2, 0]), h


@pytest.mark.parametrize("cfg", [1, 2])
def test_short_instance_runs_the_small_benchmark_configs(cfg):
    # configs 1 (one block) and 2 (192 blocks) run the short instance; test_gpu_parity checks them
    # in full, and here on a second seed
    w = W.CONFIGS[cfg]
    assert short(w)
    check_full(w.with_(seed=w.seed + 700))


@pytest.mark.parametrize("d,heads", [(128, 256), (128, 257), (64, 1024), (64, 1025)],
                         ids=["d128-256-short", "d128-257-long", "d64-1024-short", "d64-1025-long"])
def test_instance_boundary(d, heads):
    """Either side of the switch between the instances at each head dimension."""
    w = W.small(f"boundary d{d} {heads}", dqk=d, dv=d, Hq=heads, Hkv=heads, Sq=100, Sk=150, causal=True, seed=191)
    assert blocks(w) == heads and short(w) == (heads == SHORT_MAX[d])
    print(f"\n[case] {w}", flush=True)
    check_full(w)
