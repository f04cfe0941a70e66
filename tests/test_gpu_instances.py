"""GPU parity of the three instances of the fused kernel.

Which instance runs follows from the grid alone, and the library reports it (fa_fwd_rows, the query
rows of one head per workgroup): the key-halves instance (64) for the smallest grids, the short
instance (128) for mid-sized ones, and the long instance (256) for the rest and for every
d_qk = 192 problem. The small edge cases of test_gpu_parity.py have
few blocks, so they run the instance of the smallest grids; here the same cases are widened (more
heads, same per-head shape and GQA ratio, seeded afresh) until each other instance runs them, and
every output element is compared with the fp64 oracle.
"""

import numpy as np
import pytest
import torch

import paper_2609_21264_amd as fa
import workloads as W
from oracle import naive_attention
from parity import check_full, compare, rounding_bar, run_gpu, to_f64
from test_gpu_parity import SMALL_CASES

pytestmark = pytest.mark.gpu

HALF, SHORT, LONG = 64, 128, 256  # rows per workgroup of one head, by instance
NAMES = {HALF: "halves", SHORT: "short", LONG: "long"}


def rows(w):
    return fa.fa_fwd_rows(w.B, w.Hq, w.Sq, w.dqk, w.dv, w.causal)


def blocks(w):
    return w.B * w.Hq * -(-w.Sq // fa.fa_block_rows(w.dqk, w.dv, w.causal))


def widened(w, target):
    """The same per-head problem with the fewest multiples of its heads that run the instance of
    `target` rows, or None if no head count does (the instances follow each other as the grid grows:
    key halves, short, long)."""
    for m in range(1, 8192):
        v = w.with_(Hq=w.Hq * m, Hkv=w.Hkv * m)
        r = rows(v)
        if r == target:
            return v.with_(name=w.name + f" x{m} heads", seed=w.seed + 500 + target)
        if r > target:
            return None
    return None


CASES = [w for w in SMALL_CASES if (w.dqk, w.dv) != (192, 128)]
WIDE = [(w, t) for w in CASES for t in (SHORT, LONG)]


def test_small_cases_run_the_key_halves_instance():
    # the premise of this file: the edge cases of test_gpu_parity.py have few blocks
    assert CASES and all(rows(w) == HALF for w in CASES)
    assert all(rows(w) == LONG for w in SMALL_CASES if w.dqk == 192)


@pytest.mark.parametrize("w,target", WIDE, ids=[f"{w.name}-{NAMES[t]}" for w, t in WIDE])
def test_wider_instances_small_shapes_match_oracle(w, target):
    v = widened(w, target)
    print(f"\n[case] {v}", flush=True)
    check_full(v)


def _heads_for(make, target):
    """The smallest even head count whose problem `make(heads)` runs the instance of `target` rows."""
    for heads in range(2, 8192, 2):
        r = rows(make(heads))
        if r == target:
            return heads
        if r > target:
            return None
    return None


SPIKES = [(c, t) for c in (False, True) for t in (HALF, SHORT, LONG)]


@pytest.mark.parametrize("causal,target", SPIKES,
                         ids=[f"{'causal' if c else 'full'}-{NAMES[t]}" for c, t in SPIKES])
def test_rising_maxima_rebase_every_instance(causal, target):
    """Keys whose scores jump far above everything before them in the second key tile, two middle
    tiles and the last one, so that tiles are redone from their exact maximum at each position."""
    make = lambda heads: W.small("spikes", dqk=128, dv=128, Hq=heads, Hkv=heads // 2, Sq=640, Sk=640,
                                 causal=causal, seed=181)
    heads = _heads_for(make, target)
    w = make(heads)
    q, k, v = W.make_inputs(w)
    for key, factor in ((70, 4.0), (300, 8.0), (520, 16.0), (600, 32.0)):
        k[:, :, key] *= factor
    print(f"\n[case] {w}", flush=True)
    o, lse = run_gpu(q, k, v, w)
    o_ref, lse_ref = naive_attention(to_f64(q), to_f64(k), to_f64(v), w.scale, causal)
    assert np.nanmax(lse_ref) > 20.0
    compare(to_f64(o), lse.cpu().double().numpy(), o_ref, lse_ref, w.name)


ROW0 = [(d, t) for d in (64, 128) for t in (HALF, SHORT, LONG)]


@pytest.mark.parametrize("d,target", ROW0, ids=[f"d{d}-{NAMES[t]}" for d, t in ROW0])
def test_causal_first_row_bitwise_every_instance(d, target):
    # 300 rows: 2 blocks per head; row 0 sees key 0 only, so its output is V's row 0 bit for bit
    make = lambda heads: W.small("row0", dqk=d, dv=d, Hq=heads, Hkv=heads // 2, Sq=300, Sk=300, causal=True,
                                 seed=151)
    heads = _heads_for(make, target)
    w = make(heads)
    q, k, v = W.make_inputs(w)
    o, _ = run_gpu(q, k, v, w)
    o = o.cpu()
    for h in range(heads):
        assert torch.equal(o[0, h, 0], v[0, h // 2, 0]), h


@pytest.mark.parametrize("cfg", [1, 2])
def test_small_benchmark_configs_second_seed(cfg):
    # configs 1 (one block: key halves) and 2 (384 blocks: short); test_gpu_parity checks them in
    # full, and here on a second seed
    w = W.CONFIGS[cfg]
    assert rows(w) == (HALF if cfg == 1 else SHORT)
    check_full(w.with_(seed=w.seed + 700))


# (d, causal, B * Hq * ceil(Sq / 256)) of the last grid before each switch between the instances
SWITCHES = [(64, True, 320), (64, True, 1024), (64, False, 64), (64, False, 1024), (128, True, 192), (128, True, 256),
            (128, False, 128), (128, False, 256)]
BOUNDARY = [(d, c, n + side) for d, c, n in SWITCHES for side in (0, 1)]


@pytest.mark.parametrize("d,causal,heads", BOUNDARY,
                         ids=[f"d{d}-{'causal' if c else 'full'}-{h}" for d, c, h in BOUNDARY])
def test_instance_boundary(d, causal, heads):
    """Either side of each switch between the instances; one block per head (Sq = 100)."""
    make = lambda n: W.small(f"boundary d{d} {n}", dqk=d, dv=d, Hq=n, Hkv=n, Sq=100, Sk=150, causal=causal,
                             seed=191)
    w = make(heads)
    assert blocks(w) == heads
    last = heads if (d, causal, heads) in SWITCHES else heads - 1
    assert rows(make(last + 1)) > rows(make(last))
    print(f"\n[case] {w} ({NAMES[rows(w)]})", flush=True)
    check_full(w)


# At d = 64 the short instance takes 128-key tiles once Sk >= 1024 (the rows per workgroup stay 128):
# cases in the short instance's range with such keys, every output element against the oracle.
def _wide(name, Hq, Hkv, Sq, Sk, causal, seed, **kw):
    return W.small(f"wide tiles {name}", dqk=64, dv=64, Hq=Hq, Hkv=Hkv, Sq=Sq, Sk=Sk, causal=causal, seed=seed, **kw)


WIDE_TILES = [
    _wide("ragged keys", 80, 80, 100, 1100, False, 301),
    _wide("gqa4 whole tiles", 48, 12, 70, 1024, False, 302, B=2),
    _wide("causal gqa4", 56, 14, 1300, 1300, True, 303),
    _wide("causal Sq>Sk gqa2", 60, 30, 1500, 1100, True, 304),
    _wide("causal Sq<Sk", 330, 330, 40, 2100, True, 305),
    _wide("scale 0", 70, 70, 90, 1200, False, 306, scale=0.0),
    _wide("negative scale gqa7", 70, 10, 90, 1500, False, 307, scale=-0.09),
    _wide("sigma 2 causal gqa3", 330, 110, 128, 1280, True, 308, sigma=2.0),
]


@pytest.mark.parametrize("w", WIDE_TILES, ids=[w.name for w in WIDE_TILES])
def test_short_instance_wide_tiles_match_oracle(w):
    assert rows(w) == SHORT and w.Sk >= 1024
    print(f"\n[case] {w}", flush=True)
    q, k, v = W.make_inputs(w)
    o, lse = run_gpu(q, k, v, w)
    vf = to_f64(v)
    o_ref, lse_ref = naive_attention(to_f64(q), to_f64(k), vf, w.scale, w.causal)
    # sigma = 2: the bar derived from the bf16 rounding of P and O, as in the random sweep
    compare(to_f64(o), lse.cpu().double().numpy(), o_ref, lse_ref, w.name, max(1.0, w.sigma),
            o_bar=rounding_bar(vf, w.Hq) if w.sigma > 1.0 else None)


@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
def test_short_instance_wide_tiles_rebase(causal):
    """Rising maxima (keys scaled x4 .. x32 in four tiles of 128 keys) through the 128-key tiles."""
    w = _wide("spikes", 330 if causal else 80, 110 if causal else 40, 64, 1500, causal, 309)
    assert rows(w) == SHORT
    q, k, v = W.make_inputs(w)
    for key, factor in ((70, 4.0), (300, 8.0), (900, 16.0), (1490, 32.0)):
        k[:, :, key] *= factor
    print(f"\n[case] {w}", flush=True)
    o, lse = run_gpu(q, k, v, w)
    o_ref, lse_ref = naive_attention(to_f64(q), to_f64(k), to_f64(v), w.scale, causal)
    assert np.nanmax(lse_ref) > 20.0
    compare(to_f64(o), lse.cpu().double().numpy(), o_ref, lse_ref, w.name)
