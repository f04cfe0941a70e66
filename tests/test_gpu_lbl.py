"""GPU parity of the layer-by-layer (unfused) operators and their composition against the oracle.

Each operator is fed exactly the oracle's input for it (the oracle's scores, the oracle's
probabilities), so its only differences from the oracle are its own fp32 arithmetic and where that
lands relative to one bf16 rounding. The bars below are the rigorous bounds of that arithmetic:

* scores: |S - scale*q.k| <= 2^-8 |scale*q.k| + (1 + 2^-8) (d + 2) 2^-24 scale sum_t |q_t k_t|
  (fp32 accumulation of d products and the scale multiply, then one bf16 rounding);
* softmax: P within one bf16 spacing of the oracle's bf16(exp(S - LSE)), or both below 2^-126 where
  the fp32 exponential may flush; LSE within lse_tol (fp32 exp2/log2 and the row sum, see there);
* P V: |O - P.V| <= 2^-8 |P.V| + (1 + 2^-8) (Sk + 2) 2^-24 sum_j |p_j v_j|;
* the three together against exact attention: the bound of the three bf16 roundings
  (oracle.lbl_error_bound) with the fp32 terms above added.

Every operator is also checked against its extent contract: entries it must not read hold NaN, and
entries it must not write are still NaN afterwards, as are guard zones around every buffer.
"""

import math

import numpy as np
import pytest
import torch

import paper_2609_21264_amd as fa
import workloads as W
from oracle import (lbl_pv_head, lbl_scores_head, lbl_softmax_head, layer_by_layer_attention,
                    naive_attention, naive_attention_rows)
from parity import to_f64

pytestmark = pytest.mark.gpu

U = 2.0 ** -8
GUARD = 1024


def stream():
    return torch.cuda.current_stream().cuda_stream


def extent(w, i):
    """Keys the rows of i's 128-row block use: the visible keys of the block's last row, rounded up to 64."""
    last = min(w.Sq, (i // 128 + 1) * 128) - 1
    n = w.Sk if not w.causal else max(0, min(w.Sk, last + 1 + w.Sk - w.Sq))
    return -(-n // 64) * 64


def n_visible(w, i):
    return w.Sk if not w.causal else max(0, min(w.Sk, i + 1 + w.Sk - w.Sq))


def spacing(x):
    """bf16 spacing at |x| (2^-133 at zero and below the normal range)."""
    x = np.abs(np.asarray(x, dtype=np.float64))
    _, e = np.frexp(np.where(x > 0, x, 1.0))
    return np.where(x >= 2.0 ** -126, np.ldexp(1.0, e - 8), 2.0 ** -133)


def lse_tol(sk, lse):
    """fp32 error of the softmax kernel's LSE = ln2 * (M + log2 L): the row maximum of s*log2(e) is off
    by 2^-24 |LSE| relative, each exponential by 2^-23, and L sums at most 8 * ceil(Sk / 512) terms per
    lane before 6 levels of a tree: relative error (8 ceil(Sk/512) + 8) 2^-24 on L, plus one rounding
    in log2 and one in the final product."""
    terms = 8 * (-(-sk // 512)) + 8
    return terms * 2.0 ** -24 + 2.0 ** -22 * (1 + np.abs(lse))


def guarded(n, dtype):
    buf = torch.full((n + 2 * GUARD,), float("nan"), dtype=dtype, device="cuda")
    return buf, buf[GUARD:GUARD + n]


def guards_intact(buf, n):
    return bool(torch.isnan(buf[:GUARD]).all() and torch.isnan(buf[GUARD + n:]).all())


def oracle_heads(w, q, k, v):
    """Per (b, h): oracle S~, G, LSE, O and the float64 inputs of the head."""
    q64, k64, v64 = to_f64(q), to_f64(k), to_f64(v)
    out = {}
    for b in range(w.B):
        for h in range(w.Hq):
            g = h // w.group
            s = lbl_scores_head(q64[b, h], k64[b, g], w.scale)
            gp, lse = lbl_softmax_head(s, w.causal)
            out[b, h] = dict(q=q64[b, h], k=k64[b, g], v=v64[b, g], s=s, g=gp, lse=lse, o=lbl_pv_head(gp, v64[b, g]))
    return out


CASES = [
    W.small("d64 130x200", Sq=130, Sk=200, seed=71),
    W.small("d64 causal 300 gqa", Hq=4, Hkv=2, Sq=300, Sk=300, causal=True, seed=72),
    W.small("d128 causal Sq<Sk", dqk=128, dv=128, Hq=2, Hkv=1, Sq=100, Sk=333, causal=True, seed=73),
    W.small("d128 causal Sq>Sk", dqk=128, dv=128, Sq=260, Sk=70, causal=True, seed=74),
    W.small("d192/128 257x129", dqk=192, dv=128, Hq=2, Hkv=2, Sq=257, Sk=129, seed=75),
    W.small("d192/128 causal", dqk=192, dv=128, Sq=200, Sk=200, causal=True, seed=76),
    W.small("d64 decode 1x700", Hq=3, Hkv=1, Sq=1, Sk=700, seed=77),
    W.small("d128 sigma 2", dqk=128, dv=128, Sq=128, Sk=256, causal=True, sigma=2.0, seed=78),
]
IDS = [c.name for c in CASES]


@pytest.mark.parametrize("w", CASES, ids=IDS)
def test_scores_operator(w):
    q, k, v = W.make_inputs(w)
    ref = oracle_heads(w, q, k, v)
    ld = fa.fa_lbl_ld(w.Sk)
    n = w.B * w.Hq * w.Sq * ld
    buf, S = guarded(n, torch.bfloat16)
    # device copies held in variables: a temporary's memory could be handed to the next copy before the
    # kernel runs
    qd, kd = q.cuda(), k.cuda()
    st = fa.fa_lbl_scores(qd.data_ptr(), kd.data_ptr(), S.data_ptr(), w.B, w.Hq, w.Hkv, w.Sq, w.Sk,
                          w.dqk, w.scale, w.causal, stream())
    assert st == fa.FA_OK
    torch.cuda.synchronize()
    assert guards_intact(buf, n)
    got = S.view(w.B, w.Hq, w.Sq, ld).cpu().double().numpy()
    ext = np.array([extent(w, i) for i in range(w.Sq)])
    cols = np.arange(ld)[None, :]
    n_eq = n_cmp = 0
    for (b, h), r in ref.items():
        g = got[b, h]
        inside = cols < ext[:, None]
        assert np.isnan(g[~inside]).all(), "written past the extent"
        assert not np.isnan(g[inside]).any(), "entry inside the extent not written"
        keys = cols < w.Sk
        assert np.all(g[inside & ~keys] == 0), "keys past Sk must score 0"
        sel = inside[:, :w.Sk]
        exact = w.scale * (r["q"] @ r["k"].T)
        absdot = abs(w.scale) * (np.abs(r["q"]) @ np.abs(r["k"]).T)
        bound = U * np.abs(exact) + (1 + U) * (w.dqk + 2) * 2.0 ** -24 * absdot
        gk = g[:, :w.Sk]
        assert np.all(np.abs(gk - exact)[sel] <= bound[sel])
        n_eq += int(np.sum((gk == r["s"])[sel]))
        n_cmp += int(sel.sum())
    assert n_eq >= 0.99 * n_cmp, f"only {n_eq}/{n_cmp} scores equal the correctly rounded ones"


def _softmax_input(w, ref, ld):
    """[B, Hq, Sq, ld] bf16: the oracle's scores on visible keys, NaN elsewhere (never to be used)."""
    s = np.full((w.B, w.Hq, w.Sq, ld), np.nan)
    for (b, h), r in ref.items():
        for i in range(w.Sq):
            nv = n_visible(w, i)
            s[b, h, i, :nv] = r["s"][i, :nv]
    return torch.from_numpy(s).to(torch.bfloat16)


@pytest.mark.parametrize("in_place", [False, True], ids=["separate", "in-place"])
@pytest.mark.parametrize("w", CASES, ids=IDS)
def test_softmax_operator(w, in_place):
    q, k, v = W.make_inputs(w)
    ref = oracle_heads(w, q, k, v)
    ld = fa.fa_lbl_ld(w.Sk)
    n = w.B * w.Hq * w.Sq * ld
    s_in = _softmax_input(w, ref, ld).reshape(-1).cuda()
    sbuf, S = guarded(n, torch.bfloat16)
    S.copy_(s_in)
    if in_place:
        pbuf, P = sbuf, S
    else:
        pbuf, P = guarded(n, torch.bfloat16)
    lbuf, L = guarded(w.B * w.Hq * w.Sq, torch.float32)
    st = fa.fa_lbl_softmax(S.data_ptr(), P.data_ptr(), L.data_ptr(), w.B, w.Hq, w.Sq, w.Sk, w.causal, stream())
    assert st == fa.FA_OK
    torch.cuda.synchronize()
    assert guards_intact(pbuf, n) and guards_intact(lbuf, w.B * w.Hq * w.Sq)
    if not in_place:
        assert torch.equal(S.view(torch.int16), s_in.view(torch.int16)), "the input was modified"
    got = P.view(w.B, w.Hq, w.Sq, ld).cpu().double().numpy()
    lse = L.view(w.B, w.Hq, w.Sq).cpu().double().numpy()
    cols = np.arange(ld)[None, :]
    ext = np.array([extent(w, i) for i in range(w.Sq)])
    vis = np.array([n_visible(w, i) for i in range(w.Sq)])
    for (b, h), r in ref.items():
        g = got[b, h]
        inside = cols < ext[:, None]
        visible = cols < vis[:, None]
        if not in_place:
            assert np.isnan(g[~inside]).all(), "written past the extent"
        assert np.all(g[inside & ~visible] == 0), "masked entries inside the extent must be 0"
        gr = np.zeros_like(g)
        gr[:, :w.Sk] = r["g"]
        d = np.abs(g - gr)[visible]
        small = (np.abs(g) < 2.0 ** -126) & (np.abs(gr) < 2.0 ** -126)
        assert np.all((d <= spacing(gr)[visible]) | small[visible])
        fin = np.isfinite(r["lse"])
        assert np.array_equal(np.isfinite(lse[b, h]), fin)
        assert np.all(lse[b, h][~fin] == -np.inf)
        assert np.all(np.abs(lse[b, h][fin] - r["lse"][fin]) <= lse_tol(w.Sk, r["lse"][fin]))


@pytest.mark.parametrize("w", CASES, ids=IDS)
def test_pv_operator(w):
    q, k, v = W.make_inputs(w)
    ref = oracle_heads(w, q, k, v)
    ld = fa.fa_lbl_ld(w.Sk)
    n = w.B * w.Hq * w.Sq * ld
    # The oracle's probabilities inside each row's extent (0 past Sk), NaN past it: never read.
    p = np.full((w.B, w.Hq, w.Sq, ld), np.nan)
    for (b, h), r in ref.items():
        for i in range(w.Sq):
            e = extent(w, i)
            p[b, h, i, :e] = 0.0
            p[b, h, i, :min(e, w.Sk)] = r["g"][i, :min(e, w.Sk)]
    P = torch.from_numpy(p).to(torch.bfloat16).reshape(-1).cuda()
    n_o = w.B * w.Hq * w.Sq * w.dv
    obuf, O = guarded(n_o, torch.bfloat16)
    vd = v.cuda()
    st = fa.fa_lbl_pv(P.data_ptr(), vd.data_ptr(), O.data_ptr(), w.B, w.Hq, w.Hkv, w.Sq, w.Sk, w.dv,
                      w.causal, stream())
    assert st == fa.FA_OK
    torch.cuda.synchronize()
    assert guards_intact(obuf, n_o)
    got = O.view(w.B, w.Hq, w.Sq, w.dv).cpu().double().numpy()
    n_eq = n_cmp = 0
    for (b, h), r in ref.items():
        exact = r["g"] @ r["v"]
        absd = np.abs(r["g"]) @ np.abs(r["v"])
        bound = U * np.abs(exact) + (1 + U) * (w.Sk + 2) * 2.0 ** -24 * absd
        assert np.all(np.abs(got[b, h] - exact) <= bound)
        n_eq += int(np.sum(got[b, h] == r["o"]))
        n_cmp += got[b, h].size
    assert n_eq >= 0.99 * n_cmp, f"only {n_eq}/{n_cmp} outputs equal the correctly rounded ones"


def composed_bound(w, qh, kh, vh, causal_rows=None):
    """Per-row bounds of |O_gpu - O_exact| and |LSE_gpu - LSE_exact| for one head (rows at positions
    causal_rows, default 0..n-1).

    As in oracle.lbl_error_bound, with the kernels' fp32 errors folded in: each spilled score is off by
    at most D = u M + (d + 2) 2^-24 max_j scale sum_t |q_t k_t| (bf16 rounding plus fp32 accumulation),
    the softmax adds E = lse_tol to each log-probability, so each probability moves by a factor within
    exp(+-(2 D + 2 E)); rounding P and O gives (1 + u)^2, and the P V accumulation adds
    (Sk + 2) 2^-24 max|V| (probabilities sum to 1 + O(u)). The LSE is off by at most D + E."""
    exact = w.scale * (qh @ kh.T)
    absdot = abs(w.scale) * (np.abs(qh) @ np.abs(kh).T)
    n = qh.shape[0]
    if w.Sk == 0:
        return np.zeros(n), np.zeros(n)
    pos = np.arange(n) if causal_rows is None else np.asarray(causal_rows)
    vis = np.ones_like(exact, dtype=bool)
    if w.causal:
        vis = np.arange(w.Sk)[None, :] <= pos[:, None] + (w.Sk - w.Sq)
    m = np.where(vis, np.abs(exact), 0).max(axis=1)
    d = U * m + (w.dqk + 2) * 2.0 ** -24 * np.where(vis, absdot, 0).max(axis=1)
    e = lse_tol(w.Sk, m + math.log(w.Sk))
    vmax = np.abs(vh).max()
    o_bound = vmax * ((1 + U) ** 2 * np.exp(2 * d + 2 * e) - 1) + vmax * (1 + 2 * U) * (w.Sk + 2) * 2.0 ** -24
    return o_bound, d + e


COMPOSED = CASES + [
    W.small("d64 empty rows", Sq=90, Sk=20, causal=True, seed=79),
    W.small("d128 Sk 0", dqk=128, dv=128, Sq=50, Sk=0, seed=80),
    W.small("d64 B2 gqa causal", B=2, Hq=6, Hkv=2, Sq=140, Sk=333, causal=True, seed=81),
]


@pytest.mark.parametrize("w", COMPOSED, ids=[c.name for c in COMPOSED])
def test_unfused_matches_oracles(w):
    q, k, v = W.make_inputs(w)
    o, lse = fa.forward_unfused(q.cuda(), k.cuda(), v.cuda(), causal=w.causal, scale=w.scale, return_lse=True)
    torch.cuda.synchronize()
    o = to_f64(o.cpu())
    lse = lse.cpu().double().numpy()
    q64, k64, v64 = to_f64(q), to_f64(k), to_f64(v)
    o_ex, lse_ex = naive_attention(q64, k64, v64, w.scale, w.causal)
    o_lbl, lse_lbl = layer_by_layer_attention(q64, k64, v64, w.scale, w.causal)
    assert np.array_equal(np.isfinite(lse), np.isfinite(lse_ex))
    fin = np.isfinite(lse_ex)
    assert np.all(lse[~fin] == -np.inf) and np.all(o[~fin] == 0)
    for b in range(w.B):
        for h in range(w.Hq):
            g = h // w.group
            bnd, lbnd = composed_bound(w, q64[b, h], k64[b, g], v64[b, g])
            err = np.abs(o[b, h] - o_ex[b, h]).max(axis=1)
            assert np.all(err <= bnd), f"head {b},{h}: worst ratio {np.max(err / np.maximum(bnd, 1e-300)):.3f}"
            f = fin[b, h]
            assert np.all(np.abs(lse[b, h][f] - lse_ex[b, h][f]) <= lbnd[f])
    # The kernels round where the layer-by-layer oracle rounds: most outputs are bit-identical to it
    # (they differ only where an fp32 result sits next to a bf16 rounding boundary).
    if o.size:
        same = np.mean(o == o_lbl)
        assert same >= 0.95, f"only {same:.3f} of the outputs equal the layer-by-layer oracle's"
        assert np.all(np.abs(lse[fin] - lse_lbl[fin]) <= 1e-4)


def test_chunked_workspace_is_bitwise_identical():
    # Whole problem in one chunk vs. chunks of whole heads (2.5 heads of room: 2 heads, a multiple of the
    # group) vs. parts of one head (1.5 blocks of 128 rows of room: one block per chunk).
    w = W.small("chunks", dqk=128, dv=128, Hq=4, Hkv=2, Sq=300, Sk=400, causal=True, seed=82)
    q, k, v = (x.cuda() for x in W.make_inputs(w))
    ld = fa.fa_lbl_ld(w.Sk)
    full = fa.fa_lbl_workspace_bytes(w.B, w.Hq, w.Sq, w.Sk)
    assert full == w.B * w.Hq * w.Sq * ld * 2
    outs = []
    for nbytes in (full, int(2.5 * w.Sq * ld * 2), int(1.5 * 128 * ld * 2), 128 * ld * 2):
        ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        outs.append(fa.forward_unfused(q, k, v, causal=True, scale=w.scale, return_lse=True, workspace=ws))
    torch.cuda.synchronize()
    for o, l in outs[1:]:
        assert torch.equal(o.view(torch.int16), outs[0][0].view(torch.int16))
        assert torch.equal(l, outs[0][1])
    with pytest.raises(ValueError, match="FA_ERR_WORKSPACE"):
        fa.forward_unfused(q, k, v, causal=True, workspace=torch.empty(128 * ld * 2 - 2, dtype=torch.uint8,
                                                                       device="cuda"))


def test_unfused_guards_and_workspace_bounds():
    w = W.small("guards", dqk=64, dv=64, Hq=2, Hkv=1, Sq=150, Sk=190, causal=True, seed=83)
    q, k, v = (x.cuda() for x in W.make_inputs(w))
    n_o, n_l = w.Hq * w.Sq * w.dv, w.Hq * w.Sq
    nbytes = fa.fa_lbl_workspace_bytes(w.B, w.Hq, w.Sq, w.Sk)
    obuf, O = guarded(n_o, torch.bfloat16)
    lbuf, L = guarded(n_l, torch.float32)
    wbuf, WS = guarded(nbytes // 2, torch.bfloat16)
    st = fa.fa_fwd_unfused(q.data_ptr(), k.data_ptr(), v.data_ptr(), O.data_ptr(), L.data_ptr(), w.B, w.Hq, w.Hkv,
                           w.Sq, w.Sk, w.dqk, w.dv, w.scale, True, WS.data_ptr(), nbytes, stream())
    assert st == fa.FA_OK
    torch.cuda.synchronize()
    assert guards_intact(obuf, n_o) and guards_intact(lbuf, n_l) and guards_intact(wbuf, nbytes // 2)
    assert not torch.isnan(O).any() and not torch.isnan(L).any()


FULL = [W.CONFIGS[2], W.CONFIGS[3], W.CONFIGS[4]]


@pytest.mark.parametrize("w", FULL, ids=[c.name for c in FULL])
def test_unfused_full_size_sampled_rows(w):
    """The benchmark shapes in one chunk, checked on sampled rows of every head against exact attention
    within the composed bound."""
    q, k, v = W.make_inputs(w)
    o, lse = fa.forward_unfused(q.cuda(), k.cuda(), v.cuda(), causal=w.causal, scale=w.scale, return_lse=True)
    torch.cuda.synchronize()
    o, lse = o.cpu(), lse.cpu()
    rng = np.random.default_rng(w.seed)
    rows = [np.unique(np.concatenate([[0, w.Sq - 1], rng.integers(0, w.Sq, 6)])) for _ in range(w.B * w.Hq)]
    res = naive_attention_rows(lambda b, h, r: to_f64(q[b, h, r]), lambda b, g: to_f64(k[b, g]),
                               lambda b, g: to_f64(v[b, g]), w.B, w.Hq, w.Hkv, w.Sq, w.scale, w.causal, rows)
    for idx, (o_ref, lse_ref) in enumerate(res):
        b, h = divmod(idx, w.Hq)
        g = h // w.group
        r = rows[idx]
        bnd, lbnd = composed_bound(w, to_f64(q[b, h, r]), to_f64(k[b, g]), to_f64(v[b, g]), causal_rows=r)
        err = np.abs(to_f64(o[b, h, r]) - o_ref).max(axis=1)
        assert np.all(err <= bnd), f"{w.name} head {b},{h}: worst ratio {np.max(err / bnd):.3f}"
        assert np.all(np.abs(lse[b, h, r].double().numpy() - lse_ref) <= lbnd)
