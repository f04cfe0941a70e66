"""GPU parity of the decode-shaped path (fa_fwd_decode): the query heads of a key/value group and their
few rows packed into 32-column blocks, key ranges split over workgroups and merged by log-sum-exp
(Alg. 2). Compared with the fp64 oracle element by element at the bar of the prefill kernel."""

import pytest
import torch

import paper_2609_21264_amd as fa
import workloads as W
from oracle import naive_attention, naive_attention_rows
from parity import compare, to_f64

pytestmark = pytest.mark.gpu


def run(w, n_parts, inputs=None):
    q, k, v = inputs if inputs is not None else W.make_inputs(w)
    o, lse = fa.forward(q.cuda(), k.cuda(), v.cuda(), causal=w.causal, scale=w.scale, return_lse=True, decode=True,
                        n_split=n_parts)
    torch.cuda.synchronize()
    return q, k, v, o, lse


CASES = [
    # (workload, parts); columns per block = (Hq / Hkv) * Sq
    (W.small("gqa4 Sq1 4000", dqk=128, dv=128, Hq=32, Hkv=8, Sq=1, Sk=4000, seed=61), 6),
    (W.small("gqa4 Sq4 causal 3000", dqk=128, dv=128, B=2, Hq=8, Hkv=2, Sq=4, Sk=3000, causal=True, seed=62), 5),
    (W.small("gqa8 Sq4 causal 1000 d64 (32 columns)", Hq=8, Hkv=1, Sq=4, Sk=1000, causal=True, seed=63), 3),
    (W.small("mha Sq16 777 d64", Hq=4, Hkv=4, Sq=16, Sk=777, seed=64), 2),
    (W.small("gqa2 Sq16 causal d192/128", dqk=192, dv=128, Hq=2, Hkv=1, Sq=16, Sk=2100, causal=True, seed=65), 4),
    (W.small("gqa4 Sq16 causal (2 blocks)", dqk=128, dv=128, Hq=8, Hkv=2, Sq=16, Sk=1500, causal=True, seed=66), 3),
    (W.small("gqa4 Sq20 (3 blocks, ragged)", Hq=4, Hkv=1, Sq=20, Sk=900, seed=67), 2),
    (W.small("short keys 50", dqk=128, dv=128, Hq=4, Hkv=1, Sq=2, Sk=50, seed=68), 1),
    (W.small("Sq > Sk causal (empty rows)", Hq=2, Hkv=1, Sq=8, Sk=5, causal=True, seed=69), 1),
    (W.small("more parts than tiles", dqk=128, dv=128, Hq=4, Hkv=2, Sq=1, Sk=300, seed=70), 16),
    (W.small("sigma 2", dqk=128, dv=128, Hq=8, Hkv=2, Sq=2, Sk=2000, sigma=2.0, seed=71), 4),
    (W.small("sharp softmax scale 1", Hq=4, Hkv=1, Sq=3, Sk=1200, scale=1.0, seed=72), 3),
]


@pytest.mark.parametrize("w,n_parts", CASES, ids=[c[0].name for c in CASES])
def test_decode_matches_oracle(w, n_parts):
    q, k, v, o, lse = run(w, n_parts)
    o_ref, lse_ref = naive_attention(to_f64(q), to_f64(k), to_f64(v), w.scale, w.causal)
    compare(to_f64(o), lse.cpu().double().numpy(), o_ref, lse_ref, f"{w.name} parts {n_parts}", max(1.0, w.sigma))


def test_decode_no_keys():
    w = W.small("Sk 0", dqk=128, dv=128, Hq=4, Hkv=1, Sq=1, Sk=0, seed=73)
    q, k, v = W.make_inputs(w)
    o, lse = fa.forward(q.cuda(), k.cuda(), v.cuda(), scale=w.scale, return_lse=True, decode=True, n_split=2)
    torch.cuda.synchronize()
    assert torch.all(o == 0) and torch.all(lse == float("-inf"))


@pytest.mark.parametrize("name", ["decode-128k", "decode16-128k-causal", "decode-b8-8k"])
def test_decode_full_size(name):
    """The named decode workloads at full size with the suggested part count; every query row (at most
    512) is checked against the oracle."""
    w = W.EXTRA[name]
    q, k, v, o, lse = run(w, "auto")
    rows = [torch.arange(w.Sq).numpy() for _ in range(w.B * w.Hq)]
    res = naive_attention_rows(lambda b, h, r: to_f64(q[b, h][r]), lambda b, g: to_f64(k[b, g]),
                               lambda b, g: to_f64(v[b, g]), w.B, w.Hq, w.Hkv, w.Sq, w.scale, w.causal, rows)
    import numpy as np
    o_ref = np.stack([r[0] for r in res]).reshape(w.B, w.Hq, w.Sq, w.dv)
    lse_ref = np.stack([r[1] for r in res]).reshape(w.B, w.Hq, w.Sq)
    compare(to_f64(o), lse.cpu().double().numpy(), o_ref, lse_ref, name)


def test_decode_one_part_per_tile_matches_any_split():
    # The result does not depend on how the key range is cut, beyond rounding.
    w = W.small("parts", dqk=128, dv=128, Hq=8, Hkv=2, Sq=2, Sk=1024, causal=True, seed=74)
    inputs = W.make_inputs(w)
    outs = [run(w, n, inputs)[3:] for n in (1, 2, 8)]
    for o, l in outs[1:]:
        assert (o.float() - outs[0][0].float()).abs().max().item() <= 2 ** -7
        assert (l - outs[0][1]).abs().max().item() <= 1e-5


def test_decode_is_bitwise_deterministic():
    w = W.small("det", dqk=128, dv=128, Hq=8, Hkv=2, Sq=3, Sk=3000, causal=True, seed=75)
    inputs = W.make_inputs(w)
    a, b_ = run(w, 5, inputs)[3:], run(w, 5, inputs)[3:]
    assert torch.equal(a[0], b_[0]) and torch.equal(a[1], b_[1])


def test_decode_writes_only_its_buffers():
    w = W.small("guards", dqk=64, dv=64, Hq=6, Hkv=2, Sq=5, Sk=700, causal=True, seed=76)
    q, k, v = (x.cuda() for x in W.make_inputs(w))
    n_parts = 3
    nbytes = fa.fa_fwd_split_workspace_bytes(w.B, w.Hq, w.Sq, w.dv, n_parts)
    guard = 4096
    n_o, n_l = w.Hq * w.Sq * w.dv, w.Hq * w.Sq
    o_buf = torch.full((n_o + 2 * guard,), float("nan"), dtype=torch.bfloat16, device="cuda")
    l_buf = torch.full((n_l + 2 * guard,), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.full((nbytes // 4 + 2 * guard,), float("nan"), dtype=torch.float32, device="cuda")
    o, lse, wsv = o_buf[guard:guard + n_o], l_buf[guard:guard + n_l], ws[guard:guard + nbytes // 4]
    st = fa.fa_fwd_decode(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), w.B, w.Hq, w.Hkv,
                          w.Sq, w.Sk, w.dqk, w.dv, w.scale, True, n_parts, wsv.data_ptr(), nbytes,
                          torch.cuda.current_stream().cuda_stream)
    assert st == fa.FA_OK
    torch.cuda.synchronize()
    assert not torch.isnan(o).any() and not torch.isnan(lse).any()
    for buf, n in ((o_buf, n_o), (l_buf, n_l), (ws, nbytes // 4)):
        assert torch.isnan(buf[:guard]).all() and torch.isnan(buf[guard + n:]).all()
    o_ref, lse_ref = naive_attention(to_f64(q.cpu()), to_f64(k.cpu()), to_f64(v.cpu()), w.scale, True)
    compare(to_f64(o.view(1, w.Hq, w.Sq, w.dv).cpu()), lse.view(1, w.Hq, w.Sq).cpu().double().numpy(), o_ref, lse_ref,
            "guards")
