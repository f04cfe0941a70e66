"""GPU parity of split mode (fa_fwd_split): every query block's key range cut into parts that run as
separate workgroups, then a log-sum-exp merge (the paper's tile-to-tile level, Alg. 2). Compared with
the fp64 oracle element by element, at the same bar as the single-pass kernel."""

import numpy as np
import pytest
import torch

import paper_2609_21264_amd as fa
import workloads as W
from oracle import naive_attention
from parity import compare, to_f64

pytestmark = pytest.mark.gpu


def run_split(w: W.Workload, n_split: int, inputs=None):
    q, k, v = inputs if inputs is not None else W.make_inputs(w)
    o, lse = fa.forward(q.cuda(), k.cuda(), v.cuda(), causal=w.causal, scale=w.scale, return_lse=True,
                        n_split=n_split)
    torch.cuda.synchronize()
    return q, k, v, o, lse


def check_split(w: W.Workload, n_split: int):
    q, k, v, o, lse = run_split(w, n_split)
    o_ref, lse_ref = naive_attention(to_f64(q), to_f64(k), to_f64(v), w.scale, w.causal)
    return compare(to_f64(o), lse.cpu().double().numpy(), o_ref, lse_ref, f"{w.name} split {n_split}",
                   max(1.0, w.sigma))


CASES = [
    (W.small("d64 63x650 split", Sq=63, Sk=650, seed=41), 3),
    (W.small("d64 300 causal gqa split", Hq=4, Hkv=1, Sq=300, Sk=300, causal=True, seed=42), 2),
    (W.small("d64 causal Sq<Sk split", Sq=40, Sk=700, causal=True, seed=43), 5),
    (W.small("d128 257x1000 split", dqk=128, dv=128, Hq=2, Hkv=2, Sq=257, Sk=1000, seed=44), 4),
    (W.small("d128 causal Sq>Sk split", dqk=128, dv=128, Sq=300, Sk=90, causal=True, seed=45), 3),
    (W.small("d128 causal gqa split", dqk=128, dv=128, Hq=8, Hkv=2, Sq=512, Sk=512, causal=True, seed=46), 7),
    (W.small("d192/128 200x900 split", dqk=192, dv=128, Sq=200, Sk=900, seed=47), 3),
    (W.small("d192/128 causal split", dqk=192, dv=128, Hq=2, Hkv=1, Sq=333, Sk=333, causal=True, seed=48), 2),
    # more parts than key tiles: the extra parts are empty and weigh nothing in the merge
    (W.small("d64 100x150 split 16", Sq=100, Sk=150, seed=49), 16),
    # decode-like: few query rows against long keys
    (W.small("d128 decode 1x4000 gqa", dqk=128, dv=128, Hq=8, Hkv=2, Sq=1, Sk=4000, seed=50), 8),
    (W.small("d128 decode 16x3000 causal", dqk=128, dv=128, Hq=4, Hkv=1, Sq=16, Sk=3000, causal=True,
             seed=51), 12),
    (W.small("d64 decode 7x2500 causal", Hq=3, Hkv=3, Sq=7, Sk=2500, causal=True, seed=52), 6),
    # wider value range and a sharp softmax, where the parts' maxima differ a lot
    (W.small("d128 sigma 2 split", dqk=128, dv=128, Sq=128, Sk=777, sigma=2.0, seed=53), 4),
    (W.small("d64 sharp split", Sq=96, Sk=960, scale=1.0, seed=54), 5),
]


@pytest.mark.parametrize("w,n_split", CASES, ids=[f"{c[0].name}" for c in CASES])
def test_split_matches_oracle(w, n_split):
    check_split(w, n_split)


def test_split_config1_full():
    check_split(W.CONFIGS[1], 4)


def test_split_one_part_equals_single_pass_bitwise():
    # one part: O = bf16(acc / l) and LSE = m + ln l through the workspace, the same values as the
    # single-pass kernel
    w = W.small("one part", dqk=128, dv=128, Hq=4, Hkv=2, Sq=200, Sk=300, causal=True, seed=55)
    q, k, v = W.make_inputs(w)
    _, _, _, o1, l1 = run_split(w, 1, (q, k, v))
    o2, l2 = fa.forward(q.cuda(), k.cuda(), v.cuda(), causal=True, scale=w.scale, return_lse=True)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_split_is_bitwise_deterministic():
    w = W.small("det", dqk=128, dv=128, Hq=4, Hkv=1, Sq=64, Sk=2000, causal=True, seed=56)
    inputs = W.make_inputs(w)
    _, _, _, o1, l1 = run_split(w, 6, inputs)
    _, _, _, o2, l2 = run_split(w, 6, inputs)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_split_writes_only_its_buffers():
    w = W.small("guards", dqk=128, dv=128, Hq=2, Hkv=1, Sq=70, Sk=500, causal=True, seed=57)
    q, k, v = (x.cuda() for x in W.make_inputs(w))
    n_split = 3
    nbytes = fa.fa_fwd_split_workspace_bytes(w.B, w.Hq, w.Sq, w.dv, n_split)
    assert nbytes == n_split * w.B * w.Hq * w.Sq * (w.dv + 1) * 4
    guard = 4096
    n_o, n_l = w.Hq * w.Sq * w.dv, w.Hq * w.Sq
    o_buf = torch.full((n_o + 2 * guard,), float("nan"), dtype=torch.bfloat16, device="cuda")
    l_buf = torch.full((n_l + 2 * guard,), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.full((nbytes // 4 + 2 * guard,), float("nan"), dtype=torch.float32, device="cuda")
    o = o_buf[guard:guard + n_o]
    lse = l_buf[guard:guard + n_l]
    wsv = ws[guard:guard + nbytes // 4]
    st = fa.fa_fwd_split(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), w.B, w.Hq, w.Hkv,
                         w.Sq, w.Sk, w.dqk, w.dv, w.scale, True, n_split, wsv.data_ptr(), nbytes,
                         torch.cuda.current_stream().cuda_stream)
    assert st == fa.FA_OK
    torch.cuda.synchronize()
    assert not torch.isnan(o).any() and not torch.isnan(lse).any()
    for buf, n in ((o_buf, n_o), (l_buf, n_l), (ws, nbytes // 4)):
        assert torch.isnan(buf[:guard]).all() and torch.isnan(buf[guard + n:]).all()
    o_ref, lse_ref = naive_attention(to_f64(q.cpu()), to_f64(k.cpu()), to_f64(v.cpu()), w.scale, True)
    compare(to_f64(o.view(1, w.Hq, w.Sq, w.dv).cpu()), lse.view(1, w.Hq, w.Sq).cpu().double().numpy(), o_ref,
            lse_ref, "guards")
