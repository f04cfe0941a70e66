"""GPU test of the allocation-free decode entry point (fa_fwd_decode_noalloc), through the C ABI.

Its partial results live in the library's static device scratch instead of a caller workspace. Two
calls in a row on one stream, the second with a smaller problem (so the scratch holds the first
call's larger contents when the second starts), each compared with fa_fwd_decode on the same inputs
and part count (same kernels: bit for bit) and with the fp64 oracle at the acceptance bar.
"""

import pytest
import torch

import paper_2609_21264_amd as fa
import workloads as W
from oracle import naive_attention
from parity import compare, to_f64

pytestmark = pytest.mark.gpu

CALLS = [
    # (workload, parts): the first call fills more scratch than the second reads
    (W.small("noalloc gqa4 Sq4 causal 3000", dqk=128, dv=128, B=2, Hq=8, Hkv=2, Sq=4, Sk=3000, causal=True,
             seed=81), 6),
    (W.small("noalloc gqa4 Sq1 d64 700", Hq=4, Hkv=1, Sq=1, Sk=700, seed=82), 2),
]


def _decode(w, n_parts, q, k, v, noalloc):
    o = torch.full((w.B, w.Hq, w.Sq, w.dv), float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full((w.B, w.Hq, w.Sq), float("nan"), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    if noalloc:
        st = fa.fa_fwd_decode_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), w.B,
                                      w.Hq, w.Hkv, w.Sq, w.Sk, w.dqk, w.dv, w.scale, w.causal, n_parts, stream)
    else:
        nbytes = fa.fa_fwd_split_workspace_bytes(w.B, w.Hq, w.Sq, w.dv, n_parts)
        ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        st = fa.fa_fwd_decode(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), w.B, w.Hq,
                              w.Hkv, w.Sq, w.Sk, w.dqk, w.dv, w.scale, w.causal, n_parts, ws.data_ptr(), nbytes,
                              stream)
    assert st == fa.FA_OK, fa.fa_status_str(st)
    torch.cuda.synchronize()
    return o, lse


def test_noalloc_matches_decode_twice_in_a_row():
    inputs = [tuple(x.cuda() for x in W.make_inputs(w)) for w, _ in CALLS]
    torch.cuda.synchronize()
    got = []
    for (w, n_parts), (q, k, v) in zip(CALLS, inputs):
        print(f"[noalloc] {w.name}, parts {n_parts}", flush=True)
        assert fa.fa_fwd_split_workspace_bytes(w.B, w.Hq, w.Sq, w.dv, n_parts) <= fa.FA_NOALLOC_SCRATCH_BYTES
        got.append(_decode(w, n_parts, q, k, v, noalloc=True))
    for (w, n_parts), (q, k, v), (o, lse) in zip(CALLS, inputs, got):
        o_ref, lse_ref = _decode(w, n_parts, q, k, v, noalloc=False)
        assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16)), w.name
        assert torch.equal(lse.view(torch.int32), lse_ref.view(torch.int32)), w.name
        o64, lse64 = naive_attention(to_f64(q), to_f64(k), to_f64(v), w.scale, w.causal)
        compare(to_f64(o), lse.cpu().double().numpy(), o64, lse64, w.name)


def test_noalloc_rejects_more_than_the_scratch():
    w = W.small("noalloc too big", dqk=128, dv=128, Hq=1, Hkv=1, Sq=1, Sk=64, seed=83)
    q, k, v = (x.cuda() for x in W.make_inputs(w))
    o = torch.empty((1, 1, 1, 128), dtype=torch.bfloat16, device="cuda")
    parts = fa.FA_NOALLOC_SCRATCH_BYTES // (129 * 4) + 1
    st = fa.fa_fwd_decode_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), None, 1, 1, 1, 1, 64, 128,
                                  128, w.scale, False, parts, torch.cuda.current_stream().cuda_stream)
    assert st == fa.FA_ERR_WORKSPACE
