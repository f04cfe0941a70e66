"""GPU tests at the largest key length the ABI accepts (one head's K and V just under 4 GiB each).

The kernels address one head's K and V with 32-bit byte offsets from a 64-bit head base; these runs
put the last key tile at the very end of that range, and the second key/value head's base past 4 GiB.
The inputs have a closed-form answer, so the oracle needs no 4 GiB matrices: Q = e0 (every row of
every head), K = 0 except the last key K[L] = (s_h / scale) e0 with a score s_h of its own per
key/value head h, V = a except V[L] = b. A query row that sees the keys 0 .. n-1 (n <= L) gets O = a
and LSE = ln n; a row that also sees key L gets O = (L a + e^s b) / (L + e^s) and LSE = ln(L + e^s).
The last key's score sits far above the others, so the fused kernel's online softmax must rebase on
the last tile. Two query heads share each key/value head (grouped-query attention), which runs the
key-halves kernel instance; further fused runs with 100 and 129 per key/value head have enough query
blocks for the short (without a mask) and the long instance.
"""

import math

import numpy as np
import pytest
import torch

import paper_2609_21264_amd as fa
from parity import to_f64

pytestmark = pytest.mark.gpu

D = 128
SCALE = 0.125
SPIKES = (16.0, 8.0)                          # score of the last key, per key/value head
GROUP = 2                                     # query heads per key/value head
A, BV = 0.5, -1.0                             # V rows before the last, and the last
MAX_SK = (2 ** 31 - 1) // D // 64 * 64        # largest Sk with Sk * d < 2^31, a whole number of key tiles
LBL_MAX_SK = 2 ** 22                          # the layer-by-layer operators' limit


def spike_inputs(sq, sk, hkv, group=GROUP):
    q = torch.zeros(1, hkv * group, sq, D, dtype=torch.bfloat16, device="cuda")
    q[..., 0] = 1.0
    k = torch.zeros(1, hkv, sk, D, dtype=torch.bfloat16, device="cuda")
    for h in range(hkv):
        k[0, h, sk - 1, 0] = SPIKES[h] / SCALE  # 128 and 64: exact in bf16
    v = torch.full((1, hkv, sk, D), A, dtype=torch.bfloat16, device="cuda")
    v[0, :, sk - 1] = BV
    return q, k, v


def expected(sq, sk, causal, spike):
    """Closed-form O (one value per row, all dims equal) and LSE of one query head."""
    last = sk - 1
    o, lse = np.zeros(sq), np.zeros(sq)
    for i in range(sq):
        n = min(sk, i + 1 + sk - sq) if causal else sk
        if n <= last:
            o[i], lse[i] = A, math.log(n)
        else:
            e = math.exp(spike)
            o[i], lse[i] = (last * A + e * BV) / (last + e), math.log(last + e)
    return o, lse


def check(o, lse, sq, sk, causal, what, group=GROUP):
    got_o, got_lse = to_f64(o.cpu())[0], lse.cpu().double().numpy()[0]
    for hq in range(got_o.shape[0]):
        o_ref, lse_ref = expected(sq, sk, causal, SPIKES[hq // group])
        # one bf16 rounding of O plus fp32 accumulation over Sk terms; the bar of the prefill kernel
        assert np.all(np.abs(got_o[hq] - o_ref[:, None]) <= 2e-2), f"{what} head {hq}: {got_o[hq, :, 0]} vs {o_ref}"
        assert np.abs(got_lse[hq] - lse_ref).max() <= 1e-3, f"{what} head {hq}: LSE {got_lse[hq]} vs {lse_ref}"


@pytest.fixture(scope="module")
def big():
    sq = 3
    q, k, v = spike_inputs(sq, MAX_SK, hkv=2)
    yield sq, q, k, v
    del q, k, v
    torch.cuda.empty_cache()


@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
def test_fused_at_largest_key_length(big, causal):
    sq, q, k, v = big
    assert fa.fa_fwd_rows(1, q.shape[1], sq, D, D, causal) == 64
    o, lse = fa.forward(q, k, v, causal=causal, scale=SCALE, return_lse=True)
    torch.cuda.synchronize()
    check(o, lse, sq, MAX_SK, causal, f"fused causal={causal}")


@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
def test_fused_long_instance_at_largest_key_length(big, causal):
    """The same keys with 129 query heads per key/value head: 258 query blocks, more than the other
    instances take, so the long instance's loaders address the end of the 4 GiB heads."""
    sq, _, k, v = big
    group = 129
    assert fa.fa_fwd_rows(1, 2 * group, sq, D, D, causal) == 256
    q = torch.zeros(1, 2 * group, sq, D, dtype=torch.bfloat16, device="cuda")
    q[..., 0] = 1.0
    o, lse = fa.forward(q, k, v, causal=causal, scale=SCALE, return_lse=True)
    torch.cuda.synchronize()
    check(o, lse, sq, MAX_SK, causal, f"fused long causal={causal}", group)


def test_fused_short_instance_at_largest_key_length(big):
    """100 query heads per key/value head without a mask: 200 query blocks, which the short instance
    runs (causal problems at this head dimension go from the key-halves to the long instance)."""
    sq, _, k, v = big
    group = 100
    assert fa.fa_fwd_rows(1, 2 * group, sq, D, D, False) == 128
    q = torch.zeros(1, 2 * group, sq, D, dtype=torch.bfloat16, device="cuda")
    q[..., 0] = 1.0
    o, lse = fa.forward(q, k, v, causal=False, scale=SCALE, return_lse=True)
    torch.cuda.synchronize()
    check(o, lse, sq, MAX_SK, False, "fused short", group)


def test_split_at_largest_key_length(big):
    sq, q, k, v = big
    o, lse = fa.forward(q, k, v, causal=True, scale=SCALE, return_lse=True, n_split=64)
    torch.cuda.synchronize()
    check(o, lse, sq, MAX_SK, True, "split")


def test_decode_at_largest_key_length(big):
    sq, q, k, v = big
    o, lse = fa.forward(q, k, v, causal=True, scale=SCALE, return_lse=True, decode=True, n_split="auto")
    torch.cuda.synchronize()
    check(o, lse, sq, MAX_SK, True, "decode")


def test_unfused_at_its_largest_key_length():
    sq = 3
    q, k, v = spike_inputs(sq, LBL_MAX_SK, hkv=2)
    o, lse = fa.forward_unfused(q, k, v, causal=True, scale=SCALE, return_lse=True)
    torch.cuda.synchronize()
    check(o, lse, sq, LBL_MAX_SK, True, "unfused")
