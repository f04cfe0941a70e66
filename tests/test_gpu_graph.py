"""GPU tests: every entry point replayed from a captured HIP graph.

Each path (fused, split mode, decode path, unfused baseline) is captured once through the Python
binding on a side stream, then replayed several times with eager work in between: the input tensors
are overwritten in place with one of two seeded input sets, and each replay must reproduce, bit for
bit, the eager result for the inputs it saw (the kernels are deterministic). None of the paths
records a memset node; outputs and workspaces come from the graph's memory pool.
"""

import math

import pytest
import torch

import paper_2609_21264_amd as fa
import workloads as W

pytestmark = pytest.mark.gpu

# name: (B, Hq, Hkv, Sq, Sk, d_qk, d_v, causal, call)
CASES = {
    # a few query blocks: the key-halves instance
    "fused": (1, 4, 2, 300, 300, 128, 128, True, lambda q, k, v, c: fa.forward(q, k, v, causal=c, return_lse=True)),
    # 96 blocks of 256 rows at d = 64 without a mask: the short instance
    "fused-short": (1, 96, 48, 130, 200, 64, 64, False,
                    lambda q, k, v, c: fa.forward(q, k, v, causal=c, return_lse=True)),
    # more than 256 blocks at d = 128: the long instance
    "fused-long": (1, 264, 66, 130, 200, 128, 128, False,
                   lambda q, k, v, c: fa.forward(q, k, v, causal=c, return_lse=True)),
    "fused-d192": (2, 2, 1, 130, 200, 192, 128, False,
                   lambda q, k, v, c: fa.forward(q, k, v, causal=c, return_lse=True)),
    "split": (1, 4, 1, 64, 2000, 128, 128, True,
              lambda q, k, v, c: fa.forward(q, k, v, causal=c, return_lse=True, n_split=4)),
    "decode": (2, 8, 2, 2, 3000, 128, 128, True,
               lambda q, k, v, c: fa.forward(q, k, v, causal=c, return_lse=True, decode=True, n_split="auto")),
    "unfused": (1, 2, 1, 200, 300, 64, 64, True,
                lambda q, k, v, c: fa.forward_unfused(q, k, v, causal=c, return_lse=True)),
}


def inputs(case, seed):
    B, Hq, Hkv, Sq, Sk, dqk, dv, causal, _ = CASES[case]
    w = W.Workload(name=case, B=B, Hq=Hq, Hkv=Hkv, Sq=Sq, Sk=Sk, dqk=dqk, dv=dv, causal=causal,
                   scale=1.0 / math.sqrt(dqk), seed=seed)
    return W.make_inputs(w)


INSTANCE = {"fused": 64, "fused-short": 128, "fused-long": 256, "fused-d192": 256}


@pytest.mark.parametrize("case", list(CASES))
def test_graph_replay_matches_eager(case):
    causal, call = CASES[case][7], CASES[case][8]
    if case in INSTANCE:
        B, Hq, _, Sq, _, dqk, dv, _, _ = CASES[case]
        assert fa.fa_fwd_rows(B, Hq, Sq, dqk, dv, causal) == INSTANCE[case]
    sets = [inputs(case, 7100), inputs(case, 7200)]
    q, k, v = (t.cuda() for t in sets[0])

    def load(i):
        for dst, src in zip((q, k, v), sets[i]):
            dst.copy_(src)

    eager = []
    for i in range(2):
        load(i)
        o, lse = call(q, k, v, causal)
        torch.cuda.synchronize()
        eager.append((o.clone(), lse.clone()))
    assert not torch.equal(eager[0][0], eager[1][0])

    load(0)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call(q, k, v, causal)  # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        o_g, lse_g = call(q, k, v, causal)
    torch.cuda.synchronize()

    for rep, i in enumerate((1, 0, 1, 1, 0)):
        load(i)
        o_g.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(o_g, eager[i][0]), f"{case}: replay {rep} (input set {i}) differs in O"
        assert torch.equal(lse_g, eager[i][1]), f"{case}: replay {rep} (input set {i}) differs in LSE"
