"""Seeded synthetic attention workloads, shared by the oracle tests, the GPU tests and the benchmark.

This module holds shapes, seeds, random draws and measurement formulas only. It contains none of
the attention arithmetic (no products, no softmax): the fp64 oracle and the HIP kernels each
implement that on their own, and both take their inputs from here.

Inputs follow the paper's evaluation practice: every element of Q, K and V is drawn i.i.d. from
N(0, sigma^2) with sigma = 1 (Sec. "Numerical Stability", the regime of normalised activations),
at shapes of public LLM attention configurations (Sec. "Generality Across LLM Configurations",
Table 6). Draws are fp32 from torch's CPU generator (mt19937), seeded per workload, in the order
Q, K, V, then rounded to bfloat16 with round-to-nearest-even (torch's ``.to``).
"""

from __future__ import annotations

import math
from dataclasses import dataclass, replace
from typing import Dict, List, Optional, Tuple

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    """One attention problem in contiguous BHSD layout.

    Q: [B][Hq][Sq][dqk], K: [B][Hkv][Sk][dqk], V: [B][Hkv][Sk][dv], O: [B][Hq][Sq][dv],
    LSE: fp32 [B][Hq][Sq]. Query head h reads key/value head h // (Hq // Hkv).
    """

    name: str
    B: int
    Hq: int
    Hkv: int
    Sq: int
    Sk: int
    dqk: int
    dv: int
    causal: bool
    scale: float
    seed: int
    sigma: float = 1.0

    @property
    def group(self) -> int:
        return self.Hq // self.Hkv if self.Hkv else 0

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


def _wl(idx: int, name: str, B, Hq, Hkv, S, dqk, dv, causal) -> Workload:
    return Workload(name=name, B=B, Hq=Hq, Hkv=Hkv, Sq=S, Sk=S, dqk=dqk, dv=dv, causal=causal,
                    scale=1.0 / math.sqrt(dqk), seed=1000 + idx)


#: The five benchmark workloads, numbered 1..5.
CONFIGS: Dict[int, Workload] = {
    1: _wl(1, "single-head B1 H1 S256 d64 non-causal", 1, 1, 1, 256, 64, 64, False),
    2: _wl(2, "BERT-base-shaped B8 H12 S512 d64 non-causal", 8, 12, 12, 512, 64, 64, False),
    3: _wl(3, "Llama-style GQA prefill B1 Hq32 Hkv8 S8192 d128 causal", 1, 32, 8, 8192, 128, 128, True),
    4: _wl(4, "DeepSeek-style wide-head prefill B1 H128 S4096 dqk192 dv128 causal",
           1, 128, 128, 4096, 192, 128, True),
    5: _wl(5, "long-context GQA prefill B1 Hq32 Hkv8 S131072 d128 causal", 1, 32, 8, 131072, 128, 128, True),
}


#: Further workloads for split mode (few query rows against long keys), by name.
EXTRA: Dict[str, Workload] = {
    "decode-128k": Workload(name="decode B1 Hq32 Hkv8 Sq1 Sk131072 d128", B=1, Hq=32, Hkv=8, Sq=1, Sk=131072,
                            dqk=128, dv=128, causal=False, scale=1.0 / math.sqrt(128), seed=1101),
    "decode16-128k-causal": Workload(name="decode B1 Hq32 Hkv8 Sq16 Sk131072 d128 causal", B=1, Hq=32, Hkv=8,
                                     Sq=16, Sk=131072, dqk=128, dv=128, causal=True,
                                     scale=1.0 / math.sqrt(128), seed=1102),
    "decode-b8-8k": Workload(name="decode B8 Hq32 Hkv8 Sq1 Sk8192 d128", B=8, Hq=32, Hkv=8, Sq=1, Sk=8192,
                             dqk=128, dv=128, causal=False, scale=1.0 / math.sqrt(128), seed=1103),
}


def _paper(name: str, H: int, Hkv: int, S: int, d: int, causal: bool, seed: int) -> Workload:
    return Workload(name=name, B=1, Hq=H, Hkv=Hkv, Sq=S, Sk=S, dqk=d, dv=d, causal=causal,
                    scale=1.0 / math.sqrt(d), seed=seed)


#: The paper's own shapes with its XDNA 2 latencies in microseconds, as context for a like-for-like
#: comparison (the paper's hardware, not a target): the GPT-2 Small attention sweep of Table 5 (H=12,
#: d=64, causal, B=1, Sec. 6.1) and the twelve model configurations of Table 6 (Sec. 6.5).
PAPER_SWEEP: List[Tuple[str, Workload, float]] = [
    *[("Table 5", _paper(f"GPT-2 Small attention S{S}", 12, 12, S, 64, True, 1200 + i), us)
      for i, (S, us) in enumerate([(256, 300.0), (512, 600.0), (1024, 1700.0), (2048, 5200.0), (4096, 17200.0),
                                   (8192, 62000.0), (16384, 234500.0), (32768, 911100.0)])],
    ("Table 6", _paper("BERT-Base S2048", 12, 12, 2048, 64, False, 1300), 5775.0),
    ("Table 6", _paper("BERT-Large S2048", 16, 16, 2048, 64, False, 1301), 7526.0),
    ("Table 6", _paper("GPT-2 Small / OPT-125M S2048", 12, 12, 2048, 64, True, 1302), 5810.0),
    ("Table 6", _paper("GPT-2 Medium S2048", 16, 16, 2048, 64, True, 1303), 7535.0),
    ("Table 6", _paper("GPT-2 Large S2048", 20, 20, 2048, 64, True, 1304), 9196.0),
    ("Table 6", _paper("Llama-2 7B S2048", 32, 32, 2048, 128, True, 1305), 34201.0),
    ("Table 6", _paper("Llama-3 8B S2048", 32, 8, 2048, 128, True, 1306), 34076.0),
    ("Table 6", _paper("Qwen1.5-0.5B S32768", 16, 16, 32768, 64, True, 1307), 1214700.0),
    ("Table 6", _paper("Qwen2.5-0.5B-Instruct S32768", 14, 2, 32768, 64, True, 1308), 1062870.0),
    ("Table 6", _paper("Qwen1.5-0.5B S131072", 16, 16, 131072, 64, True, 1309), 18996700.0),
    ("Table 6", _paper("DeepSeek LLM 7B S4096", 32, 32, 4096, 128, True, 1310), 114443.0),
    ("Table 6", _paper("DeepSeek LLM 67B S4096", 64, 8, 4096, 128, True, 1311), 227467.0),
]


def make_inputs(w: Workload, device: str = "cpu") -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """Draw Q, K, V (bf16, contiguous BHSD) for workload ``w`` from its seed.

    The fp32 draws are rounded to bf16 before anything else sees them; the bf16 tensors are
    the exact inputs of both the oracle and the GPU path.
    """
    g = torch.Generator(device="cpu")
    g.manual_seed(w.seed)
    out = []
    for shape in ((w.B, w.Hq, w.Sq, w.dqk), (w.B, w.Hkv, w.Sk, w.dqk), (w.B, w.Hkv, w.Sk, w.dv)):
        x = torch.randn(shape, dtype=torch.float32, generator=g)
        if w.sigma != 1.0:
            x.mul_(w.sigma)
        out.append(x.to(torch.bfloat16).contiguous())
        del x
    q, k, v = out
    if device != "cpu":
        q, k, v = q.to(device), k.to(device), v.to(device)
    return q, k, v


def sample_rows(w: Workload, n: int = 64, seed_base: int = 2000) -> List[np.ndarray]:
    """Seeded query-row subset per query head (used where the full output is too large for the oracle).

    For each head h in order: ``sorted(rng.choice(Sq, n))`` without replacement, plus rows 0 and Sq-1.
    The generator is ``numpy.random.default_rng(seed_base + (seed - 1000))``.
    """
    rng = np.random.default_rng(seed_base + (w.seed - 1000))
    rows = []
    for _ in range(w.B * w.Hq):
        r = rng.choice(w.Sq, size=min(n, w.Sq), replace=False)
        r = np.union1d(r, [0, w.Sq - 1]) if w.Sq > 0 else r
        rows.append(np.asarray(sorted(r), dtype=np.int64))
    return rows


def metric_flops(w: Workload) -> float:
    """GEMM FLOPs of one forward pass in the metric's convention.

    2*B*Hq*Sq*Sk*(dqk + dv): the two contractions Q.K^T and P.V (Sec. "Operational Intensity
    Constraint"), halved exactly when causal.
    """
    f = 2.0 * w.B * w.Hq * w.Sq * w.Sk * (w.dqk + w.dv)
    return f * 0.5 if w.causal else f


def paper_flops(H: int, Lq: int, Lk: int, dk: int, dv: int, B: int = 1) -> float:
    """Effective GEMM work of the paper's throughput formula (Sec. 6.1, P_effGEMM numerator).

    2*H*Lq*Lk*(dk+dv), never halved for causal masking.
    """
    return 2.0 * B * H * Lq * Lk * (dk + dv)


def algorithmic_bytes(w: Workload, with_lse: bool = True) -> int:
    """HBM bytes a fused forward must move at minimum: read Q, K, V once, write O (bf16) and LSE (fp32)."""
    q = w.B * w.Hq * w.Sq * w.dqk
    k = w.B * w.Hkv * w.Sk * w.dqk
    v = w.B * w.Hkv * w.Sk * w.dv
    o = w.B * w.Hq * w.Sq * w.dv
    lse = w.B * w.Hq * w.Sq if with_lse else 0
    return 2 * (q + k + v + o) + 4 * lse


def visible_scores(w: Workload) -> int:
    """Number of (query, key) pairs the mask leaves visible: B*Hq*Sq*Sk, or with causal masking the sum
    over query rows i of clamp(i + 1 + Sk - Sq, 0, Sk)."""
    if not w.causal:
        return w.B * w.Hq * w.Sq * w.Sk
    per_row = np.clip(np.arange(w.Sq, dtype=np.int64) + 1 + w.Sk - w.Sq, 0, w.Sk)
    return int(w.B * w.Hq * per_row.sum())


def unfused_algorithmic_bytes(w: Workload) -> Dict[str, int]:
    """HBM bytes the layer-by-layer operators must move at minimum, per operator: the score matrix and
    the probabilities are written once and read once in bf16 over the visible pairs, next to the
    operators' own inputs and outputs (Q, K for the scores; LSE for the softmax; V, O for P V)."""
    n = visible_scores(w)
    q = 2 * w.B * w.Hq * w.Sq * w.dqk
    k = 2 * w.B * w.Hkv * w.Sk * w.dqk
    v = 2 * w.B * w.Hkv * w.Sk * w.dv
    o = 2 * w.B * w.Hq * w.Sq * w.dv
    lse = 4 * w.B * w.Hq * w.Sq
    return {"scores": 2 * n + q + k, "softmax": 4 * n + lse, "pv": 2 * n + v + o}


def small(name: str, B=1, Hq=1, Hkv=1, Sq=64, Sk=64, dqk=64, dv=64, causal=False,
          scale: Optional[float] = None, seed: int = 7, sigma: float = 1.0) -> Workload:
    """An ad-hoc workload for tests (odd shapes, edge cases)."""
    return Workload(name=name, B=B, Hq=Hq, Hkv=Hkv, Sq=Sq, Sk=Sk, dqk=dqk, dv=dv, causal=causal,
                    scale=(1.0 / math.sqrt(dqk)) if scale is None else scale, seed=seed, sigma=sigma)
