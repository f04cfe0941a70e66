"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle, element by element.

Small problems compare every element and span several tiles with ragged tails; the five benchmark
workloads run at full size in the same launch configuration the benchmark times, with configs 1-2
compared in full and 3-5 on seeded row subsets of every head.
"""

import numpy as np
import pytest
import torch

import paper_2609_21264_amd as fa
import workloads as W
from parity import check_every_element, check_full, check_rows, compare, run_gpu, to_f64
from oracle import naive_attention

pytestmark = pytest.mark.gpu


def _case(name, **kw):
    return W.small(name, **kw)


SMALL_CASES = [
    # single tile, partial tiles, several tiles with ragged tails, each head dim
    _case("d64 1x1", Sq=1, Sk=1),
    _case("d64 17x17 causal", Sq=17, Sk=17, causal=True),
    _case("d64 63x65", Sq=63, Sk=65),
    _case("d64 257 causal gqa", Hq=4, Hkv=1, Sq=257, Sk=257, causal=True, seed=11),
    _case("d64 100x257", B=2, Hq=2, Hkv=2, Sq=100, Sk=257, seed=12),
    _case("d128 65 causal", dqk=128, dv=128, Sq=65, Sk=65, causal=True, seed=13),
    _case("d128 300x300 gqa7", dqk=128, dv=128, Hq=7, Hkv=1, Sq=300, Sk=300, causal=True, seed=14),
    _case("d128 257x100 noncausal", dqk=128, dv=128, Hq=4, Hkv=4, Sq=257, Sk=100, seed=15),
    _case("d192/128 129 causal", dqk=192, dv=128, Hq=2, Hkv=2, Sq=129, Sk=129, causal=True, seed=16),
    _case("d192/128 200x333", dqk=192, dv=128, Sq=200, Sk=333, seed=17),
    # bottom-right causal with Sq != Sk (rows with no visible key when Sq > Sk)
    _case("d64 causal Sq<Sk", Sq=40, Sk=170, causal=True, seed=18),
    _case("d128 causal Sq>Sk", dqk=128, dv=128, Sq=300, Sk=90, causal=True, seed=19),
    # scale variants: zero (uniform weights), negative, large
    _case("d64 scale 0", Sq=70, Sk=130, causal=True, scale=0.0, seed=20),
    _case("d128 negative scale", dqk=128, dv=128, Sq=130, Sk=130, scale=-0.09, seed=21),
    _case("d64 sharp softmax", Sq=96, Sk=96, scale=1.0, seed=22),
    # wider value range (sigma = 2: score variance 16)
    _case("d128 sigma 2 causal", dqk=128, dv=128, Sq=192, Sk=192, causal=True, sigma=2.0, seed=23),
]


@pytest.mark.parametrize("w", SMALL_CASES, ids=[c.name for c in SMALL_CASES])
def test_small_shapes_match_oracle(w):
    print(f"\n[case] {w}", flush=True)
    check_full(w)


@pytest.mark.parametrize("cfg", [1, 2])
def test_benchmark_config_full(cfg):
    w = W.CONFIGS[cfg]
    print(f"\n[case] config {cfg}: {w}", flush=True)
    check_full(w)


@pytest.mark.parametrize("cfg", [3, 4])
def test_benchmark_config_every_element(cfg):
    w = W.CONFIGS[cfg]
    print(f"\n[case] config {cfg}, every element: {w}", flush=True)
    check_every_element(w)


@pytest.mark.parametrize("cfg,rows", [(3, 256), (4, 128), (5, 64)])
def test_benchmark_config_sampled_rows(cfg, rows):
    w = W.CONFIGS[cfg]
    print(f"\n[case] config {cfg} ({rows} rows/head): {w}", flush=True)
    check_rows(w, rows)


def test_empty_key_sequence():
    w = _case("Sk=0", Sq=70, Sk=0, causal=False)
    q = torch.randn(1, 1, 70, 64).to(torch.bfloat16)
    k = torch.zeros(1, 1, 0, 64, dtype=torch.bfloat16)
    o, lse = run_gpu(q, k, k, w)
    assert torch.all(o.cpu() == 0)
    assert torch.all(torch.isneginf(lse.cpu()))


def test_every_output_written_and_no_out_of_bounds_writes():
    w = _case("sentinel", dqk=128, dv=128, Hq=4, Hkv=2, Sq=261, Sk=261, causal=True, seed=31)
    q, k, v = (x.cuda() for x in W.make_inputs(w))
    n_o, n_l, guard = w.Hq * w.Sq * w.dv, w.Hq * w.Sq, 4096
    o_buf = torch.full((n_o + 2 * guard,), float("nan"), dtype=torch.bfloat16, device="cuda")
    l_buf = torch.full((n_l + 2 * guard,), float("nan"), dtype=torch.float32, device="cuda")
    o = o_buf[guard:guard + n_o].view(1, w.Hq, w.Sq, w.dv)
    lse = l_buf[guard:guard + n_l].view(1, w.Hq, w.Sq)
    import paper_2609_21264_amd as fa
    fa.forward(q, k, v, causal=True, scale=w.scale, return_lse=True, out=o, lse=lse)
    torch.cuda.synchronize()
    assert not torch.isnan(o).any() and not torch.isnan(lse).any()
    assert torch.isnan(o_buf[:guard]).all() and torch.isnan(o_buf[guard + n_o:]).all()
    assert torch.isnan(l_buf[:guard]).all() and torch.isnan(l_buf[guard + n_l:]).all()


def test_runs_are_bitwise_deterministic():
    w = W.CONFIGS[2]
    q, k, v = W.make_inputs(w)
    o1, l1 = run_gpu(q, k, v, w)
    o2, l2 = run_gpu(q, k, v, w)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_non_default_stream():
    w = _case("stream", dqk=128, dv=128, Hq=8, Hkv=2, Sq=500, Sk=500, causal=True, seed=41)
    q, k, v = W.make_inputs(w)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        o, lse = run_gpu(q, k, v, w, stream=s)
    o_ref, lse_ref = naive_attention(to_f64(q), to_f64(k), to_f64(v), w.scale, True)
    compare(to_f64(o), lse.cpu().double().numpy(), o_ref, lse_ref, "stream")


def test_causal_first_row_is_first_value_bitwise():
    w = _case("row0", dqk=128, dv=128, Hq=4, Hkv=2, Sq=300, Sk=300, causal=True, seed=51)
    q, k, v = W.make_inputs(w)
    o, _ = run_gpu(q, k, v, w)
    o = o.cpu()
    for h in range(4):
        assert torch.equal(o[0, h, 0], v[0, h // 2, 0])


def test_gqa_equals_repeated_kv_bitwise():
    w = _case("gqa", dqk=128, dv=128, Hq=8, Hkv=2, Sq=333, Sk=333, causal=True, seed=61)
    q, k, v = W.make_inputs(w)
    o1, l1 = run_gpu(q, k, v, w)
    kr, vr = k.repeat_interleave(4, dim=1).contiguous(), v.repeat_interleave(4, dim=1).contiguous()
    o2, l2 = run_gpu(q, kr, vr, w.with_(Hkv=8))
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_zero_queries_give_prefix_mean():
    w = _case("q0", dqk=128, dv=128, Sq=200, Sk=200, causal=True, seed=71)
    q, k, v = W.make_inputs(w)
    q = torch.zeros_like(q)
    o, lse = run_gpu(q, k, v, w)
    vf = to_f64(v)[0, 0]
    mean = np.cumsum(vf, axis=0) / np.arange(1, 201)[:, None]
    assert np.abs(to_f64(o)[0, 0] - mean).max() <= 2e-2
    assert np.abs(lse.cpu().double().numpy()[0, 0] - np.log(np.arange(1, 201))).max() <= 1e-3


def test_single_hip_runtime_mapped():
    import paper_2609_21264_amd as fa  # noqa: F401
    torch.zeros(1, device="cuda")
    maps = open("/proc/self/maps").read().splitlines()
    libs = {ln.split()[-1] for ln in maps if "libamdhip64" in ln}
    assert len(libs) == 1, libs
    assert any("libfa.so" in ln for ln in maps)


@pytest.mark.parametrize("n_split", [1, 3], ids=["fused", "split3"])
@pytest.mark.parametrize("causal", [False, True], ids=["full", "causal"])
def test_rising_maxima_rebase_at_every_position(causal, n_split):
    """Keys whose scores jump far above everything before them, in the second key tile, two middle
    tiles and the last one (scaled by 4, 8, 16 and 32: exact in bf16, scores up to ~±100 in natural
    units), so that a lane's exponential sum passes the bound and the tile is redone from its exact
    row maximum at each of those positions; every output row against the oracle."""
    w = _case("spikes", dqk=128, dv=128, Hq=2, Hkv=1, Sq=640, Sk=640, causal=causal, seed=81)
    q, k, v = W.make_inputs(w)
    for key, factor in ((70, 4.0), (300, 8.0), (520, 16.0), (600, 32.0)):
        k[:, :, key] *= factor
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    o, lse = fa.forward(qd, kd, vd, causal=causal, scale=w.scale, return_lse=True, n_split=n_split)
    torch.cuda.synchronize()
    o_ref, lse_ref = naive_attention(to_f64(q), to_f64(k), to_f64(v), w.scale, causal)
    # the spikes really dominate some rows: their LSE rises far above ln(Sk)
    assert np.nanmax(lse_ref) > 20.0
    compare(to_f64(o), lse.cpu().double().numpy(), o_ref, lse_ref, f"spikes causal={causal} split={n_split}")


def test_concurrent_threads_and_streams():
    """The library keeps no state: two host threads, each on its own stream with its own problem,
    calling the fused and split entry points concurrently, get exactly the single-stream results."""
    import threading

    cases = [_case("t0", dqk=128, dv=128, Hq=4, Hkv=2, Sq=333, Sk=517, causal=True, seed=91),
             _case("t1", dqk=64, dv=64, Hq=3, Hkv=1, Sq=200, Sk=700, causal=False, seed=92)]
    data = []
    for w in cases:
        q, k, v = (t.cuda() for t in W.make_inputs(w))
        ref = [fa.forward(q, k, v, causal=w.causal, scale=w.scale, return_lse=True, n_split=ns) for ns in (1, 3)]
        torch.cuda.synchronize()
        data.append((w, q, k, v, [(o.clone(), l.clone()) for o, l in ref]))
    errors = []

    def worker(idx):
        w, q, k, v, ref = data[idx]
        stream = torch.cuda.Stream()
        try:
            with torch.cuda.stream(stream):
                outs = []
                for rep in range(20):
                    ns = (1, 3)[rep % 2]
                    outs.append((ns, fa.forward(q, k, v, causal=w.causal, scale=w.scale, return_lse=True,
                                                n_split=ns, stream=stream)))
            stream.synchronize()
            for ns, (o, l) in outs:
                ro, rl = ref[0 if ns == 1 else 1]
                if not (torch.equal(o, ro) and torch.equal(l, rl)):
                    errors.append(f"{w.name} n_split={ns}")
        except Exception as e:  # reported in the main thread
            errors.append(f"{w.name}: {e!r}")

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(len(data))]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors


def test_fa_fwd_entry_point():
    """fa_fwd (one head dimension, no LSE) through the C ABI: the oracle's result, and bit for bit the
    output of fa_fwd_ex on the same inputs."""
    w = _case("fa_fwd d128 gqa causal", dqk=128, dv=128, B=2, Hq=8, Hkv=2, Sq=300, Sk=420, causal=True, seed=95)
    q, k, v = W.make_inputs(w)
    qd, kd, vd = q.cuda(), k.cuda(), v.cuda()
    o1 = torch.empty(w.B, w.Hq, w.Sq, w.dv, dtype=torch.bfloat16, device="cuda")
    o2 = torch.empty_like(o1)
    lse = torch.empty(w.B, w.Hq, w.Sq, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    assert fa.fa_fwd(qd.data_ptr(), kd.data_ptr(), vd.data_ptr(), o1.data_ptr(), w.B, w.Hq, w.Hkv, w.Sq, w.Sk, w.dqk,
                     w.scale, w.causal, stream) == fa.FA_OK
    assert fa.fa_fwd_ex(qd.data_ptr(), kd.data_ptr(), vd.data_ptr(), o2.data_ptr(), lse.data_ptr(), w.B, w.Hq, w.Hkv,
                        w.Sq, w.Sk, w.dqk, w.dv, w.scale, w.causal, stream) == fa.FA_OK
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)
    o_ref, lse_ref = naive_attention(to_f64(q), to_f64(k), to_f64(v), w.scale, w.causal)
    compare(to_f64(o1), lse.cpu().double().numpy(), o_ref, lse_ref, w.name)


def test_forward_rejects_out_and_lse_on_the_host():
    """A caller-supplied out or lse in host memory is rejected before any launch (its pointer would
    otherwise reach the kernel)."""
    w = _case("host out", dqk=128, dv=128, Hq=2, Hkv=1, Sq=64, Sk=64, seed=96)
    q, k, v = (x.cuda() for x in W.make_inputs(w))
    with pytest.raises(ValueError, match="out must be on"):
        fa.forward(q, k, v, out=torch.empty(1, 2, 64, 128, dtype=torch.bfloat16))
    with pytest.raises(ValueError, match="lse must be on"):
        fa.forward(q, k, v, lse=torch.empty(1, 2, 64, dtype=torch.float32))


def test_stream_on_another_device_is_rejected():
    # a torch stream must belong to the tensors' device (the kernels run on the stream's device)
    s = torch.cuda.Stream()
    with pytest.raises(ValueError, match="stream is on"):
        fa._stream(s, torch.device("cpu"))
    assert fa._stream(s, s.device)[1] == s.cuda_stream


def test_raw_stream_handle_keeps_the_split_workspace_alive():
    """A raw stream handle (an int) is wrapped so that the split-mode workspace is recorded on it: the
    result on a busy side stream equals the result on the current stream, bit for bit."""
    w = _case("raw handle split", dqk=128, dv=128, Hq=4, Hkv=2, Sq=100, Sk=3000, causal=False, seed=97)
    q, k, v = (x.cuda() for x in W.make_inputs(w))
    ref = fa.forward(q, k, v, scale=w.scale, return_lse=True, n_split=4)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    outs = []
    for _ in range(8):
        outs.append(fa.forward(q, k, v, scale=w.scale, return_lse=True, n_split=4, stream=side.cuda_stream))
        junk = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")  # reuses freed blocks at once
        junk.fill_(0xff)
    side.synchronize()
    torch.cuda.synchronize()
    for o, l in outs:
        assert torch.equal(o, ref[0]) and torch.equal(l, ref[1])
