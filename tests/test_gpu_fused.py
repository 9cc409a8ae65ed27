"""GPU parity of the attention with in-kernel selection (ugbs_attend_select).

  - given the oracle's tile scores and trigger flags: the output equals
    ugbs_attend on the oracle's kv_idx bit for bit (same block set, same
    visiting order, same arithmetic), and the fp64 oracle attention on that
    kv_idx within the attention bar (max-abs 2e-2, RMS 2e-3);
  - plain top-k (no trigger), every tile triggered, k = N_B (every tile
    saturated: dense causal attention), tiny sequences;
  - the fused layer (scores + sigma without lists, route flags, attention
    with selection) equals the layer with kv_idx lists bit for bit, on the
    same inputs (two GPU paths; the lists path is itself pinned to the
    oracle in test_gpu_parity.py).
"""
import numpy as np
import pytest

import oracle
import paper_2607_07724_amd as ugbs
from paper_2607_07724_amd import synth

from gpu_helpers import attention_error, dev, dev_bf16, host, host_bits

pytestmark = pytest.mark.gpu
ATOL_MAX, ATOL_RMS = 2e-2, 2e-3

CASES = {
    "C1": synth.WORKLOADS["C1"],
    "kmean_d128_gqa4": synth.Workload("F1", 1, 8, 2, 128, 4096, 8, 0.1, synth.KMEAN, "offset",
                                      needles=4, base_seed=51),
    "quest_d128_b2": synth.Workload("F2", 2, 8, 2, 128, 3072, 6, 0.25, synth.QUEST, "mixture",
                                    needles=4, needle_pairs=True, base_seed=52),
    "quest_d64_gqa2": synth.Workload("F3", 1, 6, 3, 64, 2048, 5, 0.4, synth.QUEST, "mixture",
                                     base_seed=53),
    "kmean_d64_mha": synth.Workload("F4", 1, 3, 3, 64, 1344, 3, 0.5, synth.KMEAN, "offset",
                                    base_seed=54),
}


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need an MI355X (gfx950) visible to torch")
    ugbs.lib()


_cache = {}


def case(name):
    if name in _cache:
        return _cache[name]
    w = CASES[name]
    inp = synth.generate(w, threads=8)
    meta = oracle.block_meta(w.backbone, inp.K)
    S = oracle.tile_scores(w.backbone, inp.Q, meta, w.Hkv)
    _cache[name] = dict(w=w, inp=inp, meta=meta, S=S)
    return _cache[name]


def problem(w, k=None, q=None):
    return ugbs.Problem.make(w.B, w.H, w.Hkv, w.N, w.d, w.k if k is None else k,
                             w.q if q is None else q, w.backbone)


def attend_select(p, inp, S, trig):
    torch = __import__("torch")
    Q, K, V = dev_bf16(inp.Q), dev_bf16(inp.K), dev_bf16(inp.V)
    O = torch.empty_like(Q)
    ugbs.ugbs_attend_select(p, Q, K, V, O, scores=dev(S), trigger=dev(np.ascontiguousarray(trig, np.uint8)))
    torch.cuda.synchronize()
    return host_bits(O)


def attend_lists(p, inp, kv):
    torch = __import__("torch")
    Q, K, V = dev_bf16(inp.Q), dev_bf16(inp.K), dev_bf16(inp.V)
    O = torch.empty_like(Q)
    ugbs.ugbs_attend(p, Q, K, V, dev(np.ascontiguousarray(kv, np.int32)), O)
    torch.cuda.synchronize()
    return host_bits(O)


def lists_for(S, k, trig):
    """The oracle's kv_idx for given trigger flags: top-2k rows with the
    expansion slots of untriggered tiles set to the sentinel."""
    idx, _ = oracle.select(S, k)
    kv = idx.copy()
    NB = S.shape[-1]
    B, H, T = S.shape[:3]
    for b in range(B):
        for t in range(T):
            if not trig[b, t]:
                kv[b, :, t, k:] = NB
    return kv


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("mode", ["route", "none", "all"])
def test_given_oracle_scores_and_flags(name, mode):
    c = case(name)
    w, inp, S = c["w"], c["inp"], c["S"]
    p = problem(w)
    if mode == "route":
        idx, sig = oracle.select(S, w.k)
        _, _, _, trig = oracle.route(sig, idx, w.k, w.q)
    else:
        trig = np.full((w.B, w.T), 1 if mode == "all" else 0, np.uint8)
    kv = lists_for(S, w.k, trig)
    got = attend_select(p, inp, S, trig)
    assert np.array_equal(got, attend_lists(p, inp, kv))
    ref = oracle.attend(inp.Q, inp.K, inp.V, kv_idx=kv)
    mx, rms = attention_error(got, ref)
    assert mx <= ATOL_MAX and rms <= ATOL_RMS, (mx, rms)


def test_heavy_ties_and_signed_zeros():
    """Quantised scores (many equal keys at the cut) with -0 and +0 mixed:
    the in-kernel threshold takes equal keys by lower block, as the lists do."""
    c = case("kmean_d64_mha")
    w, inp = c["w"], c["inp"]
    g = np.random.default_rng(6)
    S = (np.round(c["S"] * 2) / 2).astype(np.float32)
    S[np.isfinite(S) & (g.random(S.shape) < 0.3)] = np.float32(-0.0)
    for k in (3, 4, 9):
        p = problem(w, k=k)
        trig = (g.random((w.B, w.T)) < 0.5).astype(np.uint8)
        kv = lists_for(S, k, trig)
        assert np.array_equal(attend_select(p, inp, S, trig), attend_lists(p, inp, kv))


def test_budget_equal_NB_is_dense():
    c = case("quest_d64_gqa2")
    w, inp = c["w"], c["inp"]
    p = problem(w, k=w.NB)
    got = attend_select(p, inp, c["S"], np.zeros((w.B, w.T), np.uint8))
    ref = oracle.attend(inp.Q, inp.K, inp.V, dense=True)
    mx, rms = attention_error(got, ref)
    assert mx <= ATOL_MAX and rms <= ATOL_RMS


def _layers(w, inp, k=None, q=None):
    torch = __import__("torch")
    p = problem(w, k=k, q=q)
    Q, K, V = dev_bf16(inp.Q), dev_bf16(inp.K), dev_bf16(inp.V)
    b1, b2 = ugbs.Buffers(p), ugbs.Buffers(p)
    O1, O2 = torch.empty_like(Q), torch.empty_like(Q)
    ugbs.prefill(p, Q, K, V, O1, b1)
    ugbs.prefill_fused(p, Q, K, V, O2, b2)
    torch.cuda.synchronize()
    return (host_bits(O1), host(b1.sigma), host(b1.trigger), host(b1.tau)), \
           (host_bits(O2), host(b2.sigma), host(b2.trigger), host(b2.tau))


@pytest.mark.parametrize("name", list(CASES))
def test_fused_layer_equals_lists_layer(name):
    c = case(name)
    a, b = _layers(c["w"], c["inp"])
    for x, y in zip(a, b):
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8))


@pytest.mark.parametrize("k,q", [(3, 0.0), (3, 1.0), (20, 0.3), (64, 0.5)])
def test_fused_layer_budgets(k, q):
    c = case("quest_d128_b2")
    a, b = _layers(c["w"], c["inp"], k=k, q=q)
    for x, y in zip(a, b):
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8))


@pytest.mark.parametrize("N", [64, 128, 192, 320])
def test_tiny_sequences(N):
    w = synth.Workload("tiny", 1, 2, 1, 64, N, 3, 0.5, synth.QUEST, "mixture", base_seed=55)
    inp = synth.generate(w, threads=2)
    a, b = _layers(w, inp)
    assert np.array_equal(a[0], b[0])


@pytest.mark.slow
@pytest.mark.parametrize("name", ["C2", "C4", "L8"])
def test_full_size_fused_equals_lists(name):
    """32K, 128K and 256K layers in the benchmark's configuration: the fused
    layer's output, sigma and trigger flags equal the lists layer's bit for
    bit (at 256K the fused kernel holds 64 candidates per lane)."""
    w = synth.WORKLOADS[name]
    inp = synth.generate(w, threads=16)
    a, b = _layers(w, inp)
    for x, y in zip(a, b):
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8))
