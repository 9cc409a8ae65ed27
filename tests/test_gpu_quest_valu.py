"""GPU parity of the vector-ALU Quest scoring (ugbs_quest_scores_valu)
against the oracle's literal max-form tile scores (Eq. (quest-score), A.2-A.3).

The oracle's metadata is uploaded (no other GPU stage feeds these checks).
Each bound term is an exact bf16 x bf16 product, so the only difference from
the fp64 oracle is the fp32 summation of d terms in channel order:
|gpu - oracle| <= d 2^-24 max_r sum_c |q_rc| max(|kmin_c|, |kmax_c|) (plus the
final rounding of the oracle to fp32, which the same bound covers).  The
-inf pattern (entries outside C(t) = {1..t-1}) must match exactly.  The
matrix-core form of ugbs_score_select on the same inputs obeys its own bound
(2d terms), so the two GPU forms differ by at most the sum of both.
"""
import numpy as np
import pytest

import oracle
import paper_2607_07724_amd as ugbs
from paper_2607_07724_amd import synth

from gpu_helpers import bf16_to_f64, dev_bf16, dev_meta, host

pytestmark = pytest.mark.gpu

CASES = {
    "d128_b2_gqa4": synth.Workload("V1", 2, 8, 2, 128, 3072, 6, 0.25, synth.QUEST, "mixture",
                                   needles=4, needle_pairs=True, base_seed=61),
    "d64_gqa2": synth.Workload("V2", 1, 6, 3, 64, 2048, 5, 0.4, synth.QUEST, "offset", base_seed=62),
    "d256_qknorm": synth.Workload("V3", 1, 4, 2, 256, 1536, 4, 0.3, synth.QUEST, "offset",
                                  qk_norm=True, base_seed=63),
    "d128_ragged": synth.Workload("V4", 1, 2, 1, 128, 64 * 69, 4, 0.1, synth.QUEST, "mixture",
                                  base_seed=64),
    "d128_tiny": synth.Workload("V5", 1, 1, 1, 128, 192, 3, 0.0, synth.QUEST, "offset", base_seed=65),
}


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need an MI355X (gfx950) visible to torch")
    ugbs.lib()


def _bound(w, Q, meta, n_terms):
    """n_terms 2^-24 max_r sum_c |q_rc m_bc| per (b, h, t, block), m_bc the
    larger magnitude of (kmin_c, kmax_c)."""
    Qa = np.abs(bf16_to_f64(Q))
    G = w.H // w.Hkv
    out = np.empty((w.B, w.H, w.T, w.NB))
    for b in range(w.B):
        for h in range(w.H):
            Ma = np.abs(bf16_to_f64(meta[b, h // G]))            # [NB, 2, d]
            absterm = Qa[b, h] @ np.maximum(Ma[:, 0], Ma[:, 1]).T  # [N, NB]
            out[b, h] = absterm.reshape(w.T, 64, w.NB).max(axis=1) * n_terms * 2.0 ** -24 + 1e-30
    return out


@pytest.mark.parametrize("name", list(CASES))
def test_valu_scores_within_fp32_summation_bound(name):
    torch = __import__("torch")
    w = CASES[name]
    inp = synth.generate(w, threads=8)
    meta = oracle.block_meta(w.backbone, inp.K)
    S = oracle.tile_scores(w.backbone, inp.Q, meta, w.Hkv)
    p = ugbs.Problem.make(w.B, w.H, w.Hkv, w.N, w.d, w.k, w.q, w.backbone, rho=w.rho)
    Qd, Md = dev_bf16(inp.Q), dev_meta(meta)
    so = torch.full((w.B, w.H, w.T, w.NB), 7.0, dtype=torch.float32, device="cuda")
    ugbs.ugbs_quest_scores_valu(p, Qd, Md, so)
    torch.cuda.synchronize()
    got = host(so)
    fin = np.isfinite(S)
    assert np.array_equal(fin, np.isfinite(got))
    assert np.all(np.isneginf(got[~fin]))
    bound = _bound(w, inp.Q, meta, w.d)
    err = np.zeros(got.shape)
    err[fin] = np.abs(got[fin].astype(np.float64) - S[fin].astype(np.float64))
    assert np.all(err <= bound), float((err / bound).max())

    # the matrix-core form on the same inputs: within the sum of both bounds
    mf = torch.empty_like(so)
    sig = torch.empty((w.B, w.H, w.T), dtype=torch.float32, device="cuda")
    ugbs.ugbs_score_select(p, Qd, Md, None, sig, scores_out=mf)
    torch.cuda.synchronize()
    d = np.zeros(got.shape)
    d[fin] = np.abs(got[fin].astype(np.float64) - host(mf)[fin].astype(np.float64))
    assert np.all(d <= bound + _bound(w, inp.Q, meta, 2 * w.d))


def test_valu_scores_exact_on_integer_inputs():
    """Small-integer queries and keys: every product and partial sum is an
    integer below 2^24, so both GPU forms and the oracle agree exactly."""
    torch = __import__("torch")
    rng = np.random.default_rng(66)
    B, H, Hkv, N, d = 1, 4, 2, 1024, 128
    NB = N // 64

    def ints(shape):
        v = rng.integers(-8, 9, size=shape).astype(np.float32)
        return (v.view(np.uint32) >> 16).astype(np.uint16)      # exact in bf16

    Q, K = ints((B, H, N, d)), ints((B, Hkv, N, d))
    meta = oracle.block_meta(synth.QUEST, K)
    S = oracle.tile_scores(synth.QUEST, Q, meta, Hkv)
    p = ugbs.Problem.make(B, H, Hkv, N, d, 4, 0.25, ugbs.QUEST)
    so = torch.empty((B, H, NB, NB), dtype=torch.float32, device="cuda")
    ugbs.ugbs_quest_scores_valu(p, dev_bf16(Q), dev_meta(meta), so)
    torch.cuda.synchronize()
    got = host(so)
    assert np.array_equal(got, S)
