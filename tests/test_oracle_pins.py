"""Pins of the reference oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: a closed
form, a library routine (numpy / torch on the CPU), brute force on tiny
inputs, an invariant the paper states, or a hand-derived worked example.
None of these touch the GPU library.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2607_07724_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
BLK = 64


def f32(bits):
    return synth.bf16_to_f32(bits)


def small_inputs(B=1, H=4, Hkv=2, N=512, d=32, seed=7, keys="offset"):
    w = synth.Workload("T", B, H, Hkv, d, N, 3, 0.25, synth.KMEAN, keys, base_seed=seed)
    return synth.generate(w, threads=2)


# ---------------------------------------------------------------- bf16 rounding

def test_bf16_round_matches_numpy_rne_on_float32_values():
    g = np.random.default_rng(0)
    x = np.concatenate([g.standard_normal(20000).astype(np.float32),
                        (g.standard_normal(2000) * 1e-30).astype(np.float32),
                        (g.standard_normal(2000) * 1e30).astype(np.float32)])
    ref = synth.bf16_bits(x)
    got = np.array([oracle.bf16_round(float(v)) for v in x], np.uint16)
    assert np.array_equal(ref, got)


@pytest.mark.parametrize("x,expect", [
    (1.0 + 2.0 ** -8, 1.0),                  # halfway, ties to even (down)
    (1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -6),  # halfway, ties to even (up)
    (1.0 + 2.0 ** -8 + 2.0 ** -40, 1.0 + 2.0 ** -7),  # just above halfway: needs double
    (-(1.0 + 2.0 ** -8 + 2.0 ** -40), -(1.0 + 2.0 ** -7)),
    (0.0, 0.0),
    (-0.0, 0.0),                              # zero is canonical +0
])
def test_bf16_round_closed_cases(x, expect):
    bits = oracle.bf16_round(x)
    assert f32(np.array([bits], np.uint16))[0] == np.float32(expect)
    if expect == 0.0:
        assert bits == 0


# ---------------------------------------------------------------- A.1 metadata

def _nearest_bf16_exact(fr: Fraction) -> int:
    """Brute force: the bf16 bit pattern nearest to an exact rational, ties to even."""
    if fr == 0:
        return 0
    if fr < 0:
        return _nearest_bf16_exact(-fr) ^ 0x8000
    base = int(synth.bf16_bits(np.array([float(fr)], np.float32))[0])
    best = None
    for cand in range(max(0, base - 3), min(0x7F7F, base + 3) + 1):
        v = f32(np.array([cand], np.uint16))[0]
        key = (abs(Fraction(float(v)) - fr), cand & 1)
        if best is None or key < best[0]:
            best = (key, cand)
    return best[1]


def test_kmean_is_exact_mean_rounded_to_nearest_even():
    inp = small_inputs()
    meta = oracle.block_meta(oracle.KMEAN, inp.K)
    Kf = f32(inp.K)
    g = np.random.default_rng(1)
    for _ in range(40):
        b, kvh = 0, int(g.integers(0, inp.K.shape[1]))
        blk, e = int(g.integers(0, inp.K.shape[2] // BLK)), int(g.integers(0, inp.K.shape[3]))
        col = Kf[b, kvh, blk * BLK:(blk + 1) * BLK, e]
        exact = sum(Fraction(float(v)) for v in col) / BLK
        assert meta[b, kvh, blk, 0, e] == _nearest_bf16_exact(exact)


def test_kmean_exact_at_the_widest_exact_exponent_range():
    """The fp64 sum of a channel's 64 bf16 values is exact when their binary
    exponents lie within 39 of each other (8 significant bits plus 6 bits of
    carry in 53): channels mixing magnitudes 2^20 and 2^-19 of both signs,
    whose exact mean needs every low bit, still round to the nearest-even
    bf16 of the exact rational mean."""
    g = np.random.default_rng(12)
    N, d = 2 * BLK, 16
    mant = 1.0 + g.integers(0, 128, (1, 1, N, d)) / 128.0
    expo = np.where(g.random((1, 1, N, d)) < 0.5, 20, -19)
    sign = np.where(g.random((1, 1, N, d)) < 0.5, -1.0, 1.0)
    K = synth.bf16_bits((sign * mant * np.exp2(expo)).astype(np.float32))
    meta = oracle.block_meta(oracle.KMEAN, K)
    Kf = f32(K)
    for blk in range(N // BLK):
        for e in range(d):
            col = Kf[0, 0, blk * BLK:(blk + 1) * BLK, e]
            exact = sum(Fraction(float(v)) for v in col) / BLK
            assert meta[0, 0, blk, 0, e] == _nearest_bf16_exact(exact)


def test_quest_min_max_bound_every_key_and_are_attained():
    inp = small_inputs(keys="mixture")
    meta = oracle.block_meta(oracle.QUEST, inp.K)
    B, Hkv, N, d = inp.K.shape
    Kf = f32(inp.K).reshape(B, Hkv, N // BLK, BLK, d)
    lo, hi = f32(meta[:, :, :, 0]), f32(meta[:, :, :, 1])
    assert np.all(Kf >= lo[:, :, :, None, :]) and np.all(Kf <= hi[:, :, :, None, :])
    assert np.array_equal(lo, Kf.min(axis=3)) and np.array_equal(hi, Kf.max(axis=3))


def test_constant_block_ties_both_backbones():
    inp = small_inputs()
    K = inp.K.copy()
    K[0, 0, 5 * BLK:6 * BLK] = K[0, 0, 5 * BLK]      # block 5 of kv head 0: 64 equal keys
    mk = oracle.block_meta(oracle.KMEAN, K)
    mq = oracle.block_meta(oracle.QUEST, K)
    assert np.array_equal(mk[0, 0, 5, 0], K[0, 0, 5 * BLK])
    assert np.array_equal(mq[0, 0, 5, 0], K[0, 0, 5 * BLK])
    assert np.array_equal(mq[0, 0, 5, 1], K[0, 0, 5 * BLK])
    sk = oracle.tile_scores(oracle.KMEAN, inp.Q, mk, K.shape[1])
    sq = oracle.tile_scores(oracle.QUEST, inp.Q, mq, K.shape[1])
    G = inp.Q.shape[1] // K.shape[1]
    for h in range(G):                # q heads reading kv head 0
        for t in range(6 + 1, K.shape[2] // BLK):
            assert sk[0, h, t, 5] == sq[0, h, t, 5]


# ---------------------------------------------------------------- A.2/A.3 scores

def test_kmean_tile_scores_match_numpy_contraction():
    inp = small_inputs()
    meta = oracle.block_meta(oracle.KMEAN, inp.K)
    S = oracle.tile_scores(oracle.KMEAN, inp.Q, meta, inp.K.shape[1])
    B, H, N, d = inp.Q.shape
    G, T = H // inp.K.shape[1], N // BLK
    Qd = f32(inp.Q).astype(np.float64)
    Md = f32(meta[:, :, :, 0]).astype(np.float64)
    for h in range(H):
        rows = np.einsum("nd,bd->nb", Qd[0, h], Md[0, h // G])          # [N, N_B]
        tile = rows.reshape(T, BLK, T).max(axis=1).astype(np.float32)   # max over 64 rows
        for t in range(T):
            ref = np.full(T, -np.inf, np.float32)
            ref[1:t] = tile[t, 1:t]
            np.testing.assert_allclose(S[0, h, t], ref, rtol=1e-6, atol=0)


def test_quest_scores_upper_bound_rowwise_max_and_equal_split_form():
    inp = small_inputs(keys="mixture", N=384)
    meta = oracle.block_meta(oracle.QUEST, inp.K)
    S = oracle.tile_scores(oracle.QUEST, inp.Q, meta, inp.K.shape[1])
    B, H, N, d = inp.Q.shape
    G, T = H // inp.K.shape[1], N // BLK
    Qd = f32(inp.Q).astype(np.float64)
    Kd = f32(inp.K).astype(np.float64)
    lo = f32(meta[:, :, :, 0]).astype(np.float64)
    hi = f32(meta[:, :, :, 1]).astype(np.float64)
    for h in range(H):
        kv = h // G
        qp, qn = np.maximum(Qd[0, h], 0), np.minimum(Qd[0, h], 0)
        split = qp @ hi[0, kv].T + qn @ lo[0, kv].T                    # [N, N_B]
        exact_max = (Qd[0, h] @ Kd[0, kv].T).reshape(N, T, BLK).max(axis=2)
        assert np.all(split >= exact_max - 1e-9)                        # upper bound, Eq. (quest-score)
        tile = split.reshape(T, BLK, T).max(axis=1).astype(np.float32)
        for t in range(T):
            np.testing.assert_allclose(S[0, h, t, 1:t], tile[t, 1:t], rtol=1e-6, atol=0)
            assert np.all(np.isneginf(S[0, h, t, [0] + list(range(t, T))]))


# ---------------------------------------------------------------- A.4-A.6 selection

def _golden():
    with open(os.path.join(GOLDEN, "worked_examples.json")) as f:
        return json.load(f)["examples"]


@pytest.mark.parametrize("ex", _golden(), ids=lambda e: e["name"])
def test_worked_examples(ex):
    NB, t, k = ex["N_B"], ex["t"], ex["k"]
    row = np.full(NB, -7.0, np.float32)
    row[1:7] = ex["scores_blocks_1_to_6"]
    idx, sig = oracle.select(row[None, :], k, t_of_row=[t])
    assert idx[0].tolist() == ex["idx_sorted"]
    assert sig[0] == np.float32(ex["sigma"])
    T = NB
    # route one tile through both branches: triggered (q=1) and not (q=0)
    sigma = np.full((1, 1, T), -1.0, np.float32)
    isr = np.tile(np.full(2 * k, NB, np.int32), (1, 1, T, 1))
    sigma[0, 0, t] = sig[0]
    isr[0, 0, t] = idx[0]
    for q, key in ((0.0, "kv_idx_not_triggered"), (1.0, "kv_idx_triggered")):
        kv, _, _, _ = oracle.route(sigma, isr, k, q)
        assert kv[0, 0, t].tolist() == ex[key]


def _python_select(row, t, k, NB):
    """Independent second implementation with Python's sorted()."""
    F = [0] if t == 0 else [0, t]
    C = list(range(1, t))
    order = sorted(C, key=lambda b: (-(float(row[b]) + 0.0), b))
    idx = (F + order)[:2 * k]
    idx += [NB] * (2 * k - len(idx))
    m = k - len(F)
    if len(C) <= m:
        return idx, np.float32(-1.0)
    c = [np.float32(row[b]) for b in order]
    num = np.float32(c[m - 1] - c[m])
    den = np.float32(c[0] - c[m])
    return idx, (np.float32(0.0) if den == 0 else np.float32(num / den))


def test_select_matches_python_sorted_with_ties_and_signed_zeros():
    g = np.random.default_rng(3)
    NB = 40
    for trial in range(300):
        k = int(g.integers(3, 12))
        t = int(g.integers(0, NB))
        row = np.round(g.standard_normal(NB) * 2, 1).astype(np.float32)  # many exact ties
        if trial % 5 == 0:
            row[g.integers(0, NB, size=6)] = -0.0
            row[g.integers(0, NB, size=6)] = 0.0
        idx, sig = oracle.select(row[None], k, t_of_row=[t])
        ridx, rsig = _python_select(row, t, k, NB)
        assert idx[0].tolist() == ridx
        assert sig[0] == rsig


def test_select_top_set_is_the_unique_dominating_subset_brute_force():
    g = np.random.default_rng(4)
    NB = 9
    for _ in range(60):
        k = int(g.integers(3, 5))
        t = NB - 1
        row = g.integers(0, 4, size=NB).astype(np.float32)   # heavy ties
        idx, _ = oracle.select(row[None], k, t_of_row=[t])
        C = list(range(1, t))
        R = min(2 * k - 2, len(C))
        kept = set(idx[0, 2:2 + R].tolist())
        winners = []
        for S in itertools.combinations(C, R):
            dropped = [b for b in C if b not in S]
            ok = all((row[a] > row[z]) or (row[a] == row[z] and a < z) for a in S for z in dropped)
            if ok:
                winners.append(set(S))
        assert winners == [kept]
        # kept entries are in (score desc, index asc) order
        seq = idx[0, 2:2 + R].tolist()
        assert all((row[a] > row[b]) or (row[a] == row[b] and a < b) for a, b in zip(seq, seq[1:]))


def test_sigma_range_forced_blocks_and_sentinels_on_real_scores():
    inp = small_inputs(N=1024)
    meta = oracle.block_meta(oracle.KMEAN, inp.K)
    S = oracle.tile_scores(oracle.KMEAN, inp.Q, meta, inp.K.shape[1])
    for k in (3, 4, 6):
        idx, sig = oracle.select(S, k)
        T = S.shape[2]
        for t in range(T):
            rows = idx[0, :, t]
            assert np.all(rows[:, 0] == 0)
            if t > 0:
                assert np.all(rows[:, 1] == t)
            for r in rows:
                valid = r[r != T]
                n_valid = len(valid)
                assert np.all(r[n_valid:] == T)                     # sentinels trailing only
                assert len(set(valid.tolist())) == n_valid           # no duplicates
                assert np.all(valid <= t)                            # causal
            s = sig[0, :, t]
            if oracle.population(T, k)[t]:
                assert np.all((s >= 0) & (s <= 1))
            else:
                assert np.all(s == -1)


def test_sigma_closed_forms():
    # m = 1 (k = 3, t >= 2): sigma = (c0 - c1) / (c0 - c1) = 1 unless c0 == c1
    row = np.array([0, 5, 2, 2, 1, 9, 9, 9], np.float32)
    _, s = oracle.select(row[None], 3, t_of_row=[5])
    assert s[0] == 1.0
    row2 = np.array([0, 5, 5, 2, 1, 9, 9, 9], np.float32)
    _, s2 = oracle.select(row2[None], 3, t_of_row=[5])
    assert s2[0] == 0.0
    # exact tie straddling the cut (m = 2): sigma = 0
    row3 = np.array([0, 7, 3, 3, 1, 0, 9, 9], np.float32)
    _, s3 = oracle.select(row3[None], 4, t_of_row=[6])
    assert s3[0] == 0.0
    # fp32 arithmetic: (c1 - c2) / (c0 - c2) in single precision
    row4 = np.array([0, 1.1, 0.7, 0.3, 0, 0, 0, 0], np.float32)
    _, s4 = oracle.select(row4[None], 4, t_of_row=[4])
    a, b, c = np.float32(1.1), np.float32(0.7), np.float32(0.3)
    assert s4[0] == np.float32(np.float32(b - c) / np.float32(a - c))


def test_planted_exact_duplicate_block_gives_zero_margin():
    w = synth.WORKLOADS["C1"]
    inp = synth.generate(w, threads=2)
    meta = oracle.block_meta(w.backbone, inp.K)
    S = oracle.tile_scores(w.backbone, inp.Q, meta, w.Hkv)
    # blocks 2 and 4 are identical, so their scores tie exactly in every head and tile
    assert np.array_equal(S[0, :, 5:, 2], S[0, :, 5:, 4])
    idx, sig = oracle.select(S, w.k)
    hits = 0
    for h in range(w.H):
        for t in range(5, w.T):
            c = sorted(range(1, t), key=lambda b: (-S[0, h, t, b], b))
            m = w.k - 2
            if {c[m - 1], c[m]} == {2, 4}:
                assert sig[0, h, t] == 0.0
                hits += 1
            row = idx[0, h, t].tolist()
            if 4 in row:                       # lower index first on the exact tie
                assert 2 in row and row.index(2) == row.index(4) - 1
    assert hits > 0


# ---------------------------------------------------------------- A.7-A.9 route

def _pipeline(S, k, q):
    idx, sig = oracle.select(S, k)
    kv, sb, tau, trig = oracle.route(sig, idx, k, q)
    return idx, sig, kv, sb, tau, trig


def test_quantile_trigger_brute_force():
    g = np.random.default_rng(5)
    B, H, T, k = 2, 3, 50, 4
    P = oracle.population(T, k)
    n = int(P.sum())
    for trial in range(40):
        q = float(g.choice([0.0, 0.05, 0.1, 0.25, 0.4, 0.5, 0.9, 1.0, g.random()]))
        sigma = np.round(g.random((B, H, T)), 2 if trial % 2 else 6).astype(np.float32)
        sigma[:, :, ~P] = -1.0
        idx = np.tile(np.arange(2 * k, dtype=np.int32), (B, H, T, 1))
        kv, sb, tau, trig = oracle.route(sigma, idx, k, q)
        n_trig = math.ceil(q * n)
        for b in range(B):
            sbar = np.zeros(T, np.float32)
            for h in range(H):
                sbar = (sbar + sigma[b, h]).astype(np.float32)
            sbar = (sbar / np.float32(H)).astype(np.float32)
            assert np.array_equal(sb[b, P], sbar[P])
            assert np.all(sb[b, ~P] == -1)
            if n_trig == 0:
                assert trig[b].sum() == 0
                continue
            vals = sbar[P]
            # brute force: the smallest threshold v in the population with >= n_trig values <= v
            best = min(v for v in vals if np.sum(vals <= v) >= n_trig)
            assert tau[b] == best
            assert np.array_equal(trig[b].astype(bool), P & (sbar <= best))
            if len(set(vals.tolist())) == len(vals):
                assert trig[b].sum() == n_trig           # |E| = ceil(q T) with distinct values
            for t in range(T):
                for h in range(H):
                    exp_row = idx[b, h, t].copy()
                    if not trig[b, t]:
                        exp_row[k:] = T
                    assert np.array_equal(kv[b, h, t], exp_row)


def _c1_scores():
    w = synth.WORKLOADS["C1"]
    inp = synth.generate(w, threads=2)
    meta = oracle.block_meta(w.backbone, inp.K)
    return w, inp, oracle.tile_scores(w.backbone, inp.Q, meta, w.Hkv)


def test_q0_is_plain_topk_and_q1_is_uniform_2k():
    w, inp, S = _c1_scores()
    T = w.T
    for k in (3, 4):
        idx, sig, kv0, *_ = _pipeline(S, k, 0.0)
        # q = 0: the first k slots of the sorted prefix, then sentinels
        assert np.array_equal(kv0[..., :k], idx[..., :k])
        assert np.all(kv0[..., k:] == T)
        # q = 1 with budget k equals q = 0 with budget 2k (first 2k slots), bit for bit
        _, _, kv1, *_ = _pipeline(S, k, 1.0)
        _, _, kv2k, *_ = _pipeline(S, 2 * k, 0.0)
        assert np.array_equal(kv1, kv2k[..., :2 * k])
        # Observation 1: the top-k prefix is contained in the top-2k prefix
        idx2, _ = oracle.select(S, 2 * k)
        assert np.array_equal(idx[..., :k], idx2[..., :k])


def test_average_kept_blocks_grows_by_one_plus_q():
    # tiles in the population with >= 2k visible blocks and distinct head-mean sigma:
    # total slots over P = k n + k n_trig, i.e. mean k (1 + n_trig / n) -> k (1 + q)
    g = np.random.default_rng(6)
    B, H, T, k = 1, 2, 120, 4
    P = oracle.population(T, k)
    for q in (0.1, 0.25, 0.4, 0.75):
        sigma = g.random((B, H, T)).astype(np.float32)
        S = np.full((B, H, T, T), -np.inf, np.float32)
        for t in range(T):
            S[0, :, t, 1:t] = g.standard_normal((H, max(t - 1, 0)))
        idx, _ = oracle.select(S, k)
        kv, sb, tau, trig = oracle.route(sigma, idx, k, q)
        n = int(P.sum())
        n_trig = math.ceil(q * n)
        assert trig[0].sum() == n_trig
        slots = (kv[0] != T).sum(axis=-1)                         # [H, T]
        V = np.arange(T) + 1                                      # visible blocks of tile t
        expect = np.where(trig[0].astype(bool), np.minimum(2 * k, V), np.minimum(k, V))
        assert np.array_equal(slots, np.broadcast_to(expect, slots.shape))
        big = P & (V >= 2 * k)
        if big.sum() == n:    # every population tile has >= 2k visible blocks
            assert slots[:, P].sum(axis=1).tolist() == [k * n + k * n_trig] * H


def test_average_kept_identity_on_all_population_tiles():
    # T large with the population starting at 2k - 1 visible: choose k such that P has V >= 2k
    g = np.random.default_rng(8)
    B, H, T, k = 1, 3, 200, 3
    P = oracle.population(T, k)
    V = np.arange(T) + 1
    Pbig = P & (V >= 2 * k)
    sigma = g.random((B, H, T)).astype(np.float32)
    S = np.full((B, H, T, T), -np.inf, np.float32)
    for t in range(T):
        S[0, :, t, 1:t] = g.standard_normal((H, max(t - 1, 0)))
    idx, _ = oracle.select(S, k)
    kv, sb, tau, trig = oracle.route(sigma, idx, k, 0.3)
    slots = (kv[0] != T).sum(axis=-1)
    n = int(P.sum())
    n_trig = math.ceil(0.3 * n)
    small = P & ~Pbig
    extra = int(np.sum((np.minimum(2 * k, V) - 2 * k)[small & trig[0].astype(bool)]))
    assert slots[:, P].sum(axis=1).tolist() == [k * n + k * n_trig + extra] * H


# ---------------------------------------------------------------- A.10 attention

def test_dense_oracle_matches_torch_sdpa_cpu():
    torch = pytest.importorskip("torch")
    inp = small_inputs(N=256, d=32, H=4, Hkv=2)
    O = oracle.attend(inp.Q, inp.K, inp.V, dense=True)
    q = torch.from_numpy(f32(inp.Q).astype(np.float64))
    kk = torch.from_numpy(f32(inp.K).astype(np.float64)).repeat_interleave(2, dim=1)
    v = torch.from_numpy(f32(inp.V).astype(np.float64)).repeat_interleave(2, dim=1)
    N = q.shape[2]
    mask = torch.ones(N, N, dtype=torch.bool).tril()
    ref = torch.nn.functional.scaled_dot_product_attention(q, kk, v, attn_mask=mask)
    np.testing.assert_allclose(O, ref.numpy(), rtol=1e-10, atol=1e-10)


def test_budget_equal_NB_reproduces_dense():
    w, inp, S = _c1_scores()
    T = w.T
    idx, sig, kv, sb, tau, trig = _pipeline(S, T, w.q)       # k_budget = N_B: every tile saturated
    assert np.all(sig == -1) and trig.sum() == 0
    Os = oracle.attend(inp.Q, inp.K, inp.V, kv_idx=kv)
    Od = oracle.attend(inp.Q, inp.K, inp.V, dense=True)
    np.testing.assert_array_equal(Os, Od)


def test_sparse_attention_brute_force_mask_matrix():
    inp = small_inputs(N=256, d=16, H=2, Hkv=1)
    T, W = 4, 4
    kv = synth.random_kv_idx(11, 1, 2, T, W, junk=True)
    O = oracle.attend(inp.Q, inp.K, inp.V, kv_idx=kv)
    Qd, Kd, Vd = (f32(x).astype(np.float64) for x in (inp.Q, inp.K, inp.V))
    N, d = Qd.shape[2], Qd.shape[3]
    for h in range(2):
        mask = np.zeros((N, N), bool)
        for t in range(T):
            for blk in kv[0, h, t]:
                if 0 <= blk < T:
                    mask[t * BLK:(t + 1) * BLK, blk * BLK:(blk + 1) * BLK] = True
        mask &= np.tril(np.ones((N, N), bool))
        logits = (Qd[0, h] @ Kd[0, 0].T) / math.sqrt(d)
        logits[~mask] = -np.inf
        p = np.exp(logits - logits.max(axis=1, keepdims=True))
        ref = (p / p.sum(axis=1, keepdims=True)) @ Vd[0, 0]
        np.testing.assert_allclose(O[0, h], ref, rtol=1e-12, atol=1e-12)


def test_attend_units_subset_equals_full():
    inp = small_inputs(N=256, d=16, H=2, Hkv=1)
    kv = synth.random_kv_idx(12, 1, 2, 4, 4)
    full = oracle.attend(inp.Q, inp.K, inp.V, kv_idx=kv)
    units = np.array([[0, 1, 3], [0, 0, 2]], np.int32)
    sub = oracle.attend(inp.Q, inp.K, inp.V, kv_idx=kv[0, [1, 0], [3, 2]], units=units)
    np.testing.assert_array_equal(sub[0], full[0, 1, 3 * BLK:4 * BLK])
    np.testing.assert_array_equal(sub[1], full[0, 0, 2 * BLK:3 * BLK])


# ---------------------------------------------------------------- expansion factor rho

@pytest.mark.parametrize("rho", [1, 3, 4])
def test_rho_expansion(rho):
    """Section 3 step 5 with a general factor: kv_idx rows have rho k slots;
    a triggered tile keeps all of them, the others the first k.  q = 1 with
    budget k equals q = 0 with budget rho k on the first rho k slots; rho = 1
    never expands (kv_idx equals the plain top-k prefix whatever q); the
    sorted prefix of rho k is the prefix of the rho' k list for rho' > rho
    (Observation 1); the mean kept count grows by k (rho - 1) q."""
    w, inp, S = _c1_scores()
    T = w.T
    for k in (3, 4):
        idx, sig = oracle.select(S, k, rho=rho)
        assert idx.shape[-1] == rho * k
        idx8, sig8 = oracle.select(S, k, rho=8)
        assert np.array_equal(idx, idx8[..., :rho * k]) and np.array_equal(sig, sig8)
        kv1, *_ = oracle.route(sig, idx, k, 1.0, rho=rho)
        idxw, _ = oracle.select(S, rho * k, rho=1)
        kvw, *_ = oracle.route(*oracle.select(S, rho * k, rho=1)[::-1], rho * k, 0.0, rho=1)
        assert np.array_equal(kv1, kvw) and np.array_equal(kvw, idxw)
        kvq, _, _, trig = oracle.route(sig, idx, k, 0.3, rho=rho)
        for b in range(w.B):
            for t in range(T):
                keep = rho * k if trig[b, t] else k
                assert np.array_equal(kvq[b, :, t, :keep], idx[b, :, t, :keep])
                assert np.all(kvq[b, :, t, keep:] == T)
        if rho == 1:
            assert np.array_equal(kvq, idx)
    # mean slots over population tiles with >= rho k visible blocks: k (1 + (rho - 1) n_trig / n)
    g = np.random.default_rng(9)
    B, H, T, k = 1, 2, 160, 3
    P = oracle.population(T, k)
    V = np.arange(T) + 1
    sigma = g.random((B, H, T)).astype(np.float32)
    S2 = np.full((B, H, T, T), -np.inf, np.float32)
    for t in range(T):
        S2[0, :, t, 1:t] = g.standard_normal((H, max(t - 1, 0)))
    idx, _ = oracle.select(S2, k, rho=rho)
    kv, _, _, trig = oracle.route(sigma, idx, k, 0.25, rho=rho)
    slots = (kv[0] != T).sum(axis=-1)
    expect = np.where(trig[0].astype(bool), np.minimum(rho * k, V), np.minimum(k, V))
    assert np.array_equal(slots, np.broadcast_to(expect, slots.shape))
    big = P & (V >= rho * k)
    n, n_trig = int(P.sum()), math.ceil(0.25 * int(P.sum()))
    extra = int(np.sum((np.minimum(rho * k, V) - rho * k)[P & ~big & trig[0].astype(bool)]))
    assert slots[:, P].sum(axis=1).tolist() == [k * n + (rho - 1) * k * n_trig + extra] * H


# ---------------------------------------------------------------- per-row selection variant

@pytest.mark.parametrize("backbone", [oracle.KMEAN, oracle.QUEST])
def test_row_scores_are_the_contraction_and_max_to_the_tile_score(backbone):
    inp = small_inputs(keys="mixture", N=384)
    meta = oracle.block_meta(backbone, inp.K)
    R = oracle.row_scores(backbone, inp.Q, meta, inp.K.shape[1])          # [B,H,T,64,T]
    S = oracle.tile_scores(backbone, inp.Q, meta, inp.K.shape[1])
    B, H, N, d = inp.Q.shape
    G, T = H // inp.K.shape[1], N // BLK
    Qd = f32(inp.Q).astype(np.float64)
    for h in range(H):
        kv = h // G
        if backbone == oracle.KMEAN:
            ref = Qd[0, h] @ f32(meta[0, kv, :, 0]).astype(np.float64).T
        else:
            lo, hi = (f32(meta[0, kv, :, i]).astype(np.float64) for i in (0, 1))
            ref = np.maximum(Qd[0, h], 0) @ hi.T + np.minimum(Qd[0, h], 0) @ lo.T
        for t in range(T):
            got = R[0, h, t]
            np.testing.assert_allclose(got[:, 1:t], ref[64 * t:64 * t + 64, 1:t].astype(np.float32),
                                       rtol=1e-6, atol=1e-6)
            assert np.all(np.isneginf(got[:, [0] + list(range(t, T))]))
            # rounding is monotone: max over rows of the rounded scores is the tile score
            if t >= 2:
                assert np.array_equal(got[:, 1:t].max(axis=0), S[0, h, t, 1:t])


def _row_oracle_brute(rows, t, k, rho, trig):
    nf = 1 if t == 0 else 2
    nc = max(t - 1, 0)
    R = min((rho * k if trig else k) - nf, nc)
    keep = {0} | ({t} if t else set())
    for r in range(rows.shape[0]):
        c = list(range(1, t))
        # the kept set is the unique R-subset dominating every dropped candidate
        best = None
        import itertools
        for sub in itertools.combinations(c, R):
            rest = [b for b in c if b not in sub]
            key = lambda b: (float(rows[r, b]) + 0.0, -b)
            if all(key(a) > key(b) for a in sub for b in rest):
                assert best is None
                best = set(sub)
        assert best is not None or R == 0
        keep |= best or set()
    return keep


def test_select_rows_brute_force_ties_and_signed_zeros():
    g = np.random.default_rng(12)
    T = 9
    rows = np.round(g.standard_normal((6, 64, T)) * 1.5).astype(np.float32)
    rows[g.random(rows.shape) < 0.2] = np.float32(-0.0)
    rows[:, 3:, :] = rows[:, :3, :].repeat(21, axis=1)[:, :61, :]      # repeated rows
    ts = np.array([0, 2, 5, 8, 8, 7])
    trig = np.array([0, 1, 0, 0, 1, 1])
    for k, rho in ((3, 2), (4, 2), (3, 3)):
        got = oracle.select_rows(rows, ts, k, rho, trig)
        for u in range(6):
            want = _row_oracle_brute(rows[u, :4], ts[u], k, rho, trig[u])          # 4 distinct rows
            assert set(oracle.bitmap_blocks(got[u], T)) == want, (k, rho, u)


def test_select_rows_on_identical_rows_is_the_tile_selection():
    """All 64 rows equal: each row's ranking is the tile's, so the union is
    the kept prefix of the per-tile kv_idx row (triggered: rho k slots)."""
    g = np.random.default_rng(13)
    T, k = 40, 4
    S = np.full((1, 1, T, T), -np.inf, np.float32)
    for t in range(2, T):
        S[0, 0, t, 1:t] = g.standard_normal(t - 1).astype(np.float32)
    rows = np.repeat(S[0, 0][:, None, :], 64, axis=1)                        # [T, 64, T]
    for rho in (1, 2, 3):
        idx, sig = oracle.select(S, k, rho=rho)
        for trig_val in (0, 1):
            trig = np.full(T, trig_val)
            got = oracle.select_rows(rows, np.arange(T), k, rho, trig)
            for t in range(T):
                width = rho * k if trig_val else k
                want = {int(b) for b in idx[0, 0, t, :width] if b != T}
                assert set(oracle.bitmap_blocks(got[t], T)) == want


def test_select_rows_union_covers_row_argmax_and_tile_top():
    inp = small_inputs(keys="mixture", N=512)
    meta = oracle.block_meta(oracle.QUEST, inp.K)
    R = oracle.row_scores(oracle.QUEST, inp.Q, meta, inp.K.shape[1])
    S = oracle.tile_scores(oracle.QUEST, inp.Q, meta, inp.K.shape[1])
    B, H, T = R.shape[:3]
    units = oracle.all_units(B, H, T)
    rows = R.reshape(-1, 64, T)
    bits = oracle.select_rows(rows, units[:, 2], 3, 2, None)
    idx, _ = oracle.select(S, 3)
    for u, (b, h, t) in enumerate(units):
        got = set(oracle.bitmap_blocks(bits[u], T))
        if t >= 2:
            for r in range(64):
                assert int(np.argmax(rows[u, r, 1:t])) + 1 in got      # every row's best block
            assert int(idx[b, h, t, 2 if t else 1]) in got               # the tile's best candidate
        assert {0, t} <= got and max(got) <= t
    # k >= N_B: every visible block
    bits = oracle.select_rows(rows, units[:, 2], T, 2, None)
    for u, (b, h, t) in enumerate(units):
        assert oracle.bitmap_blocks(bits[u], T) == list(range(t + 1))
