"""Pins of the Appendix D diagnostics oracle (oracle/bai.py) against facts
that do not come from it: brute-force sorting, the C selection oracle's
sigma, closed forms of the noise model (a two-arm identification error is
exactly Vbar(g)), the Lemma's sandwich, the paper's bound on chi, library
normal CDF/PDF and dispersion routines, and exact row differences."""
import math
import statistics

import numpy as np
import pytest

import oracle
from oracle import bai
from paper_2607_07724_amd import synth


def _rand_scores(B, H, T, seed, levels=None):
    g = np.random.default_rng(seed)
    s = g.normal(0, 1, (B, H, T, T)).astype(np.float32)
    if levels:
        s = np.round(s * levels) / levels          # heavy ties
        s[s == 0] = -0.0
    return s.astype(np.float32)


@pytest.mark.parametrize("levels", [None, 3])
def test_tile_gaps_brute_force(levels):
    k = 3
    s = _rand_scores(1, 2, 14, 7, levels)
    got = bai.tile_gaps(s, k)
    for h in range(2):
        for t in range(14):
            nf = 1 if t == 0 else 2
            nc, m, Rp = max(t - 1, 0), k - nf, 2 * k - nf
            valid = nc >= Rp + 1
            assert got["valid"][0, h, t] == valid
            if not valid:
                continue
            c = [float(np.float32(x)) + 0.0 for x in s[0, h, t, 1:t]]   # -0 -> +0
            order = sorted(range(nc), key=lambda i: (-c[i], i))
            cs = [np.float32(c[i]) for i in order]
            g = np.float32(cs[m - 1] - cs[m])
            G = np.float32(cs[m - 1] - cs[Rp])
            r = np.float32(cs[0] - cs[m])
            sig = np.float32(0.0) if r == 0 else np.float32(g / r)
            spac = [np.float32(cs[j] - cs[j + 1]) for j in range(Rp) if j != m - 1]
            assert got["g"][0, h, t] == g and got["G"][0, h, t] == G and got["r"][0, h, t] == r
            assert got["sigma"][0, h, t].view(np.uint32) == sig.view(np.uint32)
            assert got["delta2"][0, h, t] == min(spac)


@pytest.mark.parametrize("levels", [None, 4])
def test_sigma_equals_selection_oracle(levels):
    """The C selection oracle computes sigma separately (A.6)."""
    k = 4
    s = _rand_scores(2, 3, 20, 11, levels)
    got = bai.tile_gaps(s, k)
    _, sig = oracle.select(s, k)
    v = got["valid"]
    assert v.any()
    assert np.array_equal(got["sigma"][v].view(np.uint32), sig[v].view(np.uint32))


def test_gap_invariants():
    s = _rand_scores(1, 4, 40, 3)
    got = bai.tile_gaps(s, 5)
    v = got["valid"]
    g, G, r, sg, d2 = (got[n][v] for n in ("g", "G", "r", "sigma", "delta2"))
    assert np.all(g >= 0) and np.all(G >= g) and np.all(r >= g) and np.all(d2 >= 0)
    assert np.all((sg >= 0) & (sg <= 1))
    # mask = at least rho k + 1 visible blocks
    T = s.shape[2]
    assert np.array_equal(v[0, 0], np.arange(T) >= 2 * 5)


def test_mc_expansion_never_increases_failures():
    """Observation 1 (expansion never harms): on every sample a failure of
    the expanded set is a failure of the top-k set."""
    s = _rand_scores(1, 2, 24, 5)
    z = np.random.default_rng(9).normal(0, 1, (200, 24)).astype(np.float32)
    tau = np.full((1, 2), 0.7, np.float32)
    fk, fr = bai.mc_counts(s, 4, tau, z)
    assert np.all(fr <= fk) and fk.sum() > fr.sum() > 0


def test_mc_two_arm_error_is_vbar():
    """Two contenders for the last kept slot, everything else decided: the
    identification error is P(mu_2 > mu_1) = Phi(-g / (sqrt2 tau)) exactly
    (Lemma, lower bound attained)."""
    k, T = 4, 16                     # m = 2 non-forced slots, R' = 6
    t = T - 1
    tau, gap = 1.0, 0.8
    row = np.full(T, -1e4, np.float32)
    row[1] = 1e4                     # always first
    row[5] = 10.0                    # kept, rank 1
    row[9] = 10.0 - gap              # first excluded, rank 2
    s = np.full((1, 1, T, T), -np.inf, np.float32)
    s[0, 0, t] = row
    n_s = 40000
    z = np.random.default_rng(2024).normal(0, 1, (n_s, T)).astype(np.float32)
    fk, fr = bai.mc_counts(s, k, np.full((1, 1), tau, np.float32), z)
    p = bai.vbar(gap, tau)
    est = fk[0, 0, t] / n_s
    assert abs(est - p) <= 4 * math.sqrt(p * (1 - p) / n_s)
    assert fr[0, 0, t] == 0          # the expanded set holds both contenders


def test_mc_equal_contenders_closed_form():
    """Six contenders with equal scores for m - 1 = 1 free slot (block index
    breaks the tie), the rest decided: the top-k set holds the true winner
    with probability 1/6, the expanded set (ranks 0..5) misses it with
    probability 1/6 (the sixth contender, rank R' = 6, wins)."""
    k, T = 4, 24                     # m = 2, R' = 6
    t = T - 1
    row = np.full(T, -1e4, np.float32)
    row[1] = 1e4
    row[2:8] = 10.0                  # ranks 1..6 by block index
    s = np.full((1, 1, T, T), -np.inf, np.float32)
    s[0, 0, t] = row
    n_s = 36000
    z = np.random.default_rng(31).normal(0, 1, (n_s, T)).astype(np.float32)
    fk, fr = bai.mc_counts(s, k, np.full((1, 1), 1.0, np.float32), z)
    for got, p in ((fk[0, 0, t] / n_s, 5 / 6), (fr[0, 0, t] / n_s, 1 / 6)):
        assert abs(got - p) <= 4 * math.sqrt(p * (1 - p) / n_s)


def test_mc_lemma_sandwich():
    """Equally spaced scores (spacing D) with cutoff gap g: the Lemma gives
    Vbar(g) <= E_k <= Vbar(g) (1 + chi(D))."""
    k, T = 5, 40                     # m = 3
    t = T - 1
    tau, D, gap = 1.0, 2.5, 0.6
    nc = t - 1
    c = np.zeros(nc, np.float64)
    val = 100.0
    for j in range(nc):
        c[j] = val
        val -= gap if j == 2 else D   # rank 2 -> 3 is the cutoff (m - 1 = 2)
    row = np.full(T, -np.inf, np.float32)
    row[1:t] = c.astype(np.float32)
    s = row[None, None, None, :].repeat(T, axis=2)
    s[:, :, :t] = -np.inf
    n_s = 40000
    z = np.random.default_rng(77).normal(0, 1, (n_s, T)).astype(np.float32)
    fk, _ = bai.mc_counts(s, k, np.full((1, 1), tau, np.float32), z)
    est = fk[0, 0, t] / n_s
    lo = bai.vbar(gap, tau)
    hi = lo * (1 + bai.chi(D, tau))
    se = math.sqrt(lo * (1 - lo) / n_s)
    assert lo - 4 * se <= est <= hi + 4 * se


def test_normal_functions_against_library():
    nd = statistics.NormalDist()
    for x in (-6.0, -1.3, 0.0, 0.4, 2.2, 5.0):
        assert abs(bai.Phi(x) - nd.cdf(x)) < 1e-12
        assert abs(bai.phi(x) - nd.pdf(x)) < 1e-15
    assert bai.vbar(0.0, 1.7) == 0.5


@pytest.mark.parametrize("ratio", [2.0, 2.5, 3.0, 5.0])
def test_chi_within_the_papers_bound(ratio):
    """chi <= 2.2 exp(-Delta2^2 / (4 tau^2)) once Delta2 >= 2 tau."""
    tau = 0.8
    d2 = ratio * tau
    c = bai.chi(d2, tau)
    assert c <= 2.2 * math.exp(-d2 * d2 / (4 * tau * tau))
    ref = math.fsum((m + 1) * math.exp(-(m * m) * d2 * d2 / (4 * tau * tau)) for m in range(1, 2000))
    assert abs(c - ref) <= 1e-12 * max(ref, 1e-300)
    assert math.isinf(bai.chi(0.0, tau))


@pytest.mark.parametrize("k", [2, 3, 5])
@pytest.mark.parametrize("tau,d2", [(0.5, 0.3), (1.0, 0.8), (1.0, 0.25)])
def test_eps_bar_tail_term_bounds_expanded_set_error(k, tau, d2):
    """With every secondary spacing d2, the expansion gap is at least
    G = g + (rho - 1) k d2, and the Gaussian tail ratio makes
    Vbar(G) / Vbar(g) <= exp(-((rho - 1) k d2)^2 / (4 tau^2)), the second
    term of eps_bar (divided by 1 + chi)."""
    c = bai.chi(d2, tau)
    term = (bai.eps_bar(d2, tau, k) - c) / (1 + c)
    for g in (0.0, 0.1, 0.3):
        G = g + (bai.RHO - 1) * k * d2
        assert bai.vbar(G, tau) / bai.vbar(g, tau) <= term * (1 + 1e-12)


def test_C_q_limits():
    tau, gamma = 1.0, 0.3
    for d2 in (0.5, 1.0, 3.0):
        eb = bai.eps_bar(d2, tau, k=8)
        assert bai.C_q(gamma, 0.0, tau, eb) == min(1.0, (1 + eb) / 2, eb)   # beta = 0: no band
    # the (1 + eps_bar) / 2 cap active: band term 0.51 + 0.2 > 0.6
    assert bai.C_q(1.0, 0.9, 1.0, 0.2) == 0.6
    eb = bai.eps_bar(60.0, tau, k=8)                   # spacings >> noise: eps_bar ~ 0
    assert eb < 1e-300
    band = math.sqrt(2) * 0.2 * gamma / tau * bai.phi(gamma * 0.8 / (math.sqrt(2) * tau))
    assert abs(bai.C_q(gamma, 0.2, tau, eb) - min(0.5, band)) < 1e-15


def test_head_stats_against_library_and_regret_cases():
    k = 5
    T = 48
    s = _rand_scores(1, 2, T, 21)
    gaps = bai.tile_gaps(s, k)
    assert len(set(gaps["sigma"][0, 0][gaps["valid"][0, 0]].tolist())) > 20
    n_s = 10
    # synthetic MC counts: V* decreasing in sigma for head 0 -> zero regret
    fk = np.zeros((1, 2, T), np.int32)
    fr = np.zeros((1, 2, T), np.int32)
    v = gaps["valid"][0, 0]
    order = np.argsort(gaps["sigma"][0, 0][v], kind="stable")
    ts = np.nonzero(v)[0]
    for rank, i in enumerate(order):
        fk[0, 0, ts[i]] = n_s - min(rank, n_s)
    g2 = np.random.default_rng(4)
    fk[0, 1] = g2.integers(0, n_s + 1, T)
    fr[0, 1] = np.minimum(fk[0, 1], g2.integers(0, n_s + 1, T))
    tau = np.full((1, 2), 0.9)
    for q in (0.1, 0.3, 0.5):
        st = bai.head_stats(gaps, fk, fr, tau, q, k, n_s)
        for h in range(2):
            vv = gaps["valid"][0, h]
            r = gaps["r"][0, h][vv].astype(np.float64).tolist()
            assert abs(st["r_mean"][0, h] - statistics.fmean(r)) < 1e-12
            assert abs(st["r_cv"][0, h] - statistics.pstdev(r) / statistics.fmean(r)) < 1e-12
            n = len(r)
            nq = math.ceil(q * n)
            assert st["sigma_q"][0, h] == sorted(gaps["sigma"][0, h][vv].tolist())[nq - 1]
            assert st["mc_regret"][0, h] >= 0
            assert st["C_q"][0, h] <= 1.0 and st["bound"][0, h] <= min(q, 1 - q) + st["pi2"][0, h]
        assert st["mc_regret"][0, 0] == 0.0


@pytest.mark.parametrize("backbone", [synth.KMEAN, synth.QUEST])
def test_row_roughness_closed_form(backbone):
    """Rows q_r = q_0 + r delta (bf16-exact, positive for Quest so the max
    picks kmax): adjacent per-row scores differ by delta . m_b exactly, so
    the sum is 63 sum_b (delta . m_b)^2."""
    d, N, H, Hkv = 64, 64 * 6, 2, 1
    g = np.random.default_rng(5)
    q0 = g.integers(1, 9, (H, d)).astype(np.float64)
    delta = g.integers(-2, 3, (H, d)).astype(np.float64)
    if backbone == synth.QUEST:
        delta = np.abs(delta)                                  # rows stay positive
    rows = np.arange(64)[None, :, None]
    Qf = np.zeros((1, H, N, d))
    for t in range(N // 64):
        Qf[0, :, 64 * t:64 * (t + 1)] = q0[:, None, :] + rows * delta[:, None, :]
    Q = synth.bf16_bits(Qf.astype(np.float32))
    K = synth.bf16_bits(g.integers(-4, 5, (1, Hkv, N, d)).astype(np.float32))
    meta = oracle.block_meta(backbone, K)
    sums, terms = oracle.row_roughness(backbone, Q, meta, Hkv)
    mv = synth.bf16_to_f32(meta).astype(np.float64)[0, 0]      # [NB, width, d]
    mrow = mv[:, 0] if backbone == synth.KMEAN else mv[:, 1]   # kbar or kmax
    units = oracle.all_units(1, H, N // 64)
    for u, (b, h, t) in enumerate(units):
        want = 63.0 * sum(float(delta[h] @ mrow[blk]) ** 2 for blk in range(1, t))
        assert sums[u] == want
        assert terms[u] == 63 * max(t - 1, 0)
    tau = bai.noise_scale(sums[units[:, 1] == 0], terms[units[:, 1] == 0])
    assert tau >= 0


def test_mc_mu_rounds_product_and_sum_separately():
    """mu = fp32(s + fp32(tau z)): the product is rounded before the add.
    For tau = 0.8647483, z = 0.7718125, s = 0.8033179 the exact value lies
    within half an ulp of 1.4707414 but the twice-rounded one is 1.4707415,
    equal to the kept block's score: a tie, hence an identification failure
    (the kept set must beat every other candidate strictly)."""
    from fractions import Fraction
    f32 = np.float32
    tau, zx, cx = f32(0.8647483), f32(0.7718125), f32(0.8033179)
    exact = Fraction(float(cx)) + Fraction(float(tau)) * Fraction(float(zx))
    one = f32(1.4707414)
    up = np.nextafter(one, f32(2))
    assert abs(exact - Fraction(float(one))) < abs(exact - Fraction(float(up)))  # single rounding: 1.4707414
    S = np.full((1, 1, 8, 8), -np.inf, f32)
    S[0, 0, 6, 1:6] = [up, cx, f32(0.1), f32(0.05), f32(0.0)]
    z = np.zeros((1, 8), f32)
    z[0, 2] = zx
    fk, fr = bai.mc_counts(S, 3, np.array([[tau]], f32), z)
    assert fk[0, 0, 6] == 1 and fr[0, 0, 6] == 0


# ---------------------------------------------------------------- hand-built pins
# The tests below feed the aggregate and estimator functions hand-chosen
# inputs whose outputs follow from the definitions by hand (the expected
# values are literals, derived in the comments), so that a dropped factor, a
# quantile taken one position off, or a band taken on sigma instead of g
# fails.


def test_noise_scale_linear_rows_exact():
    """Recipe step 3 on rows q_r = q_0 + r delta: every adjacent-row
    difference of the score of block b is delta . m_b, for every tile and
    every one of the row pairs, so E[(s_{r+1,b} - s_{r,b})^2] is the mean of
    (delta . m_b)^2 over the (tile, candidate) pairs, and tau^2 is half of
    it.  The expected value is computed from the dot products alone (no
    roughness sums, no per-tile pair count)."""
    d, N, H, Hkv = 64, 64 * 7, 1, 1
    g = np.random.default_rng(17)
    q0 = g.integers(1, 9, (H, d)).astype(np.float64)
    delta = g.integers(-2, 3, (H, d)).astype(np.float64)
    rows = np.arange(64)[None, :, None]
    Qf = np.zeros((1, H, N, d))
    for t in range(N // 64):
        Qf[0, :, 64 * t:64 * (t + 1)] = q0[:, None, :] + rows * delta[:, None, :]
    Q = synth.bf16_bits(Qf.astype(np.float32))
    K = synth.bf16_bits(g.integers(-4, 5, (1, Hkv, N, d)).astype(np.float32))
    meta = oracle.block_meta(synth.KMEAN, K)
    sums, terms = oracle.row_roughness(synth.KMEAN, Q, meta, Hkv)
    kbar = synth.bf16_to_f32(meta).astype(np.float64)[0, 0, :, 0]
    dots = [float(delta[0] @ kbar[b]) ** 2 for b in range(N // 64)]
    pairs = [(t, b) for t in range(N // 64) for b in range(1, t)]      # (tile, candidate)
    want = math.sqrt(sum(dots[b] for _, b in pairs) / len(pairs) / 2.0)
    assert bai.noise_scale(sums, terms) == pytest.approx(want, rel=1e-15)
    # a dropped factor 1/2 would give sqrt(2) times this value
    assert abs(bai.noise_scale(sums, terms) / want - 1.0) < 1e-12


def test_noise_scale_recovers_the_noise_model_tau():
    """Scores s[r, b] = mu_b + tau eps[r, b] with i.i.d. standard normal eps
    (the noise model of Appendix D with a common mean along the rows):
    adjacent differences have variance 2 tau^2, so the estimator returns tau
    up to sampling error (relative standard error 1/sqrt(2 n) for n terms)."""
    tau = 0.37
    g = np.random.default_rng(8)
    n_units, rows, blocks = 40, 64, 30
    sums, terms = [], []
    for _ in range(n_units):
        mu = g.normal(0, 3, blocks)
        s = mu[None, :] + tau * g.normal(0, 1, (rows, blocks))
        dif = np.diff(s, axis=0)
        sums.append(float((dif * dif).sum()))
        terms.append(dif.size)
    n = sum(terms)
    est = bai.noise_scale(np.array(sums), np.array(terms))
    assert abs(est / tau - 1.0) <= 4.0 / math.sqrt(2.0 * n)


def test_tile_gaps_hand_built_tile():
    """k = 4, rho = 2, tile t = 9: F = [0, 9], m = 2 kept candidates, R' = 6.
    Candidates (blocks 1..8) sorted: 20, 17, 16.5, 14, 11, 9, 7.5, 6.5, so
      g = c1 - c2 = 0.5, r = c0 - c2 = 3.5, sigma = 1/7 (fp32 divide),
      G = c1 - c6 = 17 - 7.5 = 9.5   (rank R' - 1 would give 8, R' + 1 10.5),
      spacings j = 0..5 without the cut j = 1: 3, 2.5, 3, 2, 1.5 -> delta2 =
      1.5 (the cut spacing 0.5 and the spacing j = 6 of 1.0 are excluded).
    Tiles 8 (7 candidates = R' + 1) and 9 are in the mask, tile 7 is not."""
    k, T = 4, 10
    s = np.full((1, 1, T, T), -np.inf, np.float32)
    s[0, 0, 9, 1:9] = [11, 16.5, 6.5, 20, 9, 14, 7.5, 17]
    s[0, 0, 8, 1:8] = [1, 2, 3, 4, 5, 6, 7]
    s[0, 0, 7, 1:7] = [1, 2, 3, 4, 5, 6]
    got = bai.tile_gaps(s, k)
    assert got["g"][0, 0, 9] == 0.5 and got["r"][0, 0, 9] == 3.5
    assert got["G"][0, 0, 9] == 9.5
    assert got["sigma"][0, 0, 9] == np.float32(0.5) / np.float32(3.5)
    assert got["delta2"][0, 0, 9] == 1.5
    assert got["valid"][0, 0].tolist() == [False] * 8 + [True, True]
    # tile 8: sorted 7..1, m = 2: g = 6 - 5, G = 6 - 1 (rank 6), r = 7 - 5
    assert (got["g"][0, 0, 8], got["G"][0, 0, 8], got["r"][0, 0, 8]) == (1, 5, 2)


def _hand_built_heads():
    """40 valid tiles (tiles 2..41 of T = 42) with
      r = 1 on the first 20 tiles and 3 on the last 20: mean 2, population
        standard deviation 1, so r_cv = beta = 0.5 exactly;
      sigma_i = j_i / 64 with j_i = 11 i mod 40 (a permutation of 0..39);
      g_i = sigma_i r_i (consistent with sigma = g / r, all exact in fp32);
      delta2_i = (7 i mod 40 + 1) / 128 (a permutation of 1..40 / 128)."""
    n, T = 40, 42
    gaps = {f: np.full((1, 1, T), np.nan, np.float32) for f in ("g", "G", "r", "sigma", "delta2")}
    gaps["valid"] = np.zeros((1, 1, T), bool)
    for i in range(n):
        t = i + 2
        r = 1.0 if i < 20 else 3.0
        j = (11 * i) % 40
        gaps["r"][0, 0, t] = r
        gaps["sigma"][0, 0, t] = j / 64
        gaps["g"][0, 0, t] = j / 64 * r
        gaps["G"][0, 0, t] = j / 64 * r + 1.0
        gaps["delta2"][0, 0, t] = ((7 * i) % 40 + 1) / 128
        gaps["valid"][0, 0, t] = True
    return gaps, n, T


def test_head_stats_hand_built_aggregates():
    """On the hand-built tile set, q = 0.25:
      n_q = ceil(0.25 * 40) = 10, sigma_(q) = the 10th smallest = 9/64,
      gamma_q = 9/64 * r_mean = 18/64 = 0.28125;
      band [gamma (1 - beta), gamma (1 + beta)] = [9/64, 27/64] on g: the
        r = 1 tiles with j in 9..27 (j = 11, 22, 15, 26, 19, 12, 23, 16, 27,
        9: ten) and the r = 3 tiles with 3 j in 9..27, i.e. j in 3..9 (j = 6,
        3, 7: three) -> band mass 13/40 (on sigma it would be 19/40);
      delta2 quantiles at sorted positions floor(0.05 * 39) = 1 and
        floor(0.5 * 39) = 19: 2/128 and 20/128; pi_2 = #(delta2 < 2/128)/40
        = 1/40 (positions 0 or 2 would give 1/128 with pi_2 = 0, or 3/128
        with pi_2 = 2/40)."""
    gaps, n, T = _hand_built_heads()
    fk = np.zeros((1, 1, T), np.int32)
    fr = np.zeros((1, 1, T), np.int32)
    st = bai.head_stats(gaps, fk, fr, np.array([[1.0]]), 0.25, 5, 4)
    assert st["n_tiles"][0, 0] == 40 and st["n_q"][0, 0] == 10
    assert st["r_mean"][0, 0] == 2.0 and st["r_cv"][0, 0] == 0.5
    assert st["sigma_q"][0, 0] == 9 / 64 and st["gamma_q"][0, 0] == 0.28125
    assert st["band_mass"][0, 0] == 13 / 40
    assert st["delta2_p05"][0, 0] == 2 / 128 and st["delta2_p50"][0, 0] == 20 / 128
    assert st["pi2"][0, 0] == 1 / 40
    # Vbar(gamma) = Phi(-gamma / (sqrt2 tau)), against the library CDF
    nd = statistics.NormalDist()
    assert st["vbar_gamma"][0, 0] == pytest.approx(nd.cdf(-0.28125 / math.sqrt(2.0)), rel=1e-12)


def test_head_stats_bound_branches():
    """The Proposition's bound min(q, 1 - q) C_q + pi_2 and the band form
    m_q / 2 C_q + pi_2 in two regimes of the hand-built set:
      tau = 1 (noise-dominated: Delta_2 = 1/64, chi ~ 1e4, eps_bar > 1):
        C_q = 1, bound = 0.25 + 1/40 = 0.275, band bound = 13/80 + 1/40;
      tau = 1e-4 (spacings >> noise: chi = 0, eps_bar = 0, and the band
        term's density is evaluated 994 standard deviations out): C_q = 0,
        both bounds = pi_2 = 1/40."""
    gaps, n, T = _hand_built_heads()
    z = np.zeros((1, 1, T), np.int32)
    st = bai.head_stats(gaps, z, z, np.array([[1.0]]), 0.25, 5, 4)
    assert st["C_q"][0, 0] == 1.0
    assert st["bound"][0, 0] == pytest.approx(0.275, rel=1e-15)
    assert st["bound_band"][0, 0] == pytest.approx(13 / 80 + 1 / 40, rel=1e-15)
    st = bai.head_stats(gaps, z, z, np.array([[1e-4]]), 0.25, 5, 4)
    assert st["chi"][0, 0] == 0.0 and st["eps_bar"][0, 0] == 0.0 and st["C_q"][0, 0] == 0.0
    assert st["bound"][0, 0] == 1 / 40 and st["bound_band"][0, 0] == 1 / 40
    # q = 0.9: min(q, 1 - q) = 0.1, n_q = 36
    st = bai.head_stats(gaps, z, z, np.array([[1.0]]), 0.9, 5, 4)
    assert st["n_q"][0, 0] == 36 and st["sigma_q"][0, 0] == 35 / 64
    assert st["bound"][0, 0] == pytest.approx(0.1 + 1 / 40, rel=1e-14)


def test_head_stats_hand_built_monte_carlo():
    """n_s = 4 samples.  V_t = (fail_k - fail_rk) / n_s.  The router's 10
    tiles (sigma = 0..9/64) get fail_k = fail_rk = 2 (V = 0); the 10 tiles
    with sigma = 30..39/64 get fail_k = 4, fail_rk = 0 (V = 1); the rest 0.
    Regret R_q = (sum of the 10 largest V - sum over the router's tiles) / n
    = (10 - 0) / 40 = 0.25; mc_err_k = (10 * 2 + 10 * 4) / (40 * 4) = 0.375,
    mc_err_rk = 20 / 160 = 0.125."""
    gaps, n, T = _hand_built_heads()
    fk = np.zeros((1, 1, T), np.int32)
    fr = np.zeros((1, 1, T), np.int32)
    for t in range(T):
        if not gaps["valid"][0, 0, t]:
            continue
        j = round(float(gaps["sigma"][0, 0, t]) * 64)
        if j < 10:
            fk[0, 0, t] = fr[0, 0, t] = 2
        elif j >= 30:
            fk[0, 0, t] = 4
    st = bai.head_stats(gaps, fk, fr, np.array([[1.0]]), 0.25, 5, 4)
    assert st["mc_regret"][0, 0] == 0.25
    assert st["mc_err_k"][0, 0] == 0.375 and st["mc_err_rk"][0, 0] == 0.125


@pytest.mark.parametrize("gamma,tau", [(0.3, 1.0), (2.0, 0.7), (0.05, 0.02)])
def test_C_q_band_term_bounds_the_band_width(gamma, tau):
    """The band term of C_q bounds the width of the boundary band in Vbar,
    Vbar(gamma (1 - beta)) - Vbar(gamma (1 + beta)) (proof of the
    Proposition: the slope phi(x / (sqrt2 tau)) / (sqrt2 tau) integrated
    over an interval of length 2 beta gamma), and is tight as beta -> 0.
    With eps_bar = 0 and the other caps inactive, C_q is the band term."""
    nd = statistics.NormalDist()
    for beta in (0.5, 0.1, 1e-4):
        lo = nd.cdf(-gamma * (1 - beta) / (math.sqrt(2.0) * tau))
        hi = nd.cdf(-gamma * (1 + beta) / (math.sqrt(2.0) * tau))
        width = lo - hi
        c = bai.C_q(gamma, beta, tau, 0.0)
        if c < 0.5:                                  # the band branch is the one taken
            assert c >= width * (1 - 1e-12)
            if beta == 1e-4:
                assert c == pytest.approx(width, rel=1e-3)
