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
