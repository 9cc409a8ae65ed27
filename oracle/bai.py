"""Reference oracle for the Appendix D diagnostics (sigma as a best-arm
identification index).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: plain numpy, slow and
literal.  Per (batch, head) it follows the empirical recipe at the end of
Appendix D:

  * per tile, from the candidate scores of C(t) sorted by (score desc, block
    asc): the cutoff gap g, the expansion gap G, the spread r and
    sigma = g / r of Eq. (gaps), with m = k - |F| non-forced kept slots and
    R' = rho k - |F| after expansion (forced blocks excluded, as for sigma);
    the smallest secondary spacing in ranks 0..R' (assumption (A1));
  * Monte Carlo of the identification errors of the empirical top-m and
    top-R' sets under mu ~ N(s, tau^2 I) (Remark on the noise-dominated
    regime), with caller-supplied standard normals shared by all tiles;
  * per head: mean and coefficient of variation of r (the proxy for beta in
    (A2)), the router's empirical quantile sigma_(q) and gamma_q, the band
    mass m_q(beta), spacing quantiles standing in for Delta_2, the closed
    forms chi, eps_bar and C_q of the Lemma and the Proposition, and the
    Monte Carlo regret R_q;
  * the noise scale tau from row-to-row score differences (recipe step 3).

Only tiles with at least rho k + 1 visible blocks (t >= 2k) enter, as in the
paper's diagnostic mask.
"""
import math

import numpy as np

RHO = 2

_F32 = np.float32


def Phi(x):
    """Standard normal CDF."""
    return 0.5 * math.erfc(-x / math.sqrt(2.0))


def phi(x):
    """Standard normal density."""
    return math.exp(-0.5 * x * x) / math.sqrt(2.0 * math.pi)


def vbar(g, tau):
    """Vbar(g) = Phi(-g / (sqrt(2) tau))."""
    return Phi(-g / (math.sqrt(2.0) * tau))


def chi(delta2, tau, max_terms=1_000_000):
    """chi = sum_{m >= 1} (m + 1) exp(-m^2 delta2^2 / (4 tau^2)), summed in
    order up to the last term that does not underflow (m^2 a <= 745); +inf
    when delta2 <= 0 or more than max_terms terms would be needed."""
    if not (delta2 > 0.0) or not (tau > 0.0):
        return math.inf
    a = delta2 * delta2 / (4.0 * tau * tau)
    M = int(math.floor(math.sqrt(745.0 / a)))
    if M > max_terms:
        return math.inf
    s = 0.0
    for m in range(1, M + 1):
        s += (m + 1) * math.exp(-(m * m) * a)
    return s


def eps_bar(delta2, tau, k, rho=RHO):
    c = chi(delta2, tau)
    if math.isinf(c):
        return math.inf
    x = (rho - 1) * k * delta2
    return c + (1.0 + c) * math.exp(-(x * x) / (4.0 * tau * tau))


def C_q(gamma, beta, tau, eb):
    """C_q = min{1, (1 + eps_bar)/2, sqrt2 beta gamma / tau phi(gamma (1-beta) / (sqrt2 tau)) + eps_bar}."""
    band = math.sqrt(2.0) * beta * gamma / tau * phi(gamma * (1.0 - beta) / (math.sqrt(2.0) * tau))
    return min(1.0, (1.0 + eb) / 2.0, band + eb)


def _canon(x):
    x = np.asarray(x, _F32).copy()
    x[x == 0] = _F32(0.0)
    return x


def _sorted_order(c):
    """Positions of the candidates by (score desc, position asc)."""
    return np.lexsort((np.arange(len(c)), -c.astype(np.float64)))


def tile_gaps(scores, k, rho=RHO):
    """scores [B, H, T, N_B] fp32 tile scores (only C(t) = 1..t-1 is read).

    Returns a dict of [B, H, T] arrays: g, G, r, sigma, delta2 (fp32, the
    differences and the division in fp32) and valid (bool, t >= 2k)."""
    scores = np.asarray(scores, _F32)
    B, H, T, NB = scores.shape
    out = {n: np.full((B, H, T), np.nan, _F32) for n in ("g", "G", "r", "sigma", "delta2")}
    out["valid"] = np.zeros((B, H, T), bool)
    for t in range(T):
        nf = 1 if t == 0 else 2
        nc = max(t - 1, 0)
        m = k - nf
        Rp = rho * k - nf
        if nc < Rp + 1 or nc <= m:
            continue
        for b in range(B):
            for h in range(H):
                c = _canon(scores[b, h, t, 1:t])
                cs = c[_sorted_order(c)]
                g = _F32(cs[m - 1] - cs[m])
                G = _F32(cs[m - 1] - cs[Rp])
                r = _F32(cs[0] - cs[m])
                sig = _F32(0.0) if r == 0 else _F32(g / r)
                sp = (cs[:Rp] - cs[1:Rp + 1]).astype(_F32)      # spacings j = 0..Rp-1
                sp = np.delete(sp, m - 1)
                out["g"][b, h, t], out["G"][b, h, t], out["r"][b, h, t] = g, G, r
                out["sigma"][b, h, t] = sig
                out["delta2"][b, h, t] = sp.min() if sp.size else np.nan
                out["valid"][b, h, t] = True
    return out


def mc_counts(scores, k, tau, z, rho=RHO):
    """Identification failures over the samples s = 0..n_s-1 of
    mu_b = fp32(s_b + fp32(tau z[s, b])) for the candidates b in C(t):

      fail_k  : the empirical top-m set (m = k - |F|) does not contain the
                true top-m of mu, i.e. not (min over it of mu > max of mu
                over the other candidates);
      fail_rk : the empirical top-R' set (R' = rho k - |F|) does not contain
                the true top-m, i.e. fewer than m of its members exceed
                every other candidate's mu.

    tau [B, H] fp32, z [n_s, N_B] fp32.  Returns (fail_k, fail_rk) int32
    [B, H, T], zero on tiles outside the diagnostic mask."""
    scores = np.asarray(scores, _F32)
    tau = np.asarray(tau, _F32)
    z = np.asarray(z, _F32)
    B, H, T, NB = scores.shape
    fk = np.zeros((B, H, T), np.int32)
    fr = np.zeros((B, H, T), np.int32)
    for t in range(T):
        nf = 1 if t == 0 else 2
        nc = max(t - 1, 0)
        m = k - nf
        Rp = rho * k - nf
        if nc < Rp + 1 or nc <= m:
            continue
        zt = z[:, 1:t]                                           # [n_s, nc]
        for b in range(B):
            for h in range(H):
                c = _canon(scores[b, h, t, 1:t])
                order = _sorted_order(c)
                in_k = np.zeros(nc, bool)
                in_k[order[:m]] = True
                in_r = np.zeros(nc, bool)
                in_r[order[:Rp]] = True
                mu = (c[None, :] + (tau[b, h] * zt).astype(_F32)).astype(_F32)
                ok_k = mu[:, in_k].min(axis=1) > mu[:, ~in_k].max(axis=1)
                top_out = mu[:, ~in_r].max(axis=1)
                ok_r = (mu[:, in_r] > top_out[:, None]).sum(axis=1) >= m
                fk[b, h, t] = int((~ok_k).sum())
                fr[b, h, t] = int((~ok_r).sum())
    return fk, fr


def noise_scale(rough_sums, terms):
    """Recipe step 3: tau^2 = E[(s_{r+1,b} - s_{r,b})^2] / 2 over adjacent rows.
    rough_sums, terms: per-unit arrays over the units of one (batch, head)."""
    n = float(np.sum(terms))
    return math.sqrt(float(np.sum(rough_sums)) / (2.0 * n)) if n > 0 else math.nan


def head_stats(gaps, fail_k, fail_rk, tau, q, k, n_s, rho=RHO):
    """Per (batch, head) aggregates over the valid tiles (Appendix D).

    tau [B, H]: the noise scale used by the closed forms.  Returns a dict of
    [B, H] float64 arrays (and int n_tiles, n_q)."""
    B, H, T = gaps["g"].shape
    keys = ("r_mean", "r_cv", "sigma_q", "gamma_q", "band_mass", "delta2_p05", "delta2_p50", "pi2",
            "tau", "chi", "eps_bar", "vbar_gamma", "C_q", "bound", "bound_band",
            "mc_err_k", "mc_err_rk", "mc_regret")
    out = {n: np.full((B, H), np.nan) for n in keys}
    out["n_tiles"] = np.zeros((B, H), np.int64)
    out["n_q"] = np.zeros((B, H), np.int64)
    for b in range(B):
        for h in range(H):
            v = gaps["valid"][b, h]
            n = int(v.sum())
            out["n_tiles"][b, h] = n
            if n == 0:
                continue
            ts = np.nonzero(v)[0]
            g = gaps["g"][b, h, ts].astype(np.float64)
            r = gaps["r"][b, h, ts].astype(np.float64)
            sig = gaps["sigma"][b, h, ts]
            d2 = gaps["delta2"][b, h, ts]
            r_mean = sum(r.tolist()) / n
            var = sum(((x - r_mean) ** 2 for x in r.tolist())) / n
            r_cv = math.sqrt(var) / r_mean if r_mean != 0 else math.nan
            nq = math.ceil(q * float(n))
            out["n_q"][b, h] = nq
            out["r_mean"][b, h], out["r_cv"][b, h] = r_mean, r_cv
            d2s = sorted(d2.tolist())
            p05 = d2s[int(math.floor(0.05 * (n - 1)))]
            out["delta2_p05"][b, h] = p05
            out["delta2_p50"][b, h] = d2s[int(math.floor(0.5 * (n - 1)))]
            out["pi2"][b, h] = sum(1 for x in d2.tolist() if x < p05) / n
            tb = float(tau[b, h])
            out["tau"][b, h] = tb
            # Monte Carlo: per-tile errors and V* estimates
            fk = fail_k[b, h, ts].astype(np.float64)
            fr = fail_rk[b, h, ts].astype(np.float64)
            if n_s > 0:
                out["mc_err_k"][b, h] = sum(fk.tolist()) / (n * n_s)
                out["mc_err_rk"][b, h] = sum(fr.tolist()) / (n * n_s)
            if nq == 0:
                continue
            # router set: the nq smallest sigma, lower tile first on ties
            by_sigma = sorted(range(n), key=lambda i: (float(sig[i]), int(ts[i])))
            sq = float(sig[by_sigma[nq - 1]])
            gamma = sq * r_mean
            beta = r_cv
            out["sigma_q"][b, h], out["gamma_q"][b, h] = sq, gamma
            lo, hi = gamma * (1.0 - beta), gamma * (1.0 + beta)
            out["band_mass"][b, h] = sum(1 for x in g.tolist() if lo <= x <= hi) / n
            if tb > 0:
                c = chi(p05, tb)
                eb = eps_bar(p05, tb, k, rho)
                cq = C_q(gamma, beta, tb, eb)
                out["chi"][b, h], out["eps_bar"][b, h], out["C_q"][b, h] = c, eb, cq
                out["vbar_gamma"][b, h] = vbar(gamma, tb)
                out["bound"][b, h] = min(q, 1.0 - q) * cq + out["pi2"][b, h]
                out["bound_band"][b, h] = 0.5 * out["band_mass"][b, h] * cq + out["pi2"][b, h]
            if n_s > 0:
                V = ((fk - fr) / n_s).tolist()
                top = sum(sorted(V, reverse=True)[:nq])
                rsig = sum(V[i] for i in by_sigma[:nq])
                out["mc_regret"][b, h] = (top - rsig) / n
    return out
