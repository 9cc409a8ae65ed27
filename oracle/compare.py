"""Comparison rules between a GPU result and the oracle's (test
infrastructure, used by ``tests/`` and the CPU-baseline leg of ``bench.py``).

End to end, the GPU's scores carry fp32 rounding, so a kept list may differ
from the oracle's where two blocks' oracle scores are within a relative
1e-3 of each other.  The rule checks the two sorted lists position by
position: for every slot j, the oracle scores of the GPU's block and of the
oracle's block at slot j must agree within

    |s_a - s_b| <= rel * max(|s_a|, |s_b|, r_t),   r_t = c_0 - c_m,

where c is the tile's candidate scores sorted descending (the oracle's) and
m = k - |F| is the number of kept candidates (r_t is the denominator of
sigma, Eq. (sigma-def): the score scale of the tile; it keeps the rule
meaningful where the scores themselves cross zero).  If every GPU score is
within eps of the oracle's, the j-th largest of each differ by at most eps,
so a correct GPU list passes with rel * scale >= 2 eps.  The rule implies
that blocks in one set but not the other score within the tolerance of the
oracle's cut, and that shared blocks keep the oracle's order up to the
tolerance (a swap across rank k with a real score gap fails at slot k).
"""
import numpy as np


def kept(row, NB):
    """The non-sentinel entries of a kv_idx / idx_sorted row, in order."""
    return [int(x) for x in row if int(x) != NB]


def near_tie_ok(gpu_row, orc_row, orc_scores, t, NB, k, rel=1e-3):
    """Return (ok, n_differing_slots) for one (b, h, t) row.

    gpu_row, orc_row: sorted kept lists padded with NB (the same width);
    orc_scores: the oracle's tile scores of this unit ([N_B], C(t) read);
    k: the budget (m = k - |F| fixes r_t)."""
    g, o = kept(gpu_row, NB), kept(orc_row, NB)
    if g == o:
        return True, 0
    nf = 1 if t == 0 else 2
    if g[:nf] != o[:nf] or len(g) != len(o):
        return False, -1
    cand_g, cand_o = g[nf:], o[nf:]
    if len(set(cand_g)) != len(cand_g) or any(not (1 <= b < t) for b in cand_g):
        return False, -1
    s = np.asarray(orc_scores, np.float64)
    c = np.sort(s[1:t])[::-1]
    m = k - nf
    r_t = float(c[0] - c[m]) if 0 <= m < len(c) else 0.0
    n_diff = 0
    for a, b in zip(cand_g, cand_o):
        if a == b:
            continue
        sa, sb = float(s[a]), float(s[b])
        if abs(sa - sb) > rel * max(abs(sa), abs(sb), r_t, 1e-30):
            return False, -1
        n_diff += 1
    return True, n_diff
