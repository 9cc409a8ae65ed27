"""The end-to-end comparison rule (oracle/compare.py): a GPU kept list may
differ from the oracle's only where oracle scores are within a relative 1e-3
(scale max(|s_a|, |s_b|, r_t), r_t = c_0 - c_m), slot by slot."""
import numpy as np

import oracle
from oracle.compare import near_tie_ok

NB = 16
T = 12      # tile 11: F = [0, 11], candidates 1..10


def _scores(vals):
    s = np.full(NB, -np.inf)
    s[1:11] = vals
    return s


def _row(blocks, width):
    r = np.full(width, NB, np.int32)
    r[:len(blocks)] = blocks
    return r


def _oracle_row(s, k, width):
    idx, _ = oracle.select(s.astype(np.float32)[None, None, None, :], k, t_of_row=np.array([11]))
    r = idx.reshape(-1)[:width].copy()
    return r


def test_equal_lists_pass():
    s = _scores([5, 9, 1, 7, 3, 8, 2, 6, 4, 0.5])
    o = _oracle_row(s, 4, 8)
    assert near_tie_ok(o, o, s, 11, NB, 4) == (True, 0)


def test_near_tie_at_the_cut_passes_and_counts():
    # blocks 2 and 6 nearly tied at the last kept slot of k = 4 (m = 2)
    s = _scores([1, 9.0, 2, 3, 4, 8.9995, 10, 0.5, 0.4, 0.3])
    o = _oracle_row(s, 4, 4)                              # [0, 11, 7, 2]
    assert o.tolist() == [0, 11, 7, 2]
    ok, n = near_tie_ok(_row([0, 11, 7, 6], 4), o, s, 11, NB, 4)
    assert ok and n == 1


def test_swap_across_rank_k_fails_even_with_a_near_tie_at_2k():
    """Same kept set at width 2k except a near-tie in the last slot, but two
    blocks with a real gap swapped across rank k: the non-triggered list and
    sigma would differ, so the row fails."""
    s = _scores([9, 8, 7, 6, 5, 4.0, 3.9995, 1, 0.5, 0])
    o = _oracle_row(s, 4, 8)
    assert o.tolist() == [0, 11, 1, 2, 3, 4, 5, 6]
    g = _row([0, 11, 1, 3, 2, 4, 5, 7], 8)               # 2 <-> 3 swapped, 7 for 6 (near-tie)
    assert near_tie_ok(g, o, s, 11, NB, 4)[0] is False
    g_ok = _row([0, 11, 1, 2, 3, 4, 5, 7], 8)
    assert near_tie_ok(g_ok, o, s, 11, NB, 4) == (True, 1)


def test_real_gap_fails_forced_and_length_checked():
    s = _scores([9, 8, 7, 6, 5, 4, 3, 2, 1, 0])
    o = _oracle_row(s, 4, 4)
    assert near_tie_ok(_row([0, 11, 1, 3], 4), o, s, 11, NB, 4)[0] is False      # 8 vs 7: real gap
    assert near_tie_ok(_row([11, 0, 1, 2], 4), o, s, 11, NB, 4)[0] is False      # forced order
    assert near_tie_ok(_row([0, 11, 1], 4), o, s, 11, NB, 4)[0] is False         # length
    assert near_tie_ok(_row([0, 11, 1, 1], 4), o, s, 11, NB, 4)[0] is False      # duplicate
    assert near_tie_ok(_row([0, 11, 1, 12], 4), o, s, 11, NB, 4)[0] is False     # not a candidate


def test_any_list_sorted_on_perturbed_scores_passes():
    """If every GPU score is within eps of the oracle's, the j-th largest of
    each differ by at most eps, so slot-wise oracle scores differ by <= 2 eps:
    a GPU list sorted on perturbed scores always passes when 2 eps is within
    the tolerance."""
    g = np.random.default_rng(3)
    for trial in range(300):
        base = g.normal(0, 1, 10)
        if trial % 3 == 0:
            base = np.round(base * 4) / 4                 # many exact ties
        s = _scores(base.astype(np.float32).astype(np.float64))
        c = np.sort(s[1:11])[::-1]
        k = int(g.integers(3, 8))
        scale = max(float(c[0] - c[k - 2]), 1e-6)
        eps = 0.4e-3 * scale
        sp = s.copy()
        sp[1:11] += g.uniform(-eps, eps, 10)
        width = 2 * k
        o = _oracle_row(s, k, width)
        gr = _oracle_row(sp, k, width)
        ok, _ = near_tie_ok(gr, o, s, 11, NB, k)
        assert ok, (trial, s, sp, o, gr)
