"""Helpers for the GPU parity tests: host<->device transfer of bf16 bit
patterns, and the comparison rules that allow near-tie differences."""
import numpy as np

BLK = 64


def torch():
    import torch as _t
    return _t


def dev_bf16(a: np.ndarray):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(t.bfloat16)


def dev(a: np.ndarray):
    return torch().from_numpy(np.ascontiguousarray(a)).cuda()


def host_bits(x) -> np.ndarray:
    return x.view(torch().int16).cpu().numpy().view(np.uint16)


def host(x) -> np.ndarray:
    return x.cpu().numpy()


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def attention_error(gpu_bits: np.ndarray, ref: np.ndarray):
    """max-abs and RMS error of bf16 GPU output against an fp64 reference."""
    g = bf16_to_f64(gpu_bits)
    d = g - ref
    return float(np.abs(d).max()), float(np.sqrt(np.mean(d * d)))


def kept_prefix(row: np.ndarray, NB: int):
    v = row[row != NB]
    return [int(x) for x in v]


def near_tie_ok(gpu_row, orc_row, orc_scores, t, NB, rel=1e-3):
    """A kept list may differ from the oracle's only through near-ties: every
    block in the symmetric difference has an oracle score within `rel`
    (relative to max(|s_b|, |s_cut|, spread)) of the oracle's last kept score.
    Returns (ok, n_differing_blocks)."""
    g, o = kept_prefix(gpu_row, NB), kept_prefix(orc_row, NB)
    if g == o:
        return True, 0
    nf = 1 if t == 0 else 2
    if g[:nf] != o[:nf] or len(g) != len(o):
        return False, -1
    diff = set(g) ^ set(o)
    if not diff:                     # same set, order differs inside near-equal scores
        gs = [orc_scores[b] for b in g[nf:]]
        # order must be non-increasing in oracle scores up to the tolerance
        spread = max(abs(orc_scores[o[nf]] - orc_scores[o[-1]]), 1e-30)
        ok = all(b2 <= b1 + rel * max(abs(b1), abs(b2), spread) for b1, b2 in zip(gs, gs[1:]))
        return ok, 0
    cand = o[nf:]
    s_cut = orc_scores[cand[-1]]
    spread = orc_scores[cand[0]] - s_cut
    for b in diff:
        if b in (0, t):
            return False, -1
        s = orc_scores[b]
        if abs(s - s_cut) > rel * max(abs(s), abs(s_cut), spread, 1e-30):
            return False, -1
    return True, len(diff)
