"""GPU parity over seeded random problem shapes.

Each seed draws one problem -- batch, query / kv heads (any GQA ratio up to
8), head dim 64 / 128 / 256, sequence length 64 .. 64 x 48 (so candidate
counts land on every position of the 16-block metadata chunks), budget k
from 3 to past N_B, expansion factor rho 1..4, q in {0, random, 1}, both
backbones, both key distributions, QK-normed rows at d 256 -- and checks
every stage of the HIP path against the oracle on the same inputs, with the
same rules as the fixed cases: metadata, selection given the oracle's tile
scores and route given the oracle's sigma bit-exact; attention on the
oracle's kv_idx within max-abs 2e-2 / RMS 2e-3; tile scores within the fp32
summation bound of the oracle's; end to end the kept lists
equal the oracle's up to near-ties; the selection inside the attention
kernel gives the lists path's output bit for bit; per-row selection on the
oracle's row scores gives the oracle's tile bitmaps bit for bit, and
attention over those bitmaps and over the same blocks listed both match the
oracle.  A second set of seeds draws longer sequences (49 to 160 blocks), so
the score kernel's metadata ring runs many chunks with a ragged last one
and budgets reach past N_B (selection widths to about a thousand); it skips
the per-row part, whose oracle grows with the square of the tile count.
"""
import numpy as np
import pytest

import oracle
import paper_2607_07724_amd as ugbs
from paper_2607_07724_amd import synth

from gpu_helpers import (attention_error, bf16_to_f64, dev, dev_bf16, dev_meta, host, host_bits,
                         meta_from_gpu, near_tie_ok)

pytestmark = pytest.mark.gpu
ATOL_MAX, ATOL_RMS = 2e-2, 2e-3
N_SEEDS = 32
N_LONG_SEEDS = 8


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need an MI355X (gfx950) visible to torch")
    ugbs.lib()  # raises if the HIP library is missing


def draw(seed: int, long: bool = False) -> synth.Workload:
    g = np.random.default_rng((7300 if long else 7100) + seed)
    Hkv = int(g.choice([1, 2, 4]))
    G = int(g.choice([1, 2, 3, 4, 5, 7, 8]))
    while Hkv * G > (8 if long else 16):
        Hkv //= 2
    while Hkv * G > (8 if long else 16):
        G //= 2
    d = int(g.choice([64, 128, 256]))
    NB = int(g.integers(49, 161)) if long else int(g.integers(1, 49))
    B = int(g.choice([1, 2]))
    k = int(g.integers(3, NB + 5))
    rho = int(g.integers(1, 5))
    q = float(g.choice([0.0, float(g.uniform(0.02, 0.98)), 1.0], p=[0.2, 0.6, 0.2]))
    backbone = int(g.choice([synth.KMEAN, synth.QUEST]))
    if long:  # both backbones; Quest at 97+ blocks (4+ of its 32-block chunks at d 128)
        backbone = synth.QUEST if seed % 2 == 0 else synth.KMEAN
        NB = int(np.random.default_rng(7500 + seed).integers(97 if backbone == synth.QUEST else 49, 161))
        k = int(g.integers(3, NB + 5))
    keys = str(g.choice(["offset", "mixture"]))
    return synth.Workload(f"rand{seed}", B, Hkv * G, Hkv, d, 64 * NB, k, q, backbone, keys,
                          needles=int(g.integers(0, 5)), needle_pairs=bool(g.integers(0, 2)),
                          base_seed=(7400 if long else 7200) + seed, rho=rho,
                          qk_norm=(d == 256 and bool(g.integers(0, 2))))


def problem(w, k=None):
    return ugbs.Problem.make(w.B, w.H, w.Hkv, w.N, w.d, w.k if k is None else k, w.q, w.backbone,
                             rho=w.rho)


def check_tile_scores(w, p, Q, meta, S):
    """GPU tile scores (the full-layout output) within the fp32 summation
    bound of the oracle's: |err| <= KD 2^-24 max_r sum_c |q_rc m_bc|."""
    torch = __import__("torch")
    so = torch.empty((w.B, w.H, w.T, w.NB), dtype=torch.float32, device="cuda")
    gidx = torch.empty((w.B, w.H, w.T, p.W), dtype=torch.int32, device="cuda")
    gsig = torch.empty((w.B, w.H, w.T), dtype=torch.float32, device="cuda")
    ugbs.ugbs_score_select(p, Q, dev_meta(meta), gidx, gsig, scores_out=so)
    torch.cuda.synchronize()
    so = host(so)
    fin = np.isfinite(S)
    assert np.array_equal(fin, np.isfinite(so))
    assert np.all(np.isneginf(so[~fin]))
    KD = w.d * (2 if w.backbone == synth.QUEST else 1)
    G = w.H // w.Hkv
    for b in range(w.B):
        Qa = np.abs(bf16_to_f64(host_bits(Q)[b]))
        for h in range(w.H):
            Ma = np.abs(bf16_to_f64(meta[b, h // G]))
            m = np.maximum(Ma[:, 0], Ma[:, 1]) if w.backbone == synth.QUEST else Ma[:, 0]
            bound = (Qa[h] @ m.T).reshape(w.T, 64, w.NB).max(axis=1) * KD * 2.0 ** -24 + 1e-30
            err = np.abs(so[b, h].astype(np.float64) - S[b, h].astype(np.float64))
            err[~fin[b, h]] = 0
            assert np.all(err <= bound), (b, h, float((err / bound).max()))


@pytest.mark.parametrize("seed", range(N_SEEDS))
def test_random_shape_against_oracle(seed):
    check_against_oracle(draw(seed))


@pytest.mark.parametrize("seed", range(N_LONG_SEEDS))
def test_random_long_shape_against_oracle(seed):
    check_against_oracle(draw(seed, long=True), rows=False)


def check_against_oracle(w, rows=True):
    torch = __import__("torch")
    print(w, flush=True)
    inp = synth.generate(w, threads=8)
    meta = oracle.block_meta(w.backbone, inp.K)
    S = oracle.tile_scores(w.backbone, inp.Q, meta, w.Hkv)
    idx, sig = oracle.select(S, w.k, rho=w.rho)
    kv, sb, tau, trig = oracle.route(sig, idx, w.k, w.q, rho=w.rho)

    p = problem(w)
    Q, K, V = dev_bf16(inp.Q), dev_bf16(inp.K), dev_bf16(inp.V)

    # metadata, bit-exact
    gmeta = torch.empty((w.B, w.Hkv, w.NB, w.d, p.meta_width), dtype=torch.bfloat16, device="cuda")
    ugbs.ugbs_block_meta(p, K, gmeta)
    torch.cuda.synchronize()
    assert np.array_equal(meta_from_gpu(host_bits(gmeta)), meta)

    check_tile_scores(w, p, Q, meta, S)

    # selection on the oracle's tile scores, bit-exact
    gidx = torch.empty((w.B, w.H, w.T, p.W), dtype=torch.int32, device="cuda")
    gsig = torch.empty((w.B, w.H, w.T), dtype=torch.float32, device="cuda")
    ugbs.ugbs_score_select(p, Q, dev_meta(meta), gidx, gsig, scores_in=dev(S))
    torch.cuda.synchronize()
    assert np.array_equal(host(gidx), idx)
    assert np.array_equal(host(gsig).view(np.uint32), sig.view(np.uint32))

    # route on the oracle's sigma and lists, bit-exact
    gkv = torch.full((w.B, w.H, w.T, p.W), -7, dtype=torch.int32, device="cuda")
    gsb = torch.empty((w.B, w.T), dtype=torch.float32, device="cuda")
    gtau = torch.empty((w.B,), dtype=torch.float32, device="cuda")
    gtrig = torch.empty((w.B, w.T), dtype=torch.uint8, device="cuda")
    ws = torch.empty((max(ugbs.ugbs_workspace_bytes(p), 256),), dtype=torch.uint8, device="cuda")
    ugbs.ugbs_route(p, dev(sig), dev(idx), gkv, ws, gsb, gtau, gtrig)
    torch.cuda.synchronize()
    assert np.array_equal(host(gkv), kv)
    assert np.array_equal(host(gsb).view(np.uint32), sb.view(np.uint32))
    assert np.array_equal(host(gtau).view(np.uint32), tau.view(np.uint32))
    assert np.array_equal(host(gtrig), trig)

    # attention on the oracle's kv_idx
    O = torch.empty_like(Q)
    ugbs.ugbs_attend(p, Q, K, V, dev(kv), O)
    torch.cuda.synchronize()
    ref = oracle.attend(inp.Q, inp.K, inp.V, kv_idx=kv)
    mx, rms = attention_error(host_bits(O), ref)
    assert mx <= ATOL_MAX and rms <= ATOL_RMS, (mx, rms)

    # end to end: kept lists equal the oracle's up to near-ties
    bufs = ugbs.Buffers(p)
    O2 = torch.empty_like(Q)
    ugbs.prefill(p, Q, K, V, O2, bufs)
    torch.cuda.synchronize()
    ekv, etrig = host(bufs.kv_idx), host(bufs.trigger)
    for b in range(w.B):
        for t in range(w.T):
            if bool(etrig[b, t]) != bool(trig[b, t]):
                assert abs(float(sb[b, t]) - float(tau[b])) <= 1e-3, (b, t)
            for h in range(w.H):
                width = w.rho * w.k if etrig[b, t] else w.k
                orow = idx[b, h, t].copy()
                orow[width:] = w.NB
                ok, _ = near_tie_ok(ekv[b, h, t], orow, S[b, h, t], t, w.NB, w.k)
                assert ok, (b, h, t, ekv[b, h, t], orow)

    # the selection inside the attention kernel: same output as the lists path
    O3 = torch.empty_like(Q)
    ugbs.prefill_fused(p, Q, K, V, O3, ugbs.Buffers(p))
    torch.cuda.synchronize()
    assert np.array_equal(host_bits(O3), host_bits(O2))

    if not rows:
        return
    # per-row selection on the oracle's row scores, then attention over the bitmaps
    rows = oracle.row_scores(w.backbone, inp.Q, meta, w.Hkv)               # [B,H,T,64,T]
    units = oracle.all_units(w.B, w.H, w.T)
    tu = np.array([trig[b, t] for b, h, t in units], np.uint8)
    obits = oracle.select_rows(rows.reshape(-1, 64, w.T), units[:, 2], w.k, w.rho, tu)
    obits = obits.reshape(w.B, w.H, w.T, -1)
    bm = torch.full((w.B, w.H, w.T, ugbs.bitmap_words(p)), -1, dtype=torch.int32, device="cuda")
    rs = np.ascontiguousarray(rows.reshape(w.B, w.H, w.T * 64, w.T))
    ugbs.ugbs_select_rows(p, dev(trig), bm, row_scores=dev(rs))
    torch.cuda.synchronize()
    assert np.array_equal(host(bm).view(np.uint32), obits)
    lists = np.full((w.B, w.H, w.T, w.NB), w.NB, np.int32)
    for b in range(w.B):
        for h in range(w.H):
            for t in range(w.T):
                blocks = oracle.bitmap_blocks(obits[b, h, t], w.NB)
                lists[b, h, t, :len(blocks)] = blocks
    O4, O5 = torch.empty_like(Q), torch.empty_like(Q)
    ugbs.ugbs_attend_bitmap(p, Q, K, V, dev(obits.view(np.int32)), O4)
    ugbs.ugbs_attend(p, Q, K, V, dev(lists), O5)
    torch.cuda.synchronize()
    ref = oracle.attend(inp.Q, inp.K, inp.V, kv_idx=lists)
    for got in (host_bits(O4), host_bits(O5)):  # same blocks, own visiting orders
        mx, rms = attention_error(got, ref)
        assert mx <= ATOL_MAX and rms <= ATOL_RMS, (mx, rms)
