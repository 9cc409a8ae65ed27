"""GPU parity of the Appendix D diagnostics against oracle/bai.py and the
roughness oracle.

Inputs of every GPU call come from the seeded generators or from the
oracle, never from another GPU call:
  - per-tile gaps, spacings and Monte Carlo failure counts, given the
    oracle's tile scores, tau and shared normals: bit-exact (same fp32
    subtract / divide, same mu = fp32(s + fp32(tau z)), same key order);
  - per-head aggregates, given the oracle's tile scores: counts, means,
    order statistics and Monte Carlo rates exact; r_cv within 1e-14
    relative; the closed forms (exp, erfc, a reordered chi sum) within 1e-9
    relative;
  - row roughness: exact on integer-valued rows (every product, difference
    and partial sum is an exact fp32 integer), within 1e-4 relative on
    Gaussian inputs (fp32 scores against fp64), and tau likewise.
The chain through ugbs_score_select's scores_out is checked for internal
consistency only (the tile kernel's sigma equals the selection kernel's).
"""
import math

import numpy as np
import pytest

import oracle
from oracle import bai
import paper_2607_07724_amd as ugbs
from paper_2607_07724_amd import synth

from gpu_helpers import dev, dev_bf16, dev_meta, host

pytestmark = pytest.mark.gpu

CASES = {
    "C1": synth.WORKLOADS["C1"],
    "kmean_d128_gqa4": synth.Workload("B1", 1, 8, 2, 128, 4096, 8, 0.1, synth.KMEAN, "offset",
                                      needles=4, base_seed=41),
    "quest_d64_b2": synth.Workload("B2", 2, 4, 2, 64, 3072, 5, 0.25, synth.QUEST, "mixture",
                                   needles=4, needle_pairs=True, base_seed=42),
    "quest_d128_k3": synth.Workload("B3", 1, 4, 1, 128, 2048, 3, 0.5, synth.QUEST, "offset",
                                    dup_pairs=True, base_seed=43),
}
N_S = 64


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
    sums, terms = oracle.row_roughness(w.backbone, inp.Q, meta, w.Hkv)
    units = oracle.all_units(w.B, w.H, w.T)
    tau = np.zeros((w.B, w.H), np.float64)
    for b in range(w.B):
        for h in range(w.H):
            sel = (units[:, 0] == b) & (units[:, 1] == h)
            tau[b, h] = bai.noise_scale(sums[sel], terms[sel])
    z = synth.mc_normals(w.seed(), N_S, w.NB)
    r = dict(w=w, inp=inp, meta=meta, S=S, rough=sums.reshape(w.B, w.H, w.T), tau=tau,
             tau32=tau.astype(np.float32), z=z)
    _cache[name] = r
    return r


def problem(w, k=None, q=None):
    return ugbs.Problem.make(w.B, w.H, w.Hkv, w.N, w.d, w.k if k is None else k,
                             w.q if q is None else q, w.backbone)


def gpu_tiles(p, S, tau32, z):
    torch = __import__("torch")
    tiles = torch.empty((p.batch * p.n_heads * p.T * ugbs.BAI_TILE_BYTES,), dtype=torch.uint8,
                        device="cuda")
    ugbs.ugbs_bai_tiles(p, dev(S), tiles, tau=dev(tau32) if tau32 is not None else None,
                        z=dev(synth.block_major(z)) if z is not None else None)
    torch.cuda.synchronize()
    return tiles, ugbs.bai_tile_records(tiles).reshape(p.batch, p.n_heads, p.T)


def gpu_heads(p, tiles, tau32, n_s):
    torch = __import__("torch")
    heads = torch.empty((p.batch * p.n_heads * ugbs.BAI_HEAD_BYTES,), dtype=torch.uint8, device="cuda")
    ugbs.ugbs_bai_heads(p, tiles, dev(tau32), n_s, heads)
    torch.cuda.synchronize()
    return ugbs.bai_head_records(heads).reshape(p.batch, p.n_heads)


def same_f32(a, b):
    """Bitwise equal fp32 arrays, NaN positions included."""
    a = np.asarray(a, np.float32)
    b = np.asarray(b, np.float32)
    return np.array_equal(np.isnan(a), np.isnan(b)) and np.array_equal(
        a[~np.isnan(a)].view(np.uint32), b[~np.isnan(b)].view(np.uint32))


def check_tiles(rec, S, k, tau32, z):
    ref = bai.tile_gaps(S, k)
    assert np.array_equal(rec["valid"].astype(bool), ref["valid"])
    for f in ("g", "G", "r", "sigma", "delta2"):
        assert same_f32(rec[f], ref[f]), f
    n_s = 0 if z is None else z.shape[0]
    if n_s:
        fk, fr = bai.mc_counts(S, k, tau32, z)
    else:
        fk = fr = np.zeros(S.shape[:3], np.int32)
    assert np.array_equal(rec["fail_k"], fk)
    assert np.array_equal(rec["fail_rk"], fr)
    return ref, fk, fr


# ---------------------------------------------------------------- tiles

@pytest.mark.parametrize("name", list(CASES))
def test_tiles_given_oracle_scores_bit_exact(name):
    c = case(name)
    w = c["w"]
    for k in sorted({3, w.k, w.k + 2}):
        p = problem(w, k=k)
        _, rec = gpu_tiles(p, c["S"], c["tau32"], c["z"])
        ref, fk, fr = check_tiles(rec, c["S"], k, c["tau32"], c["z"])
        if ref["valid"].any():
            assert (fk >= fr).all() and fk.max() > 0   # the MC sees failures at this noise level


def test_tiles_heavy_ties_and_signed_zeros():
    """Scores on a coarse grid (many equal scores, zero spacings and zero
    cutoff gaps), with -0 and +0 mixed: the same key order on both sides."""
    B, H, T = 1, 3, 40
    g = np.random.default_rng(8)
    S = g.integers(-3, 4, (B, H, T, T)).astype(np.float32) * np.float32(0.5)
    S[g.random(S.shape) < 0.2] = np.float32(-0.0)
    S[..., 0] = -np.inf
    for t in range(T):
        S[:, :, t, max(t, 1):] = -np.inf
    tau32 = np.full((B, H), 0.3, np.float32)
    z = synth.mc_normals(5, 32, T)
    for k in (3, 4, 7):
        p = ugbs.Problem.make(B, H, 1, 64 * T, 64, k, 0.3)
        tiles, rec = gpu_tiles(p, S, tau32, z)
        ref, fk, fr = check_tiles(rec, S, k, tau32, z)
        hd = gpu_heads(p, tiles, tau32, 32)
        st = bai.head_stats(ref, fk, fr, tau32, 0.3, k, 32)
        compare_heads(hd, st)


def test_tiles_without_samples_and_without_valid_tiles():
    c = case("C1")
    w = c["w"]
    p = problem(w)
    tiles, rec = gpu_tiles(p, c["S"], None, None)
    check_tiles(rec, c["S"], w.k, None, None)
    assert (rec["fail_k"] == 0).all()
    hd = gpu_heads(p, tiles, c["tau32"], 0)
    assert np.isnan(hd["mc_err_k"]).all() and np.isnan(hd["mc_regret"]).all()
    # k so large that no tile has rho k + 1 visible blocks
    p = problem(w, k=w.T // 2 + 1)
    tiles, rec = gpu_tiles(p, c["S"], c["tau32"], c["z"])
    assert not rec["valid"].any() and np.isnan(rec["sigma"]).all()
    hd = gpu_heads(p, tiles, c["tau32"], N_S)
    assert (hd["n_tiles"] == 0).all() and (hd["n_q"] == 0).all()
    for f in ("r_mean", "sigma_q", "chi", "C_q", "mc_err_k"):
        assert np.isnan(hd[f]).all()


# ---------------------------------------------------------------- heads

EXACT = ("r_mean", "sigma_q", "gamma_q", "band_mass", "delta2_p05", "delta2_p50", "pi2", "tau",
         "mc_err_k", "mc_err_rk", "mc_regret")
CLOSED = ("chi", "eps_bar", "vbar_gamma", "C_q", "bound", "bound_band")


def _close(a, b, rel):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    same_special = np.array_equal(np.isnan(a), np.isnan(b)) and np.array_equal(np.isinf(a), np.isinf(b))
    fin = np.isfinite(a) & np.isfinite(b)
    return same_special and np.all(np.abs(a[fin] - b[fin]) <= rel * np.abs(b[fin]) + 1e-300) and \
        np.array_equal(a[np.isinf(a)], b[np.isinf(b)])


def compare_heads(hd, st):
    assert np.array_equal(hd["n_tiles"], st["n_tiles"])
    assert np.array_equal(hd["n_q"], st["n_q"])
    for f in EXACT:
        a, b = hd[f], st[f]
        assert np.array_equal(np.isnan(a), np.isnan(b)), f
        assert np.array_equal(a[~np.isnan(a)], b[~np.isnan(b)]), (f, a, b)
    assert _close(hd["r_cv"], st["r_cv"], 1e-14)
    for f in CLOSED:
        assert _close(hd[f], st[f], 1e-9), (f, hd[f], st[f])


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("q", [0.05, 0.25, 1.0])
@pytest.mark.parametrize("tau_scale", [1.0, 1e-2, 1e-4])
def test_heads_given_oracle_scores(name, q, tau_scale):
    """tau_scale < 1 shrinks the measured noise scale so that chi is a
    finite sum of tens to thousands of terms and C_q drops below 1."""
    c = case(name)
    w = c["w"]
    p = problem(w, q=q)
    tau32 = (c["tau32"] * np.float32(tau_scale)).astype(np.float32)
    tiles, rec = gpu_tiles(p, c["S"], tau32, c["z"])
    ref, fk, fr = check_tiles(rec, c["S"], w.k, tau32, c["z"])
    hd = gpu_heads(p, tiles, tau32, N_S)
    st = bai.head_stats(ref, fk, fr, tau32, q, w.k, N_S)
    compare_heads(hd, st)


def test_heads_with_q_zero_and_nonpositive_tau():
    c = case("kmean_d128_gqa4")
    w = c["w"]
    p = problem(w, q=0.0)
    tau32 = c["tau32"].copy()
    tau32[0, 1] = 0.0
    tiles, rec = gpu_tiles(p, c["S"], c["tau32"], c["z"])
    ref, fk, fr = check_tiles(rec, c["S"], w.k, c["tau32"], c["z"])
    hd = gpu_heads(p, tiles, tau32, N_S)
    compare_heads(hd, bai.head_stats(ref, fk, fr, tau32, 0.0, w.k, N_S))
    assert (hd["n_q"] == 0).all() and np.isnan(hd["sigma_q"]).all()
    p = problem(w, q=0.3)
    hd = gpu_heads(p, tiles, tau32, N_S)
    st = bai.head_stats(ref, fk, fr, tau32, 0.3, w.k, N_S)
    compare_heads(hd, st)
    assert np.isnan(hd["chi"][0, 1]) and not np.isnan(hd["chi"][0, 0])


# ---------------------------------------------------------------- noise scale

def gpu_noise(p, Q, meta_np):
    torch = __import__("torch")
    rough = torch.empty((p.batch, p.n_heads, p.T), dtype=torch.float64, device="cuda")
    tau = torch.empty((p.batch, p.n_heads), dtype=torch.float32, device="cuda")
    ugbs.ugbs_noise_scale(p, Q, dev_meta(meta_np), rough, tau)
    torch.cuda.synchronize()
    return host(rough), host(tau)


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("backbone", [synth.KMEAN, synth.QUEST])
def test_noise_scale_against_oracle(name, backbone):
    c = case(name)
    w = c["w"].replace(backbone=backbone)
    p = problem(w)
    meta = oracle.block_meta(backbone, c["inp"].K)
    sums, terms = oracle.row_roughness(backbone, c["inp"].Q, meta, w.Hkv)
    rough, tau = gpu_noise(p, dev_bf16(c["inp"].Q), meta)
    ref = sums.reshape(w.B, w.H, w.T)
    assert np.all(rough[:, :, :2] == 0.0)
    rel = np.abs(rough - ref) / np.maximum(ref, 1e-300)
    assert np.all(rel[:, :, 2:] <= 1e-4), float(rel[:, :, 2:].max())
    units = oracle.all_units(w.B, w.H, w.T)
    for b in range(w.B):
        for h in range(w.H):
            sel = (units[:, 0] == b) & (units[:, 1] == h)
            t_ref = bai.noise_scale(sums[sel], terms[sel])
            assert abs(float(tau[b, h]) - t_ref) <= 1e-4 * t_ref


@pytest.mark.parametrize("backbone", [synth.KMEAN, synth.QUEST])
@pytest.mark.parametrize("d", [64, 128])
def test_noise_scale_exact_on_integer_rows(backbone, d):
    """Rows q_r = q_0 + r delta with small integers (positive for Quest):
    every fp32 score, difference, square and per-chunk sum is an exact
    integer, so the GPU sums equal the oracle's exactly."""
    H, Hkv, N = 4, 2, 64 * 40
    g = np.random.default_rng(11 + d)
    q0 = g.integers(1, 5, (H, d)).astype(np.float64)
    delta = g.integers(-1, 2, (H, d)).astype(np.float64)
    if backbone == synth.QUEST:
        delta = np.abs(delta)
    rows = np.arange(64)[None, :, None]
    Qf = np.zeros((1, H, N, d))
    for t in range(N // 64):
        Qf[0, :, 64 * t:64 * (t + 1)] = q0[:, None, :] + rows * delta[:, None, :]
    Q = synth.bf16_bits(Qf.astype(np.float32))
    K = synth.bf16_bits(g.integers(-2, 3, (1, Hkv, N, d)).astype(np.float32))
    meta = oracle.block_meta(backbone, K)
    sums, terms = oracle.row_roughness(backbone, Q, meta, Hkv)
    p = ugbs.Problem.make(1, H, Hkv, N, d, 4, 0.1, backbone)
    rough, tau = gpu_noise(p, dev_bf16(Q), meta)
    assert np.array_equal(rough.reshape(-1), sums)
    units = oracle.all_units(1, H, N // 64)
    for h in range(H):
        sel = units[:, 1] == h
        t_ref = bai.noise_scale(sums[sel], terms[sel])
        assert float(tau[0, h]) == np.float32(t_ref)


def test_noise_scale_nan_for_two_tiles():
    w = synth.WORKLOADS["C1"].replace(N=128, dup_pairs=False)
    inp = synth.generate(w, threads=2)
    meta = oracle.block_meta(w.backbone, inp.K)
    p = problem(w)
    rough, tau = gpu_noise(p, dev_bf16(inp.Q), meta)
    assert np.all(rough == 0.0) and np.isnan(tau).all()


# ---------------------------------------------------------------- chain

@pytest.mark.parametrize("name", list(CASES))
def test_chain_on_scores_out_matches_selection_sigma(name):
    """bai tiles on the GPU's own scores_out: every valid tile's sigma equals
    the selection kernel's sigma bit for bit (same scores, same order, same
    fp32 arithmetic)."""
    torch = __import__("torch")
    c = case(name)
    w = c["w"]
    p = problem(w)
    Q = dev_bf16(c["inp"].Q)
    meta = dev_meta(c["meta"])
    idx = torch.empty((w.B, w.H, w.T, p.W), dtype=torch.int32, device="cuda")
    sig = torch.empty((w.B, w.H, w.T), dtype=torch.float32, device="cuda")
    so = torch.empty((w.B, w.H, w.T, w.NB), dtype=torch.float32, device="cuda")
    ugbs.ugbs_score_select(p, Q, meta, idx, sig, scores_out=so)
    tiles = torch.empty((w.B * w.H * w.T * ugbs.BAI_TILE_BYTES,), dtype=torch.uint8, device="cuda")
    ugbs.ugbs_bai_tiles(p, so, tiles, tau=dev(c["tau32"]), z=dev(synth.block_major(c["z"])))
    torch.cuda.synchronize()
    rec = ugbs.bai_tile_records(tiles).reshape(w.B, w.H, w.T)
    v = rec["valid"].astype(bool)
    assert np.array_equal(v, bai.tile_gaps(c["S"], w.k)["valid"])
    assert np.array_equal(rec["sigma"][v].view(np.uint32), host(sig)[v].view(np.uint32))


# ---------------------------------------------------------------- full size

def _unit_oracle(S_row, t, NB, k, tau, z):
    """Oracle gaps and MC counts of one unit: its score row placed as the
    last tile of a [1, 1, t + 1, N_B] array."""
    S = np.full((1, 1, t + 1, NB), -np.inf, np.float32)
    S[0, 0, t] = S_row
    g = bai.tile_gaps(S, k)
    fk, fr = bai.mc_counts(S, k, np.array([[tau]], np.float32), z)
    return {f: g[f][0, 0, t] for f in g}, int(fk[0, 0, t]), int(fr[0, 0, t])


@pytest.mark.slow
@pytest.mark.parametrize("name", ["C2", "C3"])
def test_full_size_diagnostics(name):
    """The whole diagnostics pass at 32K / 64K in the benchmark's launch
    configuration: sampled units against the oracle (tiles given the
    oracle's scores, roughness from the same inputs), and properties of the
    per-head aggregates that hold at any size."""
    torch = __import__("torch")
    w = synth.WORKLOADS[name]
    inp = synth.generate(w, threads=16)
    p = problem(w)
    B, H, T, NB = w.B, w.H, w.T, w.NB
    Q, K = dev_bf16(inp.Q), dev_bf16(inp.K)
    meta = torch.empty((B, w.Hkv, NB, w.d, p.meta_width), dtype=torch.bfloat16, device="cuda")
    ugbs.ugbs_block_meta(p, K, meta)
    idx = torch.empty((B, H, T, p.W), dtype=torch.int32, device="cuda")
    sig = torch.empty((B, H, T), dtype=torch.float32, device="cuda")
    so = torch.empty((B, H, T, NB), dtype=torch.float32, device="cuda")
    ugbs.ugbs_score_select(p, Q, meta, idx, sig, scores_out=so)
    rough = torch.empty((B, H, T), dtype=torch.float64, device="cuda")
    tau = torch.empty((B, H), dtype=torch.float32, device="cuda")
    ugbs.ugbs_noise_scale(p, Q, meta, rough, tau)
    n_s = 128
    z = synth.mc_normals(w.seed(), n_s, NB)
    zd = dev(synth.block_major(z))
    tiles = torch.empty((B * H * T * ugbs.BAI_TILE_BYTES,), dtype=torch.uint8, device="cuda")
    ugbs.ugbs_bai_tiles(p, so, tiles, tau=tau, z=zd)
    heads = torch.empty((B * H * ugbs.BAI_HEAD_BYTES,), dtype=torch.uint8, device="cuda")
    ugbs.ugbs_bai_heads(p, tiles, tau, n_s, heads)
    torch.cuda.synchronize()

    # ---- sampled units: roughness against the oracle on the same inputs
    g = np.random.default_rng(w.seed())
    ts = sorted({2, 2 * w.k - 1, 2 * w.k, T - 1} | set(int(x) for x in g.integers(2, T, 8)))
    units = np.array([(0, int(g.integers(0, H)), t) for t in ts], np.int32)
    meta_np = oracle.block_meta(w.backbone, inp.K, nthreads=16)
    sums, _ = oracle.row_roughness(w.backbone, inp.Q, meta_np, w.Hkv, units=units, nthreads=16)
    rg = host(rough)
    for i, (b, h, t) in enumerate(units):
        assert abs(rg[b, h, t] - sums[i]) <= 1e-4 * sums[i], (b, h, t)
    # tau is the stated function of the roughness sums
    terms = 63.0 * (T - 1) * (T - 2) / 2
    assert np.allclose(host(tau), np.sqrt(rg.sum(axis=2) / (2 * terms)).astype(np.float32), rtol=1e-6)

    # ---- sampled tiles given the oracle's scores: bit-exact
    S = oracle.tile_scores(w.backbone, inp.Q, meta_np, w.Hkv, units=units, nthreads=16)
    sin = torch.full((B, H, T, NB), -np.inf, dtype=torch.float32, device="cuda")
    for i, (b, h, t) in enumerate(units):
        sin[b, h, t] = torch.from_numpy(S[i]).cuda()
    tau_in = np.full((B, H), 0.05, np.float32)
    t2 = torch.empty_like(tiles)
    ugbs.ugbs_bai_tiles(p, sin, t2, tau=dev(tau_in), z=zd)
    torch.cuda.synchronize()
    rec = ugbs.bai_tile_records(t2).reshape(B, H, T)
    for i, (b, h, t) in enumerate(units):
        ref, fk, fr = _unit_oracle(S[i], int(t), NB, w.k, float(tau_in[b, h]), z)
        r = rec[b, h, t]
        assert bool(r["valid"]) == bool(ref["valid"]), (b, h, t)
        for f in ("g", "G", "r", "sigma", "delta2"):
            assert same_f32(r[f], ref[f]), (f, b, h, t)
        assert (int(r["fail_k"]), int(r["fail_rk"])) == (fk, fr), (b, h, t)
    del sin, t2

    # ---- the GPU chain: properties of tiles and heads at full size
    rec = ugbs.bai_tile_records(tiles).reshape(B, H, T)
    hd = ugbs.bai_head_records(heads).reshape(B, H)
    v = rec["valid"].astype(bool)
    t_idx = np.arange(T)
    assert np.array_equal(v, np.broadcast_to(t_idx >= 2 * w.k, v.shape))
    sg = host(sig)
    assert np.array_equal(rec["sigma"][v].view(np.uint32), sg[v].view(np.uint32))
    assert (rec["fail_k"] >= rec["fail_rk"]).all()
    n = T - 2 * w.k
    nq = math.ceil(w.q * n)
    for b in range(B):
        for h in range(H):
            x = hd[b, h]
            s_h = rec["sigma"][b, h][v[b, h]]
            d_h = rec["delta2"][b, h][v[b, h]]
            assert x["n_tiles"] == n and x["n_q"] == nq
            assert (s_h < x["sigma_q"]).sum() < nq <= (s_h <= x["sigma_q"]).sum()
            assert x["pi2"] == (d_h < x["delta2_p05"]).sum() / n
            assert x["delta2_p05"] == np.sort(d_h)[int(math.floor(0.05 * (n - 1)))]
            assert x["mc_err_rk"] <= x["mc_err_k"] and x["mc_regret"] >= 0
            assert x["C_q"] <= 1.0 and x["bound"] <= min(w.q, 1 - w.q) + x["pi2"] + 1e-15
            assert x["tau"] == float(host(tau)[b, h])


def test_mc_mu_is_rounded_twice():
    """mu = fp32(s + fp32(tau z)) with both roundings: a tile built so that a
    fused multiply-add would change one comparison.  With tau = 0.8647483,
    z = 0.7718125 and s = 0.8033179, the two roundings give 1.4707415 and a
    single rounding 1.4707414; the kept block's mu is exactly 1.4707415, so
    the outside block ties it (a failure) only under double rounding."""
    f32 = np.float32
    T = 8
    tau, zx, cx = f32(0.8647483), f32(0.7718125), f32(0.8033179)
    mu_x = f32(cx + f32(tau * zx))
    assert mu_x == f32(1.4707415)
    S = np.full((1, 1, T, T), -np.inf, f32)
    g = np.random.default_rng(3)
    for t in range(2, T):
        S[0, 0, t, 1:t] = g.uniform(-1, 0, t - 1).astype(f32)
    # tile 6, k = 3: m = 1 kept, R' = 4; block 1 is the kept one, block 2 the runner-up
    S[0, 0, 6, 1:6] = [mu_x, cx, f32(0.1), f32(0.05), f32(0.0)]
    z = np.zeros((1, T), f32)
    z[0, 2] = zx
    p = ugbs.Problem.make(1, 1, 1, 64 * T, 64, 3, 0.5)
    tau32 = np.array([[tau]], f32)
    _, rec = gpu_tiles(p, S, tau32, z)
    check_tiles(rec, S, 3, tau32, z)
    assert rec["fail_k"][0, 0, 6] == 1 and rec["fail_rk"][0, 0, 6] == 0
