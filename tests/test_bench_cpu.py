"""Host logic of bench.py: the work counts behind its TFLOP/s figures, the
staleness rule of the recorded HBM traffic, and the one-GPU contract."""
import json
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2607_07724_amd import synth  # noqa: E402


def _pairs_brute(kv_idx, T):
    """Attended (query, key) pairs by enumeration: row i of tile t sees key j
    of a listed block b <= t when 64 b + j <= 64 t + i."""
    total = 0
    B, H = kv_idx.shape[:2]
    for b in range(B):
        for h in range(H):
            for t in range(T):
                blocks = {int(x) for x in kv_idx[b, h, t] if 0 <= x <= t}
                for blk in blocks:
                    for i in range(64):
                        for j in range(64):
                            total += (64 * blk + j) <= (64 * t + i)
    return total


def test_attention_flops_count_exact_causal_pairs():
    rng = np.random.default_rng(5)
    B, H, T, W, d = 1, 2, 9, 4, 64
    kv = np.full((B, H, T, W), T, np.int32)          # sentinel = N_B
    for h in range(H):
        for t in range(T):
            n = min(W, t + 1)
            row = rng.choice(t + 1, size=n, replace=False)
            kv[0, h, t, :n] = row
    kv[0, 1, 3, -1] = -1                               # junk entries are not attended
    got = bench.flops_attention(kv, T, d)
    assert got == 4.0 * d * _pairs_brute(kv, T)


def test_score_flops_count_rows_times_candidates():
    B, H, T, d = 1, 3, 7, 64
    for backbone, kd in ((0, d), (1, 2 * d)):
        brute = sum(2 * kd * 64 * max(t - 1, 0) for _ in range(B * H) for t in range(T))
        assert bench.flops_scores(B, H, T, d, backbone) == brute


def test_traffic_record_is_used_only_for_the_source_it_was_taken_on(tmp_path, monkeypatch):
    (tmp_path / "profiles").mkdir()
    src_dir = tmp_path / "paper_2607_07724_amd" / "csrc"
    src_dir.mkdir(parents=True)
    (src_dir / "attend.hip").write_bytes(b"kernel source A")
    (src_dir / "attend_common.h").write_bytes(b"helpers A")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    sha = bench.attention_source_sha256()
    rec = {"attend_kernel<128>": {"source_sha256": sha, "fetch_bytes": 100.4, "write_bytes": 20.2}}
    (tmp_path / "profiles" / "traffic.json").write_text(json.dumps(rec))
    c4 = synth.WORKLOADS["C4"]
    assert bench.measured_traffic(c4, None) == 121
    assert bench.measured_traffic(c4, 0.25) is None               # another workload
    assert bench.measured_traffic(synth.WORKLOADS["C2"], None) is None
    (src_dir / "attend_common.h").write_bytes(b"helpers B")      # an included header changed since
    assert bench.measured_traffic(c4, None) is None
    (src_dir / "attend_common.h").write_bytes(b"helpers A")
    assert bench.measured_traffic(c4, None) == 121
    (src_dir / "attend.hip").write_bytes(b"kernel source B")      # kernel changed since
    assert bench.measured_traffic(c4, None) is None


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_selection_stats_by_hand():
    """Two kv heads x two sibling query heads, three population tiles
    (k = 1 so every tile t >= 1 is in it); lists chosen so every overlap is
    known: head 0 keeps {0,1} at every tile, head 1 {0,2} at tiles 1-2 and
    {0,1} at tile 3, heads 2/3 (the second kv head) identical lists {1, 2}."""
    w = synth.Workload("t", 1, 4, 2, 64, 64 * 4, 1, 0.5, 0, "offset")
    NB = w.NB
    kv = np.full((1, 4, 4, 2), NB, np.int32)
    kv[0, 0, :] = [0, 1]
    kv[0, 1, :] = [0, 2]
    kv[0, 1, 3] = [0, 1]
    kv[0, 2:, :] = [1, 2]
    trig = np.zeros((1, 4), np.uint8)
    st = bench.selection_stats(kv, trig, w)
    assert st["mean_kept_blocks"] == 2.0
    # adjacent tiles (1,2), (2,3) of every head: 1, 1/3 for head 1, 1 otherwise
    assert st["jaccard_adjacent_tiles"] == round((6 * 1 + 1 + 1 / 3) / 8, 4)
    # sibling pairs at tiles 1..3: kv head 0: 1/3, 1/3, 1; kv head 1: 1, 1, 1
    assert st["jaccard_sibling_heads"] == round((1 / 3 + 1 / 3 + 1 + 3) / 6, 4)
    # unions: kv head 0 {0,1,2},{0,1,2},{0,1}; kv head 1 {1,2} x3; lists sum 4 each
    assert st["sibling_union_blocks"] == round((3 + 3 + 2 + 2 + 2 + 2) / 6, 2)
    assert st["sibling_union_over_sum"] == round(14 / 24, 4)


def test_cpu_leg_parity_on_oracle_outputs():
    """The CPU leg's parity check, fed the oracle's own routed lists and its
    attention rounded to bf16 as the 'GPU' result, reports every sampled row
    equal and the output within tolerance; a planted wrong block fails it."""
    import oracle
    w = synth.WORKLOADS["C1"]
    inp = synth.generate(w, threads=4)
    meta = oracle.block_meta(w.backbone, inp.K)
    S = oracle.tile_scores(w.backbone, inp.Q, meta, w.Hkv)
    idx, sig = oracle.select(S, w.k)
    kv, sb, tau, trig = oracle.route(sig, idx, w.k, w.q)
    units = bench.cpu_sample_units(w, 24)
    ref = oracle.attend(inp.Q, inp.K, inp.V, kv_idx=kv)
    O_units = np.stack([synth.bf16_bits(ref[b, h, 64 * t:64 * t + 64].astype(np.float32))
                        for b, h, t in units])
    r = bench.cpu_baseline(w, inp, units, kv, trig.astype(np.uint8), O_units, threads=2)
    assert r["parity"]["ok"] and r["parity"]["kv_rows_equal"] == len(units)
    assert r["cores"] == 2 and r["host_logical_cpus"] >= 1
    b, h, t = units[0]
    bad = kv.copy()
    row = [x for x in bad[b, h, t] if x != w.NB]
    spare = [x for x in range(1, t) if x not in row]
    if spare:
        bad[b, h, t, len(row) - 1] = spare[-1]
        r2 = bench.cpu_baseline(w, inp, units, bad, trig.astype(np.uint8), O_units, threads=2)
        assert r2["parity"]["kv_rows_beyond_near_ties"] >= 1 and not r2["parity"]["ok"]


def test_stage_roofline_holds_quest_scoring_to_the_sparse_peak():
    """The Quest score contraction runs on the 2:4-sparse instruction, so its
    dense-equivalent FLOP are held to the 5.0 PFLOP/s sparse peak; K-mean
    and the attention to the 2.5 PFLOP/s dense one."""
    for backbone, peak in ((synth.QUEST, 5000.0), (synth.KMEAN, 2500.0)):
        w = synth.WORKLOADS["C2"].replace(backbone=backbone)
        st = bench.stage_roofline(w, [1.0, 1.0, 1.0, 1.0], 2.5e12, 2.5e12, 10)
        assert st["score_select"]["mfma_peak_TFLOPs"] == peak
        assert st["score_select"]["frac_mfma"] == round(2500.0 / peak, 4)
        assert st["attend"]["mfma_peak_TFLOPs"] == 2500.0 and st["attend"]["frac_mfma"] == 1.0
