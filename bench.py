"""Benchmark: routed block-sparse causal prefill on one MI355X.

One step = one pass of the whole pipeline for one layer (block metadata ->
tile scores + top-2k + sigma -> quantile route -> sparse attention) over one
batch of synthetic input already resident in HBM.  Default workload: the
Mistral-Nemo attention shape (32 query / 8 kv heads, d 128) at N = 131072,
Quest backbone, k 64, q 0.1 (Table 3 context length; Section 4.1 shapes).

Printed (one JSON line): pipeline time and effective TFLOP/s, per-stage
times, the same-run dense causal attention (torch SDPA and this library's
kernel with every block listed), the roofline figures of the dominant
kernel (timed live with HIP events on its stream), and the reference oracle
timed on the host cores over a bounded sample of the same workload.
"""
import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "routed block-sparse prefill ms + TFLOP/s vs dense at 32K-128K, 1 MI355X"
PEAK_BF16_TFLOPS = 2500.0
# the 2:4-sparse bf16 instruction the Quest scoring runs on, dense-equivalent FLOP
PEAK_BF16_SPARSE_TFLOPS = 5000.0
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=None, choices=["C1", "C2", "C3", "C4", "C6", "P7", "L8"])
    ap.add_argument("--q", type=float, default=None)
    ap.add_argument("--cpu-units", type=int, default=3072, help="oracle sample size (tile, head units)")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--json-out", default=None)
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run a plain streaming kernel (1 GiB in, 1 GiB out) to scale HBM counters")
    ap.add_argument("--no-probe", action="store_true", help="skip the measured copy / GEMM peaks")
    ap.add_argument("--no-cold", action="store_true", help="skip the cold-cache steps")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the fused-selection, per-row selection and graph-replay variants")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the 32K-256K sweep (C2, C3, C4 at q 0.05 / 0.25, and the 256K layer L8 "
                         "with lists and fused selection)")
    ap.add_argument("--no-stack", action="store_true",
                    help="skip the 28-layer 128K stack (28/4 heads, both backbones) routed vs dense")
    ap.add_argument("--stack-steps", type=int, default=2, help="timed passes over the 28-layer stack")
    ap.add_argument("--bai", action="store_true",
                    help="time the Appendix D diagnostics pass instead (default workload C2)")
    ap.add_argument("--samples", type=int, default=256, help="Monte Carlo samples of the diagnostics")
    ap.add_argument("--oracle-layers", default=None,
                    help="CPU-baseline leg over whole layers: comma-separated layers (of --workload, "
                         "default the 28-layer stack); the oracle runs on each whole layer (every tile "
                         "and head) on the host cores, is timed, and the GPU pipeline is compared with it")
    ap.add_argument("--oracle-backbone", default=None, choices=["quest", "kmean"],
                    help="backbone for --oracle-layers (default: the workload's own)")
    ap.add_argument("--oracle-threads", type=int, default=None,
                    help="host threads for the oracle (default: the job's CPU share; 1 = single-threaded)")
    return ap.parse_args()


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def flops_attention(kv_idx: np.ndarray, NB: int, d: int) -> float:
    """4 d per attended (query, key) pair; exact causal pair count per unit."""
    T = kv_idx.shape[2]
    t = np.arange(T)[None, None, :, None]
    valid = (kv_idx >= 0) & (kv_idx <= t)
    diag = (kv_idx == t) & valid
    full = valid & ~diag
    pairs = full.sum(dtype=np.int64) * 64 * 64 + diag.sum(dtype=np.int64) * (64 * 65 // 2)
    return 4.0 * d * float(pairs)


def flops_scores(B: int, H: int, T: int, d: int, backbone: int) -> float:
    """2 * KD per (row, candidate block): KD = d (K-mean) or 2d (Quest split form)."""
    KD = d * (2 if backbone == 1 else 1)
    cand = sum(max(t - 1, 0) for t in range(T))
    return 2.0 * KD * B * H * 64 * cand


ATTENTION_SOURCES = ("attend.hip", "attend_common.h", "select_common.h", "ugbs_internal.h")


def attention_source_sha256():
    """SHA-256 over the attention kernel's translation unit and the headers
    it includes (in a fixed order), the key of the recorded traffic."""
    import hashlib
    h = hashlib.sha256()
    for name in ATTENTION_SOURCES:
        p = os.path.join(ROOT, "paper_2607_07724_amd", "csrc", name)
        if os.path.exists(p):
            with open(p, "rb") as f:
                h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def measured_traffic(w, q_override):
    """HBM bytes per attention launch from the committed rocprofv3 counter
    passes (FETCH_SIZE + WRITE_SIZE, each scaled by what the counter reads
    for a streaming kernel of known size), or None when the attention source
    has changed since the counters were taken or the workload differs."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if w.name != "C4" or q_override not in (None, 0.1) or not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f).get("attend_kernel<128>")
    if rec is None or rec.get("source_sha256") != attention_source_sha256():
        return None
    return round(rec["fetch_bytes"] + rec["write_bytes"])


def host_cores(requested=None):
    """The host's CPU facts and the thread count the oracle uses: the
    process's affinity set, capped by the job's CPU share when the
    environment states one (OMP_NUM_THREADS), or the requested count."""
    nproc = os.cpu_count() or 1
    try:
        affinity = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        affinity = nproc
    share_env = os.environ.get("OMP_NUM_THREADS")
    share = int(share_env) if share_env and share_env.isdigit() and int(share_env) > 0 else None
    threads = requested if requested else min(affinity, share or affinity)
    return {"threads": int(threads), "host_logical_cpus": nproc, "affinity_cpus": affinity,
            "job_cpu_share": share, "host_cpu": _cpu_name()}


def stage_roofline(w, stage_ms, f_sc, f_att, n_trig):
    """Per-stage work over time against the stage's roof: metadata, the
    selection route and (as bytes) the score+select stage against HBM, the
    score contraction and the attention against bf16 MFMA."""
    B, H, Hkv, N, NB, T, d = w.B, w.H, w.Hkv, w.N, w.NB, w.T, w.d
    W = w.rho * w.k
    c = 2 if w.backbone == 1 else 1
    meta_b = B * Hkv * N * d * 2 + B * Hkv * NB * d * 2 * c
    packed = B * H * (T - 1) * (T - 2) // 2 * 4
    score_b = B * H * N * d * 2 + B * Hkv * NB * d * 2 * c + 2 * packed + B * H * T * (W + 1) * 4
    route_b = B * H * T * 4 + (T - n_trig) * B * H * (W - w.k) * 4 + B * T * 9

    def hbm(by, ms):
        gbs = by / (ms * 1e-3) / 1e9
        return {"bytes": int(by), "GBps": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM_GBS, 4)}

    def mfma(fl, ms, peak=PEAK_BF16_TFLOPS):
        tf = fl / (ms * 1e-3) / 1e12
        return {"flop": fl, "TFLOPs": round(tf, 2), "mfma_peak_TFLOPs": peak, "frac_mfma": round(tf / peak, 4)}

    # Quest scores run on the 2:4-sparse instruction (twice the dense rate);
    # its FLOP are counted dense-equivalent, so they are held to that peak
    score_peak = PEAK_BF16_SPARSE_TFLOPS if w.backbone == 1 else PEAK_BF16_TFLOPS

    return {
        "block_meta": {"ms": round(float(stage_ms[0]), 4), "bound": "hbm", **hbm(meta_b, stage_ms[0])},
        "score_select": {"ms": round(float(stage_ms[1]), 4), "bound": "mfma",
                         **mfma(f_sc, stage_ms[1], score_peak), **hbm(score_b, stage_ms[1])},
        "route": {"ms": round(float(stage_ms[2]), 4), "bound": "hbm (launch latency)",
                  **hbm(route_b, stage_ms[2])},
        "attend": {"ms": round(float(stage_ms[3]), 4), "bound": "mfma", **mfma(f_att, stage_ms[3])},
    }


def selection_stats(kv, trig, w):
    """Overlap of the kept block sets: Jaccard index of adjacent tiles of a
    head and of the sibling query heads of one kv head at one tile, and the
    union over all sibling heads of a tile relative to the sum of their
    lists (the share of K/V fetches a kernel staging blocks once per sibling
    group could save)."""
    B, H, T, W = kv.shape
    NB, G = w.NB, w.H // w.Hkv
    words = (NB + 63) // 64
    bits = np.zeros((B, H, T, words), np.uint64)
    b_i, h_i, t_i, s_i = np.nonzero((kv >= 0) & (kv < NB))
    blk = kv[b_i, h_i, t_i, s_i].astype(np.int64)
    np.bitwise_or.at(bits, (b_i, h_i, t_i, blk // 64), np.left_shift(np.uint64(1), (blk % 64).astype(np.uint64)))
    cnt = np.bitwise_count(bits).sum(axis=-1).astype(np.float64)

    def jacc(a, b):
        inter = np.bitwise_count(a & b).sum(axis=-1).astype(np.float64)
        uni = np.bitwise_count(a | b).sum(axis=-1).astype(np.float64)
        return float(np.mean(inter / np.maximum(uni, 1)))

    pop = np.arange(T) >= w.k               # tiles with more candidates than kept slots
    tt = np.nonzero(pop[1:] & pop[:-1])[0]
    adj = jacc(bits[:, :, tt], bits[:, :, tt + 1]) if len(tt) else None
    sib = []
    grp = bits.reshape(B, w.Hkv, G, T, words)[:, :, :, pop]
    for i in range(G):
        for j in range(i + 1, G):
            sib.append(jacc(grp[:, :, i], grp[:, :, j]))
    union = np.bitwise_or.reduce(grp, axis=2)
    ucnt = np.bitwise_count(union).sum(axis=-1).astype(np.float64)
    lsum = cnt.reshape(B, w.Hkv, G, T)[:, :, :, pop].sum(axis=2)
    return {"mean_kept_blocks": round(float(cnt.mean()), 3),
            "triggered_tiles": int(trig.sum()),
            "jaccard_adjacent_tiles": None if adj is None else round(adj, 4),
            "jaccard_sibling_heads": round(float(np.mean(sib)), 4) if sib else None,
            "sibling_union_blocks": round(float(ucnt.mean()), 2),
            "sibling_list_blocks": round(float(lsum.mean()), 2),
            "sibling_union_over_sum": round(float(ucnt.sum() / max(lsum.sum(), 1)), 4)}


def make_pipeline_step(ugbs, p, Q, K, V, O, bufs, stream):
    def step(ev=None):
        rec = (lambda i: ev[i].record(stream)) if ev is not None else (lambda i: None)
        rec(0)
        ugbs.ugbs_block_meta(p, K, bufs.meta)
        rec(1)
        ugbs.ugbs_score_select(p, Q, bufs.meta, bufs.idx_sorted, bufs.sigma, workspace=bufs.workspace)
        rec(2)
        ugbs.ugbs_route(p, bufs.sigma, bufs.idx_sorted, bufs.kv_idx, bufs.workspace,
                        bufs.sigma_bar, bufs.tau, bufs.trigger)
        rec(3)
        ugbs.ugbs_attend(p, Q, K, V, bufs.kv_idx, O)
        rec(4)
    return step


def time_steps(torch, dev, step, steps, warmup, n_ev=5):
    """Warm up, then time `steps` calls of step(events) bracketed by
    synchronisations; returns (wall ms per step, [steps, n_ev - 1] stage ms)."""
    for _ in range(warmup):
        step()
    torch.cuda.synchronize(dev)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(n_ev)] for _ in range(steps)]
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    for i in range(steps):
        step(evs[i])
    torch.cuda.synchronize(dev)
    wall = 1e3 * (time.perf_counter() - t0) / steps
    st = np.array([[evs[i][j].elapsed_time(evs[i][j + 1]) for j in range(n_ev - 1)] for i in range(steps)])
    return wall, st


def time_dense(torch, dev, ugbs, synth, w, Q, K, V, stream, sdpa_reps=3, own_reps=2):
    """Same-run dense causal attention on the same inputs: torch SDPA (GQA
    heads expanded outside the timed region) and this library's kernel with
    every causal block listed."""
    import torch.nn.functional as F
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    f_dense = 4.0 * w.d * w.B * w.H * (w.N * (w.N + 1) / 2)
    sd_ms = None
    try:
        from torch.nn.attention import SDPBackend, sdpa_kernel
        G = w.H // w.Hkv
        Ke, Ve = K.repeat_interleave(G, dim=1), V.repeat_interleave(G, dim=1)
        with sdpa_kernel([SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION]):
            F.scaled_dot_product_attention(Q, Ke, Ve, is_causal=True)
            torch.cuda.synchronize(dev)
            e0.record(stream)
            for _ in range(sdpa_reps):
                F.scaled_dot_product_attention(Q, Ke, Ve, is_causal=True)
            e1.record(stream)
            torch.cuda.synchronize(dev)
        sd_ms = e0.elapsed_time(e1) / sdpa_reps
        del Ke, Ve
    except Exception as ex:  # keep the routed figures even if SDPA is unavailable
        log(f"torch SDPA failed: {ex!r}")
    kvd = torch.from_numpy(synth.dense_kv_idx(w.B, w.H, w.T)).to(dev)
    pd = ugbs.Problem.make(w.B, w.H, w.Hkv, w.N, w.d, w.NB, 0.0, w.backbone, rho=1)   # every block: W = N_B
    Od = torch.empty_like(Q)
    ugbs.ugbs_attend(pd, Q, K, V, kvd, Od)
    torch.cuda.synchronize(dev)
    e0.record(stream)
    for _ in range(own_reps):
        ugbs.ugbs_attend(pd, Q, K, V, kvd, Od)
    e1.record(stream)
    torch.cuda.synchronize(dev)
    ud_ms = e0.elapsed_time(e1) / own_reps
    del kvd, Od
    return {
        "torch_sdpa_ms": None if sd_ms is None else round(sd_ms, 3),
        "torch_sdpa_TFLOPs": None if sd_ms is None else round(f_dense / (sd_ms * 1e-3) / 1e12, 1),
        "ugbs_attend_dense_ms": round(ud_ms, 3),
        "ugbs_attend_dense_TFLOPs": round(f_dense / (ud_ms * 1e-3) / 1e12, 1),
        "dense_flop": f_dense,
    }


def layer_record(w, ms, stage_avg, kv, trig, needles):
    f_att = flops_attention(kv, w.NB, w.d)
    f_sc = flops_scores(w.B, w.H, w.T, w.d, w.backbone)
    hits = [int(np.any(kv[b, h, i // 64] == j // 64)) for (b, h, i, j) in needles]
    sel = selection_stats(kv, trig, w)
    sel["needle_hit_rate"] = float(np.mean(hits)) if hits else None
    return {"ms_per_step": round(ms, 4),
            "TFLOPs": round((f_sc + f_att) / (ms * 1e-3) / 1e12, 2),
            "stages": stage_roofline(w, stage_avg, f_sc, f_att, int(trig.sum())),
            "selection": sel}, f_sc, f_att


def run_sweep(torch, dev, ugbs, synth, a, c4_inputs):
    """The 32K-128K range of the metric: C2 (32K) and C3 (64K) at their own
    settings, and the 128K layer at q 0.05 and 0.25 (the same inputs as the
    headline line, only the route and attention differ); each with its
    same-run dense causal attention."""
    out = []
    stream = torch.cuda.current_stream(dev)
    cases = [(synth.WORKLOADS["C2"], None), (synth.WORKLOADS["C3"], None),
             (synth.WORKLOADS["C4"].replace(q=0.05), c4_inputs),
             (synth.WORKLOADS["C4"].replace(q=0.25), c4_inputs),
             (synth.WORKLOADS["L8"], None)]
    for w, given in cases:
        if given is None:
            inp = synth.generate(w, threads=16)
            cv = lambda x: torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)
            Q, K, V = cv(inp.Q), cv(inp.K), cv(inp.V)
            needles = inp.needles
            del inp
        else:
            Q, K, V, needles = given
        p = ugbs.Problem.make(w.B, w.H, w.Hkv, w.N, w.d, w.k, w.q, w.backbone)
        bufs = ugbs.Buffers(p, device=dev)
        O = torch.empty_like(Q)
        step = make_pipeline_step(ugbs, p, Q, K, V, O, bufs, stream)
        ms, st = time_steps(torch, dev, step, max(3, min(a.steps, 10)), max(1, min(a.warmup, 3)))
        rec, f_sc, f_att = layer_record(w, ms, st.mean(axis=0), bufs.kv_idx.cpu().numpy(),
                                        bufs.trigger.cpu().numpy(), needles)
        rec = {"workload": w.name, "seq_len": w.N, "q_heads": w.H, "kv_heads": w.Hkv, "k_budget": w.k,
               "q": w.q, "backbone": "quest" if w.backbone == 1 else "kmean", **rec}
        if w.N > 131072:
            # beyond 128K the selection inside the attention kernel is timed too
            # (the regime where the paper expects the fusion to pay)
            rec["fused_selection"] = run_fused(torch, dev, ugbs, p, Q, K, V, O, stream,
                                               argparse.Namespace(steps=max(3, min(a.steps, 10)),
                                                                  warmup=max(1, min(a.warmup, 3))), f_att)
        if not a.no_dense:
            dn = time_dense(torch, dev, ugbs, synth, w, Q, K, V, stream,
                            sdpa_reps=2 if w.N >= 131072 else 3, own_reps=1 if w.N >= 131072 else 2)
            dn["routed_over_sdpa"] = None if dn["torch_sdpa_ms"] is None else round(ms / dn["torch_sdpa_ms"], 4)
            rec["dense"] = dn
        log(f"sweep {w.name} q {w.q}: {ms:.3f} ms/step, attention {rec['stages']['attend']}")
        out.append(rec)
        del bufs, O
        if given is None:
            del Q, K, V
    torch.cuda.empty_cache()
    return out


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py runs on exactly one GPU (asked for --gpus {a.gpus}); sharding the path "
              "across GPUs (by kv-head group) is not built: one GPU's share is what is measured",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2607_07724_amd as ugbs
    from paper_2607_07724_amd import synth

    w = synth.WORKLOADS[a.workload or ("C2" if a.bai else "C4")]
    if a.q is not None:
        w = w.replace(q=a.q)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if a.bai:
        return run_bai(a, torch, dev, ugbs, synth, w)
    if a.oracle_layers:
        return run_oracle_layers(a, torch, dev, ugbs, synth)
    if a.calibrate_copy:
        # a plain streaming kernel of known size: reads 1 GiB, writes 1 GiB
        src = torch.empty(1 << 29, dtype=torch.int16, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(2):
            torch.add(src, 1, out=dst)
        torch.cuda.synchronize(dev)
        del src, dst
        log("calibration: 2 x elementwise add, 1 GiB read + 1 GiB written each")
    headline = a.workload is None and a.q is None
    log(f"workload {w.name}: B={w.B} H={w.H}/{w.Hkv} d={w.d} N={w.N} k={w.k} q={w.q} backbone={w.backbone}")
    t0 = time.time()
    inp = synth.generate(w, threads=16)
    log(f"inputs generated in {time.time() - t0:.1f}s")

    def to_dev(x):
        return torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)

    Q, K, V = to_dev(inp.Q), to_dev(inp.K), to_dev(inp.V)
    p = ugbs.Problem.make(w.B, w.H, w.Hkv, w.N, w.d, w.k, w.q, w.backbone, rho=w.rho)
    bufs = ugbs.Buffers(p, device=dev)
    O = torch.empty_like(Q)
    stream = torch.cuda.current_stream(dev)
    step = make_pipeline_step(ugbs, p, Q, K, V, O, bufs, stream)
    ms_per_step, stage_ms = time_steps(torch, dev, step, a.steps, a.warmup)
    stage_avg = stage_ms.mean(axis=0)
    step_ms = stage_ms.sum(axis=1)
    log(f"timed {a.steps} steps: {ms_per_step:.3f} ms/step; stages {np.round(stage_avg, 4).tolist()}")

    kv = bufs.kv_idx.cpu().numpy()
    trig = bufs.trigger.cpu().numpy()
    layer, f_sc, f_att = layer_record(w, ms_per_step, stage_avg, kv, trig, inp.needles)
    f_dense = 4.0 * w.d * w.B * w.H * (w.N * (w.N + 1) / 2)

    graph = fused = rows = quest_forms = None
    if not a.no_variants:
        graph = run_graph(torch, dev, step, O, stream, a)
        fused = run_fused(torch, dev, ugbs, p, Q, K, V, O, stream, a, f_att)
        rows = run_rows(torch, dev, ugbs, w, p, Q, K, V, stream, a, inp.needles)
        if w.backbone == ugbs.QUEST:
            quest_forms = run_quest_forms(torch, dev, ugbs, w, p, Q, bufs, stream, a)

    cold = None
    if not a.no_cold:
        # caches cold: a 1 GiB write (twice the 256 MB last-level cache) before each single step
        flush = torch.empty(1 << 28, dtype=torch.int32, device=dev)
        cold_ms = []
        for i in range(3):
            flush.fill_(i)
            torch.cuda.synchronize(dev)
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
            step(ev)
            torch.cuda.synchronize(dev)
            cold_ms.append([ev[j].elapsed_time(ev[j + 1]) for j in range(4)])
        del flush
        cm = np.array(cold_ms)
        cold = {"ms_median": round(float(np.median(cm.sum(axis=1))), 4),
                "stages_ms_median": np.round(np.median(cm, axis=0), 4).tolist(),
                "runs": 3, "flush": "1 GiB device write before each step"}
        log(f"cold: {cold}")

    att_ms = float(stage_avg[3])
    kept = (kv != w.NB).sum(axis=-1)
    bytes_kv_gathered = 2.0 * float(kept.sum()) * 64 * w.d * 2
    roofline = {
        "kernel": f"attend_kernel<{w.d}, 0> (kv_idx lists)",
        "bound": "mfma",
        "achieved": round(f_att / (att_ms * 1e-3) / 1e12, 2),
        "peak": PEAK_BF16_TFLOPS,
        "unit": "TFLOP/s",
        "frac": round(f_att / (att_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "traffic": measured_traffic(w, a.q),
        "flop_per_launch": f_att,
        "gathered_kv_bytes_per_launch": bytes_kv_gathered,
        "gathered_kv_GBps": round(bytes_kv_gathered / (att_ms * 1e-3) / 1e9, 1),
        "flop_per_staged_kv_byte": round(f_att / bytes_kv_gathered, 2),
    }

    dense = None
    if not a.no_dense:
        dense = time_dense(torch, dev, ugbs, synth, w, Q, K, V, stream)
        dense["routed_over_sdpa"] = (None if dense["torch_sdpa_ms"] is None
                                     else round(ms_per_step / dense["torch_sdpa_ms"], 4))
        log(f"dense: {dense}")

    probe = None
    if not a.no_probe:
        probe = measured_peaks(torch, dev, stream)
        log(f"measured peaks: {probe}")
        roofline["measured_peak_TFLOPs"] = probe["gemm_bf16_TFLOPs"]
        roofline["frac_of_measured_peak"] = round(roofline["achieved"] / probe["gemm_bf16_TFLOPs"], 4)
        if probe["mfma_loop_bf16_TFLOPs"]:
            roofline["mfma_loop_TFLOPs"] = probe["mfma_loop_bf16_TFLOPs"]
            roofline["frac_of_mfma_loop"] = round(roofline["achieved"] / probe["mfma_loop_bf16_TFLOPs"], 4)

    # GPU outputs of the units the CPU leg samples, copied before the big legs free memory
    cpu = None
    sample = None
    if not a.no_cpu:
        sample = cpu_sample_units(w, a.cpu_units)
        idx_t = torch.from_numpy(sample.astype(np.int64)).to(dev)
        Ou = O.view(w.B, w.H, w.T, 64, w.d)[idx_t[:, 0], idx_t[:, 1], idx_t[:, 2]]
        gpu_O_sample = Ou.view(torch.int16).cpu().numpy().view(np.uint16)
        del idx_t, Ou

    sweep = None
    if headline and not a.no_sweep:
        sweep = run_sweep(torch, dev, ugbs, synth, a, (Q, K, V, inp.needles))

    del bufs, O
    torch.cuda.empty_cache()
    stack = None
    if headline and not a.no_stack:
        del Q, K, V
        torch.cuda.empty_cache()
        stack = run_stack(torch, dev, ugbs, synth, a.stack_steps)

    if not a.no_cpu:
        cpu = cpu_baseline(w, inp, sample, kv, trig, gpu_O_sample, a.oracle_threads)
        log(f"cpu baseline: {cpu}")

    value = (f_sc + f_att) / (ms_per_step * 1e-3) / 1e12
    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"{w.name}: Mistral-Nemo-shaped causal GQA prefill layer" if w.name == "C4" else w.name,
            "batch": w.B, "q_heads": w.H, "kv_heads": w.Hkv, "head_dim": w.d, "seq_len": w.N,
            "block": 64, "k_budget": w.k, "q": w.q, "rho": w.rho,
            "backbone": "quest" if w.backbone == 1 else "kmean", "seed": w.seed(0),
        },
        "flop": {"score": f_sc, "attention": f_att, "dense_equivalent_TFLOPs":
                 round(f_dense / (ms_per_step * 1e-3) / 1e12, 1)},
        "stages": layer["stages"],
        "dense": dense,
        "selection": layer["selection"],
        "fused_selection": fused,
        "row_selection": rows,
        "quest_scoring_forms": quest_forms,
        "ms_per_step_median": round(float(np.median(step_ms)), 4),
        "graph_replay": graph,
        "cold": cold,
        "measured_peaks": probe,
        "sweep": sweep,
        "stack": stack,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    line = json.dumps(out)
    print(line, flush=True)
    if a.json_out:
        with open(a.json_out, "w") as f:
            f.write(line + "\n")


def run_graph(torch, dev, step, O, stream, a):
    """The same layer captured once in a HIP graph and replayed (no host
    launch gaps between the kernels); its output must equal the eager one."""
    try:
        O_eager = O.clone()
        side = torch.cuda.Stream(dev)
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            step()
        stream.wait_stream(side)
        torch.cuda.synchronize(dev)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        for _ in range(a.warmup):
            g.replay()
        torch.cuda.synchronize(dev)
        t0 = time.perf_counter()
        for _ in range(a.steps):
            g.replay()
        torch.cuda.synchronize(dev)
        graph_ms = 1e3 * (time.perf_counter() - t0) / a.steps
        res = {"ms_per_step": round(graph_ms, 4),
               "output_identical": bool(torch.equal(O.view(torch.int16), O_eager.view(torch.int16)))}
        del g, O_eager
        log(f"graph replay: {res}")
        return res
    except Exception as ex:  # reported, never fatal: the eager layer is the measured one
        log(f"graph capture failed: {ex!r}")
        return {"error": repr(ex)}


def run_fused(torch, dev, ugbs, p, Q, K, V, O, stream, a, f_att):
    """The same layer with the selection inside the attention kernel (no kv_idx lists)."""
    fb = ugbs.Buffers(p, device=dev)
    Of = torch.empty_like(Q)

    def step_fused(ev=None):
        rec = (lambda i: ev[i].record(stream)) if ev is not None else (lambda i: None)
        rec(0)
        ugbs.ugbs_block_meta(p, K, fb.meta)
        rec(1)
        ugbs.ugbs_score_select(p, Q, fb.meta, None, fb.sigma, workspace=fb.workspace)
        rec(2)
        ugbs.ugbs_route(p, fb.sigma, None, None, fb.workspace, fb.sigma_bar, fb.tau, fb.trigger)
        rec(3)
        ugbs.ugbs_attend_select(p, Q, K, V, Of, workspace=fb.workspace)
        rec(4)

    ms, st = time_steps(torch, dev, step_fused, a.steps, a.warmup)
    fst = st.mean(axis=0)
    same = bool(torch.equal(O.view(torch.int16), Of.view(torch.int16)))
    log(f"fused: {ms:.3f} ms/step; stages {np.round(fst, 4).tolist()}; output identical: {same}")
    del fb, Of
    return {"ms_per_step": round(ms, 4),
            "stages_ms": {"block_meta": round(float(fst[0]), 4), "score_sigma": round(float(fst[1]), 4),
                          "route_flags": round(float(fst[2]), 4), "attend_select": round(float(fst[3]), 4)},
            "attend_select_TFLOPs": round(f_att / (fst[3] * 1e-3) / 1e12, 2),
            "output_identical": same}


def run_quest_forms(torch, dev, ugbs, w, p, Q, bufs, stream, a):
    """Quest tile scores in both forms, each into a full [B, H, T, N_B] tensor:
    the per-channel vector-ALU form (one bf16 dot2 per bound term) and the
    2:4-sparse matrix-core form inside ugbs_score_select (which also runs the
    selection; the selection alone is timed from the same scores through
    scores_in, so the matrix-core scoring time is the difference)."""
    so_v = torch.empty((w.B, w.H, w.T, w.NB), dtype=torch.float32, device=dev)
    so_m = torch.empty_like(so_v)
    idx = torch.empty_like(bufs.idx_sorted)
    sig = torch.empty_like(bufs.sigma)

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize(dev)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record(stream)
        for _ in range(reps):
            fn()
        ev[1].record(stream)
        torch.cuda.synchronize(dev)
        return ev[0].elapsed_time(ev[1]) / reps

    reps = max(2, a.steps // 2)
    ms_valu = timed(lambda: ugbs.ugbs_quest_scores_valu(p, Q, bufs.meta, so_v), reps)
    ms_mfma_sel = timed(lambda: ugbs.ugbs_score_select(p, Q, bufs.meta, idx, sig, scores_out=so_m), reps)
    ms_sel = timed(lambda: ugbs.ugbs_score_select(p, Q, bufs.meta, idx, sig, scores_in=so_m), reps)
    fin = torch.isfinite(so_m)
    same_inf = bool(torch.equal(fin, torch.isfinite(so_v)))
    rel = float(((so_v - so_m).abs()[fin] / so_m.abs()[fin].clamp_min(1e-30)).max())
    # bound terms: d per (row, candidate block); one dot2 instruction lane-op each
    terms = float(w.B * w.H) * sum(max(t - 1, 0) for t in range(w.T)) * 64 * w.d
    valu_peak = 256 * 64 * 2.4e9          # lane-ops per second: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
    rec = {"valu_dot2_ms": round(ms_valu, 4),
           "mfma_score_plus_select_ms": round(ms_mfma_sel, 4),
           "select_only_ms": round(ms_sel, 4),
           "mfma_score_ms": round(ms_mfma_sel - ms_sel, 4),
           "valu_over_mfma": round(ms_valu / max(ms_mfma_sel - ms_sel, 1e-9), 2),
           "bound_terms": terms,
           "valu_frac_of_dot2_peak": round(terms / (ms_valu * 1e-3) / valu_peak, 4),
           "same_inf_pattern": same_inf, "max_rel_diff": rel}
    log(f"quest forms: {rec}")
    del so_v, so_m, idx, sig
    return rec


def run_rows(torch, dev, ugbs, w, p, Q, K, V, stream, a, needles):
    """Per-row selection into tile bitmaps (union over each tile's rows)."""
    rb = ugbs.Buffers(p, device=dev)
    Or = torch.empty_like(Q)
    bm = torch.empty((w.B, w.H, w.T, ugbs.bitmap_words(p)), dtype=torch.int32, device=dev)

    def step_rows(ev=None):
        rec = (lambda i: ev[i].record(stream)) if ev is not None else (lambda i: None)
        rec(0)
        ugbs.ugbs_block_meta(p, K, rb.meta)
        ugbs.ugbs_score_select(p, Q, rb.meta, None, rb.sigma, workspace=rb.workspace)
        ugbs.ugbs_route(p, rb.sigma, None, None, rb.workspace, rb.sigma_bar, rb.tau, rb.trigger)
        rec(1)
        ugbs.ugbs_select_rows(p, rb.trigger, bm, Q=Q, meta=rb.meta)
        rec(2)
        ugbs.ugbs_attend_bitmap(p, Q, K, V, bm, Or)
        rec(3)

    ms, st = time_steps(torch, dev, step_rows, a.steps, a.warmup, n_ev=4)
    rst = st.mean(axis=0)
    bmh = bm.cpu().numpy().view(np.uint32)
    kept_rows = np.unpackbits(bmh.view(np.uint8), axis=-1).reshape(w.B, w.H, w.T, -1).sum(axis=-1)
    # attention flop from the bitmaps' block sets: every set holds its diagonal block t
    f_rows = 4.0 * w.d * float((kept_rows - 1).sum() * 64 * 64 + kept_rows.size * (64 * 65 // 2))
    hits = [int((int(bmh[b, h, i // 64, (j // 64) // 32]) >> ((j // 64) % 32)) & 1) for (b, h, i, j) in needles]
    log(f"rows: {ms:.3f} ms/step; stages {np.round(rst, 4).tolist()}; mean kept {kept_rows.mean():.2f}")
    del rb, Or, bm
    return {"ms_per_step": round(ms, 4),
            "stages_ms": {"meta_score_sigma_route": round(float(rst[0]), 4),
                          "select_rows": round(float(rst[1]), 4), "attend_bitmap": round(float(rst[2]), 4)},
            "attend_bitmap_TFLOPs": round(f_rows / (rst[2] * 1e-3) / 1e12, 2),
            "mean_kept_blocks": round(float(kept_rows.mean()), 3),
            "needle_hit_rate": float(np.mean(hits)) if hits else None}


BAI_METRIC = "Appendix D diagnostics pass: (batch, head, tile) units per second, 1 MI355X"


def run_bai(a, torch, dev, ugbs, synth, w):
    """One step = the Appendix D diagnostics of one layer: tile scores into
    HBM (ugbs_score_select with scores_out), row roughness and the noise
    scale, per-tile gaps with the Monte Carlo over `--samples` shared normal
    draws, and the per-head aggregates."""
    log(f"diagnostics workload {w.name}: B={w.B} H={w.H}/{w.Hkv} d={w.d} N={w.N} k={w.k} "
        f"q={w.q} backbone={w.backbone} samples={a.samples}")
    inp = synth.generate(w, threads=16)

    def to_dev(x):
        return torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)

    Q, K = to_dev(inp.Q), to_dev(inp.K)
    p = ugbs.Problem.make(w.B, w.H, w.Hkv, w.N, w.d, w.k, w.q, w.backbone)
    B, H, T, NB = w.B, w.H, w.T, w.NB
    meta = torch.empty((B, w.Hkv, NB, w.d, p.meta_width), dtype=torch.bfloat16, device=dev)
    idx = torch.empty((B, H, T, p.W), dtype=torch.int32, device=dev)
    sig = torch.empty((B, H, T), dtype=torch.float32, device=dev)
    scores = torch.empty((B, H, T, NB), dtype=torch.float32, device=dev)
    rough = torch.empty((B, H, T), dtype=torch.float64, device=dev)
    tau = torch.empty((B, H), dtype=torch.float32, device=dev)
    z = torch.from_numpy(synth.block_major(synth.mc_normals(w.seed(), a.samples, NB))).to(dev)
    tiles = torch.empty((B * H * T * ugbs.BAI_TILE_BYTES,), dtype=torch.uint8, device=dev)
    heads = torch.empty((B * H * ugbs.BAI_HEAD_BYTES,), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    ugbs.ugbs_block_meta(p, K, meta)

    def step(ev=None):
        rec = (lambda i: ev[i].record(stream)) if ev is not None else (lambda i: None)
        rec(0)
        ugbs.ugbs_score_select(p, Q, meta, idx, sig, scores_out=scores)
        rec(1)
        ugbs.ugbs_noise_scale(p, Q, meta, rough, tau)
        rec(2)
        ugbs.ugbs_bai_tiles(p, scores, tiles, tau=tau, z=z)
        rec(3)
        ugbs.ugbs_bai_heads(p, tiles, tau, a.samples, heads)
        rec(4)

    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize(dev)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(a.steps)]
    t0 = time.perf_counter()
    for i in range(a.steps):
        step(evs[i])
    torch.cuda.synchronize(dev)
    ms_per_step = 1e3 * (time.perf_counter() - t0) / a.steps
    st = np.array([[evs[i][j].elapsed_time(evs[i][j + 1]) for j in range(4)] for i in range(a.steps)]).mean(axis=0)
    log(f"timed {a.steps} steps: {ms_per_step:.3f} ms/step; stages {np.round(st, 4).tolist()}")
    rec = ugbs.bai_tile_records(tiles).reshape(B, H, T)
    hd = ugbs.bai_head_records(heads).reshape(B, H)
    n_valid = int(rec["valid"].sum())
    # per-unit algorithmic work of the tile kernel: one read of the candidate
    # scores from HBM, and per (sample, candidate) one fp32 multiply and one add
    cand = np.array([max(t - 1, 0) for t in range(T)], np.float64)
    valid_t = rec["valid"][0, 0].astype(bool)
    bytes_tiles = 4.0 * B * H * cand.sum() + 32.0 * B * H * T
    flop_mc = 2.0 * a.samples * B * H * cand[valid_t].sum()
    units = B * H * T
    tiles_ms = float(st[2])
    f_rough = flops_scores(B, H, T, w.d, w.backbone)
    stages = {
        "score_select_scores_out": {"ms": round(float(st[0]), 4),
                                    "scores_GBps": round(4.0 * B * H * T * NB / (st[0] * 1e-3) / 1e9, 1)},
        "noise_scale": {"ms": round(float(st[1]), 4),
                        "TFLOPs": round(f_rough / (st[1] * 1e-3) / 1e12, 2)},
        "bai_tiles": {"ms": round(tiles_ms, 4),
                      "scores_GBps": round(bytes_tiles / (tiles_ms * 1e-3) / 1e9, 1),
                      "mc_TFLOPs": round(flop_mc / (tiles_ms * 1e-3) / 1e12, 3)},
        "bai_heads": {"ms": round(float(st[3]), 4)},
    }
    dom = int(np.argmax(st))
    name = ["score_select", "noise_scale", "bai_tiles", "bai_heads"][dom]
    if name == "bai_tiles":
        ach = flop_mc / (tiles_ms * 1e-3) / 1e12
        roof = {"kernel": "bai_tile_kernel", "bound": "alu", "achieved": round(ach, 3),
                "peak": 157.3, "unit": "TFLOP/s", "frac": round(ach / 157.3, 5), "traffic": None,
                "flop_per_launch": flop_mc, "note": "fp32 vector peak; 2 flop per (sample, candidate)"}
    elif name == "noise_scale":
        ach = f_rough / (st[1] * 1e-3) / 1e12
        roof = {"kernel": "score_kernel (roughness mode)", "bound": "mfma", "achieved": round(ach, 2),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4),
                "traffic": None, "flop_per_launch": f_rough}
    else:
        by = 4.0 * B * H * T * NB
        ach = by / (st[0] * 1e-3) / 1e9
        roof = {"kernel": name, "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": None}
    cpu = None if a.no_cpu else cpu_baseline_bai(w, inp, a.samples)
    out = {
        "metric": BAI_METRIC,
        "value": round(units / (ms_per_step * 1e-3), 1),
        "unit": "units/s",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"{w.name} diagnostics: B {B}, {H} q / {w.Hkv} kv heads, d {w.d}, "
                               f"N {w.N}, k {w.k}, q {w.q}, {a.samples} Monte Carlo samples",
                   "backbone": "quest" if w.backbone == 1 else "kmean", "seed": w.seed(0)},
        "stages": stages,
        "valid_tiles": n_valid,
        "head0": {f: float(hd[f][0, 0]) for f in ("r_cv", "sigma_q", "tau", "delta2_p05", "chi", "C_q",
                                                   "bound", "mc_err_k", "mc_err_rk", "mc_regret")},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    line = json.dumps(out)
    print(line, flush=True)
    if a.json_out:
        with open(a.json_out, "w") as f:
            f.write(line + "\n")


def cpu_baseline_bai(w, inp, n_s, kv_heads=2):
    """The diagnostics oracle on a bounded sample: block metadata, tile
    scores and row roughness of the query heads of `kv_heads` kv heads,
    then their tile gaps, Monte Carlo counts and head aggregates; rate in
    (b, h, t) units/s."""
    import oracle
    from oracle import bai
    hc = host_cores()
    threads = hc["threads"]
    G = w.H // w.Hkv
    nh = G * kv_heads
    Q1 = np.ascontiguousarray(inp.Q[:1, :nh])
    K1 = np.ascontiguousarray(inp.K[:1, :kv_heads])
    t0 = time.perf_counter()
    meta = oracle.block_meta(w.backbone, K1, nthreads=threads)
    S = oracle.tile_scores(w.backbone, Q1, meta, kv_heads, nthreads=threads)
    sums, terms = oracle.row_roughness(w.backbone, Q1, meta, kv_heads, nthreads=threads)
    units = oracle.all_units(1, nh, w.T)
    tau = np.array([[bai.noise_scale(sums[units[:, 1] == h], terms[units[:, 1] == h])
                     for h in range(nh)]], np.float32)
    z = synth_normals(w, n_s)
    gaps = bai.tile_gaps(S, w.k)
    fk, fr = bai.mc_counts(S, w.k, tau, z)
    bai.head_stats(gaps, fk, fr, tau, w.q, w.k, n_s)
    secs = time.perf_counter() - t0
    return {"value": round(nh * w.T / secs, 3), "unit": "units/s", "cores": threads, "kind": "oracle",
            "seconds": round(secs, 2),
            "sample": f"batch 0, query heads 0..{nh - 1} ({kv_heads} kv heads) of {w.name}: their "
                      f"{nh * w.T} tiles through metadata, tile scores, row roughness, gaps, "
                      f"{n_s}-sample Monte Carlo and head aggregates",
            **{k: v for k, v in hc.items() if k != "threads"}}


def synth_normals(w, n_s):
    from paper_2607_07724_amd import synth
    return synth.mc_normals(w.seed(), n_s, w.NB)


def measured_peaks(torch, dev, stream):
    """Practical ceilings measured on this GPU: a streaming elementwise add
    (1 GiB read + 1 GiB written) and a large bf16 GEMM (8192^3)."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    src = torch.ones(1 << 29, dtype=torch.int16, device=dev)
    dst = torch.empty_like(src)
    torch.add(src, 1, out=dst)
    torch.cuda.synchronize(dev)
    e0.record(stream)
    for _ in range(5):
        torch.add(src, 1, out=dst)
    e1.record(stream)
    torch.cuda.synchronize(dev)
    copy_gbps = 5 * 2 * (1 << 30) / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    n = 8192
    A = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    B = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
    C = A @ B
    torch.cuda.synchronize(dev)
    e0.record(stream)
    for _ in range(10):
        torch.matmul(A, B, out=C)
    e1.record(stream)
    torch.cuda.synchronize(dev)
    gemm = 10 * 2.0 * n ** 3 / (e0.elapsed_time(e1) * 1e-3) / 1e12
    del A, B, C
    loops = mfma_loop_peaks(torch, dev, stream)
    fill = lds_fill_rates(torch, dev, stream)
    return {"copy_GBps": round(copy_gbps, 1), "gemm_bf16_TFLOPs": round(gemm, 1), **loops, "lds_fill": fill,
            "copy": "torch elementwise add, 1 GiB in + 1 GiB out", "gemm": "torch.matmul bf16 8192^3",
            "mfma_loop": "libugbs_probe: 2048 workgroups x 4 waves, back-to-back 16x16x32 bf16 MFMA "
                         "(dense) or 16x16x64 bf16 2:4-sparse MFMA (dense-equivalent FLOP) on 8 "
                         "accumulator chains per wave, operands toggling every iteration"}


def lds_fill_rates(torch, dev, stream, iters=800):
    """The attention kernel's staging path on its own: 16 KiB tiles chosen at
    random from a region that fits one XCD's L2 (2 MiB), the memory-side
    cache (64 MiB) or neither (2 GiB), streamed into LDS by direct loads,
    four 2-wave workgroups per CU with two tiles in flight each.  Bytes per
    second, and per clock and CU at the clock the kernel ran at."""
    import ctypes
    from paper_2607_07724_amd import build
    if not os.path.exists(build.PROBE_LIB):
        return None
    L = ctypes.CDLL(build.PROBE_LIB)
    L.ugbs_probe_fill.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_uint, ctypes.c_int, ctypes.c_int,
                                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    L.ugbs_probe_out_floats.argtypes = [ctypes.c_int]
    n_cu = torch.cuda.get_device_properties(dev).multi_processor_count
    n_wg = 4 * n_cu
    src = torch.ones(1 << 30, dtype=torch.int16, device=dev)      # 2 GiB
    clk = torch.zeros(2, dtype=torch.int64, device=dev)
    out = torch.empty(L.ugbs_probe_out_floats(n_wg), dtype=torch.float32, device=dev)
    st = ctypes.c_void_p(stream.cuda_stream)
    res = {}
    for name, mib in (("l2_resident_2MiB", 2), ("memory_side_cache_64MiB", 64), ("hbm_2GiB", 2048)):
        args = (2, ctypes.c_void_p(src.data_ptr()), mib * 64, n_wg, iters, ctypes.c_void_p(clk.data_ptr()),
                ctypes.c_void_p(out.data_ptr()), st)
        assert L.ugbs_probe_fill(*args) == 0
        torch.cuda.synchronize(dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        assert L.ugbs_probe_fill(*args) == 0
        e1.record(stream)
        torch.cuda.synchronize(dev)
        sec = e0.elapsed_time(e1) * 1e-3
        ticks, real = clk.cpu().tolist()
        ghz = ticks / (real / 100e6) / 1e9 if real > 0 else None
        by = n_wg * iters * 16384
        res[name] = {"TBps": round(by / sec / 1e12, 2), "clock_GHz": round(ghz, 2) if ghz else None,
                     "bytes_per_clk_per_cu": round(by / sec / n_cu / (ghz * 1e9), 1) if ghz else None}
    del src, out
    res["pattern"] = "16 KiB tiles, random per workgroup, direct-to-LDS, 4 x 2-wave workgroups per CU, 2 tiles in flight"
    return res


def mfma_loop_peaks(torch, dev, stream, n_wg=2048, iters=4000, reps=5):
    """Matrix-core ceilings of this GPU under a sustained load: TFLOP/s of a
    tight loop of dense and of 2:4-sparse bf16 matrix instructions."""
    import ctypes
    from paper_2607_07724_amd import build
    if not os.path.exists(build.PROBE_LIB):
        log(f"{build.PROBE_LIB} is not built: no matrix-core loop ceilings")
        return {"mfma_loop_bf16_TFLOPs": None, "smfmac_loop_bf16_TFLOPs": None}
    L = ctypes.CDLL(build.PROBE_LIB)
    L.ugbs_probe_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    L.ugbs_probe_flop.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int]
    L.ugbs_probe_flop.restype = ctypes.c_double
    L.ugbs_probe_out_floats.argtypes = [ctypes.c_int]
    out = torch.empty(L.ugbs_probe_out_floats(n_wg), dtype=torch.float32, device=dev)
    st = ctypes.c_void_p(stream.cuda_stream)
    res = {}
    for kind, key in ((0, "mfma_loop_bf16_TFLOPs"), (1, "smfmac_loop_bf16_TFLOPs")):
        assert L.ugbs_probe_mfma(kind, n_wg, iters, ctypes.c_void_p(out.data_ptr()), st) == 0
        torch.cuda.synchronize(dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            assert L.ugbs_probe_mfma(kind, n_wg, iters, ctypes.c_void_p(out.data_ptr()), st) == 0
        e1.record(stream)
        torch.cuda.synchronize(dev)
        res[key] = round(reps * L.ugbs_probe_flop(kind, n_wg, iters) / (e0.elapsed_time(e1) * 1e-3) / 1e12, 1)
    del out
    return res


def run_stack(torch, dev, ugbs, synth, steps):
    """28-layer attention-only stack at the 28/4-head d 128 shape, N = 131072:
    per-layer inputs (independent seeds) resident in HBM, per-layer quantile;
    routed pipeline for both backbones vs dense causal attention, summed over
    the layers."""
    import torch.nn.functional as F
    w0 = synth.WORKLOADS["C5"]
    L = w0.layers
    t0 = time.time()
    layers = []
    for layer in range(L):
        inp = synth.generate(w0, layer=layer, threads=16)
        cv = lambda x: torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)
        layers.append((cv(inp.Q), cv(inp.K), cv(inp.V)))
        del inp
        if layer % 7 == 6:
            log(f"stack: {layer + 1}/{L} layers generated and uploaded ({time.time() - t0:.0f}s)")
    stream = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    out = {"layers": L, "workload": "C5: 28-layer stack, 28 q / 4 kv heads, d 128, N 131072, k 64, q 0.1"}
    O = torch.empty_like(layers[0][0])
    for name, bb in (("kmean", synth.KMEAN), ("quest", synth.QUEST)):
        p = ugbs.Problem.make(w0.B, w0.H, w0.Hkv, w0.N, w0.d, w0.k, w0.q, bb)
        bufs = ugbs.Buffers(p, device=dev)
        for Q, K, V in layers[:2]:
            ugbs.prefill(p, Q, K, V, O, bufs)
        torch.cuda.synchronize(dev)
        reps = max(1, steps)
        e0.record(stream)
        for _ in range(reps):
            for Q, K, V in layers:
                ugbs.prefill(p, Q, K, V, O, bufs)
        e1.record(stream)
        torch.cuda.synchronize(dev)
        ms = e0.elapsed_time(e1) / reps
        out[name] = {"routed_ms": round(ms, 2), "per_layer_ms": round(ms / L, 3), "passes": reps}
        log(f"stack {name}: {ms:.1f} ms per 28-layer pass")
        del bufs
    G = w0.H // w0.Hkv
    try:
        from torch.nn.attention import SDPBackend, sdpa_kernel
        with sdpa_kernel([SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION]):
            Ke, Ve = layers[0][1].repeat_interleave(G, dim=1), layers[0][2].repeat_interleave(G, dim=1)
            F.scaled_dot_product_attention(layers[0][0], Ke, Ve, is_causal=True)
            torch.cuda.synchronize(dev)
            del Ke, Ve
            # GQA heads expanded per layer outside the timed windows (as in the single-layer leg)
            sd = 0.0
            for Q, K, V in layers:
                Ke, Ve = K.repeat_interleave(G, dim=1), V.repeat_interleave(G, dim=1)
                torch.cuda.synchronize(dev)
                e0.record(stream)
                F.scaled_dot_product_attention(Q, Ke, Ve, is_causal=True)
                e1.record(stream)
                torch.cuda.synchronize(dev)
                sd += e0.elapsed_time(e1)
                del Ke, Ve
        out["dense_sdpa_ms"] = round(sd, 1)
        for name in ("kmean", "quest"):
            out[name]["routed_over_sdpa"] = round(out[name]["routed_ms"] / sd, 4)
    except Exception as ex:
        log(f"stack SDPA failed: {ex!r}")
    kvd = torch.from_numpy(synth.dense_kv_idx(w0.B, w0.H, w0.T)).to(dev)
    pd = ugbs.Problem.make(w0.B, w0.H, w0.Hkv, w0.N, w0.d, w0.NB, 0.0, w0.backbone, rho=1)
    e0.record(stream)
    for Q, K, V in layers:
        ugbs.ugbs_attend(pd, Q, K, V, kvd, O)
    e1.record(stream)
    torch.cuda.synchronize(dev)
    out["dense_ugbs_ms"] = round(e0.elapsed_time(e1), 1)
    del layers, O, kvd
    torch.cuda.empty_cache()
    log(f"stack: {out}")
    return out


def cpu_sample_units(w, n_units):
    """The (batch, head, tile) units the CPU leg samples: random heads and
    tiles of the quantile population (t >= k)."""
    g = np.random.default_rng(w.seed(0))
    return np.stack([g.integers(0, w.B, n_units).astype(np.int32),
                     g.integers(0, w.H, n_units).astype(np.int32),
                     g.integers(w.k, w.T, n_units).astype(np.int32)], axis=1)


def cpu_baseline(w, inp, units, gpu_kv, gpu_trig, gpu_O_units, threads=None):
    """The reference oracle on a bounded sample of the same workload, timed
    on the host cores: block metadata for every kv head, then tile scores,
    sorted top-2k + sigma, and exact fp64 attention for the sampled (tile,
    head) units over the GPU's kv_idx rows of those units (the route needs
    every tile, so the GPU's trigger flags cut the oracle's lists).  The same
    computation checks the GPU run on the sample: kv_idx rows against the
    oracle's under the near-tie rule, and the GPU's output against the
    oracle's attention (max-abs 2e-2, RMS 2e-3)."""
    import oracle
    from oracle.compare import near_tie_ok
    hc = host_cores(threads)
    nt = hc["threads"]
    t0 = time.perf_counter()
    meta = oracle.block_meta(w.backbone, inp.K, nthreads=nt)
    t1 = time.perf_counter()
    S = oracle.tile_scores(w.backbone, inp.Q, meta, w.Hkv, units=units, nthreads=nt)
    idx, sig = oracle.select(S, w.k, t_of_row=units[:, 2], rho=w.rho)
    t2 = time.perf_counter()
    g_rows = np.stack([gpu_kv[b, h, t] for b, h, t in units])
    ref = oracle.attend(inp.Q, inp.K, inp.V, kv_idx=g_rows, units=units, nthreads=nt)
    t3 = time.perf_counter()
    KD = w.d * (2 if w.backbone == 1 else 1)
    f_sc = float(sum(2 * KD * 64 * max(int(t) - 1, 0) for t in units[:, 2]))
    # every row lists its own (diagonal) block plus n - 1 earlier ones
    f_at = float(sum(4 * w.d * (64 * 64 * (int((r != w.NB).sum()) - 1) + 64 * 65 // 2) for r in g_rows))
    secs = t3 - t0
    # parity on the sample
    bad = exempt = equal = 0
    for i, (b, h, t) in enumerate(units):
        width = w.rho * w.k if gpu_trig[b, t] else w.k
        orow = idx[i].copy()
        orow[width:] = w.NB
        ok, nd = near_tie_ok(g_rows[i], orow, S[i], int(t), w.NB, w.k)
        bad += not ok
        exempt += ok and nd > 0
        equal += ok and nd == 0
    got = (gpu_O_units.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    d = got - ref
    mx, rms = float(np.abs(d).max()), float(np.sqrt(np.mean(d * d)))
    return {
        "value": round((f_sc + f_at) / secs / 1e12, 6),
        "unit": "TFLOP/s",
        "cores": nt,
        "kind": "oracle",
        "seconds": round(secs, 2),
        "seconds_meta_scores_attend": [round(t1 - t0, 2), round(t2 - t1, 2), round(t3 - t2, 2)],
        "sample": f"block metadata for all {w.B * w.Hkv} kv heads, then scores + sorted top-2k + sigma "
                  f"and exact fp64 attention (over the GPU's kv_idx rows) for {len(units)} random "
                  f"(tile >= k, head) units of the same {w.name} inputs; the route needs every tile "
                  f"and is not part of the sample",
        **{k: v for k, v in hc.items() if k != "threads"},
        "parity": {"units": int(len(units)), "kv_rows_equal": int(equal),
                   "kv_rows_near_tie_exempt": int(exempt), "kv_rows_beyond_near_ties": int(bad),
                   "attention_max_abs": mx, "attention_rms": rms,
                   "ok": bad == 0 and mx <= 2e-2 and rms <= 2e-3},
    }


def run_oracle_layers(a, torch, dev, ugbs, synth):
    """CPU-baseline leg over whole layers: the reference oracle on every
    tile and head of a workload's layers (default the 28-layer stack), its
    stage times on the host cores, and the GPU pipeline's kv_idx and output
    compared with it
    (kv_idx rows equal up to near-ties, trigger flips only within 1e-3 of
    tau, attention on the rows with equal lists within max-abs 2e-2 / RMS
    2e-3)."""
    import oracle
    from oracle.compare import near_tie_ok
    w = synth.WORKLOADS[a.workload or "C5"]
    if a.q is not None:
        w = w.replace(q=a.q)
    if a.oracle_backbone:
        w = w.replace(backbone=synth.QUEST if a.oracle_backbone == "quest" else synth.KMEAN)
    bb_name = "quest" if w.backbone == synth.QUEST else "kmean"
    hc = host_cores(a.oracle_threads)
    threads = hc["threads"]
    res = []
    for layer in [int(x) for x in a.oracle_layers.split(",")]:
        inp = synth.generate(w, layer=layer, threads=16)
        cv = lambda x: torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)
        Q, K, V = cv(inp.Q), cv(inp.K), cv(inp.V)
        p = ugbs.Problem.make(w.B, w.H, w.Hkv, w.N, w.d, w.k, w.q, w.backbone, rho=w.rho)
        bufs = ugbs.Buffers(p, device=dev)
        O = torch.empty_like(Q)
        ugbs.prefill(p, Q, K, V, O, bufs)
        torch.cuda.synchronize(dev)
        g_kv, g_trig = bufs.kv_idx.cpu().numpy(), bufs.trigger.cpu().numpy()
        g_O = O.view(torch.int16).cpu().numpy().view(np.uint16)
        del Q, K, V, bufs, O
        log(f"oracle layer {layer}: GPU pipeline done")
        t0 = time.perf_counter()
        meta = oracle.block_meta(w.backbone, inp.K, nthreads=threads)
        t1 = time.perf_counter()
        S = oracle.tile_scores(w.backbone, inp.Q, meta, w.Hkv, nthreads=threads)
        t2 = time.perf_counter()
        log(f"oracle layer {layer}: metadata {t1 - t0:.1f}s, tile scores {t2 - t1:.1f}s")
        idx, sig = oracle.select(S, w.k, rho=w.rho)
        kv, sb, tau, trig = oracle.route(sig, idx, w.k, w.q, rho=w.rho)
        t3 = time.perf_counter()
        log(f"oracle layer {layer}: selection + route {t3 - t2:.1f}s")
        units = oracle.all_units(w.B, w.H, w.T)
        ref = np.empty((len(units), 64, w.d), np.float64)
        n_parts = 16
        for i, part in enumerate(np.array_split(np.arange(len(units)), n_parts)):
            ref[part] = oracle.attend(inp.Q, inp.K, inp.V, kv_idx=kv.reshape(-1, kv.shape[-1])[part],
                                      units=units[part], nthreads=threads)
            log(f"oracle layer {layer}: attention {i + 1}/{n_parts} ({time.perf_counter() - t3:.0f}s)")
        t4 = time.perf_counter()
        # comparisons
        flips = int((g_trig != trig).sum())
        flips_ok = all(abs(float(sb[b, t]) - float(tau[b])) <= 1e-3 for b, t in zip(*np.nonzero(g_trig != trig)))
        rows_eq = (g_kv == kv).all(axis=-1)
        bad = 0
        for b, h, t in zip(*np.nonzero(~rows_eq)):
            width = w.rho * w.k if g_trig[b, t] else w.k
            orow = idx[b, h, t].copy()
            orow[width:] = w.NB
            bad += not near_tie_ok(g_kv[b, h, t], orow, S[b, h, t], int(t), w.NB, w.k)[0]
        gO = ((g_O.astype(np.uint32) << 16).view(np.float32).astype(np.float64)).reshape(len(units), 64, w.d)
        eq = rows_eq.reshape(-1)
        d = gO[eq] - ref[eq]
        mx, rms = float(np.abs(d).max()), float(np.sqrt(np.mean(d * d)))
        KD = w.d * (2 if w.backbone == synth.QUEST else 1)
        f_sc = float(sum(2 * KD * 64 * max(t - 1, 0) for t in range(w.T)) * w.B * w.H)
        f_at = float(sum(4 * w.d * (64 * 64 * (int((r != w.NB).sum()) - 1) + 64 * 65 // 2)
                         for r in kv.reshape(-1, kv.shape[-1])))
        r = {"layer": layer, "backbone": bb_name,
             "oracle_seconds": {"meta": round(t1 - t0, 2), "scores": round(t2 - t1, 2),
                                "select_route": round(t3 - t2, 2), "attend": round(t4 - t3, 2),
                                "total": round(t4 - t0, 2)},
             "oracle_TFLOPs": round((f_sc + f_at) / (t4 - t0) / 1e12, 6), "cores": threads,
             "rows": int(rows_eq.size), "rows_equal": int(rows_eq.sum()),
             "rows_differing_beyond_near_ties": bad, "trigger_flips": flips,
             "trigger_flips_within_1e-3_of_tau": flips_ok,
             "attention_on_equal_rows": {"max_abs": mx, "rms": rms},
             "parity_ok": bad == 0 and flips_ok and mx <= 2e-2 and rms <= 2e-3}
        log(f"oracle layer {layer}: {r}")
        res.append(r)
        del S, ref, gO, inp
    print(json.dumps({"mode": "oracle_full_layers",
                      "workload": {"name": w.name, "batch": w.B, "q_heads": w.H, "kv_heads": w.Hkv,
                                   "head_dim": w.d, "seq_len": w.N, "k_budget": w.k, "q": w.q,
                                   "rho": w.rho, "backbone": bb_name},
                      **{k: v for k, v in hc.items() if k != "threads"}, "layers": res}), flush=True)


def _cpu_name():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


if __name__ == "__main__":
    main()
