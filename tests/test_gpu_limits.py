"""GPU parity at the largest sizes the ABI accepts: N_B = 4096 blocks (N =
262144; and 2048, the largest that keeps 32 candidates per lane) and kv_idx
rows of up to 4096 slots (rho k = UGBS_MAX_KV_WIDTH).

Selection on given tile scores and the route are compared with the oracle
bit for bit; the budgets reach R = rho k - |F| far above the 128 winners
the register sort handles (the LDS sort path), up to every candidate of
the last tile.  Attention over 4096-slot rows is compared with the oracle
on sampled tiles (the full fp64 oracle at this size takes minutes).
"""
import numpy as np
import pytest

import oracle
import paper_2607_07724_amd as ugbs
from paper_2607_07724_amd import synth

from gpu_helpers import attention_error, dev, dev_bf16, host, host_bits

pytestmark = pytest.mark.gpu
ATOL_MAX, ATOL_RMS = 2e-2, 2e-3
B, H, HKV, D, N = 1, 2, 1, 64, 131072
NB = N // 64


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need an MI355X (gfx950) visible to torch")
    ugbs.lib()  # raises if the HIP library is missing


_scores = {}


def scores(nb=NB):
    """[B, H, T, N_B] fp32 tile scores with heavy ties and signed zeros on
    one head and distinct values on the other."""
    if nb not in _scores:
        g = np.random.default_rng(2048 + nb)
        S = np.empty((B, H, nb, nb), np.float32)
        S[0, 0] = np.round(g.standard_normal((nb, nb)) * 3.0)   # small integers: many ties
        S[0, 0][g.random((nb, nb)) < 0.05] = -0.0
        S[0, 1] = g.standard_normal((nb, nb)).astype(np.float32)
        _scores[nb] = S
    return _scores[nb]


@pytest.mark.parametrize("nb", [2048, 4096])
@pytest.mark.parametrize("k,rho", [(3, 2), (64, 2), (700, 2), (1024, 2), (2048, 2), (512, 8), (1365, 3), (4096, 1)])
def test_selection_and_route_at_maximum_width(k, rho, nb):
    torch = __import__("torch")
    N, NB = 64 * nb, nb
    S = scores(nb)
    p = ugbs.Problem.make(B, H, HKV, N, D, k, 0.1, synth.KMEAN, rho=rho)
    assert p.W == rho * k <= ugbs.MAX_KV_WIDTH
    Q = torch.zeros((B, H, N, D), dtype=torch.bfloat16, device="cuda")
    meta = torch.zeros((B, HKV, NB, D, 1), dtype=torch.bfloat16, device="cuda")
    idx = torch.empty((B, H, NB, p.W), dtype=torch.int32, device="cuda")
    sig = torch.empty((B, H, NB), dtype=torch.float32, device="cuda")
    ugbs.ugbs_score_select(p, Q, meta, idx, sig, scores_in=dev(S))
    torch.cuda.synchronize()
    ridx, rsig = oracle.select(S, k, rho=rho)
    assert np.array_equal(host(idx), ridx)
    assert np.array_equal(host(sig).view(np.uint32), rsig.view(np.uint32))
    for q in (0.1, 1.0):
        pq = ugbs.Problem.make(B, H, HKV, N, D, k, q, synth.KMEAN, rho=rho)
        kv = torch.full_like(idx, -7)
        sb = torch.empty((B, NB), dtype=torch.float32, device="cuda")
        tau = torch.empty((B,), dtype=torch.float32, device="cuda")
        trig = torch.empty((B, NB), dtype=torch.uint8, device="cuda")
        ws = torch.empty((max(ugbs.ugbs_workspace_bytes(pq), 256),), dtype=torch.uint8, device="cuda")
        ugbs.ugbs_route(pq, dev(rsig), dev(ridx), kv, ws, sb, tau, trig)
        torch.cuda.synchronize()
        kv_ref, sb_ref, tau_ref, trig_ref = oracle.route(rsig, ridx, k, q, rho=rho)
        assert np.array_equal(host(kv), kv_ref)
        assert np.array_equal(host(sb).view(np.uint32), sb_ref.view(np.uint32))
        assert np.array_equal(host(tau).view(np.uint32), tau_ref.view(np.uint32))
        assert np.array_equal(host(trig), trig_ref)


def test_attention_over_4096_slot_rows_on_sampled_tiles():
    torch = __import__("torch")
    w = synth.Workload("limits", B, H, HKV, D, N, 2048, 0.1, synth.KMEAN, "offset", base_seed=2049)
    inp = synth.generate(w, threads=16)
    # 4096 slots per row: random visible blocks (up to all of them), junk entries, sentinels
    kv = synth.random_kv_idx(2050, B, H, NB, ugbs.MAX_KV_WIDTH, shuffle=True, junk=True)
    p = ugbs.Problem.make(B, H, HKV, N, D, 2048, 0.1, synth.KMEAN)
    Q, K, V = dev_bf16(inp.Q), dev_bf16(inp.K), dev_bf16(inp.V)
    O = torch.empty_like(Q)
    ugbs.ugbs_attend(p, Q, K, V, dev(kv), O)
    torch.cuda.synchronize()
    Ob = host_bits(O)
    g = np.random.default_rng(2051)
    ts = np.concatenate([[0, 1, NB - 1], g.choice(NB, 13, replace=False)])
    units = np.array([(0, h, int(t)) for h in range(H) for t in ts], np.int32)
    ref = oracle.attend(inp.Q, inp.K, inp.V, kv_idx=kv[0][units[:, 1], units[:, 2]], units=units)
    for i, (b, h, t) in enumerate(units):
        mx, rms = attention_error(Ob[b, h, 64 * t:64 * t + 64], ref[i])
        assert mx <= ATOL_MAX and rms <= ATOL_RMS, (h, t, mx, rms)
