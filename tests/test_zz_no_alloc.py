"""ugbs_route_noalloc (the route for callers that cannot allocate) against
ugbs_route and the oracle's route, through the C ABI: two calls in a row on
one GPU, the second with a smaller problem (the static scratch then holds
the first call's larger contents), in place, out of place and flags only.
Every output must be bit-identical."""
import ctypes

import numpy as np
import pytest

import oracle
import paper_2607_07724_amd as ugbs

from gpu_helpers import dev, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need an MI355X (gfx950) visible to torch")
    ugbs.lib()


def _inputs(B, H, T, k, rho, seed, levels):
    """Oracle selection on random tile scores with heavy ties (so sigma_bar
    ties at tau occur): sigma [B,H,T] and idx_sorted [B,H,T,rho k]."""
    g = np.random.default_rng(seed)
    S = np.round(g.normal(0, 1, (B, H, T, T)) * levels) / levels
    S = S.astype(np.float32)
    idx, sig = oracle.select(S, k, rho=rho)
    return sig, idx


def _call_noalloc(p, sigma, idx, kv, sb, tau, trig):
    L = ugbs.lib()
    ptr = lambda t: None if t is None else ctypes.c_void_p(t.data_ptr())
    import torch
    st = L.ugbs_route_noalloc(ctypes.byref(p), ptr(sigma), ptr(idx), ptr(kv), ptr(sb), ptr(tau), ptr(trig),
                              ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, ugbs.ugbs_status_string(st)


def _call_route(p, sigma, idx, kv, sb, tau, trig, ws):
    L = ugbs.lib()
    ptr = lambda t: None if t is None else ctypes.c_void_p(t.data_ptr())
    import torch
    st = L.ugbs_route(ctypes.byref(p), ptr(sigma), ptr(idx), ptr(kv), ptr(sb), ptr(tau), ptr(trig), ptr(ws),
                      ws.numel(), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, ugbs.ugbs_status_string(st)


def _check_case(B, H, T, k, q, rho, seed, levels):
    import torch
    N = 64 * T
    p = ugbs.Problem.make(B, H, 1, N, 64, k, q, ugbs.KMEAN, rho=rho)
    sig, idx = _inputs(B, H, T, k, rho, seed, levels)
    kv_o, sb_o, tau_o, trig_o = oracle.route(sig, idx, k, q, rho=rho)
    W = rho * k
    sigma = dev(sig)
    out = {}
    for name in ("noalloc", "route"):
        idx_d = dev(idx)
        kv = torch.empty((B, H, T, W), dtype=torch.int32, device="cuda")
        sb = torch.empty((B, T), dtype=torch.float32, device="cuda")
        tau = torch.empty((B,), dtype=torch.float32, device="cuda")
        trig = torch.empty((B, T), dtype=torch.uint8, device="cuda")
        idx_ip = dev(idx)
        sb2 = torch.empty_like(sb)
        tau2 = torch.empty_like(tau)
        trig2 = torch.empty_like(trig)
        trig3 = torch.empty_like(trig)
        if name == "noalloc":
            _call_noalloc(p, sigma, idx_d, kv, sb, tau, trig)            # out of place
            _call_noalloc(p, sigma, idx_ip, idx_ip, sb2, tau2, trig2)    # in place
            _call_noalloc(p, sigma, None, None, None, None, trig3)       # flags only
        else:
            ws = torch.empty((ugbs.ugbs_workspace_bytes(p),), dtype=torch.uint8, device="cuda")
            _call_route(p, sigma, idx_d, kv, sb, tau, trig, ws)
            _call_route(p, sigma, idx_ip, idx_ip, sb2, tau2, trig2, ws)
            _call_route(p, sigma, None, None, None, None, trig3, ws)
        torch.cuda.synchronize()
        out[name] = [host(x) for x in (kv, sb, tau, trig, idx_ip, sb2, tau2, trig2, trig3)]
    a, b = out["noalloc"], out["route"]
    for x, y in zip(a, b):
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8))
    kv, sb, tau, trig, kv_ip, sb2, tau2, trig2, trig3 = a
    assert np.array_equal(kv, kv_o) and np.array_equal(kv_ip, kv_o)
    assert np.array_equal(sb.view(np.uint32), sb_o.view(np.uint32))
    assert np.array_equal(tau.view(np.uint32), tau_o.view(np.uint32))
    assert np.array_equal(trig.astype(bool), trig_o) and np.array_equal(trig2, trig) and np.array_equal(trig3, trig)
    return int(trig.sum())


def test_noalloc_route_equals_route_twice_second_smaller():
    n1 = _check_case(B=2, H=8, T=256, k=8, q=0.3, rho=2, seed=11, levels=3)
    n2 = _check_case(B=1, H=4, T=40, k=5, q=0.5, rho=3, seed=12, levels=2)
    assert n1 > 0 and n2 > 0


def test_noalloc_route_at_the_largest_batch_the_scratch_holds():
    """Batch 64 at T = 2048 (N = 131072) fills 656 KB of the 1 MiB array."""
    import torch
    B, H, T, k, q = 64, 1, 2048, 64, 0.1
    p = ugbs.Problem.make(B, H, 1, 64 * T, 64, k, q, ugbs.KMEAN)
    g = np.random.default_rng(5)
    sig = np.round(g.random((B, H, T)) * 50).astype(np.float32) / 50
    sig[:, :, :k] = -1.0                                            # saturated tiles (outside the population)
    sigma = dev(sig)
    trig_a = torch.empty((B, T), dtype=torch.uint8, device="cuda")
    trig_b = torch.empty_like(trig_a)
    sb_a = torch.empty((B, T), dtype=torch.float32, device="cuda")
    sb_b = torch.empty_like(sb_a)
    ws = torch.empty((ugbs.ugbs_workspace_bytes(p),), dtype=torch.uint8, device="cuda")
    _call_noalloc(p, sigma, None, None, sb_a, None, trig_a)
    _call_route(p, sigma, None, None, sb_b, None, trig_b, ws)
    torch.cuda.synchronize()
    assert torch.equal(trig_a, trig_b) and torch.equal(sb_a.view(torch.int32), sb_b.view(torch.int32))
    assert int(trig_a.sum()) >= 64 * int(np.ceil(q * (T - k)))
