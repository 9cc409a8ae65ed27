"""The benchmark's ceiling probes (libugbs_probe.so) run and report sane
values: the matrix-instruction loops leave finite accumulator sums, and the
LDS-fill loop records both clock counters and keeps LDS contents that are
the source tile's (every element of the source is 1.0 in bf16)."""
import ctypes
import math
import os

import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def probe():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need an MI355X (gfx950) visible to torch")
    from paper_2607_07724_amd import build
    if not os.path.exists(build.PROBE_LIB):
        pytest.fail(f"{build.PROBE_LIB} is not built")
    L = ctypes.CDLL(build.PROBE_LIB)
    L.ugbs_probe_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    L.ugbs_probe_fill.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_uint, ctypes.c_int, ctypes.c_int,
                                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    L.ugbs_probe_out_floats.argtypes = [ctypes.c_int]
    return torch, L


@pytest.mark.parametrize("kind", [0, 1])
def test_mfma_loop_sums_are_finite(probe, kind):
    torch, L = probe
    n_wg = 16
    out = torch.full((L.ugbs_probe_out_floats(n_wg),), float("nan"), dtype=torch.float32, device="cuda")
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    assert L.ugbs_probe_mfma(kind, n_wg, 20, ctypes.c_void_p(out.data_ptr()), st) == 0
    torch.cuda.synchronize()
    assert bool(torch.isfinite(out).all())


@pytest.mark.parametrize("depth", [1, 2])
def test_fill_loop_records_clocks_and_tiles(probe, depth):
    torch, L = probe
    n_wg, n_tiles = 32, 16
    src = torch.ones(n_tiles * 8192, dtype=torch.bfloat16, device="cuda")      # 16 tiles of 16 KiB
    clk = torch.zeros(2, dtype=torch.int64, device="cuda")
    out = torch.zeros(L.ugbs_probe_out_floats(n_wg), dtype=torch.float32, device="cuda")
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    assert L.ugbs_probe_fill(depth, ctypes.c_void_p(src.data_ptr()), n_tiles, n_wg, 10,
                             ctypes.c_void_p(clk.data_ptr()), ctypes.c_void_p(out.data_ptr()), st) == 0
    torch.cuda.synchronize()
    ticks, real = clk.cpu().tolist()
    assert ticks > 0 and real > 0
    ghz = ticks / (real / 100e6) / 1e9
    assert 0.5 < ghz < 4.0, ghz
    # out[128 wg + i] is the 16-bit pattern of LDS element i of workgroup wg
    # as a float (bf16 1.0 = 0x3F80); the fill loop writes 128 per workgroup
    got = out[: 128 * n_wg]
    assert bool((got == float(0x3F80)).all()), got[:8]
    assert not math.isnan(float(got.sum()))
