"""The layer captured in a HIP graph and replayed.

Every entry point enqueues on the caller's stream and neither allocates,
synchronises nor clears memory with memset nodes, so the four calls of a
layer (and of the fused variant) can be captured once and replayed.  Each
replay is checked bit for bit against the eager layer on the same inputs,
with eager kernels that overwrite the outputs in between the replays.
"""
import numpy as np
import pytest
import torch

import paper_2607_07724_amd as ugbs
from paper_2607_07724_amd import synth

from gpu_helpers import dev_bf16

pytestmark = pytest.mark.gpu

WORKLOADS = {
    "C1": synth.WORKLOADS["C1"],
    # 8 / 2 heads, d 128, N 8192, Quest, k 8, q 0.3: several tiles per XCD
    "mid": synth.Workload("mid", 1, 8, 2, 128, 8192, 8, 0.3, synth.QUEST, "mixture", needles=4),
}


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs an MI355X (gfx950)")


@pytest.mark.parametrize("name", sorted(WORKLOADS))
@pytest.mark.parametrize("fused", [False, True])
def test_graph_replays_equal_the_eager_layer(name, fused):
    _need_gpu()
    w = WORKLOADS[name]
    inp = synth.generate(w, threads=4)
    Q, K, V = dev_bf16(inp.Q), dev_bf16(inp.K), dev_bf16(inp.V)
    p = ugbs.Problem.make(w.B, w.H, w.Hkv, w.N, w.d, w.k, w.q, w.backbone)
    run = ugbs.prefill_fused if fused else ugbs.prefill

    bufs_e = ugbs.Buffers(p)
    O_e = torch.empty_like(Q)
    run(p, Q, K, V, O_e, bufs_e)
    torch.cuda.synchronize()

    bufs_g = ugbs.Buffers(p)
    O_g = torch.empty_like(Q)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):          # warm-up outside the capture
        run(p, Q, K, V, O_g, bufs_g)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run(p, Q, K, V, O_g, bufs_g)
    torch.cuda.synchronize()

    for rep in range(3):
        # eager work between the replays: clobber every output
        O_g.fill_(float("nan"))
        bufs_g.sigma.fill_(-7.0)
        bufs_g.trigger.fill_(3)
        if not fused:
            bufs_g.kv_idx.fill_(-5)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(O_g.view(torch.int16), O_e.view(torch.int16)), (name, fused, rep)
        assert torch.equal(bufs_g.sigma.view(torch.int32), bufs_e.sigma.view(torch.int32)), (name, fused, rep)
        assert torch.equal(bufs_g.trigger, bufs_e.trigger), (name, fused, rep)
        if not fused:
            assert torch.equal(bufs_g.kv_idx, bufs_e.kv_idx), (name, fused, rep)
