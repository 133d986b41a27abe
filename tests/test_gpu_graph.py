"""The static-mask plan path under HIP graph capture.

sa_bsattn_fwd_plan enqueues only the attention kernel (no allocation, no
memset, no synchronisation), so a caller can capture it into a graph and
replay it.  The test captures it on torch's capture stream, replays the graph
several times with other eager work and synchronisations in between, and
checks every replay bit for bit against the eager call.
"""

import numpy as np
import pytest

from workloads import pack_rows

pytestmark = pytest.mark.gpu


def test_plan_forward_replays_in_a_graph():
    import torch
    from paper_2606_23019_amd import binding
    assert torch.cuda.is_available()
    B, H, N, d, blk = 2, 3, 1000, 128, 128
    n = -(-N // blk)
    rng = np.random.default_rng(7)
    bm = rng.random((H, n, n)) < 0.4
    bm[:, np.arange(n), np.arange(n)] = True
    packed = pack_rows(bm)
    g = torch.Generator(device="cuda")
    g.manual_seed(8)
    q, k, v = (torch.randn((B, H, N, d), generator=g, device="cuda").to(torch.bfloat16)
               for _ in range(3))
    plan = binding.Plan(packed, B, H, N, blk, blk)
    ref_out, ref_lse = plan(q, k, v)
    torch.cuda.synchronize()

    out = torch.zeros_like(q)
    lse = torch.zeros((B, H, N), dtype=torch.float32, device="cuda")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):           # warm-up outside the graph
        plan(q, k, v, out=out, lse=lse)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        plan(q, k, v, out=out, lse=lse)
    for rep in range(4):
        out.fill_(float("nan"))
        lse.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        junk = (q.float() * 2).sum()        # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(out, ref_out) and torch.equal(lse, ref_lse), "replay %d" % rep
        assert torch.isfinite(junk).item()
    del graph
    plan.close()
