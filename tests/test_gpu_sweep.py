"""Parity at the density / block-size sweep's own shape (H40, N32768, d128).

Each point builds its masks with the sweep's generator and runs the prepared
call that the sweep times (pre-pass, schedule, then the attention kernel
alone), plus a plan with float32 out on the same inputs.  16 seeded query
blocks per point are checked against the float64 reference: the bf16 out with
the allowance for its own rounding, the float32 out against the plain bounds
with none.  The plan's bf16 out must equal the prepared call's bit for bit,
and the float32 out must round to it.
"""

import numpy as np
import pytest

from helpers import compare, compare_strict, gather_rows, reference_items
from workloads import masks_for, qkv_for, sample_items, sweep_point

pytestmark = pytest.mark.gpu

POINTS = [(rho, blk, kind) for blk in (64, 128) for kind in ("structured", "uniform")
          for rho in (0.05, 0.5)]


@pytest.mark.parametrize("rho,blk,kind", POINTS, ids=lambda x: str(x))
def test_sweep_point_parity(rho, blk, kind):
    import torch
    from paper_2606_23019_amd import binding
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    wl = sweep_point(rho, blk, kind)
    packed, bm, dens = masks_for(wl)
    q, k, v = qkv_for(wl, device="cuda")
    mask = binding.mask_to_device(packed)
    counts, lists = binding.mask_prepass(mask, wl.H, wl.n_qb, wl.n_kb)
    order = binding.schedule(counts, wl.B, wl.H, wl.n_qb)
    out, lse = binding.bsattn_fwd_prepared(q, k, v, counts, lists, order, blk, blk, wl.scale)
    plan = binding.Plan(packed, wl.B, wl.H, wl.N, blk, blk)
    assert plan.executed_blocks == int(bm.sum())
    o_plan, l_plan = plan(q, k, v, wl.scale)
    out32, lse32 = plan.fwd_f32out(q, k, v, wl.scale)
    torch.cuda.synchronize()
    plan.close()
    assert torch.equal(o_plan.view(torch.int16), out.view(torch.int16))
    assert torch.equal(l_plan, lse) and torch.equal(lse32, lse)
    assert torch.equal(out32.to(torch.bfloat16).view(torch.int16), out.view(torch.int16))
    items = sample_items(wl, bm, 16)
    ref = reference_items(q, k, v, packed, blk, blk, wl.scale, items)
    ro = np.concatenate([ref[it][0] for it in items])
    rl = np.concatenate([ref[it][1] for it in items])
    gl = gather_rows(lse, items, blk, wl.N)
    stats = compare(gather_rows(out, items, blk, wl.N), gl, ro, rl)
    strict = compare_strict(gather_rows(out32, items, blk, wl.N), gl, ro, rl)
    print(wl.name, "density %.4f" % dens.mean(), "bf16", stats, "fp32 out", strict)
    del q, k, v, out, lse, o_plan, l_plan, out32, lse32
    torch.cuda.empty_cache()
