#!/usr/bin/env python3
"""Benchmark of the block-sparse attention forward on one MI355X.

A step is one call of ``sa_bsattn_fwd`` (mask pre-pass, schedule and the
attention kernel) on resident inputs of the Wan2.1-14B-like 480p shape
(B=1, H=40, N=32768, d=128, 128 x 128 blocks, structured per-head masks with
density U[0.05, 0.6]).  The metric is effective TFLOP/s: 4 * 128 * 128 * 128
flops per executed (enabled) block divided by the step time.

Printed (one JSON line on stdout): the metric, the fraction of the bf16 MFMA
peak, speedup over the same kernel with an all-ones mask, a roofline record
for the attention kernel (timed with events on the stream it runs on) and the
CPU reference timed on a bounded sample of the same workload.

  python bench.py [--steps K] [--warmup W] [--workload 14b-480p]
  python bench.py --sweep out.json     # density / block sweep, extra file
"""

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0          # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "attn_fwd_14b480p_hbm_traffic.txt")
# The sources whose change invalidates the committed counter summary: the
# attention kernel, and the pre-pass/schedule file, whose launch order sets the
# L2 reuse of the K/V stream.
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2606_23019_amd", "csrc", f)
                  for f in ("attn_fwd.hip", "prepass.hip")]


def kernel_sources_sha():
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def flops_per_block(wl):
    return 4.0 * wl.blk_q * wl.blk_k * wl.d


def _events_time(fn, steps):
    """Run fn() ``steps`` times between two events on the current stream; ms per call."""
    import torch
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    s.record()
    for _ in range(steps):
        fn()
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / steps


def _per_launch_time(fn, steps):
    """Average duration of the kernel launched by fn(): an event pair around every launch."""
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    torch.cuda.synchronize()
    for a, b in evs:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    t = np.array([a.elapsed_time(b) for a, b in evs])
    return float(t.mean()), float(np.median(t))


def _graph_time(fn, launches=20, replays=10):
    """GPU time per call of fn() without host launch gaps: ``launches`` calls are
    captured into one HIP graph, which is replayed ``replays`` times between two
    events (ms per call).  For kernels of a few microseconds, an event pair
    around each call from Python would time the host instead."""
    import torch
    fn()  # outputs and workspaces of the first call come from the ordinary pool
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(launches):
            fn()
    graph.replay()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(replays):
        graph.replay()
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / (replays * launches)
    del graph
    return ms


class Case:
    """Device-resident inputs and prepared schedule of one workload."""

    def __init__(self, wl, dense=False, qkv=None):
        import torch
        from paper_2606_23019_amd import binding
        from workloads import masks_for, qkv_for
        self.wl = wl
        if dense:
            n_qb, n_kb = wl.n_qb, wl.n_kb
            bm = np.ones((wl.H, n_qb, n_kb), dtype=bool)
            from workloads import pack_rows
            packed = pack_rows(bm)
            dens = np.ones(wl.H)
        else:
            packed, bm, dens = masks_for(wl)
        self.packed, self.bm, self.dens = packed, bm, dens
        self.mask = binding.mask_to_device(packed)
        self.q, self.k, self.v = qkv if qkv is not None else qkv_for(wl, device="cuda")
        self.out = torch.empty_like(self.q)
        self.lse = torch.empty((wl.B, wl.H, wl.N), dtype=torch.float32, device="cuda")
        self.executed = wl.B * int(bm.sum())
        self.flops = self.executed * flops_per_block(wl)
        self.counts, self.lists = binding.mask_prepass(self.mask, wl.H, wl.n_qb, wl.n_kb)
        self.order = binding.schedule(self.counts, wl.B, wl.H, wl.n_qb)
        torch.cuda.synchronize()

    def step(self):
        from paper_2606_23019_amd import binding
        binding.bsattn_fwd(self.q, self.k, self.v, self.mask, self.wl.blk_q, self.wl.blk_k,
                           self.wl.scale, out=self.out, lse=self.lse)

    def attention_only(self):
        from paper_2606_23019_amd import binding
        binding.bsattn_fwd_prepared(self.q, self.k, self.v, self.counts, self.lists, self.order,
                                    self.wl.blk_q, self.wl.blk_k, self.wl.scale, out=self.out,
                                    lse=self.lse)


def parity_spot_check(case, n_items=4):
    """Sampled check of the last output against the CPU reference (not timed)."""
    import torch
    import oracle
    from workloads import sample_items
    wl = case.wl
    items = sample_items(wl, case.bm, n_items)
    worst = dict(out_max_abs=0.0, lse_max_abs=0.0)
    n_kb = wl.n_kb
    for (b, h, u) in items:
        r0, r1 = u * wl.blk_q, min((u + 1) * wl.blk_q, wl.N)

        def bits(t):
            return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        allowed = oracle.block_mask(case.packed[h:h + 1, u:u + 1], n_kb)[0, 0]
        ro, rl = oracle.attention_block(bits(case.q[b, h, r0:r1]), bits(case.k[b, h]),
                                        bits(case.v[b, h]), allowed, wl.blk_k, wl.scale)
        go = case.out[b, h, r0:r1].float().cpu().numpy()
        gl = case.lse[b, h, r0:r1].cpu().numpy()
        worst["out_max_abs"] = max(worst["out_max_abs"], float(np.abs(go - ro).max()))
        worst["lse_max_abs"] = max(worst["lse_max_abs"], float(np.abs(gl - rl).max()))
    return worst


def cpu_baseline(case, budget_s=12.0):
    """The CPU reference, as it stands, on a bounded sample of the same workload."""
    import torch
    import oracle
    wl = case.wl
    rng = np.random.default_rng(wl.sample_seed + 17)
    n_kb = wl.n_kb
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    # per-head host copies are part of the setup, not of the timed work
    heads = sorted(set(int(h) for h in rng.integers(0, wl.H, size=4)))
    host = {}
    for h in heads:
        host[h] = tuple(t[0, h].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
                        for t in (case.q, case.k, case.v))
    items = [(h, int(u)) for h in heads for u in rng.permutation(wl.n_qb)]
    rng.shuffle(items)
    done_blocks, n_done, t_used = 0, 0, 0.0
    for (h, u) in items:
        qb, kb, vb = host[h]
        allowed = oracle.block_mask(case.packed[h:h + 1, u:u + 1], n_kb)[0, 0]
        r0, r1 = u * wl.blk_q, min((u + 1) * wl.blk_q, wl.N)
        t0 = time.perf_counter()
        oracle.attention_block(qb[r0:r1], kb, vb, allowed, wl.blk_k, wl.scale)
        t_used += time.perf_counter() - t0
        done_blocks += int(allowed.sum())
        n_done += 1
        if t_used >= budget_s:
            break
    value = done_blocks * flops_per_block(wl) / t_used / 1e12
    return {"value": value, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": "%d query blocks (%d executed 128x128 blocks) of heads %s of %s, float64 "
                      "NumPy on %d host threads, %.1f s" % (n_done, done_blocks, heads, wl.name,
                                                            threads, t_used)}


def traffic_record():
    """HBM bytes per attention launch from the committed counter summary, if it still
    describes the current kernel source."""
    if not os.path.exists(TRAFFIC_SUMMARY):
        return None
    kv = {}
    for line in open(TRAFFIC_SUMMARY):
        if ":" in line and not line.startswith("#"):
            a, b = line.split(":", 1)
            kv[a.strip()] = b.strip()
    if kv.get("kernel_source_sha256_16") != kernel_sources_sha():
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def run_sweep(path, steps, warmup):
    import torch
    from workloads import SWEEP_BLKS, SWEEP_KINDS, SWEEP_RHOS, sweep_point
    rows = []
    for blk in SWEEP_BLKS:
        dense_wl = sweep_point(1.0, blk, "structured")
        dense = Case(dense_wl, dense=True)
        qkv = (dense.q, dense.k, dense.v)
        for _ in range(warmup):
            dense.attention_only()
        t_dense, _ = _per_launch_time(dense.attention_only, steps)
        for kind in SWEEP_KINDS:
            for rho in SWEEP_RHOS:
                wl = sweep_point(rho, blk, kind)
                c = dense if rho >= 1.0 else Case(wl, qkv=qkv)
                for _ in range(warmup):
                    c.attention_only()
                t, _ = _per_launch_time(c.attention_only, steps)
                tf = c.flops / (t * 1e-3) / 1e12
                rows.append(dict(blk=blk, kind=kind, rho=rho, ms=t, tflops=tf,
                                 pct_peak=100 * tf / PEAK_BF16_TFLOPS, speedup_vs_dense=t_dense / t,
                                 speedup_x_rho=rho * t_dense / t))
                log(json.dumps(rows[-1]))
                if c is not dense:
                    del c
        del dense, qkv
        torch.cuda.empty_cache()
    with open(path, "w") as f:
        json.dump(rows, f, indent=1)
    return rows


# Sequence lengths of the dense-overhead sweep (the paper's kernel comparison
# spans 1K .. 262K tokens) and the head count used at each, chosen so that one
# launch stays within tens of milliseconds.
OVERHEAD_POINTS = [(1024, 40), (2048, 40), (4096, 40), (8192, 40), (16384, 40), (32768, 40),
                   (65536, 10), (131072, 3), (262144, 1)]


def run_overhead(path, steps, warmup):
    """0 %-sparsity cost of the CRM machinery: the attention kernel driven by an all-ones
    mask (and the one-shot call with pre-pass and schedule) against the maskless dense
    path of the same kernel, with torch's SDPA as an outside reference."""
    import torch
    import torch.nn.functional as F
    from paper_2606_23019_amd import binding
    from workloads import Workload, pack_rows
    rows = []
    for N, H in OVERHEAD_POINTS:
        wl = Workload(name="dense_h%d_n%d" % (H, N), B=1, H=H, N=N, d=128, blk_q=128, blk_k=128,
                      grid=(1, 1, N), mask_kind="dense", rho=1.0)
        g = torch.Generator(device="cuda")
        g.manual_seed(4000 + N)
        q, k, v = (torch.randn((1, H, N, 128), generator=g, device="cuda").to(torch.bfloat16)
                   for _ in range(3))
        out = torch.empty_like(q)
        lse = torch.empty((1, H, N), dtype=torch.float32, device="cuda")
        n = wl.n_qb
        mask = binding.mask_to_device(pack_rows(np.ones((H, n, n), dtype=bool)))
        counts, lists = binding.mask_prepass(mask, H, n, n)
        order = binding.schedule(counts, 1, H, n)
        flops = 4.0 * H * N * N * 128

        def f_dense():
            binding.dense_attn_fwd(q, k, v, 128, wl.scale, out=out, lse=lse)

        def f_kernel():
            binding.bsattn_fwd_prepared(q, k, v, counts, lists, order, 128, 128, wl.scale,
                                        out=out, lse=lse)

        def f_oneshot():
            binding.bsattn_fwd(q, k, v, mask, 128, 128, wl.scale, out=out, lse=lse)

        def f_sdpa():
            # fused backends only: the unfused math path would materialise N x N scores
            from torch.nn.attention import SDPBackend, sdpa_kernel
            with sdpa_kernel([SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION]):
                F.scaled_dot_product_attention(q, k, v, scale=wl.scale)
        res = dict(N=N, H=H, d=128, blk=128)
        # Kernels that allocate nothing are timed as graph replays (GPU time
        # only); the one-shot call allocates its stream-ordered workspace and
        # SDPA may allocate too, so those two keep an event pair per call,
        # which at small N also times the host.
        for name, fn, graph in (("maskless", f_dense, True), ("crm_kernel", f_kernel, True),
                                ("crm_oneshot", f_oneshot, False), ("torch_sdpa", f_sdpa, False)):
            try:
                for _ in range(warmup):
                    fn()
                t = _graph_time(fn, launches=steps) if graph else _per_launch_time(fn, steps)[0]
            except RuntimeError as e:  # an SDPA backend that refuses the shape
                log("%s at N=%d: %s" % (name, N, str(e).splitlines()[0]))
                res[name + "_ms"] = res[name + "_tflops"] = None
                continue
            res[name + "_ms"] = t
            res[name + "_tflops"] = flops / (t * 1e-3) / 1e12
            res[name + "_timing"] = "graph replay" if graph else "event pair per call"
        res["overhead_kernel"] = res["crm_kernel_ms"] / res["maskless_ms"] - 1.0
        res["overhead_oneshot"] = res["crm_oneshot_ms"] / res["maskless_ms"] - 1.0
        res["sdpa_over_maskless"] = (res["torch_sdpa_ms"] / res["maskless_ms"]
                                     if res["torch_sdpa_ms"] else None)
        log(json.dumps(res))
        rows.append(res)
        del q, k, v, out, lse, mask, counts, lists, order
        torch.cuda.empty_cache()
    with open(path, "w") as f:
        json.dump(rows, f, indent=1)
    return rows


# Mask instantiation sizes: (label, H, blocks per side, thresholds per map).
INSTANTIATE_POINTS = [("14b-480p", 40, 256, 1), ("14b-480p", 40, 256, 50),
                      ("14b-720p", 40, 591, 1), ("14b-720p", 40, 591, 50),
                      ("262k-tokens", 40, 2048, 1), ("262k-tokens", 40, 2048, 8)]


GRAPH_TIMING = "GPU time per call: calls captured in one HIP graph, replayed between events"


def run_instantiate(path, steps, warmup):
    """sa_mask_instantiate against its HBM roofline: T read once (4 B per block),
    one bit per block and threshold written."""
    import torch
    from paper_2606_23019_amd import binding
    rows = []
    for label, H, n, n_p in INSTANTIATE_POINTS:
        g = torch.Generator(device="cuda")
        g.manual_seed(5000 + n)
        T = torch.rand((H, n, n), generator=g, device="cuda")
        p = torch.rand((n_p, H), generator=g, device="cuda")
        W = (n + 63) // 64
        out = torch.empty((n_p, H, n, W), dtype=torch.int64, device="cuda")

        def fn():
            binding.mask_instantiate(T, p, out=out)
        for _ in range(warmup):
            fn()
        t = _graph_time(fn, launches=steps)
        nbytes = 4.0 * H * n * n + 8.0 * n_p * H * n * W + 4.0 * n_p * H
        rec = dict(shape=label, H=H, n_blocks=n, n_thresholds=n_p, us=t * 1e3, timing=GRAPH_TIMING,
                   algorithmic_bytes=nbytes, gbs=nbytes / (t * 1e-3) / 1e9,
                   frac_hbm_peak=nbytes / (t * 1e-3) / 1e9 / PEAK_HBM_GBS)
        log(json.dumps(rec))
        rows.append(rec)
        del T, p, out
        torch.cuda.empty_cache()
    with open(path, "w") as f:
        json.dump(rows, f, indent=1)
    return rows


# Fidelity profiling sizes: (workload, sampled rows per head, candidate thresholds).
FIDELITY_POINTS = [("14b-480p", 16, 16), ("14b-720p", 16, 16), ("14b-720p", 32, 64)]


def run_fidelity(path, steps, warmup):
    """sa_fidelity_profile against its HBM roofline: every head's K is read once
    (B H N d 2 bytes); the sampled rows' Q, the block log-masses (written, then
    read), the rows' threshold-map rows and the outputs are small beside it."""
    import torch
    from paper_2606_23019_amd import binding
    from workloads import SHORT, qkv_for, stratified_rows, threshold_maps
    rows_out = []
    for name, R, K in FIDELITY_POINTS:
        wl = SHORT[name]
        q, k, v = qkv_for(wl, device="cuda")
        del v
        T = torch.from_numpy(threshold_maps(wl.H, wl.n_qb, wl.n_kb, wl.blk_q, wl.grid,
                                            seed=wl.mask_seed)).cuda()
        rows = torch.from_numpy(stratified_rows(wl.N, wl.H, n_strata=R, seed=wl.sample_seed)).cuda()
        p = torch.linspace(0.0, 1.0, K, device="cuda")

        def fn():
            binding.fidelity_profile(q, k, rows, T, p, wl.blk_q, wl.scale)
        for _ in range(warmup):
            fn()
        t = _graph_time(fn, launches=steps)
        BH = wl.B * wl.H
        nbytes = (2.0 * BH * wl.N * wl.d + 2.0 * BH * R * wl.d + 2 * 4.0 * BH * R * wl.n_kb
                  + 4.0 * wl.H * R * wl.n_kb + 4.0 * BH * R * K + 4.0 * BH * K)
        flops = 2.0 * BH * wl.N * 32 * wl.d   # MFMA work incl. the padding of R to 32 columns
        rec = dict(workload=wl.name, rows_per_head=R, candidates=K, ms=t, timing=GRAPH_TIMING,
                   algorithmic_bytes=nbytes, gbs=nbytes / (t * 1e-3) / 1e9,
                   frac_hbm_peak=nbytes / (t * 1e-3) / 1e9 / PEAK_HBM_GBS,
                   mfma_tflops=flops / (t * 1e-3) / 1e12)
        log(json.dumps(rec))
        rows_out.append(rec)
        del q, k, T, rows, p
        torch.cuda.empty_cache()
    with open(path, "w") as f:
        json.dump(rows_out, f, indent=1)
    return rows_out


def run_resize(path, steps, warmup):
    """Threshold-map and mask resize 480p -> 720p (40 heads, 256^2 -> 591^2 blocks) and a
    4x upscale of 720p maps, against HBM: each base entry read (cached re-reads are
    not counted), each target entry written."""
    import torch
    from paper_2606_23019_amd import binding
    from workloads import SHORT
    a, b = SHORT["14b-480p"], SHORT["14b-720p"]
    rows = []
    for label, H, nq, tq in (("480p->720p", a.H, a.n_qb, b.n_qb), ("720p->4x", b.H, b.n_qb, 4 * b.n_qb)):
        g = torch.Generator(device="cuda")
        g.manual_seed(6000 + tq)
        T = torch.rand((H, nq, nq), generator=g, device="cuda")
        masks = binding.mask_instantiate(T, torch.full((1, H), 0.3, device="cuda"))[0].contiguous()
        for kind in ("map", "mask"):
            if kind == "map":
                def fn():
                    binding.resize_threshold_map(T, tq, tq)
                nbytes = 4.0 * H * nq * nq + 4.0 * H * tq * tq
            else:
                def fn():
                    binding.resize_mask(masks, nq, tq, tq)
                nbytes = 8.0 * H * nq * ((nq + 63) // 64) + 8.0 * H * tq * ((tq + 63) // 64)
            for _ in range(warmup):
                fn()
            t = _graph_time(fn, launches=steps)
            rec = dict(resize=label, kind=kind, H=H, base=nq, target=tq, us=t * 1e3, timing=GRAPH_TIMING,
                       algorithmic_bytes=nbytes, gbs=nbytes / (t * 1e-3) / 1e9,
                       frac_hbm_peak=nbytes / (t * 1e-3) / 1e9 / PEAK_HBM_GBS)
            log(json.dumps(rec))
            rows.append(rec)
        del T, masks
        torch.cuda.empty_cache()
    with open(path, "w") as f:
        json.dump(rows, f, indent=1)
    return rows


def reference_gemm(attention_tflops, n=8192, reps=10):
    """A measured practical bf16 MFMA rate on the same GPU: torch.matmul of two
    n x n bf16 matrices (the vendor GEMM library), so that the attention kernel
    can be read against what a plain dense contraction reaches under the same
    clock and power limits, beside the 2.5 PFLOP/s data-sheet figure."""
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(77)
    a = torch.randn((n, n), generator=g, device="cuda").to(torch.bfloat16)
    b = torch.randn((n, n), generator=g, device="cuda").to(torch.bfloat16)
    for _ in range(3):
        c = a @ b
    ms = _events_time(lambda: a @ b, reps)
    del a, b, c
    torch.cuda.empty_cache()
    tflops = 2.0 * n ** 3 / (ms * 1e-3) / 1e12
    return {"what": "torch.matmul bf16 %dx%dx%d" % (n, n, n), "tflops": round(tflops, 1),
            "attention_kernel_frac_of_it": round(attention_tflops / tflops, 4)}


def mfma_microbench(attention_tflops, iters=100000, reps=3):
    """The sustained bf16 MFMA rate of this GPU: the probe kernel of
    libsa_mfma_peak.so (one workgroup of 8 wavefronts per CU, four independent
    32x32x16 accumulators per wavefront, register operands holding random bf16
    values), timed with events over ~50 ms launches, so the clock settles where
    the power limit puts it."""
    import ctypes
    import torch
    from paper_2606_23019_amd import build as _b
    if not os.path.exists(_b.MFMA_PEAK_PATH):
        return None
    lib = ctypes.CDLL(_b.MFMA_PEAK_PATH)
    lib.sa_mfma_peak.restype = ctypes.c_int
    lib.sa_mfma_peak.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                 ctypes.c_void_p]
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    g = torch.Generator(device="cuda")
    g.manual_seed(78)
    src = torch.randn((2 * 4 * 64 * 8,), generator=g, device="cuda").to(torch.bfloat16)
    out = torch.empty((n_cu * 8 * 64,), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream

    def launch():
        if lib.sa_mfma_peak(src.data_ptr(), out.data_ptr(), n_cu, iters, stream) != 0:
            raise RuntimeError("sa_mfma_peak launch failed")
    launch()
    ms = _events_time(launch, reps)
    tflops = n_cu * 8 * iters * 16 * 32768 / (ms * 1e-3) / 1e12
    return {"what": "v_mfma_f32_32x32x16_bf16 on random register operands, 8 wavefronts per CU "
                    "x %d CUs, %.1f ms per launch" % (n_cu, ms),
            "tflops": round(tflops, 1), "frac_of_2500": round(tflops / PEAK_BF16_TFLOPS, 4),
            "attention_kernel_frac_of_it": round(attention_tflops / tflops, 4)}


COPY_BYTES = 1 << 30


def profile_run(case, steps, warmup):
    """Launches for counter collection: the attention kernel, then a plain copy of
    COPY_BYTES (read COPY_BYTES, write COPY_BYTES) to calibrate byte counters."""
    import torch
    for _ in range(warmup):
        case.attention_only()
    for _ in range(steps):
        case.attention_only()
    src = torch.empty(COPY_BYTES // 2, dtype=torch.bfloat16, device="cuda").normal_()
    dst = torch.empty_like(src)
    for _ in range(steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"profile_run": case.wl.name, "attention_launches": warmup + steps,
                      "copy_launches": steps, "copy_bytes_each_way": COPY_BYTES}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=12)
    ap.add_argument("--workload", default="14b-480p")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sweep", default=None, help="also run the density/block sweep into this file")
    ap.add_argument("--configs", default=None, help="also time every named workload into this file")
    ap.add_argument("--overhead", default=None,
                    help="also run the 0 %%-sparsity overhead sweep (1K..262K tokens) into this file")
    ap.add_argument("--instantiate", default=None,
                    help="also time mask instantiation from threshold maps into this file")
    ap.add_argument("--fidelity", default=None,
                    help="also time the Hellinger fidelity profile into this file")
    ap.add_argument("--resize", default=None,
                    help="also time the conservative resize of maps and masks into this file")
    ap.add_argument("--profile", action="store_true",
                    help="counter-collection run: attention kernel launches plus a plain 1 GiB "
                         "device copy (the HBM byte-counter calibration), nothing else")
    ap.add_argument("--profile-density", type=float, default=None,
                    help="with --profile: run the sweep point of this density (H40 N32768 d128) "
                         "instead of the workload")
    ap.add_argument("--profile-blk", type=int, default=128, choices=(64, 128),
                    help="block size of the --profile-density point")
    ap.add_argument("--profile-kind", default="structured", choices=("structured", "uniform"),
                    help="mask kind of the --profile-density point")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the block-sparse forward is a single-GPU kernel "
              "here (heads shard across GPUs with no exchange); run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from workloads import SHORT
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    from paper_2606_23019_amd import binding
    binding.load(build_if_missing=True)

    wl = SHORT[args.workload]
    if args.profile and args.profile_density is not None:
        from workloads import sweep_point
        wl = sweep_point(args.profile_density, args.profile_blk, args.profile_kind)
    log("workload", wl.name)
    case = Case(wl)
    if args.profile:
        profile_run(case, args.steps, args.warmup)
        return
    for _ in range(args.warmup):
        case.step()
    torch.cuda.synchronize()
    ms_step = _events_time(case.step, args.steps)
    value = case.flops / (ms_step * 1e-3) / 1e12

    # attention kernel alone, event pair around every launch on its stream
    for _ in range(args.warmup):
        case.attention_only()
    ms_attn, ms_attn_med = _per_launch_time(case.attention_only, args.steps)
    achieved = case.flops / (ms_attn * 1e-3) / 1e12

    # same kernel, all-ones mask, same inputs
    dense = Case(wl, dense=True, qkv=(case.q, case.k, case.v))
    dense_steps = max(3, args.steps // 4)
    for _ in range(2):
        dense.attention_only()
    ms_dense, _ = _per_launch_time(dense.attention_only, dense_steps)
    dense_tflops = dense.flops / (ms_dense * 1e-3) / 1e12

    def maskless():
        binding.dense_attn_fwd(case.q, case.k, case.v, wl.blk_q, wl.scale, out=dense.out,
                               lse=dense.lse)
    for _ in range(2):
        maskless()
    ms_maskless, _ = _per_launch_time(maskless, dense_steps)
    del dense
    torch.cuda.empty_cache()

    case.step()
    torch.cuda.synchronize()
    parity = parity_spot_check(case)
    gemm = reference_gemm(achieved)
    mfma_probe = mfma_microbench(achieved)

    traffic = traffic_record()
    rec = {
        "metric": "block-sparse attn fwd effective TFLOP/s",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": wl.name, "B": wl.B, "H": wl.H, "N": wl.N, "d": wl.d,
            "blk_q": wl.blk_q, "blk_k": wl.blk_k, "mask": wl.mask_kind,
            "density_range": list(wl.rho_range) if wl.rho_range else wl.rho,
            "mean_density": round(float(case.dens.mean()), 4),
            "executed_blocks": case.executed, "executed_tflop": round(case.flops / 1e12, 4),
        },
        "pct_bf16_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "attention_kernel_ms": round(ms_attn, 4),
        "attention_kernel_ms_median": round(ms_attn_med, 4),
        "dense_mask_ms": round(ms_dense, 4),
        "dense_mask_tflops": round(dense_tflops, 3),
        "speedup_vs_dense": round(ms_dense / ms_attn, 3),
        "maskless_dense_ms": round(ms_maskless, 4),
        "crm_overhead_at_density_1": round(ms_dense / ms_maskless - 1.0, 4),
        "parity_spot_check": parity,
        "reference_gemm": gemm,
        "mfma_microbench": mfma_probe,
        "roofline": {
            "bound": "mfma", "achieved": round(achieved, 3), "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic,
        },
    }
    if args.configs:
        from workloads import SHORT as ALL
        res = {}
        for name, w in ALL.items():
            c = Case(w)
            for _ in range(args.warmup):
                c.attention_only()
            t, _ = _per_launch_time(c.attention_only, args.steps)
            # the same kernel on an all-ones mask, same inputs (speedup vs dense)
            d = Case(w, dense=True, qkv=(c.q, c.k, c.v))
            for _ in range(2):
                d.attention_only()
            td, _ = _per_launch_time(d.attention_only, max(3, args.steps // 4))
            del d
            c.attention_only()
            torch.cuda.synchronize()
            res[name] = dict(workload=w.name, ms=t, tflops=c.flops / (t * 1e-3) / 1e12,
                             mean_density=float(c.dens.mean()), executed_blocks=c.executed,
                             executed_tflop=c.flops / 1e12, dense_mask_ms=td,
                             speedup_vs_dense=td / t, parity_spot_check=parity_spot_check(c))
            log(json.dumps(res[name]))
            del c
            torch.cuda.empty_cache()
        with open(args.configs, "w") as f:
            json.dump(res, f, indent=1)
    if args.sweep:
        run_sweep(args.sweep, args.steps, args.warmup)
    if args.overhead:
        run_overhead(args.overhead, max(5, args.steps // 2), 2)
    if args.instantiate:
        run_instantiate(args.instantiate, args.steps, args.warmup)
    if args.fidelity:
        run_fidelity(args.fidelity, args.steps, args.warmup)
    if args.resize:
        run_resize(args.resize, args.steps, args.warmup)
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(case)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
