#!/usr/bin/env python3
"""Benchmark of the batched speculative verify step on one MI355X.

Workload: one Llama-3-8B-shaped decoder layer plus the LM head (bf16,
random-init N(0, 0.02)), context 1024 for every sequence, KV block 16, draft
distributions softmax(N(0, 2^2)) -- the small-batch, memory-bound regime.  A
timed step is the whole hot path: the verify step (embedding, norms, GEMMs,
RoPE, paged verify attention, LM head, acceptance) and the KV append of the
accepted rows; the cache's context lengths are restored after each step so
every step sees the same state.

Prints one JSON line: verified tokens/s at the headline point B=8, k=5, the
(B, k) cost table of the grid B in {1,2,4,8} x k in {0..5}, the LM-head
GEMM's roofline fraction, and the CPU oracle timed on the host as a baseline.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def gemm_source_digest():
    import hashlib
    path = os.path.join(ROOT, "paper_2512_22420_amd", "csrc", "gemm.hip")
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def measured_traffic(M):
    """HBM bytes per launch of the LM-head GEMM from the committed counter
    summary, if it was taken on the current GEMM source at this M; else None."""
    path = os.path.join(ROOT, "profiles", "lm_head_gemm_traffic.json")
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("gemm_source_sha256_16") != gemm_source_digest() or rec.get("M") != M:
        return None
    return rec.get("hbm_bytes_per_launch")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--grid-reps", type=int, default=30)
    ap.add_argument("--no-grid", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--B", type=int, default=8)
    ap.add_argument("--k", type=int, default=5)
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run a plain 1 GiB device copy (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the verify step shards by sequence "
              "across GPUs without any exchange, which this single-GPU build does not implement.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2512_22420_amd import binding as nb
    from paper_2512_22420_amd import roofline as R
    from paper_2512_22420_amd import workload as W
    from paper_2512_22420_amd.device import DeviceCache, DeviceModel, StepIO, Workspace, device_error, kv_append, verify

    wl = W.WORKLOADS["llama8b-layer-small-batch"]
    shape = wl.shape
    k_max = max(k for _, k in wl.grid)
    B_max = max(B for B, _ in wl.grid)
    torch.cuda.set_device(0)
    t0 = time.time()
    weights = W.make_weights(shape, seed=0)
    model = DeviceModel(shape, weights)
    log(f"weights generated and uploaded in {time.time() - t0:.1f} s")
    ws = Workspace(shape, B_max, k_max)
    stream = torch.cuda.current_stream()

    def setup(B, k):
        ctx = wl.ctx(B, seed=0)
        c = W.make_context(shape, ctx, k_max, seed=0)
        d = W.make_drafts(shape, B, k, seed=0)
        cache = DeviceCache(c)
        io = StepIO(shape, d, keep_logits=False)
        ctx0 = cache.context_lens.clone()
        return c, d, cache, io, ctx0

    def step(cache, io, ctx0):
        verify(model, cache, io, ws)
        kv_append(model, cache, io, ws)
        cache.context_lens.copy_(ctx0)

    # ---------------- headline: K timed steps at (B, k) ----------------
    B, k = args.B, args.k
    _, _, cache, io, ctx0 = setup(B, k)
    for _ in range(args.warmup):
        step(cache, io, ctx0)
    torch.cuda.synchronize()
    assert device_error(ws) == 0, "device error during warmup"
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step(cache, io, ctx0)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_total = ev0.elapsed_time(ev1)
    ms_per_step = ms_total / args.steps
    acc = io.accepted_len.cpu().numpy()
    verified = B * (k + 1)
    value = verified / (ms_per_step / 1e3)
    log(f"headline B={B} k={k}: {ms_per_step * 1e3:.1f} us/step, {value:.0f} verified tok/s (wall {wall:.3f} s)")
    model_pt = R.step_model(shape, B, k, [1024] * B)

    # ---------------- dominant kernel: the LM-head GEMM ----------------
    M = B * (k + 1)
    x = torch.zeros((M, shape.d_model), dtype=torch.int16, device="cuda")
    y = torch.empty((M, shape.vocab), dtype=torch.float32, device="cuda")
    s = stream.cuda_stream
    gws_n = nb.gemm_workspace_bytes(nb.NJ_BF16, M, shape.vocab, shape.d_model, nb.NJ_GEMM_STORE)
    gws = torch.empty(gws_n, dtype=torch.uint8, device="cuda")
    nb.workspace_init(gws.data_ptr(), gws_n, s)

    def lm_head():
        nb.gemm(nb.NJ_BF16, x.data_ptr(), model.lm_head.data_ptr(), y.data_ptr(), M, shape.vocab, shape.d_model,
                nb.NJ_GEMM_STORE, gws.data_ptr(), gws_n, s)

    for _ in range(5):
        lm_head()
    reps = max(20, args.steps)
    g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    g0.record(stream)
    for _ in range(reps):
        lm_head()
    g1.record(stream)
    torch.cuda.synchronize()
    lm_us = g0.elapsed_time(g1) / reps * 1e3
    lm_bytes = R.lm_head_bytes(shape, M)
    lm_gbs = lm_bytes / (lm_us * 1e-6) / 1e9
    log(f"lm_head gemm M={M}: {lm_us:.1f} us, {lm_gbs:.0f} GB/s")
    roofline = {"kernel": "gemm_bf16 (LM head, M=%d, N=%d, K=%d)" % (M, shape.vocab, shape.d_model),
                "bound": "hbm", "achieved": round(lm_gbs, 1), "peak": R.HBM_BYTES_PER_S / 1e9, "unit": "GB/s",
                "frac": round(lm_gbs / (R.HBM_BYTES_PER_S / 1e9), 4),
                "traffic": measured_traffic(M),
                "algorithmic_bytes_per_launch": lm_bytes, "avg_launch_us": round(lm_us, 2)}
    del x, y, gws
    if args.calib_copy:
        src = torch.empty(2 ** 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # ---------------- the (B, k) cost table ----------------
    grid = []
    if not args.no_grid:
        flush = torch.empty(512 * 2 ** 20 // 4, dtype=torch.float32, device="cuda")
        for (gB, gk) in wl.grid:
            _, d, gcache, gio, gctx0 = setup(gB, gk)
            for _ in range(3):
                step(gcache, gio, gctx0)
            times_cold, times_warm = [], []
            for rep in range(args.grid_reps):
                flush.fill_(float(rep))  # evict the 256 MB last-level cache between cold reps
                a, b2 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(stream)
                verify(model, gcache, gio, ws)
                b2.record(stream)
                c1, c2 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                c1.record(stream)
                verify(model, gcache, gio, ws)
                c2.record(stream)
                torch.cuda.synchronize()
                times_cold.append(a.elapsed_time(b2) * 1e3)
                times_warm.append(c1.elapsed_time(c2) * 1e3)
            assert device_error(ws) == 0
            acc = gio.accepted_len.cpu().numpy()
            t_us = float(np.median(times_cold))
            mp = R.step_model(shape, gB, gk, [1024] * gB)
            grid.append({"B": gB, "k": gk, "verify_us": round(t_us, 1),
                         "verify_us_warm": round(float(np.median(times_warm)), 1),
                         "verified_tok_s": round(gB * (gk + 1) / (t_us * 1e-6)),
                         "goodput_tok_s": round(float((acc + 1).sum()) / (t_us * 1e-6)),
                         "acceptance": round(float(acc.sum()) / (gB * gk), 3) if gk else None,
                         "roofline_us": round(mp["t_roof_s"] * 1e6, 1),
                         "roofline_frac": round(mp["t_roof_s"] * 1e6 / t_us, 3)})
            log(f"grid B={gB} k={gk}: {t_us:.1f} us cold, {np.median(times_warm):.1f} us warm, "
                f"roofline {mp['t_roof_s'] * 1e6:.1f} us")
        del flush

    # ---------------- CPU baseline: the oracle on the host ----------------
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        try:
            from threadpoolctl import threadpool_info
            threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
        except Exception:  # pragma: no cover
            threads = len(os.sched_getaffinity(0))
        # the headline configuration, repeated until at least 10 s of host work
        cB, ck = B, k
        c = W.make_context(shape, wl.ctx(cB, seed=0), k_max, seed=0)
        d = W.make_drafts(shape, cB, ck, seed=0)
        n_steps, tc = 0, 0.0
        while tc < 10.0:
            t1 = time.perf_counter()
            oracle.verify_step(weights, shape, c["k_pages"], c["v_pages"], c["block_table"], c["context_lens"],
                               d["last_tokens"], d["draft_tokens"], d["draft_probs"], d["uniforms"])
            tc += time.perf_counter() - t1
            n_steps += 1
        cpu = {"value": round(n_steps * cB * (ck + 1) / tc, 3), "unit": "verified tokens/s", "cores": threads,
               "kind": "oracle",
               "sample": f"{n_steps} fp64 oracle verify steps at B={cB} k={ck} ctx 1024 (the headline workload), "
                         f"{tc:.1f} s, NumPy/OpenBLAS on {threads} threads"}
        log(f"cpu oracle: {n_steps} steps in {tc:.1f} s at B={cB} k={ck} on {threads} threads")

    out = {
        "metric": "verified tokens/s per verify step over (batch,k) grid; % HBM or MFMA roofline",
        "value": round(value, 1),
        "unit": "verified tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (random-init N(0,0.02) weights, N(0,1)*0.5 KV pages, softmax(N(0,4)) drafts)",
        "config": {"workload": "llama3-8b-layer+lm_head verify step, B=%d k=%d ctx 1024 (small-batch grid)" % (B, k),
                   "B": B, "k": k, "ctx": 1024, "M": M, "d_model": shape.d_model, "vocab": shape.vocab,
                   "kv_block": 16, "step": "verify_step + kv_append"},
        "roofline_step": {"t_roof_us": round(model_pt["t_roof_s"] * 1e6, 1),
                          "frac": round(model_pt["t_roof_s"] * 1e3 / ms_per_step, 4),
                          "bytes": model_pt["bytes"]},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "grid": grid,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
