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


# --------------------------------------------------------------------------
# Report mode: cost table of the large-batch / full-depth configurations
# --------------------------------------------------------------------------
def report(args):
    """Time the verify step over a workload's (B, k) grid and print one JSON
    line with the cost table.  Inputs are generated on the GPU with torch's
    seeded generator (same distributions as the CPU generator, not the same
    bits: these runs are timed, not checked; the parity tests use the CPU
    generator).  Drafts follow the beta-mixed draft model,
    q_i = softmax(beta * l_i + (1 - beta) * N(0, 4)), with the target logits l_i
    of a device pre-pass over the window."""
    import torch

    from paper_2512_22420_amd import binding as nb
    from paper_2512_22420_amd import roofline as R
    from paper_2512_22420_amd import workload as W
    from paper_2512_22420_amd.device import DeviceCache, DeviceModel, Workspace, device_error, kv_append, verify

    wl = W.WORKLOADS[args.workload]
    shape = wl.shape
    grid = list(wl.grid)
    if args.points:
        keep = {tuple(int(v) for v in p.split("x")) for p in args.points.split(",")}
        grid = [g for g in grid if g in keep]
    betas = [float(b) for b in args.beta.split(",")]
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    gen = torch.Generator(device="cuda")
    gen.manual_seed(0)

    def normal_bf16(shape_, std):
        out = torch.empty(shape_, dtype=torch.bfloat16, device="cuda")
        flat = out.view(-1)
        step = 1 << 26
        for i in range(0, flat.numel(), step):  # bounded fp32 temporaries
            n = min(step, flat.numel() - i)
            flat[i:i + n] = (torch.randn(n, generator=gen, device="cuda") * std).to(torch.bfloat16)
        return out.view(torch.int16)

    t0 = time.time()
    ones = torch.ones(shape.d_model, dtype=torch.bfloat16, device="cuda").view(torch.int16)
    w = {"embed": normal_bf16((shape.vocab, shape.d_model), 0.02),
         "lm_head": normal_bf16((shape.vocab, shape.d_model), 0.02), "final_norm": ones, "layers": []}
    for _ in range(shape.n_layers):
        w["layers"].append({"attn_norm": ones, "ffn_norm": ones,
                            "w_qkv": normal_bf16((shape.qkv_dim, shape.d_model), 0.02),
                            "w_o": normal_bf16((shape.d_model, shape.n_heads * shape.head_dim), 0.02),
                            "w_gate_up": normal_bf16((2 * shape.ffn_dim, shape.d_model), 0.02),
                            "w_down": normal_bf16((shape.d_model, shape.ffn_dim), 0.02)})
    model = DeviceModel(shape, w)
    torch.cuda.synchronize()
    log(f"{wl.name}: weights generated on the device in {time.time() - t0:.1f} s")
    B_max = max(B for B, _ in grid)
    k_max = max(k for _, k in grid)
    ws = Workspace(shape, B_max, k_max)
    s = stream.cuda_stream

    class IO:
        pass

    rows = []
    for (B, k) in grid:
        ctx = wl.ctx(B, seed=0)
        table, num_blocks, max_blocks = W.make_block_table(shape, ctx, k_max, seed=0)
        c = {"k_pages": [normal_bf16((num_blocks, shape.n_kv_heads, 16, shape.head_dim), 0.5)
                         for _ in range(shape.n_layers)],
             "v_pages": [normal_bf16((num_blocks, shape.n_kv_heads, shape.head_dim, 16), 0.5)
                         for _ in range(shape.n_layers)],
             "block_table": torch.from_numpy(table).cuda(), "context_lens": torch.from_numpy(ctx).cuda(),
             "num_blocks": num_blocks}
        cache = DeviceCache(c)
        cache.max_blocks = max_blocks
        ctx0 = cache.context_lens.clone()
        for beta in (betas if k else [None]):
            io = IO()
            io.B, io.k = B, k
            io.last_tokens = torch.randint(0, shape.vocab, (B,), generator=gen, device="cuda", dtype=torch.int32)
            io.uniforms = torch.rand((B, k + 1), generator=gen, device="cuda")
            io.accepted_len = torch.zeros(B, dtype=torch.int32, device="cuda")
            io.next_tokens = torch.zeros((B, k + 1), dtype=torch.int32, device="cuda")
            io.draft_tokens = torch.zeros((B, k), dtype=torch.int32, device="cuda") if k else None
            io.draft_probs = torch.full((B, k, shape.vocab), 1.0 / shape.vocab, device="cuda") if k else None
            io.logits = torch.empty((B, k + 1, shape.vocab), dtype=torch.float32, device="cuda") if k else None
            for i in range(k):  # beta-mixed drafts from a causal pre-pass
                verify(model, cache, io, ws)
                z = beta * io.logits[:, i, :] + (1.0 - beta) * 2.0 * torch.randn(
                    (B, shape.vocab), generator=gen, device="cuda")
                q = torch.softmax(z, dim=-1)
                io.draft_probs[:, i] = q
                io.draft_tokens[:, i] = torch.multinomial(q, 1, generator=gen).squeeze(1).to(torch.int32)
            io.logits = None
            verify(model, cache, io, ws)
            torch.cuda.synchronize()
            assert device_error(ws) == 0, "device error"
            reps = args.grid_reps
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
            tv, ts = [], []
            for _ in range(reps):
                ev[0].record(stream)
                verify(model, cache, io, ws)
                ev[1].record(stream)
                kv_append(model, cache, io, ws)
                ev[2].record(stream)
                cache.context_lens.copy_(ctx0)
                torch.cuda.synchronize()
                tv.append(ev[0].elapsed_time(ev[1]) * 1e3)
                ts.append(ev[0].elapsed_time(ev[2]) * 1e3)
            assert device_error(ws) == 0, "device error"
            acc = io.accepted_len.cpu().numpy()
            t_us = float(np.median(tv))
            mp = R.step_model(shape, B, k, ctx)
            # the step's GEMMs alone, with layer 0's weights (every layer has the same shapes)
            M = B * (k + 1)
            x = normal_bf16((M, max(shape.d_model, shape.ffn_dim, shape.n_heads * shape.head_dim)), 1.0)
            y = torch.zeros((M, max(shape.vocab, 2 * shape.ffn_dim, shape.qkv_dim)), dtype=torch.float32,
                            device="cuda")
            lw = model.layers[0]
            gl = [(lw["w_qkv"], shape.qkv_dim, shape.d_model, nb.NJ_GEMM_STORE, shape.n_layers),
                  (lw["w_o"], shape.d_model, shape.n_heads * shape.head_dim, nb.NJ_GEMM_RESIDUAL, shape.n_layers),
                  (lw["w_gate_up"], 2 * shape.ffn_dim, shape.d_model, nb.NJ_GEMM_SWIGLU, shape.n_layers),
                  (lw["w_down"], shape.d_model, shape.ffn_dim, nb.NJ_GEMM_RESIDUAL, shape.n_layers),
                  (model.lm_head, shape.vocab, shape.d_model, nb.NJ_GEMM_STORE, 1)]
            gemm_us = 0.0
            for wt, N, K, epi, mult in gl:
                n = nb.gemm_workspace_bytes(nb.NJ_BF16, M, N, K, epi)
                gws = torch.empty(n, dtype=torch.uint8, device="cuda")
                nb.workspace_init(gws.data_ptr(), n, s)
                # the tiled kernel's inputs in the k-blocked layout, as the step writes them
                flag = nb.NJ_GEMM_KBLOCKED
                call = lambda: nb.gemm(nb.NJ_BF16, x.data_ptr(), wt.data_ptr(), y.data_ptr(), M, N, K, epi | flag,
                                       gws.data_ptr(), n, s)
                try:
                    call()
                except nb.NightjarError:  # a streaming-kernel plan: row-major x
                    flag = 0
                    call()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                for _ in range(5):
                    call()
                e1.record(stream)
                torch.cuda.synchronize()
                gemm_us += e0.elapsed_time(e1) / 5 * 1e3 * mult
            del x, y
            gemm_roof_us = max(mp["weight_bytes"] / R.HBM_BYTES_PER_S, mp["gemm_flops"] / R.BF16_MFMA_FLOPS) * 1e6
            row = {"B": B, "k": k, "M": M, "beta": beta, "verify_us": round(t_us, 1),
                   "step_us": round(float(np.median(ts)), 1),
                   "verified_tok_s": round(M / (t_us * 1e-6)),
                   "goodput_tok_s": round(float((acc + 1).sum()) / (t_us * 1e-6)),
                   "acceptance": round(float(acc.sum()) / (B * k), 3) if k else None,
                   "roofline_us": round(mp["t_roof_s"] * 1e6, 1),
                   "roofline_frac": round(mp["t_roof_s"] * 1e6 / t_us, 3),
                   "gemm_us": round(gemm_us, 1), "gemm_roofline_us": round(gemm_roof_us, 1),
                   "gemm_mfma_frac": round(mp["gemm_flops"] / R.BF16_MFMA_FLOPS * 1e6 / gemm_us, 3),
                   "gemm_share": round(gemm_us / t_us, 3),
                   "kv_gb": round(mp["kv_bytes"] / 1e9, 3), "ctx_mean": round(float(np.mean(ctx)), 1)}
            rows.append(row)
            log(f"{wl.name} B={B} k={k} beta={beta}: verify {t_us:.1f} us, step {row['step_us']} us, "
                f"{row['verified_tok_s']} tok/s, roofline {row['roofline_us']} us ({row['roofline_frac']:.2f}), "
                f"GEMMs {gemm_us:.1f} us at {row['gemm_mfma_frac']:.2f} of MFMA peak, acceptance {row['acceptance']}")
        del cache, c
        torch.cuda.empty_cache()
    print(json.dumps({"report": wl.name, "unit": "verified tokens/s", "dtype": "bf16",
                      "data": "synthetic, generated on the device (torch seeded generator)", "grid": rows}),
          flush=True)


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
    ap.add_argument("--workload", default="llama8b-layer-small-batch",
                    help="another workload prints its (B, k) cost table instead of the headline line: "
                         "llama8b-layer-large-batch, llama8b-32layer, qwen7b-28layer")
    ap.add_argument("--points", default="", help="report mode: only these grid points, e.g. 64x4,128x5")
    ap.add_argument("--beta", default="0.7", help="report mode: beta(s) of the beta-mixed draft model")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the verify step shards by sequence "
              "across GPUs without any exchange, which this single-GPU build does not implement.", file=sys.stderr)
        sys.exit(2)
    if args.workload != "llama8b-layer-small-batch":
        if args.grid_reps == 30:
            args.grid_reps = 10
        report(args)
        return

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
    # Every step starts from the same state: each one gets its own copy of the
    # pre-step context lengths (the KV append advances them in place), so the
    # timed region holds exactly verify_step + kv_append per step; the pages
    # the append writes are rewritten with the same values each step.
    B, k = args.B, args.k
    _, _, cache, io, ctx0 = setup(B, k)
    ctx_bufs = [ctx0.clone() for _ in range(args.warmup + args.steps)]
    for i in range(args.warmup):
        cache.context_lens = ctx_bufs[i]
        verify(model, cache, io, ws)
        kv_append(model, cache, io, ws)
    torch.cuda.synchronize()
    assert device_error(ws) == 0, "device error during warmup"
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        cache.context_lens = ctx_bufs[args.warmup + i]
        verify(model, cache, io, ws)
        kv_append(model, cache, io, ws)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_total = ev0.elapsed_time(ev1)
    ms_per_step = ms_total / args.steps
    assert all(torch.equal(c, ctx_bufs[-1]) for c in ctx_bufs[args.warmup:]), "steps diverged"
    cache.context_lens = ctx0
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
    roofline = {"kernel": "gemm_logits_kernel (LM head, M=%d, N=%d, K=%d)" % (M, shape.vocab, shape.d_model),
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
        # cold reps: reading 640 MB evicts the 256 MB last-level cache (a read,
        # so no dirty lines are left to be written back during the timed step)
        flush = torch.zeros(640 * 2 ** 20 // 4, dtype=torch.float32, device="cuda")
        flush_sum = torch.zeros(1, dtype=torch.float32, device="cuda")
        for (gB, gk) in wl.grid:
            _, d, gcache, gio, gctx0 = setup(gB, gk)
            for _ in range(3):
                step(gcache, gio, gctx0)
            times_cold, times_warm = [], []
            for rep in range(args.grid_reps):
                torch.sum(flush, dim=0, keepdim=True, out=flush_sum)
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
        del flush, flush_sum

    # ---------------- CPU baseline: the oracle on the host ----------------
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        cores = len(os.sched_getaffinity(0))
        blas = "unknown BLAS"
        threads = cores
        try:
            from threadpoolctl import threadpool_info
            libs = [p for p in threadpool_info() if p.get("user_api") == "blas"]
            if libs:
                threads = max(p.get("num_threads", 1) for p in libs)
                blas = ", ".join(sorted({f"{p.get('internal_api', '?')} {p.get('version') or ''}".strip()
                                         for p in libs}))
        except ImportError:  # pragma: no cover
            pass
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
        cpu = {"value": round(n_steps * cB * (ck + 1) / tc, 3), "unit": "verified tokens/s", "cores": cores,
               "kind": "oracle", "blas": blas, "blas_threads": threads,
               "sample": f"{n_steps} fp64 oracle verify steps at B={cB} k={ck} ctx 1024 (the headline workload), "
                         f"{tc:.1f} s; NumPy with {blas} on {threads} BLAS threads, {cores} cores in the affinity mask"}
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
