#!/usr/bin/env python3
"""Benchmark of the batched speculative verify step on one MI355X.

Headline workload: one Llama-3-8B-shaped decoder layer plus the LM head (bf16,
random-init N(0, 0.02)), context 1024 for every sequence, KV block 16, draft
distributions softmax(N(0, 2^2)), B=8 sequences with k=5 drafts -- the
small-batch, memory-bound regime.  A timed step is the whole hot path: the
verify step (embedding, norms, GEMMs, RoPE, paged verify attention, LM head,
acceptance) and the KV append of the accepted rows; every step starts from the
same cache state.

Prints one JSON line with:
* value: verified tokens/s at the headline point (B * (k+1) per step time);
* roofline: the LM-head kernel as it runs inside the step (folded final norm,
  softmax-statistics epilogue, the step's own activations), timed with HIP
  events around its launch on the library's stream (nightjar_profile_*);
* kernels: every kernel class of the headline step with its time and roofline
  fraction;
* grid: the (B, k) cost table of the small-batch grid B in {1,2,4,8} x k in {0..5};
* large_batch: B in {64, 128} x k in {3, 4, 5} of the same layer with beta-mixed
  drafts (beta 0.7), contexts lognormal (median 768, clipped to [128, 2048]):
  step time, step roofline fraction, and the GEMM kernels' fraction of the bf16
  MFMA peak (from the in-step kernel times);
* llama8b_32layer: the 32-layer 8B-shaped stack at B=64, k=4 (contexts lognormal,
  median 1024, clipped to [128, 4096]);
* cpu_baseline: the CPU oracle timed on the host at the headline workload.
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
# shared pieces
# --------------------------------------------------------------------------
class StepInputs:
    """A step's device inputs and outputs (the fields the device helpers read)."""


def device_model(shape, seed):
    """Random-init weights generated on the device (torch's seeded generator)."""
    import torch

    from paper_2512_22420_amd import workload as W
    from paper_2512_22420_amd.device import DeviceModel
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    w = W.device_weights(shape, gen)
    model = DeviceModel(shape, w)
    del w
    torch.cuda.empty_cache()
    return model


def device_case(model, shape, ctx, k, k_max, beta, seed, ws):
    """Cache with contexts `ctx` (pages generated on the device) and a step's
    inputs with beta-mixed drafts, q_i = softmax(beta * l_i + (1 - beta) * N(0, 4)),
    l_i the target logits of window row i from a causal pre-pass through the
    step itself (these runs are timed, not checked)."""
    import torch

    from paper_2512_22420_amd import workload as W
    from paper_2512_22420_amd.device import DeviceCache, verify
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    B = len(ctx)
    table, num_blocks, max_blocks = W.make_block_table(shape, ctx, k_max, seed=seed)
    kp, vp = W.device_pages(shape, num_blocks, gen)
    cache = DeviceCache({"k_pages": kp, "v_pages": vp, "block_table": torch.from_numpy(table).cuda(),
                         "context_lens": torch.from_numpy(np.asarray(ctx, np.int32)).cuda(),
                         "num_blocks": num_blocks})
    cache.max_blocks = max_blocks
    io = StepInputs()
    io.B, io.k = B, k
    V = shape.vocab
    io.last_tokens = torch.randint(0, V, (B,), generator=gen, device="cuda", dtype=torch.int32)
    io.uniforms = torch.rand((B, k + 1), generator=gen, device="cuda", dtype=torch.float32)
    io.accepted_len = torch.zeros(B, dtype=torch.int32, device="cuda")
    io.next_tokens = torch.zeros((B, k + 1), dtype=torch.int32, device="cuda")
    io.draft_tokens = torch.zeros((B, k), dtype=torch.int32, device="cuda") if k else None
    io.draft_probs = torch.full((B, k, V), 1.0 / V, device="cuda", dtype=torch.float32) if k else None
    io.logits = torch.empty((B, k + 1, V), dtype=torch.float32, device="cuda") if k else None
    for i in range(k):
        verify(model, cache, io, ws)
        z = beta * io.logits[:, i, :] + (1.0 - beta) * 2.0 * torch.randn((B, V), generator=gen, device="cuda", dtype=torch.float32)
        q = torch.softmax(z, dim=-1)
        io.draft_probs[:, i] = q
        io.draft_tokens[:, i] = torch.multinomial(q, 1, generator=gen).squeeze(1).to(torch.int32)
    io.logits = None
    return cache, io


def kernel_table(shape, B, k, ctx, prof, steps):
    """Per kernel class: time per step, its algorithmic bytes / FLOPs per step
    and the fraction of the roofline bound (HBM 8 TB/s, bf16 MFMA 2.5 PF/s)."""
    from paper_2512_22420_amd import roofline as R
    s = shape
    M = B * (k + 1)
    L = s.n_layers
    HD, qkv, F, d, V = s.n_heads * s.head_dim, s.qkv_dim, s.ffn_dim, s.d_model, s.vocab
    kv_read = sum(int(c) for c in ctx) * s.n_kv_heads * s.head_dim * 2 * 2
    # (bytes, flops) per launch
    algo = {
        "qkv": (R.gemm_bytes(M, qkv, d, 2, 2), 2 * M * qkv * d),
        "o": (R.gemm_bytes(M, d, HD, 2, 8), 2 * M * d * HD),
        "gate_up": (R.gemm_bytes(M, 2 * F, d, 2, 0) + M * F * 2, 2 * M * 2 * F * d),
        "down": (R.gemm_bytes(M, d, F, 2, 8), 2 * M * d * F),
        "lm_head": (R.lm_head_bytes(s, M), 2 * M * V * d),
        "attention": (kv_read + M * HD * 2 * 2, 4 * (k + 1) * HD * sum(int(c) + (k + 2) / 2 for c in ctx)),
        "accept": (2 * B * V * 4 + B * k * 8, 0),
    }
    out = {}
    for name, (us, n) in prof.items():
        if n == 0:
            continue
        row = {"us_per_launch": round(us, 2), "launches_per_step": round(n / steps, 2),
               "us_per_step": round(us * n / steps, 2)}
        if name in algo:
            by, fl = algo[name]
            t_hbm, t_mfma = by / R.HBM_BYTES_PER_S, fl / R.BF16_MFMA_FLOPS
            row["bound"] = "mfma" if t_mfma > t_hbm else "hbm"
            row["gb_s"] = round(by / (us * 1e-6) / 1e9, 1)
            if fl:
                row["tflop_s"] = round(fl / (us * 1e-6) / 1e12, 1)
            row["frac"] = round(max(t_hbm, t_mfma) / (us * 1e-6), 3)
        out[name] = row
    return out


def profiled(run_step, steps):
    """Mean in-step kernel times over `steps` steps (HIP events around each
    launch site inside the library)."""
    import torch

    from paper_2512_22420_amd import binding as nb
    torch.cuda.synchronize()
    nb.profile_enable(True)
    for _ in range(steps):
        run_step()
    torch.cuda.synchronize()
    prof = nb.profile_read()
    nb.profile_enable(False)
    return prof


def gemm_mfma_frac(shape, B, k, prof, steps):
    from paper_2512_22420_amd import roofline as R
    M = B * (k + 1)
    flops = 2 * M * (shape.n_layers * R.layer_params(shape) + shape.vocab * shape.d_model)
    us = sum(prof[n][0] * prof[n][1] for n in ("qkv", "o", "gate_up", "down", "lm_head")) / steps
    return round(flops / R.BF16_MFMA_FLOPS / (us * 1e-6), 3), round(us, 1)


def timed_cold(run, reps, flush, flush_out):
    """Median event time of `run` with the last-level cache evicted before each
    rep (reading 640 MB: no dirty lines left to write back in the timed rep)."""
    import torch
    stream = torch.cuda.current_stream()
    ts = []
    for _ in range(reps):
        torch.sum(flush, dim=0, keepdim=True, out=flush_out)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        run()
        b.record(stream)
        torch.cuda.synchronize()
        ts.append(a.elapsed_time(b) * 1e3)
    return float(np.median(ts))


def large_point(model, shape, B, k, ctx, ws, beta, seed, reps, flush, flush_out, label):
    """One (B, k) point with beta-mixed drafts: cold verify time, in-step kernel
    times, step roofline fraction, GEMM fraction of the MFMA peak."""
    import torch

    from paper_2512_22420_amd import roofline as R
    from paper_2512_22420_amd.device import device_error, kv_append, verify
    cache, io = device_case(model, shape, ctx, k, k, beta, seed, ws)
    ctx0 = cache.context_lens.clone()  # a copy: the KV append advances cache.context_lens in place

    def vstep():
        verify(model, cache, io, ws)

    def full():
        verify(model, cache, io, ws)
        kv_append(model, cache, io, ws)
        cache.context_lens.copy_(ctx0)
    for _ in range(2):
        full()
    torch.cuda.synchronize()
    assert device_error(ws) == 0, f"device error at {label}"
    t_us = timed_cold(vstep, reps, flush, flush_out)
    t_step = timed_cold(full, reps, flush, flush_out)
    psteps = 3
    prof = profiled(vstep, psteps)
    acc = io.accepted_len.cpu().numpy()
    mp = R.step_model(shape, B, k, ctx)
    gf, gus = gemm_mfma_frac(shape, B, k, prof, psteps)
    row = {"B": B, "k": k, "M": B * (k + 1), "beta": beta, "verify_us": round(t_us, 1), "step_us": round(t_step, 1),
           "verified_tok_s": round(B * (k + 1) / (t_us * 1e-6)),
           "goodput_tok_s": round(float((acc + 1).sum()) / (t_us * 1e-6)),
           "acceptance": round(float(acc.sum()) / (B * k), 3) if k else None,
           "roofline_us": round(mp["t_roof_s"] * 1e6, 1), "roofline_frac": round(mp["t_roof_s"] * 1e6 / t_us, 3),
           "gemm_us_in_step": gus, "gemm_mfma_frac": gf,
           "kernels": kernel_table(shape, B, k, ctx, prof, psteps), "ctx_mean": round(float(np.mean(ctx)), 1)}
    log(f"{label} B={B} k={k}: verify {t_us:.1f} us (step {t_step:.1f}), roofline {row['roofline_frac']:.3f}, "
        f"GEMMs {gus:.1f} us at {gf:.3f} of MFMA peak, acceptance {row['acceptance']}")
    del cache, io
    torch.cuda.empty_cache()
    return row


def sd_table(tmodel, tshape, dshape, B, ctx_len, gammas, reps=10):
    """Whole speculative-decoding steps (nightjar_sd_step: k+1 draft forwards
    with their appends, the target's verify step and append) for each k, with
    the draft chain and the verify step also timed alone.  The random-init
    draft agrees with the random-init target about as often as chance, so the
    acceptance here is near 0; goodput at the paper's acceptance rates follows
    from the step time as (1 - a^(k+1)) / (1 - a) committed tokens per step."""
    import torch

    from paper_2512_22420_amd import binding as nb
    from paper_2512_22420_amd import workload as W
    from paper_2512_22420_amd.device import DeviceCache
    dmodel = device_model(dshape, 7)
    kmax = max(gammas)
    ctx = np.full(B, ctx_len, np.int32)
    table, num_blocks, max_blocks = W.make_block_table(tshape, ctx, kmax + 1, seed=3)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(3)
    tk, tv = W.device_pages(tshape, num_blocks, gen)
    dk, dv = W.device_pages(dshape, num_blocks, gen)
    bt = torch.from_numpy(table).cuda()
    ctx_dev = torch.from_numpy(ctx).cuda()
    ctx0 = ctx_dev.clone()
    tcache = DeviceCache({"k_pages": tk, "v_pages": tv, "block_table": bt, "context_lens": ctx_dev,
                          "num_blocks": num_blocks})
    dcache = DeviceCache({"k_pages": dk, "v_pages": dv, "block_table": bt, "context_lens": ctx_dev,
                          "num_blocks": num_blocks})
    s = torch.cuda.current_stream().cuda_stream
    tn = nb.workspace_bytes(tmodel.desc, B, kmax)
    tws = torch.empty(tn, dtype=torch.uint8, device="cuda")
    nb.workspace_init(tws.data_ptr(), tn, s)
    dn = nb.sd_workspace_bytes(dmodel.desc, B)
    dws = torch.empty(dn, dtype=torch.uint8, device="cuda")
    nb.workspace_init(dws.data_ptr(), dn, s)
    V = tshape.vocab
    last = torch.randint(0, V, (B,), generator=gen, device="cuda", dtype=torch.int32)
    rows = []
    for k in gammas:
        du = torch.rand((B, k + 1), generator=gen, device="cuda", dtype=torch.float32)
        u = torch.rand((B, k + 1), generator=gen, device="cuda", dtype=torch.float32)
        dt = torch.zeros((B, max(k, 1)), dtype=torch.int32, device="cuda")
        dq = torch.zeros((B, max(k, 1), V), device="cuda", dtype=torch.float32)
        acc = torch.zeros(B, dtype=torch.int32, device="cuda")
        nxt = torch.zeros((B, k + 1), dtype=torch.int32, device="cuda")

        def step():
            ctx_dev.copy_(ctx0)
            nb.sd_step(tmodel.desc, tmodel.c, tcache.c, dmodel.desc, dmodel.c, dcache.c, bt.data_ptr(), max_blocks,
                       ctx_dev.data_ptr(), last.data_ptr(), du.data_ptr(), u.data_ptr(), B, k, dt.data_ptr(),
                       dq.data_ptr(), acc.data_ptr(), nxt.data_ptr(), tws.data_ptr(), tn, dws.data_ptr(), dn, s)

        def chain():
            ctx_dev.copy_(ctx0)
            for i in range(k + 1):
                nb.draft_step(dmodel.desc, dmodel.c, dcache.c, bt.data_ptr(), max_blocks, ctx_dev.data_ptr(),
                              last.data_ptr(), du.data_ptr(), B, dt.data_ptr(), max(k, 1), dq.data_ptr(),
                              max(k, 1) * V, dws.data_ptr(), dn, s)
        for f in (step, chain):
            f()
        torch.cuda.synchronize()
        assert nb.device_error(tws.data_ptr(), tn, s) == 0 and nb.device_error(dws.data_ptr(), dn, s) == 0

        def timed(f):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(reps):
                f()
            b.record()
            torch.cuda.synchronize()
            return a.elapsed_time(b) / reps * 1e3
        t_step = timed(step)
        t_chain = timed(chain) if k else 0.0
        a_n = acc.cpu().numpy()
        row = {"k": k, "B": B, "sd_step_us": round(t_step, 1), "draft_forwards": k + 1 if k else 0,
               "draft_chain_us": round(t_chain, 1), "verify_and_append_us": round(t_step - t_chain, 1),
               "committed_tokens_s": round(float((a_n + 1).sum()) / (t_step * 1e-6)),
               "goodput_tok_s_at_acceptance": {str(al): round(B * (1 - al ** (k + 1)) / (1 - al) / (t_step * 1e-6))
                                               for al in (0.53, 0.69)}}
        rows.append(row)
        log(f"sd step B={B} k={k}: {t_step:.1f} us (draft chain {t_chain:.1f} us), "
            f"goodput at acceptance 0.69: {row['goodput_tok_s_at_acceptance']['0.69']} tok/s")
    del dmodel, tcache, dcache, tws, dws
    torch.cuda.empty_cache()
    return {"target": tshape.name, "draft": dshape.name, "ctx": ctx_len, "rows": rows}


def elastic_costs(tshape, dshape, moves=292):
    """Costs of the elastic pool's data movement (Sec. 6.2, 6.4): the draft
    model's weights (bf16) offloaded to pinned host memory and reloaded, on a
    side stream, and a contraction migrating `moves` KV blocks of the 32-layer
    target pool (the paper migrates 292 blocks)."""
    import torch

    from paper_2512_22420_amd import binding as nb
    from paper_2512_22420_amd import roofline as R
    from paper_2512_22420_amd import workload as W
    from paper_2512_22420_amd.device import DeviceCache, model_desc
    nbytes = 2 * (dshape.n_layers * R.layer_params(dshape) + 2 * dshape.vocab * dshape.d_model)
    dev = torch.empty(nbytes // 2, dtype=torch.int16, device="cuda")
    host = torch.empty(nbytes // 2, dtype=torch.int16, pin_memory=True)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())

    def timed(fn):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(side)
        fn()
        b.record(side)
        side.synchronize()
        return a.elapsed_time(b) * 1e3
    off = timed(lambda: nb.offload(dev.data_ptr(), host.data_ptr(), nbytes, side.cuda_stream))
    rel = timed(lambda: nb.reload(host.data_ptr(), dev.data_ptr(), nbytes, side.cuda_stream))
    del dev, host
    # contraction: blocks [nb/2, nb/2 + moves) move to [0, moves)
    nblk = 2 * moves + 8
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)
    kp, vp = W.device_pages(tshape, nblk, gen)
    cache = DeviceCache({"k_pages": kp, "v_pages": vp, "block_table": torch.zeros((1, 1), dtype=torch.int32,
                         device="cuda"), "context_lens": torch.zeros(1, dtype=torch.int32, device="cuda"),
                         "num_blocks": nblk})
    src = torch.arange(nblk // 2, nblk // 2 + moves, dtype=torch.int32, device="cuda")
    dst = torch.arange(0, moves, dtype=torch.int32, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    desc = model_desc(tshape)
    mig = lambda: nb.kv_migrate(desc, cache.c, src.data_ptr(), dst.data_ptr(), moves, err.data_ptr(),
                                side.cuda_stream)
    mig()
    side.synchronize()
    assert int(err.item()) == 0
    t_mig = min(timed(mig) for _ in range(5))
    mbytes = 2 * moves * tshape.n_layers * 2 * tshape.n_kv_heads * 16 * tshape.head_dim * 2  # read + write
    out = {"draft_bytes": nbytes, "offload_ms": round(off / 1e3, 2), "offload_gb_s": round(nbytes / off / 1e3, 1),
           "reload_ms": round(rel / 1e3, 2), "reload_gb_s": round(nbytes / rel / 1e3, 1),
           "migrate_blocks": moves, "migrate_us": round(t_mig, 1),
           "migrate_gb_s": round(mbytes / t_mig / 1e3, 1), "migrate_hbm_frac": round(mbytes / t_mig / 1e3 / 8000, 3)}
    log(f"elastic: offload {out['offload_ms']} ms ({out['offload_gb_s']} GB/s), reload {out['reload_ms']} ms, "
        f"migrate {moves} blocks in {t_mig:.1f} us ({out['migrate_gb_s']} GB/s)")
    del cache, kp, vp
    torch.cuda.empty_cache()
    return out


# --------------------------------------------------------------------------
# Report mode: the full (B, k) cost table of another configuration
# --------------------------------------------------------------------------
def report(args):
    """Time the verify step over a workload's whole (B, k) grid and print one
    JSON line with the cost table (inputs generated on the device)."""
    import torch

    from paper_2512_22420_amd import workload as W
    from paper_2512_22420_amd.device import Workspace

    wl = W.WORKLOADS[args.workload]
    shape = wl.shape
    grid = list(wl.grid)
    if args.points:
        keep = {tuple(int(v) for v in p.split("x")) for p in args.points.split(",")}
        grid = [g for g in grid if g in keep]
    betas = [float(b) for b in args.beta.split(",")]
    torch.cuda.set_device(0)
    t0 = time.time()
    model = device_model(shape, 0)
    log(f"{wl.name}: weights generated on the device in {time.time() - t0:.1f} s")
    ws = Workspace(shape, max(B for B, _ in grid), max(k for _, k in grid))
    flush = torch.zeros(640 * 2 ** 20 // 4, dtype=torch.float32, device="cuda")
    flush_out = torch.zeros(1, dtype=torch.float32, device="cuda")
    rows = []
    for (B, k) in grid:
        ctx = wl.ctx(B, seed=0)
        for beta in (betas if k else [None]):
            rows.append(large_point(model, shape, B, k, ctx, ws, beta if beta is not None else 0.0, 0,
                                    args.grid_reps, flush, flush_out, wl.name))
    print(json.dumps({"report": wl.name, "unit": "verified tokens/s", "dtype": "bf16",
                      "data": "synthetic, generated on the device (torch seeded generator)", "grid": rows}),
          flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--grid-reps", type=int, default=20)
    ap.add_argument("--no-grid", action="store_true")
    ap.add_argument("--no-large", action="store_true", help="skip the large-batch and 32-layer points")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also copy a 1 GiB device buffer three times: a dispatch of known HBM traffic "
                         "(1,048,576 KiB read and written) that scales the FETCH_SIZE / WRITE_SIZE counters")
    ap.add_argument("--B", type=int, default=8)
    ap.add_argument("--k", type=int, default=5)
    ap.add_argument("--workload", default="llama8b-layer-small-batch",
                    help="another workload prints its whole (B, k) cost table instead of the headline line: "
                         "llama8b-layer-large-batch, llama8b-32layer, qwen7b-28layer")
    ap.add_argument("--points", default="", help="report mode: only these grid points, e.g. 64x4,128x5")
    ap.add_argument("--beta", default="0.7", help="report mode: beta(s) of the beta-mixed draft model")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the verify step shards by sequence "
              "across GPUs without any exchange, which this single-GPU build does not implement.", file=sys.stderr)
        sys.exit(2)
    if args.workload != "llama8b-layer-small-batch":
        report(args)
        return

    import torch

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
        return cache, io, ctx0

    # ---------------- headline: K timed steps at (B, k) ----------------
    # Every step starts from the same state: each one gets its own copy of the
    # pre-step context lengths (the KV append advances them in place), so the
    # timed region holds exactly verify_step + kv_append per step; the pages
    # the append writes are rewritten with the same values each step.
    B, k = args.B, args.k
    cache, io, ctx0 = setup(B, k)
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
    ms_per_step = ev0.elapsed_time(ev1) / args.steps
    assert all(torch.equal(c, ctx_bufs[-1]) for c in ctx_bufs[args.warmup:]), "steps diverged"
    cache.context_lens = ctx0
    verified = B * (k + 1)
    value = verified / (ms_per_step / 1e3)
    log(f"headline B={B} k={k}: {ms_per_step * 1e3:.1f} us/step, {value:.0f} verified tok/s (wall {wall:.3f} s)")
    model_pt = R.step_model(shape, B, k, [1024] * B)

    # ---------------- the headline step's kernels, timed inside the step ----------------
    M = B * (k + 1)
    psteps = max(20, args.steps)

    ctx_start = ctx0.clone()

    def head_step():
        verify(model, cache, io, ws)
        kv_append(model, cache, io, ws)
        cache.context_lens.copy_(ctx_start)
    prof = profiled(head_step, psteps)
    assert device_error(ws) == 0, "device error in the profiled steps"
    kernels = kernel_table(shape, B, k, [1024] * B, prof, psteps)
    lm_us = prof["lm_head"][0]
    lm_bytes = R.lm_head_bytes(shape, M)
    lm_gbs = lm_bytes / (lm_us * 1e-6) / 1e9
    log(f"in-step LM head (M={M}): {lm_us:.1f} us per launch, {lm_gbs:.0f} GB/s")
    roofline = {"kernel": "LM head inside the step: gemm_stream_kernel<kEpiLogits> (folded final RMSNorm, "
                          "softmax-statistics epilogue), M=%d, N=%d, K=%d" % (M, shape.vocab, shape.d_model),
                "bound": "hbm", "achieved": round(lm_gbs, 1), "peak": R.HBM_BYTES_PER_S / 1e9, "unit": "GB/s",
                "frac": round(lm_gbs / (R.HBM_BYTES_PER_S / 1e9), 4),
                "traffic": measured_traffic(M),
                "algorithmic_bytes_per_launch": lm_bytes, "avg_launch_us": round(lm_us, 2),
                "timing": "HIP events around the launch on the library's stream, %d steps" % psteps}

    # ---------------- the (B, k) cost table of the small-batch grid ----------------
    flush = torch.zeros(640 * 2 ** 20 // 4, dtype=torch.float32, device="cuda")
    flush_out = torch.zeros(1, dtype=torch.float32, device="cuda")
    grid = []
    if not args.no_grid:
        for (gB, gk) in wl.grid:
            gcache, gio, gctx0 = setup(gB, gk)

            def gstep():
                verify(model, gcache, gio, ws)
            for _ in range(3):
                gstep()
            t_us = timed_cold(gstep, args.grid_reps, flush, flush_out)
            a, b2 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for _ in range(5):
                gstep()
            b2.record(stream)
            torch.cuda.synchronize()
            warm = a.elapsed_time(b2) / 5 * 1e3
            assert device_error(ws) == 0
            acc = gio.accepted_len.cpu().numpy()
            mp = R.step_model(shape, gB, gk, [1024] * gB)
            grid.append({"B": gB, "k": gk, "verify_us": round(t_us, 1), "verify_us_warm": round(warm, 1),
                         "verified_tok_s": round(gB * (gk + 1) / (t_us * 1e-6)),
                         "goodput_tok_s": round(float((acc + 1).sum()) / (t_us * 1e-6)),
                         "acceptance": round(float(acc.sum()) / (gB * gk), 3) if gk else None,
                         "roofline_us": round(mp["t_roof_s"] * 1e6, 1),
                         "roofline_frac": round(mp["t_roof_s"] * 1e6 / t_us, 3)})
            log(f"grid B={gB} k={gk}: {t_us:.1f} us cold, {warm:.1f} us warm, roofline {mp['t_roof_s'] * 1e6:.1f} us")
            del gcache, gio

    # ---------------- compute-bound points: large batch, 32 layers ----------------
    large, deep = [], None
    if not args.no_large:
        lwl = W.WORKLOADS["llama8b-layer-large-batch"]
        lmodel = device_model(shape, 0)  # the same layer, weights generated on the device
        lws = Workspace(shape, 128, 5)
        for (lB, lk) in [(64, 3), (64, 4), (64, 5), (128, 3), (128, 4), (128, 5)]:
            large.append(large_point(lmodel, shape, lB, lk, lwl.ctx(lB, seed=0), lws, 0.7, 1, 10, flush, flush_out,
                                     "large-batch"))
        del lmodel, lws
        torch.cuda.empty_cache()
        dwl = W.WORKLOADS["llama8b-32layer"]
        t1 = time.time()
        dmodel = device_model(dwl.shape, 0)
        log(f"32-layer stack generated on the device in {time.time() - t1:.1f} s")
        dws = Workspace(dwl.shape, 64, 4)
        deep = large_point(dmodel, dwl.shape, 64, 4, dwl.ctx(64, seed=0), dws, 0.7, 2, 10, flush, flush_out,
                           "32-layer")
        # whole speculative-decoding steps: the 32-layer target with a 1B-class draft
        sd = sd_table(dmodel, dwl.shape, W.LLAMA1B_DRAFT, 8, 1024, [0, 1, 3, 5])
        elastic = elastic_costs(dwl.shape, W.LLAMA1B_DRAFT)
        del dmodel, dws
        torch.cuda.empty_cache()
    del flush, flush_out

    # ---------------- CPU baseline: the oracle on the host ----------------
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        cores = len(os.sched_getaffinity(0))
        blas, threads = "unknown BLAS", cores
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
        c = W.make_context(shape, wl.ctx(B, seed=0), k_max, seed=0)
        d = W.make_drafts(shape, B, k, seed=0)
        n_steps, tc = 0, 0.0
        while tc < 10.0:
            t1 = time.perf_counter()
            oracle.verify_step(weights, shape, c["k_pages"], c["v_pages"], c["block_table"], c["context_lens"],
                               d["last_tokens"], d["draft_tokens"], d["draft_probs"], d["uniforms"])
            tc += time.perf_counter() - t1
            n_steps += 1
        cpu = {"value": round(n_steps * B * (k + 1) / tc, 3), "unit": "verified tokens/s", "cores": cores,
               "kind": "oracle", "blas": blas, "blas_threads": threads,
               "sample": f"{n_steps} fp64 oracle verify steps at B={B} k={k} ctx 1024 (the headline workload), "
                         f"{tc:.1f} s; NumPy with {blas} on {threads} BLAS threads, {cores} cores in the affinity mask"}
        log(f"cpu oracle: {n_steps} steps in {tc:.1f} s at B={B} k={k} on {threads} threads")

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
        "data": "synthetic (random-init N(0,0.02) weights, N(0,1)*0.5 KV pages, softmax(N(0,4)) drafts; "
                "beta-mixed drafts for the large-batch and 32-layer points)",
        "config": {"workload": "llama3-8b-layer+lm_head verify step, B=%d k=%d ctx 1024 (small-batch grid)" % (B, k),
                   "B": B, "k": k, "ctx": 1024, "M": M, "d_model": shape.d_model, "vocab": shape.vocab,
                   "kv_block": 16, "step": "verify_step + kv_append"},
        "roofline_step": {"t_roof_us": round(model_pt["t_roof_s"] * 1e6, 1),
                          "frac": round(model_pt["t_roof_s"] * 1e3 / ms_per_step, 4),
                          "bytes": model_pt["bytes"]},
        "roofline": roofline,
        "kernels": kernels,
        "cpu_baseline": cpu,
        "grid": grid,
        "large_batch": large,
        "llama8b_32layer": deep,
        "sd_step": sd if not args.no_large else None,
        "elastic": elastic if not args.no_large else None,
    }
    if args.calib_copy:
        src = torch.empty(2 ** 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
