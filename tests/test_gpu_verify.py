"""End-to-end GPU parity of the verify step and the KV append through the C ABI.

Forward: fp32 model -> target probabilities within 1e-3 max-abs of the oracle;
bf16 models -> logits within 1e-2 relative L2 per row.  Decisions: bit-exact
except flagged ones (see parity.py).  Also: KV append placement, paging
invariance, determinism, device-side error reporting, HIP-graph replay.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2512_22420_amd import binding as nb
from paper_2512_22420_amd import workload as W
from paper_2512_22420_amd.device import (DeviceCache, DeviceModel, StepIO, Workspace, device_error, kv_append,
                                        model_desc, verify)

import rounding_model as RM
from parity import compare, record, rel_l2_rows, self_check

pytestmark = pytest.mark.gpu

# two-layer bf16 GQA model with the production head dim; vocab not a multiple of 256
SMALL_BF16 = dataclasses.replace(W.LLAMA8B_LAYER, name="bf16-small", n_layers=2, d_model=512, n_heads=8,
                                 n_kv_heads=2, ffn_dim=1024, vocab=4112)
# Qwen-like grouping: 7 query heads per KV head (k=7 packs 56 query rows per KV head)
QWEN_SMALL = dataclasses.replace(W.QWEN7B, name="qwen-small", n_layers=2, d_model=1792, n_heads=14, n_kv_heads=2,
                                 ffn_dim=1536, vocab=6016)


def _oracle(x, shape):
    return oracle.verify_step(x["weights"], shape, x["k_pages"], x["v_pages"], x["block_table"], x["context_lens"],
                              x["last_tokens"], x["draft_tokens"], x["draft_probs"], x["uniforms"])


def _inputs(shape, ctx, k, seed, weights=None, k_max=None):
    w = weights if weights is not None else W.make_weights(shape, seed)
    c = W.make_context(shape, ctx, k if k_max is None else k_max, seed)
    d = W.make_drafts(shape, len(ctx), k, seed)
    return {"weights": w, **c, **d}


def _run(shape, x, model=None, ws=None):
    model = model or DeviceModel(shape, x["weights"])
    cache = DeviceCache(x)
    io = StepIO(shape, x)
    ws = ws or Workspace(shape, io.B, io.k)
    verify(model, cache, io, ws)
    err = device_error(ws)
    return model, cache, io, ws, err


def _decisions_ok(io, ref, x, gpu_logits=None, min_checked=0):
    """Decisions against the oracle (flagged ones excluded and counted) and,
    with the GPU's logits, every decision against the rule on those logits.
    min_checked: floor on the decisions compared with the oracle."""
    acc, nxt = io.accepted_len.cpu().numpy(), io.next_tokens.cpu().numpy()
    res = compare(acc, nxt, ref["logits"], x["draft_tokens"], x["draft_probs"], x["uniforms"], gpu_logits=gpu_logits)
    sres = None
    if gpu_logits is not None:
        sres = self_check(acc, nxt, gpu_logits, x["draft_tokens"], x["draft_probs"], x["uniforms"])
        assert not sres["mismatches"], sres["mismatches"][:5]
        B = len(acc)
        assert sres["margin"] <= max(1, B // 4), sres
        assert sres["checked"] >= B - sres["margin"], sres
    record(res, sres)
    assert not res["mismatches"], res["mismatches"][:5]
    assert res["checked"] >= min_checked, (res, min_checked)
    return res


# --------------------------------------------------------------------------
def test_tiny_f32_step_matches_oracle():
    x = W.tiny_inputs(seed=0, k=3)
    shape = x["shape"]
    _, _, io, _, err = _run(shape, x)
    assert err == 0
    ref = _oracle(x, shape)
    p_gpu = oracle.softmax(io.logits.cpu().numpy().astype(np.float64))
    assert np.abs(p_gpu - ref["probs"]).max() <= 1e-3
    assert np.abs(io.logits.cpu().numpy() - ref["logits"]).max() < 1e-4
    res = _decisions_ok(io, ref, x)
    assert res["checked"] >= 1


@pytest.mark.parametrize("k", [0, 1, 3, 7])
def test_small_bf16_ragged_contexts(k):
    ctx = np.array([0, 5, 37, 100, 16, 250], dtype=np.int32)  # empty, partial blocks, exact block, long
    x = _inputs(SMALL_BF16, ctx, k, seed=1)
    _, _, io, _, err = _run(SMALL_BF16, x)
    assert err == 0
    ref = _oracle(x, SMALL_BF16)
    gl = io.logits.cpu().numpy()
    assert rel_l2_rows(gl, ref["logits"]).max() <= 1e-2
    _decisions_ok(io, ref, x, gpu_logits=gl)


@pytest.mark.parametrize("k", [2, 4, 7])
def test_qwen_grouping_many_query_rows(k):
    """G = 7: k=2 -> 21 query rows per KV head (2 tiles), k=4 -> 35 (3), k=7 -> 56 (4)."""
    ctx = np.array([300, 0, 47, 129], dtype=np.int32)
    x = _inputs(QWEN_SMALL, ctx, k, seed=20 + k)
    _, _, io, _, err = _run(QWEN_SMALL, x)
    assert err == 0
    ref = _oracle(x, QWEN_SMALL)
    gl = io.logits.cpu().numpy()
    assert rel_l2_rows(gl, ref["logits"]).max() <= 1e-2
    _decisions_ok(io, ref, x, gpu_logits=gl)


def test_large_batch_lognormal_contexts():
    """B=24, k=5 (M = 144 rows: three 64-row blocks in every GEMM), contexts
    lognormal (median 768, sigma 0.5, clipped to [128, 2048]) as in the large-batch grid."""
    B, k = 24, 5
    ctx = W.ctx_lengths("lognormal", B, seed=3, median=768, sigma=0.5, lo=128, hi=2048)
    x = _inputs(SMALL_BF16, ctx, k, seed=31)
    _, _, io, _, err = _run(SMALL_BF16, x)
    assert err == 0
    ref = _oracle(x, SMALL_BF16)
    gl = io.logits.cpu().numpy()
    assert rel_l2_rows(gl, ref["logits"]).max() <= 1e-2
    res = _decisions_ok(io, ref, x, gpu_logits=gl)
    assert res["checked"] >= B // 2


def _within_storage_model(shape, weights, x, k, ref_logits, gpu_logits):
    """Per-row logits errors within those of the bf16 storage model of the
    same path (folded or unfused norms, as the library runs this window)."""
    B = len(x["context_lens"])
    fused = nb.step_folds_norms(model_desc(shape), B, k)
    toks = oracle.window_tokens(x["last_tokens"], x["draft_tokens"])
    m = RM.forward(weights, shape, x["k_pages"], x["v_pages"], x["block_table"], x["context_lens"], toks, fused)
    return RM.assert_within_model(gpu_logits, m, ref_logits)


@pytest.fixture(scope="module")
def llama_layer():
    shape = W.LLAMA8B_LAYER
    weights = W.make_weights(shape, 0)
    return shape, weights, DeviceModel(shape, weights)


@pytest.mark.parametrize("B,k", [(1, 0), (8, 0), (8, 5), (3, 2)])
def test_llama8b_layer_full_size(llama_layer, B, k):
    """The 8B-shaped layer + LM head at the sizes the benchmark runs (context 1024)."""
    shape, weights, model = llama_layer
    x = _inputs(shape, np.full(B, 1024, dtype=np.int32), k, seed=0, weights=weights, k_max=5)
    _, _, io, _, err = _run(shape, x, model=model)
    assert err == 0
    ref = _oracle(x, shape)
    gl = io.logits.cpu().numpy()
    assert rel_l2_rows(gl, ref["logits"]).max() <= 1e-2
    # at V = 128256 a 1e-3 relative logit difference moves about half the draws
    # across a running-sum boundary (straddles, flagged); the accept tests are
    # compared with the oracle, the draws with the rule on the GPU's logits
    res = _decisions_ok(io, ref, x, gpu_logits=gl, min_checked=B // 2 if k else 0)
    if k == 0:
        sres = self_check(io.accepted_len.cpu().numpy(), io.next_tokens.cpu().numpy(), gl, x["draft_tokens"],
                          x["draft_probs"], x["uniforms"])
        assert res["checked"] + sres["checked"] >= B // 2


@pytest.mark.parametrize("B,k", [(32, 3), (64, 5)])
def test_llama8b_layer_tiled_gemms(llama_layer, B, k):
    """Windows of 128 and 384 rows: the LDS-tiled GEMMs with their inputs written
    k-blocked by the norm, attention and SwiGLU producers, contexts lognormal
    as in the large-batch grid.  The logits bound is the relative L2 over the
    whole logits tensor; single rows of a window this large pass 1e-2 from
    bf16 storage alone (the storage model puts row 14 of the 128-row case at
    1.08e-2), so rows are held to the storage model's own row errors
    (rounding_model.assert_within_model)."""
    shape, weights, model = llama_layer
    ctx = W.ctx_lengths("lognormal", B, seed=5, median=768, sigma=0.5, lo=128, hi=2048)
    x = _inputs(shape, ctx, k, seed=1, weights=weights, k_max=5)
    _, _, io, _, err = _run(shape, x, model=model)
    assert err == 0
    ref = _oracle(x, shape)
    gl = io.logits.cpu().numpy()
    r = np.asarray(ref["logits"])
    assert np.linalg.norm(gl - r) / np.linalg.norm(r) <= 1e-2
    _within_storage_model(shape, weights, x, k, r, gl)
    _decisions_ok(io, ref, x, gpu_logits=gl, min_checked=B // 2)


@pytest.mark.parametrize("B,k", [(16, 4), (16, 5)])
def test_llama8b_layer_wide_persistent_lm_head(llama_layer, B, k):
    """Windows of 80 and 96 rows: the persistent LM-head kernel with 5 and 6
    row tiles (one group per workgroup) and its softmax statistics feeding the
    acceptance.  These windows take the unfused path (bf16 normed GEMM inputs),
    whose storage roundings alone put row 62 of the 80-row case at 1.06e-2
    (the storage model); rows are held to the model's row errors."""
    shape, weights, model = llama_layer
    ctx = W.ctx_lengths("lognormal", B, seed=6, median=768, sigma=0.5, lo=128, hi=2048)
    x = _inputs(shape, ctx, k, seed=3, weights=weights, k_max=5)
    _, _, io, _, err = _run(shape, x, model=model)
    assert err == 0
    ref = _oracle(x, shape)
    gl = io.logits.cpu().numpy()
    r = np.asarray(ref["logits"])
    assert np.linalg.norm(gl - r) / np.linalg.norm(r) <= 1e-2
    _within_storage_model(shape, weights, x, k, r, gl)
    _decisions_ok(io, ref, x, gpu_logits=gl, min_checked=B // 2)


# --------------------------------------------------------------------------
@pytest.mark.parametrize("shape,ctx,k", [(W.TINY_F32, [32, 48], 3), (SMALL_BF16, [0, 15, 31, 77], 5)],
                         ids=["f32", "bf16"])
def test_kv_append_commits_accepted_rows_only(shape, ctx, k):
    x = _inputs(shape, np.array(ctx, dtype=np.int32), k, seed=2)
    model, cache, io, ws, err = _run(shape, x)
    assert err == 0
    before_k = [t.cpu().numpy().copy() for t in cache.k_pages]
    before_v = [t.cpu().numpy().copy() for t in cache.v_pages]
    kv_append(model, cache, io, ws)
    assert device_error(ws) == 0
    acc = io.accepted_len.cpu().numpy()
    new_ctx = cache.context_lens.cpu().numpy()
    assert np.array_equal(new_ctx, np.array(ctx) + acc + 1)
    ref = _oracle(x, shape)
    view = np.uint16 if shape.dtype == "bf16" else np.float32
    tol = 2 ** -7 if shape.dtype == "bf16" else 1e-4
    for l in range(shape.n_layers):
        kp = cache.k_pages[l].cpu().numpy().view(view)
        vp = cache.v_pages[l].cpu().numpy().view(view)
        touched = np.zeros(kp.shape[:1] + kp.shape[2:3], dtype=bool)  # [blocks, slots]
        for b in range(len(ctx)):
            for j in range(acc[b] + 1):
                pos = ctx[b] + j
                blk, slot = x["block_table"][b][pos // 16], pos % 16
                touched[blk, slot] = True
                gk = oracle.widen(kp[blk, :, slot, :], shape.dtype)
                gv = oracle.widen(vp[blk, :, :, slot], shape.dtype)
                rk, rv = ref["win_k"][l][b, j], ref["win_v"][l][b, j]
                assert np.abs(gk - rk).max() <= tol * max(1.0, np.abs(rk).max())
                assert np.abs(gv - rv).max() <= tol * max(1.0, np.abs(rv).max())
        bk = before_k[l].view(view)
        bv = before_v[l].view(view)
        for blk in range(kp.shape[0]):
            for slot in range(16):
                if not touched[blk, slot]:
                    assert np.array_equal(kp[blk, :, slot, :], bk[blk, :, slot, :])
                    assert np.array_equal(vp[blk, :, :, slot], bv[blk, :, :, slot])


def test_gamma0_chain_tiny_f32():
    """Plain decoding through verify + append, several steps, against the oracle's chain."""
    shape = W.TINY_F32
    x = _inputs(shape, np.array([3, 20], dtype=np.int32), 0, seed=5, k_max=8)
    model = DeviceModel(shape, x["weights"])
    cache = DeviceCache(x)
    ws = Workspace(shape, 2, 0)
    kp, vp, ctx = x["k_pages"], x["v_pages"], x["context_lens"].copy()
    last = x["last_tokens"].copy()
    rng = np.random.default_rng(0)
    for step in range(8):
        u = rng.random((2, 1), dtype=np.float32)
        d = {"last_tokens": last, "draft_tokens": np.zeros((2, 0), np.int32),
             "draft_probs": np.zeros((2, 0, shape.vocab), np.float32), "uniforms": u}
        io = StepIO(shape, d)
        verify(model, cache, io, ws)
        kv_append(model, cache, io, ws)
        assert device_error(ws) == 0
        ref = oracle.verify_step(x["weights"], shape, kp, vp, x["block_table"], ctx, last, d["draft_tokens"],
                                 d["draft_probs"], u)
        res = compare(io.accepted_len.cpu().numpy(), io.next_tokens.cpu().numpy(), ref["logits"], d["draft_tokens"],
                      d["draft_probs"], u, gpu_logits=io.logits.cpu().numpy())
        assert not res["mismatches"] and res["flagged"] == 0, (step, res)
        kp, vp, ctx = oracle.kv_append(kp, vp, x["block_table"], ctx, ref["accepted_len"], ref["win_k"],
                                       ref["win_v"], 16, "f32")
        assert np.array_equal(cache.context_lens.cpu().numpy(), ctx)
        last = ref["next_tokens"][:, 0].astype(np.int32)


def test_block_table_permutation_is_invisible():
    x = _inputs(SMALL_BF16, np.array([40, 3, 64], dtype=np.int32), 4, seed=6)
    model, _, io1, _, _ = _run(SMALL_BF16, x)
    perm = np.random.default_rng(1).permutation(x["num_blocks"])
    inv = np.argsort(perm)
    y = dict(x)
    y["k_pages"] = [a[inv] for a in x["k_pages"]]
    y["v_pages"] = [a[inv] for a in x["v_pages"]]
    y["block_table"] = np.where(x["block_table"] >= 0, perm[np.maximum(x["block_table"], 0)], -1).astype(np.int32)
    _, _, io2, _, _ = _run(SMALL_BF16, y, model=model)
    assert torch.equal(io1.logits, io2.logits)
    assert torch.equal(io1.next_tokens, io2.next_tokens)


def test_repeated_steps_are_bitwise_identical():
    x = _inputs(SMALL_BF16, np.array([200, 17, 1, 90, 33, 64, 128, 5], dtype=np.int32), 5, seed=7)
    model, cache, io, ws, _ = _run(SMALL_BF16, x)
    first = (io.logits.clone(), io.next_tokens.clone(), io.accepted_len.clone())
    for _ in range(3):
        verify(model, cache, io, ws)
        assert torch.equal(io.logits, first[0])
        assert torch.equal(io.next_tokens, first[1])
        assert torch.equal(io.accepted_len, first[2])


def test_device_errors_are_reported_without_faults():
    x = _inputs(SMALL_BF16, np.array([20, 40], dtype=np.int32), 2, seed=8)
    model, cache, io, ws, err = _run(SMALL_BF16, x)
    assert err == 0
    io.last_tokens[1] = SMALL_BF16.vocab + 5
    verify(model, cache, io, ws)
    assert device_error(ws) & nb.NJ_DEV_BAD_TOKEN
    io.last_tokens[1] = 0
    saved = cache.block_table.clone()
    cache.block_table[0, 0] = x["num_blocks"] + 100
    verify(model, cache, io, ws)
    assert device_error(ws) & nb.NJ_DEV_BAD_BLOCK
    cache.block_table.copy_(saved)
    # -1 (an unused entry) for a block inside the context is a bad block too;
    # the kernel reads its window block instead, so nothing faults
    cache.block_table[0, 0] = -1
    verify(model, cache, io, ws)
    assert device_error(ws) & nb.NJ_DEV_BAD_BLOCK
    cache.block_table.copy_(saved)
    cache.context_lens[0] = cache.max_blocks * 16  # no room for the window
    verify(model, cache, io, ws)
    assert device_error(ws) & nb.NJ_DEV_BAD_CONTEXT
    cache.context_lens[0] = 20
    verify(model, cache, io, ws)
    assert device_error(ws) == 0


def test_hip_graph_replay_matches_eager():
    x = _inputs(SMALL_BF16, np.array([50, 9, 130], dtype=np.int32), 3, seed=9)
    model, cache, io, ws, _ = _run(SMALL_BF16, x)
    eager = (io.logits.clone(), io.next_tokens.clone(), io.accepted_len.clone())
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            verify(model, cache, io, ws, stream=s.cuda_stream)
    torch.cuda.current_stream().wait_stream(s)
    for rep in range(3):
        io.logits.zero_()
        io.next_tokens.fill_(-9)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(io.logits, eager[0]), rep
        assert torch.equal(io.next_tokens, eager[1]), rep
        assert torch.equal(io.accepted_len, eager[2]), rep
        verify(model, cache, io, ws)  # eager work between replays
        torch.cuda.synchronize()


def test_steps_of_different_sizes_share_one_workspace():
    """A workspace sized for the largest step serves smaller and larger steps in
    any order: results equal those on a fresh workspace, bitwise."""
    shape = SMALL_BF16
    weights = W.make_weights(shape, 11)
    model = DeviceModel(shape, weights)
    shared = Workspace(shape, 6, 7)
    sizes = [(2, 1), (6, 7), (1, 0), (4, 3), (6, 7), (3, 5)]
    for B, k in sizes:
        x = _inputs(shape, np.arange(B, dtype=np.int32) * 37 + 5, k, seed=B * 10 + k, weights=weights)
        _, _, io_s, _, err_s = _run(shape, x, model=model, ws=shared)
        _, _, io_f, _, err_f = _run(shape, x, model=model)
        assert err_s == 0 and err_f == 0
        assert torch.equal(io_s.logits, io_f.logits), (B, k)
        assert torch.equal(io_s.next_tokens, io_f.next_tokens), (B, k)


@pytest.mark.parametrize("k", [3, 12])
def test_stale_workspace_contents_never_reach_the_outputs(k):
    """A step reads no workspace memory that it has not written first (beyond
    the error word and the split-K counters, which workspace_init zeroes and
    every kernel leaves at zero): with the rest of the workspace filled with
    0xFF bytes (NaN bit patterns), outputs equal those of a fresh workspace,
    bitwise.  The contexts leave some KV splits of the attention empty."""
    ctx = np.array([0, 5, 37, 100, 16, 250], dtype=np.int32)
    x = _inputs(SMALL_BF16, ctx, k, seed=21)
    model, _, io_f, _, err_f = _run(SMALL_BF16, x)
    ws = Workspace(SMALL_BF16, len(ctx), k)
    zero_prefix = 256 + 1024 * 256  # error word, split-K arrival counters (1024, 256 bytes apart)
    ws.buf[zero_prefix:].fill_(255)
    _, _, io_s, _, err_s = _run(SMALL_BF16, x, model=model, ws=ws)
    assert err_f == 0 and err_s == 0
    assert torch.equal(io_s.logits, io_f.logits)
    assert torch.equal(io_s.next_tokens, io_f.next_tokens)
    assert torch.equal(io_s.accepted_len, io_f.accepted_len)
