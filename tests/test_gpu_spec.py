"""The draft chain and the whole speculative-decoding step on the GPU
(nightjar_draft_step, nightjar_sd_step) against the oracle's composition
(oracle/spec_step.py; Sec. 2.2 and Sec. 3.1: k drafts proposed one at a time,
verified in one target forward, n + 1 tokens committed, both caches
finalised before the next step).  The draft chain's draws are compared like
the target's (parity.py margins); once a sequence's chain differs by a flagged
draw its later positions are not compared."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from oracle import spec_step as S
from paper_2512_22420_amd import binding as nb
from paper_2512_22420_amd import workload as W
from paper_2512_22420_amd.device import DeviceCache, DeviceModel, device_error, model_desc

from parity import CDF_MARGIN, compare

pytestmark = pytest.mark.gpu

DRAFT_F32 = dataclasses.replace(W.TINY_F32, name="tiny-draft", d_model=128, n_heads=2, n_kv_heads=2, ffn_dim=256)
SMALL_BF16 = dataclasses.replace(W.LLAMA8B_LAYER, name="bf16-small", n_layers=2, d_model=512, n_heads=8,
                                 n_kv_heads=2, ffn_dim=1024, vocab=4112)
DRAFT_BF16 = dataclasses.replace(SMALL_BF16, name="bf16-draft", n_layers=1, d_model=256, n_heads=2, n_kv_heads=2,
                                 ffn_dim=512)


def _s():
    return torch.cuda.current_stream().cuda_stream


def _ws(desc, B, k, sd=False):
    n = nb.sd_workspace_bytes(desc, B) if sd else nb.workspace_bytes(desc, B, k)
    t = torch.empty(n, dtype=torch.uint8, device="cuda")
    nb.workspace_init(t.data_ptr(), n, _s())
    return t, n


@pytest.mark.parametrize("shape", [W.TINY_F32, SMALL_BF16], ids=["f32", "bf16"])
def test_draft_step_matches_oracle(shape):
    B = 6
    ctx = np.array([0, 5, 16, 37, 100, 250], np.int32)
    c = W.make_context(shape, ctx, 2, seed=4)
    w = W.make_weights(shape, 4)
    model = DeviceModel(shape, w)
    cache = DeviceCache(c)
    rng = np.random.default_rng(4)
    last = rng.integers(0, shape.vocab, B).astype(np.int32)
    u = rng.random(B).astype(np.float32)
    ws, n = _ws(model.desc, B, 0)
    k_t = 3  # write into column 1 of a [B][3] / [B][3][V] layout
    tok = torch.full((B, k_t), -5, dtype=torch.int32, device="cuda")
    probs = torch.full((B, k_t, shape.vocab), -1.0, device="cuda", dtype=torch.float32)
    dl, du = torch.from_numpy(last).cuda(), torch.from_numpy(u).cuda()
    nb.draft_step(model.desc, model.c, cache.c, cache.block_table.data_ptr(), cache.max_blocks,
                  cache.context_lens.data_ptr(), dl.data_ptr(), du.data_ptr(), B, tok.data_ptr() + 4, k_t,
                  probs.data_ptr() + 4 * shape.vocab, k_t * shape.vocab, ws.data_ptr(), n, _s())
    assert device_error_ws(ws, n) == 0
    t_ref, q_ref, r = S.draft_forward(w, shape, c["k_pages"], c["v_pages"], c["block_table"], ctx, last, u)
    got_t = tok.cpu().numpy()
    got_q = probs.cpu().numpy()
    assert np.all(got_t[:, [0, 2]] == -5) and np.all(got_q[:, [0, 2]] == -1.0)  # only column 1 written
    q = got_q[:, 1].astype(np.float64)
    if shape.dtype == "f32":
        assert np.abs(q - q_ref).max() <= 1e-5
    else:
        assert np.abs(q - q_ref).sum(axis=1).max() <= 2e-2  # total variation, bf16 logits
    assert np.abs(q.sum(axis=1) - 1).max() <= 1e-4
    res = compare(np.zeros(B, np.int32), got_t[:, 1:2], r["logits"], np.zeros((B, 0), np.int32),
                  np.zeros((B, 0, shape.vocab)), u[:, None], gpu_logits=np.log(np.maximum(q, 1e-300))[:, None])
    assert not res["mismatches"] and res["checked"] >= B // 2


def device_error_ws(ws, n):
    return nb.device_error(ws.data_ptr(), n, _s())


def _sd_setup(tshape, dshape, k, B, steps, ctx):
    ct = W.make_context(tshape, ctx, steps * (k + 1) + 1, seed=0)
    cd = W.make_context(dshape, ctx, steps * (k + 1) + 1, seed=1)
    cd["block_table"] = ct["block_table"]  # one shared table; the draft pool is as large as the target's
    assert cd["num_blocks"] == ct["num_blocks"]
    return ct, cd


def _sd_run(mt, md, cache_t, cache_d, tws, tn, dws, dn, last, du, u, B, k, V):
    dt = torch.zeros((B, k), dtype=torch.int32, device="cuda")
    dq = torch.zeros((B, k, V), device="cuda", dtype=torch.float32)
    acc = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    nxt = torch.full((B, k + 1), -7, dtype=torch.int32, device="cuda")
    dl, ddu, dtu = (torch.from_numpy(a).cuda() for a in (last, du, u))
    nb.sd_step(mt.desc, mt.c, cache_t.c, md.desc, md.c, cache_d.c, cache_t.block_table.data_ptr(),
               cache_t.max_blocks, cache_t.context_lens.data_ptr(), dl.data_ptr(), ddu.data_ptr(), dtu.data_ptr(),
               B, k, dt.data_ptr(), dq.data_ptr(), acc.data_ptr(), nxt.data_ptr(), tws.data_ptr(), tn,
               dws.data_ptr(), dn, _s())
    assert device_error_ws(tws, tn) == 0 and device_error_ws(dws, dn) == 0
    return dt.cpu().numpy(), dq.cpu().numpy(), acc.cpu().numpy(), nxt.cpu().numpy()


def test_sd_step_bf16_invariants():
    """bf16 models (a 2-layer target, a 1-layer draft, vocab 4112): the step's
    structure -- accepted prefix = drafts, n + 1 tokens, -1 padding, contexts
    advanced by n + 1, q rows normalised -- over three consecutive steps, and
    the first chain position's q against the oracle (total variation 2e-2)."""
    B, k, steps = 4, 4, 3
    ctx = np.array([20, 0, 47, 130], np.int32)
    ct, cd = _sd_setup(SMALL_BF16, DRAFT_BF16, k, B, steps, ctx)
    wt, wd = W.make_weights(SMALL_BF16, 5), W.make_weights(DRAFT_BF16, 6)
    mt, md = DeviceModel(SMALL_BF16, wt), DeviceModel(DRAFT_BF16, wd)
    cache_t, cache_d = DeviceCache(ct), DeviceCache(cd)
    tws, tn = _ws(mt.desc, B, k)
    dws, dn = _ws(md.desc, B, 0, sd=True)
    rng = np.random.default_rng(8)
    last = rng.integers(0, SMALL_BF16.vocab, B).astype(np.int32)
    for step in range(steps):
        c0 = cache_t.context_lens.cpu().numpy()
        du = rng.random((B, k + 1)).astype(np.float32)
        u = rng.random((B, k + 1)).astype(np.float32)
        g_drafts, g_q, g_acc, g_nxt = _sd_run(mt, md, cache_t, cache_d, tws, tn, dws, dn, last, du, u, B, k,
                                              SMALL_BF16.vocab)
        if step == 0:
            _, q0, _ = S.draft_forward(wd, DRAFT_BF16, cd["k_pages"], cd["v_pages"], cd["block_table"], ctx, last,
                                       du[:, 0])
            assert np.abs(g_q[:, 0] - q0).sum(axis=1).max() <= 2e-2
        assert np.abs(g_q.sum(axis=-1) - 1).max() <= 1e-4
        assert np.all((g_acc >= 0) & (g_acc <= k))
        for b in range(B):
            assert list(g_nxt[b, : g_acc[b]]) == list(g_drafts[b, : g_acc[b]])
            assert np.all(g_nxt[b, g_acc[b] + 1:] == -1) and g_nxt[b, g_acc[b]] >= 0
        assert np.array_equal(cache_t.context_lens.cpu().numpy(), c0 + g_acc + 1)
        last = np.array([g_nxt[b, g_acc[b]] for b in range(B)], np.int32)


@pytest.mark.parametrize("k", [3, 1])
def test_sd_steps_match_the_oracle_composition(k):
    tshape, dshape = W.TINY_F32, DRAFT_F32
    """Three consecutive whole steps (draft chain, verify, both appends): drafts,
    q, accepted lengths, emitted tokens, context lengths and the pages of both
    caches at the committed positions."""
    B, steps = 4, 3
    ctx = np.array([20, 0, 47, 130], np.int32)
    ct, cd = _sd_setup(tshape, dshape, k, B, steps, ctx)
    wt, wd = W.make_weights(tshape, 5), W.make_weights(dshape, 6)
    mt, md = DeviceModel(tshape, wt), DeviceModel(dshape, wd)
    cache_t, cache_d = DeviceCache(ct), DeviceCache(cd)
    tws, tn = _ws(mt.desc, B, k)
    dws, dn = _ws(md.desc, B, 0, sd=True)
    rng = np.random.default_rng(7)
    last = rng.integers(0, tshape.vocab, B).astype(np.int32)
    tgt = {"weights": wt, "shape": tshape, "k_pages": ct["k_pages"], "v_pages": ct["v_pages"]}
    drf = {"weights": wd, "shape": dshape, "k_pages": cd["k_pages"], "v_pages": cd["v_pages"]}
    cx = ctx.copy()
    live = np.ones(B, bool)  # sequences whose GPU and oracle histories still agree
    for step in range(steps):
        du = rng.random((B, k + 1)).astype(np.float32)
        u = rng.random((B, k + 1)).astype(np.float32)
        g_drafts, g_q, g_acc, g_nxt = _sd_run(mt, md, cache_t, cache_d, tws, tn, dws, dn, last, du, u, B, k,
                                              tshape.vocab)
        out = S.sd_step(tgt, drf, ct["block_table"], cx, last, du, u, k)
        g_ctx = cache_t.context_lens.cpu().numpy()
        for b in range(B):
            if not live[b]:
                continue
            if not np.array_equal(g_drafts[b], out["drafts"][b]):
                # a chain draw may only differ where the draw sits within the margin
                i = int(np.nonzero(g_drafts[b] != out["drafts"][b])[0][0])
                c = np.cumsum(out["q"][b, i])
                tgt_u = du[b, i] * c[-1]
                j = int(out["drafts"][b, i])
                assert min(abs(tgt_u - (c[j - 1] if j else 0.0)), abs(c[j] - tgt_u)) < CDF_MARGIN, (step, b, i)
                live[b] = False
                continue
            assert np.abs(g_q[b] - out["q"][b]).sum(axis=-1).max() <= 1e-5
            res = compare(g_acc[b:b + 1], g_nxt[b:b + 1], out["logits"][b:b + 1], out["drafts"][b:b + 1],
                          out["q"][b:b + 1], u[b:b + 1])
            assert not res["mismatches"], (step, b, res)
            if res["flagged"]:
                live[b] = False
                continue
            assert g_ctx[b] == out["context_lens"][b] == cx[b] + g_acc[b] + 1
        assert live.sum() >= B - 1
        # the next step: both sides continue from their own outputs
        last_g = np.array([g_nxt[b, g_acc[b]] for b in range(B)], np.int32)
        last_o = np.array([out["next_tokens"][b, out["accepted_len"][b]] for b in range(B)], np.int32)
        live &= last_g == last_o
        last = last_o  # inputs come from the oracle; dead sequences are not compared
        cache_t.context_lens.copy_(torch.from_numpy(out["context_lens"]).cuda())
        tgt = {**tgt, "k_pages": out["target_pages"][0], "v_pages": out["target_pages"][1]}
        drf = {**drf, "k_pages": out["draft_pages"][0], "v_pages": out["draft_pages"][1]}
        cx = out["context_lens"]
