"""Pins of the whole speculative-decoding step of the oracle (oracle/spec_step.py).

* Draft = target (the same weights): the chain samples the target itself, so
  every draft is accepted (q = p) and the k+1 committed tokens are the target's
  own autoregressive samples: the chain's k tokens with the draft uniforms and
  the bonus with the target's last uniform (Sec. 2.2, Sec. 3.1).  The rollout
  is the oracle's gamma = 0 chain, itself pinned against the HuggingFace Llama
  model in test_oracle_forward.py.
* Invariants of any step: 0 <= n <= k, the committed prefix is the drafts, the
  context grows by n + 1, and the draft cache agrees with the target's on every
  committed position's logits afterwards (the next step sees both in step).
"""
import dataclasses

import numpy as np

import oracle
from oracle import spec_step as S
from paper_2512_22420_amd import workload as W


def _model(shape, seed, ctx, k):
    c = W.make_context(shape, ctx, 3 * (k + 1), seed=0)  # both caches share one table (seed 0)
    src = W.make_context(shape, ctx, 3 * (k + 1), seed=seed)
    return {"weights": W.make_weights(shape, seed), "shape": shape, "k_pages": src["k_pages"],
            "v_pages": src["v_pages"]}, c


def test_draft_equal_to_target_commits_the_targets_own_samples():
    shape = W.TINY_F32
    ctx = np.array([20, 33], np.int32)
    k = 3
    tgt, c = _model(shape, 1, ctx, k)
    drf = dict(tgt)
    rng = np.random.default_rng(0)
    du = rng.random((2, k + 1)).astype(np.float32)
    u = rng.random((2, k + 1)).astype(np.float32) * 0.999
    out = S.sd_step(tgt, drf, c["block_table"], ctx, np.array([5, 900], np.int32), du, u, k)
    assert list(out["accepted_len"]) == [k, k]
    # the target's own rollout with the same uniforms: gamma = 0 steps with appends
    kp, vp, cx = tgt["k_pages"], tgt["v_pages"], ctx.copy()
    last = np.array([5, 900], np.int32)
    for i in range(k + 1):
        ui = u[:, k:k + 1] if i == k else du[:, i:i + 1]
        r = oracle.verify_step(tgt["weights"], shape, kp, vp, c["block_table"], cx, last, np.zeros((2, 0), np.int32),
                               np.zeros((2, 0, shape.vocab), np.float32), ui)
        tok = r["next_tokens"][:, 0]
        assert list(tok) == list(out["next_tokens"][:, i])
        kp, vp, cx = oracle.kv_append(kp, vp, c["block_table"], cx, r["accepted_len"], r["win_k"], r["win_v"], 16,
                                      "f32")
        last = tok.astype(np.int32)


def test_step_invariants_and_caches_in_step():
    shape = W.TINY_F32
    dshape = dataclasses.replace(W.TINY_F32, name="tiny-draft", d_model=128, n_heads=2, n_kv_heads=2, ffn_dim=256)
    ctx = np.array([16, 40, 3], np.int32)
    k = 4
    tgt, c = _model(shape, 2, ctx, k)
    drf, _ = _model(dshape, 3, ctx, k)
    rng = np.random.default_rng(1)
    last = np.array([7, 1500, 42], np.int32)
    cx = ctx.copy()
    for step in range(3):
        du = rng.random((3, k + 1)).astype(np.float32)
        u = rng.random((3, k + 1)).astype(np.float32)
        out = S.sd_step(tgt, drf, c["block_table"], cx, last, du, u, k)
        n = out["accepted_len"]
        assert np.all((n >= 0) & (n <= k))
        for b in range(3):
            assert list(out["next_tokens"][b, : n[b]]) == list(out["drafts"][b, : n[b]])
        assert np.array_equal(out["context_lens"], cx + n + 1)
        # the draft cache holds the keys and values of the committed tokens
        # [last, d_1..d_n] at positions ctx .. ctx+n, as a draft forward over
        # exactly those tokens computes them
        dk, dv = out["draft_pages"]
        for b in range(3):
            toks = np.concatenate([[last[b]], out["drafts"][b, : n[b]]])[None, :]
            _, wk, wv = oracle.forward_window(drf["weights"], drf["shape"], drf["k_pages"], drf["v_pages"],
                                              c["block_table"][b:b + 1], cx[b:b + 1], toks)
            for j in range(n[b] + 1):
                pos = cx[b] + j
                blk, slot = c["block_table"][b][pos // 16], pos % 16
                np.testing.assert_allclose(dk[0][blk, :, slot, :], wk[0][0, j], rtol=0, atol=1e-12)
                np.testing.assert_allclose(dv[0][blk, :, :, slot], wv[0][0, j], rtol=0, atol=1e-12)
        # next step's caches: the target's appended pages, the draft's pages
        tgt = {**tgt, "k_pages": out["target_pages"][0], "v_pages": out["target_pages"][1],
               "shape": dataclasses.replace(tgt["shape"], dtype="f32")}
        drf = {**drf, "k_pages": dk, "v_pages": dv, "shape": dataclasses.replace(drf["shape"], dtype="f32")}
        last = np.array([out["next_tokens"][b, n[b]] for b in range(3)], np.int32)
        cx = out["context_lens"]
