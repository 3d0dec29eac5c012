"""Plain reference of a whole speculative-decoding step with a draft model
(TEST INFRASTRUCTURE: only tests/ may use it; the library shares no code with
it).

Sec. 2.2 and Sec. 3.1 of the paper: a small draft model proposes k tokens one
at a time, sampling each from its own distribution q_i; the target scores all
of them in one forward pass and accepts the longest prefix that passes the
speculative test, then adds one token; the committed tokens are the accepted
drafts plus that token.  Sec. 6.5: the step is finalised (both KV caches
hold exactly the committed tokens) before the next one starts.

Composition, each piece being the oracle's own verify step and KV append:
* draft forward i (i = 0..k) is a k = 0 verify step of the draft model on the
  previous token (the last committed token, then draft i), drawing draft i+1
  with draft uniform i and recording q_i = its distribution; forward k only
  adds draft k's keys and values (its draw is not used), so the draft cache
  holds every token the target may commit;
* the target verifies [last, d_1..d_k] with q_0..q_{k-1} and the target uniforms;
* the target appends n + 1 rows; the draft cache keeps the same n + 1 new
  positions (its context length is set to the target's).
"""
from __future__ import annotations

import numpy as np

import dataclasses

from .verify_step import kv_append, verify_step, widen


def _values(model):
    """The model with every tensor widened to fp64 values and a shape that says
    so (the KV append returns fp64 pages, so a chain works on values)."""
    s = model["shape"]
    if s.dtype == "f32":
        return model
    w = model["weights"]
    w64 = {"embed": widen(w["embed"], s.dtype), "lm_head": widen(w["lm_head"], s.dtype),
           "final_norm": widen(w["final_norm"], s.dtype),
           "layers": [{n: widen(a, s.dtype) for n, a in lw.items()} for lw in w["layers"]]}
    return {"weights": w64, "shape": dataclasses.replace(s, dtype="f32"),
            "k_pages": [widen(a, s.dtype) for a in model["k_pages"]],
            "v_pages": [widen(a, s.dtype) for a in model["v_pages"]]}


def draft_forward(weights, shape, k_pages, v_pages, block_table, context_lens, last_tokens, uniforms):
    """One draft token per sequence: (tokens [B], q [B, V], the step's record)."""
    B = len(last_tokens)
    r = verify_step(weights, shape, k_pages, v_pages, block_table, context_lens, np.asarray(last_tokens),
                    np.zeros((B, 0), np.int32), np.zeros((B, 0, shape.vocab), np.float32),
                    np.asarray(uniforms, np.float32).reshape(B, 1))
    return r["next_tokens"][:, 0].astype(np.int32), r["probs"][:, 0], r


def sd_step(target, draft, block_table, context_lens, last_tokens, draft_uniforms, uniforms, k):
    """target / draft: dicts with weights, shape, k_pages, v_pages.  Returns the
    committed outcome, the drafts and q, and both caches after the step."""
    B = len(last_tokens)
    target, draft = _values(target), _values(draft)
    ctx0 = np.asarray(context_lens, np.int32)
    dkp, dvp, dctx = draft["k_pages"], draft["v_pages"], ctx0.copy()
    drafts = np.zeros((B, k), np.int32)
    q = np.zeros((B, k, target["shape"].vocab))
    for i in range(k + 1):
        tok_in = last_tokens if i == 0 else drafts[:, i - 1]
        t, qi, r = draft_forward(draft["weights"], draft["shape"], dkp, dvp, block_table, dctx, tok_in,
                                 draft_uniforms[:, i])
        if i < k:
            drafts[:, i], q[:, i] = t, qi
        dkp, dvp, dctx = kv_append(dkp, dvp, block_table, dctx, np.zeros(B, np.int32), r["win_k"], r["win_v"],
                                   draft["shape"].block_size, "f32")
    R = verify_step(target["weights"], target["shape"], target["k_pages"], target["v_pages"], block_table, ctx0,
                    last_tokens, drafts, q, uniforms)
    tkp, tvp, tctx = kv_append(target["k_pages"], target["v_pages"], block_table, ctx0, R["accepted_len"],
                               R["win_k"], R["win_v"], target["shape"].block_size, "f32")
    return {"accepted_len": R["accepted_len"], "next_tokens": R["next_tokens"], "logits": R["logits"],
            "drafts": drafts, "q": q, "target_pages": (tkp, tvp), "draft_pages": (dkp, dvp),
            "context_lens": tctx}
