"""End-to-end parity at the large configurations, the whole batch on the GPU
and a subset of its sequences checked by the oracle (sequences are independent
in the verify step), with beta-mixed drafts from the oracle's own target
logits so that accepted drafts and bonus draws are compared at the real
vocabulary sizes:

* the 8B-shaped layer + LM head at B = 128, k = 5 (768 window rows, the largest
  point of the large-batch grid; contexts lognormal, median 768, clipped to
  [128, 2048]), beta = 0.7, 12 sequences checked;
* the 32-layer Llama-3-8B-shaped stack at B = 64, k = 4 (contexts lognormal,
  median 1024, clipped to [128, 4096]), beta = 0.7, 2 sequences checked;
* the 28-layer Qwen2.5-7B-shaped stack at B = 256, k = 7 (contexts uniform in
  [1024, 4096]), beta = 0.9, 2 sequences checked.

Logits: per-row errors against the oracle within those of the bf16 storage
model of the same path (rounding_model.py); for the one-layer case also
relative L2 <= 1e-2 over the checked rows.  Through 28 and 32 layers the
storage roundings alone compound past 1e-2 (each layer adds its own rounding
error to a residual stream the next layers amplify), so the deep stacks are
held to the model's own error instead of a fixed 1e-2.  Decisions: bit-exact
except flagged ones (parity.py), every decision also checked against the rule
on the GPU's logits.
"""
import gc

import numpy as np
import pytest
import torch

from paper_2512_22420_amd import workload as W

import rounding_model as RM
from bigcfg import BigCase, BigModel
from paper_2512_22420_amd import binding as nb
from paper_2512_22420_amd.device import model_desc
from parity import compare, record, self_check

pytestmark = pytest.mark.gpu


def _check(case, model, min_checked, overall_1e2):
    acc, nxt, gl, acc_all, err = case.run(model)
    assert err == 0
    ref = case.oracle(model)
    r = np.asarray(ref["logits"])
    fused = nb.step_folds_norms(model_desc(model.shape), case.B, case.k)
    toks = np.concatenate([case.sub_last[:, None], case.sub_drafts], axis=1)
    m = RM.forward(model.w64, model.shape64, case.sub_k, case.sub_v, case.sub_table, case.sub_ctx, toks, fused)
    eg, em = RM.assert_within_model(gl, m, r)
    total = np.linalg.norm(gl - r) / np.linalg.norm(r)
    total_m = np.linalg.norm(m - r) / np.linalg.norm(r)
    print(f"logits rel-L2: gpu {total:.3e} (rows mean {eg.mean():.3e} max {eg.max():.3e}); "
          f"storage model {total_m:.3e} (rows mean {em.mean():.3e} max {em.max():.3e})")
    if overall_1e2:
        assert total <= 1e-2
    res = compare(acc, nxt, r, case.sub_drafts, case.sub_probs, case.sub_u, gpu_logits=gl)
    sres = self_check(acc, nxt, gl, case.sub_drafts, case.sub_probs, case.sub_u)
    record(res, sres)
    assert not res["mismatches"], res["mismatches"][:5]
    assert not sres["mismatches"], sres["mismatches"][:5]
    assert res["checked"] >= min_checked, res
    # the beta-mixed drafts are accepted: multi-position accepts happen in the checked rows
    assert acc.sum() >= 1 and np.all((acc_all >= 0) & (acc_all <= case.k))
    return res


def _free(*objs):
    for o in objs:
        del o
    gc.collect()
    torch.cuda.empty_cache()


def test_llama8b_layer_b128_k5_beta_drafts():
    shape = W.LLAMA8B_LAYER
    model = BigModel(shape, seed=11)
    ctx = W.WORKLOADS["llama8b-layer-large-batch"].ctx(128, seed=0)
    checked = sorted(set(list(range(0, 128, 11)) + [int(np.argmax(ctx))]))
    case = BigCase(model, ctx, 5, checked, beta=0.7, seed=12)
    _check(case, model, min_checked=len(checked), overall_1e2=True)
    _free(case, model)


def test_llama8b_32_layers_b64_k4_subset():
    shape = W.LLAMA8B
    model = BigModel(shape, seed=21)
    ctx = W.WORKLOADS["llama8b-32layer"].ctx(64, seed=0)
    checked = [int(np.argmax(ctx)), 5]
    case = BigCase(model, ctx, 4, checked, beta=0.7, seed=22)
    _check(case, model, min_checked=2, overall_1e2=False)
    _free(case, model)


def test_qwen7b_28_layers_b256_k7_subset():
    shape = W.QWEN7B
    model = BigModel(shape, seed=31)
    ctx = W.WORKLOADS["qwen7b-28layer"].ctx(256, seed=0)
    checked = [int(np.argmax(ctx)), 200]
    case = BigCase(model, ctx, 7, checked, beta=0.9, seed=32)
    _check(case, model, min_checked=2, overall_1e2=False)
    _free(case, model)
