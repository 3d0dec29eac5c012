"""nightjar_accept_noalloc (no workspace: a fixed device array as scratch)
against nightjar_accept through the C ABI: the same kernels, so the same
accepted lengths and tokens bit for bit, on two calls in a row, the second
with a smaller input (the array keeps the first call's contents)."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2512_22420_amd import binding as nb
from paper_2512_22420_amd import workload as W
from paper_2512_22420_amd.device import model_desc

from parity import compare

pytestmark = pytest.mark.gpu


def _s():
    return torch.cuda.current_stream().cuda_stream


def _case(B, k, V, seed):
    rng = np.random.default_rng(seed)
    logits = (rng.standard_normal((B, k + 1, V)) * 2).astype(np.float32)
    z = 0.7 * logits[:, :k].astype(np.float64) + 0.3 * rng.standard_normal((B, k, V)) * 2.0
    q = oracle.softmax(z).astype(np.float32)
    drafts = np.array([[oracle.invcdf(q[b, i].astype(np.float64), rng.random()) for i in range(k)]
                       for b in range(B)], dtype=np.int32).reshape(B, k)
    u = rng.random((B, k + 1), dtype=np.float32)
    return logits, drafts, q, u


def _both(V, logits, drafts, q, u):
    B, T, _ = logits.shape
    k = T - 1
    desc = model_desc(dataclasses.replace(W.TINY_F32, vocab=V))
    dl, dd, dq, du = (torch.from_numpy(a).cuda() for a in (logits, drafts, q, u))
    # reference: the workspace entry point
    n = nb.accept_workspace_bytes(V, B, k)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    nb.workspace_init(ws.data_ptr(), n, _s())
    acc_w = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    nxt_w = torch.full((B, T), -7, dtype=torch.int32, device="cuda")
    nb.accept(desc, dl.data_ptr(), dd.data_ptr(), dq.data_ptr(), du.data_ptr(), B, k, acc_w.data_ptr(),
              nxt_w.data_ptr(), ws.data_ptr(), n, _s())
    err_w = nb.device_error(ws.data_ptr(), n, _s())
    # the entry point without a workspace
    acc = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    nxt = torch.full((B, T), -7, dtype=torch.int32, device="cuda")
    err = torch.full((1,), 12345, dtype=torch.int32, device="cuda")
    nb.accept_noalloc(desc, dl.data_ptr(), dd.data_ptr(), dq.data_ptr(), du.data_ptr(), B, k, acc.data_ptr(),
                      nxt.data_ptr(), err.data_ptr(), _s())
    torch.cuda.synchronize()
    return acc.cpu().numpy(), nxt.cpu().numpy(), int(err.item()), acc_w.cpu().numpy(), nxt_w.cpu().numpy(), err_w


def test_accept_noalloc_matches_workspace_entry_point():
    for (B, k, V, seed) in [(64, 5, 128256, 1), (8, 3, 32000, 2)]:  # second call smaller than the first
        logits, drafts, q, u = _case(B, k, V, seed)
        acc, nxt, err, acc_w, nxt_w, err_w = _both(V, logits, drafts, q, u)
        assert err == 0 and err_w == 0
        assert np.array_equal(acc, acc_w) and np.array_equal(nxt, nxt_w), (B, k, V)
        res = compare(acc, nxt, logits, drafts, q, u)
        assert not res["mismatches"] and res["checked"] >= B // 2


def test_accept_noalloc_reports_bad_drafts_and_rejects_oversize():
    B, k, V = 4, 2, 1000
    logits, drafts, q, u = _case(B, k, V, 3)
    drafts[1, 0] = V + 3
    acc, nxt, err, _, _, err_w = _both(V, logits, drafts, q, u)
    assert err & nb.NJ_DEV_BAD_TOKEN and err_w & nb.NJ_DEV_BAD_TOKEN
    desc = model_desc(dataclasses.replace(W.TINY_F32, vocab=152064))
    rc = nb.lib().nightjar_accept_noalloc(__import__("ctypes").byref(desc), 16, 16, 16, 16, 256, 15, 16, 16, 16, 0)
    assert rc == nb.NJ_EINVAL and "scratch" in nb.last_error()
