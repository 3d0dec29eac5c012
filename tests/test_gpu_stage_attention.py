"""Stage parity of the attention inputs and of the paged verify attention,
through the C ABI entry points nightjar_rmsnorm_rope and
nightjar_attn_verify, element by element against the oracle's rms_norm, rope
and attention (Sec. 2.1: paged KV blocks reached through a block table;
Sec. 2.2: the k+1 window rows of a sequence are scored together).

Tolerances (bf16 storage of q, K/V, the probabilities fed to the P.V product
and the output; fp32 sums): one bf16 rounding is at most 2^-9 relative, about
1.1e-3 rms, and an output passes through two or three of them, so each
(row, head) vector is held to a relative L2 error of 1e-2 (attention) or 5e-3
(projection + RoPE).  fp32 paths are held to 1e-5 relative.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2512_22420_amd import binding as nb
from paper_2512_22420_amd import workload as W
from paper_2512_22420_amd.device import model_desc, pack_weight

pytestmark = pytest.mark.gpu


def _dev(a):
    a = np.ascontiguousarray(a)
    return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).cuda()


def _s():
    return torch.cuda.current_stream().cuda_stream


def _store(x, dtype):
    return W.f32_to_bf16_bits(x.astype(np.float32)) if dtype == "bf16" else x.astype(np.float32)


def _host(t, dtype):
    a = t.cpu().numpy()
    return oracle.widen(a.view(np.uint16) if dtype == "bf16" else a, dtype)


def _ws(nbytes):
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    nb.workspace_init(ws.data_ptr(), nbytes, _s())
    return ws


def _rel_rows(got, ref):
    got = got.reshape(-1, got.shape[-1])
    ref = ref.reshape(-1, ref.shape[-1])
    return np.linalg.norm(got - ref, axis=1) / np.maximum(np.linalg.norm(ref, axis=1), 1e-30)


# shapes: the 8B head layout (G = 4), the Qwen head layout (G = 7), the tiny fp32 model
L8 = W.LLAMA8B_LAYER
QW = W.QWEN7B
TF = W.TINY_F32


def _attn_case(shape, ctx, k, seed):
    rng = np.random.default_rng(seed)
    B, T = len(ctx), k + 1
    H, Hkv, D = shape.n_heads, shape.n_kv_heads, shape.head_dim
    c = W.make_context(dataclasses.replace(shape, n_layers=1), ctx, k, seed=seed)
    q = _store(rng.standard_normal((B * T, H, D)), shape.dtype)
    wk = np.zeros((B, Hkv, 16, D), np.float32)
    wv = np.zeros((B, Hkv, D, 16), np.float32)
    wk[:, :, :T, :] = rng.standard_normal((B, Hkv, T, D)) * 0.5
    wv[:, :, :, :T] = rng.standard_normal((B, Hkv, D, T)) * 0.5
    return c, q, _store(wk, shape.dtype), _store(wv, shape.dtype)


def _attn_oracle(shape, c, q, wk, wv, ctx, k):
    dt = shape.dtype
    B, T = len(ctx), k + 1
    H, D = shape.n_heads, shape.head_dim
    kp, vp = oracle.widen(c["k_pages"][0], dt), oracle.widen(c["v_pages"][0], dt)
    qf = oracle.widen(q, dt).reshape(B, T, H, D)
    kwin = oracle.widen(wk, dt)[:, :, :T, :].transpose(0, 2, 1, 3)   # [B, T, Hkv, D]
    vwin = oracle.widen(wv, dt)[:, :, :, :T].transpose(0, 3, 1, 2)
    out = np.empty((B, T, H, D))
    for b in range(B):
        kc, vc = oracle.gather_cache(kp, vp, c["block_table"][b], int(ctx[b]), 16)
        out[b] = oracle.attention(qf[b], kc, vc, kwin[b], vwin[b])
    return out.reshape(B * T, H, D)


def _attn_gpu(shape, c, q, wk, wv, ctx, k, table=None):
    B, T = len(ctx), k + 1
    desc = model_desc(shape)
    n = nb.attn_workspace_bytes(desc, B, k)
    ws = _ws(n)
    dq, dkp, dvp, dwk, dwv = _dev(q), _dev(c["k_pages"][0]), _dev(c["v_pages"][0]), _dev(wk), _dev(wv)
    dt = _dev(c["block_table"] if table is None else table)
    dc = _dev(np.asarray(ctx, np.int32))
    out = torch.full((B * T, shape.n_heads * shape.head_dim), -1,
                     dtype=torch.int16 if shape.dtype == "bf16" else torch.float32, device="cuda")
    nb.attn_verify(desc, dq.data_ptr(), dkp.data_ptr(), dvp.data_ptr(), c["num_blocks"], dwk.data_ptr(),
                   dwv.data_ptr(), dt.data_ptr(), c["block_table"].shape[1], dc.data_ptr(), B, k, out.data_ptr(),
                   ws.data_ptr(), n, _s())
    err = nb.device_error(ws.data_ptr(), n, _s())
    return _host(out, shape.dtype).reshape(B * T, shape.n_heads, shape.head_dim), err


def _many(B, seed):
    """B short contexts (0..40 tokens) with every 50th one long (1500..2047): the
    work list gives the long ones several splits and the short ones one."""
    rng = np.random.default_rng(seed)
    ctx = rng.integers(0, 41, size=B)
    ctx[::50] = rng.integers(1500, 2048, size=len(ctx[::50]))
    return ctx.tolist()


@pytest.mark.parametrize("shape,ctx,k", [
    (L8, [0, 5, 16, 37, 1000, 2047], 3),          # ragged: empty, partial, exact block, long
    (L8, [2047, 0, 3], 15),                       # R = 16 x 4 = 64 query rows; empty KV splits of short rows
    (L8, [1024] * 8, 5),                          # the headline shape
    (L8, [0], 0),                                 # window only, one row
    (QW, [300, 0, 47, 4000], 8),                  # G = 7: 63 query rows
    (QW, [129, 1], 2),
    (TF, [32, 48, 0], 3),                         # fp32 path
    (L8, _many(64, 3), 4),                        # work list: the one-wave path at its largest batch
    (L8, _many(65, 4), 2),                        # work list: the block-wide path at its smallest batch
    (L8, _many(600, 1), 3),                       # work list: more sequences than half its threads
    (L8, _many(1100, 2), 1),                      # work list: five sequences per thread (contexts re-read)
], ids=["8b-ragged", "8b-r64", "8b-headline", "8b-window-only", "g7-r63", "g7-k2", "f32", "8b-b64-work-list",
        "8b-b65-work-list", "8b-b600-work-list", "8b-b1100-work-list"])
def test_attn_verify_matches_oracle(shape, ctx, k):
    ctx = np.asarray(ctx, np.int32)
    c, q, wk, wv = _attn_case(shape, ctx, k, seed=int(ctx.sum()) + k)
    got, err = _attn_gpu(shape, c, q, wk, wv, ctx, k)
    assert err == 0
    ref = _attn_oracle(shape, c, q, wk, wv, ctx, k)
    r = _rel_rows(got, ref)
    if shape.dtype == "bf16":
        assert r.max() <= 1e-2, (r.max(), np.unravel_index(r.argmax(), got.shape[:2]))
    else:
        assert np.abs(got - ref).max() <= 1e-5 * max(1.0, np.abs(ref).max())


def test_attn_verify_paging_is_invisible():
    """Relabelled physical blocks with their contents moved: bitwise the same output."""
    shape, ctx, k = L8, np.array([700, 33, 0, 1500], np.int32), 4
    c, q, wk, wv = _attn_case(shape, ctx, k, seed=3)
    got1, _ = _attn_gpu(shape, c, q, wk, wv, ctx, k)
    perm = np.random.default_rng(2).permutation(c["num_blocks"])
    inv = np.argsort(perm)
    c2 = dict(c)
    c2["k_pages"] = [c["k_pages"][0][inv]]
    c2["v_pages"] = [c["v_pages"][0][inv]]
    table = np.where(c["block_table"] >= 0, perm[np.maximum(c["block_table"], 0)], -1).astype(np.int32)
    got2, _ = _attn_gpu(shape, c2, q, wk, wv, ctx, k, table=table)
    assert np.array_equal(got1, got2)


def test_attn_verify_flags_bad_blocks_without_faults():
    shape, ctx, k = L8, np.array([100, 40], np.int32), 2
    c, q, wk, wv = _attn_case(shape, ctx, k, seed=4)
    for bad in (-1, c["num_blocks"], 1 << 30):
        t = c["block_table"].copy()
        t[1, 1] = bad
        _, err = _attn_gpu(shape, c, q, wk, wv, ctx, k, table=t)
        assert err & nb.NJ_DEV_BAD_BLOCK, bad


# --------------------------------------------------------------------------
# RMSNorm + QKV projection + RoPE + window store
# --------------------------------------------------------------------------
def _pre_case(shape, B, k, seed):
    rng = np.random.default_rng(seed)
    M = B * (k + 1)
    h = (rng.standard_normal((M, shape.d_model)) * rng.uniform(0.05, 3.0, size=(M, 1))).astype(np.float32)
    g = _store(1.0 + 0.2 * rng.standard_normal(shape.d_model), shape.dtype)
    w = _store(rng.standard_normal((shape.qkv_dim, shape.d_model)) * 0.02, shape.dtype)
    return h, g, w


@pytest.mark.parametrize("shape,ctx,k", [
    (L8, [0, 17, 1000], 5),                             # 18 rows: norm folded into the QKV GEMM, RoPE in its epilogue
    (L8, [1024] * 8, 5),                                # 48 rows, the headline window
    (L8, list(range(0, 64 * 31, 31)), 5),               # 384 rows: norm kernel, tiled GEMM, RoPE kernel
    (QW, [4000, 3, 1500], 7),                           # Qwen layout (d 3584, G 7), theta 1e6
    (TF, [32, 48], 3),                                  # fp32 path
], ids=["8b-18rows", "8b-48rows", "8b-384rows", "qwen-24rows", "f32"])
def test_rmsnorm_rope_matches_oracle(shape, ctx, k):
    ctx = np.asarray(ctx, np.int32)
    B, T = len(ctx), k + 1
    M = B * T
    H, Hkv, D = shape.n_heads, shape.n_kv_heads, shape.head_dim
    h, g, w = _pre_case(shape, B, k, seed=M)
    desc = model_desc(shape)
    n = nb.rmsnorm_rope_workspace_bytes(desc, B, k)
    ws = _ws(n)
    bf = shape.dtype == "bf16"
    et = torch.int16 if bf else torch.float32
    dh, dg, dc = _dev(h), _dev(g), _dev(ctx)
    dw = pack_weight(_dev(w)) if bf else _dev(w)
    q = torch.full((M, H, D), -1, dtype=et, device="cuda")
    wk = torch.full((B, Hkv, 16, D), -1, dtype=et, device="cuda")
    wv = torch.full((B, Hkv, D, 16), -1, dtype=et, device="cuda")
    nb.rmsnorm_rope(desc, dh.data_ptr(), dg.data_ptr(), dw.data_ptr(), dc.data_ptr(), B, k, q.data_ptr(),
                    wk.data_ptr(), wv.data_ptr(), ws.data_ptr(), n, _s())
    assert nb.device_error(ws.data_ptr(), n, _s()) == 0
    # oracle: x = RMSNorm(h) * g, [q|k|v] = x W^T, RoPE at ctx_b + i
    x = oracle.rms_norm(h.astype(np.float64), oracle.widen(g, shape.dtype), shape.rms_eps)
    qkv = oracle.linear(x, w, shape.dtype)
    pos = (ctx[:, None] + np.arange(T)[None, :]).reshape(-1)
    rq = oracle.rope(qkv[:, : H * D].reshape(M, H, D), pos, shape.rope_theta)
    rk = oracle.rope(qkv[:, H * D: (H + Hkv) * D].reshape(M, Hkv, D), pos, shape.rope_theta).reshape(B, T, Hkv, D)
    rv = qkv[:, (H + Hkv) * D:].reshape(B, T, Hkv, D)
    gq = _host(q, shape.dtype)
    gk = _host(wk, shape.dtype)
    gv = _host(wv, shape.dtype)
    gk_rows = gk[:, :, :T, :].transpose(0, 2, 1, 3)
    gv_rows = gv[:, :, :, :T].transpose(0, 3, 1, 2)
    tol = 5e-3 if bf else 1e-5
    for got, ref in ((gq, rq), (gk_rows, rk), (gv_rows, rv)):
        r = _rel_rows(got, ref)
        assert r.max() <= tol, r.max()
    # slots past the window are zero
    assert np.all(gk[:, :, T:, :] == 0) and np.all(gv[:, :, :, T:] == 0)
