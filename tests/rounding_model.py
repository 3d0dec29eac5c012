"""The bf16 storage model of the verify step's forward pass (test
infrastructure).

It computes what the oracle computes, in fp64, but rounds to bf16 (nearest,
ties to even) at the points where the bf16 C ABI stores an intermediate in
bf16: the normed GEMM inputs, the rotated queries and keys and the values, the
attention probabilities that enter the P.V product, the attention output, and
the SwiGLU activations.  Everything else (residual stream, sums, logits) stays
exact.  The model is the error floor of any implementation with these storage
points: the GPU path is held to a bound derived from the model's own error
against the oracle, row by row.

Two forms of the RMSNorm before a GEMM:
* unfused: x = bf16(RMSNorm(h) * gain), then x . W^T;
* fused (the norm folded into the GEMM): x = bf16(h * gain), then
  (x . W^T) / rms(h).
The probabilities are rounded relative to the row's maximum score, which
matches the GPU's online softmax in distribution, not element by element.

Arrays are widened with `dtype` ("bf16": uint16 bit patterns; "f32": values
already widened, e.g. fp64 copies); the arithmetic follows oracle.verify_step
and reuses its building blocks.
"""
from __future__ import annotations

import numpy as np

import oracle
from paper_2512_22420_amd import workload as W


def bf16(x) -> np.ndarray:
    """Round to bf16 (via fp32, nearest-even) and widen back to fp64."""
    return oracle.widen(W.f32_to_bf16_bits(np.asarray(x, dtype=np.float32)), "bf16")


def forward(weights, shape, k_pages, v_pages, block_table, context_lens, tokens, fused: bool, dtype: str = None,
            rnd=bf16):
    """Logits [B, T, V] of the window tokens [B, T] with bf16 storage points
    (`rnd` the rounding applied there; the identity gives the oracle's logits)."""
    bf16 = rnd
    s = shape
    dt = s.dtype if dtype is None else dtype
    H, Hkv, D, F = s.n_heads, s.n_kv_heads, s.head_dim, s.ffn_dim
    G = H // Hkv
    B, T = tokens.shape
    pos = (np.asarray(context_lens, np.int64)[:, None] + np.arange(T)[None, :]).reshape(-1)
    h = oracle.widen(weights["embed"][np.asarray(tokens).reshape(-1)], dt)

    def normed_gemm(h, gain, w):
        r = 1.0 / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + s.rms_eps)
        g = oracle.widen(gain, dt)
        if fused:
            return oracle.linear(bf16(h * g), w, dt) * r
        return oracle.linear(bf16(h * r * g), w, dt)

    for l, lw in enumerate(weights["layers"]):
        qkv = normed_gemm(h, lw["attn_norm"], lw["w_qkv"])
        q = bf16(oracle.rope(qkv[:, : H * D].reshape(-1, H, D), pos, s.rope_theta))
        k = bf16(oracle.rope(qkv[:, H * D: (H + Hkv) * D].reshape(-1, Hkv, D), pos, s.rope_theta))
        v = bf16(qkv[:, (H + Hkv) * D:].reshape(-1, Hkv, D))
        o = np.empty_like(q)
        for b in range(B):
            rows = slice(b * T, (b + 1) * T)
            kc, vc = oracle.gather_cache(k_pages[l], v_pages[l], block_table[b], int(context_lens[b]), s.block_size)
            keys = np.concatenate([oracle.widen(kc, dt), k[rows]])
            vals = np.concatenate([oracle.widen(vc, dt), v[rows]])
            C = keys.shape[0] - T
            mask = np.zeros((T, C + T))
            for i in range(T):
                mask[i, C + i + 1:] = -np.inf
            for g in range(Hkv):
                qq = q[rows][:, g * G:(g + 1) * G, :].transpose(1, 0, 2).reshape(G * T, D)
                sc = (qq @ keys[:, g, :].T / np.sqrt(D)).reshape(G, T, -1) + mask
                p = np.exp(sc - sc.max(axis=2, keepdims=True))
                oo = (bf16(p) @ vals[:, g, :]) / p.sum(axis=2, keepdims=True)
                o[rows, g * G:(g + 1) * G, :] = oo.transpose(1, 0, 2)
        h = h + oracle.linear(bf16(o).reshape(-1, H * D), lw["w_o"], dt)
        gu = normed_gemm(h, lw["ffn_norm"], lw["w_gate_up"])
        h = h + oracle.linear(bf16(oracle.silu(gu[:, :F]) * gu[:, F:]), lw["w_down"], dt)
    return normed_gemm(h, weights["final_norm"], weights["lm_head"]).reshape(B, T, s.vocab)


def row_errors(logits, ref):
    a = np.asarray(logits, dtype=np.float64).reshape(-1, np.shape(ref)[-1])
    r = np.asarray(ref, dtype=np.float64).reshape(-1, np.shape(ref)[-1])
    return np.linalg.norm(a - r, axis=1) / np.linalg.norm(r, axis=1)


# The GPU path against the model: its per-row errors against the oracle may
# exceed the model's by these factors (the model rounds the probabilities
# against the row maximum, the GPU against a running maximum per KV chunk, and
# accumulates in fp32: same distribution of errors, not the same elements).
MEAN_FACTOR = 1.25
MAX_FACTOR = 1.35


def assert_within_model(gpu_logits, model_logits, ref_logits):
    """The GPU's logits error is statistically that of the storage model: mean
    and maximum row error within MEAN_FACTOR / MAX_FACTOR of the model's.
    Returns (gpu row errors, model row errors)."""
    eg = row_errors(gpu_logits, ref_logits)
    em = row_errors(model_logits, ref_logits)
    assert eg.mean() <= MEAN_FACTOR * em.mean(), (eg.mean(), em.mean())
    assert eg.max() <= MAX_FACTOR * em.max(), (eg.max(), em.max(), int(eg.argmax()))
    return eg, em
