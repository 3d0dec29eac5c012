"""Plain CPU oracle of the batched speculative verify step.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run this module.  The
product path (the HIP library and its binding) never calls it, and it shares
no code with that path: it reads the same seeded inputs and nothing else.

What it computes (Nightjar, arXiv 2512.22420):

* Sec. 2.2 (Speculative Decoding): a draft model proposes gamma tokens; the
  target model scores all of them in one forward pass; a wrong draft is thrown
  away at the first error and replaced by a corrected token.
* Sec. 3.1 and Sec. 5.1 (goodput): a step commits the n accepted drafts plus
  one extra target token, so gamma drafts give n+1 tokens, 0 <= n <= gamma.
* Sec. 1 and Sec. 6.5: the output distribution equals the target model's.
  The paper states no formula for the test; it cites the standard speculative
  sampling method (Leviathan et al., 2023), which is what `accept` runs:
  accept draft x_i with probability min(1, p_i(x_i)/q_i(x_i)); at the first
  rejection draw from the normalised residual max(0, p_i - q_i); if every
  draft is accepted draw the bonus token from p_gamma.
* Sec. 2.1 (PagedAttention): cached keys and values live in fixed-size blocks
  reached through a per-sequence block table.
* Sec. 4 / Sec. 6.5: gamma = 0 is plain autoregressive decoding, and a step is
  finalised (its accepted tokens' KV written) before the next one starts.

The target is a Llama-style decoder (RMSNorm, rotate-half RoPE, grouped-query
attention, SwiGLU FFN, untied LM head).  Every floating-point step runs in
fp64 on the exact stored weight values (bf16 bit patterns are widened
exactly; large matrices are widened one block of rows at a time).  Readings of points the paper leaves open are listed where they are
used; all of them are also collected in the design notes of the repository.

Parity: the acceptance rule and the inverse-CDF draw are pinned by exact
enumeration (the output distribution equals the target's), the forward pass by
an independent Llama implementation (HuggingFace ``transformers``) on the same
weights, the paging by block-table permutation invariance.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np


# --------------------------------------------------------------------------
# Storage decoding
# --------------------------------------------------------------------------
def widen(a: np.ndarray, dtype: str) -> np.ndarray:
    """Stored tensor -> fp64.  bf16 bit patterns (uint16) are widened exactly."""
    if dtype == "bf16":
        bits = np.asarray(a, dtype=np.uint16).astype(np.uint32) << 16
        return bits.view(np.float32).astype(np.float64)
    return np.asarray(a, dtype=np.float64)


# --------------------------------------------------------------------------
# Decoder building blocks
# --------------------------------------------------------------------------
def rms_norm(h: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """h / sqrt(mean(h^2) + eps) * gain, over the last axis."""
    return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps) * gain


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding.  x [T, heads, D], pos [T].

    Dim pair (j, j + D/2) turns by pos * theta^(-2j/D):
    (a, b) -> (a cos - b sin, b cos + a sin).
    """
    D = x.shape[-1]
    half = D // 2
    inv_freq = theta ** (-2.0 * np.arange(half, dtype=np.float64) / D)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * cos - b * sin, b * cos + a * sin], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def softmax(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, dtype=np.float64)
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def gather_cache(k_page: np.ndarray, v_page: np.ndarray, table_row: np.ndarray,
                 n_tokens: int, block_size: int) -> Tuple[np.ndarray, np.ndarray]:
    """Cached keys/values of one sequence in logical order (PagedAttention, Sec. 2.1).

    Token t lives in physical block table_row[t // block_size] at slot
    t % block_size.  K pages are [blocks][Hkv][slot][D]; V pages are
    [blocks][Hkv][D][slot].  Returns K, V as [n_tokens, Hkv, D].
    """
    t = np.arange(n_tokens)
    blk = np.asarray(table_row)[t // block_size]
    slot = t % block_size
    K = k_page[blk, :, slot, :]      # advanced indices first: [T, Hkv, D]
    V = v_page[blk, :, :, slot]      # [T, Hkv, D]
    return K, V


def attention(q: np.ndarray, k_cache: np.ndarray, v_cache: np.ndarray,
              k_win: np.ndarray, v_win: np.ndarray) -> np.ndarray:
    """Verify attention of one sequence.

    q [T, H, D] are the T = gamma+1 window queries; the keys are the cached
    ones [C, Hkv, D] followed by the window's own [T, Hkv, D].  Window query i
    sees every cached key and window keys 0..i.  Query head h reads KV head
    h // (H / Hkv).  Scores are scaled by 1/sqrt(D).
    """
    T, H, D = q.shape
    C, Hkv = k_cache.shape[0], k_cache.shape[1]
    G = H // Hkv
    keys = np.concatenate([k_cache, k_win], axis=0)     # [C+T, Hkv, D]
    vals = np.concatenate([v_cache, v_win], axis=0)
    visible = np.ones((T, C + T), dtype=bool)
    for i in range(T):
        visible[i, C + i + 1:] = False
    out = np.empty_like(q)
    for h in range(H):
        g = h // G
        s = q[:, h, :] @ keys[:, g, :].T / np.sqrt(D)   # [T, C+T]
        s = np.where(visible, s, -np.inf)
        p = softmax(s)
        out[:, h, :] = p @ vals[:, g, :]
    return out


# --------------------------------------------------------------------------
# Forward over the verify window
# --------------------------------------------------------------------------
def linear(x: np.ndarray, w: np.ndarray, dtype: str, rows: int = 8192) -> np.ndarray:
    """x @ W^T for a weight stored [N, K]; W is widened to fp64 one block of rows
    at a time so that no full fp64 copy of a large matrix is made."""
    out = np.empty((x.shape[0], w.shape[0]))
    for r0 in range(0, w.shape[0], rows):
        out[:, r0: r0 + rows] = x @ widen(w[r0: r0 + rows], dtype).T
    return out


def forward_window(weights: Dict, shape, k_pages: Sequence[np.ndarray], v_pages: Sequence[np.ndarray],
                   block_table: np.ndarray, context_lens: np.ndarray,
                   tokens: np.ndarray) -> Tuple[np.ndarray, List[np.ndarray], List[np.ndarray]]:
    """Target forward over each sequence's window tokens against its paged cache.

    tokens [B, T]: window token ids (last committed token, then the drafts);
    window row i of sequence b sits at position context_lens[b] + i.  The
    linear layers act on every row independently, so all B*T rows go through
    them together; attention is per sequence.
    Returns logits [B, T, V] and, per layer, the window's post-RoPE keys and
    its values, each [B, T, Hkv, D].
    """
    s, dt = shape, shape.dtype
    H, Hkv, D, F = s.n_heads, s.n_kv_heads, s.head_dim, s.ffn_dim
    B, T = tokens.shape
    pos = (np.asarray(context_lens, dtype=np.int64)[:, None] + np.arange(T)[None, :]).reshape(-1)
    h = widen(weights["embed"][np.asarray(tokens).reshape(-1)], dt)     # [B*T, d]
    win_k, win_v = [], []
    for l, lw in enumerate(weights["layers"]):
        x = rms_norm(h, widen(lw["attn_norm"], dt), s.rms_eps)
        qkv = linear(x, lw["w_qkv"], dt)
        q = rope(qkv[:, : H * D].reshape(-1, H, D), pos, s.rope_theta)
        k = rope(qkv[:, H * D: (H + Hkv) * D].reshape(-1, Hkv, D), pos, s.rope_theta)
        v = qkv[:, (H + Hkv) * D:].reshape(-1, Hkv, D)
        o = np.empty_like(q)
        for b in range(B):
            rows = slice(b * T, (b + 1) * T)
            kc, vc = gather_cache(k_pages[l], v_pages[l], block_table[b], int(context_lens[b]), s.block_size)
            o[rows] = attention(q[rows], widen(kc, dt), widen(vc, dt), k[rows], v[rows])
        win_k.append(k.reshape(B, T, Hkv, D))
        win_v.append(v.reshape(B, T, Hkv, D))
        h = h + linear(o.reshape(-1, H * D), lw["w_o"], dt)
        x = rms_norm(h, widen(lw["ffn_norm"], dt), s.rms_eps)
        gu = linear(x, lw["w_gate_up"], dt)
        h = h + linear(silu(gu[:, :F]) * gu[:, F:], lw["w_down"], dt)
    x = rms_norm(h, widen(weights["final_norm"], dt), s.rms_eps)
    logits = linear(x, weights["lm_head"], dt).reshape(B, T, s.vocab)
    return logits, win_k, win_v


# --------------------------------------------------------------------------
# Acceptance (speculative sampling)
# --------------------------------------------------------------------------
def invcdf(weights: np.ndarray, u: float) -> int:
    """Draw an index from non-negative weights with one uniform u in [0, 1).

    S = sum of the weights; C_j the inclusive running sum in index order (fp64).
    Returns the smallest j with C_j > u*S.  A zero-weight index is never
    returned: if rounding leaves no such j (u close to 1), the last index with
    positive weight is returned.
    """
    wts = np.asarray(weights, dtype=np.float64)
    c = np.cumsum(wts)
    target = float(u) * c[-1]
    hit = np.nonzero(c > target)[0]
    if hit.size:
        return int(hit[0])
    return int(np.nonzero(wts > 0)[0][-1])


def accept(p: np.ndarray, q: np.ndarray, drafts: Sequence[int], u: Sequence[float]) -> Tuple[int, List[int]]:
    """Speculative acceptance for one sequence.

    p [gamma+1, V]: target distributions at the window rows (row i is the
    target's distribution for the token after window token i).
    q [gamma, V]: the draft's distributions it sampled drafts[i] from.
    u [gamma+1]: u[0..gamma-1] are the accept tests, u[gamma] the one draw of
    the corrected or bonus token.

    Draft i is accepted iff u[i] < p_i(x)/q_i(x) (q_i(x) = 0 counts as an
    accept).  With u uniform on [0, 1) this accepts with probability exactly
    min(1, p/q), and a draft the target gives probability 0 is never accepted.  At the first rejection n the token is drawn from max(0, p_n - q_n)
    (from p_n if that residual is all zero, which only rounding can cause);
    with all gamma accepted the bonus is drawn from p_gamma.
    Returns (n, tokens) with tokens = drafts[:n] + [drawn], length n+1.
    """
    gamma = len(drafts)
    n = 0
    while n < gamma:
        x = int(drafts[n])
        px, qx = float(p[n, x]), float(q[n, x])
        if qx > 0.0 and not (float(u[n]) < px / qx):
            break
        n += 1
    if n < gamma:
        r = np.maximum(0.0, p[n] - np.asarray(q[n], dtype=np.float64))
        if not np.any(r > 0):
            r = p[n]
    else:
        r = p[gamma]
    y = invcdf(r, float(u[gamma]))
    return n, [int(t) for t in drafts[:n]] + [y]


# --------------------------------------------------------------------------
# The verify step and the KV append
# --------------------------------------------------------------------------
def window_tokens(last_tokens: np.ndarray, draft_tokens: np.ndarray) -> np.ndarray:
    """[B, gamma+1] window ids: the last committed token, then the drafts."""
    return np.concatenate([np.asarray(last_tokens)[:, None], np.asarray(draft_tokens).reshape(len(last_tokens), -1)], axis=1).astype(np.int64)


def verify_step(weights, shape, k_pages, v_pages, block_table, context_lens,
                last_tokens, draft_tokens, draft_probs, uniforms) -> Dict:
    """One verify step for B sequences with gamma drafts each.

    Returns accepted_len [B], next_tokens [B, gamma+1] (-1 past the n+1
    emitted tokens), logits [B, gamma+1, V], target probabilities, and the
    window keys/values that a KV append would commit.
    """
    B = len(last_tokens)
    toks = window_tokens(last_tokens, draft_tokens)
    gamma = toks.shape[1] - 1
    logits, win_k, win_v = forward_window(weights, shape, k_pages, v_pages, block_table, context_lens, toks)
    probs = softmax(logits)
    acc = np.zeros(B, dtype=np.int32)
    nxt = np.full((B, gamma + 1), -1, dtype=np.int32)
    for b in range(B):
        n, out = accept(probs[b], draft_probs[b] if gamma else np.zeros((0, shape.vocab)),
                        toks[b, 1:], uniforms[b])
        acc[b] = n
        nxt[b, : n + 1] = out
    return {"accepted_len": acc, "next_tokens": nxt, "logits": logits, "probs": probs,
            "win_k": win_k, "win_v": win_v}


def kv_append(k_pages, v_pages, block_table, context_lens, accepted_len, win_k, win_v,
              block_size: int, dtype: str):
    """Commit window rows 0..n_b of each sequence to its pages (Sec. 6.5).

    Row j goes to logical position context_lens[b] + j, i.e. block
    block_table[b][pos // block_size], slot pos % block_size.  Rows past n_b
    (rejected drafts) are not written.  Returns fp64 copies of the pages and the
    new context lengths context_lens[b] + n_b + 1.
    """
    kp = [widen(a, dtype).copy() for a in k_pages]
    vp = [widen(a, dtype).copy() for a in v_pages]
    ctx = np.asarray(context_lens, dtype=np.int64).copy()
    for b in range(len(ctx)):
        for j in range(int(accepted_len[b]) + 1):
            pos = int(ctx[b]) + j
            blk, slot = int(block_table[b][pos // block_size]), pos % block_size
            for l in range(len(kp)):
                kp[l][blk, :, slot, :] = win_k[l][b, j]
                vp[l][blk, :, :, slot] = win_v[l][b, j]
        ctx[b] += int(accepted_len[b]) + 1
    return kp, vp, ctx.astype(np.int32)
