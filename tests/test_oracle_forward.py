"""Pins of the oracle's target forward, paging and KV append.

The paper prints no logits or worked example of the forward pass, so the
oracle's decoder is pinned against an independent Llama implementation
(HuggingFace ``transformers``, fp64, eager attention) on the same weights:

* verify-window logits over a paged cache filled from the library model's own
  prefill equal the library model's full no-cache forward over prefix+window;
* gamma = 0 steps chained with the KV append reproduce autoregressive sampling
  from the library model (Sec. 4: gamma = 0 is plain decoding; Sec. 6.5: each
  step is finalised before the next);
* block-table permutations leave outputs unchanged (PagedAttention, Sec. 2.1);
* special cases: RoPE at position 0, norm preservation, RMSNorm of a constant,
  a single key, dense causal attention against torch's SDPA.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2512_22420_amd import workload as W



@pytest.fixture(autouse=True)
def _float64_default():
    """The HF reference model is built in fp64; the default dtype is restored
    afterwards so that no other module sees it (device inputs are fp32)."""
    old = torch.get_default_dtype()
    torch.set_default_dtype(torch.float64)
    yield
    torch.set_default_dtype(old)

# tiny shapes: the tiny fp32 case, and a 2-layer GQA variant (4 query heads on 2 KV heads)
SHAPES = [
    W.TINY_F32,
    dataclasses.replace(W.TINY_F32, name="tiny-gqa-2l", n_layers=2, n_kv_heads=2, d_model=128,
                        head_dim=32, ffn_dim=200, vocab=300, rope_theta=5e5),
]


def _hf_model(shape, weights):
    from transformers import LlamaConfig, LlamaForCausalLM
    s = shape
    cfg = LlamaConfig(vocab_size=s.vocab, hidden_size=s.d_model, intermediate_size=s.ffn_dim,
                      num_hidden_layers=s.n_layers, num_attention_heads=s.n_heads,
                      num_key_value_heads=s.n_kv_heads, head_dim=s.head_dim, rms_norm_eps=s.rms_eps,
                      rope_theta=s.rope_theta, max_position_embeddings=8192, tie_word_embeddings=False,
                      attention_bias=False, mlp_bias=False, attn_implementation="eager")
    m = LlamaForCausalLM(cfg).double().eval()

    def t(a):
        a = W.bf16_bits_to_f32(a) if s.dtype == "bf16" else a
        return torch.from_numpy(np.asarray(a, dtype=np.float64).copy())

    H, Hkv, D, F = s.n_heads, s.n_kv_heads, s.head_dim, s.ffn_dim
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(t(weights["embed"]))
        m.lm_head.weight.copy_(t(weights["lm_head"]))
        m.model.norm.weight.copy_(t(weights["final_norm"]))
        for l, lw in enumerate(weights["layers"]):
            L = m.model.layers[l]
            qkv = t(lw["w_qkv"])
            L.self_attn.q_proj.weight.copy_(qkv[: H * D])
            L.self_attn.k_proj.weight.copy_(qkv[H * D: (H + Hkv) * D])
            L.self_attn.v_proj.weight.copy_(qkv[(H + Hkv) * D:])
            L.self_attn.o_proj.weight.copy_(t(lw["w_o"]))
            gu = t(lw["w_gate_up"])
            L.mlp.gate_proj.weight.copy_(gu[:F])
            L.mlp.up_proj.weight.copy_(gu[F:])
            L.mlp.down_proj.weight.copy_(t(lw["w_down"]))
            L.input_layernorm.weight.copy_(t(lw["attn_norm"]))
            L.post_attention_layernorm.weight.copy_(t(lw["ffn_norm"]))
    return m


def _hf_logits(m, ids):
    with torch.no_grad():
        return m(torch.tensor([list(ids)])).logits[0].numpy()


def _hf_prefill(m, ids):
    """Post-RoPE keys and values the library model caches for a prompt: per layer [Hkv, T, D]."""
    with torch.no_grad():
        out = m(torch.tensor([list(ids)]), use_cache=True)
    pkv = out.past_key_values
    return [(pkv.layers[l].keys[0].numpy(), pkv.layers[l].values[0].numpy()) for l in range(len(pkv.layers))]


def _write_prefix(ctxd, shape, b, kv):
    """Store a sequence's prefix keys/values into fp64 copies of the pages."""
    bs = shape.block_size
    for l, (K, V) in enumerate(kv):
        for t in range(K.shape[1]):
            blk = ctxd["block_table"][b][t // bs]
            ctxd["k_pages"][l][blk, :, t % bs, :] = K[:, t, :]
            ctxd["v_pages"][l][blk, :, :, t % bs] = V[:, t, :]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: s.name)
def test_window_logits_match_library_model(shape):
    rng = np.random.default_rng(5)
    weights = W.make_weights(shape, seed=3, std=0.05)
    m = _hf_model(shape, weights)
    ctx = np.array([21, 37, 16], dtype=np.int32)  # ragged, one exactly a block
    k = 4
    cd = W.make_context(shape, ctx, k, seed=3)
    cd["k_pages"] = [np.asarray(a, dtype=np.float64).copy() for a in cd["k_pages"]]
    cd["v_pages"] = [np.asarray(a, dtype=np.float64).copy() for a in cd["v_pages"]]
    seqs = [rng.integers(0, shape.vocab, size=c + k + 1) for c in ctx]
    for b, ids in enumerate(seqs):
        _write_prefix(cd, shape, b, _hf_prefill(m, ids[: ctx[b]]))
    toks = np.stack([ids[c: c + k + 1] for ids, c in zip(seqs, ctx)])
    logits, win_k, win_v = oracle.forward_window(weights, shape, cd["k_pages"], cd["v_pages"],
                                                 cd["block_table"], ctx, toks)
    for b, ids in enumerate(seqs):
        ref = _hf_logits(m, ids)[ctx[b]:]
        err = np.abs(logits[b] - ref).max() / np.abs(ref).max()
        # the library computes RoPE angles and RMSNorm in fp32, the rest in fp64
        assert err < 2e-6, err
        # the window keys/values are what the library caches for those positions
        kv = _hf_prefill(m, ids)
        for l in range(shape.n_layers):
            for mine, lib in ((win_k[l][b], kv[l][0]), (win_v[l][b], kv[l][1])):
                lib = lib[:, ctx[b]:].transpose(1, 0, 2)
                assert np.abs(mine - lib).max() / np.abs(lib).max() < 2e-6


def test_planted_mistakes_are_caught_by_library_comparison():
    """Mutations of the oracle's forward (transposed W_o, wrong GQA map, RoPE sign)
    must move the logits far outside the tolerance used above."""
    shape = SHAPES[1]
    weights = W.make_weights(shape, seed=3, std=0.05)
    m = _hf_model(shape, weights)
    ids = np.random.default_rng(1).integers(0, shape.vocab, size=24)
    ref = _hf_logits(m, ids)[19:]
    cd = W.make_context(shape, [19], 4, seed=3)
    cd["k_pages"] = [np.asarray(a, dtype=np.float64).copy() for a in cd["k_pages"]]
    cd["v_pages"] = [np.asarray(a, dtype=np.float64).copy() for a in cd["v_pages"]]
    _write_prefix(cd, shape, 0, _hf_prefill(m, ids[:19]))
    vs = __import__("sys").modules["oracle.verify_step"]

    def run():
        lg, _, _ = vs.forward_window(weights, shape, cd["k_pages"], cd["v_pages"],
                                     cd["block_table"], np.array([19]), ids[None, 19:])
        return np.abs(lg[0] - ref).max() / np.abs(ref).max()

    assert run() < 2e-6
    orig_rope, orig_attn = vs.rope, vs.attention
    try:
        vs.rope = lambda x, pos, th: orig_rope(x, -np.asarray(pos), th)
        assert run() > 1e-3
        vs.rope = orig_rope

        def attn_bad_gqa(q, kc, vc, kw, vw):
            G = q.shape[1] // kc.shape[1]
            perm = [(h % kc.shape[1]) * G + h // kc.shape[1] for h in range(q.shape[1])]
            return orig_attn(q[:, perm], kc, vc, kw, vw)[:, np.argsort(perm)]
        vs.attention = attn_bad_gqa
        assert run() > 1e-3
    finally:
        vs.rope, vs.attention = orig_rope, orig_attn
    w2 = {**weights, "layers": [dict(weights["layers"][0], w_o=np.ascontiguousarray(weights["layers"][0]["w_o"].T)),
                                weights["layers"][1]]}
    lg, _, _ = vs.forward_window(w2, shape, cd["k_pages"], cd["v_pages"], cd["block_table"],
                                 np.array([19]), ids[None, 19:])
    assert np.abs(lg[0] - ref).max() / np.abs(ref).max() > 1e-3


def test_gamma0_chain_reproduces_autoregressive_sampling():
    """20 gamma=0 steps with KV append == sampling the library model token by token."""
    shape = SHAPES[1]
    weights = W.make_weights(shape, seed=4, std=0.05)
    m = _hf_model(shape, weights)
    steps = 20
    cd = W.make_context(shape, [0], steps, seed=4)
    kp = [np.asarray(a, dtype=np.float64).copy() for a in cd["k_pages"]]
    vp = [np.asarray(a, dtype=np.float64).copy() for a in cd["v_pages"]]
    ctx = np.array([0], dtype=np.int32)
    rng = np.random.default_rng(9)
    seq = [int(rng.integers(shape.vocab))]
    for step in range(steps):
        u = rng.random(1).astype(np.float32)
        r = oracle.verify_step(weights, shape, kp, vp, cd["block_table"], ctx, np.array([seq[-1]]),
                               np.zeros((1, 0), np.int32), np.zeros((1, 0, shape.vocab), np.float32),
                               u[None, :])
        assert r["accepted_len"][0] == 0
        y = int(r["next_tokens"][0, 0])
        # library model: full forward, softmax, inverse CDF by searchsorted
        lg = _hf_logits(m, seq)[-1]
        p = np.exp(lg - lg.max())
        c = np.cumsum(p)
        assert y == int(np.searchsorted(c, float(u[0]) * c[-1], side="right")), step
        kp, vp, ctx = oracle.kv_append(kp, vp, cd["block_table"], ctx, r["accepted_len"], r["win_k"], r["win_v"],
                                       shape.block_size, "f32")
        assert ctx[0] == step + 1
        seq.append(y)


def test_block_table_permutation_invariance():
    """Relabelling physical blocks (and moving their contents) changes nothing."""
    x = W.tiny_inputs(seed=2, k=3)
    s = x["shape"]
    r1 = oracle.verify_step(x["weights"], s, x["k_pages"], x["v_pages"], x["block_table"], x["context_lens"],
                            x["last_tokens"], x["draft_tokens"], x["draft_probs"], x["uniforms"])
    perm = np.random.default_rng(0).permutation(x["num_blocks"])  # new id of old block
    inv = np.argsort(perm)
    kp = [a[inv] for a in x["k_pages"]]
    vp = [a[inv] for a in x["v_pages"]]
    bt = np.where(x["block_table"] >= 0, perm[np.maximum(x["block_table"], 0)], -1).astype(np.int32)
    r2 = oracle.verify_step(x["weights"], s, kp, vp, bt, x["context_lens"], x["last_tokens"], x["draft_tokens"],
                            x["draft_probs"], x["uniforms"])
    assert np.array_equal(r1["logits"], r2["logits"])
    assert np.array_equal(r1["next_tokens"], r2["next_tokens"])


def test_window_row_depends_only_on_its_prefix():
    """Causality in the window: row i's logits do not depend on drafts after i."""
    x = W.tiny_inputs(seed=3, k=5)
    s = x["shape"]
    toks = oracle.window_tokens(x["last_tokens"], x["draft_tokens"])
    full, _, _ = oracle.forward_window(x["weights"], s, x["k_pages"], x["v_pages"], x["block_table"], x["context_lens"], toks)
    for T in (1, 3):
        part, _, _ = oracle.forward_window(x["weights"], s, x["k_pages"], x["v_pages"], x["block_table"], x["context_lens"],
                                           toks[:, :T])
        np.testing.assert_allclose(part, full[:, :T], rtol=0, atol=1e-12)


def test_kv_append_writes_only_accepted_rows():
    x = W.tiny_inputs(seed=4, k=3)
    s = x["shape"]
    r = oracle.verify_step(x["weights"], s, x["k_pages"], x["v_pages"], x["block_table"], x["context_lens"],
                           x["last_tokens"], x["draft_tokens"], x["draft_probs"], x["uniforms"])
    acc = np.array([3, 1], dtype=np.int32)  # force one full accept and one early stop
    kp, vp, ctx = oracle.kv_append(x["k_pages"], x["v_pages"], x["block_table"], x["context_lens"], acc,
                                   r["win_k"], r["win_v"], s.block_size, s.dtype)
    assert list(ctx) == [x["context_lens"][0] + 4, x["context_lens"][1] + 2]
    touched = set()
    for b in range(2):
        for j in range(acc[b] + 1):
            pos = x["context_lens"][b] + j
            blk, slot = x["block_table"][b][pos // 16], pos % 16
            touched.add((blk, slot))
            np.testing.assert_array_equal(kp[0][blk, :, slot, :], r["win_k"][0][b, j])
            np.testing.assert_array_equal(vp[0][blk, :, :, slot], r["win_v"][0][b, j])
    for blk in range(x["num_blocks"]):
        for slot in range(16):
            if (blk, slot) not in touched:
                assert np.array_equal(kp[0][blk, :, slot, :], x["k_pages"][0][blk, :, slot, :])
                assert np.array_equal(vp[0][blk, :, :, slot], x["v_pages"][0][blk, :, :, slot])


# --------------------------------------------------------------------------
# building blocks
# --------------------------------------------------------------------------
def test_rope_special_cases():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 3, 64))
    np.testing.assert_array_equal(oracle.rope(x, np.zeros(5), 1e4), x)
    y = oracle.rope(x, np.arange(5) * 37 + 11, 1e4)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)
    # dim pair 0 turns by exactly pos radians
    a, b = x[1, 0, 0], x[1, 0, 32]
    np.testing.assert_allclose(oracle.rope(x, np.full(5, 2.0), 1e4)[1, 0, [0, 32]],
                               [a * np.cos(2) - b * np.sin(2), b * np.cos(2) + a * np.sin(2)], rtol=1e-13)
    # scores depend only on the position difference
    q, k = rng.standard_normal((1, 1, 64)), rng.standard_normal((1, 1, 64))
    s1 = (oracle.rope(q, np.array([40]), 1e4) * oracle.rope(k, np.array([33]), 1e4)).sum()
    s2 = (oracle.rope(q, np.array([1007]), 1e4) * oracle.rope(k, np.array([1000]), 1e4)).sum()
    assert abs(s1 - s2) < 1e-10


def test_rmsnorm_of_constant_is_gain():
    g = np.linspace(0.5, 2.0, 8)
    np.testing.assert_allclose(oracle.rms_norm(np.full(8, 3.0), g, 0.0), g, rtol=1e-15)
    np.testing.assert_allclose(oracle.rms_norm(np.full(8, -2.0), g, 0.0), -g, rtol=1e-15)


def test_attention_single_key_returns_value():
    rng = np.random.default_rng(1)
    q = rng.standard_normal((1, 4, 16))
    kw, vw = rng.standard_normal((1, 2, 16)), rng.standard_normal((1, 2, 16))
    out = oracle.attention(q, np.zeros((0, 2, 16)), np.zeros((0, 2, 16)), kw, vw)
    np.testing.assert_allclose(out, vw[:, [0, 0, 1, 1]], rtol=1e-15)


def test_window_attention_with_empty_cache_is_causal_sdpa():
    rng = np.random.default_rng(2)
    T, H, Hkv, D = 6, 8, 2, 32
    q, kw, vw = rng.standard_normal((T, H, D)), rng.standard_normal((T, Hkv, D)), rng.standard_normal((T, Hkv, D))
    out = oracle.attention(q, np.zeros((0, Hkv, D)), np.zeros((0, Hkv, D)), kw, vw)
    Q = torch.from_numpy(q).permute(1, 0, 2)
    K = torch.from_numpy(kw).permute(1, 0, 2).repeat_interleave(H // Hkv, dim=0)
    V = torch.from_numpy(vw).permute(1, 0, 2).repeat_interleave(H // Hkv, dim=0)
    ref = torch.nn.functional.scaled_dot_product_attention(Q, K, V, is_causal=True).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-13)


def test_widen_bf16_bit_patterns():
    bits = np.array([0x3F80, 0xC000, 0x3E80, 0x0000, 0x8000, 0x3F81, 0x7F7F], dtype=np.uint16)
    vals = oracle.widen(bits, "bf16")
    assert list(vals[:5]) == [1.0, -2.0, 0.25, 0.0, -0.0]
    assert vals[5] == 1.0 + 2.0 ** -7
    assert vals[6] == (2.0 - 2.0 ** -7) * 2.0 ** 127


# --------------------------------------------------------------------------
# the composed step at gamma > 0 (which target row scores which draft)
# --------------------------------------------------------------------------
def _self_draft_case(shape, weights, m, ctx, k, seed):
    """Prefixes cached from the library model's prefill, and k drafts sampled
    from the library model itself token by token (q_i = its own p_i), so every
    draft must be accepted (Sec. 2.2: a draft the target agrees with is kept)
    and the extra token is the target's own next sample (Sec. 3.1: n accepted
    plus one).  Returns the inputs and, per sequence, the library model's
    sample at window position k drawn with the step's last uniform."""
    rng = np.random.default_rng(seed)
    cd = W.make_context(shape, ctx, k, seed=seed)
    cd["k_pages"] = [np.asarray(a, dtype=np.float64).copy() for a in cd["k_pages"]]
    cd["v_pages"] = [np.asarray(a, dtype=np.float64).copy() for a in cd["v_pages"]]
    B = len(ctx)
    last = np.zeros(B, np.int32)
    drafts = np.zeros((B, k), np.int32)
    dprobs = np.zeros((B, k, shape.vocab), np.float32)
    unif = np.zeros((B, k + 1), np.float32)
    bonus = []
    for b in range(B):
        ids = list(rng.integers(0, shape.vocab, size=int(ctx[b]) + 1))
        if ctx[b] > 0:
            _write_prefix(cd, shape, b, _hf_prefill(m, ids[: ctx[b]]))
        last[b] = ids[-1]
        unif[b, :k] = rng.random(k) * 0.9  # accept tests, away from ratio 1
        unif[b, k] = rng.random()
        for i in range(k + 1):
            lg = _hf_logits(m, ids)[-1]
            p = np.exp(lg - lg.max())
            c = np.cumsum(p)
            v = rng.random() if i < k else float(unif[b, k])
            y = int(np.searchsorted(c, v * c[-1], side="right"))
            if i < k:
                dprobs[b, i] = (p / c[-1]).astype(np.float32)
                drafts[b, i] = y
                ids.append(y)
            else:
                bonus.append(y)
    return cd, last, drafts, dprobs, unif, bonus


@pytest.mark.parametrize("k", [1, 4])
def test_self_drafts_are_all_accepted_and_bonus_is_library_sample(k):
    """With q_i equal to the target's own p_i every draft passes (u < p/q = 1),
    and the bonus token is the library model's autoregressive sample at window
    position k with the last uniform.  This pins that window row i scores draft
    i+1 and that the bonus comes from row k."""
    shape = SHAPES[1]
    weights = W.make_weights(shape, seed=6, std=0.05)
    m = _hf_model(shape, weights)
    ctx = np.array([13, 30, 0], dtype=np.int32)
    cd, last, drafts, dprobs, unif, bonus = _self_draft_case(shape, weights, m, ctx, k, seed=10 + k)
    r = oracle.verify_step(weights, shape, cd["k_pages"], cd["v_pages"], cd["block_table"], ctx, last, drafts,
                           dprobs, unif)
    assert list(r["accepted_len"]) == [k] * len(ctx)
    for b in range(len(ctx)):
        assert list(r["next_tokens"][b]) == list(drafts[b]) + [bonus[b]]


def test_misaligned_rows_fail_the_self_draft_pin():
    """Planted mistake: scoring draft i with target row i+1 (an off-by-one
    between rows and drafts) must break the self-draft property above."""
    shape = SHAPES[1]
    weights = W.make_weights(shape, seed=6, std=0.05)
    m = _hf_model(shape, weights)
    ctx = np.array([13, 30, 0], dtype=np.int32)
    k = 4
    cd, last, drafts, dprobs, unif, bonus = _self_draft_case(shape, weights, m, ctx, k, seed=14)
    vs = __import__("sys").modules["oracle.verify_step"]
    orig = vs.accept

    def shifted(p, q, d, u):
        return orig(np.concatenate([p[1:], p[-1:]], axis=0), q, d, u)
    try:
        vs.accept = shifted
        r = oracle.verify_step(weights, shape, cd["k_pages"], cd["v_pages"], cd["block_table"], ctx, last, drafts,
                               dprobs, unif)
    finally:
        vs.accept = orig
    ok = all(r["accepted_len"][b] == k and list(r["next_tokens"][b]) == list(drafts[b]) + [bonus[b]]
             for b in range(len(ctx)))
    assert not ok


def test_window_rows_equal_a_chain_of_gamma0_steps():
    """A gamma = k window equals k+1 chained gamma = 0 steps fed the same tokens
    (each followed by the KV append of its one row): row i of the window is the
    gamma = 0 step at position ctx + i, and when every draft is accepted the
    bonus equals the gamma = 0 step's draw with the same uniform (Sec. 4:
    gamma = 0 is plain decoding)."""
    x = W.tiny_inputs(seed=7, k=4)
    s = x["shape"]
    k = 4
    # drafts the step must accept: q_i = the window's own p_i, accept uniforms 0
    toks = oracle.window_tokens(x["last_tokens"], x["draft_tokens"])
    logits, _, _ = oracle.forward_window(x["weights"], s, x["k_pages"], x["v_pages"], x["block_table"],
                                         x["context_lens"], toks)
    q = oracle.softmax(logits[:, :k]).astype(np.float32)
    u = x["uniforms"].copy()
    u[:, :k] = 0.0
    r = oracle.verify_step(x["weights"], s, x["k_pages"], x["v_pages"], x["block_table"], x["context_lens"],
                           x["last_tokens"], x["draft_tokens"], q, u)
    assert list(r["accepted_len"]) == [k, k]
    kp, vp, ctx = x["k_pages"], x["v_pages"], x["context_lens"].copy()
    for i in range(k + 1):
        ui = u[:, k:k + 1] if i == k else np.full((2, 1), 0.5, np.float32)
        ri = oracle.verify_step(x["weights"], s, kp, vp, x["block_table"], ctx, toks[:, i].astype(np.int32),
                                np.zeros((2, 0), np.int32), np.zeros((2, 0, s.vocab), np.float32), ui)
        np.testing.assert_allclose(ri["logits"][:, 0], r["logits"][:, i], rtol=0, atol=1e-10)
        if i == k:
            assert list(ri["next_tokens"][:, 0]) == list(r["next_tokens"][:, k])
        kp, vp, ctx = oracle.kv_append(kp, vp, x["block_table"], ctx, ri["accepted_len"], ri["win_k"], ri["win_v"],
                                       s.block_size, s.dtype)
