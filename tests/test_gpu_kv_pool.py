"""KV-pool contraction on the GPU (Sec. 6.4, Step 4): nightjar_kv_migrate
copies blocks bit for bit as the reference's Step 4 does, and a verify step on
the contracted pool (tables rewritten by nightjar_contraction_plan) gives
bitwise the outputs of the step on the expanded pool (the attention reads
blocks only through the tables; Sec. 6.5: migration never changes outputs)."""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import kv_pool as ref
from paper_2512_22420_amd import binding as nb
from paper_2512_22420_amd import workload as W
from paper_2512_22420_amd.device import (DeviceCache, DeviceModel, StepIO, Workspace, device_error, kv_append,
                                        model_desc, verify)

pytestmark = pytest.mark.gpu

SMALL_BF16 = dataclasses.replace(W.LLAMA8B_LAYER, name="bf16-small", n_layers=2, d_model=512, n_heads=8,
                                 n_kv_heads=2, ffn_dim=1024, vocab=4112)


def _s():
    return torch.cuda.current_stream().cuda_stream


def _expanded_pool(shape, ctx, k, seed):
    """A pool twice the size the sequences need, their blocks spread over all of
    it; the top quarter of the ids is the region being reclaimed."""
    c = W.make_context(shape, ctx, k, seed=seed, spare=1.0)
    kb = (3 * c["num_blocks"]) // 4
    live = set(int(x) for x in c["block_table"].ravel() if x >= 0)
    free = np.array([i for i in np.random.default_rng(seed).permutation(c["num_blocks"]) if i not in live], np.int32)
    return c, kb, free


@pytest.mark.parametrize("shape", [dataclasses.replace(W.LLAMA8B_LAYER, n_layers=3), W.TINY_F32],
                         ids=["8b-heads-3-layers", "f32"])
def test_kv_migrate_is_the_reference_copy(shape):
    ctx = np.array([700, 33, 0, 1500, 250, 16], np.int32)
    c, kb, free = _expanded_pool(shape, ctx, 5, seed=4)
    p = ref.contraction_plan(c["block_table"], free, kb)
    assert len(p["src"]) > 10
    cache = DeviceCache(c)
    src = torch.tensor(p["src"], dtype=torch.int32, device="cuda")
    dst = torch.tensor(p["dst"], dtype=torch.int32, device="cuda")
    err = torch.full((1,), 99, dtype=torch.int32, device="cuda")
    nb.kv_migrate(model_desc(shape), cache.c, src.data_ptr(), dst.data_ptr(), len(p["src"]), err.data_ptr(), _s())
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    want_k, want_v = ref.migrate(c["k_pages"], c["v_pages"], p["src"], p["dst"])
    view = np.uint16 if shape.dtype == "bf16" else np.float32
    for l in range(shape.n_layers):
        assert np.array_equal(cache.k_pages[l].cpu().numpy().view(view), want_k[l])
        assert np.array_equal(cache.v_pages[l].cpu().numpy().view(view), want_v[l])


def test_kv_migrate_flags_bad_ids_and_skips_them():
    shape = SMALL_BF16
    c = W.make_context(shape, np.array([40, 70], np.int32), 3, seed=5, spare=1.0)
    cache = DeviceCache(c)
    before = [t.clone() for t in cache.k_pages]
    n = c["num_blocks"]
    src = torch.tensor([0, n + 5], dtype=torch.int32, device="cuda")
    dst = torch.tensor([-1, 1], dtype=torch.int32, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    nb.kv_migrate(model_desc(shape), cache.c, src.data_ptr(), dst.data_ptr(), 2, err.data_ptr(), _s())
    torch.cuda.synchronize()
    assert int(err.item()) & nb.NJ_DEV_BAD_BLOCK
    for a, b in zip(before, cache.k_pages):
        assert torch.equal(a, b)


@pytest.mark.parametrize("shape,k", [(SMALL_BF16, 4), (W.TINY_F32, 3)], ids=["bf16", "f32"])
def test_step_after_contraction_is_bitwise_unchanged(shape, k):
    ctx = np.array([300, 5, 129, 47, 0, 260], np.int32)
    c, kb, free = _expanded_pool(shape, ctx, k, seed=6)
    d = W.make_drafts(shape, len(ctx), k, seed=6)
    model = DeviceModel(shape, W.make_weights(shape, seed=6))
    cache = DeviceCache(c)
    io = StepIO(shape, d)
    ws = Workspace(shape, len(ctx), k)
    verify(model, cache, io, ws)
    assert device_error(ws) == 0
    before = (io.logits.clone(), io.next_tokens.clone(), io.accepted_len.clone())
    # contract: plan on the host, migrate on the device, new tables
    src, dst, table, new_free = nb.contraction_plan(c["block_table"], free, kb, c["num_blocks"])
    assert len(src) > 0 and np.all(table[table >= 0] < kb)
    ds = torch.from_numpy(src).cuda()
    dd = torch.from_numpy(dst).cuda()
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    nb.kv_migrate(model_desc(shape), cache.c, ds.data_ptr(), dd.data_ptr(), len(src), err.data_ptr(), _s())
    cache.block_table.copy_(torch.from_numpy(table).cuda())
    # the reclaimed blocks are overwritten (the region goes back to the draft model)
    for l in range(shape.n_layers):
        cache.k_pages[l][kb:].fill_(-1)
        cache.v_pages[l][kb:].fill_(-1)
    verify(model, cache, io, ws)
    assert device_error(ws) == 0 and int(err.item()) == 0
    assert torch.equal(io.logits, before[0])
    assert torch.equal(io.next_tokens, before[1]) and torch.equal(io.accepted_len, before[2])
    # the KV append after contraction writes below the boundary only
    kv_append(model, cache, io, ws)
    assert device_error(ws) == 0
    for l in range(shape.n_layers):
        assert torch.all(cache.k_pages[l][kb:].view(-1) == -1)


def test_offload_reload_round_trip_on_a_side_stream():
    """Sec. 6.2: the draft weights go to pinned host memory and back with
    asynchronous copies on a side stream; the bytes come back unchanged."""
    n = 48 << 20
    g = torch.Generator(device="cuda")
    g.manual_seed(1)
    src = torch.randint(-30000, 30000, (n // 2,), dtype=torch.int16, device="cuda", generator=g)
    host = torch.empty(n // 2, dtype=torch.int16, pin_memory=True)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    nb.offload(src.data_ptr(), host.data_ptr(), n, side.cuda_stream)
    side.synchronize()
    assert torch.equal(host, src.cpu())
    dst = torch.zeros_like(src)
    side.wait_stream(torch.cuda.current_stream())
    nb.reload(host.data_ptr(), dst.data_ptr(), n, side.cuda_stream)
    side.synchronize()
    assert torch.equal(dst, src)
    with pytest.raises(nb.NightjarError):
        nb.offload(0, host.data_ptr(), n, side.cuda_stream)
