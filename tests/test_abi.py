"""The C-ABI library loads, exports every entry point the header declares, and
rejects bad arguments on the host (no device work is needed for these)."""
import ctypes
import os

import pytest

from paper_2512_22420_amd import binding as nb
from paper_2512_22420_amd import workload as W
from paper_2512_22420_amd.device import model_desc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "nightjar.h")

pytestmark = pytest.mark.skipif(not os.path.exists(nb.LIB_PATH), reason="libnightjar.so not built")


def test_exports_every_declared_function():
    import glob
    names = nb.header_functions(HEADER)
    assert "nightjar_verify_step" in names and "nightjar_kv_append" in names
    headers = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))
    assert len(headers) >= 2
    L = nb.lib()
    for h in headers:
        for n in nb.header_functions(h):
            assert hasattr(L, n), (h, n)
            assert n in nb._SIGS, (h, n)  # the binding declares it too


def test_struct_sizes_match_header_layout():
    assert ctypes.sizeof(nb.ModelDesc) == 11 * 4
    assert ctypes.sizeof(nb.LayerWeights) == 6 * 8
    assert ctypes.sizeof(nb.Weights) == 4 * 8
    assert ctypes.sizeof(nb.KvCache) == 3 * 8


def test_workspace_bytes_monotone_and_validating():
    d = model_desc(W.LLAMA8B_LAYER)
    small = nb.workspace_bytes(d, 1, 0)
    big = nb.workspace_bytes(d, 8, 5)
    assert 0 < small < big
    assert big % 256 == 0
    with pytest.raises(nb.NightjarError):
        nb.workspace_bytes(d, 1, 16)  # the window must fit one 16-token block
    bad = model_desc(W.LLAMA8B_LAYER)
    bad.block_size = 32
    assert nb.lib().nightjar_workspace_bytes(ctypes.byref(bad), 1, 0) == 0
    assert "block_size" in nb.last_error()
    bad = model_desc(W.LLAMA8B_LAYER)
    bad.n_kv_heads = 5
    assert nb.lib().nightjar_workspace_bytes(ctypes.byref(bad), 1, 0) == 0


def test_verify_step_rejects_bad_arguments_on_host():
    d = model_desc(W.TINY_F32)
    w = nb.Weights()
    kv = nb.KvCache()
    rc = nb.lib().nightjar_verify_step(ctypes.byref(d), ctypes.byref(w), ctypes.byref(kv), 0, 1, 0, 0, 0, 0, 0,
                                       2, 3, 0, 0, 0, 0, 0, 0)
    assert rc == nb.NJ_EINVAL and "weights" in nb.last_error()
    rc = nb.lib().nightjar_verify_step(None, ctypes.byref(w), ctypes.byref(kv), 0, 1, 0, 0, 0, 0, 0,
                                       2, 3, 0, 0, 0, 0, 0, 0)
    assert rc == nb.NJ_EINVAL and "desc" in nb.last_error()
    rc = nb.lib().nightjar_verify_step(ctypes.byref(d), ctypes.byref(w), ctypes.byref(kv), 0, 1, 0, 0, 0, 0, 0,
                                       2, 16, 0, 0, 0, 0, 0, 0)
    assert rc == nb.NJ_EINVAL and "k must be" in nb.last_error()


def test_gemm_rejects_bad_shapes_on_host():
    L = nb.lib()
    big = 1 << 30
    assert L.nightjar_gemm(nb.NJ_BF16, 16, 16, 16, 4, 32, 40, nb.NJ_GEMM_STORE, 256, big, 0) == nb.NJ_EINVAL  # K % 32
    assert L.nightjar_gemm(nb.NJ_BF16, 16, 16, 16, 4, 24, 64, nb.NJ_GEMM_STORE, 256, big, 0) == nb.NJ_EINVAL  # N % 16
    assert L.nightjar_gemm(nb.NJ_BF16, 16, 16, 16, 4, 30, 64, nb.NJ_GEMM_SWIGLU, 256, big, 0) == nb.NJ_EINVAL
    assert L.nightjar_gemm(nb.NJ_BF16, 0, 16, 16, 4, 32, 64, nb.NJ_GEMM_STORE, 256, big, 0) == nb.NJ_EINVAL
    assert L.nightjar_gemm(nb.NJ_BF16, 16, 16, 16, 0, 32, 64, nb.NJ_GEMM_STORE, 256, big, 0) == nb.NJ_EINVAL
    assert L.nightjar_gemm(7, 16, 16, 16, 1, 32, 64, nb.NJ_GEMM_STORE, 256, big, 0) == nb.NJ_EINVAL
    # a workspace smaller than the split-K scratch is refused before any launch
    need = nb.gemm_workspace_bytes(nb.NJ_BF16, 48, 4096, 14336, nb.NJ_GEMM_RESIDUAL)
    assert need > 256
    assert L.nightjar_gemm(nb.NJ_BF16, 16, 16, 16, 48, 4096, 14336, nb.NJ_GEMM_RESIDUAL, 256, need - 256, 0) == nb.NJ_EINVAL
    assert "workspace" in nb.last_error()


def test_kv_append_requires_a_preceding_verify_step():
    d = model_desc(W.TINY_F32)
    ptrs = (ctypes.c_void_p * 1)(16)
    kv = nb.KvCache(ctypes.cast(ptrs, ctypes.POINTER(ctypes.c_void_p)), ctypes.cast(ptrs, ctypes.POINTER(ctypes.c_void_p)), 4)
    rc = nb.lib().nightjar_kv_append(ctypes.byref(d), ctypes.byref(kv), 16, 4, 16, 16, 2, 3, 256, 1 << 20, 0)
    assert rc == nb.NJ_EINVAL and "no verify step" in nb.last_error()


def test_gemm_with_plan_rejects_impossible_plans_on_host():
    L = nb.lib()
    ws = 1 << 30
    st = nb.NJ_GEMM_STORE
    # tiled kernels need K % 64 == 0
    assert L.nightjar_gemm_with_plan(nb.NJ_BF16, 16, 16, 16, 200, 256, 96, st, nb.NJ_GEMM_TILE_128x128, 0, 256, ws, 0) \
        == nb.NJ_EINVAL
    assert "K % 64" in nb.last_error()
    # a run that cuts tiles between workgroups may have at most 1024 of them
    assert nb.lib().nightjar_gemm_plan_workspace_bytes(nb.NJ_BF16, 768, 128256, 4096, st, nb.NJ_GEMM_TILE_128x128, 2) == 0
    assert "at most 1024 workgroups" in nb.last_error()
    assert nb.lib().nightjar_gemm_plan_workspace_bytes(nb.NJ_BF16, 768, 4096, 4096, st, nb.NJ_GEMM_TILE_128x128,
                                                       -1100) == 0
    # stream-K grids: tiled kernels only, and not the 256x256 tile
    assert nb.lib().nightjar_gemm_plan_workspace_bytes(nb.NJ_BF16, 768, 4096, 4096, st, nb.NJ_GEMM_TILE_256x256,
                                                       -100) == 0
    assert "256x256" in nb.last_error()
    assert nb.lib().nightjar_gemm_plan_workspace_bytes(nb.NJ_BF16, 768, 4096, 4096, st, nb.NJ_GEMM_TILE_128x256,
                                                       -100) > 0
    # a grid of 3 x 12 workgroups on 12 tiles is a plain 3-way split, which the 256x256 tile runs
    assert nb.lib().nightjar_gemm_plan_workspace_bytes(nb.NJ_BF16, 768, 1024, 4096, st, nb.NJ_GEMM_TILE_256x256,
                                                       -36) > 0
    # auto plan takes no split; fp32 has one kernel; bad kernel id
    assert L.nightjar_gemm_plan_workspace_bytes(nb.NJ_BF16, 64, 256, 256, st, nb.NJ_GEMM_AUTO, 2) == 0
    assert L.nightjar_gemm_plan_workspace_bytes(nb.NJ_F32, 64, 256, 256, st, nb.NJ_GEMM_STREAM, 0) == 0
    assert L.nightjar_gemm_plan_workspace_bytes(nb.NJ_BF16, 64, 256, 256, st, nb.NJ_GEMM_TILE_96x128 + 1, 0) == 0
    assert L.nightjar_gemm_plan_workspace_bytes(nb.NJ_BF16, 64, 256, 256, st, nb.NJ_GEMM_STREAM, -1) == 0
    # the workspace grows with the split (fp32 partials per chunk)
    a = nb.gemm_plan_workspace_bytes(nb.NJ_BF16, 384, 4096, 4096, st, nb.NJ_GEMM_TILE_256x256, 1)
    b = nb.gemm_plan_workspace_bytes(nb.NJ_BF16, 384, 4096, 4096, st, nb.NJ_GEMM_TILE_256x256, 4)
    assert b >= a + 4 * 384 * 4096 * 4
    # a workspace one byte short is refused before any launch
    assert L.nightjar_gemm_with_plan(nb.NJ_BF16, 16, 16, 16, 384, 4096, 4096, st, nb.NJ_GEMM_TILE_256x256, 4, 256,
                                     b - 1, 0) == nb.NJ_EINVAL


def test_stage_entries_reject_bad_arguments_on_host():
    desc = model_desc(W.QWEN7B)  # G = 7: k = 9 gives 70 query rows per KV head
    n = nb.attn_workspace_bytes(desc, 1, 9)
    rc = nb.lib().nightjar_attn_verify(ctypes.byref(desc), 16, 16, 16, 4, 16, 16, 16, 4, 16, 1, 9, 16, 256, n, 0)
    assert rc == nb.NJ_EINVAL and "64 query rows" in nb.last_error()
    rc = nb.lib().nightjar_attn_verify(ctypes.byref(desc), 16, 16, 16, 4, 16, 16, 16, 4, 16, 1, 2, 16, 256, 255, 0)
    assert rc == nb.NJ_EINVAL and "workspace" in nb.last_error()
    rc = nb.lib().nightjar_attn_verify(ctypes.byref(desc), 0, 16, 16, 4, 16, 16, 16, 4, 16, 1, 2, 16, 256, n, 0)
    assert rc == nb.NJ_EINVAL and "NULL" in nb.last_error()
    d8 = model_desc(W.LLAMA8B_LAYER)
    m = nb.rmsnorm_rope_workspace_bytes(d8, 2, 3)
    assert m > nb.rmsnorm_rope_workspace_bytes(d8, 1, 3) > 0
    rc = nb.lib().nightjar_rmsnorm_rope(ctypes.byref(d8), 16, 16, 16, 16, 2, 3, 16, 16, 8, 256, m, 0)
    assert rc == nb.NJ_EINVAL and "aligned" in nb.last_error()
    rc = nb.lib().nightjar_rmsnorm_rope(ctypes.byref(d8), 16, 16, 16, 16, 2, 16, 16, 16, 16, 256, m, 0)
    assert rc == nb.NJ_EINVAL


@pytest.mark.parametrize("shape,max_B,max_k", [(W.LLAMA8B_LAYER, 128, 5), (W.QWEN7B, 256, 7), (W.LLAMA1B_DRAFT, 64, 4)],
                         ids=["8b-layer", "qwen7b", "1b-draft"])
def test_max_workspace_serves_every_smaller_window(shape, max_B, max_k):
    """nightjar_workspace_bytes(max_B, max_k) is enough for every (B, k) below
    it, whatever GEMM plan (split partials included) the smaller window picks."""
    L = nb.lib()
    d = model_desc(shape)
    top = L.nightjar_workspace_bytes(ctypes.byref(d), max_B, max_k)
    assert top > 0
    Bs = sorted(set(list(range(1, 17)) + list(range(16, max_B + 1, 7)) + [max_B]))
    for B in Bs:
        for k in range(max_k + 1):
            need = L.nightjar_workspace_bytes(ctypes.byref(d), B, k)
            assert 0 < need <= top, (B, k, need, top)
