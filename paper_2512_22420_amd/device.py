"""Device-memory plumbing for the binding: upload a model, a paged cache and a
step's inputs as torch tensors and build the C structs that point at them.
PyTorch is used for allocation and streams only; all compute is in the HIP
library.
"""
from __future__ import annotations

import ctypes
from typing import Dict, Optional

import numpy as np
import torch

from . import binding as nb


def _to_dev(a, device) -> torch.Tensor:
    if isinstance(a, torch.Tensor):  # already resident (bf16 bits as int16, or fp32/int32)
        return a
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(device)


def _ptr(t: Optional[torch.Tensor]) -> int:
    return 0 if t is None else t.data_ptr()


def pack_weight(w: torch.Tensor, stream: Optional[int] = None) -> torch.Tensor:
    """Packed copy (the layout of nightjar_pack_weight) of a bf16 [N][K]
    weight matrix resident on the device as int16 bits."""
    N, K = w.shape
    s = torch.cuda.current_stream().cuda_stream if stream is None else stream
    out = torch.empty(nb.packed_weight_elems(N, K), dtype=torch.int16, device=w.device)
    nb.pack_weight(w.data_ptr(), out.data_ptr(), N, K, s)
    return out


def model_desc(shape) -> nb.ModelDesc:
    return nb.ModelDesc(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim,
                        shape.ffn_dim, shape.vocab, shape.block_size, shape.rms_eps, shape.rope_theta,
                        nb.NJ_BF16 if shape.dtype == "bf16" else nb.NJ_F32)


class DeviceModel:
    """Weights resident on the device, plus the descriptor structs."""

    def __init__(self, shape, weights: Dict, device="cuda"):
        self.shape = shape
        self.desc = model_desc(shape)
        # bf16 GEMM weights go to the packed layout the GEMM kernels read
        mat = (lambda a: pack_weight(_to_dev(a, device))) if shape.dtype == "bf16" else (lambda a: _to_dev(a, device))
        self.embed = _to_dev(weights["embed"], device)
        self.final_norm = _to_dev(weights["final_norm"], device)
        self.lm_head = mat(weights["lm_head"])
        names = ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down")
        self.layers = [{n: (mat(lw[n]) if n.startswith("w_") else _to_dev(lw[n], device)) for n in names}
                       for lw in weights["layers"]]
        self._c_layers = (nb.LayerWeights * shape.n_layers)(
            *[nb.LayerWeights(*[_ptr(l[n]) for n in names]) for l in self.layers])
        self.c = nb.Weights(_ptr(self.embed), _ptr(self.final_norm), _ptr(self.lm_head),
                            ctypes.cast(self._c_layers, ctypes.POINTER(nb.LayerWeights)))


class DeviceCache:
    """Paged KV cache and block table on the device."""

    def __init__(self, ctx: Dict, device="cuda"):
        self.k_pages = [_to_dev(a, device) for a in ctx["k_pages"]]
        self.v_pages = [_to_dev(a, device) for a in ctx["v_pages"]]
        self.block_table = _to_dev(ctx["block_table"], device)
        self.context_lens = _to_dev(ctx["context_lens"], device)
        self.num_blocks = int(ctx["num_blocks"])
        self.max_blocks = int(ctx["block_table"].shape[1])
        self._kp = (ctypes.c_void_p * len(self.k_pages))(*[_ptr(t) for t in self.k_pages])
        self._vp = (ctypes.c_void_p * len(self.v_pages))(*[_ptr(t) for t in self.v_pages])
        self.c = nb.KvCache(ctypes.cast(self._kp, ctypes.POINTER(ctypes.c_void_p)),
                            ctypes.cast(self._vp, ctypes.POINTER(ctypes.c_void_p)), self.num_blocks)


class Workspace:
    def __init__(self, shape, max_B: int, max_k: int, device="cuda", stream: int = 0):
        self.nbytes = nb.workspace_bytes(model_desc(shape), max_B, max_k)
        self.buf = torch.empty(self.nbytes, dtype=torch.uint8, device=device)
        nb.workspace_init(self.ptr, self.nbytes, stream)

    @property
    def ptr(self) -> int:
        return self.buf.data_ptr()


class StepIO:
    """One step's inputs and outputs on the device."""

    def __init__(self, shape, drafts: Dict, device="cuda", keep_logits: bool = True):
        B, k = drafts["draft_tokens"].shape
        self.B, self.k = B, k
        self.last_tokens = _to_dev(drafts["last_tokens"], device)
        self.draft_tokens = _to_dev(drafts["draft_tokens"], device) if k else None
        self.draft_probs = _to_dev(drafts["draft_probs"], device) if k else None
        self.uniforms = _to_dev(drafts["uniforms"], device)
        self.accepted_len = torch.full((B,), -7, dtype=torch.int32, device=device)
        self.next_tokens = torch.full((B, k + 1), -7, dtype=torch.int32, device=device)
        self.logits = torch.empty((B, k + 1, shape.vocab), dtype=torch.float32, device=device) if keep_logits else None


def _expect(t: Optional[torch.Tensor], dtype, numel: int, name: str) -> None:
    """The C ABI takes raw pointers: a tensor of another dtype or size would be
    reinterpreted, so it is refused here."""
    if t is None:
        return
    if t.dtype != dtype or t.numel() != numel or not t.is_contiguous():
        raise TypeError(f"{name}: need a contiguous {dtype} tensor of {numel} elements, "
                        f"got {t.dtype} {tuple(t.shape)}")


def verify(model: DeviceModel, cache: DeviceCache, io: StepIO, ws: Workspace, stream: Optional[int] = None):
    B, k, V = io.B, io.k, model.shape.vocab
    _expect(io.last_tokens, torch.int32, B, "last_tokens")
    _expect(io.draft_tokens, torch.int32, B * k, "draft_tokens")
    _expect(io.draft_probs, torch.float32, B * k * V, "draft_probs")
    _expect(io.uniforms, torch.float32, B * (k + 1), "uniforms")
    _expect(io.accepted_len, torch.int32, B, "accepted_len")
    _expect(io.next_tokens, torch.int32, B * (k + 1), "next_tokens")
    _expect(io.logits, torch.float32, B * (k + 1) * V, "logits")
    _expect(cache.context_lens, torch.int32, B, "context_lens")
    s = torch.cuda.current_stream().cuda_stream if stream is None else stream
    nb.verify_step(model.desc, model.c, cache.c, _ptr(cache.block_table), cache.max_blocks, _ptr(cache.context_lens),
                   _ptr(io.last_tokens), _ptr(io.draft_tokens), _ptr(io.draft_probs), _ptr(io.uniforms), io.B, io.k,
                   _ptr(io.accepted_len), _ptr(io.next_tokens), _ptr(io.logits), ws.ptr, ws.nbytes, s)


def kv_append(model: DeviceModel, cache: DeviceCache, io: StepIO, ws: Workspace, stream: Optional[int] = None):
    s = torch.cuda.current_stream().cuda_stream if stream is None else stream
    nb.kv_append(model.desc, cache.c, _ptr(cache.block_table), cache.max_blocks, _ptr(cache.context_lens),
                 _ptr(io.accepted_len), io.B, io.k, ws.ptr, ws.nbytes, s)


def device_error(ws: Workspace, stream: Optional[int] = None) -> int:
    s = torch.cuda.current_stream().cuda_stream if stream is None else stream
    return nb.device_error(ws.ptr, ws.nbytes, s)
