"""ctypes binding of libnightjar.so: the C ABI of ``include/nightjar.h`` with the
same names.  Argument marshalling only; every step runs in the HIP library.
Device pointers are passed as Python ints (e.g. ``tensor.data_ptr()``), the
stream as a ``hipStream_t`` int (``torch.cuda.current_stream().cuda_stream``).
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libnightjar.so")

NJ_F32, NJ_BF16 = 0, 1
NJ_OK, NJ_EINVAL, NJ_EDEVICE, NJ_EHIP, NJ_EAGAIN = 0, -1, -2, -3, -4
NJ_DEV_BAD_TOKEN, NJ_DEV_BAD_BLOCK, NJ_DEV_BAD_CONTEXT, NJ_DEV_BAD_ACCEPT, NJ_DEV_SPLIT_WAIT = 1, 2, 4, 8, 16
NJ_GEMM_STORE, NJ_GEMM_RESIDUAL, NJ_GEMM_SWIGLU = 0, 1, 2
NJ_GEMM_KBLOCKED = 16  # flag: x (and a SwiGLU y) k-blocked, [K/32][M][32]
NJ_GEMM_AUTO, NJ_GEMM_STREAM, NJ_GEMM_TILE_256x256, NJ_GEMM_TILE_128x256, NJ_GEMM_TILE_128x128 = 0, 1, 2, 3, 4
NJ_GEMM_TILE_192x256 = 6
NJ_GEMM_TILE_160x256, NJ_GEMM_TILE_96x256, NJ_GEMM_TILE_96x128 = 7, 8, 9
NJ_GEMM_STREAM_DEEP = 5

_vp = ctypes.c_void_p
_i32 = ctypes.c_int32
_sz = ctypes.c_size_t


class ModelDesc(ctypes.Structure):
    _fields_ = [("n_layers", _i32), ("d_model", _i32), ("n_heads", _i32), ("n_kv_heads", _i32),
                ("head_dim", _i32), ("ffn_dim", _i32), ("vocab", _i32), ("block_size", _i32),
                ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float), ("dtype", _i32)]


class LayerWeights(ctypes.Structure):
    _fields_ = [("attn_norm", _vp), ("w_qkv", _vp), ("w_o", _vp), ("ffn_norm", _vp),
                ("w_gate_up", _vp), ("w_down", _vp)]


class Weights(ctypes.Structure):
    _fields_ = [("embed", _vp), ("final_norm", _vp), ("lm_head", _vp), ("layers", ctypes.POINTER(LayerWeights))]


class KvCache(ctypes.Structure):
    _fields_ = [("k_pages", ctypes.POINTER(_vp)), ("v_pages", ctypes.POINTER(_vp)), ("num_blocks", _i32)]


class PlannerConfig(ctypes.Structure):
    _fields_ = [("max_batch", _i32), ("max_gamma", _i32), ("seed", ctypes.c_uint64), ("prev_per_batch", _i32),
                ("unplayed_latency", ctypes.c_double)]


class PlannerBState(ctypes.Structure):
    _fields_ = [("block", _i32), ("block_len", ctypes.c_int64), ("bin", ctypes.c_int64), ("round", ctypes.c_int64),
                ("gamma", _i32), ("steps", ctypes.c_int64), ("bins", ctypes.c_int64),
                ("explore_bins", ctypes.c_int64)]


class ElasticConfig(ctypes.Structure):
    _fields_ = [("n_orig", _i32), ("n_draft", _i32), ("tau_low", _i32), ("t_persist", _i32),
                ("reload_persist", _i32), ("max_migrate", _i32)]


class NightjarError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"nightjar error {code}: {msg}")
        self.code = code


_LIB = None

_SIGS = {
    "nightjar_workspace_bytes": (_sz, [ctypes.POINTER(ModelDesc), _i32, _i32]),
    "nightjar_workspace_init": (ctypes.c_int, [_vp, _sz, _vp]),
    "nightjar_step_folds_norms": (ctypes.c_int, [ctypes.POINTER(ModelDesc), _i32, _i32]),
    "nightjar_verify_step": (ctypes.c_int, [ctypes.POINTER(ModelDesc), ctypes.POINTER(Weights), ctypes.POINTER(KvCache),
                                            _vp, _i32, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp, _vp,
                                            _vp, _sz, _vp]),
    "nightjar_kv_append": (ctypes.c_int, [ctypes.POINTER(ModelDesc), ctypes.POINTER(KvCache), _vp, _i32, _vp, _vp,
                                          _i32, _i32, _vp, _sz, _vp]),
    "nightjar_draft_step": (ctypes.c_int, [ctypes.POINTER(ModelDesc), ctypes.POINTER(Weights), ctypes.POINTER(KvCache),
                                           _vp, _i32, _vp, _vp, _vp, _i32, _vp, _i32, _vp, ctypes.c_int64, _vp, _sz,
                                           _vp]),
    "nightjar_sd_workspace_bytes": (_sz, [ctypes.POINTER(ModelDesc), _i32]),
    "nightjar_sd_step": (ctypes.c_int, [ctypes.POINTER(ModelDesc), ctypes.POINTER(Weights), ctypes.POINTER(KvCache),
                                        ctypes.POINTER(ModelDesc), ctypes.POINTER(Weights), ctypes.POINTER(KvCache),
                                        _vp, _i32, _vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _sz, _vp,
                                        _sz, _vp]),
    "nightjar_device_error": (ctypes.c_int, [_vp, _sz, _vp]),
    "nightjar_last_error": (ctypes.c_char_p, []),
    "nightjar_accept": (ctypes.c_int, [ctypes.POINTER(ModelDesc), _vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp, _vp,
                                       _sz, _vp]),
    "nightjar_gemm": (ctypes.c_int, [_i32, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _vp, _sz, _vp]),
    "nightjar_gemm_workspace_bytes": (_sz, [_i32, _i32, _i32, _i32, _i32]),
    "nightjar_gemm_with_plan": (ctypes.c_int, [_i32, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _sz,
                                               _vp]),
    "nightjar_gemm_plan_workspace_bytes": (_sz, [_i32, _i32, _i32, _i32, _i32, _i32, _i32]),
    "nightjar_accept_workspace_bytes": (_sz, [_i32, _i32, _i32]),
    "nightjar_rmsnorm_rope_workspace_bytes": (_sz, [ctypes.POINTER(ModelDesc), _i32, _i32]),
    "nightjar_rmsnorm_rope": (ctypes.c_int, [ctypes.POINTER(ModelDesc), _vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp,
                                             _vp, _vp, _sz, _vp]),
    "nightjar_attn_workspace_bytes": (_sz, [ctypes.POINTER(ModelDesc), _i32, _i32]),
    "nightjar_attn_verify": (ctypes.c_int, [ctypes.POINTER(ModelDesc), _vp, _vp, _vp, _i32, _vp, _vp, _vp, _i32,
                                            _vp, _i32, _i32, _vp, _vp, _sz, _vp]),
    "nightjar_accept_noalloc": (ctypes.c_int, [ctypes.POINTER(ModelDesc), _vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp,
                                               _vp, _vp]),
    "nightjar_planner_create": (_vp, [ctypes.POINTER(PlannerConfig)]),
    "nightjar_planner_destroy": (None, [_vp]),
    "nightjar_planner_set_switch_cost": (ctypes.c_int, [_vp, _vp, _i32, _vp, _i32, _vp]),
    "nightjar_planner_switch_cost": (ctypes.c_double, [_vp, _i32, _i32]),
    "nightjar_planner_select": (ctypes.c_int, [_vp, _i32, _i32, _i32, ctypes.POINTER(_i32)]),
    "nightjar_planner_observe": (ctypes.c_int, [_vp, _i32, _i32, ctypes.c_double, _i32]),
    "nightjar_planner_bstate": (ctypes.c_int, [_vp, _i32, ctypes.POINTER(PlannerBState)]),
    "nightjar_planner_arm": (ctypes.c_int, [_vp, _i32, _i32, ctypes.POINTER(ctypes.c_double),
                                            ctypes.POINTER(ctypes.c_int64)]),
    "nightjar_contraction_plan": (ctypes.c_int, [_vp, _i32, _i32, _vp, _i32, _i32, _i32, _vp, _vp, _i32,
                                                 ctypes.POINTER(_i32), _vp, ctypes.POINTER(_i32)]),
    "nightjar_kv_migrate": (ctypes.c_int, [ctypes.POINTER(ModelDesc), ctypes.POINTER(KvCache), _vp, _vp, _i32, _vp,
                                           _vp]),
    "nightjar_profile_enable": (ctypes.c_int, [_i32]),
    "nightjar_profile_read": (ctypes.c_int, [_i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]),
    "nightjar_elastic_create": (_vp, [ctypes.POINTER(ElasticConfig)]),
    "nightjar_elastic_destroy": (None, [_vp]),
    "nightjar_elastic_step": (ctypes.c_int, [_vp, _i32, _i32, _i32, _i32, ctypes.POINTER(_i32)]),
    "nightjar_elastic_done": (ctypes.c_int, [_vp, _i32]),
    "nightjar_elastic_state": (ctypes.c_int, [_vp, ctypes.POINTER(_i32), ctypes.POINTER(_i32), ctypes.POINTER(_i32)]),
    "nightjar_offload": (ctypes.c_int, [_vp, _vp, _sz, _vp]),
    "nightjar_reload": (ctypes.c_int, [_vp, _vp, _sz, _vp]),
    "nightjar_packed_weight_elems": (_sz, [_i32, _i32]),
    "nightjar_pack_weight": (ctypes.c_int, [_vp, _vp, _i32, _i32, _vp]),
}


def lib() -> ctypes.CDLL:
    """Load the built library; fails loudly if it is missing (there is no fallback)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2512_22420_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype, fn.argtypes = res, args
        _LIB = L
    return _LIB


def last_error() -> str:
    return lib().nightjar_last_error().decode()


def _check(rc: int) -> int:
    if rc < 0:
        raise NightjarError(rc, last_error())
    return rc


def workspace_bytes(desc: ModelDesc, max_B: int, max_k: int) -> int:
    n = lib().nightjar_workspace_bytes(ctypes.byref(desc), max_B, max_k)
    if n == 0:
        raise NightjarError(NJ_EINVAL, last_error())
    return n


def step_folds_norms(desc: ModelDesc, B: int, k: int) -> bool:
    return bool(_check(lib().nightjar_step_folds_norms(ctypes.byref(desc), B, k)))


def workspace_init(workspace: int, nbytes: int, stream: int = 0) -> None:
    _check(lib().nightjar_workspace_init(workspace, nbytes, stream))


def verify_step(desc, weights, kv, block_table, max_blocks, context_lens, last_tokens, draft_tokens, draft_probs,
                uniforms, B, k, accepted_len, next_tokens, target_logits, workspace, workspace_nbytes,
                stream: int = 0) -> None:
    _check(lib().nightjar_verify_step(ctypes.byref(desc), ctypes.byref(weights), ctypes.byref(kv), block_table,
                                      max_blocks, context_lens, last_tokens, draft_tokens, draft_probs, uniforms,
                                      B, k, accepted_len, next_tokens, target_logits, workspace, workspace_nbytes,
                                      stream))


def kv_append(desc, kv, block_table, max_blocks, context_lens, accepted_len, B, k, workspace, workspace_nbytes,
              stream: int = 0) -> None:
    _check(lib().nightjar_kv_append(ctypes.byref(desc), ctypes.byref(kv), block_table, max_blocks, context_lens,
                                    accepted_len, B, k, workspace, workspace_nbytes, stream))


def draft_step(desc, weights, kv, block_table, max_blocks, context_lens, last_tokens, uniforms, B, token_out,
               token_stride, probs_out, probs_stride, workspace, workspace_nbytes, stream: int = 0) -> None:
    _check(lib().nightjar_draft_step(ctypes.byref(desc), ctypes.byref(weights), ctypes.byref(kv), block_table,
                                     max_blocks, context_lens, last_tokens, uniforms, B, token_out, token_stride,
                                     probs_out, probs_stride, workspace, workspace_nbytes, stream))


def sd_workspace_bytes(draft_desc, B) -> int:
    n = lib().nightjar_sd_workspace_bytes(ctypes.byref(draft_desc), B)
    if n == 0:
        raise NightjarError(NJ_EINVAL, last_error())
    return n


def sd_step(tdesc, tw, tkv, ddesc, dw, dkv, block_table, max_blocks, context_lens, last_tokens, draft_uniforms,
            uniforms, B, k, draft_tokens, draft_probs, accepted_len, next_tokens, target_ws, target_ws_nbytes,
            draft_ws, draft_ws_nbytes, stream: int = 0) -> None:
    _check(lib().nightjar_sd_step(ctypes.byref(tdesc), ctypes.byref(tw), ctypes.byref(tkv), ctypes.byref(ddesc),
                                  ctypes.byref(dw), ctypes.byref(dkv), block_table, max_blocks, context_lens,
                                  last_tokens, draft_uniforms, uniforms, B, k, draft_tokens, draft_probs,
                                  accepted_len, next_tokens, target_ws, target_ws_nbytes, draft_ws, draft_ws_nbytes,
                                  stream))


def device_error(workspace: int, workspace_nbytes: int, stream: int = 0) -> int:
    return _check(lib().nightjar_device_error(workspace, workspace_nbytes, stream))


def accept_workspace_bytes(vocab, B, k) -> int:
    n = lib().nightjar_accept_workspace_bytes(vocab, B, k)
    if n == 0:
        raise NightjarError(NJ_EINVAL, last_error())
    return n


def accept(desc, logits, draft_tokens, draft_probs, uniforms, B, k, accepted_len, next_tokens, workspace,
           workspace_nbytes, stream: int = 0) -> None:
    _check(lib().nightjar_accept(ctypes.byref(desc), logits, draft_tokens, draft_probs, uniforms, B, k,
                                 accepted_len, next_tokens, workspace, workspace_nbytes, stream))


def gemm_workspace_bytes(dtype, M, N, K, epilogue) -> int:
    n = lib().nightjar_gemm_workspace_bytes(dtype, M, N, K, epilogue)
    if n == 0:
        raise NightjarError(NJ_EINVAL, last_error())
    return n


def gemm(dtype, x, w, y, M, N, K, epilogue, workspace, workspace_nbytes, stream: int = 0) -> None:
    _check(lib().nightjar_gemm(dtype, x, w, y, M, N, K, epilogue, workspace, workspace_nbytes, stream))


def gemm_plan_workspace_bytes(dtype, M, N, K, epilogue, kernel, split_k) -> int:
    n = lib().nightjar_gemm_plan_workspace_bytes(dtype, M, N, K, epilogue, kernel, split_k)
    if n == 0:
        raise NightjarError(NJ_EINVAL, last_error())
    return n


def gemm_with_plan(dtype, x, w, y, M, N, K, epilogue, kernel, split_k, workspace, workspace_nbytes,
                   stream: int = 0) -> None:
    _check(lib().nightjar_gemm_with_plan(dtype, x, w, y, M, N, K, epilogue, kernel, split_k, workspace,
                                         workspace_nbytes, stream))


def accept_noalloc(desc, logits, draft_tokens, draft_probs, uniforms, B, k, accepted_len, next_tokens, device_error,
                   stream: int = 0) -> None:
    _check(lib().nightjar_accept_noalloc(ctypes.byref(desc), logits, draft_tokens, draft_probs, uniforms, B, k,
                                         accepted_len, next_tokens, device_error, stream))


def rmsnorm_rope_workspace_bytes(desc, B, k) -> int:
    n = lib().nightjar_rmsnorm_rope_workspace_bytes(ctypes.byref(desc), B, k)
    if n == 0:
        raise NightjarError(NJ_EINVAL, last_error())
    return n


def rmsnorm_rope(desc, h, attn_norm, w_qkv, context_lens, B, k, q_out, win_k, win_v, workspace, workspace_nbytes,
                 stream: int = 0) -> None:
    _check(lib().nightjar_rmsnorm_rope(ctypes.byref(desc), h, attn_norm, w_qkv, context_lens, B, k, q_out, win_k,
                                       win_v, workspace, workspace_nbytes, stream))


def attn_workspace_bytes(desc, B, k) -> int:
    n = lib().nightjar_attn_workspace_bytes(ctypes.byref(desc), B, k)
    if n == 0:
        raise NightjarError(NJ_EINVAL, last_error())
    return n


def attn_verify(desc, q, k_pages, v_pages, num_blocks, win_k, win_v, block_table, max_blocks, context_lens, B, k,
                out, workspace, workspace_nbytes, stream: int = 0) -> None:
    _check(lib().nightjar_attn_verify(ctypes.byref(desc), q, k_pages, v_pages, num_blocks, win_k, win_v,
                                      block_table, max_blocks, context_lens, B, k, out, workspace, workspace_nbytes,
                                      stream))


def packed_weight_elems(N, K) -> int:
    n = lib().nightjar_packed_weight_elems(N, K)
    if n == 0:
        raise NightjarError(NJ_EINVAL, last_error())
    return n


def pack_weight(src, dst, N, K, stream: int = 0) -> None:
    _check(lib().nightjar_pack_weight(src, dst, N, K, stream))


def contraction_plan(block_table, free_list, k_boundary: int, k_total: int):
    """nightjar_contraction_plan on numpy arrays (host memory).  Returns
    (src, dst, new_table, new_free); raises NightjarError (code NJ_EAGAIN when
    the contraction must be deferred)."""
    import numpy as np
    table = np.ascontiguousarray(block_table, dtype=np.int32).copy()
    free = np.ascontiguousarray(free_list, dtype=np.int32)
    B, mb = table.shape
    cap = max(1, int((table >= k_boundary).sum()))
    src = np.zeros(cap, np.int32)
    dst = np.zeros(cap, np.int32)
    new_free = np.zeros(max(1, len(free)), np.int32)
    nm, nf = _i32(0), _i32(0)
    _check(lib().nightjar_contraction_plan(table.ctypes.data, B, mb, free.ctypes.data if len(free) else None,
                                           len(free), k_boundary, k_total, src.ctypes.data, dst.ctypes.data, cap,
                                           ctypes.byref(nm), new_free.ctypes.data, ctypes.byref(nf)))
    return src[:nm.value].copy(), dst[:nm.value].copy(), table, new_free[:nf.value].copy()


def kv_migrate(desc, kv, src, dst, n, device_error, stream: int = 0) -> None:
    _check(lib().nightjar_kv_migrate(ctypes.byref(desc), ctypes.byref(kv), src, dst, n, device_error, stream))


NJ_POOL_RESIDENT, NJ_POOL_OFFLOADING, NJ_POOL_OFFLOADED, NJ_POOL_EXPANDED, NJ_POOL_CONTRACTING, NJ_POOL_RELOADING = \
    range(6)
NJ_ACT_NONE, NJ_ACT_OFFLOAD_DRAFT, NJ_ACT_EXPAND, NJ_ACT_CONTRACT, NJ_ACT_RELOAD_DRAFT = range(5)


class Elastic:
    """The elastic pool controller of include/nightjar_memory.h; marshalling only."""

    def __init__(self, n_orig, n_draft, tau_low, t_persist=3, reload_persist=3, max_migrate=1 << 30):
        cfg = ElasticConfig(n_orig, n_draft, tau_low, t_persist, reload_persist, max_migrate)
        self._e = lib().nightjar_elastic_create(ctypes.byref(cfg))
        if not self._e:
            raise NightjarError(NJ_EINVAL, last_error())

    def __del__(self):
        if getattr(self, "_e", None) and _LIB is not None:
            _LIB.nightjar_elastic_destroy(self._e)
            self._e = None

    def step(self, n_free, n_waiting, speculating, live_above=0) -> int:
        a = _i32(-1)
        _check(lib().nightjar_elastic_step(self._e, n_free, n_waiting, int(speculating), live_above, ctypes.byref(a)))
        return a.value

    def done(self, action) -> None:
        _check(lib().nightjar_elastic_done(self._e, action))

    def state(self):
        st, pb, ga = _i32(), _i32(), _i32()
        _check(lib().nightjar_elastic_state(self._e, ctypes.byref(st), ctypes.byref(pb), ctypes.byref(ga)))
        return st.value, pb.value, bool(ga.value)


def offload(device_src, host_dst, nbytes, stream: int = 0) -> None:
    _check(lib().nightjar_offload(device_src, host_dst, nbytes, stream))


def reload(host_src, device_dst, nbytes, stream: int = 0) -> None:
    _check(lib().nightjar_reload(host_src, device_dst, nbytes, stream))


class Planner:
    """The planner of include/nightjar_planner.h (Algorithm 1), one object per
    decision loop; marshalling only."""

    def __init__(self, max_batch: int, max_gamma: int, seed: int = 0, prev_per_batch: bool = False,
                 unplayed_latency: float = 0.0):
        cfg = PlannerConfig(max_batch, max_gamma, seed, int(prev_per_batch), unplayed_latency)
        self._p = lib().nightjar_planner_create(ctypes.byref(cfg))
        if not self._p:
            raise NightjarError(NJ_EINVAL, last_error())

    def __del__(self):
        if getattr(self, "_p", None) and _LIB is not None:
            _LIB.nightjar_planner_destroy(self._p)
            self._p = None

    def set_switch_cost(self, lengths, batches, seconds) -> None:
        nl, nbt = len(lengths), len(batches)
        la = (_i32 * nl)(*lengths)
        ba = (_i32 * nbt)(*batches)
        flat = [float(v) for row in seconds for v in row]
        sa = (ctypes.c_double * len(flat))(*flat)
        _check(lib().nightjar_planner_set_switch_cost(self._p, ctypes.cast(la, _vp), nl, ctypes.cast(ba, _vp), nbt,
                                                      ctypes.cast(sa, _vp)))

    def switch_cost(self, delta_max: int, B: int) -> float:
        v = lib().nightjar_planner_switch_cost(self._p, delta_max, B)
        if v < 0:
            raise NightjarError(NJ_EINVAL, last_error())
        return v

    def select(self, B: int, delta_max: int = 0, gamma_limit: int = 15) -> int:
        g = _i32(-1)
        _check(lib().nightjar_planner_select(self._p, B, delta_max, gamma_limit, ctypes.byref(g)))
        return g.value

    def observe(self, B: int, gamma: int, step_seconds: float, committed_tokens: int) -> None:
        _check(lib().nightjar_planner_observe(self._p, B, gamma, step_seconds, committed_tokens))

    def bstate(self, B: int) -> PlannerBState:
        st = PlannerBState()
        _check(lib().nightjar_planner_bstate(self._p, B, ctypes.byref(st)))
        return st

    def arm(self, B: int, gamma: int):
        m, n = ctypes.c_double(), ctypes.c_int64()
        _check(lib().nightjar_planner_arm(self._p, B, gamma, ctypes.byref(m), ctypes.byref(n)))
        return m.value, n.value


PROF_KERNELS = ("embed", "qkv", "norm", "rope", "attention", "o", "gate_up", "down", "lm_head", "accept",
                "kv_append")


def profile_enable(on: bool) -> None:
    _check(lib().nightjar_profile_enable(int(on)))


def profile_read() -> dict:
    """{kernel class: (mean us per launch, launches)} since profile_enable."""
    out = {}
    for i, name in enumerate(PROF_KERNELS):
        m, n = ctypes.c_double(), ctypes.c_int64()
        _check(lib().nightjar_profile_read(i, ctypes.byref(m), ctypes.byref(n)))
        out[name] = (m.value, n.value)
    return out


def header_functions(header_path: str):
    """Names of the functions declared in the C header (used by the ABI tests)."""
    import re
    text = open(header_path).read()
    return sorted(set(re.findall(r"\b(nightjar_[a-z_]+)\s*\(", text)))
