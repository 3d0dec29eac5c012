"""CPU oracle of the batched speculative verify step and of the planner (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg use it;
the HIP library never does.
"""
from .verify_step import (accept, attention, forward_window, gather_cache, invcdf,  # noqa: F401
                          kv_append, linear, rms_norm, rope, silu, softmax, verify_step, widen,
                          window_tokens)
from . import elastic, kv_pool, planner, spec_step  # noqa: F401
