"""The elastic pool controller (include/nightjar_memory.h) against the plain
reference oracle/elastic.py, and the reference against Sec. 6.1 of the paper:

* a load surge: with speculation off and fewer than tau_low free blocks for
  T_persist = 3 steps the draft is offloaded, then the pool expands by
  N_draft blocks; two low steps are not enough (persistence window);
* while the pool is expanded or the draft is away, the planner may not
  speculate (gamma limit 0);
* the load falls: contraction waits for an empty queue and N_draft + tau_low
  free blocks over the reload window, and for the region to drain (at most
  max_migrate live blocks above the boundary); then the draft is reloaded and
  speculation is allowed again;
* speculating steps never count toward an offload.
Random traces: the library's actions and states equal the reference's.
"""
import os

import numpy as np
import pytest

from oracle import elastic as ref
from paper_2512_22420_amd import binding as nb

pytestmark = pytest.mark.skipif(not os.path.exists(nb.LIB_PATH), reason="libnightjar.so not built")


def _run(ctrl, trace, done_lag=1):
    """Feed (n_free, waiting, speculating, live_above) steps; asynchronous
    actions complete `done_lag` steps later.  Returns the actions and the
    gamma-allowed flag of every step."""
    pending, acts, allowed = [], [], []
    for t, (free, wait, spec, live) in enumerate(trace):
        for (due, a) in list(pending):
            if due == t:
                ctrl.done(a)
                pending.remove((due, a))
        a = ctrl.step(free, wait, spec, live)
        acts.append(a)
        if a in (ref.OFFLOAD_DRAFT, ref.CONTRACT, ref.RELOAD_DRAFT):
            pending.append((t + done_lag, a))
        allowed.append(ctrl.gamma_allowed() if hasattr(ctrl, "gamma_allowed") else ctrl.state()[2])
    return acts, allowed


def test_reference_surge_and_recovery():
    e = ref.Elastic(n_orig=1000, n_draft=200, tau_low=50, t_persist=3, reload_persist=3, max_migrate=10)
    # speculating under pressure: nothing happens
    trace = [(20, 5, True, 0)] * 5
    # speculation off, pressure for 2 steps, relief, then 3 steps of pressure
    trace += [(20, 5, False, 0)] * 2 + [(300, 5, False, 0)] + [(20, 5, False, 0)] * 3
    # offload completes the next step; still under pressure: expand
    trace += [(20, 5, False, 0)] * 2
    # load falls, but 30 live blocks sit above the boundary: deferred
    trace += [(600, 0, False, 30)] * 4
    # drained: contract, then reload, then resident
    trace += [(600, 0, False, 5)] * 6
    acts, allowed = _run(e, trace)
    order = [a for a in acts if a != ref.NONE]
    assert order == [ref.OFFLOAD_DRAFT, ref.EXPAND, ref.CONTRACT, ref.RELOAD_DRAFT]
    first_off = acts.index(ref.OFFLOAD_DRAFT)
    assert first_off == 10  # the third consecutive low step after the relief step (index 7)
    assert acts.index(ref.EXPAND) == first_off + 1  # the offload lands one step later, the pressure persists
    assert acts.index(ref.CONTRACT) >= len(trace) - 6  # not while 30 blocks were live above the boundary
    # speculation allowed only while the draft is resident
    assert all(allowed[:first_off]) and not any(allowed[first_off: acts.index(ref.RELOAD_DRAFT) + 1])
    assert allowed[-1]


def test_reference_pool_size_and_done_checks():
    e = ref.Elastic(n_orig=100, n_draft=40, tau_low=10)
    for _ in range(3):
        e.step(5, 3, False)
    assert e.state == ref.OFFLOADING and e.pool_blocks() == 100
    with pytest.raises(ValueError):
        e.done(ref.RELOAD_DRAFT)
    e.done(ref.OFFLOAD_DRAFT)
    assert e.step(5, 3, False) == ref.EXPAND and e.pool_blocks() == 140


def _random_trace(rng, n):
    out = []
    load = 0.5
    for _ in range(n):
        load = min(1.0, max(0.0, load + rng.normal(0, 0.15)))
        free = int((1.0 - load) * 1300)
        wait = int(max(0, rng.normal(load * 10 - 4, 2)))
        spec = bool(rng.random() < (0.8 if load < 0.4 else 0.1))
        live = int(rng.integers(0, 60))
        out.append((free, wait, spec, live))
    return out


@pytest.mark.parametrize("seed", range(5))
def test_library_equals_reference(seed):
    rng = np.random.default_rng(seed)
    trace = _random_trace(rng, 3000)
    kw = dict(n_orig=1000, n_draft=300, tau_low=60, t_persist=3, reload_persist=4, max_migrate=25)
    r, l = ref.Elastic(**kw), nb.Elastic(**kw)
    for lag in (1,):
        ar, gr = _run(r, trace, lag)
        al, gl = _run(l, trace, lag)
        assert ar == al and gr == gl
        assert sum(a != ref.NONE for a in ar) > 10  # the trace exercises the machine


def test_library_validates():
    with pytest.raises(nb.NightjarError):
        nb.Elastic(0, 10, 5)
    e = nb.Elastic(100, 40, 10)
    with pytest.raises(nb.NightjarError):
        e.done(nb.NJ_ACT_CONTRACT)
    assert e.state() == (nb.NJ_POOL_RESIDENT, 100, True)
