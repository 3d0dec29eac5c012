"""The speculative-length planner (Sec. 5, Algorithm 1) through the C ABI of
include/nightjar_planner.h, against the plain reference in oracle/planner.py,
and both against what the paper fixes:

* the worked trace of Sec. 5.2: batch sizes (3,4,4,2,4,4,4) give five local
  rounds on the B = 4 timeline;
* the block / bin schedule: blocks of H = 2^(j-1) rounds made of bins of
  floor(sqrt(H)) rounds, so O(sqrt(T_B)) bins (and switches) after T_B steps
  (Appendix A);
* exploitation converges to argmin_gamma of the mean latency per token, and the
  regret grows sublinearly (Appendix A);
* the switching term of Eq. (exploitation_min) keeps speculation off when
  C_switch / gamma outweighs the gain;
* C_switch from the paper's Table ttft_diff is returned exactly at the
  profiled points and interpolated between them.
The library and the reference draw exploration from the same published
generator (splitmix64), so their decisions must agree step for step.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import planner as ref
from paper_2512_22420_amd import binding as nb

HERE = os.path.dirname(os.path.abspath(__file__))
pytestmark = pytest.mark.skipif(not os.path.exists(nb.LIB_PATH), reason="libnightjar.so not built")


def _table():
    t = json.load(open(os.path.join(HERE, "golden", "switch_cost_ttft_diff.json")))
    return t["lengths"], t["batches"], [[v / 1e3 for v in row] for row in t["ms"]]


# --------------------------------------------------------------------------
# the reference against the paper
# --------------------------------------------------------------------------
def test_reference_worked_trace_gives_five_local_rounds():
    p = ref.Planner(max_batch=8, max_gamma=4, seed=1)
    for B in (3, 4, 4, 2, 4, 4, 4):
        p.select(B)
    assert p.state[4]["steps"] == 5 and p.state[3]["steps"] == 1 and p.state[2]["steps"] == 1
    # blocks of 1, 1, then 4 rounds (two bins of two): rounds 1, 2, 3 and 5 start bins
    assert p.state[4]["bins"] == 4
    assert (p.state[4]["j"], p.state[4]["H"], p.state[4]["b"], p.state[4]["tau"]) == (3, 4, 2, 2)


def _bins_after(T):
    """Closed form of the schedule: block j has H = 2^(j-1) rounds split into
    floor(sqrt(H)) bins of floor(sqrt(H)) rounds."""
    bins, t, j = 0, 0, 1
    while t < T:
        H = 2 ** (j - 1)
        r = math.isqrt(H)
        for _ in range(r):
            if t >= T:
                break
            bins += 1
            t += r
        j += 1
    return bins


@pytest.mark.parametrize("T", [1, 7, 100, 1000, 20000])
def test_reference_bin_count_matches_closed_form_and_grows_as_sqrt(T):
    p = ref.Planner(max_batch=1, max_gamma=3, seed=2)
    for _ in range(T):
        p.select(1)
    assert p.state[1]["bins"] == _bins_after(T)
    assert p.state[1]["bins"] <= 4 * math.sqrt(T) + 2


def _stream(mu, noise, seed):
    rng = np.random.default_rng(seed)
    return lambda g: max(1e-6, mu[g] * (1.0 + noise * rng.standard_normal()))


def test_reference_converges_to_the_best_arm_with_sublinear_regret():
    mu = [5e-3, 3e-3, 2e-3, 2.5e-3, 4e-3]  # seconds per token; gamma* = 2
    p = ref.Planner(max_batch=1, max_gamma=4, seed=3)
    lat = _stream(mu, 0.2, 0)
    regret, marks = 0.0, {}
    arms = []
    for t in range(1, 160001):
        g = p.select(1)
        arms.append(g)
        p.observe(1, g, lat(g), 1)
        regret += mu[g] - min(mu)
        if t in (2500, 160000):
            marks[t] = regret
    assert np.mean(np.array(arms[-20000:]) == 2) > 0.9
    # a 64x longer horizon: regret per step falls by more than 3x, and the
    # regret grows by less than 64^0.75 (linear regret would grow 64x)
    assert marks[160000] / 160000 < 0.33 * marks[2500] / 2500
    assert marks[160000] / marks[2500] < 64 ** 0.75


def test_reference_switch_cost_keeps_speculation_off():
    """mu_0 = 2.0 ms/token, mu_3 = 1.9 ms/token: with C_switch = 30 ms the
    switching term 30/3 = 10 ms outweighs the 0.1 ms gain, so after gamma = 0
    exploitation stays at 0; without the table it switches to 3."""
    for cost, want in ((0.030, 0), (None, 3)):
        table = None if cost is None else {"lengths": [0], "batches": [1], "seconds": [[cost]]}
        p = ref.Planner(max_batch=1, max_gamma=3, seed=4, unplayed_latency=1.0, switch_table=table)
        for g, m in ((0, 2.0e-3), (3, 1.9e-3), (1, 5e-3), (2, 5e-3)):
            p.observe(1, g, m, 1)
        p.prev_global = 0
        p.state[1]["b"] = 10 ** 9  # exploration probability ~0 from here on
        assert p.select(1, delta_max=100) == want


def test_reference_interpolates_the_paper_table():
    L, Bs, S = _table()
    for i, l in enumerate(L):
        for j, b in enumerate(Bs):
            assert ref.interp_switch_cost(L, Bs, S, l, b) == S[i][j]
    assert math.isclose(ref.interp_switch_cost(L, Bs, S, 384, 32), (S[1][0] + S[2][0]) / 2, rel_tol=1e-12)
    assert math.isclose(ref.interp_switch_cost(L, Bs, S, 256, 2 ** 5.5), (S[1][0] + S[1][1]) / 2, rel_tol=1e-12)
    assert ref.interp_switch_cost(L, Bs, S, 4096, 1000) == S[2][1]  # clamped at the table's edge
    assert ref.interp_switch_cost(L, Bs, S, 0, 1) == S[0][0]


# --------------------------------------------------------------------------
# the library against the reference
# --------------------------------------------------------------------------
def _drive_both(max_batch, max_gamma, seed, steps, prev_per_batch, unplayed, table, trace_seed):
    rng = np.random.default_rng(trace_seed)
    lib = nb.Planner(max_batch, max_gamma, seed, prev_per_batch, unplayed)
    orc = ref.Planner(max_batch, max_gamma, seed, prev_per_batch, unplayed,
                      None if table is None else {"lengths": table[0], "batches": table[1], "seconds": table[2]})
    if table is not None:
        lib.set_switch_cost(*table)
    mu = rng.uniform(1e-3, 5e-3, size=(max_batch + 1, max_gamma + 1))
    for t in range(steps):
        B = int(rng.integers(1, max_batch + 1))
        delta = int(rng.integers(0, 700))
        limit = int(rng.integers(0, max_gamma + 1)) if rng.random() < 0.1 else max_gamma
        g1 = lib.select(B, delta, limit)
        g2 = orc.select(B, delta, limit)
        assert g1 == g2, (t, B, g1, g2)
        step_s = float(mu[B, g1] * (1 + 0.3 * rng.standard_normal()) ** 2) * (g1 + 1)
        committed = int(rng.integers(1, g1 + 2)) * B
        lib.observe(B, g1, step_s, committed)
        orc.observe(B, g1, step_s, committed)
    for B in range(1, max_batch + 1):
        st, so = lib.bstate(B), orc.state[B]
        assert (st.block, st.block_len, st.bin, st.round, st.steps, st.bins, st.explore_bins) == \
            (so["j"], so["H"], so["b"], so["tau"], so["steps"], so["bins"], so["explore"])
        for g in range(max_gamma + 1):
            m, n = lib.arm(B, g)
            s = orc.sums.get((B, g))
            assert n == (s[1] if s else 0)
            assert m == pytest.approx(orc.mean(B, g), rel=1e-12)


@pytest.mark.parametrize("prev_per_batch,unplayed,with_table", [(False, 0.0, True), (True, 0.0, True),
                                                                (False, 1.0, False), (True, 3e-3, True)])
def test_library_decisions_equal_the_reference(prev_per_batch, unplayed, with_table):
    _drive_both(16, 5, 123, 6000, prev_per_batch, unplayed, _table() if with_table else None, 7)


def test_library_worked_trace_and_schedule():
    p = nb.Planner(8, 4, seed=1)
    for B in (3, 4, 4, 2, 4, 4, 4):
        p.select(B)
    s = p.bstate(4)
    assert (s.steps, s.bins, s.block, s.block_len, s.bin, s.round) == (5, 4, 3, 4, 2, 2)
    assert p.bstate(3).steps == 1 and p.bstate(2).steps == 1
    q = nb.Planner(1, 3, seed=2)
    for _ in range(20000):
        q.select(1)
    assert q.bstate(1).bins == _bins_after(20000)


def test_library_arm_is_locked_within_a_bin_and_respects_the_limit():
    p = nb.Planner(1, 5, seed=9)
    rng = np.random.default_rng(0)
    prev_bins, arm = 0, None
    for t in range(5000):
        g = p.select(1, 0, 5)
        st = p.bstate(1)
        started = st.bins != prev_bins
        if not started:
            assert g == arm, t  # no switch inside a bin
        arm, prev_bins = g, st.bins
        p.observe(1, g, float(rng.uniform(1e-3, 2e-3)), 1)
    for _ in range(200):
        assert p.select(1, 0, 0) == 0  # draft model offloaded: only plain decoding


def test_library_switch_cost_table():
    L, Bs, S = _table()
    p = nb.Planner(64, 4)
    assert p.switch_cost(300, 40) == 0.0  # no table: the original loss
    p.set_switch_cost(L, Bs, S)
    for i, l in enumerate(L):
        for j, b in enumerate(Bs):
            assert p.switch_cost(l, b) == pytest.approx(S[i][j], rel=1e-15)
    for d, b in ((384, 32), (256, 45), (100, 64), (700, 48), (300, 8)):
        assert p.switch_cost(d, b) == pytest.approx(ref.interp_switch_cost(L, Bs, S, d, b), rel=1e-12)
    with pytest.raises(nb.NightjarError):
        p.set_switch_cost([256, 128], Bs, S)  # lengths must increase
    with pytest.raises(nb.NightjarError):
        nb.Planner(0, 4)
    with pytest.raises(nb.NightjarError):
        nb.Planner(4, 16)


def test_library_decision_time_is_negligible():
    """Sec. 5.2 reports ~1e-5 s per arm selection; one select + observe here
    must stay far below a decoding step (tens of microseconds at most)."""
    import time
    p = nb.Planner(256, 7, seed=5)
    rng = np.random.default_rng(1)
    Bs = rng.integers(1, 257, size=20000)
    t0 = time.perf_counter()
    for B in Bs:
        g = p.select(int(B), 64, 7)
        p.observe(int(B), g, 1e-2, int(B))
    per = (time.perf_counter() - t0) / len(Bs)
    assert per < 1e-4, per
