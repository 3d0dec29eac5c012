"""KV-pool contraction (Sec. 6.4, Steps 1-5): the library's plan
(include/nightjar_memory.h) against the plain reference oracle/kv_pool.py, and
the reference against what the section fixes:

* after the plan no table entry is at or above the boundary;
* the map is one-to-one onto free blocks below the boundary, a shared block
  moves once, and blocks below the boundary never move;
* with the data copied as the map says (Step 4), every sequence sees the same
  keys and values at every logical position (decoding is unaffected: the
  attention reads blocks only through the tables);
* the free list afterwards holds exactly the free blocks below the boundary
  that were not taken;
* with too few free blocks below the boundary nothing changes (deferred).
"""
import os

import numpy as np
import pytest

import oracle
from oracle import kv_pool as ref
from paper_2512_22420_amd import binding as nb
from paper_2512_22420_amd import workload as W

pytestmark = pytest.mark.skipif(not os.path.exists(nb.LIB_PATH), reason="libnightjar.so not built")


def _pool_case(seed, B=12, k_total=300, k_boundary=220, shared=3, spare_low=10):
    """Tables whose blocks are spread over the whole pool (some shared by two
    rows, as prefix sharing does), -1 past each row's blocks; the free list is
    every unused block, shuffled."""
    rng = np.random.default_rng(seed)
    lens = rng.integers(1, 12, size=B)
    used_total = int(lens.sum())
    assert used_total + spare_low < k_total
    ids = rng.permutation(k_total)[:used_total]
    mb = int(lens.max())
    table = np.full((B, mb), -1, np.int32)
    off = 0
    for b in range(B):
        table[b, : lens[b]] = ids[off: off + lens[b]]
        off += lens[b]
    for _ in range(shared):  # a row reuses another row's first block
        a, c = rng.choice(B, 2, replace=False)
        table[c, 0] = table[a, 0]
    live = set(int(x) for x in table.ravel() if x >= 0)
    free = np.array([i for i in rng.permutation(k_total) if i not in live], np.int32)
    return table, free, k_boundary, k_total


@pytest.mark.parametrize("seed", range(6))
def test_reference_plan_properties(seed):
    table, free, kb, kt = _pool_case(seed)
    p = ref.contraction_plan(table, free, kb)
    new = p["table"]
    assert np.all(new[new >= 0] < kb)
    assert len(set(p["dst"])) == len(p["dst"]) and all(d < kb for d in p["dst"])
    assert sorted(p["src"]) == sorted(set(int(x) for x in table.ravel() if x >= kb))
    assert all(int(d) in set(int(f) for f in free) for d in p["dst"])
    # blocks below the boundary keep their ids
    low = table < kb
    assert np.array_equal(new[low], table[low])
    assert p["free"] == [int(f) for f in free if f < kb and f not in set(p["dst"])]
    # data: every logical position of every row reads the same values after Step 4
    shape = W.TINY_F32
    rng = np.random.default_rng(seed)
    kp = [rng.standard_normal((kt, shape.n_kv_heads, 16, 8))]
    vp = [rng.standard_normal((kt, shape.n_kv_heads, 8, 16))]
    kp2, vp2 = ref.migrate(kp, vp, p["src"], p["dst"])
    for b in range(table.shape[0]):
        n = int((table[b] >= 0).sum()) * 16
        k1, v1 = oracle.gather_cache(kp[0], vp[0], table[b], n, 16)
        k2, v2 = oracle.gather_cache(kp2[0], vp2[0], new[b], n, 16)
        assert np.array_equal(k1, k2) and np.array_equal(v1, v2)


def test_reference_defers_without_room():
    table, free, kb, kt = _pool_case(1)
    need = len(set(int(x) for x in table.ravel() if x >= kb))
    few = np.array([f for f in free if f < kb][: need - 1] + [f for f in free if f >= kb], np.int32)
    with pytest.raises(ref.Deferred):
        ref.contraction_plan(table, few, kb)


@pytest.mark.parametrize("seed", range(6))
def test_library_plan_equals_reference(seed):
    table, free, kb, kt = _pool_case(seed)
    src, dst, new, new_free = nb.contraction_plan(table, free, kb, kt)
    p = ref.contraction_plan(table, free, kb)
    assert list(src) == p["src"] and list(dst) == p["dst"]
    assert np.array_equal(new, p["table"])
    assert list(new_free) == p["free"]


def test_library_plan_defers_and_validates():
    table, free, kb, kt = _pool_case(2)
    need = len(set(int(x) for x in table.ravel() if x >= kb))
    few = np.array([f for f in free if f < kb][: need - 1], np.int32)
    with pytest.raises(nb.NightjarError) as e:
        nb.contraction_plan(table, few, kb, kt)
    assert e.value.code == nb.NJ_EAGAIN
    with pytest.raises(nb.NightjarError) as e:  # a free block that a table still uses
        nb.contraction_plan(table, np.append(free, table[0, 0]), kb, kt)
    assert e.value.code == nb.NJ_EINVAL
    with pytest.raises(nb.NightjarError):  # an id past the pool
        t2 = table.copy()
        t2[0, 0] = kt
        nb.contraction_plan(t2, free, kb, kt)
    # nothing above the boundary: no moves, the free list just trimmed
    src, dst, new, nf = nb.contraction_plan(np.where(table >= kb, -1, table), free, kb, kt)
    assert len(src) == 0 and list(nf) == [int(f) for f in free if f < kb]
