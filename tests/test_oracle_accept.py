"""Pins of the oracle's acceptance rule and inverse-CDF draw.

The paper (Sec. 1, Sec. 6.5) claims speculative decoding is lossless: the
committed tokens are distributed exactly as the target model would produce
them autoregressively.  Sec. 3.1 / Sec. 5.1: a step commits n accepted drafts
plus one token, 0 <= n <= gamma.  Sec. 2.2: a wrong draft is dropped at the
first error and replaced.  These tests turn those statements into exact
checks of ``oracle.accept`` / ``oracle.invcdf``:

* exact enumeration over draft tuples and over the pieces on which the
  oracle's output is constant in each uniform: the distribution of the first
  N committed tokens equals prod_t p(y_t | y_<t) to 1e-12, for any schedule
  of speculative lengths (including gamma = 0);
* invariants over many random cases.
"""
import itertools

import numpy as np
import pytest

import oracle


# --------------------------------------------------------------------------
# A tiny "language model" pair: deterministic distributions over V tokens
# for every prefix, with some exact zeros.
# --------------------------------------------------------------------------
class TablePair:
    def __init__(self, V, seed, zero_frac=0.25, same=False):
        self.V, self.seed, self.zero_frac, self.same = V, seed, zero_frac, same
        self.cache = {}

    def _dist(self, prefix, which):
        key = (which, tuple(prefix))
        if key not in self.cache:
            rng = np.random.default_rng([self.seed, 0 if which == "p" else 1, len(prefix), *prefix])
            w = rng.gamma(0.7, size=self.V)
            w[rng.random(self.V) < self.zero_frac] = 0.0
            if w.sum() == 0:
                w[rng.integers(self.V)] = 1.0
            self.cache[key] = w / w.sum()
        return self.cache[key]

    def p(self, prefix):
        return self._dist(prefix, "p")

    def q(self, prefix):
        return self._dist(prefix, "p" if self.same else "q")


def _pieces(breaks):
    """Sorted distinct breakpoints in [0,1] -> (midpoint, length) of each piece."""
    b = np.unique(np.clip(np.concatenate([[0.0, 1.0], breaks]), 0.0, 1.0))
    return [(0.5 * (lo + hi), hi - lo) for lo, hi in zip(b[:-1], b[1:]) if hi > lo]


def step_distribution(pair, prefix, gamma):
    """Exact distribution of the tokens one verify step commits after `prefix`.

    Enumerates every draft tuple (weighted by the draft's probability) and every
    piece of the uniforms on which the oracle's output is constant.
    """
    out = {}
    V = pair.V
    for d in itertools.product(range(V), repeat=gamma):
        pd, ctx = 1.0, list(prefix)
        for x in d:
            pd *= pair.q(ctx)[x]
            ctx.append(x)
        if pd == 0.0:
            continue
        P = np.array([pair.p(list(prefix) + list(d[:i])) for i in range(gamma + 1)])
        Q = np.array([pair.q(list(prefix) + list(d[:i])) for i in range(gamma)]).reshape(gamma, V)
        # accept-test pieces: u_i < min(1, p/q) accepts
        acc_pieces = []
        for i in range(gamma):
            r = min(1.0, P[i, d[i]] / Q[i, d[i]])
            acc_pieces.append(_pieces(np.array([r])))
        # final-draw pieces: union of the breakpoints of every candidate row
        cands = [P[gamma]] + [np.maximum(0.0, P[i] - Q[i]) for i in range(gamma)] + list(P[:gamma])
        br = []
        for w in cands:
            if w.sum() > 0:
                br.extend(np.cumsum(w) / w.sum())
        fin_pieces = _pieces(np.array(br))
        for combo in itertools.product(*acc_pieces):
            pu = np.prod([c[1] for c in combo]) if combo else 1.0
            if pu == 0.0:
                continue
            for um, ul in fin_pieces:
                u = [c[0] for c in combo] + [um]
                n, toks = oracle.accept(P, Q, list(d), u)
                key = tuple(toks)
                out[key] = out.get(key, 0.0) + pd * pu * ul
    return out


def committed_distribution(pair, schedule, N):
    """Distribution of the first N committed tokens when each step uses the next
    speculative length of `schedule` (cycled)."""
    dist = {}

    def rec(prefix, prob, step):
        if len(prefix) >= N:
            key = tuple(prefix[:N])
            dist[key] = dist.get(key, 0.0) + prob
            return
        gamma = schedule[step % len(schedule)]
        for toks, pr in step_distribution(pair, prefix, gamma).items():
            rec(prefix + list(toks), prob * pr, step + 1)

    rec([], 1.0, 0)
    return dist


def autoregressive_distribution(pair, N):
    dist = {}
    for y in itertools.product(range(pair.V), repeat=N):
        pr = 1.0
        for t in range(N):
            pr *= pair.p(list(y[:t]))[y[t]]
            if pr == 0.0:
                break
        if pr > 0.0:
            dist[y] = pr
    return dist


def _assert_same(d1, d2, tol=1e-12):
    keys = set(d1) | set(d2)
    err = max(abs(d1.get(k, 0.0) - d2.get(k, 0.0)) for k in keys)
    assert err < tol, err
    assert abs(sum(d1.values()) - 1.0) < tol


@pytest.mark.parametrize("V,schedule,N,seed", [
    (3, [1], 3, 0),
    (3, [2], 3, 1),
    (4, [3], 4, 2),
    (3, [2, 0, 3, 1], 4, 3),
    (4, [0], 3, 4),
])
def test_committed_tokens_follow_target_distribution(V, schedule, N, seed):
    pair = TablePair(V, seed)
    _assert_same(committed_distribution(pair, schedule, N), autoregressive_distribution(pair, N))


@pytest.mark.parametrize("gamma", [1, 2, 3])
def test_first_token_marginal_is_p0(gamma):
    pair = TablePair(4, 10 + gamma)
    marg = np.zeros(4)
    for toks, pr in step_distribution(pair, [], gamma).items():
        marg[toks[0]] += pr
    np.testing.assert_allclose(marg, pair.p([]), atol=1e-13, rtol=0)


def test_identical_draft_is_always_fully_accepted():
    pair = TablePair(3, 7, same=True)
    for toks, pr in step_distribution(pair, [], 3).items():
        assert len(toks) == 4  # n == gamma, plus the bonus token


def test_step_length_distribution_matches_closed_form():
    """With one draft, P(accept) = sum_x min(p(x), q(x)) (overlap of p and q)."""
    pair = TablePair(4, 21)
    dist = step_distribution(pair, [], 1)
    p_acc = sum(pr for toks, pr in dist.items() if len(toks) == 2)
    assert abs(p_acc - np.minimum(pair.p([]), pair.q([])).sum()) < 1e-13


# --------------------------------------------------------------------------
# inverse CDF
# --------------------------------------------------------------------------
def test_invcdf_matches_searchsorted_and_never_picks_zero_weight():
    rng = np.random.default_rng(0)
    for _ in range(2000):
        V = int(rng.integers(1, 40))
        w = rng.random(V)
        w[rng.random(V) < 0.4] = 0.0
        if w.sum() == 0:
            w[-1] = 0.5
        u = rng.random()
        j = oracle.invcdf(w, u)
        c = np.cumsum(w)
        assert j == np.searchsorted(c, u * c[-1], side="right")
        assert w[j] > 0


def test_invcdf_edges():
    assert oracle.invcdf(np.array([0.0, 1.0, 0.0]), 0.0) == 1
    assert oracle.invcdf(np.array([0.25, 0.25, 0.5, 0.0]), np.nextafter(1.0, 0.0)) == 2
    assert oracle.invcdf(np.array([0.5, 0.5]), 0.5) == 1  # C_0 = 0.5 is not > 0.5
    # no index passes u*S because of rounding -> last positive weight
    w = np.array([1e-300, 0.0])
    assert oracle.invcdf(w, 1.0) == 0


# --------------------------------------------------------------------------
# invariants
# --------------------------------------------------------------------------
def test_acceptance_invariants_random():
    rng = np.random.default_rng(1)
    for _ in range(3000):
        V = int(rng.integers(2, 12))
        gamma = int(rng.integers(0, 6))
        P = rng.gamma(0.5, size=(gamma + 1, V))
        P /= P.sum(1, keepdims=True)
        Q = rng.gamma(0.5, size=(gamma, V))
        Q /= np.maximum(Q.sum(1, keepdims=True), 1e-300)
        d = [int(oracle.invcdf(Q[i], rng.random())) for i in range(gamma)]
        u = rng.random(gamma + 1)
        n, toks = oracle.accept(P, Q, d, u)
        assert 0 <= n <= gamma
        assert len(toks) == n + 1
        assert toks[:n] == d[:n]
        for i in range(n):
            assert u[i] < P[i, d[i]] / Q[i, d[i]]
        if n < gamma:
            assert u[n] >= P[n, d[n]] / Q[n, d[n]]
            y = toks[n]
            assert y != d[n]
            assert P[n, y] > Q[n, y]
        assert 0 <= toks[-1] < V


def test_certain_accept_and_certain_reject():
    P = np.array([[0.5, 0.5, 0.0], [0.2, 0.3, 0.5]])
    Q = np.array([[0.0, 0.5, 0.5]])
    # p(1)/q(1) = 1: always accepted, even with u just below 1
    n, toks = oracle.accept(P, Q, [1], [0.999999, 0.0])
    assert n == 1 and toks == [1, 0]
    # p(2) = 0: always rejected, even with u = 0; residual max(0, p - q) = [0.5, 0, 0]
    n, toks = oracle.accept(P, Q, [2], [0.0, 0.7])
    assert n == 0 and toks == [0]
    # a draft with q = 0 (never sampled by a real draft) counts as accepted
    n, toks = oracle.accept(P, Q, [0], [0.9, 0.1])
    assert n == 1 and toks == [0, 0]
