"""Plain reference of the Nightjar speculative-length planner (TEST
INFRASTRUCTURE: only tests/ and bench.py's CPU leg may use it; the library's
planner shares no code with it).

Follows Sec. 5 of the paper step by step:

* Sec. 5.1: at each decoding step the batch size B is given; the loss of a
  step is its latency per committed token plus, when speculation is switched
  back on (previous arm 0, this arm > 0), the draft model's KV-reconstruction
  cost C_switch divided by the arm.
* Sec. 5.2, Algorithm 1: every batch size keeps its own hierarchy (block j_B,
  block length H_B, bin b_B, round tau_B), all starting at 1.  When tau_B is 1
  a new bin starts: with probability 1/b_B it explores (arm uniform over
  {0..Gamma_max}), otherwise it exploits Eq. (exploitation_min), the arm that
  minimises the empirical mean latency per token plus the switching term.  The
  arm is played for every step of the bin.  After each step tau_B grows; past
  sqrt(H_B) the bin ends (b_B grows, tau_B back to 1); b_B past sqrt(H_B) ends
  the block (j_B grows, H_B = 2^(j_B - 1), b_B back to 1).
* Table "ttft_diff": C_switch is looked up from an offline table over
  (input length, batch size) and interpolated between profiled points.

Readings where the paper leaves a choice (the library's header lists the
same): gamma_{t-1} is the previous step's arm of the whole system (or of the
same B); before the first step there is no penalty; arms never played at B
take a configured estimate (0: optimistic); ties go to the smallest arm;
interpolation is bilinear, linear in the length and in log2 of the batch size,
clamped at the table's edges; an arm limit (e.g. 0 while the draft model is
offloaded) restricts both exploration and exploitation and caps a locked arm.

Random numbers: the exploration draws come from splitmix64 (Steele, Lea and
Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014), written
here from its published definition; a uniform in [0, 1) is the top 53 bits of
an output times 2^-53.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence

MASK64 = (1 << 64) - 1


class SplitMix64:
    def __init__(self, seed: int):
        self.state = seed & MASK64

    def next(self) -> int:
        self.state = (self.state + 0x9E3779B97F4A7C15) & MASK64
        z = self.state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
        return z ^ (z >> 31)

    def uniform(self) -> float:
        return (self.next() >> 11) * 2.0 ** -53


def interp_switch_cost(lengths: Sequence[int], batches: Sequence[int], table: Sequence[Sequence[float]],
                       delta: int, B: int) -> float:
    """C_switch(delta, B): bilinear over (length, log2 batch), clamped to the table."""
    def axis_pos(axis: List[float], v: float):
        if len(axis) == 1 or v <= axis[0]:
            return 0, 0.0
        if v >= axis[-1]:
            return len(axis) - 2, 1.0
        i = max(j for j in range(len(axis)) if axis[j] <= v)
        return i, (v - axis[i]) / (axis[i + 1] - axis[i])

    la = [float(x) for x in lengths]
    ba = [math.log2(b) for b in batches]
    i, wl = axis_pos(la, float(delta))
    j, wb = axis_pos(ba, math.log2(max(B, 1)))

    def at(a, b):
        return table[min(a, len(la) - 1)][min(b, len(ba) - 1)]
    c0 = (1 - wb) * at(i, j) + wb * at(i, j + 1)
    c1 = (1 - wb) * at(i + 1, j) + wb * at(i + 1, j + 1)
    return (1 - wl) * c0 + wl * c1


class Planner:
    """Algorithm 1, one decision per decoding step (select), feedback per step (observe)."""

    def __init__(self, max_batch: int, max_gamma: int, seed: int, prev_per_batch: bool = False,
                 unplayed_latency: float = 0.0, switch_table: Optional[Dict] = None):
        self.max_gamma = max_gamma
        self.rng = SplitMix64(seed)
        self.prev_per_batch = prev_per_batch
        self.unplayed = unplayed_latency
        self.table = switch_table
        # per-B hierarchy: j_B, H_B, b_B, tau_B, the locked arm, the previous arm at B
        self.state = {B: {"j": 1, "H": 1, "b": 1, "tau": 1, "arm": 0, "prev": None, "steps": 0, "bins": 0,
                          "explore": 0} for B in range(1, max_batch + 1)}
        self.sums = {}    # (B, gamma) -> [sum of latency per token, count]
        self.prev_global = None

    def mean(self, B: int, g: int) -> float:
        s = self.sums.get((B, g))
        return s[0] / s[1] if s else self.unplayed

    def switch_cost(self, delta: int, B: int) -> float:
        if not self.table:
            return 0.0
        return interp_switch_cost(self.table["lengths"], self.table["batches"], self.table["seconds"], delta, B)

    def select(self, B: int, delta_max: int = 0, gamma_limit: Optional[int] = None) -> int:
        st = self.state[B]
        limit = self.max_gamma if gamma_limit is None else min(gamma_limit, self.max_gamma)
        prev = st["prev"] if self.prev_per_batch else self.prev_global
        if st["tau"] == 1:                        # a bin starts
            st["bins"] += 1
            u = self.rng.uniform()
            if u < 1.0 / st["b"]:                 # exploration, probability 1/b_B
                st["arm"] = min(int(self.rng.uniform() * (limit + 1)), limit)
                st["explore"] += 1
            else:                                 # exploitation, Eq. (exploitation_min)
                c = self.switch_cost(delta_max, B) if prev == 0 else 0.0
                vals = [self.mean(B, g) + (c / g if (prev == 0 and g > 0) else 0.0) for g in range(limit + 1)]
                st["arm"] = min(range(limit + 1), key=lambda g: (vals[g], g))
        played = min(st["arm"], limit)
        st["steps"] += 1
        st["tau"] += 1
        if st["tau"] > math.sqrt(st["H"]):        # the bin is complete
            st["b"] += 1
            st["tau"] = 1
            if st["b"] > math.sqrt(st["H"]):      # the block is complete
                st["j"] += 1
                st["H"] = 2 ** (st["j"] - 1)
                st["b"] = 1
        st["prev"] = played
        self.prev_global = played
        return played

    def observe(self, B: int, gamma: int, step_seconds: float, committed_tokens: int) -> None:
        s = self.sums.setdefault((B, gamma), [0.0, 0])
        s[0] += step_seconds / committed_tokens
        s[1] += 1
