"""Plain reference of the elastic KV-pool controller (TEST INFRASTRUCTURE:
only tests/ may use it; the library shares no code with it).

Sec. 6.1 of the paper:
* expansion needs speculation disabled with the draft model already offloaded,
  fewer than tau_low free blocks, and that low-memory state lasting T_persist
  scheduling steps; the offload that precedes it happens in the same
  low-memory state with speculation off;
* contraction (which reloads the draft afterwards) needs an empty waiting queue
  and more than N_draft + tau_low free blocks, lasting several steps, and is
  drain-aware: it waits while too many live blocks sit in the region to give
  back;
* speculation stays off while the draft is not on the GPU (Sec. 6.5: memory is
  only moved while decoding is plain).
Sec. 6.2: offload and reload are asynchronous copies; the controller waits for
their completion.  Sec. 6.4: the draft is reloaded once the pool has shrunk.
"""
from __future__ import annotations

RESIDENT, OFFLOADING, OFFLOADED, EXPANDED, CONTRACTING, RELOADING = range(6)
NONE, OFFLOAD_DRAFT, EXPAND, CONTRACT, RELOAD_DRAFT = range(5)


class Elastic:
    def __init__(self, n_orig, n_draft, tau_low, t_persist=3, reload_persist=3, max_migrate=1 << 30):
        self.n_orig, self.n_draft, self.tau_low = n_orig, n_draft, tau_low
        self.t_persist, self.reload_persist, self.max_migrate = t_persist, reload_persist, max_migrate
        self.state = RESIDENT
        self.low_steps = 0      # consecutive steps: few free blocks, no speculation
        self.quiet_steps = 0    # consecutive steps: nobody waiting, room for the draft and the buffer
        self.reload_after_shrink = False

    def step(self, n_free, n_waiting, speculating, live_above=0):
        self.low_steps = self.low_steps + 1 if (n_free < self.tau_low and not speculating) else 0
        quiet = n_waiting == 0 and n_free > self.n_draft + self.tau_low
        self.quiet_steps = self.quiet_steps + 1 if quiet else 0
        if self.state == RESIDENT and self.low_steps >= self.t_persist:
            self.state = OFFLOADING
            return OFFLOAD_DRAFT
        if self.state == OFFLOADED:
            if self.reload_after_shrink:
                self.reload_after_shrink = False
                self.state = RELOADING
                return RELOAD_DRAFT
            if self.low_steps >= self.t_persist:
                self.state = EXPANDED
                return EXPAND
            if self.quiet_steps >= self.reload_persist:
                self.state = RELOADING
                return RELOAD_DRAFT
        if self.state == EXPANDED and self.quiet_steps >= self.reload_persist and live_above <= self.max_migrate:
            self.state = CONTRACTING
            return CONTRACT
        return NONE

    def done(self, action):
        if action == OFFLOAD_DRAFT and self.state == OFFLOADING:
            self.state = OFFLOADED
        elif action == CONTRACT and self.state == CONTRACTING:
            self.state = OFFLOADED
            self.reload_after_shrink = True
        elif action == RELOAD_DRAFT and self.state == RELOADING:
            self.state = RESIDENT
        else:
            raise ValueError(f"action {action} not in flight in state {self.state}")

    def pool_blocks(self):
        return self.n_orig + (self.n_draft if self.state in (EXPANDED, CONTRACTING) else 0)

    def gamma_allowed(self):
        return self.state == RESIDENT
