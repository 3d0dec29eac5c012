"""Decision parity between the GPU's acceptance outputs and the oracle.

Accept tests: a decision whose ratio p(x)/q(x) is within RATIO_MARGIN of its
uniform is flagged and excluded (the tolerance the target statement sets).
Draws: a draw whose u*S lies within CDF_MARGIN of a running-sum boundary of the
drawn entry is flagged.  CDF_MARGIN follows from the arithmetic: the kernel
evaluates each weight p_j (or max(0, p_j - q_j)) in fp32, so any running sum of
weights carries at most ~eps32 * (sum p + sum q) = 2.4e-7 absolute error; 1e-6
leaves 4x headroom.  With ``gpu_logits`` given, decisions that the GPU's own
logits and the oracle's logits take differently ("straddles": a logit error
moved p/q or a boundary across u) are flagged too.  After the first flagged
decision of a sequence its later positions are not compared, since they are
conditioned differently.

``self_check`` is the second half: every decision of the GPU, flagged or not,
must be the one the acceptance rule takes on the GPU's own logits (softmax in
fp64 on the host), except within the same margins measured on those logits.
Straddles are excluded from the oracle comparison but still checked here, so a
test never passes on decisions that no one compared.

Every comparison is recorded in ``REPORT`` and printed in pytest's terminal
summary (checked, flagged and self-checked counts per test).
"""
import os

import numpy as np

import oracle

RATIO_MARGIN = 1e-3
CDF_MARGIN = 1e-6


def _draw_weights(p, q, n, k):
    if n < k:
        w = np.maximum(0.0, p[n] - q[n])
        return w if np.any(w > 0) else p[n]
    return p[k]


def compare(gpu_acc, gpu_next, ref_logits, drafts, dprobs, uniforms, gpu_logits=None):
    """Returns dict(checked, flagged, mismatches=[...])."""
    B = len(gpu_acc)
    k = drafts.shape[1] if drafts.ndim == 2 else 0
    out = {"checked": 0, "flagged": 0, "mismatches": [], "accepted": 0}
    for b in range(B):
        p = oracle.softmax(np.asarray(ref_logits[b], dtype=np.float64))
        pg = oracle.softmax(np.asarray(gpu_logits[b], dtype=np.float64)) if gpu_logits is not None else None
        q = np.asarray(dprobs[b], dtype=np.float64) if k else np.zeros((0, p.shape[1]))
        u = np.asarray(uniforms[b], dtype=np.float64)
        flagged = False
        n = 0
        while n < k:
            x = int(drafts[b, n])
            r = p[n, x] / q[n, x] if q[n, x] > 0 else np.inf
            if abs(r - u[n]) < RATIO_MARGIN:
                flagged = True
                break
            if pg is not None:
                rg = pg[n, x] / q[n, x] if q[n, x] > 0 else np.inf
                if (u[n] < r) != (u[n] < rg):
                    flagged = True
                    break
            out["checked"] += 1
            acc = u[n] < r
            if acc != (int(gpu_acc[b]) > n):
                out["mismatches"].append((b, n, "accept", bool(acc), int(gpu_acc[b])))
                flagged = True  # do not compare further positions of this sequence
                break
            if not acc:
                break
            n += 1
        if flagged:
            out["flagged"] += 1
            continue
        if int(gpu_acc[b]) != n:
            out["mismatches"].append((b, n, "accepted_len", n, int(gpu_acc[b])))
            continue
        if list(gpu_next[b, :n]) != [int(t) for t in drafts[b, :n]]:
            out["mismatches"].append((b, n, "prefix"))
            continue
        w = _draw_weights(p, q, n, k)
        c = np.cumsum(w)
        target = u[k] * c[-1]
        j = oracle.invcdf(w, u[k])
        lo = c[j - 1] if j > 0 else 0.0
        if abs(target - lo) < CDF_MARGIN or abs(c[j] - target) < CDF_MARGIN:
            out["flagged"] += 1
            continue
        if pg is not None:
            wg = _draw_weights(pg, q, n, k)
            if oracle.invcdf(wg, u[k]) != j:
                out["flagged"] += 1
                continue
        out["checked"] += 1
        out["accepted"] += n
        if int(gpu_next[b, n]) != j:
            out["mismatches"].append((b, n, "draw", j, int(gpu_next[b, n])))
        if any(int(t) != -1 for t in gpu_next[b, n + 1:]):
            out["mismatches"].append((b, n, "padding"))
    return out


def self_check(gpu_acc, gpu_next, gpu_logits, drafts, dprobs, uniforms):
    """The rule applied to the GPU's own logits, position by position.

    Returns dict(checked, margin, mismatches): `checked` counts decisions
    compared (accept tests and draws), `margin` those within RATIO_MARGIN /
    CDF_MARGIN on these logits (a fp32 vs fp64 evaluation may take them either
    way; the rest of that sequence is then skipped)."""
    B = len(gpu_acc)
    k = drafts.shape[1] if drafts.ndim == 2 else 0
    out = {"checked": 0, "margin": 0, "mismatches": []}
    for b in range(B):
        p = oracle.softmax(np.asarray(gpu_logits[b], dtype=np.float64))
        q = np.asarray(dprobs[b], dtype=np.float64) if k else np.zeros((0, p.shape[1]))
        u = np.asarray(uniforms[b], dtype=np.float64)
        n, skip = 0, False
        while n < k:
            x = int(drafts[b, n])
            r = p[n, x] / q[n, x] if q[n, x] > 0 else np.inf
            if abs(r - u[n]) < RATIO_MARGIN:
                skip = True
                break
            out["checked"] += 1
            acc = u[n] < r
            if acc != (int(gpu_acc[b]) > n):
                out["mismatches"].append((b, n, "accept(self)", bool(acc), int(gpu_acc[b])))
                skip = True
                break
            if not acc:
                break
            n += 1
        if skip:
            out["margin"] += 1
            continue
        if int(gpu_acc[b]) != n or list(gpu_next[b, :n]) != [int(t) for t in drafts[b, :n]]:
            out["mismatches"].append((b, n, "prefix(self)"))
            continue
        w = _draw_weights(p, q, n, k)
        c = np.cumsum(w)
        target = u[k] * c[-1]
        j = oracle.invcdf(w, u[k])
        lo = c[j - 1] if j > 0 else 0.0
        if abs(target - lo) < CDF_MARGIN or abs(c[j] - target) < CDF_MARGIN:
            out["margin"] += 1
            continue
        out["checked"] += 1
        if int(gpu_next[b, n]) != j:
            out["mismatches"].append((b, n, "draw(self)", j, int(gpu_next[b, n])))
    return out


REPORT = []


def record(res, selfres=None):
    """Keep a comparison's counts for the terminal summary (test id from pytest's environment)."""
    name = os.environ.get("PYTEST_CURRENT_TEST", "?").split(" (")[0]
    REPORT.append((name, res.get("checked", 0), res.get("flagged", 0), res.get("accepted", 0),
                   None if selfres is None else selfres["checked"], None if selfres is None else selfres["margin"]))


def rel_l2_rows(a, b):
    a = np.asarray(a, dtype=np.float64).reshape(-1, a.shape[-1])
    b = np.asarray(b, dtype=np.float64).reshape(-1, b.shape[-1])
    return np.linalg.norm(a - b, axis=1) / np.linalg.norm(b, axis=1)
