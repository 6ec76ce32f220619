"""Causality-guided bucket routing (Sec. 5), from its description.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

Prefix tree: a node at depth k is the key (prompt_id, (s_1, ..., s_k)), s_i the
composite state of the i-th tool return.  Every node keeps a histogram of the remaining
trajectory length seen from that point, in bins aligned to the bucket length
thresholds.  Traces are inserted by walking their return states and recording the
residual at every visited node (Phase 3; App. B.1).  A lookup walks the observed
returns; an unseen node backs off to its parent (Phase 2).

Readings: a root above every prompt (depth -1) collects all traces and answers for an
unseen prompt; bin k holds residuals in [edge[k-1], edge[k]) with edge[-1] = 0 and the
last bin open-ended; probabilities are count / total of the node.

Routing (Phase 2): B* = argmin over buckets B of sum_k p_k Tdec(B, k) + C_mig(B_cur, B),
C_mig(B, B) = 0; ties go to the lowest bucket index.
"""
from __future__ import annotations

import bisect


class PrefixTreeRef:
    def __init__(self, bin_edges):
        self.edges = [int(e) for e in bin_edges]
        self.counts = {}           # key -> list of counts; key () is the root

    def _bin(self, residual: int) -> int:
        return bisect.bisect_right(self.edges, int(residual))

    def _record(self, key, residual):
        c = self.counts.setdefault(key, [0] * (len(self.edges) + 1))
        c[self._bin(residual)] += 1

    def insert(self, prompt_id, states, residual):
        self._record((), residual[0])
        key = (int(prompt_id), ())
        self._record(key, residual[0])
        for k, s in enumerate(states):
            key = (int(prompt_id), tuple(int(x) for x in states[:k + 1]))
            self._record(key, residual[k + 1])

    def lookup(self, prompt_id, states):
        """(probabilities, depth) of the deepest existing node on the path."""
        if () not in self.counts:
            raise ValueError("empty tree")
        key, depth = (), -1
        if (int(prompt_id), ()) in self.counts:
            key, depth = (int(prompt_id), ()), 0
            for k in range(len(states)):
                nxt = (int(prompt_id), tuple(int(x) for x in states[:k + 1]))
                if nxt not in self.counts:
                    break
                key, depth = nxt, k + 1
        c = self.counts[key]
        total = sum(c)
        return [x / total for x in c], depth


def route_ref(hist, t_dec, c_mig, current):
    """(best bucket, cost) of the argmin rule."""
    best, best_cost = None, None
    for b in range(len(t_dec)):
        cost = 0.0
        for k in range(len(hist)):
            cost += hist[k] * t_dec[b][k]
        if b != current:
            cost += c_mig[current][b]
        if best is None or cost < best_cost:
            best, best_cost = b, cost
    return best, best_cost
