"""vTime fair scheduler (two-layer, with vTime lift) -- test infrastructure only.

The control-plane algorithm that decides which tenant's model-function
invocation (e.g. one denoising step) runs next on an idle executor
(Sec. 6 "Ensure Fairness in Multi-tenant Serving", Alg. 1).  Readings for what
the paper leaves open:

* vTime: a tenant is charged the estimated execution time at dispatch and the
  difference (measured - estimated) when the invocation completes;
* Active tenants are those with ready or running invocations; a tenant with
  ready work that was not active (new, or back after having none) is lifted
  to the minimum vTime of the tenants that are active; with no other active
  tenant its vTime is kept;
* Layer 1: R = tenants with ready invocations, C = {u in R : v_u - min_R v <= Delta};
* Layer 2: over the ready invocations N of tenants in C, the waiting time
  w = now - ready time, the remaining critical-path time r and the estimated
  execution time e are each divided by their maximum over N (0 when that
  maximum is 0); score = w^ - r^ - e^; the highest score wins, ties to the
  earlier ready time, then the smaller invocation id.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple


@dataclasses.dataclass
class Invocation:
    fn_id: int
    tenant: int
    est: float          # estimated execution time (the dispatch charge)
    remaining: float    # remaining critical-path time of its workflow
    ready_at: float


class VTimeScheduler:
    def __init__(self, delta: float):
        self.delta = float(delta)
        self.v: Dict[int, float] = {}
        self.active: Dict[int, bool] = {}
        self.ready: List[Invocation] = []
        self.running: Dict[int, Invocation] = {}

    def submit(self, tenant, fn_id, est, remaining, now):
        """An invocation becomes ready (its predecessors finished)."""
        self.v.setdefault(tenant, 0.0)
        self.active.setdefault(tenant, False)
        self.ready.append(Invocation(fn_id, tenant, float(est), float(remaining), float(now)))

    def _has_work(self, u):
        return any(n.tenant == u for n in self.ready) or \
            any(n.tenant == u for n in self.running.values())

    def schedule(self, now) -> Optional[Tuple[int, int, float]]:
        """Pick the next invocation (Alg. 1 Schedule); returns (fn_id, tenant,
        charged estimate) or None when nothing is ready."""
        if not self.ready:
            return None
        tenants_ready = sorted({n.tenant for n in self.ready})
        # vTime lift for new / returning tenants
        active_before = [u for u, a in self.active.items() if a]
        for u in tenants_ready:
            if not self.active[u]:
                if active_before:
                    self.v[u] = min(self.v[x] for x in active_before)
                self.active[u] = True
        # Layer 1: fairness filter
        vmin = min(self.v[u] for u in tenants_ready)
        cand = {u for u in tenants_ready if self.v[u] - vmin <= self.delta}
        # Layer 2: normalised priority score
        N = [n for n in self.ready if n.tenant in cand]
        wmax = max(now - n.ready_at for n in N)
        rmax = max(n.remaining for n in N)
        emax = max(n.est for n in N)

        def norm(x, m):
            return x / m if m > 0 else 0.0

        def key(n):
            s = norm(now - n.ready_at, wmax) - norm(n.remaining, rmax) - norm(n.est, emax)
            return (-s, n.ready_at, n.fn_id)

        best = min(N, key=key)
        self.ready.remove(best)
        self.running[best.fn_id] = best
        self.v[best.tenant] += best.est
        return best.fn_id, best.tenant, best.est

    def complete(self, fn_id, measured):
        """Alg. 1 OnComplete: replace the estimate by the measured time."""
        n = self.running.pop(fn_id)
        self.v[n.tenant] += float(measured) - n.est
        if not self._has_work(n.tenant):
            self.active[n.tenant] = False
