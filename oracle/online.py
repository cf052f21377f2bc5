"""Oracle of the online route compactor and its achieved share A.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).  Plain Python, one
global event loop over arrivals and deadline triggers, for the test sizes.

The runtime of Section 9 ("The next systems test") queues events by route and
deadline, launches a route only when its queue reaches the safe-suffix
threshold K_r, and sends to the CPU what a deadline or a capacity limit keeps
from batching.  The paper names the policy but does not fix it; the frozen
policy written here is:

* events arrive in release order (ties by event index) into a FIFO queue of
  their route; an event is released at t_i and must start on the device no
  later than d_i = t_i + delta; a launch at host time tau starts on the device
  at tau + L (L, the launch latency, at most delta);
* a queue's trigger is the latest launch time of its oldest event,
  t_oldest + delta - L.  Arrivals at or before a trigger are taken first.  At
  the trigger, a queue of at least K_r events is launched whole (every member
  has t_j <= tau, and its device start tau + L is within every member's
  deadline, the oldest's being the earliest); a shorter queue sends its
  oldest event to the CPU and the next oldest sets the new trigger;
* a queue that reaches its capacity C (C >= K_r) is launched at once, at the
  arrival time of the event that filled it; with C < K_r nothing ever
  launches, and an arrival that finds its queue full goes to the CPU;
* triggers of several routes at the same time are taken in route order
  (routes do not interact, so this fixes only the listing order).

z_i = 1 for every event of a launched batch and 0 for every event sent to
the CPU; A = sum z_i / |E| (Section 9, the achieved share) and the recovery
R_A = (A - F) / (P* - F) when P* > F (Eq. online-recovery).  Every launched
batch is feasible in the sense of Eq. feasible-batch, so A <= P*.
"""
from __future__ import annotations

from typing import Dict, List


def _k(k, r) -> int:
    return int(k[r]) if isinstance(k, (list, tuple, dict)) else int(k)


def online_compactor(t, r, K, delta: int, latency: int = 0, capacity=None):
    """Run the frozen policy.  Returns a dict: ``accelerated`` (sum of z),
    ``fallback_deadline``, ``fallback_capacity``, ``batches`` (a list of
    (route, launch time, [event indices in release order]) in launch order),
    ``z`` (per event, 0 or 1)."""
    assert 0 <= latency <= delta
    n = len(t)
    order = sorted(range(n), key=lambda i: (int(t[i]), i))
    cap = float("inf") if capacity is None else int(capacity)
    queues: Dict[int, List[int]] = {}
    z = [0] * n
    batches = []
    fb_deadline = fb_capacity = 0
    p = 0
    while True:
        trig = None
        for rr in sorted(queues):
            q = queues[rr]
            if q:
                tau = int(t[q[0]]) + delta - latency
                if trig is None or tau < trig[0]:
                    trig = (tau, rr)
        if p < n and (trig is None or int(t[order[p]]) <= trig[0]):
            i = order[p]
            p += 1
            rr = int(r[i])
            q = queues.setdefault(rr, [])
            if len(q) >= cap:
                fb_capacity += 1
                continue
            q.append(i)
            if len(q) == cap and cap >= _k(K, rr):
                batches.append((rr, int(t[i]), list(q)))
                for j in q:
                    z[j] = 1
                queues[rr] = []
        elif trig is not None:
            tau, rr = trig
            q = queues[rr]
            if len(q) >= _k(K, rr):
                batches.append((rr, tau, list(q)))
                for j in q:
                    z[j] = 1
                queues[rr] = []
            else:
                q.pop(0)
                fb_deadline += 1
        else:
            break
    return {"accelerated": sum(z), "fallback_deadline": fb_deadline,
            "fallback_capacity": fb_capacity, "batches": batches, "z": z}


def recovery(a: int, f: int, p_star: int):
    """R_A = (A - F) / (P* - F) (Eq. online-recovery); None when P* = F."""
    return None if p_star == f else (a - f) / (p_star - f)
