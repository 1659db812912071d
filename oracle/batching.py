"""Inference-queue batching -- oracle (test infrastructure only).

App. A.3 "Inference Queue Composition": the scheduler looks at queued
requests in arrival order and forms the largest FIFO prefix that is
compatible at the shared frozen-prefix boundary and allowed by the batching
timeout and the maximum batch size; compatibility is a property of the
base-model interface, not of the tenant.

Readings (the paper names the rule, not its corner cases):
  * a prefix is contiguous from the oldest queued request -- a request that
    does not fit is never skipped, it waits for a later batch;
  * compatible = same prefix signature and same feature width as the oldest
    request of the prefix;
  * the maximum batch size counts samples; whole requests only; the oldest
    request is always taken, even when it alone exceeds the maximum;
  * the prefix is released as soon as it cannot grow any more (it is full,
    or the next queued request is incompatible or would overflow it), or
    once the oldest request has waited ``timeout`` (``now - arrival >=
    timeout``).

Written as plain loops over a list.
"""
from __future__ import annotations

from typing import List, Tuple


def current_prefix(queue: List[Tuple[int, int, int, int, int]], max_batch: int):
    """queue: [(id, sig, d, n_samples, arrival)] in arrival order.
    Returns (k, final): the first k requests form the prefix; final = it
    cannot grow any more."""
    if not queue:
        return 0, False
    head = queue[0]
    k, total = 0, 0
    for item in queue:
        if (item[1], item[2]) != (head[1], head[2]):
            return k, True
        if k > 0 and total + item[3] > max_batch:
            return k, True
        total += item[3]
        k += 1
        if total >= max_batch:
            return k, True
    return k, False


def simulate(events, max_batch: int, timeout: int):
    """Replay a trace of ("submit", id, sig, d, n, t) and ("poll", t) events.
    Returns the released batches as (poll time, [ids])."""
    queue: List[Tuple[int, int, int, int, int]] = []
    out = []
    for ev in events:
        if ev[0] == "submit":
            _, rid, sig, d, n, t = ev
            queue.append((rid, sig, d, n, t))
        else:
            t = ev[1]
            if not queue:
                continue
            k, final = current_prefix(queue, max_batch)
            if final or t - queue[0][4] >= timeout:
                out.append((t, [q[0] for q in queue[:k]]))
                queue = queue[k:]
    return out
