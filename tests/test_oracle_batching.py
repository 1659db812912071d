"""Pins of the inference-queue batching oracle (App. A.3): brute force over
every prefix, structural properties of released batches, closed-form traces."""
import itertools
import random

from oracle import batching as B


def brute_prefix(queue, max_batch):
    """Largest k such that queue[:k] satisfies the rule, by trying every k."""
    best = 0
    for k in range(1, len(queue) + 1):
        head = queue[0]
        ok = all((q[1], q[2]) == (head[1], head[2]) for q in queue[:k])
        size = sum(q[3] for q in queue[:k])
        if ok and (k == 1 or size <= max_batch):
            best = k
    if best == 0:
        return 0, False
    size = sum(q[3] for q in queue[:best])
    can_grow = best < len(queue)  # a longer prefix would have been accepted above
    final = size >= max_batch or can_grow
    return best, final


def test_prefix_matches_brute_force():
    rng = random.Random(0)
    for _ in range(3000):
        n = rng.randint(0, 7)
        queue = [(i, rng.choice([1, 2]), rng.choice([64, 64, 128]), rng.randint(1, 4), i) for i in range(n)]
        mb = rng.randint(1, 8)
        assert B.current_prefix(queue, mb) == brute_prefix(queue, mb), (queue, mb)


def test_hand_trace():
    # 1, 2 share the interface, 3 does not: {1, 2} is final at once; {3} is
    # final once 4 (another interface) arrives; {4} alone waits for its timeout
    ev = [("submit", 1, 7, 128, 1, 0), ("submit", 2, 7, 128, 2, 10), ("submit", 3, 9, 128, 1, 20),
          ("poll", 15), ("submit", 4, 7, 128, 1, 30), ("poll", 31), ("poll", 129), ("poll", 130)]
    assert B.simulate(ev, max_batch=4, timeout=100) == [(15, [1, 2]), (31, [3]), (130, [4])]


def test_full_batches_of_unit_requests():
    # one interface, one sample per request, no timeout pressure: batches of
    # exactly max_batch in arrival order
    ev = []
    for i in range(10):
        ev += [("submit", i, 5, 64, 1, i), ("poll", i)]
    out = B.simulate(ev, max_batch=4, timeout=10 ** 9)
    assert [ids for _, ids in out] == [[0, 1, 2, 3], [4, 5, 6, 7]]


def test_timeout_zero_releases_every_poll():
    ev = [("submit", 0, 1, 8, 2, 0), ("submit", 1, 1, 8, 1, 0), ("poll", 0), ("submit", 2, 1, 8, 1, 1), ("poll", 1)]
    assert B.simulate(ev, max_batch=100, timeout=0) == [(0, [0, 1]), (1, [2])]


def test_oversize_first_request_goes_alone():
    ev = [("submit", 0, 1, 8, 9, 0), ("submit", 1, 1, 8, 1, 0), ("poll", 0)]
    assert B.simulate(ev, max_batch=4, timeout=10 ** 9) == [(0, [0])]


def test_released_batches_properties():
    rng = random.Random(1)
    for trial in range(300):
        mb, to = rng.randint(1, 6), rng.choice([0, 5, 50, 10 ** 9])
        t, ev, meta = 0, [], {}
        for i in range(rng.randint(1, 25)):
            t += rng.randint(0, 10)
            sig = rng.choice([3, 3, 4])
            n = rng.randint(1, 3)
            meta[i] = (sig, n)
            ev.append(("submit", i, sig, 32, n, t))
            if rng.random() < 0.6:
                ev.append(("poll", t))
        ev += [("poll", t + 10 ** 10)] * 30  # late polls: every prefix has expired
        out = B.simulate(ev, mb, to)
        flat = list(itertools.chain.from_iterable(ids for _, ids in out))
        # FIFO: released ids are exactly the submitted ids in arrival order
        assert flat == sorted(meta)
        for _, ids in out:
            sigs = {meta[i][0] for i in ids}
            assert len(sigs) == 1  # compatible batch
            size = sum(meta[i][1] for i in ids)
            assert len(ids) == 1 or size <= mb
