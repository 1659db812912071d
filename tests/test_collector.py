"""The C-ABI collector (jn_collector_*) against the batching oracle: same
released batches (ids and poll times) on random arrival traces, bit-exact;
error statuses leave the queue untouched.  Host only."""
import random

import pytest

from oracle import batching as B


@pytest.fixture(scope="module")
def jn():
    import paper_2607_16074_amd as lib
    return lib


def run_c(jn, events, max_batch, timeout, cap=4096):
    c = jn.Collector(max_batch, timeout)
    out = []
    for ev in events:
        if ev[0] == "submit":
            _, rid, sig, d, n, t = ev
            c.submit(rid, sig, d, n, t)
        else:
            ids = c.poll(ev[1], cap)
            if ids:
                out.append((ev[1], ids))
    return out, c


def test_random_traces_match_oracle(jn):
    rng = random.Random(7)
    for trial in range(400):
        mb, to = rng.randint(1, 8), rng.choice([0, 3, 40, 10 ** 12])
        t, ev = 0, []
        for i in range(rng.randint(0, 40)):
            t += rng.choice([0, 0, 1, 5, 30])
            ev.append(("submit", 1000 + i, rng.choice([11, 11, 11, 12, 2 ** 63 + 5]), rng.choice([768, 768, 2048]),
                       rng.randint(1, 5), t))
            if rng.random() < 0.5:
                ev.append(("poll", t + rng.randint(0, 50)))
                t = max(t, ev[-1][1])
        ev += [("poll", t + 10 ** 13)] * 45
        got, _ = run_c(jn, ev, mb, to)
        assert got == B.simulate(ev, mb, to), trial


def test_status_deadline(jn):
    c = jn.Collector(4, 100)
    assert c.status() == (0, -1)
    c.submit(1, 5, 64, 1, 10)
    assert c.status() == (1, 110)          # waits for its timeout
    c.submit(2, 6, 64, 1, 20)
    assert c.status() == (2, 10)           # blocked by an incompatible request: ready now
    assert c.poll(11) == [1]
    assert c.status() == (1, 120)


def test_errors_leave_queue_untouched(jn):
    with pytest.raises(jn.JNError):
        jn.Collector(0, 10)
    with pytest.raises(jn.JNError):
        jn.Collector(4, -1)
    c = jn.Collector(8, 0)
    c.submit(1, 5, 64, 2, 100)
    with pytest.raises(jn.JNError):
        c.submit(2, 5, 64, 1, 99)          # arrival before the last queued one
    with pytest.raises(jn.JNError):
        c.submit(2, 5, 64, 0, 100)         # no samples
    c.submit(2, 5, 64, 1, 100)
    c.submit(3, 5, 64, 1, 100)
    with pytest.raises(jn.JNError) as e:
        c.poll(100, cap=2)                 # ready batch has 3 requests
    assert "ENOSPACE" in str(e.value)
    assert c.status()[0] == 3
    assert c.poll(100, cap=3) == [1, 2, 3]
