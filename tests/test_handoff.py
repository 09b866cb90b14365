"""The aligned batch handoff (hs_handoff_*; §5.2 "Aligned Batch Handoff"):
host logic, run on the CPU.  Batches of B_align requests in arrival order, an
under-filled batch after the timeout, a row budget for packed prefill, and a
brute-force comparison with a plain model of the rule."""
from __future__ import annotations

import random

import pytest


def _hs():
    import paper_2603_12707_amd as hs
    return hs


def test_full_batch_of_align_requests_goes_at_once():
    hs = _hs()
    h = hs.Handoff(align=32, timeout_ms=500.0)
    for r in range(31):
        h.push(r, 600, now_ms=float(r))
    assert h.pop(40.0) == ([], 0, pytest.approx(460.0))  # 31 wait; the oldest has 460 ms left
    h.push(31, 600, now_ms=41.0)
    batch, rows, wait = h.pop(41.0)
    assert batch == list(range(32)) and rows == 32 * 600 and wait == -1
    assert h.pending() == 0


def test_underfilled_batch_goes_after_the_timeout():
    hs = _hs()
    h = hs.Handoff(align=32, timeout_ms=500.0)
    for r, t in [(7, 0.0), (3, 100.0), (9, 250.0)]:
        h.push(r, 10 + r, now_ms=t)
    assert h.pop(499.9)[0] == []
    batch, rows, _ = h.pop(500.0)
    assert batch == [7, 3, 9] and rows == 17 + 13 + 19


def test_more_than_align_waiting_leaves_the_rest_in_order():
    hs = _hs()
    h = hs.Handoff(align=4, timeout_ms=1000.0)
    for r in range(10):
        h.push(100 + r, 1, now_ms=0.0)
    assert h.pop(1.0)[0] == [100, 101, 102, 103]
    b, _, wait = h.pop(1.0)
    assert b == [104, 105, 106, 107] and wait == 999.0  # 2 left, their timeout 999 ms away
    assert h.pop(1.0)[0] == [] and h.pending() == 2
    assert h.pop(1000.0)[0] == [108, 109]


def test_row_budget_closes_a_batch_early():
    hs = _hs()
    h = hs.Handoff(align=32, max_rows=2000, timeout_ms=500.0)
    for r, rows in enumerate([700, 800, 600, 100]):
        h.push(r, rows, now_ms=0.0)
    batch, rows, wait = h.pop(0.0)                   # 700 + 800 fit, + 600 does not: the budget closes the batch
    assert batch == [0, 1] and rows == 1500 and wait == 500.0
    assert h.pop(0.0)[0] == []                       # 600 + 100 fit and more could follow: not due
    assert h.pop(500.0) == ([2, 3], 700, -1)
    big = hs.Handoff(align=8, max_rows=100, timeout_ms=500.0)
    big.push(1, 5000, now_ms=0.0)                    # a request above the budget still goes, alone
    big.push(2, 10, now_ms=0.0)
    assert big.pop(0.0)[0] == [1]


def test_errors():
    hs = _hs()
    for args in [(0, 0, 8, 500.0), (4, -1, 8, 500.0), (4, 0, 3, 500.0), (4, 0, 8, -1.0), (4, 0, 8, float("nan"))]:
        with pytest.raises(hs.HsError) as e:
            hs.Handoff(*args)
        assert e.value.code == hs.HS_E_INVALID
    h = hs.Handoff(align=2, max_pending=3, timeout_ms=500.0)
    with pytest.raises(hs.HsError) as e:
        h.push(-1, 5, now_ms=0.0)
    assert e.value.code == hs.HS_E_INVALID
    with pytest.raises(hs.HsError) as e:
        h.push(1, 0, now_ms=0.0)
    assert e.value.code == hs.HS_E_INVALID
    h.push(1, 5, now_ms=10.0)
    with pytest.raises(hs.HsError) as e:
        h.push(2, 5, now_ms=9.0)                     # time runs backwards
    assert e.value.code == hs.HS_E_INVALID
    h.push(2, 5, now_ms=10.0)
    h.push(3, 5, now_ms=11.0)
    with pytest.raises(hs.HsError) as e:
        h.push(4, 5, now_ms=12.0)                    # max_pending waiting
    assert e.value.code == hs.HS_E_CAPACITY


def _model_pop(queue, now, align, max_rows, timeout):
    """The rule written out: the longest arrival-order prefix of at most align
    requests within the row budget (one request always), due when it is full
    by count, closed by the budget with more waiting, or timed out."""
    k, rows, full = 0, 0, False
    for req, r, t in queue:
        if k == align:
            break
        if k > 0 and max_rows > 0 and rows + r > max_rows:
            full = True
            break
        rows += r
        k += 1
    if not queue or not (k == align or full or now - queue[0][2] >= timeout):
        return [], 0
    out = [q[0] for q in queue[:k]]
    del queue[:k]
    return out, rows


@pytest.mark.parametrize("seed", range(6))
def test_random_arrivals_match_the_rule(seed):
    hs = _hs()
    rng = random.Random(seed)
    align, max_rows, timeout = rng.choice([1, 3, 8, 32]), rng.choice([0, 900, 5000]), rng.choice([0.0, 50.0, 500.0])
    h = hs.Handoff(align=align, max_rows=max_rows, max_pending=100000, timeout_ms=timeout)
    queue, now, nxt = [], 0.0, 0
    for _ in range(400):
        now += rng.choice([0.0, 0.5, 3.0, 40.0])
        if rng.random() < 0.6:
            rows = rng.randint(1, 1500)
            h.push(nxt, rows, now_ms=now)
            queue.append((nxt, rows, now))
            nxt += 1
        else:
            got, got_rows, _ = h.pop(now)
            want, want_rows = _model_pop(queue, now, align, max_rows, timeout)
            assert (got, got_rows) == (want, want_rows)
    assert h.pending() == len(queue)
