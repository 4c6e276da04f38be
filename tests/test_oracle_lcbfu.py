"""Pins of the oracle's LCBFU maintainer and hole handling (Sec. 5.4).

Checked against the section's worked score example (tests/golden/lcbfu_example.txt),
hand-built states whose eviction order, holes and row compaction are worked out by
hand, and invariants of the policy (the state limit, exactly |K-set| evictions per
prompt at the limit, every evicted score <= every surviving score) on random streams
with an independent sort-based statement of the eviction set.
"""
import os

import numpy as np
import pytest

from oracle.lcbfu import LCBFU

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
K5 = [5, 10, 15, 20, 25]


def _use(c, entry, slot, times):
    row = c.rows.index(entry)
    c.access([row] * times, [c.slot_k[slot]] * times)


def _golden_example():
    out = []
    for line in open(os.path.join(GOLDEN, "lcbfu_example.txt")):
        if line.strip() and not line.startswith("#"):
            k, f, s = (int(v) for v in line.split())
            out.append((k, f, s))
    return out


def test_paper_score_example():
    """The K = 25 state used 100 times outranks the K = 5 state used 200 times."""
    ex = _golden_example()
    c = LCBFU([5, 25], state_capacity=4, entry_capacity=8)
    c.insert(2)                                   # e0, e1: f = 1 each
    (k_lo, f_lo, s_lo), (k_hi, f_hi, s_hi) = ex
    _use(c, 1, c.slot_k.index(k_lo), f_lo - 1)    # e1 K=5: 200 uses
    _use(c, 0, c.slot_k.index(k_hi), f_hi - 1)    # e0 K=25: 100 uses
    _use(c, 0, 0, 399)                            # e0 K=5: 400 uses -> 2000
    _use(c, 1, 1, 89)                             # e1 K=25: 90 uses -> 2250
    assert c.score((1, 0)) == s_lo and c.score((0, 1)) == s_hi
    c.insert(1)                                   # full: two evictions
    assert (1, 0) not in c.states and (0, 0) not in c.states   # 1000 then 2000 go
    assert (0, 1) in c.states and (1, 1) in c.states
    assert c.evicted == 2


def test_score_is_product_not_count_or_k():
    """K = 25 used once (25) goes before K = 5 used 10 times (50): neither the count
    alone (LFU) nor K alone would order them this way."""
    c = LCBFU([5, 25], state_capacity=4, entry_capacity=8)
    c.insert(2)
    _use(c, 0, 0, 9)       # e0 K=5: f 10 -> 50
    _use(c, 1, 0, 9)       # e1 K=5: f 10 -> 50
    _use(c, 1, 1, 4)       # e1 K=25: f 5 -> 125; e0 K=25 stays 25
    c.insert(1)            # evicts e0 K=25 (25), then the first-stored 50: e0 K=5
    # e0 lost every state: dropped from the vector DB (e1 moves to row 0), and the
    # new prompt reuses id 0 with fresh counts
    assert c.dropped == 1 and c.rows == [1, 0]
    assert set(c.states) == {(1, 0), (1, 1), (0, 0), (0, 1)}
    assert c.states[(0, 0)]["f"] == 1 and c.states[(0, 0)]["seq"] == 4


def test_no_eviction_below_limit_then_exactly_k_set_per_prompt():
    c = LCBFU(K5, state_capacity=20, entry_capacity=20)
    for i in range(4):
        c.insert(1)
        assert c.evicted == 0 and len(c.states) == 5 * (i + 1)
    for i in range(6):
        before = c.evicted
        c.insert(1)
        assert c.evicted - before == 5 and len(c.states) == 20


def test_partial_fill_evicts_only_the_overflow():
    c = LCBFU([5, 10, 15], state_capacity=7, entry_capacity=10)
    c.insert(2)                                # 6 states
    c.insert(1)                                # 9 > 7: two evictions
    assert c.evicted == 2 and len(c.states) == 7
    c.insert(1)
    assert c.evicted == 5 and len(c.states) == 7


def test_new_state_score_is_its_k_and_ties_go_to_the_oldest():
    c = LCBFU([5, 10], state_capacity=4, entry_capacity=8)
    c.insert(2)
    assert [c.score((0, s)) for s in range(2)] == [5, 10]
    c.insert(1)              # evicts e0 K=5 then e1 K=5 (both 5, e0 stored first)
    assert set(c.states) == {(0, 1), (1, 1), (2, 0), (2, 1)}


def test_batch_evicts_before_storing():
    """A batch never evicts its own new states, even though they score lowest."""
    c = LCBFU([5, 10], state_capacity=6, entry_capacity=8)
    c.insert(3)
    for e in range(3):
        _use(c, e, 0, 50)
        _use(c, e, 1, 50)
    plan = c.insert(2)        # 4 evictions: the three K=5 states (255), then e0 K=10
    assert c.evicted == 4 and c.dropped == 1
    assert plan["entries"] == [0, 3]          # e0's id is free again, then 3
    assert all(c.states[(e, s)]["f"] == 1 for e in (0, 3) for s in range(2))
    assert set(c.states) - {(0, 0), (0, 1), (3, 0), (3, 1)} == {(1, 1), (2, 1)}


def test_hole_choice_by_hand():
    c = LCBFU(K5, state_capacity=10, entry_capacity=10)
    c.insert(2)
    for s in (1, 3):                      # e0 keeps K = 5, 15, 25
        c.free_pool.add(c.states.pop((0, s))["pool"])
    for s in range(4):                    # e1 keeps K = 25 only
        c.free_pool.add(c.states.pop((1, s))["pool"])
    want0 = {0: 0, 4: 0, 5: 5, 9: 5, 10: 5, 14: 5, 15: 15, 20: 15, 24: 15, 25: 25, 50: 25}
    for k, kp in want0.items():
        assert c.choose_k(0, k) == kp, k
    for k, kp in {5: 0, 20: 0, 24: 0, 25: 25}.items():
        assert c.choose_k(1, k) == kp, k
    assert c.choose_k(-1, 25) == 0


def test_row_compaction_by_hand():
    """Rows [e0 e1 e2 e3 e4]; e1 and e4 lose their last state: e3 (the one live row
    at or past the new count 3) fills row 1; rows become [e0 e3 e2], then the
    new prompt takes the lowest free id (1) at row 3."""
    c = LCBFU([5], state_capacity=5, entry_capacity=8)
    c.insert(5)
    for e in (0, 2, 3):
        _use(c, e, 0, 3)
    plan = c.insert(2)      # evicts e1 then e4 (score 5, seq order)
    assert plan["moves"] == [(3, 1)] and plan["kept"] == 3
    assert c.rows == [0, 3, 2, 1, 4]
    assert plan["entries"] == [1, 4]


def test_access_counts_only_the_served_state():
    c = LCBFU(K5, state_capacity=10, entry_capacity=10)
    c.insert(2)
    c.access([1, 0, 1], [15, 0, 15])
    assert c.states[(1, 2)]["f"] == 3
    assert all(c.states[(e, s)]["f"] == 1 for e in range(2) for s in range(5)
               if (e, s) != (1, 2))


def test_errors():
    with pytest.raises(ValueError):
        LCBFU([5, 5], 10, 10)
    with pytest.raises(ValueError):
        LCBFU([0, 5], 10, 10)
    with pytest.raises(ValueError):
        LCBFU([5, 10], 10, 9)
    c = LCBFU(K5, state_capacity=9, entry_capacity=9)
    with pytest.raises(ValueError):
        c.insert(2)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_random_stream_invariants(seed):
    """Random accesses and inserts: the limit holds, the evicted set is the `need`
    smallest (score, age) states of a snapshot (sorted independently), every
    evicted score <= every kept score, and rows / table / free lists stay coherent."""
    rng = np.random.default_rng(seed)
    c = LCBFU(K5, state_capacity=60, entry_capacity=64)
    for step in range(120):
        if c.rows and rng.random() < 0.6:
            b = int(rng.integers(1, 4))
            rows = rng.integers(0, len(c.rows), size=b)
            ks = [c.choose_k(int(r), int(rng.choice([0, 5, 10, 15, 20, 25, 30])))
                  for r in rows]
            c.access([int(r) for r in rows], ks)
            continue
        m = int(rng.integers(1, 4))
        # states are named by their sequence number: entry ids are reused
        snap = {v["seq"]: c.score(k) for k, v in c.states.items()}
        need = max(0, len(snap) + 5 * m - 60)
        want = set(sorted(snap, key=lambda q: (snap[q], q))[:need])
        c.insert(m)
        gone = set(snap) - {v["seq"] for v in c.states.values()}
        assert gone == want
        if gone and set(snap) - gone:
            assert max(snap[q] for q in gone) <= min(snap[q] for q in set(snap) - gone)
        assert len(c.states) <= 60
        live = {e for e, _ in c.states}
        assert sorted(c.rows) == sorted(live) and len(set(c.rows)) == len(c.rows)
        used = {v["pool"] for v in c.states.values()}
        assert len(used) == len(c.states) and not used & c.free_pool
        assert len(used) + len(c.free_pool) == 60
        assert not live & c.free_entries and len(live) + len(c.free_entries) == 64


def test_two_row_compaction_and_lowest_first_reuse_by_hand():
    """Rows [e0 .. e6], one state each; e0 and e2 are evicted: the new count is 5,
    rows 5 and 6 (e5, e6) fill rows 0 and 2 in that order, and the two new prompts
    take ids 0, 2 and pool slots 0, 2 (lowest free first)."""
    c = LCBFU([5], state_capacity=7, entry_capacity=8)
    first = c.insert(7)
    assert first["pools"] == [[p] for p in range(7)]
    for e in (1, 3, 4, 5, 6):
        _use(c, e, 0, 2)
    plan = c.insert(2)
    assert plan["moves"] == [(5, 0), (6, 2)] and plan["kept"] == 5
    assert c.rows == [5, 1, 6, 3, 4, 0, 2]
    assert plan["entries"] == [0, 2] and plan["pools"] == [[0], [2]]
    assert plan["touched"] == [0, 2]
