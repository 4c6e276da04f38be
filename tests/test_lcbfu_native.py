"""The native LCBFU maintainer (host C++ behind the C ABI; no GPU) against the
oracle's maintainer (Sec. 5.4): identical insert plans (entry ids, pool states,
row moves, kept rows, table updates), tables, row maps and access counts after
every operation of random request streams, plus its argument checks."""
import numpy as np
import pytest

from oracle.lcbfu import LCBFU


def _same_state(nat, ora):
    table, rows, counts = nat.export()
    assert rows.tolist() == ora.rows
    want = np.full_like(table, -1)
    want_counts = np.zeros_like(counts)
    for (e, s), st in ora.states.items():
        want[e, s] = st["pool"]
        want_counts[st["pool"]] = st["f"]
    np.testing.assert_array_equal(table, want)
    np.testing.assert_array_equal(counts, want_counts)
    info = nat.info()
    assert info["states"] == len(ora.states) and info["evicted"] == ora.evicted
    assert info["dropped"] == ora.dropped and info["stored"] == ora.seq


def _same_plan(p, q, S):
    assert p["entries"].tolist() == q["entries"]
    assert p["pools"].tolist() == q["pools"]
    assert list(zip(p["move_src"].tolist(), p["move_dst"].tolist())) == q["moves"]
    assert p["kept"] == q["kept"]
    assert p["upd"][:, 0].tolist() == q["touched"]


@pytest.mark.parametrize("slot_k,cap,seed", [([5, 10, 15, 20, 25], 60, 0),
                                             ([5, 10, 15, 20, 25], 61, 1),
                                             ([25, 5, 15], 20, 2),
                                             ([7], 9, 3),
                                             ([5, 10, 15, 20, 25], 500, 4)])
def test_native_matches_oracle_on_random_streams(slot_k, cap, seed):
    import paper_2312_04429_amd as P
    S = len(slot_k)
    ecap = cap + 3
    nat = P.NvLCBFU(slot_k, cap, ecap)
    ora = LCBFU(slot_k, cap, ecap)
    rng = np.random.default_rng(seed)
    ks_all = [0] + sorted(slot_k) + [max(slot_k) + 5]
    steps = 400 if cap < 100 else 1500
    for step in range(steps):
        if ora.rows and rng.random() < 0.65:
            b = int(rng.integers(1, 9))
            rows = rng.integers(0, len(ora.rows), size=b)
            ks = [ora.choose_k(int(r), int(rng.choice(ks_all))) for r in rows]
            nat.access(rows, ks)
            ora.access([int(r) for r in rows], ks)
        else:
            m = int(rng.integers(1, max(2, min(4, cap // S) + 1)))
            p = nat.insert(m)
            q = ora.insert(m)
            _same_plan(p, q, S)
            table = nat.export()[0]
            for rec in p["upd"]:
                assert rec[1:].tolist() == table[rec[0]].tolist()
        if step % 7 == 0 or step == steps - 1:
            _same_state(nat, ora)
    _same_state(nat, ora)
    assert ora.evicted > 0 and ora.dropped > 0


def test_paper_example_through_the_native_maintainer():
    """Sec. 5.4's scores: K = 25 used 100 times (2500) outlives K = 5 used 200 times (1000)."""
    import paper_2312_04429_amd as P
    c = P.NvLCBFU([5, 25], 4, 8)
    c.insert(2)
    c.access([1] * 199, [5] * 199)       # e1 K=5 -> f 200
    c.access([0] * 99, [25] * 99)        # e0 K=25 -> f 100
    c.access([0] * 399, [5] * 399)       # e0 K=5 -> 2000
    c.access([1] * 89, [25] * 89)        # e1 K=25 -> 2250
    table, _, counts = c.export()
    assert counts[table[1, 0]] * 5 == 1000 and counts[table[0, 1]] * 25 == 2500
    c.insert(1)
    table, rows, _ = c.export()
    assert table[1, 0] == -1 and table[0, 0] == -1 and table[0, 1] >= 0 and table[1, 1] >= 0


def test_native_argument_checks():
    import paper_2312_04429_amd as P
    from paper_2312_04429_amd import _native as N
    for args in [([5, 5], 10, 10), ([0, 5], 10, 10), ([5], 10, 9), ([5], 0, 0),
                 (list(range(1, 18)), 100, 100)]:
        with pytest.raises(N.NvError):
            P.NvLCBFU(*args)
    c = P.NvLCBFU([5, 10], 6, 6)
    with pytest.raises(N.NvError):
        c.insert(4)                      # 8 states > 6
    c.insert(1)
    with pytest.raises(N.NvError):
        c.access([1], [5])               # row out of range
    with pytest.raises(N.NvError):
        c.access([0], [7])               # not a slot's K
    before = c.export()[2].copy()
    with pytest.raises(N.NvError):
        c.access([0, 0], [5, 15])        # second one invalid: nothing applied
    np.testing.assert_array_equal(c.export()[2], before)
    c.access([0, 0], [0, -1])            # K <= 0: no state served
    np.testing.assert_array_equal(c.export()[2], before)
