"""Pins for the paged-KV bookkeeping model (lowest-free-id reading) by brute force."""
import random

import pytest

from oracle.pages import OutOfPages, PagePool


def _brute_lowest(used, n):
    return min(set(range(n)) - used)


def test_lowest_free_id_under_random_interleaving():
    rng = random.Random(0)
    n = 64
    pool = PagePool(n)
    used = set()
    live = []
    for step in range(3000):
        op = rng.random()
        if op < 0.15 and len(live) < 8:
            seq = step
            length = rng.randint(0, 40)
            need = -(-length // 16)
            if need <= n - len(used):
                expect = sorted(set(range(n)) - used)[:need]
                pool.add_seq(seq, length)
                assert pool.tables[seq] == expect
                used |= set(expect)
                live.append(seq)
        elif op < 0.8 and live:
            seq = rng.choice(live)
            L = pool.lens[seq]
            if L % 16 == 0 and len(used) < n:
                expect = _brute_lowest(used, n)
                pool.append(seq, 1)
                assert pool.tables[seq][-1] == expect
                used.add(expect)
            elif L % 16 != 0:
                before = list(pool.tables[seq])
                pool.append(seq, 1)
                assert pool.tables[seq] == before
        elif op < 0.9 and live:
            seq = rng.choice(live)
            cut = rng.randint(0, pool.lens[seq])
            keep = -(-cut // 16)
            used -= set(pool.tables[seq][keep:])
            pool.truncate(seq, cut)
        elif live:
            seq = live.pop(rng.randrange(len(live)))
            used -= set(pool.tables[seq])
            pool.free_seq(seq)
        assert sorted(pool.free) == sorted(set(range(n)) - used)


def test_probe_scratch_restores_tables_bit_exact():
    pool = PagePool(100)
    pool.add_seq(0, 4096 // 64)
    pool.add_seq(1, 33)
    pool.append(0, 5)
    snap_tables = {k: list(v) for k, v in pool.tables.items()}
    snap_free = sorted(pool.free)
    L = pool.lens[1]
    pool.append(1, 8 + 4 - 1)  # suffix S=8 plus T-1=3 fed-back trial tokens
    assert len(pool.tables[1]) == -(-(L + 11) // 16)
    pool.truncate(1, L)
    assert pool.tables == snap_tables and sorted(pool.free) == snap_free and pool.lens[1] == L


def test_exhaustion_is_all_or_nothing():
    pool = PagePool(4)
    pool.add_seq(0, 40)  # 3 pages
    snap = ({k: list(v) for k, v in pool.tables.items()}, sorted(pool.free), dict(pool.lens))
    with pytest.raises(OutOfPages):
        pool.add_seq(1, 20)  # needs 2
    with pytest.raises(OutOfPages):
        pool.append(0, 30)  # needs 2 more
    assert ({k: list(v) for k, v in pool.tables.items()}, sorted(pool.free), dict(pool.lens)) == snap


def test_fork_shares_full_pages_and_copies_the_partial_one():
    # hand-derived: a 37-token request holds pages [0, 1, 2]; its fork shares 0 and 1 and
    # copies page 2 into the lowest free page, 3
    pool = PagePool(8)
    pool.add_seq(0, 37)
    assert pool.fork(0, 1) == (2, 3)
    assert pool.tables[1] == [0, 1, 3] and pool.lens[1] == 37
    # the request's next token lands in its own page 2, the fork's in its copy
    pool.append(0, 1)
    pool.append(1, 12)  # 37 + 12 = 49 crosses a page boundary: takes page 4
    assert pool.tables[0] == [0, 1, 2] and pool.tables[1] == [0, 1, 3, 4]
    # freeing the fork returns only its private pages; shared ones stay with the request
    pool.free_seq(1)
    assert sorted(pool.free) == [3, 4, 5, 6, 7] and pool.tables[0] == [0, 1, 2]
    # a request ending on a page boundary forks without a copy
    pool.add_seq(2, 32)
    assert pool.fork(2, 3) is None and pool.tables[3] == pool.tables[2]
    # a shared page is freed only when its last holder lets go
    pool.free_seq(2)
    assert set(pool.tables[3]).isdisjoint(pool.free)
    pool.free_seq(3)
    assert sorted(pool.free) == [3, 4, 5, 6, 7]


def test_truncation_may_not_end_inside_a_shared_page():
    pool = PagePool(8)
    pool.add_seq(0, 40)
    pool.fork(0, 1)
    with pytest.raises(ValueError):
        pool.truncate(0, 20)  # page 1 (positions 16..31) is shared with the fork
    pool.truncate(0, 32)  # a page boundary is fine
    assert pool.tables[0] == [0, 1] and pool.tables[1][:2] == [0, 1]


def test_fork_refcounts_under_random_interleaving():
    # brute force: a page is free exactly when no table holds it
    rng = random.Random(5)
    n = 40
    pool = PagePool(n)
    live = []
    for step in range(4000):
        op = rng.random()
        try:
            if op < 0.1 and len(live) < 10:
                seq = step
                pool.add_seq(seq, rng.randint(0, 50))
                live.append(seq)
            elif op < 0.2 and live and len(live) < 10:
                src = rng.choice(live)
                pool.fork(src, step)
                live.append(step)
            elif op < 0.75 and live:
                pool.append(rng.choice(live), rng.randint(1, 9))
            elif op < 0.88 and live:
                seq = rng.choice(live)
                try:
                    pool.truncate(seq, rng.randint(0, pool.lens[seq]))
                except ValueError:
                    pass
            elif live:
                pool.free_seq(live.pop(rng.randrange(len(live))))
        except OutOfPages:
            pass
        held = [p for t in pool.tables.values() for p in t]
        assert sorted(set(held) | set(pool.free)) == list(range(n))
        assert set(held).isdisjoint(pool.free)
        for p in set(held):
            assert pool.refs[p] == held.count(p)
