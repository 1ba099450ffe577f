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
