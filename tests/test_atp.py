"""ATP cue detection: the oracle's bitmap pinned by hand and by brute force, and the C ABI's
bitmap builder checked against it (CPU).  The device match runs in test_gpu_5_atp_conclusion."""
import random

import numpy as np
import pytest

from oracle import atp as A
from paper_2606_31580_amd import laser as L


def test_oracle_bitmap_by_hand():
    # ids 0, 31, 32, 69 over a 70-token vocabulary: words 0..2
    assert A.bitmap([0, 31, 32, 69], 70) == [1 | (1 << 31), 1, 1 << 5]
    assert A.bitmap([], 33) == [0, 0]


def test_oracle_bitmap_brute_force():
    rng = random.Random(5)
    for vocab in (1, 31, 32, 33, 100, 257):
        ids = rng.sample(range(vocab), k=min(vocab, 7))
        words = A.bitmap(ids, vocab)
        for t in range(vocab):
            assert ((words[t // 32] >> (t % 32)) & 1) == int(t in ids)
        assert sum(bin(w).count("1") for w in words) == len(set(ids))
        assert A.cue_flags([-1, vocab, vocab + 40], ids, vocab) == [0, 0, 0]


@pytest.mark.parametrize("vocab", [1, 32, 2048, 152064])
def test_native_bitmap_matches_oracle(vocab):
    rng = random.Random(vocab)
    ids = [rng.randrange(vocab) for _ in range(min(vocab, 64))]
    got = L.laser_atp_bitmap(ids, vocab)
    assert [int(x) for x in got] == A.bitmap(ids, vocab)


def test_native_bitmap_errors():
    with pytest.raises(L.LaserError):
        L.laser_atp_bitmap([5], 5)
    with pytest.raises(L.LaserError):
        L.laser_atp_bitmap([-1], 5)
    with pytest.raises(L.LaserError):
        L.laser_atp_bitmap([], 0)
