"""ATP cue detection as token-set membership (Section 3.1).

Oracle (test infrastructure).  The paper marks ATPs by linguistic cues such as "Wait" or
"Alternatively" between reasoning chunks.  With the cues given as token ids, a freshly
generated token is an ATP cue exactly when it is one of those ids.  The bitmap is the
set written as bits: bit b of word w is set exactly when token 32 w + b is a cue.

Pinned in tests/test_atp.py by a hand-written bitmap and by brute force over a small
vocabulary.
"""
from __future__ import annotations

from typing import List, Sequence


def is_cue(token: int, cue_ids: Sequence[int], vocab: int) -> bool:
    return 0 <= token < vocab and token in set(cue_ids)


def cue_flags(tokens: Sequence[int], cue_ids: Sequence[int], vocab: int) -> List[int]:
    return [int(is_cue(int(t), cue_ids, vocab)) for t in tokens]


def bitmap(cue_ids: Sequence[int], vocab: int) -> List[int]:
    ids = set(int(i) for i in cue_ids)
    return [sum(1 << b for b in range(32) if 32 * w + b in ids) for w in range((vocab + 31) // 32)]
