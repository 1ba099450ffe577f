"""Riding probes at the 8B shape, batch 8: forwards of 40 to 52 rows against the oracle.

The benchmark's batch-8 pattern: every forward decodes the 8 requests (ragged contexts of
3,000-14,000 positions) and a seeded half of them start a probe, each on a fork whose 8
suffix rows ride in that forward and whose 3 trial rows ride one per forward in the next
three.  The fourth forward carries 8 decode rows, 32 suffix rows and 12 trial rows (52 rows:
matrix-core projections over four 16-row tiles, the row-wave kernel for gate/up and the
O/down projections, shared-prefix attention for each request and its forks).

Sampled outputs are checked against the oracle one by one: every decode row of three
requests in every forward (logits, greedy token, max-probability), and the two probes of
the first forward that finish in the 52-row forward (trial inputs forced to the oracle's
tokens: every trial's logits, token, max-probability, and the confidence).  Page tables of
all requests and forks are checked after every forward.  The final norm gain is 4, so the
max-probabilities spread over (0, 1) (a flat random-init model gives about 1/V), and the
probes' confidences drive laser_exit_decision against the oracle controller.
"""
import gc
import sys
import time

import numpy as np
import pytest
import torch

from gpu_helpers import check_exit_decisions, kv_pair, make_pair, require_gpu, riding_forwards, set_final_gain
from oracle.transformer import SeqState
from paper_2606_31580_amd import synth
from paper_2606_31580_amd.configs import LLAMA_8B

pytestmark = pytest.mark.gpu

S, T = 8, 4
T0 = [time.time()]


def log(*a):
    print(f"[{time.time() - T0[0]:6.1f}s]", *a, flush=True)
    sys.stdout.flush()


def test_llama8b_b8_riding_52_row_forward():
    T0[0] = time.time()
    require_gpu()
    shape = LLAMA_8B
    V = shape.vocab
    lens = synth.make_ragged_lengths(8, 3000, 14000)
    cap = max(lens) + 64
    model, orc, _ = make_pair(shape, max_rows=64, max_positions=cap, weights_on_device=True, cache_oracle=True,
                              oracle_dtype=np.float32)
    n_forks = 16
    num_pages = sum(n // 16 + 2 for n in lens) + 3 * n_forks + 16
    kv, opool = kv_pair(model, shape, num_pages=num_pages, max_seqs=8 + n_forks, max_pages_per_seq=cap // 16 + 1)
    schedule = synth.make_mixed_schedule(8, 4)
    checked = {(0, schedule[0][0]), (0, schedule[0][1])}
    check_rows = sorted({schedule[0][0], schedule[0][1], [b for b in range(8) if b not in schedule[0]][0]})
    states = {}
    for b, n in enumerate(lens):
        K0, V0 = synth.make_prefill_kv(shape, n, b, device="cuda")
        kv.add_seq(b, n)
        opool.add_seq(b, n)
        kv.import_kv(b, K0, V0)
        if b in check_rows:
            states[b] = SeqState.from_prefill(shape, synth.to_numpy(K0), synth.to_numpy(V0), cap, dtype=np.float32)
        del K0, V0
    suffix = [int(t) for t in synth.make_suffix(S, V)]
    log(f"8B lens {lens}: setup done; probes {schedule}, checked rows {check_rows}")
    set_final_gain(model, orc, 4.0)
    pairs = riding_forwards(model, orc, kv, opool, states, list(range(8)), schedule, checked,
                            list(range(8, 8 + n_forks)), suffix, S, T, 5023, "8B riding", check_rows=check_rows,
                            log=log)
    assert len(pairs) == 2
    n = check_exit_decisions(pairs, "8B")
    log(f"8B: {n} exit decisions compared")
    kv.destroy()
    model.destroy()
    del orc, states
    gc.collect()
    torch.cuda.empty_cache()
