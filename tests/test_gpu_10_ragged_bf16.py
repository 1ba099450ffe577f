"""GPU parity on a small bf16 decoder whose widths leave ragged tails everywhere.

The full-size shapes have row lengths that are multiples of 512, so every projection's
chunks fill whole waves and every matrix-core K step is whole.  This decoder (2 layers,
d_model 960, 6 query / 2 KV heads of 128, FFN 2600, vocabulary 4099, QKV bias) gives:
  * one-chunk-per-thread GEMVs whose rows (120 and 96 chunks of 16 bytes) leave part of the
    last wave idle, and a down projection (325 chunks) that takes three chunks per thread
    over 128 threads with the last pass partly past the row;
  * matrix-core projections with K = 2600 (81 whole 32-column steps and a partial one);
  * an LM head whose last row group is partly past the vocabulary;
  * contexts that end inside a page.
  * QKV of forwards of 33 to 64 rows over 512-column slices of K with K = 960 (the second
    slice ends 64 columns past K) and 80 row groups (the last workgroup of 16 groups full,
    five workgroups per slice), with the QKV bias added after the slices are summed.
The final-norm gain is 8, so the max-probabilities and confidences sit well inside (0, 1).
Decode rows go through the VALU path at one and two rows and the matrix cores at three;
the probe chunks always run on the matrix cores.
"""
import pytest

from gpu_helpers import check_exit_decisions, kv_pair, make_pair, riding_forwards, set_final_gain
from oracle.transformer import SeqState
from paper_2606_31580_amd import synth
from paper_2606_31580_amd.configs import ModelShape
from test_gpu_2_full_shapes import Setup

pytestmark = pytest.mark.gpu

RAGGED = ModelShape("ragged-bf16-2L-d960", 2, 960, 6, 2, 128, 2600, 4099, False, True, "bf16", 1.0e4, 1.0e-6)


def run(lens, steps, probe_seqs):
    st = Setup(RAGGED, lens)
    set_final_gain(st.model, st.orc, 8.0)
    st.decode(steps)
    st.probe(probe_seqs)
    st.release()


def test_ragged_bf16_one_row():
    run([700], 3, [0])


def test_ragged_bf16_two_rows():
    run([37, 1000], 2, [0, 1])


def test_ragged_bf16_three_rows_matrix_cores():
    run([37, 300, 1001], 2, [2])


def test_ragged_bf16_riding_wide_forwards():
    """Six requests with probes riding along: forward 0 carries 6 decode rows and 6 x 8 suffix
    rows (54 rows, four activation tiles), forward 2 another 4 probes' suffixes beside 6
    decode and 6 trial rows (44 rows, three tiles); the QKV projection of both runs over K
    slices.  Every decode row, and the probes started in forward 0 on requests 1 and 4, are
    checked against the oracle."""
    S, T = 8, 4
    lens = [37, 300, 1001, 700, 17, 450]
    cap = max(lens) + 64
    model, orc, _ = make_pair(RAGGED, max_rows=64, max_positions=cap, weights_on_device=True, cache_oracle=True)
    n_forks = 10
    kv, opool = kv_pair(model, RAGGED, num_pages=sum(n // 16 + 2 for n in lens) + 3 * n_forks + 16,
                        max_seqs=len(lens) + n_forks, max_pages_per_seq=cap // 16 + 1)
    states = {}
    for b, n in enumerate(lens):
        K0, V0 = synth.make_prefill_kv(RAGGED, n, b, device="cuda")
        kv.add_seq(b, n)
        opool.add_seq(b, n)
        kv.import_kv(b, K0, V0)
        states[b] = SeqState.from_prefill(RAGGED, synth.to_numpy(K0), synth.to_numpy(V0), cap)
    set_final_gain(model, orc, 8.0)
    suffix = [int(t) for t in synth.make_suffix(S, RAGGED.vocab)]
    starts = [list(range(6)), [], [0, 2, 3, 5], []]
    pairs = riding_forwards(model, orc, kv, opool, states, list(range(6)), starts, {(0, 1), (0, 4)},
                            list(range(6, 6 + n_forks)), suffix, S, T, 6011, "ragged riding")
    assert len(pairs) == 2
    check_exit_decisions(pairs, "ragged")
    kv.destroy()
    model.destroy()
