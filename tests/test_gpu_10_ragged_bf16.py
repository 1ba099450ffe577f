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
The final-norm gain is 8, so the max-probabilities and confidences sit well inside (0, 1).
Decode rows go through the VALU path at one and two rows and the matrix cores at three;
the probe chunks always run on the matrix cores.
"""
import pytest

from gpu_helpers import set_final_gain
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
