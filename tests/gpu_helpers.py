"""Shared helpers of the GPU parity tests: build the device model/KV and the matching oracle.

Both sides get the same seeded inputs from paper_2606_31580_amd.synth; the oracle gets
host copies (bf16 as bit patterns).  Nothing here computes any of the method.
"""
import numpy as np
import torch

from oracle.pages import PagePool as OraclePool
from oracle.transformer import DecoderOracle, SeqState, lm_stats
from paper_2606_31580_amd import laser as L
from paper_2606_31580_amd import synth

# Tolerances fixed by the parity protocol: logits within 2e-2 absolute, confidence (and
# max-probabilities) within 1e-3, greedy tokens exact wherever the oracle's top-2 margin
# exceeds 1e-2, exit decisions exact wherever |C - lambda| > 1e-3.
LOGIT_TOL = 2e-2
PROB_TOL = 1e-3
MARGIN = 1e-2


def require_gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    return torch.device("cuda:0")


def make_pair(shape, max_rows, max_positions, weights_on_device=False, cache_oracle=False):
    """(device weights, oracle) for `shape` from the seeded generator."""
    dev = require_gpu()
    if weights_on_device:
        w_dev = synth.make_weights(shape, device=dev)
    else:
        w_dev = {k: v.to(dev) for k, v in synth.make_weights(shape).items()}
    host = {k: synth.to_numpy(v) for k, v in w_dev.items()}
    orc = DecoderOracle(shape, host, cache_weights=cache_oracle)
    model = L.Model(shape, w_dev, max_rows=max_rows, max_positions=max_positions, poison=True)
    return model, orc, w_dev


def kv_pair(model, shape, num_pages, max_seqs, max_pages_per_seq):
    return L.KVCache(model, num_pages, max_seqs, max_pages_per_seq, poison=True), OraclePool(num_pages)


def export_seq(kv, shape, seq):
    n = kv.seq_len(seq)
    dt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
    K = torch.empty((shape.n_layers, n, shape.n_kv_heads, shape.head_dim), dtype=dt, device="cuda")
    V = torch.empty_like(K)
    kv.export_kv(seq, K, V)
    torch.cuda.synchronize()
    return K.float().cpu().numpy().astype(np.float64), V.float().cpu().numpy().astype(np.float64)


def compare_logits(gpu_row, ref_row, what=""):
    g = np.asarray(gpu_row, dtype=np.float64)
    err = float(np.max(np.abs(g - ref_row)))
    assert err <= LOGIT_TOL, f"{what}: logits differ by {err}"
    return err


def check_token(gpu_tok, ref_row, what=""):
    tok, _, margin = lm_stats(ref_row)
    if margin > MARGIN:
        assert int(gpu_tok) == tok, f"{what}: token {gpu_tok} vs oracle {tok} (margin {margin})"
    return tok
