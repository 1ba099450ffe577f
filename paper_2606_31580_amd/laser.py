"""ctypes binding of liblaser.so (C ABI in include/laser.h).

Functions keep the C names and signatures (argument marshalling only); every step of
the hot path runs in the library's HIP kernels.  `Model` and `KVCache` are thin owners
of the device memory (allocated with PyTorch) that the library borrows.  Loading fails
loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, Optional, Sequence

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "lib", "liblaser.so")

OK, ERR_INVALID_ARG, ERR_OUT_OF_PAGES, ERR_HIP, ERR_UNSUPPORTED, ERR_STATE = 0, -1, -2, -3, -4, -5
DTYPE_F32, DTYPE_BF16, DTYPE_FP8_E4M3 = 0, 1, 2
CONTINUE, EARLY_EXIT, BUDGET_EXHAUSTED = 0, 1, 2
K_EMBED, K_QKV, K_ATTN, K_OPROJ, K_GATEUP, K_DOWN, K_LMHEAD, K_OTHER = range(8)
KERNEL_CLASSES = {"embed": 0, "qkv": 1, "attn": 2, "oproj": 3, "gateup": 4, "down": 5, "lmhead": 6, "other": 7}


class LaserError(RuntimeError):
    def __init__(self, code: int, fn: str, msg: str):
        super().__init__(f"{fn} failed ({code}): {msg}")
        self.code = code


class laser_params(C.Structure):
    _fields_ = [(n, C.c_double) for n in ("lambda_base", "beta", "gamma", "alpha", "L_target", "lambda_min", "lambda_max")] + [
        ("B_base", C.c_int), ("B_min", C.c_int), ("f_min", C.c_double), ("f_max", C.c_double), ("p_min", C.c_int), ("p_max", C.c_int)]


class laser_load_state(C.Structure):
    _fields_ = [("L_bar", C.c_double)]


class laser_model_desc(C.Structure):
    _fields_ = [(n, C.c_int) for n in ("n_layers", "d_model", "n_q_heads", "n_kv_heads", "head_dim", "d_ffn", "vocab",
                                       "tied_embeddings", "qkv_bias", "dtype")] + [
        ("rope_theta", C.c_float), ("rms_eps", C.c_float), ("max_positions", C.c_int), ("kv_dtype", C.c_int)]


class laser_sim_config(C.Structure):
    _fields_ = [("method", C.c_int), ("fixed_lambda", C.c_double), ("max_probes", C.c_int),
                ("max_think_tokens", C.c_int)] + [(n, C.c_double) for n in (
                    "prefill_ms", "prefill_ms_per_token", "decode_ms", "decode_ms_per_ctx", "probe_ms",
                    "probe_ms_per_ctx", "slo_s")]


class laser_sim_request(C.Structure):
    _fields_ = [("arrival_s", C.c_double), ("prompt_len", C.c_int32), ("n_chunks", C.c_int32),
                ("conclusion_tokens", C.c_int32), ("nothink_correct", C.c_int32)]


class laser_sim_result(C.Structure):
    _fields_ = [(n, C.c_double) for n in ("start_s", "finish_s", "latency_s", "lambda_last")] + [
        (n, C.c_int32) for n in ("budget", "chunks", "probes", "think_tokens", "outcome", "correct")]


class laser_sim_summary(C.Structure):
    _fields_ = [("n", C.c_int32)] + [(n, C.c_double) for n in (
        "mean_latency_s", "p95_latency_s", "throughput_qps", "slo_rate", "accuracy", "mean_tokens",
        "early_exit_rate")]


SIM_VANILLA, SIM_FIXED, SIM_LASER, SIM_THRESHOLD_ONLY, SIM_BUDGET_ONLY, SIM_NOTHINKING = range(6)
SIM_FINISHED, SIM_EXITED, SIM_EXHAUSTED, SIM_CAPPED, SIM_SKIPPED = range(5)

_P = C.c_void_p
_I = C.c_int
_I32P = C.POINTER(C.c_int32)
_SIGS = {
    "laser_last_error": (C.c_char_p, []),
    "laser_abi_version": (_I, []),
    "laser_params_default": (None, [C.POINTER(laser_params)]),
    "laser_ema_update": (_I, [C.POINTER(laser_params), C.POINTER(laser_load_state), _I]),
    "laser_threshold": (_I, [C.POINTER(laser_params), C.c_double, C.POINTER(C.c_double)]),
    "laser_budget": (_I, [C.POINTER(laser_params), _I, _I, C.POINTER(_I)]),
    "laser_exit_decision": (_I, [C.POINTER(laser_params), C.POINTER(laser_load_state), C.c_float, _I, _I, _I,
                                 C.POINTER(_I), C.POINTER(C.c_double)]),
    "laser_pages_create": (_I, [_I, _I, _I, _I, C.POINTER(_P)]),
    "laser_pages_add_seq": (_I, [_P, _I, _I]),
    "laser_pages_append": (_I, [_P, _I, _I]),
    "laser_pages_truncate": (_I, [_P, _I, _I]),
    "laser_pages_free_seq": (_I, [_P, _I]),
    "laser_pages_fork": (_I, [_P, _I, _I]),
    "laser_pages_table": (_I, [_P, _I, _I32P, _I, C.POINTER(_I)]),
    "laser_pages_seq_len": (_I, [_P, _I, C.POINTER(_I)]),
    "laser_pages_num_free": (_I, [_P, C.POINTER(_I)]),
    "laser_pages_destroy": (_I, [_P]),
    "laser_model_create": (_I, [C.POINTER(laser_model_desc), C.POINTER(_P)]),
    "laser_model_set_tensor": (_I, [_P, C.c_char_p, _P, C.c_size_t]),
    "laser_workspace_size": (_I, [_P, _I, C.POINTER(C.c_size_t)]),
    "laser_model_finalize": (_I, [_P, _I, _P, C.c_size_t, _P]),
    "laser_model_destroy": (_I, [_P]),
    "laser_kv_pool_bytes": (_I, [_P, _I, C.POINTER(C.c_size_t)]),
    "laser_kv_create": (_I, [_P, _I, _I, _I, _P, _P, _P, C.POINTER(_P)]),
    "laser_kv_add_seq": (_I, [_P, _I, _I]),
    "laser_kv_import": (_I, [_P, _I, _P, _P, _I, _P]),
    "laser_kv_export": (_I, [_P, _I, _P, _P, _P]),
    "laser_kv_free_seq": (_I, [_P, _I]),
    "laser_kv_fork": (_I, [_P, _I, _I, _P]),
    "laser_kv_seq_len": (_I, [_P, _I, C.POINTER(_I)]),
    "laser_kv_page_table": (_I, [_P, _I, _I32P, _I, C.POINTER(_I)]),
    "laser_kv_destroy": (_I, [_P]),
    "laser_prefill": (_I, [_P, _P, _I, _P, _I, _P, _P]),
    "laser_decode_step": (_I, [_P, _P, _I, _I32P, _P, _P, _P, _P, _P]),
    "laser_decode_step_static": (_I, [_P, _P, _I, _I32P, _P, _P, _P, _P, _P]),
    "laser_probe_confidence": (_I, [_P, _P, _I, _I32P, _P, _I, _I, _P, _P, _P, _P]),
    "laser_step_mixed": (_I, [_P, _P, _I, _I32P, _P, _P, _P, _I, _I32P, _P, _I, _I, _P, _P, _P]),
    "laser_forward": (_I, [_P, _P, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "laser_confidence": (_I, [_P, _P, _I, _I, _P, _P]),
    "laser_timing_enable": (_I, [_P, _I, _I]),
    "laser_timing_read": (_I, [_P, _I, C.POINTER(C.c_double), C.POINTER(_I)]),
    "laser_model_set_graphs": (_I, [_P, _I]),
    "laser_model_set_gemm_kernel": (_I, [_P, _I]),
    "laser_model_set_attn_merge": (_I, [_P, _I, _I]),
    "laser_model_set_oproj_merge": (_I, [_P, _I]),
    "laser_model_graph_stats": (_I, [_P, C.POINTER(C.c_longlong), C.POINTER(C.c_int)]),
    "laser_model_tile_bytes": (_I, [_P, C.POINTER(C.c_size_t)]),
    "laser_model_set_tiles": (_I, [_P, _P, C.c_size_t, _P]),
    "laser_atp_bitmap": (_I, [_P, _I, _I, _P]),
    "laser_atp_match": (_I, [_P, _I, _P, _I, _P, _P]),
    "laser_simulate": (_I, [C.POINTER(laser_params), C.POINTER(laser_sim_config), _I, C.POINTER(laser_sim_request),
                            _P, _P, _P, C.POINTER(laser_sim_result), C.POINTER(laser_sim_summary)]),
}

_lib = None


def lib() -> C.CDLL:
    """The loaded liblaser.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_31580_amd.build`")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def exported_symbols():
    return list(_SIGS)


def check(code: int, fn: str) -> int:
    if code != OK:
        raise LaserError(code, fn, lib().laser_last_error().decode())
    return code


def _call(name, *args):
    return check(getattr(lib(), name)(*args), name)


def _i32arr(vals: Sequence[int]):
    return (C.c_int32 * len(vals))(*[int(v) for v in vals])


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


# --------------------------------------------------------------------------- controller

def laser_params_default() -> laser_params:
    p = laser_params()
    lib().laser_params_default(C.byref(p))
    return p


def laser_ema_update(p: laser_params, state: laser_load_state, active_requests: int) -> None:
    _call("laser_ema_update", C.byref(p), C.byref(state), active_requests)


def laser_threshold(p: laser_params, L_bar: float) -> float:
    out = C.c_double()
    _call("laser_threshold", C.byref(p), L_bar, C.byref(out))
    return out.value


def laser_budget(p: laser_params, prompt_len: int, active_requests: int) -> int:
    out = C.c_int()
    _call("laser_budget", C.byref(p), prompt_len, active_requests, C.byref(out))
    return out.value


def laser_exit_decision(p: laser_params, state: laser_load_state, confidence: float, active_requests: int, k_done: int,
                        B_i: int):
    d, lam = C.c_int(), C.c_double()
    _call("laser_exit_decision", C.byref(p), C.byref(state), confidence, active_requests, k_done, B_i, C.byref(d),
          C.byref(lam))
    return d.value, lam.value


# --------------------------------------------------------------------------- page pool

class PagePool:
    """Host page pool (laser_pages_*)."""

    def __init__(self, num_pages: int, page_size: int = 16, max_seqs: int = 64, max_pages_per_seq: int = 4096):
        h = C.c_void_p()
        _call("laser_pages_create", num_pages, page_size, max_seqs, max_pages_per_seq, C.byref(h))
        self.h = h
        self.max_pages_per_seq = max_pages_per_seq

    def add_seq(self, seq, length):
        _call("laser_pages_add_seq", self.h, seq, length)

    def append(self, seq, n=1):
        _call("laser_pages_append", self.h, seq, n)

    def truncate(self, seq, length):
        _call("laser_pages_truncate", self.h, seq, length)

    def free_seq(self, seq):
        _call("laser_pages_free_seq", self.h, seq)

    def fork(self, src, dst):
        _call("laser_pages_fork", self.h, src, dst)

    def table(self, seq):
        buf = (C.c_int32 * self.max_pages_per_seq)()
        n = C.c_int()
        _call("laser_pages_table", self.h, seq, buf, self.max_pages_per_seq, C.byref(n))
        return list(buf[: n.value])

    def seq_len(self, seq):
        n = C.c_int()
        _call("laser_pages_seq_len", self.h, seq, C.byref(n))
        return n.value

    def num_free(self):
        n = C.c_int()
        _call("laser_pages_num_free", self.h, C.byref(n))
        return n.value

    def destroy(self):
        if self.h:
            _call("laser_pages_destroy", self.h)
            self.h = None


# --------------------------------------------------------------------------- model / KV (device)

def desc_from_shape(shape, max_positions: int = 16640) -> laser_model_desc:
    return laser_model_desc(
        shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.d_ffn, shape.vocab,
        int(shape.tied_embeddings), int(shape.qkv_bias), DTYPE_BF16 if shape.dtype == "bf16" else DTYPE_F32,
        float(shape.rope_theta), float(shape.rms_eps), int(max_positions),
        DTYPE_FP8_E4M3 if getattr(shape, "kv_dtype", "") == "fp8" else 0)


def _stream_ptr(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


class Model:
    """A finalized model over device weights (dict name -> torch tensor on the GPU)."""

    def __init__(self, shape, weights: Dict[str, "object"], max_rows: int = 16, max_positions: int = 16640, stream=None,
                 poison: bool = False, tiles: bool = True):
        import torch
        self.shape = shape
        self.weights = weights  # kept alive: the library borrows them
        self.desc = desc_from_shape(shape, max_positions)
        h = C.c_void_p()
        _call("laser_model_create", C.byref(self.desc), C.byref(h))
        self.h = h
        for name, t in weights.items():
            assert t.is_cuda and t.is_contiguous()
            _call("laser_model_set_tensor", self.h, name.encode(), t.data_ptr(), t.numel() * t.element_size())
        nbytes = C.c_size_t()
        _call("laser_workspace_size", self.h, max_rows, C.byref(nbytes))
        self.workspace = torch.empty(nbytes.value, dtype=torch.uint8, device=next(iter(weights.values())).device)
        self.max_rows = max_rows
        if poison:  # tests: NaN bytes everywhere, so any read of unwritten workspace shows
            self.workspace.fill_(0xFF)
        _call("laser_model_finalize", self.h, max_rows, self.workspace.data_ptr(), nbytes.value, _stream_ptr(stream))
        self.tile_buf = None
        if tiles:
            self.set_tiles(True, stream)

    def set_tiles(self, on: bool, stream=None):
        """Matrix-core weight tiles for forwards of more than 4 rows (a second copy of the weights)."""
        import torch
        if on and self.tile_buf is None:
            nb = C.c_size_t()
            _call("laser_model_tile_bytes", self.h, C.byref(nb))
            self.tile_buf = torch.empty(nb.value, dtype=torch.uint8, device=self.workspace.device)
        if on:
            _call("laser_model_set_tiles", self.h, self.tile_buf.data_ptr(), self.tile_buf.numel(), _stream_ptr(stream))
        else:
            _call("laser_model_set_tiles", self.h, None, 0, _stream_ptr(stream))

    def set_graphs(self, on: bool):
        """Replay forwards from captured HIP graphs (default) or launch kernels one by one."""
        _call("laser_model_set_graphs", self.h, int(on))

    def graph_stats(self):
        """(forwards captured into graphs so far, graphs cached now)."""
        n, c = C.c_longlong(), C.c_int()
        _call("laser_model_graph_stats", self.h, C.byref(n), C.byref(c))
        return n.value, c.value

    def set_attn_merge(self, fused: bool, max_splits: int = 56):
        """One-row attention groups merged inside the attention kernel (fused) or by the merge kernel (default)."""
        _call("laser_model_set_attn_merge", self.h, int(fused), int(max_splits))

    def set_oproj_merge(self, mode: int):
        """Where the split merge of 1-2 row forwards runs: 0 the merge kernel, 1 (default) the
        O-projection's launch for projections of at least 16 MiB of weights, 2 that launch always."""
        _call("laser_model_set_oproj_merge", self.h, int(mode))

    def set_gemm_kernel(self, mode: int):
        """Matrix-core projection kernel: 0 by cost (default), 1 K-split waves, 2 row waves."""
        _call("laser_model_set_gemm_kernel", self.h, int(mode))

    def timing_enable(self, cls: int, on: bool = True):
        _call("laser_timing_enable", self.h, cls, int(on))

    def timing_read(self, cls: int):
        ms, n = C.c_double(), C.c_int()
        _call("laser_timing_read", self.h, cls, C.byref(ms), C.byref(n))
        return ms.value, n.value

    def destroy(self):
        if self.h:
            _call("laser_model_destroy", self.h)
            self.h = None


class KVCache:
    """Paged KV cache: device pools and block table allocated here, bookkeeping in the library."""

    def __init__(self, model: Model, num_pages: int, max_seqs: int, max_pages_per_seq: int, poison: bool = False):
        import torch
        dev = model.workspace.device
        nb = C.c_size_t()
        _call("laser_kv_pool_bytes", model.h, num_pages, C.byref(nb))
        self.k_pool = torch.empty(nb.value, dtype=torch.uint8, device=dev)
        self.v_pool = torch.empty(nb.value, dtype=torch.uint8, device=dev)
        self.block_table = torch.zeros(max_seqs * max_pages_per_seq, dtype=torch.int32, device=dev)
        if poison:  # tests: unwritten KV slots read as NaN
            self.k_pool.fill_(0xFF)
            self.v_pool.fill_(0xFF)
        self.model = model
        self.max_pages_per_seq = max_pages_per_seq
        h = C.c_void_p()
        _call("laser_kv_create", model.h, num_pages, max_seqs, max_pages_per_seq, self.k_pool.data_ptr(),
              self.v_pool.data_ptr(), self.block_table.data_ptr(), C.byref(h))
        self.h = h

    def add_seq(self, seq: int, length: int):
        _call("laser_kv_add_seq", self.h, seq, length)

    def import_kv(self, seq: int, k, v, stream=None):
        _call("laser_kv_import", self.h, seq, k.data_ptr(), v.data_ptr(), k.shape[1], _stream_ptr(stream))

    def export_kv(self, seq: int, k, v, stream=None):
        _call("laser_kv_export", self.h, seq, k.data_ptr(), v.data_ptr(), _stream_ptr(stream))

    def free_seq(self, seq: int):
        _call("laser_kv_free_seq", self.h, seq)

    def fork(self, src: int, dst: int, stream=None):
        """dst (a free slot) starts as a copy of src that shares src's full pages."""
        _call("laser_kv_fork", self.h, src, dst, _stream_ptr(stream))

    def seq_len(self, seq: int) -> int:
        n = C.c_int()
        _call("laser_kv_seq_len", self.h, seq, C.byref(n))
        return n.value

    def page_table(self, seq: int):
        buf = (C.c_int32 * self.max_pages_per_seq)()
        n = C.c_int()
        _call("laser_kv_page_table", self.h, seq, buf, self.max_pages_per_seq, C.byref(n))
        return list(buf[: n.value])

    def destroy(self):
        if self.h:
            _call("laser_kv_destroy", self.h)
            self.h = None


# --------------------------------------------------------------------------- hot path

def laser_prefill(model: Model, kv: KVCache, seq_id: int, d_tokens, d_logits_last=None, stream=None):
    _call("laser_prefill", model.h, kv.h, seq_id, d_tokens.data_ptr(), d_tokens.numel(), _ptr(d_logits_last),
          _stream_ptr(stream))


def laser_decode_step(model: Model, kv: KVCache, seq_ids: Sequence[int], d_tokens, d_next, d_max_prob, d_logits=None,
                      stream=None):
    _call("laser_decode_step", model.h, kv.h, len(seq_ids), _i32arr(seq_ids), d_tokens.data_ptr(), d_next.data_ptr(),
          d_max_prob.data_ptr(), _ptr(d_logits), _stream_ptr(stream))


def laser_decode_step_static(model: Model, kv: KVCache, seq_ids: Sequence[int], d_tokens, d_next, d_max_prob,
                             d_logits=None, stream=None):
    """laser_decode_step with its scratch in the library's static device array (allocates nothing)."""
    _call("laser_decode_step_static", model.h, kv.h, len(seq_ids), _i32arr(seq_ids), d_tokens.data_ptr(),
          d_next.data_ptr(), d_max_prob.data_ptr(), _ptr(d_logits), _stream_ptr(stream))


def laser_probe_confidence(model: Model, kv: KVCache, seq_ids: Sequence[int], d_suffix, T: int, d_conf, d_argmax,
                           d_logits=None, stream=None):
    _call("laser_probe_confidence", model.h, kv.h, len(seq_ids), _i32arr(seq_ids), d_suffix.data_ptr(), d_suffix.numel(), T,
          d_conf.data_ptr(), d_argmax.data_ptr(), _ptr(d_logits), _stream_ptr(stream))


class laser_span(C.Structure):
    _fields_ = [("seq", C.c_int32), ("n_tokens", C.c_int32), ("tok_sel", C.c_int32), ("tok_off", C.c_int32),
                ("out", C.c_int32), ("out_sel", C.c_int32), ("out_off", C.c_int32)]


def span(seq, n_tokens, tok_sel=0, tok_off=0, out=None):
    """A laser_span; out = (out_sel, out_off) to emit the last row's token and max-prob."""
    o = out is not None
    return laser_span(seq, n_tokens, tok_sel, tok_off, int(o), out[0] if o else 0, out[1] if o else 0)


def laser_forward(model: Model, kv: KVCache, spans: Sequence[laser_span], d_tok0, d_tok1=None, d_out_tok0=None,
                  d_out_p0=None, d_out_tok1=None, d_out_p1=None, d_out_logits0=None, d_out_logits1=None, stream=None):
    arr = (laser_span * len(spans))(*spans)
    _call("laser_forward", model.h, kv.h, len(spans), arr, _ptr(d_tok0), _ptr(d_tok1), _ptr(d_out_tok0),
          _ptr(d_out_p0), _ptr(d_out_tok1), _ptr(d_out_p1), _ptr(d_out_logits0), _ptr(d_out_logits1),
          _stream_ptr(stream))


def laser_confidence(model: Model, d_p, T: int, n: int, d_conf, stream=None):
    _call("laser_confidence", model.h, _ptr(d_p), T, n, _ptr(d_conf), _stream_ptr(stream))


def laser_step_mixed(model: Model, kv: KVCache, seq_ids: Sequence[int], d_tokens, d_next, d_max_prob,
                     probe_idx: Sequence[int], d_suffix, T: int, d_conf, d_argmax, stream=None):
    n = len(probe_idx)
    _call("laser_step_mixed", model.h, kv.h, len(seq_ids), _i32arr(seq_ids), d_tokens.data_ptr(), d_next.data_ptr(),
          d_max_prob.data_ptr(), n, _i32arr(probe_idx) if n else None, _ptr(d_suffix) if n else None,
          d_suffix.numel() if n else 0, T, _ptr(d_conf) if n else None, _ptr(d_argmax) if n else None, _stream_ptr(stream))


# --------------------------------------------------------------------------- serving simulation

def sim_config(method: int, costs: dict, fixed_lambda: float = 0.95, max_probes: int = 0, max_think_tokens: int = 0,
               slo_s: float = 30.0) -> laser_sim_config:
    """A laser_sim_config; costs holds the six cost-model fields (milliseconds)."""
    cfg = laser_sim_config(method=method, fixed_lambda=fixed_lambda, max_probes=max_probes,
                           max_think_tokens=max_think_tokens, slo_s=slo_s)
    for k in ("prefill_ms", "prefill_ms_per_token", "decode_ms", "decode_ms_per_ctx", "probe_ms", "probe_ms_per_ctx"):
        setattr(cfg, k, float(costs.get(k, 0.0)))
    return cfg


def laser_simulate(params: laser_params, cfg: laser_sim_config, arrivals, traces: dict):
    """Runs laser_simulate on arrival times (s) and traces (the arrays of synth.make_sim_traces).

    Returns (results: list of laser_sim_result, summary: laser_sim_summary).
    """
    import numpy as np

    n = len(arrivals)
    reqs = (laser_sim_request * max(n, 1))()
    for i in range(n):
        reqs[i] = laser_sim_request(float(arrivals[i]), int(traces["prompt_len"][i]), int(traces["n_chunks"][i]),
                                    int(traces["conclusion_tokens"][i]), int(traces["nothink_correct"][i]))
    tok = np.ascontiguousarray(traces["chunk_tokens"], dtype=np.int32)
    conf = np.ascontiguousarray(traces["confidence"], dtype=np.float32)
    corr = np.ascontiguousarray(traces["correct"], dtype=np.uint8)
    out = (laser_sim_result * max(n, 1))()
    summ = laser_sim_summary()
    _call("laser_simulate", C.byref(params), C.byref(cfg), n, reqs, tok.ctypes.data if tok.size else None,
          conf.ctypes.data if conf.size else None, corr.ctypes.data if corr.size else None, out, C.byref(summ))
    return [out[i] for i in range(n)], summ


# --------------------------------------------------------------------------- ATP cues

def laser_atp_bitmap(ids: Sequence[int], vocab: int):
    """Bitmap words (numpy uint32, (vocab + 31) // 32) of the ATP cue token set."""
    import numpy as np

    words = np.zeros((vocab + 31) // 32, dtype=np.uint32)
    arr = np.ascontiguousarray(np.asarray(list(ids), dtype=np.int32))
    _call("laser_atp_bitmap", arr.ctypes.data if arr.size else None, int(arr.size), vocab, words.ctypes.data)
    return words


def laser_atp_match(d_tokens, d_bitmap, vocab: int, d_flags, n: Optional[int] = None, stream=None) -> None:
    """d_flags[i] = 1 if d_tokens[i] is an ATP cue token (device tensors, int32 / uint32 words)."""
    n = d_tokens.numel() if n is None else n
    _call("laser_atp_match", d_tokens.data_ptr(), n, d_bitmap.data_ptr(), vocab, d_flags.data_ptr(), _stream_ptr(stream))
