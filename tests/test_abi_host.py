"""Host-side tests of liblaser.so through its C ABI (no device work; runs on CPU)."""
import ctypes as C
import math
import os
import random
import re

import pytest

from oracle import controller as OC
from oracle.pages import OutOfPages, PagePool as OraclePool
from paper_2606_31580_amd import laser as L
from paper_2606_31580_amd.configs import QWEN_7B, TINY

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    return L.lib()


def test_exports_every_declared_symbol(lib):
    header = open(os.path.join(ROOT, "include", "laser.h")).read()
    declared = set(re.findall(r"\b(laser_[a-z0-9_]+)\s*\(", header))
    assert len(declared) >= 35
    for name in declared:
        assert hasattr(lib, name), name
    assert set(L.exported_symbols()) <= declared
    assert lib.laser_abi_version() == 3


def _params_from(p: OC.LaserParams):
    q = L.laser_params_default()
    for f in ("lambda_base", "beta", "gamma", "alpha", "L_target", "lambda_min", "lambda_max", "B_base", "B_min", "f_min",
              "f_max", "p_min", "p_max"):
        setattr(q, f, getattr(p, f))
    return q


def test_defaults_match_paper(lib):
    p = L.laser_params_default()
    ref = OC.LaserParams()
    for f in ("lambda_base", "beta", "gamma", "alpha", "L_target", "lambda_min", "lambda_max", "B_base", "B_min", "f_min",
              "f_max", "p_min", "p_max"):
        assert getattr(p, f) == getattr(ref, f), f


def test_threshold_and_ema_match_oracle(lib):
    for beta in (0.04, 0.1, 0.0):
        ref = OC.LaserParams(beta=beta)
        p = _params_from(ref)
        for i in range(400):
            Lb = i * 0.1
            assert L.laser_threshold(p, Lb) == pytest.approx(OC.adaptive_threshold(Lb, ref), abs=1e-15)
        st = L.laser_load_state(0.0)
        Lb = 0.0
        rng = random.Random(1)
        for _ in range(200):
            load = rng.randint(0, 40)
            L.laser_ema_update(p, st, load)
            Lb = OC.ema_update(Lb, load, ref.alpha)
            assert st.L_bar == pytest.approx(Lb, abs=1e-12)


def test_budget_matches_exact_oracle(lib):
    for ref in (OC.LaserParams(), OC.LaserParams(L_target=7.0, f_min=0.5, f_max=2.0, p_min=20, p_max=500, B_base=12)):
        p = _params_from(ref)
        for plen in range(0, 600, 3):
            for load in range(0, 70):
                assert L.laser_budget(p, plen, load) == OC.allocate_budget(plen, load, ref), (plen, load)


def test_exit_decision_matches_oracle(lib):
    ref = OC.LaserParams()
    p = _params_from(ref)
    rng = random.Random(2)
    st = L.laser_load_state(0.0)
    Lb = 0.0
    for _ in range(2000):
        B = rng.randint(1, 12)
        k = rng.randint(0, B - 1)
        load = rng.randint(0, 30)
        conf = rng.choice([rng.random(), 0.97, 0.95, 0.9315153137095996, rng.uniform(0.9, 1.0)])
        conf = float(C.c_float(conf).value)  # the ABI takes float confidence
        d, lam = L.laser_exit_decision(p, st, conf, load, k, B)
        d2, lam2, Lb = OC.exit_decision(Lb, conf, load, k, B, ref)
        assert lam == pytest.approx(lam2, abs=1e-15)
        if abs(conf - lam2) > 1e-12:
            assert d == d2


def test_controller_argument_errors(lib):
    p = L.laser_params_default()
    st = L.laser_load_state(0.0)
    with pytest.raises(L.LaserError) as e:
        L.laser_exit_decision(p, st, 0.5, 1, 3, 3)  # k_done >= B_i
    assert e.value.code == L.ERR_INVALID_ARG and "k_done" in str(e.value)
    assert st.L_bar == 0.0  # untouched on error
    with pytest.raises(L.LaserError):
        L.laser_exit_decision(p, st, float("nan"), 1, 0, 3)
    with pytest.raises(L.LaserError):
        L.laser_budget(p, -1, 1)
    bad = L.laser_params_default()
    bad.L_target = 0.0
    with pytest.raises(L.LaserError):
        L.laser_threshold(bad, 1.0)
    assert lib.laser_threshold(None, C.c_double(1.0), None) == L.ERR_INVALID_ARG


def test_page_pool_matches_oracle_policy(lib):
    rng = random.Random(3)
    n = 48
    pool = L.PagePool(n, 16, 16, 64)
    ref = OraclePool(n)
    live = []
    for step in range(3000):
        op = rng.random()
        try:
            if op < 0.15 and len(live) < 12:
                seq = next(s for s in range(16) if s not in live)
                length = rng.randint(0, 70)
                try:
                    ref.add_seq(seq, length)
                    ok = True
                except OutOfPages:
                    ok = False
                if ok:
                    pool.add_seq(seq, length)
                    live.append(seq)
                else:
                    with pytest.raises(L.LaserError) as e:
                        pool.add_seq(seq, length)
                    assert e.value.code == L.ERR_OUT_OF_PAGES
            elif op < 0.8 and live:
                seq = rng.choice(live)
                k = rng.randint(1, 20)
                try:
                    ref.append(seq, k)
                    ok = True
                except OutOfPages:
                    ok = False
                if ok:
                    pool.append(seq, k)
                else:
                    with pytest.raises(L.LaserError) as e:
                        pool.append(seq, k)
                    assert e.value.code == L.ERR_OUT_OF_PAGES
            elif op < 0.86 and live:
                seq = rng.choice(live)
                cut = rng.randint(0, ref.lens[seq])
                try:
                    ref.truncate(seq, cut)
                    ok = True
                except ValueError:  # would end inside a shared page
                    ok = False
                if ok:
                    pool.truncate(seq, cut)
                else:
                    with pytest.raises(L.LaserError) as e:
                        pool.truncate(seq, cut)
                    assert e.value.code == L.ERR_INVALID_ARG
            elif op < 0.92 and live and len(live) < 12:
                src = rng.choice(live)
                dst = next(s for s in range(16) if s not in live)
                try:
                    ref.fork(src, dst)
                    ok = True
                except OutOfPages:
                    ok = False
                if ok:
                    pool.fork(src, dst)
                    live.append(dst)
                else:
                    with pytest.raises(L.LaserError) as e:
                        pool.fork(src, dst)
                    assert e.value.code == L.ERR_OUT_OF_PAGES
            elif live:
                seq = live.pop(rng.randrange(len(live)))
                ref.free_seq(seq)
                pool.free_seq(seq)
        finally:
            pass
        for s in live:
            assert pool.table(s) == ref.tables[s]
            assert pool.seq_len(s) == ref.lens[s]
        assert pool.num_free() == len(ref.free)
    pool.destroy()


def test_page_pool_errors(lib):
    pool = L.PagePool(4, 16, 4, 2)
    pool.add_seq(0, 20)
    with pytest.raises(L.LaserError) as e:
        pool.add_seq(0, 1)
    assert e.value.code == L.ERR_INVALID_ARG
    with pytest.raises(L.LaserError) as e:
        pool.append(0, 20)  # would need a third page for this sequence
    assert e.value.code == L.ERR_INVALID_ARG
    assert pool.table(0) == [0, 1] and pool.seq_len(0) == 20
    with pytest.raises(L.LaserError):
        pool.add_seq(7, 1)
    h = pool.h
    pool.destroy()
    assert lib.laser_pages_destroy(h) == L.ERR_STATE  # a stale handle is detected


def test_model_validation_without_device(lib):
    bad = L.desc_from_shape(TINY)
    bad.head_dim = 96
    h = C.c_void_p()
    assert lib.laser_model_create(C.byref(bad), C.byref(h)) == L.ERR_UNSUPPORTED
    assert lib.laser_model_create(None, C.byref(h)) == L.ERR_INVALID_ARG
    d = L.desc_from_shape(QWEN_7B)
    assert lib.laser_model_create(C.byref(d), C.byref(h)) == L.OK
    # shapes and names are checked before anything is recorded; fake addresses are never dereferenced
    assert lib.laser_model_set_tensor(h, b"layers.0.wq", 4096, 3584 * 3584 * 2) == L.OK
    assert lib.laser_model_set_tensor(h, b"layers.0.wq", 4096, 123) == L.ERR_INVALID_ARG
    assert lib.laser_model_set_tensor(h, b"layers.28.wq", 4096, 3584 * 3584 * 2) == L.ERR_INVALID_ARG
    assert lib.laser_model_set_tensor(h, b"nonsense", 4096, 4) == L.ERR_INVALID_ARG
    assert "nonsense" in lib.laser_last_error().decode()
    nbytes = C.c_size_t()
    assert lib.laser_workspace_size(h, 0, C.byref(nbytes)) == L.ERR_INVALID_ARG
    assert lib.laser_workspace_size(h, 8, C.byref(nbytes)) == L.OK and nbytes.value > 0
    # hot-path calls before finalize are refused without touching the device
    toks = (C.c_int32 * 1)(0)
    assert lib.laser_decode_step(h, None, 1, toks, None, None, None, None, None) == L.ERR_STATE
    assert lib.laser_model_finalize(h, 8, None, 0, None) in (L.ERR_STATE, L.ERR_INVALID_ARG)
    assert lib.laser_model_destroy(h) == L.OK
    assert lib.laser_model_destroy(h) == L.ERR_STATE


def test_bench_refuses_several_gpus():
    # one GPU only: the benchmark exits with a message before anything touches a device
    import subprocess
    import sys

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""
