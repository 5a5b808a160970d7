"""The C ABI on the CPU: the library loads, exports every declared entry point,
validates its arguments before touching the GPU, and its host-side
fingerprint sampling matches the oracle bit for bit."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import synth
from oracle import xcache_oracle as xo
from paper_2604_20289_amd import xcache as xcp

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "xcache.h")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:xc_status|const char\*)\s+(xc_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_symbol():
    lib = xcp.load_library()
    names = _declared()
    assert len(names) >= 11
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(names) == sorted(xcp.EXPORTED)


def test_status_strings():
    assert xcp.xc_status_string(xcp.XC_OK) == "XC_OK"
    assert xcp.xc_status_string(xcp.XC_ERR_UNSUPPORTED) == "XC_ERR_UNSUPPORTED"
    assert xcp.xc_status_string(99) == "XC_ERR_UNKNOWN"


def _init_status(model, gate, weights=None, nbytes=None):
    lib = xcp.load_library()
    mc = xcp.model_config(model) if model is not None else None
    gc = xcp.gate_config(gate) if gate is not None else None
    if weights is None:
        weights = np.zeros(synth.weights_numel(model) if model is not None else 1, np.float32)
    h = ctypes.c_void_p()
    return lib.xc_init(ctypes.byref(mc) if mc else None, ctypes.byref(gc) if gc else None,
                       weights.ctypes.data, weights.nbytes if nbytes is None else nbytes, None, ctypes.byref(h))


W0 = synth.workload(0)


@pytest.mark.parametrize("change,want", [
    (dict(n_blocks=0), xcp.XC_ERR_INVALID_ARG),
    (dict(hidden=130), xcp.XC_ERR_INVALID_ARG),          # != heads * head_dim
    (dict(temb_dim=63), xcp.XC_ERR_INVALID_ARG),
    (dict(action_dim=65), xcp.XC_ERR_INVALID_ARG),
    (dict(dtype=7), xcp.XC_ERR_INVALID_ARG),
    (dict(n_steps=0), xcp.XC_ERR_INVALID_ARG),
    (dict(kv_window=0), xcp.XC_ERR_INVALID_ARG),
    (dict(groups=()), xcp.XC_ERR_INVALID_ARG),
    (dict(groups=(synth.ViewGroup(1, 0, 4, 4),)), xcp.XC_ERR_INVALID_ARG),
    (dict(dtype="bf16"), xcp.XC_ERR_UNSUPPORTED),         # head_dim 32 has no bf16 MFMA path
    (dict(n_heads=1, head_dim=256, hidden=256), xcp.XC_ERR_UNSUPPORTED),
    (dict(rope=2), xcp.XC_ERR_INVALID_ARG),
    (dict(rope=1, rope_theta=1.0), xcp.XC_ERR_INVALID_ARG),
    (dict(rope=1, rope_theta=math.nan), xcp.XC_ERR_INVALID_ARG),
    (dict(rope=1, groups=(synth.ViewGroup(1, 1, 1024, 1),)), xcp.XC_ERR_INVALID_ARG),
    (dict(rope=1, n_heads=8, head_dim=15, hidden=120), xcp.XC_ERR_INVALID_ARG),   # odd head_dim
    (dict(cond_len=-1), xcp.XC_ERR_INVALID_ARG),
    (dict(cond_len=4097), xcp.XC_ERR_INVALID_ARG),
])
def test_init_rejects_bad_model(change, want):
    m = synth.with_model(W0, **change).model
    weights = np.zeros(max(1, synth.weights_numel(m)) if m.n_blocks > 0 else 1, np.float32)
    assert _init_status(m, W0.gate, weights) == want


@pytest.mark.parametrize("change", [
    # 4 x 4,198,400 = 16,793,600 visible keys > 2^24: the attention kernel's V^T staging offset would wrap
    dict(kv_window=4, groups=(synth.ViewGroup(4, 1, 1024, 1025),)),
    # hidden 4096, L = 2^21: ceil(L/32) * 2 * C * 4 = 2^31 bytes of column-sum partials per kind
    dict(n_heads=32, head_dim=128, hidden=4096, kv_window=1, groups=(synth.ViewGroup(1, 1, 2048, 1024),)),
    dict(n_heads=32, head_dim=128, hidden=4096, kv_window=1, dtype="bf16",
         groups=(synth.ViewGroup(2, 1, 1024, 1024),)),
])
def test_init_rejects_shapes_past_32bit_offsets(change):
    """Shapes whose kernel offsets would not fit in 32 bits are refused before
    anything is allocated (the weight blob is not even looked at)."""
    m = synth.with_model(W0, **change).model
    assert _init_status(m, W0.gate, np.zeros(1, np.float32)) == xcp.XC_ERR_UNSUPPORTED
    # one fewer camera row / window chunk is inside the limits: validation then reaches the size check
    smaller = dict(change)
    if change["kv_window"] > 1:
        smaller["kv_window"] = 3
    else:
        g = change["groups"][0]
        smaller["groups"] = (synth.ViewGroup(g.views, g.frames, g.height - 1, g.width),)
    m2 = synth.with_model(W0, **smaller).model
    assert _init_status(m2, W0.gate, np.zeros(1, np.float32)) == xcp.XC_ERR_INVALID_ARG


@pytest.mark.parametrize("change,want", [
    (dict(kv_protect=0), xcp.XC_ERR_UNSUPPORTED),
    (dict(kv_protect=2), xcp.XC_ERR_INVALID_ARG),
    (dict(warmup=0), xcp.XC_ERR_INVALID_ARG),
    (dict(alpha=1.5), xcp.XC_ERR_INVALID_ARG),
    (dict(step0_mode=3), xcp.XC_ERR_INVALID_ARG),
    (dict(fp_mode=2), xcp.XC_ERR_INVALID_ARG),
    (dict(fp_refresh=2), xcp.XC_ERR_INVALID_ARG),
    (dict(fp_budget=0), xcp.XC_ERR_INVALID_ARG),
    (dict(tau_floor=math.nan), xcp.XC_ERR_INVALID_ARG),
    (dict(eps=-1.0), xcp.XC_ERR_INVALID_ARG),
    (dict(max_stale=-1), xcp.XC_ERR_INVALID_ARG),
    (dict(enabled=2), xcp.XC_ERR_INVALID_ARG),
])
def test_init_rejects_bad_gate(change, want):
    g = synth.with_gate(W0, **change).gate
    assert _init_status(W0.model, g) == want


def test_init_rejects_null_and_size_mismatch():
    lib = xcp.load_library()
    assert _init_status(None, W0.gate) == xcp.XC_ERR_INVALID_ARG
    assert _init_status(W0.model, None) == xcp.XC_ERR_INVALID_ARG
    w = np.zeros(synth.weights_numel(W0.model), np.float32)
    assert _init_status(W0.model, W0.gate, w, w.nbytes - 4) == xcp.XC_ERR_INVALID_ARG
    mc, gc = xcp.model_config(W0.model), xcp.gate_config(W0.gate)
    assert lib.xc_init(ctypes.byref(mc), ctypes.byref(gc), w.ctypes.data, w.nbytes, None, None) == \
        xcp.XC_ERR_INVALID_ARG
    assert lib.xc_init(ctypes.byref(mc), ctypes.byref(gc), None, w.nbytes, None,
                       ctypes.byref(ctypes.c_void_p())) == xcp.XC_ERR_INVALID_ARG


def test_calls_on_null_handle():
    lib = xcp.load_library()
    a = np.zeros(8, np.float32)
    assert lib.xc_forward_chunk(None, 0, 1.0, a.ctypes.data, 1, 1, 0) == xcp.XC_ERR_INVALID_ARG
    assert lib.xc_kv_update(None, 0.0, a.ctypes.data, 1, None) == xcp.XC_ERR_INVALID_ARG
    assert lib.xc_stats(None, None, None, None, None, None, None, None) == xcp.XC_ERR_INVALID_ARG
    assert lib.xc_reset(None) == xcp.XC_ERR_INVALID_ARG
    assert lib.xc_destroy(None) == xcp.XC_OK
    assert lib.xc_axpby(None, 1.0, 1, 1.0, 1, 1, 4) == xcp.XC_ERR_INVALID_ARG
    assert lib.xc_profile(None, 1) == xcp.XC_ERR_INVALID_ARG
    assert lib.xc_set_condition(None, a.ctypes.data, 1) == xcp.XC_ERR_INVALID_ARG
    assert lib.xc_forward_chunk_noalloc(None, 0, 1.0, a.ctypes.data, 1, 1, 0) == xcp.XC_ERR_INVALID_ARG
    assert lib.xc_read_cache(None, xcp.XC_CACHE_KEYS, 0, 0, 1, 1) == xcp.XC_ERR_INVALID_ARG


def test_measurement_aids_reject_bad_arguments():
    """Checked before any HIP call: runs without a GPU."""
    lib = xcp.load_library()
    t = ctypes.c_double(-1.0)
    assert lib.xc_mfma_rate(0, 1, None, None) == xcp.XC_ERR_INVALID_ARG
    assert lib.xc_mfma_rate(5, 1, None, ctypes.byref(t)) == xcp.XC_ERR_INVALID_ARG
    assert lib.xc_mfma_rate(-1, 0, None, ctypes.byref(t)) == xcp.XC_ERR_INVALID_ARG
    assert lib.xc_lds_dma_rate(128, None, None) == xcp.XC_ERR_INVALID_ARG
    assert lib.xc_lds_dma_rate(96, None, ctypes.byref(t)) == xcp.XC_ERR_INVALID_ARG


def test_weight_blob_size_includes_cross_attention_tensors():
    m = synth.with_model(W0, cond_len=16).model
    short = np.zeros(synth.weights_numel(W0.model), np.float32)   # the blob without the cross tensors
    assert _init_status(m, W0.gate, short) == xcp.XC_ERR_INVALID_ARG


def _variants():
    ws = [synth.workload(i) for i in range(5)]
    out = [(w.model, w.gate) for w in ws]
    two = synth.with_model(W0, groups=(synth.ViewGroup(1, 2, 4, 4), synth.ViewGroup(1, 2, 4, 4)))
    out.append((two.model, two.gate))
    out.append((W0.model, synth.with_gate(W0, fp_mode=xo.FP_LINSPACE1D).gate))
    out.append((ws[2].model, synth.with_gate(ws[2], fp_mode=xo.FP_LINSPACE1D).gate))
    split = synth.with_model(ws[3], groups=(synth.ViewGroup(2, 3, 18, 32), synth.ViewGroup(4, 3, 18, 32),
                                            synth.ViewGroup(1, 3, 18, 32)))
    out.append((split.model, split.gate))
    odd = synth.with_model(W0, groups=(synth.ViewGroup(3, 5, 7, 11), synth.ViewGroup(2, 1, 1, 40)))
    out.append((odd.model, synth.with_gate(odd, fp_budget=17).gate))
    return out


@pytest.mark.parametrize("model,gate", _variants())
def test_fingerprint_rows_match_oracle(model, gate):
    want = np.concatenate([r.reshape(-1) for r in xo.fingerprint_rows(model.groups, gate.fp_budget, gate.fp_mode)])
    got = xcp.xc_fingerprint_rows(model, gate)
    np.testing.assert_array_equal(got, want)


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU; --gpus N > 1 exits with a message before any device work."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=root)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""
