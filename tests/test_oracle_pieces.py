"""Pins of the oracle's pieces against things other than itself.

Each test checks one oracle function against a textbook value, a library
routine, a closed form or a brute-force loop on tiny inputs.
"""
import math
import os

import numpy as np
import pytest
import torch

import synth
from oracle import xcache_oracle as xo

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --- bf16 rounding ----------------------------------------------------------

def test_bf16_round_matches_torch_on_float32_values():
    rng = np.random.default_rng(5)
    x = (rng.standard_normal(200_000) * rng.choice([1e-3, 1.0, 1e3], 200_000)).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = xo.bf16_round(x.astype(np.float64))
    np.testing.assert_array_equal(got, ref)


def test_bf16_round_ties_to_even_and_exact_values():
    u = 2.0 ** -7  # bf16 spacing at 1.0
    vals = np.array([1.0, 1.0 + u / 2, 1.0 + 3 * u / 2, -1.0 - u / 2, 0.0, 1.0 + u / 2 + 1e-12])
    want = np.array([1.0, 1.0, 1.0 + 2 * u, -1.0, 0.0, 1.0 + u])
    np.testing.assert_array_equal(xo.bf16_round(vals), want)


# --- elementwise and norms ----------------------------------------------------

def test_spot_values():
    assert xo.silu(np.array(1.0)) == pytest.approx(0.7310585786300049, abs=1e-15)
    assert xo.gelu_tanh(np.array(1.0)) == pytest.approx(0.8411919906082768, abs=1e-15)
    # tanh form differs from the erf form by about 1.5e-4 at x = 1
    assert abs(xo.gelu_tanh(np.array(1.0)) - 0.8413447460685429) > 1e-4


def test_gelu_silu_match_torch():
    x = np.linspace(-8, 8, 4001)
    tx = torch.from_numpy(x)
    np.testing.assert_allclose(xo.gelu_tanh(x), torch.nn.functional.gelu(tx, approximate="tanh").numpy(),
                               rtol=0, atol=1e-14)
    np.testing.assert_allclose(xo.silu(x), torch.nn.functional.silu(tx).numpy(), rtol=0, atol=1e-14)


def test_layer_norm_and_rms_match_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 33)) * 3 + 1.5
    g = rng.standard_normal(33)
    tx = torch.from_numpy(x)
    np.testing.assert_allclose(xo.layer_norm(x), torch.nn.functional.layer_norm(tx, (33,), eps=1e-6).numpy(),
                               atol=1e-12)
    np.testing.assert_allclose(xo.rms_norm(x, g),
                               torch.nn.functional.rms_norm(tx, (33,), torch.from_numpy(g), eps=1e-6).numpy(),
                               atol=1e-12)


def test_timestep_embedding_closed_form():
    e0 = xo.timestep_embedding(0.0, 8)
    np.testing.assert_array_equal(e0, [1, 1, 1, 1, 0, 0, 0, 0])
    e = xo.timestep_embedding(1.0, 4)  # frequencies 1 and 10000^-0.5 = 0.01
    np.testing.assert_allclose(e, [math.cos(1), math.cos(0.01), math.sin(1), math.sin(0.01)], atol=1e-15)


# --- attention ------------------------------------------------------------------

def _attention_loops(q, k, v):
    out = []
    d = len(q[0])
    for qi in q:
        sc = [sum(qi[c] * kj[c] for c in range(d)) / math.sqrt(d) for kj in k]
        mx = max(sc)
        w = [math.exp(s - mx) for s in sc]
        z = sum(w)
        out.append([sum(w[j] * v[j][c] for j in range(len(k))) / z for c in range(d)])
    return np.array(out)


@pytest.mark.parametrize("lq,lk,d", [(1, 1, 4), (5, 16, 8), (16, 48, 4), (3, 7, 2)])
def test_attention_brute_force(lq, lk, d):
    rng = np.random.default_rng(lq * 100 + lk)
    q, k, v = (rng.standard_normal((n, d)) * 2 for n in (lq, lk, lk))
    np.testing.assert_allclose(xo.softmax_attention(q, k, v),
                               _attention_loops(q.tolist(), k.tolist(), v.tolist()), atol=1e-12)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None], torch.from_numpy(k)[None], torch.from_numpy(v)[None])[0].numpy()
    np.testing.assert_allclose(xo.softmax_attention(q, k, v), ref, atol=1e-12)


def test_attention_closed_forms():
    rng = np.random.default_rng(2)
    k = rng.standard_normal((9, 4))
    v = rng.standard_normal((9, 4))
    # q = 0: uniform weights -> mean of V
    np.testing.assert_allclose(xo.softmax_attention(np.zeros((2, 4)), k, v), np.tile(v.mean(0), (2, 1)), atol=1e-14)
    # identical keys: uniform weights -> mean of V
    kk = np.tile(k[:1], (9, 1))
    np.testing.assert_allclose(xo.softmax_attention(rng.standard_normal((3, 4)), kk, v),
                               np.tile(v.mean(0), (3, 1)), atol=1e-14)
    # one dominant key picks its value
    q = np.array([[50.0, 0, 0, 0]])
    k2 = np.eye(4)[[0, 1, 2, 3, 1]]
    np.testing.assert_allclose(xo.softmax_attention(q, k2, v[:5]), v[:1], atol=1e-10)


# --- fingerprint indices (Section 2.3.1) ------------------------------------------

def _golden_lines(kind):
    with open(os.path.join(GOLDEN, "fingerprint_indices.txt")) as f:
        for line in f:
            if line.startswith(kind + " "):
                lhs, rhs = line[len(kind) + 1:].split("->")
                yield [int(t) for t in lhs.split()], [int(t) for t in rhs.split()]


def test_axis_indices_golden():
    n = 0
    for (dim, k), want in _golden_lines("axis"):
        assert xo.axis_indices(dim, k) == want, (dim, k)
        n += 1
    assert n >= 8


def test_axis_counts_golden():
    n = 0
    for (F, H, W, K), want in _golden_lines("counts"):
        assert list(xo.axis_counts(F, H, W, K)) == want, (F, H, W, K)
        n += 1
    assert n >= 5


def test_fingerprint_rows_structure():
    g = synth.ViewGroup(6, 3, 15, 26)
    rows = xo.fingerprint_rows([g], 32)[0]
    assert rows.shape == (6, 40)
    T = 3 * 15 * 26
    # camera v's sample is camera 0's shifted by v*T; frame 0 only; (h, w) grid product
    for v in range(6):
        np.testing.assert_array_equal(rows[v] - v * T, rows[0])
    hs, ws = [0, 3, 7, 10, 14], [0, 3, 7, 10, 14, 17, 21, 25]
    np.testing.assert_array_equal(rows[0], [h * 26 + w for h in hs for w in ws])
    # small grids keep every token; several groups are offset by the earlier groups' tokens
    small = [synth.ViewGroup(1, 2, 4, 4), synth.ViewGroup(2, 1, 2, 3)]
    r = xo.fingerprint_rows(small, 32)
    np.testing.assert_array_equal(r[0], [list(range(32))])
    np.testing.assert_array_equal(r[1], [[32 + i for i in range(6)], [38 + i for i in range(6)]])
    # 1-D fallback: K uniformly spaced tokens along the camera's flattened axis
    r1 = xo.fingerprint_rows([synth.ViewGroup(2, 4, 4, 4)], 32, xo.FP_LINSPACE1D)[0]
    np.testing.assert_array_equal(r1[0], [(i * 63) // 31 for i in range(32)])
    np.testing.assert_array_equal(r1[1], 64 + r1[0])


def test_fingerprint_global_channel_is_camera_mean():
    groups = [synth.ViewGroup(2, 1, 3, 3), synth.ViewGroup(1, 1, 2, 2)]
    x = np.arange(22 * 3, dtype=np.float64).reshape(22, 3)
    fp = xo.fingerprint(x, groups, xo.fingerprint_rows(groups, 32))
    np.testing.assert_allclose(fp[0][1], np.concatenate([x[0:9].mean(0), x[9:18].mean(0)]))
    np.testing.assert_allclose(fp[1][1], x[18:22].mean(0))
    np.testing.assert_array_equal(fp[0][0], x[:18].reshape(-1))


# --- metrics (Eq. 5-6) ------------------------------------------------------------

def test_metric_hand_vectors():
    prev = np.array([1.0, 0, 0, 0])
    cur = np.array([0.6, 0.8, 0, 0])
    assert xo.cosine(cur, prev) == pytest.approx(0.6, abs=1e-15)
    assert xo.max_deviation(cur, prev, 1e-6) == pytest.approx(0.8 / (0.25 + 1e-6), rel=1e-14)
    assert xo.cosine(np.zeros(4), prev) == 0.0
    assert xo.cosine(-prev, prev) == -1.0


def test_metric_scale_invariance():
    rng = np.random.default_rng(3)
    a, b = rng.standard_normal(100), rng.standard_normal(100)
    assert xo.cosine(7 * a, 7 * b) == pytest.approx(xo.cosine(a, b), rel=1e-13)
    assert xo.max_deviation(7 * a, 7 * b, 0.0) == pytest.approx(xo.max_deviation(a, b, 0.0), rel=1e-13)


def test_gate_metrics_aggregation():
    e = np.eye(4)
    fp_prev = [(e[0], e[0]), (e[1], e[1])]
    # group 0 spatial cos 0.6, group 1 global cos 0.8; group 1 spatial deviation largest
    fp = [(np.array([0.6, 0.8, 0, 0]), e[0]), (np.array([0, 1.0, 3.0, 0]), np.array([0, 0.8, 0.6, 0]))]
    s, d = xo.gate_metrics(fp, fp_prev, None, None, 0.0)
    assert s == pytest.approx(min(0.6, 1 / math.sqrt(10), 0.8))
    assert d == pytest.approx(max(0.8 / 0.25, 3.0 / 0.25))
    # the action channel takes part in the min-cosine only
    s2, d2 = xo.gate_metrics(fp_prev, fp_prev, np.array([1.0, 0]), np.array([1.0, 1.0]), 0.0)
    assert s2 == pytest.approx(1 / math.sqrt(2))
    assert d2 == 0.0


# --- threshold, EMA, decision (Eq. 7-9, Section 2.5) ------------------------------

def test_threshold_and_ema_closed_forms():
    g = synth.GateParams()
    assert xo.cosine_threshold(g, None, 1) == 0.97                 # first evaluation: the floor
    assert xo.cosine_threshold(g, 0.999, 1) == pytest.approx(0.979)  # ema - m above the floor
    assert xo.cosine_threshold(g, 0.98, 1) == 0.97                  # floor binds
    strict = synth.GateParams(step0_mode=xo.STEP0_STRICT)
    assert xo.cosine_threshold(strict, 0.98, 0) == 0.999
    assert xo.cosine_threshold(strict, 0.98, 1) == 0.97
    fixed = synth.GateParams(adaptive=0, tau_cos_fixed=0.5)
    assert xo.cosine_threshold(fixed, 0.999, 2) == 0.5
    # constant s is a fixed point; two updates give the closed form
    e = None
    for _ in range(5):
        e = xo.ema_update(g, e, 0.9)
    assert e == pytest.approx(0.9, abs=1e-15)
    e = xo.ema_update(g, xo.ema_update(g, None, 0.5), 1.0)
    assert e == pytest.approx(0.3 * 1.0 + 0.7 * 0.5)


def test_skip_rule_truth_table():
    g = synth.GateParams(tau_dev=2.0)
    assert xo.skip_rule(g, 0.98, 1.0, 0.98, 0)          # s == tau skips (>=)
    assert not xo.skip_rule(g, 0.98, 2.0, 0.97, 0)      # d == tau_dev recomputes (<)
    assert not xo.skip_rule(g, 0.969, 0.1, 0.97, 0)
    assert xo.skip_rule(g, 0.99, 0.1, 0.97, 10**6)      # staleness bound off
    gm = synth.GateParams(max_stale=2)
    assert xo.skip_rule(gm, 0.99, 0.1, 0.97, 1)
    assert not xo.skip_rule(gm, 0.99, 0.1, 0.97, 2)     # at most M consecutive skips
