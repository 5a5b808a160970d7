"""Pins of the oracle's block and of its cached rollout (whole-stream invariants).

The DiT block is checked against a pure-Python loop version on tiny shapes;
the rollout against invariants the method fixes: thresholds at zero give no
skips and the uncached output, a skipped block adds exactly its cached
residual, the KV-update pass is never gated, warmup/anchor/step-0/staleness
rules, FIFO eviction and the order-independence of the key/value window.
"""
import math

import numpy as np
import pytest

import synth
from oracle import xcache_oracle as xo

TINY = synth.Workload(
    "tiny",
    synth.ModelShape(2, 4, 2, 2, 8, 4, 2, synth.F32, 2, 2, (synth.ViewGroup(1, 1, 1, 3),)),
    synth.GateParams(),
    synth.StreamParams(3, 0.9, 0.05),
)


def _loop_block(m, p, x, cond, past):
    """The block written out element by element (tiny shapes only)."""
    L, C, H, d, Dm = m.tokens, m.hidden, m.n_heads, m.head_dim, m.mlp_hidden
    sil = [c / (1 + math.exp(-c)) for c in cond]
    mod = [sum(p["w_ada"][i][j] * sil[j] for j in range(len(cond))) + p["b_ada"][i] for i in range(6 * C)]
    sh1, sc1, g1, sh2, sc2, g2 = (mod[i * C:(i + 1) * C] for i in range(6))

    def ln_mod(row, sc, sh):
        mu = sum(row) / C
        var = sum((r - mu) ** 2 for r in row) / C
        return [(row[c] - mu) / math.sqrt(var + 1e-6) * (1 + sc[c]) + sh[c] for c in range(C)]

    def lin(vec, w, bias):
        return [sum(w[o][i] * vec[i] for i in range(len(vec))) + bias[o] for o in range(len(bias))]

    def rms(vec, gain):
        r = math.sqrt(sum(v * v for v in vec) / len(vec) + 1e-6)
        return [vec[i] / r * gain[i] for i in range(len(vec))]

    h = [ln_mod(list(x[i]), sc1, sh1) for i in range(L)]
    q = [lin(h[i], p["wq"], p["bq"]) for i in range(L)]
    k = [lin(h[i], p["wk"], p["bk"]) for i in range(L)]
    v = [lin(h[i], p["wv"], p["bv"]) for i in range(L)]
    qh = [[rms(q[i][hd * d:(hd + 1) * d], p["gq"]) for hd in range(H)] for i in range(L)]
    kh = [[rms(k[i][hd * d:(hd + 1) * d], p["gk"]) for hd in range(H)] for i in range(L)]
    vh = [[v[i][hd * d:(hd + 1) * d] for hd in range(H)] for i in range(L)]
    y = []
    for i in range(L):
        o = []
        for hd in range(H):
            keys = [pk[hd][j] for pk, _ in past for j in range(L)] + [kh[j][hd] for j in range(L)]
            vals = [pv[hd][j] for _, pv in past for j in range(L)] + [vh[j][hd] for j in range(L)]
            sc = [sum(qh[i][hd][c] * kk[c] for c in range(d)) / math.sqrt(d) for kk in keys]
            mx = max(sc)
            w = [math.exp(s - mx) for s in sc]
            z = sum(w)
            o += [sum(w[j] * vals[j][c] for j in range(len(keys))) / z for c in range(d)]
        a = lin(o, p["wo"], p["bo"])
        x1 = [x[i][c] + g1[c] * a[c] for c in range(C)]
        h2 = ln_mod(x1, sc2, sh2)
        u = lin(h2, p["w1"], p["b1"])
        u = [0.5 * t * (1 + math.tanh(math.sqrt(2 / math.pi) * (t + 0.044715 * t ** 3))) for t in u]
        mlp = lin(u, p["w2"], p["b2"])
        y.append([x1[c] + g2[c] * mlp[c] for c in range(C)])
    return np.array(y)


def test_block_matches_loop_version():
    m = TINY.model
    rng = np.random.default_rng(11)
    blob = (rng.standard_normal(synth.weights_numel(m)) * 0.7).astype(np.float32)
    orc = xo.XCacheOracle(m, TINY.gate, blob)
    x = rng.standard_normal((3, 4))
    cond = orc.cond(300.0, np.array([0.3, -1.2]))
    past = [(rng.standard_normal((2, 3, 2)), rng.standard_normal((2, 3, 2)))]
    orc.ring[1] = list(past)
    y, (k, v) = orc.block(1, x, cond)
    p = {n: a.tolist() for n, a in orc.blocks[1].p.items()}
    want = _loop_block(m, p, x.tolist(), cond.tolist(), [(pk.tolist(), pv.tolist()) for pk, pv in past])
    np.testing.assert_allclose(y, want, atol=1e-12)
    assert k.shape == (2, 3, 2) and v.shape == (2, 3, 2)


def test_block_weight_layout_is_out_by_in():
    """Wq[i, j] couples input channel j to output channel i (y = x W^T + b)."""
    m = TINY.model
    blob = np.zeros(synth.weights_numel(m), np.float32)
    orc = xo.XCacheOracle(m, TINY.gate, blob)
    p = orc.blocks[0].p
    p["b_ada"][2 * 4:3 * 4] = 1.0        # gate1 = 1, every other modulation 0
    p["wv"][0, 3] = 1.0                  # v channel 0 <- h channel 3
    p["wo"][2, 0] = 1.0                  # out channel 2 <- o channel 0
    x = np.array([[0.0, 0.0, 0.0, 2.0], [0.0, 0.0, 0.0, 2.0], [0.0, 0.0, 0.0, 2.0]]) + np.arange(3)[:, None]
    y, _ = orc.block(0, x, orc.cond(0.0, np.zeros(2)))
    h3 = xo.layer_norm(x)[:, 3]
    # identical rows in h -> every query sees identical values -> o channel 0 = h channel 3
    np.testing.assert_allclose(y - x, np.outer(h3, [0, 0, 1, 0]), atol=1e-12)


def test_zero_adaln_makes_every_block_identity():
    w = synth.workload(0)
    blob = synth.make_weights(w.model)
    for b in range(w.model.n_blocks):
        t = synth.split_block_weights(w.model, blob, b)
        t["w_ada"][...] = 0
        t["b_ada"][...] = 0
    orc = xo.XCacheOracle(w.model, synth.GateParams(enabled=0), blob)
    x = np.random.default_rng(0).standard_normal((64, 128))
    np.testing.assert_array_equal(orc.forward_chunk(0, 1000.0, np.ones(8), x), x)
    np.testing.assert_array_equal(orc.kv_update(0.0, np.ones(8), x), x)


def test_bf16_rounding_points_are_bf16_values():
    w = synth.workload(1)
    m = synth.with_model(w, n_blocks=2, hidden=64, n_heads=2, head_dim=32, mlp_hidden=128,
                         groups=(synth.ViewGroup(1, 3, 4, 4),)).model
    orc = xo.XCacheOracle(m, w.gate, synth.make_weights(m))
    x = np.random.default_rng(0).standard_normal((48, 64))
    a = np.zeros(16)
    orc.forward_chunk(0, 1000.0, a, x)
    orc.kv_update(0.0, a, x)
    for arr in [orc.ring[1][0][0], orc.ring[1][0][1], orc.rhat[(0, 1)], orc.blocks[0].p["wq"]]:
        np.testing.assert_array_equal(xo.bf16_round(arr), arr)


# --- whole-stream invariants -----------------------------------------------------

def _run(w, n_chunks=None, seed=0, weights=None, kv_input=None, flags=lambda n, t: 0):
    m = w.model
    n_chunks = n_chunks or w.stream.n_chunks
    blob = synth.make_weights(m, seed) if weights is None else weights
    orc = xo.XCacheOracle(m, w.gate, blob)
    eps = list(synth.latent_stream(m, w.stream, seed, n_chunks))
    acts = list(synth.action_stream(m, w.stream, seed, n_chunks))
    taus = synth.timesteps(m)
    passes, records = [], []
    for n in range(n_chunks):
        x = eps[n].astype(np.float64)
        for t in range(m.n_steps):
            y = orc.forward_chunk(t, taus[t], acts[n], x, flags(n, t))
            passes.append(y)
            records.append((n, t, orc.last))
            if t + 1 < m.n_steps:
                sg = synth.sampler_sigma(m, t + 1)
                x = (1 - sg) * y + sg * eps[n]
        clean = y if kv_input is None else kv_input(n, eps[n])
        passes.append(orc.kv_update(0.0, acts[n], clean))
    return orc, passes, records


def test_zero_thresholds_equal_uncached():
    w = synth.workload(0)
    orc, p_gate, rec = _run(synth.with_gate(w, adaptive=0, tau_cos_fixed=0.0, tau_dev=0.0))
    _, p_off, _ = _run(synth.with_gate(w, enabled=0))
    assert orc.skips == 0
    for a, b in zip(p_gate, p_off):
        np.testing.assert_array_equal(a, b)


def test_always_skip_adds_cached_residual_exactly():
    w = synth.with_gate(synth.workload(0), adaptive=0, tau_cos_fixed=-1.0, tau_dev=math.inf, front_anchors=0)
    m = w.model
    orc = xo.XCacheOracle(m, w.gate, synth.make_weights(m))
    eps = list(synth.latent_stream(m, w.stream, 0, 2))
    acts = list(synth.action_stream(m, w.stream, 0, 2))
    orc.forward_chunk(0, 1000.0, acts[0], eps[0])
    orc.kv_update(0.0, acts[0], eps[0])
    x = eps[1].astype(np.float64)
    y = orc.forward_chunk(0, 1000.0, acts[1], x)
    assert [r["decision"] for r in orc.last] == [xo.DEC_SKIP] * m.n_blocks
    want = x.copy()
    for b in range(m.n_blocks):
        want = want + orc.rhat[(0, b)]
    np.testing.assert_array_equal(y, want)


def test_kv_update_is_never_gated():
    base = synth.workload(0)
    skip_all = synth.with_gate(base, adaptive=0, tau_cos_fixed=-1.0, tau_dev=math.inf, front_anchors=0)
    feed = lambda n, eps: eps.astype(np.float64)  # same clean latent on both sides keeps the rings equal
    o1, p1, r1 = _run(skip_all, 4, kv_input=feed)
    o2, p2, _ = _run(synth.with_gate(base, enabled=0), 4, kv_input=feed)
    S = base.model.n_steps
    assert o1.skips == base.model.n_blocks * S * 3
    for n in range(4):
        np.testing.assert_array_equal(p1[n * (S + 1) + S], p2[n * (S + 1) + S])
    assert o1.kv_block_evals == 4 * base.model.n_blocks


def test_identical_chunks_skip_everything_after_warmup():
    # one visible chunk (no past keys), frozen noise and action: every chunk repeats the first
    w = synth.with_stream(synth.with_model(synth.workload(0), kv_window=1), rho=1.0, action_sigma=0.0)
    orc, p_gate, rec = _run(w, 4)
    _, p_off, _ = _run(synth.with_gate(w, enabled=0), 4)
    B, S = w.model.n_blocks, w.model.n_steps
    for n, t, r in rec:
        want = [xo.DEC_FORCED] * B if n == 0 else [xo.DEC_FORCED] + [xo.DEC_SKIP] * (B - 1)
        assert [x["decision"] for x in r] == want
        if n > 0:
            assert r[1]["s"] == pytest.approx(1.0, abs=1e-12) and r[1]["d"] < 1e-12
    assert orc.skips == (B - 1) * S * 3
    assert orc.evals_post_warmup == B * S * 3
    for a, b in zip(p_gate, p_off):
        np.testing.assert_allclose(a, b, atol=1e-12)


def test_warmup_anchor_step0_staleness_rules():
    w = synth.with_stream(synth.workload(0), rho=0.999)
    # a 4-block model with both anchors, M = 1, strict step 0 never passes 0.999 here
    w = synth.with_model(w, n_blocks=4)
    w = synth.with_gate(w, adaptive=1, tau_floor=0.9, tau_dev=2.0, back_anchors=1, max_stale=1,
                        warmup=2, step0_mode=xo.STEP0_FORCE)
    orc, _, rec = _run(w, 6)
    prev = {}
    skipped_any = False
    for n, t, r in rec:
        dec = [x["decision"] for x in r]
        assert dec[0] == xo.DEC_FORCED and dec[-1] == xo.DEC_FORCED    # anchors
        if n < 2 or t == 0:
            assert dec == [xo.DEC_FORCED] * 4                           # warmup, step-0 force
        for b in (1, 2):
            if dec[b] == xo.DEC_SKIP:
                skipped_any = True
                assert prev.get((t, b)) != xo.DEC_SKIP                  # M = 1
            prev[(t, b)] = dec[b]
    assert skipped_any


def test_force_full_flag_computes_and_refreshes():
    w = synth.with_stream(synth.with_gate(synth.workload(0), adaptive=1, tau_floor=0.9, tau_dev=2.0), rho=0.999)
    orc, _, rec = _run(w, 4, flags=lambda n, t: xo.FORCE_FULL if n == 2 else 0)
    for n, t, r in rec:
        if n == 2:
            assert all(x["decision"] == xo.DEC_FORCED for x in r)
    assert any(x["decision"] == xo.DEC_SKIP for n, t, r in rec if n == 3 for x in r)


def test_fingerprint_refresh_modes():
    """Every evaluation replaces the cached fingerprint by default; in the
    refresh-on-compute mode a skipped evaluation leaves the one of the last
    computed pass (here chunk 0, since every later gated evaluation skips)."""
    import copy
    base = synth.with_stream(synth.with_gate(synth.workload(0), adaptive=0, tau_cos_fixed=-1.0, tau_dev=math.inf,
                                             front_anchors=0), rho=0.9)
    snaps = {}
    for mode in (xo.FP_REFRESH_EVERY, xo.FP_REFRESH_ON_COMPUTE):
        w = synth.with_gate(base, fp_refresh=mode)
        m = w.model
        orc = xo.XCacheOracle(m, w.gate, synth.make_weights(m))
        eps = list(synth.latent_stream(m, w.stream, 0, 3))
        acts = list(synth.action_stream(m, w.stream, 0, 3))
        after0, svals = None, []
        for n in range(3):
            x = eps[n].astype(np.float64)
            for t in range(m.n_steps):
                y = orc.forward_chunk(t, 1000.0 * (1 - t / m.n_steps), acts[n], x)
                if n > 0:
                    assert all(r["decision"] == xo.DEC_SKIP for r in orc.last)
                    svals.append(orc.last[0]["s"])
                x = y
            orc.kv_update(0.0, acts[n], y)
            if n == 0:
                after0 = copy.deepcopy(orc.fp_prev)
        same = all(np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
                   for k in after0 for a, b in zip(after0[k], orc.fp_prev[k]))
        assert same == (mode == xo.FP_REFRESH_ON_COMPUTE)
        snaps[mode] = svals
    # chunk 1 compares with chunk 0 in both modes; chunk 2 with chunk 1 (every) or chunk 0 (on compute)
    S = base.model.n_steps
    assert snaps[0][:S] == snaps[1][:S]
    assert snaps[0][S:] != snaps[1][S:]


def test_fifo_eviction_keeps_last_window():
    w = synth.with_model(synth.workload(0), kv_window=3)
    m = w.model
    orc = xo.XCacheOracle(m, synth.GateParams(enabled=0), synth.make_weights(m))
    clean = [np.random.default_rng(n).standard_normal((64, 128)) for n in range(5)]
    kvs = []
    for n in range(5):
        c = orc.cond(0.0, np.zeros(8))
        _, kv = orc.block(0, clean[n], c)   # block 0's K/V of this chunk, given the ring so far
        orc.kv_update(0.0, np.zeros(8), clean[n])
        kvs.append(kv)
        assert len(orc.ring[0]) == min(n + 1, 2)
        for got, want in zip(orc.ring[0], kvs[-2:]):
            np.testing.assert_array_equal(got[0], want[0])
            np.testing.assert_array_equal(got[1], want[1])


def test_window_order_does_not_matter():
    w = synth.with_model(synth.workload(0), kv_window=3)
    m = w.model
    orc = xo.XCacheOracle(m, synth.GateParams(enabled=0), synth.make_weights(m))
    rng = np.random.default_rng(4)
    for n in range(2):
        orc.kv_update(0.0, np.zeros(8), rng.standard_normal((64, 128)))
    x = rng.standard_normal((64, 128))
    y1 = orc.forward_chunk(1, 750.0, np.zeros(8), x)
    for b in range(m.n_blocks):
        orc.ring[b].reverse()
    y2 = orc.forward_chunk(1, 750.0, np.zeros(8), x)
    np.testing.assert_allclose(y1, y2, atol=1e-12)
    assert not np.allclose(y1, x)


def test_skip_rate_denominator_counts_all_blocks_after_warmup():
    w = synth.with_stream(synth.with_gate(synth.workload(0), adaptive=1, tau_floor=0.9, tau_dev=2.0), rho=0.999)
    orc, _, rec = _run(w, 5)
    B, S = w.model.n_blocks, w.model.n_steps
    assert orc.evals_post_warmup == B * S * 4
    assert orc.skips == sum(1 for n, t, r in rec for x in r if x["decision"] == xo.DEC_SKIP)
    assert orc.skips > 0


def test_row_restricted_checking_mode():
    """The oracle's row-restricted mode returns exactly the selected rows of the full computation
    (a block's output row depends on the other tokens only through keys and values)."""
    w = synth.with_stream(synth.with_gate(synth.workload(0), adaptive=1, tau_floor=0.9, tau_dev=2.0), rho=0.999)
    m = w.model
    blob = synth.make_weights(m)
    rows = np.array([0, 5, 17, 33, 63])
    full = xo.XCacheOracle(m, w.gate, blob)
    part = xo.XCacheOracle(m, w.gate, blob)
    taus = synth.timesteps(m)
    for n, (eps, a) in enumerate(zip(synth.latent_stream(m, w.stream, 0, 3), synth.action_stream(m, w.stream, 0, 3))):
        y_full = full.forward_chunk(0, taus[0], a, eps)
        y_part = part.forward_chunk(0, taus[0], a, eps, rows=rows)
        np.testing.assert_allclose(y_part, y_full[rows], rtol=1e-12, atol=1e-12)
        assert [i["decision"] for i in full.last] == [i["decision"] for i in part.last]
        # the restricted pass left the last block's residual cache alone: continue both on the full path
        part.rhat = {k: v.copy() for k, v in full.rhat.items()}
        k_full = full.kv_update(0.0, a, y_full)
        k_part = part.kv_update(0.0, a, y_full, rows=rows)
        np.testing.assert_allclose(k_part, k_full[rows], rtol=1e-12, atol=1e-12)
        for b in range(m.n_blocks):
            for (k1, v1), (k2, v2) in zip(full.ring[b], part.ring[b]):
                np.testing.assert_array_equal(k1, k2)
                np.testing.assert_array_equal(v1, v2)
