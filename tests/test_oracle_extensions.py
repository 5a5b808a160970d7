"""Pins of the oracle's optional block extensions: the 3-D rotary position
embedding of the self-attention queries / keys and the cross-attention layer
to a condition token sequence (the WAN-style blocks of the paper's model,
Section 3.1; conditions injected through cross-attention, Sections 2.1 and
2.3.2).

The rotary embedding is pinned by its axis split, a worked example in complex
arithmetic with the frequencies written out by hand, the shift invariance of
rotated dot products, and whole-stream translation invariance; the
cross-attention layer by closed forms (one condition token, duplicated tokens,
permuted tokens, a zero output projection) and the whole extended block by an
element-by-element loop version on tiny shapes.
"""
import cmath
import math

import numpy as np
import pytest

import synth
from oracle import xcache_oracle as xo


def test_rope_axis_split():
    # frame axis gets d - 4 floor(d/6), rows and columns 2 floor(d/6) each
    assert xo.rope_axis_dims(128) == (44, 42, 42)
    assert xo.rope_axis_dims(64) == (24, 20, 20)
    assert xo.rope_axis_dims(32) == (12, 10, 10)
    assert xo.rope_axis_dims(12) == (4, 4, 4)


def test_rope_worked_example_in_complex_form():
    # d = 12, theta = 100: two pairs per axis with frequencies 1 and 100^(-1/2);
    # the token sits at frame 2, row 1, column 3
    x = np.arange(1.0, 13.0).reshape(1, 1, 12)
    pos = np.array([[2.0, 1.0, 3.0]])
    got = xo.apply_rope(x, pos, 100.0)[0, 0]
    omega = [1.0, 0.1, 1.0, 0.1, 1.0, 0.1]
    p = [2.0, 2.0, 1.0, 1.0, 3.0, 3.0]
    for j in range(6):
        z = complex(x[0, 0, 2 * j], x[0, 0, 2 * j + 1]) * cmath.exp(1j * p[j] * omega[j])
        assert got[2 * j] == pytest.approx(z.real, abs=1e-12)
        assert got[2 * j + 1] == pytest.approx(z.imag, abs=1e-12)


def test_rope_zero_position_is_identity_and_rotation_keeps_pair_norms():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 3, 32))
    np.testing.assert_array_equal(xo.apply_rope(x, np.zeros((5, 3)), 1e4), x)
    pos = rng.integers(0, 50, size=(5, 3)).astype(np.float64)
    y = xo.apply_rope(x, pos, 1e4)
    np.testing.assert_allclose(y[..., 0::2] ** 2 + y[..., 1::2] ** 2, x[..., 0::2] ** 2 + x[..., 1::2] ** 2,
                               rtol=1e-12)


def test_rope_scores_depend_only_on_position_differences():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((6, 2, 32))
    k = rng.standard_normal((6, 2, 32))
    pq = rng.integers(0, 40, size=(6, 3)).astype(np.float64)
    pk = rng.integers(0, 40, size=(6, 3)).astype(np.float64)
    shift = np.array([[7.0, -3.0, 11.0]])
    a = np.einsum("ihd,jhd->hij", xo.apply_rope(q, pq, 1e4), xo.apply_rope(k, pk, 1e4))
    b = np.einsum("ihd,jhd->hij", xo.apply_rope(q, pq + shift, 1e4), xo.apply_rope(k, pk + shift, 1e4))
    np.testing.assert_allclose(a, b, atol=1e-10)
    # and they do depend on the difference
    c = np.einsum("ihd,jhd->hij", xo.apply_rope(q, pq + shift, 1e4), xo.apply_rope(k, pk, 1e4))
    assert np.abs(a - c).max() > 1e-2


def test_token_positions_hand_case():
    groups = (synth.ViewGroup(2, 2, 2, 3), synth.ViewGroup(1, 1, 1, 2))
    pos = xo.token_positions(groups, 1)
    assert pos.shape == (2 * 12 + 2, 3)
    assert tuple(pos[0]) == (2, 0, 0)      # generation 1, frames per chunk 2
    assert tuple(pos[7]) == (3, 0, 1)      # f = 1, h = 0, w = 1
    assert tuple(pos[12]) == (2, 0, 0)     # second camera restarts its grid
    assert tuple(pos[24]) == (1, 0, 0)     # second group: one frame per chunk
    assert tuple(pos[25]) == (1, 0, 1)


# --- cross-attention ---------------------------------------------------------------

CROSS = synth.Workload(
    "tiny-cross",
    synth.ModelShape(2, 24, 2, 12, 16, 4, 2, synth.F32, 2, 2, (synth.ViewGroup(1, 2, 2, 2),),
                     rope=1, rope_theta=100.0, cond_len=3),
    synth.GateParams(),
    synth.StreamParams(3, 0.9, 0.05),
)


def _oracle(m, seed=3, scale=0.3):
    rng = np.random.default_rng(seed)
    blob = (rng.standard_normal(synth.weights_numel(m)) * scale).astype(np.float32)
    return xo.XCacheOracle(m, synth.GateParams(enabled=0), blob), rng


def test_single_condition_token_adds_its_projected_value_to_every_row():
    orc, rng = _oracle(CROSS.model)
    c = rng.standard_normal((1, 24))
    orc.set_condition(c)
    p = orc.blocks[0].p
    x1 = rng.standard_normal((8, 24))
    got = orc.cross_attention(0, x1) - x1
    v = c @ p["wv_c"].T + p["bv_c"]            # softmax over one key is 1
    want = v @ p["wo_c"].T + p["bo_c"]
    np.testing.assert_allclose(got, np.repeat(want, 8, axis=0), atol=1e-12)


def test_duplicated_and_permuted_condition_tokens():
    orc, rng = _oracle(CROSS.model)
    c = rng.standard_normal((3, 24))
    x1 = rng.standard_normal((8, 24))
    orc.set_condition(c)
    base = orc.cross_attention(1, x1)
    orc.set_condition(c[[2, 0, 1]])
    np.testing.assert_allclose(orc.cross_attention(1, x1), base, atol=1e-12)
    orc.set_condition(c[:1])
    one = orc.cross_attention(1, x1)
    orc.set_condition(c[[0, 0, 0]])
    np.testing.assert_allclose(orc.cross_attention(1, x1), one, atol=1e-12)


def test_zero_cross_output_projection_equals_model_without_cross_attention():
    m = CROSS.model
    m0 = synth.with_model(CROSS, cond_len=0).model
    orc, rng = _oracle(m)
    blob0 = np.zeros(synth.weights_numel(m0), np.float32)
    orc0 = xo.XCacheOracle(m0, synth.GateParams(enabled=0), blob0)
    for b in range(m.n_blocks):
        orc.blocks[b].p["wo_c"][...] = 0.0
        orc.blocks[b].p["bo_c"][...] = 0.0
        for name in orc0.blocks[b].p:
            orc0.blocks[b].p[name][...] = orc.blocks[b].p[name]
    orc.set_condition(rng.standard_normal((3, 24)))
    x = rng.standard_normal((8, 24))
    a = np.array([0.2, -0.4])
    np.testing.assert_array_equal(orc.forward_chunk(0, 700.0, a, x), orc0.forward_chunk(0, 700.0, a, x))


def test_rope_stream_is_translation_invariant_without_past_chunks():
    # a one-chunk window: generation n's attention sees only its own chunk,
    # whose frame positions all move by F from one generation to the next
    m = synth.with_model(CROSS, kv_window=1).model
    orc, rng = _oracle(m)
    orc.set_condition(rng.standard_normal((2, 24)))
    x = rng.standard_normal((8, 24))
    a = np.array([0.1, 0.3])
    outs = []
    for _n in range(3):
        outs.append(orc.forward_chunk(0, 500.0, a, x))
        orc.kv_update(0.0, a, x)
    np.testing.assert_allclose(outs[1], outs[0], atol=1e-12)
    np.testing.assert_allclose(outs[2], outs[0], atol=1e-12)
    # with a past chunk visible the positions matter
    m2 = synth.with_model(CROSS, kv_window=2).model
    o2, rng2 = _oracle(m2)
    o2.set_condition(rng2.standard_normal((2, 24)))
    o2.kv_update(0.0, a, x)
    y_rope = o2.forward_chunk(0, 500.0, a, x)
    m3 = synth.with_model(CROSS, kv_window=2, rope=0).model
    o3, rng3 = _oracle(m3)
    o3.set_condition(rng3.standard_normal((2, 24)))
    o3.kv_update(0.0, a, x)
    assert np.abs(o3.forward_chunk(0, 500.0, a, x) - y_rope).max() > 1e-6


def _loop_extended_block(m, p, x, cond, ctoks, n, theta):
    """The extended block written out element by element (tiny shapes only):
    adaLN, self-attention with the 3-D rotary embedding (frame position n F + f),
    cross-attention to ctoks, MLP."""
    L, C, H, d = m.tokens, m.hidden, m.n_heads, m.head_dim
    g = m.groups[0]
    sil = [c / (1 + math.exp(-c)) for c in cond]
    mod = [sum(p["w_ada"][i][j] * sil[j] for j in range(len(cond))) + p["b_ada"][i] for i in range(6 * C)]
    sh1, sc1, g1, sh2, sc2, g2 = (mod[i * C:(i + 1) * C] for i in range(6))

    def norm(row):
        mu = sum(row) / C
        var = sum((r - mu) ** 2 for r in row) / C
        return [(row[c] - mu) / math.sqrt(var + 1e-6) for c in range(C)]

    def lin(vec, w, bias):
        return [sum(w[o][i] * vec[i] for i in range(len(vec))) + bias[o] for o in range(len(bias))]

    def rms(vec, gain):
        r = math.sqrt(sum(v * v for v in vec) / len(vec) + 1e-6)
        return [vec[i] / r * gain[i] for i in range(len(vec))]

    # d = 12: pairs (0,1), (2,3) follow the frame axis, (4,5), (6,7) the row
    # axis, (8,9), (10,11) the column axis; frequencies 1 and theta^(-1/2)
    freq = [1.0, theta ** -0.5] * 3
    axis = [0, 0, 1, 1, 2, 2]

    def rot(vec, t):
        f, rem = divmod(t, g.height * g.width)
        pos = (n * g.frames + f, rem // g.width, rem % g.width)
        out = list(vec)
        for j in range(6):
            ang = pos[axis[j]] * freq[j]
            a, b = vec[2 * j], vec[2 * j + 1]
            out[2 * j] = a * math.cos(ang) - b * math.sin(ang)
            out[2 * j + 1] = a * math.sin(ang) + b * math.cos(ang)
        return out

    def attend(qv, keys, vals):
        sc = [sum(qv[c] * kk[c] for c in range(d)) / math.sqrt(d) for kk in keys]
        mx = max(sc)
        w = [math.exp(s - mx) for s in sc]
        z = sum(w)
        return [sum(w[j] * vals[j][c] for j in range(len(keys))) / z for c in range(d)]

    h = [[a * (1 + s) + t for a, s, t in zip(norm(list(x[i])), sc1, sh1)] for i in range(L)]
    q = [lin(h[i], p["wq"], p["bq"]) for i in range(L)]
    k = [lin(h[i], p["wk"], p["bk"]) for i in range(L)]
    v = [lin(h[i], p["wv"], p["bv"]) for i in range(L)]
    qh = [[rot(rms(q[i][hd * d:(hd + 1) * d], p["gq"]), i) for hd in range(H)] for i in range(L)]
    kh = [[rot(rms(k[i][hd * d:(hd + 1) * d], p["gk"]), i) for hd in range(H)] for i in range(L)]
    vh = [[v[i][hd * d:(hd + 1) * d] for hd in range(H)] for i in range(L)]
    ck = [lin(c, p["wk_c"], p["bk_c"]) for c in ctoks]
    cv = [lin(c, p["wv_c"], p["bv_c"]) for c in ctoks]
    ckh = [[rms(ck[j][hd * d:(hd + 1) * d], p["gk_c"]) for hd in range(H)] for j in range(len(ctoks))]
    cvh = [[cv[j][hd * d:(hd + 1) * d] for hd in range(H)] for j in range(len(ctoks))]
    y = []
    for i in range(L):
        o = []
        for hd in range(H):
            o += attend(qh[i][hd], [kh[j][hd] for j in range(L)], [vh[j][hd] for j in range(L)])
        a = lin(o, p["wo"], p["bo"])
        x1 = [x[i][c] + g1[c] * a[c] for c in range(C)]
        hc = [a * w + b for a, w, b in zip(norm(x1), p["ln3_w"], p["ln3_b"])]
        qc = lin(hc, p["wq_c"], p["bq_c"])
        oc = []
        for hd in range(H):
            oc += attend(rms(qc[hd * d:(hd + 1) * d], p["gq_c"]), [ckh[j][hd] for j in range(len(ctoks))],
                         [cvh[j][hd] for j in range(len(ctoks))])
        ac = lin(oc, p["wo_c"], p["bo_c"])
        x1 = [x1[c] + ac[c] for c in range(C)]
        h2 = [a * (1 + s) + t for a, s, t in zip(norm(x1), sc2, sh2)]
        u = lin(h2, p["w1"], p["b1"])
        u = [0.5 * t * (1 + math.tanh(math.sqrt(2 / math.pi) * (t + 0.044715 * t ** 3))) for t in u]
        mlp = lin(u, p["w2"], p["b2"])
        y.append([x1[c] + g2[c] * mlp[c] for c in range(C)])
    return np.array(y)


def test_extended_block_matches_loop_version():
    m = CROSS.model
    orc, rng = _oracle(m, seed=5, scale=0.4)
    ctoks = rng.standard_normal((3, 24))
    orc.set_condition(ctoks)
    orc.n = 2                                   # frame positions 4 and 5
    x = rng.standard_normal((8, 24))
    cond = orc.cond(250.0, np.array([0.5, -0.7]))
    y, _ = orc.block(1, x, cond)
    p = {name: a.tolist() for name, a in orc.blocks[1].p.items()}
    want = _loop_extended_block(m, p, x.tolist(), cond.tolist(), ctoks.tolist(), 2, m.rope_theta)
    np.testing.assert_allclose(y, want, atol=1e-11)


def test_extended_zero_thresholds_equal_uncached():
    m = CROSS.model
    orc, rng = _oracle(m, seed=7, scale=0.2)
    blob = (np.random.default_rng(7).standard_normal(synth.weights_numel(m)) * 0.2).astype(np.float32)
    gated = xo.XCacheOracle(m, synth.GateParams(adaptive=0, tau_cos_fixed=2.0, tau_dev=0.0, front_anchors=0),
                            blob)
    plain = xo.XCacheOracle(m, synth.GateParams(enabled=0), blob)
    c = rng.standard_normal((3, 24))
    gated.set_condition(c)
    plain.set_condition(c)
    for n in range(3):
        x = rng.standard_normal((8, 24))
        a = rng.standard_normal(2)
        for t in range(m.n_steps):
            np.testing.assert_array_equal(gated.forward_chunk(t, 1000.0 - 400 * t, a, x),
                                          plain.forward_chunk(t, 1000.0 - 400 * t, a, x))
        gated.kv_update(0.0, a, x)
        plain.kv_update(0.0, a, x)
    assert gated.skips == 0
