"""Pins of the oracle's gate state over several evaluations of one (t, b):
the order in which the threshold reads the EMA (Section 2.4, Eq. 8-9), the
action channel inside the min-cosine (Section 2.3.2, Eq. 5) and the staleness
count that every recompute restarts (Section 2.5).  The expected values are
hand-worked literals in ``gate_sequences``; the streams make each block the
identity so that the cosines are the chosen ones.
"""
import math

import numpy as np
import pytest

import gate_sequences as gs
from oracle import xcache_oracle as xo


def run_oracle(seq):
    m = gs.model()
    orc = xo.XCacheOracle(m, seq.gate, gs.identity_weights(m))
    got = []
    for x, a in zip(gs.latents(m, seq), gs.actions(m, seq)):
        y = orc.forward_chunk(0, 1000.0, a, x.astype(np.float64))
        np.testing.assert_array_equal(y, x)         # identity blocks, skipped or not
        info = orc.last[1]
        ema = orc.ema.get((0, 1), math.nan)
        got.append((info["decision"], info["s"], info["tau"], ema))
        orc.kv_update(0.0, a, y)
    return orc, got


@pytest.mark.parametrize("seq", gs.ALL, ids=lambda s: s.name)
def test_hand_worked_sequence(seq):
    orc, got = run_oracle(seq)
    assert [g[0] for g in got] == seq.decision
    for n, (dec, s, tau, ema) in enumerate(got):
        for name, val, want in (("s", s, seq.s[n]), ("tau", tau, seq.tau[n]), ("ema", ema, seq.ema[n])):
            if math.isnan(want):
                assert math.isnan(val), (seq.name, n, name, val)
            else:
                assert val == pytest.approx(want, abs=1e-6), (seq.name, n, name, val, want)
    st = orc.stats()
    assert st["skips"] == seq.decision.count(gs.S)
    assert st["gated_evals"] == len(seq.decision) - 1
    assert orc.last[0]["decision"] == xo.DEC_FORCED           # the front anchor


def test_planted_mistakes_fail_the_sequences(monkeypatch):
    """Each mistake the sequences exist to catch, planted in the oracle, changes
    at least one hand-worked decision."""
    def fails(seq):
        try:
            _, got = run_oracle(seq)
        except AssertionError:
            return True
        return [g[0] for g in got] != seq.decision

    orig_thr, orig_metrics, orig_rule = xo.cosine_threshold, xo.gate_metrics, xo.skip_rule

    # (a) the threshold reads the EMA after this evaluation's update
    with monkeypatch.context() as mp:
        state = {}

        def thr_after_update(g, ema, t):
            s = state["s"]
            return orig_thr(g, xo.ema_update(g, ema, s), t)

        def metrics_spy(*a, **k):
            s, d = orig_metrics(*a, **k)
            state["s"] = s
            return s, d
        mp.setattr(xo, "cosine_threshold", thr_after_update)
        mp.setattr(xo, "gate_metrics", metrics_spy)
        assert fails(gs.EMA_ORDER)

    # (b) the action channel left out of the min-cosine
    with monkeypatch.context() as mp:
        mp.setattr(xo, "gate_metrics", lambda fp, fp0, a, a0, eps: orig_metrics(fp, fp0, None, None, eps))
        assert fails(gs.ACTION_CHANNEL)

    # (c) the staleness count never restarted by a recompute
    with monkeypatch.context() as mp:
        class NoReset(np.ndarray):
            def __setitem__(self, key, value):
                if np.all(np.asarray(value) == 0):
                    return
                super().__setitem__(key, value)

        orig_reset = xo.XCacheOracle.reset

        def reset(self):
            orig_reset(self)
            self.stale = self.stale.view(NoReset)
        mp.setattr(xo.XCacheOracle, "reset", reset)
        assert fails(gs.STALE_M2) and fails(gs.STALE_M1)

    # (d) alpha applied to the old EMA instead of the new cosine
    with monkeypatch.context() as mp:
        mp.setattr(xo, "ema_update", lambda g, ema, s: s if ema is None else (1 - g.alpha) * s + g.alpha * ema)
        assert fails(gs.EMA_ORDER)

    # (e) the action compared with the first generation's instead of the previous one's
    with monkeypatch.context() as mp:
        orig_kv = xo.XCacheOracle.kv_update

        def kv_keep_first(self, tau, action, x, rows=None):
            first = self.action_prev
            out = orig_kv(self, tau, action, x, rows)
            if first is not None:
                self.action_prev = first
            return out
        mp.setattr(xo.XCacheOracle, "kv_update", kv_keep_first)
        assert fails(gs.ACTION_CHANNEL)
    assert xo.skip_rule is orig_rule
