"""The hand-worked gate sequences of ``gate_sequences`` through the C ABI: the
device's decisions, cosines, thresholds and EMA must be the literal values
worked out from Eq. 5, 7-9 and Section 2.5 (not only the oracle's)."""
import math

import numpy as np
import pytest

import gate_sequences as gs

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seq", gs.ALL, ids=lambda s: s.name)
def test_device_follows_hand_worked_sequence(seq):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_20289_amd.xcache import XCache
    m = gs.model()
    print(f"[gate-seq] {seq.name}", flush=True)
    xc = XCache(m, seq.gate, gs.identity_weights(m), torch.cuda.current_stream().cuda_stream)
    try:
        dev = torch.device("cuda")
        y_d = torch.empty((m.tokens, m.hidden), dtype=torch.float32, device=dev)
        for n, (x, a) in enumerate(zip(gs.latents(m, seq), gs.actions(m, seq))):
            x_d = torch.from_numpy(x).to(dev)
            xc.forward_chunk(0, 1000.0, a, x_d, y_d)
            st = xc.stats()
            np.testing.assert_array_equal(y_d.cpu().numpy(), x)     # identity blocks
            assert int(st["last_decision"][1]) == seq.decision[n], (seq.name, n, st["last_decision"])
            assert int(st["last_decision"][0]) == gs.F
            if not math.isnan(seq.s[n]):
                assert st["last_cos"][1] == pytest.approx(seq.s[n], abs=2e-6), (seq.name, n)
                assert st["last_tau"][1] == pytest.approx(seq.tau[n], abs=2e-6), (seq.name, n)
            if not math.isnan(seq.ema[n]):
                assert st["ema"][0, 1] == pytest.approx(seq.ema[n], abs=2e-6), (seq.name, n)
            xc.kv_update(0.0, a, y_d)
        st = xc.stats()
        assert st["skips"] == seq.decision.count(gs.S)
        assert st["gated_evals"] == len(seq.decision) - 1
    finally:
        xc.close()
