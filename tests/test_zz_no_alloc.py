"""xc_forward_chunk_noalloc (per-pass scratch in the library's static device
array) against xc_forward_chunk (the handle's own buffers): two handles with
the same model, weights and inputs run the same passes, one through each
entry point; every pass output must agree to the parity bar (relative L2
2e-2 for bf16) and every decision must be the same.

First the multi-camera shapes (one block, 7020 tokens, window of 3 chunks):
at 21060 keys the attention's unconstrained key split needs more partials
than the static array holds, so the no-alloc pass splits less.  Then a
smaller model (768 tokens, two blocks, natural skips), whose passes find the
array holding the first model's contents."""
import math

import numpy as np
import pytest

import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _pair_run(w, n_chunks, steps):
    from lockstep import rel_l2
    from paper_2604_20289_amd.xcache import XCache
    m = w.model
    blob = synth.make_weights(m)
    stream = torch.cuda.current_stream().cuda_stream
    ref = XCache(m, w.gate, blob, stream)
    noa = XCache(m, w.gate, blob, stream)
    worst = 0.0
    try:
        dev = torch.device("cuda")
        L, C = m.tokens, m.hidden
        y_r = torch.empty((L, C), dtype=torch.float32, device=dev)
        y_n = torch.empty_like(y_r)
        taus = synth.timesteps(m)
        eps = synth.latent_stream(m, w.stream, 0, n_chunks)
        acts = synth.action_stream(m, w.stream, 0, n_chunks)
        for n, e, a in zip(range(n_chunks), eps, acts):
            x = torch.from_numpy(e).to(dev)
            for t in steps:
                ref.forward_chunk(t, taus[t], a, x, y_r)
                noa.forward_chunk_noalloc(t, taus[t], a, x, y_n)
                s_r, s_n = ref.stats(), noa.stats()
                np.testing.assert_array_equal(s_r["last_decision"], s_n["last_decision"])
                err = rel_l2(y_n.cpu().numpy(), y_r.cpu().numpy())
                res = rel_l2((y_n - x).cpu().numpy(), (y_r - x).cpu().numpy())
                worst = max(worst, err, res)
                print(f"[no-alloc] {w.name} n={n} t={t} rel-L2 y {err:.2e} y-x {res:.2e} "
                      f"decisions {s_n['last_decision'].tolist()}", flush=True)
                assert err <= 2e-2 and res <= 2e-2
            ref.kv_update(0.0, a, y_r)
            noa.kv_update(0.0, a, y_r)
        s_r, s_n = ref.stats(), noa.stats()
        for k in ("skips", "gated_evals", "evals_post_warmup"):
            assert s_r[k] == s_n[k], k
        np.testing.assert_array_equal(s_r["skip_counts"], s_n["skip_counts"])
        return s_n, worst
    finally:
        ref.close()
        noa.close()


def test_no_alloc_entry_point_matches_forward_chunk():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    # 1) multi-camera shapes, one block that always computes (the gate is evaluated and fails)
    big = synth.with_model(synth.with_gate(synth.workload(2), front_anchors=0, adaptive=0, tau_cos_fixed=2.0),
                           n_blocks=1)
    st, worst = _pair_run(big, 3, [0])
    assert st["skips"] == 0 and st["gated_evals"] == 2
    # 2) a smaller model right after: single-camera shapes, two blocks, Table 1 gate with natural skips
    small = synth.with_stream(synth.with_model(synth.workload(1), n_blocks=2), rho=0.999)
    st, worst2 = _pair_run(small, 3, range(small.model.n_steps))
    print(f"[no-alloc] skips {st['skips']} worst rel-L2 {max(worst, worst2):.2e}", flush=True)
    assert st["skips"] > 0


def test_no_alloc_entry_point_errors_change_nothing():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_20289_amd import xcache as xcp
    w = synth.workload(0)
    m = w.model
    xc = xcp.XCache(m, w.gate, synth.make_weights(m), torch.cuda.current_stream().cuda_stream)
    try:
        x = torch.zeros((m.tokens, m.hidden), dtype=torch.float32, device="cuda")
        with pytest.raises(xcp.XCacheError) as e:
            xc.forward_chunk_noalloc(m.n_steps, 0.0, np.zeros(m.action_dim), x, x)
        assert e.value.status == xcp.XC_ERR_INVALID_ARG
        with pytest.raises(xcp.XCacheError) as e:
            xc.forward_chunk_noalloc(0, math.nan, np.zeros(m.action_dim), x, x)
        assert e.value.status == xcp.XC_ERR_INVALID_ARG
        assert xc.stats()["last_step"] == -1
    finally:
        xc.close()
