"""GPU parity: the HIP library against the CPU oracle, pass by pass.

fp32 model: max-abs 1e-4 on every pass output.  bf16 models: relative L2
2e-2.  Decisions must agree wherever a metric is outside a relative 1e-3 band
around its threshold (see ``lockstep``)."""
import dataclasses
import math

import numpy as np
import pytest

import synth
from oracle import xcache_oracle as xo

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

W0 = synth.workload(0)
W1 = synth.workload(1)
TOL32 = 1e-4
TOLBF = 2e-2


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _ls(w, **kw):
    _need_gpu()
    from lockstep import Lockstep
    print(f"[parity] {w.name} gate={w.gate} stream={w.stream}", flush=True)
    return Lockstep(w, **kw)


CFG0_VARIANTS = {
    "stated-0.05": W0,
    "zero-thresholds": synth.with_gate(W0, adaptive=0, tau_cos_fixed=0.0, tau_dev=0.0),
    "always-skip": synth.with_gate(W0, adaptive=0, tau_cos_fixed=-1.0, tau_dev=math.inf),
    "table1": synth.with_gate(W0, adaptive=1, tau_floor=0.97, tau_dev=2.0),
    "table1-rho0.999": synth.with_stream(synth.with_gate(W0, adaptive=1, tau_floor=0.97, tau_dev=2.0), rho=0.999),
    "two-groups": synth.with_stream(synth.with_model(
        synth.with_gate(W0, adaptive=1, tau_floor=0.97, tau_dev=2.0),
        groups=(synth.ViewGroup(1, 2, 4, 4), synth.ViewGroup(1, 2, 4, 4))), rho=0.999),
    "linspace1d": synth.with_stream(synth.with_gate(W0, adaptive=1, tau_floor=0.97, tau_dev=2.0,
                                                    fp_mode=xo.FP_LINSPACE1D), rho=0.999),
    "step0-force": synth.with_stream(synth.with_gate(W0, adaptive=1, tau_floor=0.97, tau_dev=2.0,
                                                     step0_mode=xo.STEP0_FORCE), rho=0.999),
    "step0-strict": synth.with_stream(synth.with_gate(W0, adaptive=1, tau_floor=0.97, tau_dev=2.0,
                                                      step0_mode=xo.STEP0_STRICT), rho=0.999),
    "max-stale-1": synth.with_stream(synth.with_gate(W0, adaptive=1, tau_floor=0.97, tau_dev=2.0,
                                                     max_stale=1), rho=0.999),
    "back-anchor-4blk": synth.with_stream(synth.with_model(
        synth.with_gate(W0, adaptive=1, tau_floor=0.97, tau_dev=2.0, back_anchors=1), n_blocks=4), rho=0.999),
    "refresh-on-compute": synth.with_stream(synth.with_gate(W0, adaptive=1, tau_floor=0.97, tau_dev=2.0,
                                                            fp_refresh=xo.FP_REFRESH_ON_COMPUTE), rho=0.999),
    # the gate-stress stream's mechanisms at the tiny shape: an i.i.d. redraw every 3rd chunk (scene
    # cut) and a large action step every 2nd chunk, over an otherwise slowly varying stream
    "scene-cut-steer": synth.with_stream(synth.with_gate(W0, adaptive=1, tau_floor=0.9, tau_dev=2.0),
                                         rho=0.999, cut_every=3, big_every=2, big_sigma=1.0, n_chunks=7),
    "gate-off": synth.with_gate(W0, enabled=0),
    "window-1": synth.with_stream(synth.with_model(synth.with_gate(W0, adaptive=1, tau_floor=0.9, tau_dev=2.0),
                                                   kv_window=1), rho=0.999),
}


@pytest.mark.parametrize("name", list(CFG0_VARIANTS))
def test_cfg0_variants(name):
    ls = _ls(CFG0_VARIANTS[name])
    try:
        st = ls.run(6, tol_abs=TOL32)
        print(f"[parity] {name}: skips={st['skips']} evals={st['evals_post_warmup']} band={ls.band_hits} "
              f"worst={max(ls.worst.values()):.2e}", flush=True)
        if name == "zero-thresholds":
            assert st["skips"] == 0
        if name == "always-skip":
            assert st["skips"] == 5 * 4 * 1   # 5 post-warmup chunks x 4 steps x 1 gated block
        if name == "scene-cut-steer":
            assert st["skips"] > 0
    finally:
        ls.close()


def test_cfg0_force_full_every_other_chunk():
    w = CFG0_VARIANTS["table1-rho0.999"]
    ls = _ls(w)
    try:
        st = ls.run(6, tol_abs=TOL32, flags=lambda n, t: xo.FORCE_FULL if n % 2 == 0 else 0)
        assert st["skips"] > 0
    finally:
        ls.close()


def test_kv_update_without_output():
    """No output buffer for the KV-update pass: the last block stops after its
    key/value projection, and every later pass still matches the oracle (fp32
    and bf16, the last block gated in both)."""
    for w, kw in ((CFG0_VARIANTS["table1-rho0.999"], dict(tol_abs=TOL32)), (BF_RAGGED, dict(tol_rel_l2=TOLBF))):
        ls = _ls(w)
        try:
            ls.run(4, kv_out=False, **kw)
        finally:
            ls.close()


def test_cfg0_natural_skips_happen():
    ls = _ls(CFG0_VARIANTS["table1-rho0.999"])
    try:
        st = ls.run(6, tol_abs=TOL32)
        assert st["skips"] > 0
    finally:
        ls.close()


def test_zero_thresholds_bitwise_equal_to_gate_off():
    """Thresholds at zero: no skips, and the output equals the uncached path bit for bit."""
    _need_gpu()
    from paper_2604_20289_amd.xcache import XCache
    dev = torch.device("cuda")
    outs = []
    for w in (CFG0_VARIANTS["zero-thresholds"], CFG0_VARIANTS["gate-off"]):
        blob = synth.make_weights(w.model)
        xc = XCache(w.model, w.gate, blob, torch.cuda.current_stream().cuda_stream)
        res = []
        for n, eps, a in zip(range(4), synth.latent_stream(w.model, w.stream, 0, 4),
                             synth.action_stream(w.model, w.stream, 0, 4)):
            x = torch.from_numpy(eps).to(dev)
            y = torch.empty_like(x)
            for t, tau in enumerate(synth.timesteps(w.model)):
                xc.forward_chunk(t, tau, a, x, y)
                res.append(y.cpu().numpy().copy())
                x = y.clone()
            xc.kv_update(0.0, a, y)
        outs.append(res)
        xc.close()
    for a, b in zip(*outs):
        np.testing.assert_array_equal(a, b)


# ---- bf16 ---------------------------------------------------------------------

BF_RAGGED = synth.Workload(
    "bf16-ragged-3blk-h256-L300",
    synth.ModelShape(3, 256, 2, 128, 512, 256, 16, synth.BF16, 4, 3, (synth.ViewGroup(2, 3, 5, 10),)),
    synth.GateParams(),
    synth.StreamParams(5, 0.999, 0.02),
)


def test_bf16_ragged_multitile_parity():
    """L = 300 (ragged against the 128-row tiles and 64-key tiles), head_dim 128,
    a 3-chunk window, natural skips."""
    ls = _ls(BF_RAGGED)
    try:
        st = ls.run(5, tol_rel_l2=TOLBF)
        print(f"[parity] bf16-ragged skips={st['skips']} band={ls.band_hits} worst={max(ls.worst.values()):.2e}",
              flush=True)
        assert st["skips"] > 0
    finally:
        ls.close()


def test_bf16_head64_always_skip_and_table1():
    w = synth.with_model(BF_RAGGED, n_heads=4, head_dim=64, groups=(synth.ViewGroup(1, 3, 7, 9),))
    for gate in (synth.with_gate(w, adaptive=0, tau_cos_fixed=-1.0, tau_dev=math.inf).gate, w.gate):
        ls = _ls(synth.Workload(w.name, w.model, gate, w.stream))
        try:
            ls.run(4, tol_rel_l2=TOLBF)
        finally:
            ls.close()


# widths whose LayerNorm launch (which also runs the skip path, Eq. 4) takes
# the 8- and 16-vector-per-lane instantiations: the multi-camera hidden size
# 1536 (MLP 6144) and 4096 (MLP 1024 to keep the oracle quick); two cameras of
# 150 tokens, so the gate's global channel comes from the MLP-down column sums
BF_WIDE = {
    1536: synth.Workload(
        "bf16-wide-3blk-h1536-L300",
        synth.ModelShape(3, 1536, 12, 128, 6144, 256, 16, synth.BF16, 4, 2, (synth.ViewGroup(2, 1, 10, 15),)),
        synth.GateParams(),
        synth.StreamParams(4, 0.999, 0.02)),
    4096: synth.Workload(
        "bf16-wide-2blk-h4096-L300",
        synth.ModelShape(2, 4096, 32, 128, 1024, 256, 16, synth.BF16, 4, 2, (synth.ViewGroup(2, 1, 10, 15),)),
        synth.GateParams(),
        synth.StreamParams(3, 0.999, 0.02)),
}


@pytest.mark.parametrize("width", sorted(BF_WIDE))
@pytest.mark.parametrize("gate", ["always-skip", "table1"])
def test_bf16_wide_skip_path(width, gate):
    """Skipped blocks at C >= 1024 against the oracle: the pass output, the pass
    residual, every refreshed r_hat and the key/value caches, with skips > 0."""
    w = BF_WIDE[width]
    if gate == "always-skip":
        w = synth.with_gate(w, adaptive=0, tau_cos_fixed=-1.0, tau_dev=math.inf)
    ls = _ls(w, compute=np.float32)
    try:
        st = ls.run(w.stream.n_chunks, tol_rel_l2=TOLBF)
        print(f"[parity] {w.name} {gate}: skips={st['skips']} of {st['evals_post_warmup']} band={ls.band_hits} "
              f"r_hat checked={ls.residuals_checked} kv slots={ls.kv_slots_checked} "
              f"worst={max(ls.worst.values()):.2e}", flush=True)
        assert st["skips"] > 0
        if gate == "always-skip":
            B, S = w.model.n_blocks, w.model.n_steps
            assert st["skips"] == (w.stream.n_chunks - 1) * S * (B - 1)
    finally:
        ls.close()


# Hidden sizes that are no multiple of 256 put the QKV projection (and the
# cross-attention q and condition key / value projections) on the
# two-workgroup GEMM and its QKV epilogue, whose tile height (64 * MT rows)
# the library picks from the tile count on 256 CUs: N = 3C = 1152 at L = 300
# takes MT = 1 (its per-lane sums of squares padded from 16 to 32 for the
# reduce-scatter); N = 1920 (C = 640, 5 heads of 128) takes MT = 3 at L = 5000
# (48 padded to 64) and MT = 4 at L = 7000, where the output and MLP-down
# products take MT = 2; hidden 2048 at L = 7020 puts those two on MT = 4.
BF_TWO_WG = {
    "h384-d64-L300-rope-cross": synth.with_model(synth.Workload(
        "bf16-2wg-3blk-h384-d64-L300",
        synth.ModelShape(3, 384, 6, 64, 768, 256, 16, synth.BF16, 4, 3, (synth.ViewGroup(2, 3, 5, 10),)),
        synth.GateParams(), synth.StreamParams(4, 0.999, 0.02)), rope=1, cond_len=40),
    "h384-d128-L300": synth.Workload(
        "bf16-2wg-3blk-h384-d128-L300",
        synth.ModelShape(3, 384, 3, 128, 768, 256, 16, synth.BF16, 4, 3, (synth.ViewGroup(2, 3, 5, 10),)),
        synth.GateParams(), synth.StreamParams(4, 0.999, 0.02)),
    "h640-d128-L5000-mt3": synth.Workload(
        "bf16-2wg-1blk-h640-d128-L5000",
        synth.ModelShape(1, 640, 5, 128, 1280, 256, 16, synth.BF16, 2, 2, (synth.ViewGroup(2, 1, 50, 50),)),
        synth.GateParams(), synth.StreamParams(2, 0.999, 0.02)),
    "h640-d128-L7000-mt4": synth.with_model(synth.Workload(
        "bf16-2wg-1blk-h640-d128-L7000",
        synth.ModelShape(1, 640, 5, 128, 1280, 256, 16, synth.BF16, 2, 2, (synth.ViewGroup(2, 1, 50, 70),)),
        synth.GateParams(), synth.StreamParams(2, 0.999, 0.02)), rope=1),
    # the output and MLP-down products (N = 2048, no multiple of 192) on 256-row tiles
    "h2048-d128-L7020-oproj-down-mt4": synth.Workload(
        "bf16-2wg-1blk-h2048-d128-L7020",
        synth.ModelShape(1, 2048, 16, 128, 2048, 256, 16, synth.BF16, 1, 2, (synth.ViewGroup(2, 1, 54, 65),)),
        synth.GateParams(), synth.StreamParams(2, 0.999, 0.02)),
}


@pytest.mark.parametrize("name", list(BF_TWO_WG))
def test_bf16_two_workgroup_qkv_epilogue(name):
    """The two-workgroup kernel's QKV epilogue (per-head RMSNorm, rotation, q /
    K / V^T cache stores) at every tile height, head_dim 64 and 128, against
    the oracle: pass outputs, residuals, r_hat and the key / value caches."""
    w = BF_TWO_WG[name]
    ls = _ls(w, compute=np.float32)
    try:
        st = ls.run(w.stream.n_chunks, tol_rel_l2=TOLBF)
        print(f"[parity] {w.name}: skips={st['skips']} r_hat checked={ls.residuals_checked} "
              f"kv slots={ls.kv_slots_checked} worst={max(ls.worst.values()):.2e}", flush=True)
        assert ls.kv_slots_checked > 0
    finally:
        ls.close()


# The wide kernel's QKV epilogue with head_dim 64 (one wave per head): wide
# tiles serve the QKV product only where they fill the chip (the multi-camera
# token count), so this case runs at L = 7020 with hidden 1536 in 24 heads,
# one block, two chunks, rotary embedding.
BF_WIDE_D64 = synth.with_model(synth.Workload(
    "bf16-wide-1blk-h1536-d64-L7020",
    synth.ModelShape(1, 1536, 24, 64, 6144, 256, 16, synth.BF16, 2, 2, (synth.ViewGroup(2, 1, 54, 65),)),
    synth.GateParams(), synth.StreamParams(2, 0.999, 0.02)), rope=1)


def test_bf16_wide_qkv_epilogue_head64():
    w = BF_WIDE_D64
    ls = _ls(w, compute=np.float32)
    try:
        ls.run(w.stream.n_chunks, tol_rel_l2=TOLBF)
        print(f"[parity] {w.name}: kv slots={ls.kv_slots_checked} worst={max(ls.worst.values()):.2e}", flush=True)
        assert ls.kv_slots_checked > 0
    finally:
        ls.close()


@pytest.mark.slow
def test_cfg1_prefix_parity():
    """Single-camera bf16 configuration, first 4 chunks, Table-1 gate."""
    ls = _ls(W1, compute=np.float32)
    try:
        st = ls.run(4, tol_rel_l2=TOLBF)
        print(f"[parity] cfg1 skips={st['skips']} band={ls.band_hits} worst={max(ls.worst.values()):.2e}",
              flush=True)
    finally:
        ls.close()


def test_determinism_bf16():
    """Same inputs twice: bitwise-equal outputs and identical decisions."""
    _need_gpu()
    from paper_2604_20289_amd.xcache import XCache
    w = BF_RAGGED
    dev = torch.device("cuda")
    runs = []
    for _ in range(2):
        xc = XCache(w.model, w.gate, synth.make_weights(w.model), torch.cuda.current_stream().cuda_stream)
        res = []
        for n, eps, a in zip(range(3), synth.latent_stream(w.model, w.stream, 0, 3),
                             synth.action_stream(w.model, w.stream, 0, 3)):
            x = torch.from_numpy(eps).to(dev)
            y = torch.empty_like(x)
            for t, tau in enumerate(synth.timesteps(w.model)):
                xc.forward_chunk(t, tau, a, x, y)
                res.append(y.cpu().numpy().copy())
                x = y.clone()
            xc.kv_update(0.0, a, y)
        st = xc.stats()
        res.append(st["skip_counts"].copy())
        runs.append(res)
        xc.close()
    for a, b in zip(*runs):
        np.testing.assert_array_equal(a, b)


DEGENERATE = {
    # one block, no anchors: the only block is gated
    "one-block-no-anchor": synth.with_stream(synth.with_model(
        synth.with_gate(W0, adaptive=1, tau_floor=0.9, tau_dev=2.0, front_anchors=0), n_blocks=1), rho=0.999),
    # a single denoising step per chunk
    "one-step": synth.with_stream(synth.with_model(
        synth.with_gate(W0, adaptive=1, tau_floor=0.9, tau_dev=2.0), n_steps=1), rho=0.999),
    # every block an anchor: nothing is ever gated
    "all-anchors": synth.with_gate(W0, adaptive=1, tau_floor=0.9, tau_dev=2.0, front_anchors=1, back_anchors=1),
    # warmup of two generations and a longer window than the stream
    "warmup2-window4": synth.with_stream(synth.with_model(
        synth.with_gate(W0, adaptive=1, tau_floor=0.9, tau_dev=2.0, warmup=2), kv_window=4), rho=0.999),
}


@pytest.mark.parametrize("name", list(DEGENERATE))
def test_degenerate_configs(name):
    ls = _ls(DEGENERATE[name])
    try:
        st = ls.run(5, tol_abs=TOL32)
        if name == "all-anchors":
            assert st["gated_evals"] == 0 and st["skips"] == 0
    finally:
        ls.close()


def test_bf16_three_view_groups():
    """Three view groups with different grids (front/side/rear-like), one back anchor."""
    w = synth.Workload(
        "bf16-three-groups",
        synth.ModelShape(3, 256, 4, 64, 512, 256, 16, synth.BF16, 4, 2,
                         (synth.ViewGroup(2, 2, 6, 10), synth.ViewGroup(3, 2, 4, 7), synth.ViewGroup(1, 3, 5, 5))),
        synth.GateParams(back_anchors=1),
        synth.StreamParams(4, 0.999, 0.02),
    )
    ls = _ls(w)
    try:
        ls.run(4, tol_rel_l2=TOLBF)
    finally:
        ls.close()


def test_bf16_persistent_gemm_widths():
    """Widths that are multiples of 192 (hidden 384, MLP 768) take the
    persistent 256 x 192 projection kernel; L = 300 leaves a ragged last row
    tile."""
    w = synth.Workload(
        "bf16-h384-L300",
        synth.ModelShape(2, 384, 3, 128, 768, 256, 16, synth.BF16, 4, 2, (synth.ViewGroup(2, 3, 5, 10),)),
        synth.GateParams(),
        synth.StreamParams(4, 0.999, 0.02),
    )
    ls = _ls(w)
    try:
        ls.run(4, tol_rel_l2=TOLBF)
    finally:
        ls.close()


# ---- WAN-style block extensions: 3-D rotary embedding and cross-attention ---------

EXT_VARIANTS = {
    "fp32-rope": synth.with_model(W0, rope=1),
    "fp32-cross": synth.with_model(W0, cond_len=8),
    "fp32-rope-cross-table1": synth.with_stream(synth.with_model(
        synth.with_gate(W0, adaptive=1, tau_floor=0.97, tau_dev=2.0), rope=1, cond_len=8), rho=0.999),
    "fp32-rope-cross-always-skip": synth.with_model(
        synth.with_gate(W0, adaptive=0, tau_cos_fixed=-1.0, tau_dev=math.inf), rope=1, cond_len=8),
    "fp32-rope-two-groups": synth.with_stream(synth.with_model(
        synth.with_gate(W0, adaptive=1, tau_floor=0.97, tau_dev=2.0), rope=1, cond_len=5,
        groups=(synth.ViewGroup(1, 2, 4, 4), synth.ViewGroup(2, 1, 3, 5))), rho=0.999),
}


@pytest.mark.parametrize("name", list(EXT_VARIANTS))
def test_extension_fp32_variants(name):
    """Rotary embedding and cross-attention on the tiny float32 model, pass by
    pass, with the condition replaced (and its token count changed) mid-rollout."""
    w = EXT_VARIANTS[name]
    ls = _ls(w)
    try:
        m = w.model
        cond_fn = None
        if m.cond_len > 0:
            cond_fn = lambda n: synth.condition_tokens(m, 10 + n, n_tokens=1 + (3 * n) % m.cond_len) \
                if n in (2, 4) else None
        st = ls.run(w.stream.n_chunks, tol_abs=TOL32, cond_fn=cond_fn)
        print(f"[parity] {name} skips={st['skips']} band={ls.band_hits} worst={max(ls.worst.values()):.2e}",
              flush=True)
    finally:
        ls.close()


BF_EXT = synth.with_model(BF_RAGGED, rope=1, cond_len=77)


def test_extension_bf16_ragged_parity():
    """bf16, head_dim 128, L = 300 and 77 condition tokens (ragged against the
    tiles), rotary embedding over a 3-chunk window, natural skips; the
    condition is replaced by 64 tokens before chunk 2 and by 5 before chunk 3."""
    ls = _ls(BF_EXT)
    try:
        m = BF_EXT.model
        cond_fn = lambda n: {2: synth.condition_tokens(m, 21, n_tokens=64),
                             3: synth.condition_tokens(m, 22, n_tokens=5)}.get(n)
        st = ls.run(5, tol_rel_l2=TOLBF, cond_fn=cond_fn)
        print(f"[parity] bf16-ext skips={st['skips']} band={ls.band_hits} worst={max(ls.worst.values()):.2e}",
              flush=True)
        assert st["skips"] > 0
    finally:
        ls.close()


def test_extension_bf16_head64_kv_without_output():
    w = synth.with_model(BF_RAGGED, n_heads=4, head_dim=64, groups=(synth.ViewGroup(1, 3, 7, 9),), rope=1,
                         cond_len=33)
    ls = _ls(w)
    try:
        ls.run(4, tol_rel_l2=TOLBF, kv_out=False)
    finally:
        ls.close()


def test_condition_required_and_validated():
    _need_gpu()
    from paper_2604_20289_amd import xcache as xcp
    w = synth.with_model(W0, cond_len=4)
    dev = torch.device("cuda")
    xc = xcp.XCache(w.model, w.gate, synth.make_weights(w.model), torch.cuda.current_stream().cuda_stream)
    try:
        x = torch.zeros((w.model.tokens, w.model.hidden), dtype=torch.float32, device=dev)
        a = np.zeros(w.model.action_dim, np.float32)
        with pytest.raises(xcp.XCacheError) as e:
            xc.forward_chunk(0, 1000.0, a, x, x)
        assert e.value.status == xcp.XC_ERR_STATE
        with pytest.raises(xcp.XCacheError) as e:
            xc.set_condition(np.zeros((5, w.model.hidden), np.float32))     # more than cond_len
        assert e.value.status == xcp.XC_ERR_INVALID_ARG
        bad = np.zeros((2, w.model.hidden), np.float32)
        bad[1, 3] = np.nan
        with pytest.raises(xcp.XCacheError) as e:
            xc.set_condition(bad)
        assert e.value.status == xcp.XC_ERR_INVALID_ARG
        xc.set_condition(np.ones((4, w.model.hidden), np.float32))
        xc.forward_chunk(0, 1000.0, a, x, x)
        torch.cuda.synchronize()
    finally:
        xc.close()
    plain = xcp.XCache(W0.model, W0.gate, synth.make_weights(W0.model), torch.cuda.current_stream().cuda_stream)
    try:
        with pytest.raises(xcp.XCacheError) as e:
            plain.set_condition(np.ones((1, W0.model.hidden), np.float32))
        assert e.value.status == xcp.XC_ERR_STATE
    finally:
        plain.close()


def test_action_fixed_per_generation():
    """One chunk has one action (the condition channel changes once per
    generation, Section 2.3.2): a pass of the same generation with another
    action is refused with no state change; the clean pass releases it."""
    _need_gpu()
    from paper_2604_20289_amd import xcache as xcp
    w = W0
    dev = torch.device("cuda")
    xc = xcp.XCache(w.model, w.gate, synth.make_weights(w.model), torch.cuda.current_stream().cuda_stream)
    try:
        x = torch.randn((w.model.tokens, w.model.hidden), dtype=torch.float32, device=dev)
        y = torch.empty_like(x)
        a0 = np.zeros(w.model.action_dim, np.float32)
        a1 = a0.copy()
        a1[0] = 0.5
        xc.forward_chunk(0, 900.0, a0, x, y)
        before = xc.stats()
        for call in (lambda: xc.forward_chunk(1, 800.0, a1, x, y),
                     lambda: xc.kv_update(synth.KV_UPDATE_TIMESTEP, a1, x, None)):
            with pytest.raises(xcp.XCacheError) as e:
                call()
            assert e.value.status == xcp.XC_ERR_STATE
        after = xc.stats()
        assert (after["last_step"], after["generations"], after["kv_block_evals"]) == \
            (before["last_step"], before["generations"], before["kv_block_evals"])
        xc.forward_chunk(1, 800.0, a0, x, y)
        xc.kv_update(synth.KV_UPDATE_TIMESTEP, a0, x, None)
        xc.forward_chunk(0, 900.0, a1, x, y)        # the next generation takes a new action
        xc.reset()
        xc.forward_chunk(0, 900.0, a0, x, y)        # and so does a reset rollout
        torch.cuda.synchronize()
        assert xc.stats()["generations"] == 0
    finally:
        xc.close()


def test_bf16_small_cameras_read_the_block_input():
    """Cameras of 25 tokens (fewer than the 32-token blocks of the MLP-down
    column-sum partials): the gate reads the camera means from the block input
    itself; 12 cameras in one view group, natural skips."""
    w = synth.with_model(BF_RAGGED, groups=(synth.ViewGroup(12, 1, 5, 5),))
    ls = _ls(w)
    try:
        st = ls.run(5, tol_rel_l2=TOLBF)
        print(f"[parity] bf16-small-cameras skips={st['skips']} band={ls.band_hits}", flush=True)
    finally:
        ls.close()


def _tiny(base, name, group, **stream):
    w = synth.with_stream(synth.with_model(base, groups=(group,)), n_chunks=4, **stream)
    return dataclasses.replace(w, name=name)


TINY = {
    "fp32-L1": _tiny(W0, "tiny-fp32-2blk-h128-L1", synth.ViewGroup(1, 1, 1, 1), rho=0.999),
    "fp32-L33": _tiny(W0, "tiny-fp32-2blk-h128-L33", synth.ViewGroup(1, 1, 3, 11), rho=0.999),
    "bf16-L1": _tiny(BF_RAGGED, "tiny-bf16-3blk-h256-L1", synth.ViewGroup(1, 1, 1, 1)),
    "bf16-L33": _tiny(BF_RAGGED, "tiny-bf16-3blk-h256-L33", synth.ViewGroup(1, 1, 3, 11)),
}


@pytest.mark.parametrize("name", sorted(TINY))
@pytest.mark.parametrize("gate", ["always-skip", "table1"])
def test_tiny_token_counts(name, gate):
    """Degenerate sizes: one token (every tile almost all padding, a camera of
    one token whose fingerprint and mean are the token itself) and 33 tokens
    (one past a 32-row block); both below the 64-key and 256-query tiles."""
    w = TINY[name]
    if gate == "always-skip":
        w = synth.with_gate(w, adaptive=0, tau_cos_fixed=-1.0, tau_dev=math.inf)
    else:
        w = synth.with_gate(w, adaptive=1, tau_floor=0.97, tau_dev=2.0)
    tol = dict(tol_abs=TOL32) if w.model.dtype == synth.F32 else dict(tol_rel_l2=TOLBF)
    ls = _ls(w, compute=np.float32 if w.model.dtype == synth.BF16 else np.float64)
    try:
        st = ls.run(w.stream.n_chunks, **tol)
        print(f"[parity] {name} {gate}: skips={st['skips']} of {st['evals_post_warmup']} band={ls.band_hits} "
              f"worst={max(ls.worst.values()):.2e}", flush=True)
        if gate == "always-skip":
            assert st["skips"] > 0
    finally:
        ls.close()
