"""Benchmark of the cached chunk forward on one MI355X.

A step is one generation chunk: S denoising passes (with the sampler update
between them) plus the KV-update pass, over the multi-camera bf16 DiT
workload (20 blocks, hidden 1536, 12 heads x 128, MLP 6144; 6 cameras x 3
latent frames x 15 x 26 patches = 7020 tokens; a 3-chunk key/value window =
21060 keys; 4 steps).  Inputs are synthetic and seeded (weights N(0, 0.02^2),
an AR(1) latent stream with rho 0.97, a 16-d action random walk with sigma
0.03) and resident in HBM before the timed region; the gate uses Table 1's
defaults.

Runs, in order:
  1. gate on, `warmup` untimed chunks then `steps` timed chunks -> mean
     chunk latency (the reported value; the paper reports the average
     per-chunk DiT time) and the block skip rate over the timed chunks;
  2. the skip path alone (a gate that skips every block after the warmup
     chunk) -> time per skipped block and the per-launch averages of its
     kernels; the gate comparison that reads the block input, with that
     input in the last-level cache and after a 1 GiB write evicted it;
  3. the same stream at tau_floor 0.95 (the value the paper's Section 2.4
     text gives; Table 1 says 0.97);
  4. gate off (every block computed, same kernels), same chunks ->
     full-compute latency and effective block TFLOP/s; then the same chunks
     again with HIP events around every kernel launch -> per-kernel
     durations and the roofline of the dominant kernel (attention);
  5. the gate-stress stream (same shapes; scene cut every 8th chunk, a
     steering step every 5th) -> its latency and skip rate;
  6. the CPU oracle on a bounded sample (one computed block at the full
     shape, float64 numpy on the host cores), scaled to ms per chunk.
Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

METRIC = "chunk latency ms + block TFLOP/s vs MFMA peak + block skip rate, 1 GPU"
PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0

# HBM-side bytes per full-window attention op (main dispatch + merge of the
# key-split partials) from the rocprofv3 FETCH_SIZE and WRITE_SIZE passes,
# scaled by a 512 MiB copy-kernel calibration; valid only for the workload and
# the kernel source they were taken on (sha1 prefix of the file).
MEASURED_TRAFFIC = {
    "attention": {"source": "paper_2604_20289_amd/csrc/xc_attention.hip", "sha1": "ccad982ddaa23cb7",
                  "workload": "multi-camera-bf16-dit-20blk-h1536-L7020", "bytes": (358.8 + 88.5) * 1e6},
}


def measured_traffic(kernel, workload):
    import hashlib
    rec = MEASURED_TRAFFIC.get(kernel)
    if not rec or rec["workload"] != workload:
        return None
    with open(os.path.join(ROOT, rec["source"]), "rb") as f:
        if hashlib.sha1(f.read()).hexdigest()[:16] != rec["sha1"]:
            return None
    return rec["bytes"]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def block_flops(m, n_keys):
    L, C, Dm = m.tokens, m.hidden, m.mlp_hidden
    f = 6.0 * L * C * C + 2.0 * L * C * C + 4.0 * L * C * Dm + 4.0 * L * n_keys * C
    if m.cond_len > 0:  # cross-attention: q and output projections, attention over the condition
        f += 4.0 * L * C * C + 4.0 * L * m.cond_len * C
    return f


def attention_flops(m, n_keys):
    return 4.0 * m.tokens * n_keys * m.n_heads * m.head_dim


def run_stream(xc, m, eps_dev, actions, n_warm, n_timed, torch, profile=False, force_every=0, per_chunk=None,
               at_timed=None, flush=None):
    """Drive n_warm + n_timed chunks; returns, per timed chunk, (chunk ms, ms of
    the S denoising passes, ms of the KV-update pass).  force_every = P > 0
    computes every block of the denoising passes of chunks n with n % P == 0
    (the paper's periodic whole-generation refresh); per_chunk, a list, then
    receives each chunk's skip count (the stream is synchronised per chunk).
    at_timed(xc) is called once, synchronised, before the first timed chunk;
    flush(), when given, is enqueued before every timed pass (outside the
    chunk's events it is not: use it only for per-kernel timings)."""
    L, C = m.tokens, m.hidden
    taus = synth.timesteps(m)
    x = torch.empty((L, C), dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    ev = []
    for n in range(n_warm + n_timed):
        eps = eps_dev[n]
        timed = n >= n_warm
        if timed and n == n_warm:
            torch.cuda.synchronize()
            if at_timed is not None:
                at_timed(xc)
            if profile:
                xc.profile(True)
        if timed:
            e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            e[0].record()
        x.copy_(eps)
        fl = xcp_force_full if force_every and n % force_every == 0 else 0
        for t in range(m.n_steps):
            if flush is not None and timed:
                flush()
            xc.forward_chunk(t, taus[t], actions[n], x, y, fl)
            if t + 1 < m.n_steps:
                sg = synth.sampler_sigma(m, t + 1)
                xc.axpby(1.0 - sg, y, sg, eps, x, L * C)
        if timed:
            e[1].record()
        xc.kv_update(synth.KV_UPDATE_TIMESTEP, actions[n], y, None)
        if timed:
            e[2].record()
            ev.append(e)
        if per_chunk is not None:
            per_chunk.append(xc.stats()["skips"])
    torch.cuda.synchronize()
    if profile:
        xc.profile(False)
    return [(e[0].elapsed_time(e[2]), e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2])) for e in ev]


xcp_force_full = 1  # the library's forward flag that computes every block (set from the binding in main)


def kernel_table(xc, xcp):
    out = {}
    for k in range(xcp.XC_KERN_COUNT):
        n, tot = xc.kernel_times(k, clear=True)
        if n:
            out[xcp.KERNEL_NAMES[k]] = {"launches": n, "avg_us": 1e3 * tot / n, "total_ms": tot}
    return out


def cpu_baseline(w, weights, seed):
    """The oracle, as it is, on one computed block at the full shape (full key window)."""
    from oracle import xcache_oracle as xo
    m = w.model
    small = synth.with_model(w, n_blocks=1).model
    blob = weights[: synth.block_numel(m)]
    orc = xo.XCacheOracle(small, synth.GateParams(enabled=0), blob)
    if m.cond_len > 0:
        orc.set_condition(synth.condition_tokens(m, seed))
    rng = np.random.default_rng(seed + 7)
    L, H, d = m.tokens, m.n_heads, m.head_dim
    orc.ring[0] = [(xo.bf16_round(rng.standard_normal((H, L, d))), xo.bf16_round(rng.standard_normal((H, L, d))))
                   for _ in range(m.kv_window - 1)]
    x = next(synth.latent_stream(m, w.stream, seed, 1)).astype(np.float64)
    cond = orc.cond(1000.0, np.zeros(m.action_dim))
    # repeat the block until about 10 s of CPU work (at least twice)
    n_eval, t0 = 0, time.perf_counter()
    while n_eval < 2 or time.perf_counter() - t0 < 10.0:
        orc.block(0, x, cond)
        n_eval += 1
    total = time.perf_counter() - t0
    dt = total / n_eval
    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info
        blas = max((p.get("num_threads", 0) for p in threadpool_info() if p.get("user_api") == "blas"), default=0)
    except Exception:  # threadpoolctl missing: report the affinity count only
        blas = 0
    per_chunk_ms = dt * 1e3 * m.n_blocks * (m.n_steps + 1)
    return {"value": per_chunk_ms, "unit": "ms/chunk", "cores": min(cores, blas) if blas else cores,
            "kind": "oracle", "blas_threads": blas, "cpus_available": cores,
            "sample": (f"{n_eval} computed block evaluations at the full shape (L={L}, {m.kv_window * L} keys), "
                       f"float64 numpy, {total:.1f} s in total, {dt:.1f} s each, scaled x"
                       f"{m.n_blocks * (m.n_steps + 1)} block evaluations to a full-compute chunk")}


def gate_bytes(m, gate, xcp, folded):
    """Algorithmic bytes of one gate-comparison launch: the cached fingerprint
    read and the current one written, the spatial rows gathered, and the
    global channel's source (one read of the block input, or the previous
    block's MLP-down column-sum partials)."""
    L, C = m.tokens, m.hidden
    n_srows = len(xcp.xc_fingerprint_rows(m, gate))
    fp_rows = n_srows + sum(g.views for g in m.groups)
    if folded:
        return 4.0 * n_srows * C + 8.0 * fp_rows * C + 16.0 * ((L + 31) // 32) * C
    return 4.0 * L * C + 8.0 * fp_rows * C


def skip_path(w, m, eps_dev, actions, make_xc, n_timed, torch, xcp):
    """Every gated block skips: no anchor, fixed cosine threshold -1 and no
    deviation bound.  After the warmup chunk each denoising pass is the
    conditioning plus B skipped blocks (gate comparison, decision, the
    skip-add inside the first LayerNorm launch, and the block's other
    launches returning at entry).  Reports the per-skipped-block time from
    pass events and the per-launch averages of one more chunk's passes."""
    g = synth.with_gate(w, front_anchors=0, back_anchors=0, adaptive=0, tau_cos_fixed=-1.0, tau_dev=math.inf).gate
    xc = make_xc(g)
    L, C = m.tokens, m.hidden
    taus = synth.timesteps(m)
    x = torch.empty((L, C), dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    pass_ms = []
    n_all = 1 + n_timed + 1
    for n in range(n_all):
        x.copy_(eps_dev[n])
        last = n == n_all - 1
        if last:
            torch.cuda.synchronize()
            xc.profile(True)
        for t in range(m.n_steps):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            ev[0].record()
            xc.forward_chunk(t, taus[t], actions[n], x, y)
            ev[1].record()
            if 1 <= n < n_all - 1:
                pass_ms.append(ev)
            if t + 1 < m.n_steps:
                sg = synth.sampler_sigma(m, t + 1)
                xc.axpby(1.0 - sg, y, sg, eps_dev[n], x, L * C)
        if last:
            torch.cuda.synchronize()
            xc.profile(False)
        xc.kv_update(synth.KV_UPDATE_TIMESTEP, actions[n], y, None)
    torch.cuda.synchronize()
    kt = kernel_table(xc, xcp)
    st = xc.stats()
    xc.close()
    ms = [e[0].elapsed_time(e[1]) for e in pass_ms]
    per_block_us = 1e3 * statistics.mean(ms) / m.n_blocks
    kernels = {}
    folded = m.dtype == synth.BF16 and min(gr.frames * gr.height * gr.width for gr in m.groups) >= 32
    for k, v in kt.items():
        e = {"launches": v["launches"], "avg_us": round(v["avg_us"], 2)}
        if k == "skip_add":
            e["bytes"] = 10.0 * L * C if m.dtype == synth.BF16 else 12.0 * L * C
            e["gbs"] = round(e["bytes"] / (v["avg_us"] * 1e-6) / 1e9, 1)
            e["hbm_frac"] = round(e["gbs"] / PEAK_HBM_GBS, 4)
        if k == "gate":
            # block 0 reads its input; the others take the previous block's sums
            b_all = gate_bytes(m, g, xcp, False) + (m.n_blocks - 1) * gate_bytes(m, g, xcp, folded)
            e["bytes_mean"] = b_all / m.n_blocks
            e["gbs"] = round(e["bytes_mean"] / (v["avg_us"] * 1e-6) / 1e9, 1)
        kernels[k] = e
    return {"pass_ms_mean": round(statistics.mean(ms), 3), "per_skipped_block_us": round(per_block_us, 2),
            "skips": st["skips"], "kernels": kernels,
            "note": "every gated block skipped (no anchor, cosine threshold -1): a pass = conditioning + "
                    f"{m.n_blocks} skipped blocks; per-skipped-block time = pass time / blocks"}


def cold_gate(w, m, eps_dev, actions, make_xc, torch, xcp, n_pass=8):
    """The gate comparison that reads the block input (one gated block, no
    anchor), timed per launch with the input in the last-level cache (the
    previous launch wrote it) and after a 1 GiB write evicts it."""
    wg = synth.with_gate(synth.with_model(w, n_blocks=1), front_anchors=0, adaptive=0, tau_cos_fixed=-1.0,
                         tau_dev=math.inf)
    m1 = wg.model
    flush_buf = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    out = {}
    for mode in ("in_stream", "cold"):
        xc = xcp.XCache(m1, wg.gate, make_xc.weights[: synth.block_numel(m1)], make_xc.stream)
        if make_xc.cond is not None:
            xc.set_condition(make_xc.cond)
        L, C = m1.tokens, m1.hidden
        x = torch.empty((L, C), dtype=torch.float32, device="cuda")
        y = torch.empty_like(x)
        for n in range(2):
            x.copy_(eps_dev[n])
            if n == 1:
                torch.cuda.synchronize()
                xc.profile(True)
            for i in range(n_pass if n == 1 else 1):
                if n == 1 and mode == "cold":
                    flush_buf.fill_(float(i))
                xc.forward_chunk(0, 1000.0, actions[n], x, y)
            if n == 1:
                torch.cuda.synchronize()
                xc.profile(False)
            xc.kv_update(synth.KV_UPDATE_TIMESTEP, actions[n], y, None)
        cnt, tot = xc.kernel_times(xcp.XC_KERN_GATE, clear=True)
        xc.close()
        b = gate_bytes(m1, wg.gate, xcp, False)
        us = 1e3 * tot / cnt
        out[mode] = {"launches": cnt, "avg_us": round(us, 2), "bytes": b, "gbs": round(b / (us * 1e-6) / 1e9, 1),
                     "hbm_frac": round(b / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    del flush_buf
    return out


def ablations(w, m, weights, eps_dev, actions, make_xc, args, torch):
    """Synthetic analogues of the paper's gate ablations (Section 4.4): the same stream under
    step-0 handling, anchor, staleness, refresh and threshold variants; skip rate and latency only."""
    from paper_2604_20289_amd import xcache as xcp
    variants = [
        ("table1", {}),
        ("step0_force", {"step0_mode": xcp.XC_STEP0_FORCE}),
        ("step0_strict", {"step0_mode": xcp.XC_STEP0_STRICT}),
        ("front_anchors_0", {"front_anchors": 0}),
        ("back_anchors_1", {"back_anchors": 1}),
        ("max_stale_1", {"max_stale": 1}),
        ("fp_refresh_on_compute", {"fp_refresh": xcp.XC_FP_REFRESH_ON_COMPUTE}),
        ("fixed_tau_0.97", {"adaptive": 0, "tau_cos_fixed": 0.97}),
    ] + [(f"tau_floor_{tf:.2f}", {"tau_floor": tf}) for tf in (0.93, 0.95, 0.96, 0.97, 0.98, 0.99)]
    out = {"metric": "gate ablations: block skip rate and gate-on chunk latency", "workload": w.name,
           "warmup": args.warmup, "steps": args.steps, "data": "synthetic", "variants": {}}
    B, S = m.n_blocks, m.n_steps
    for name, kw in variants:
        wv = synth.with_gate(w, **kw)
        xc = make_xc(wv.gate)
        ms = [v[0] for v in run_stream(xc, m, eps_dev, actions, args.warmup, args.steps, torch)]
        st = xc.stats()
        xc.close()
        per_block = np.asarray(st["skip_counts"]).reshape(S, B).sum(axis=0).astype(int).tolist()
        out["variants"][name] = {"gate": kw, "skip_rate": round(st["skips"] / max(1, st["evals_post_warmup"]), 4),
                                 "mean_ms": round(statistics.mean(ms), 3),
                                 "median_ms": round(statistics.median(ms), 3),
                                 "skips_per_block": per_block}
        log(f"ablation {name}: skip rate {out['variants'][name]['skip_rate']}, {out['variants'][name]['mean_ms']} ms")
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=12, help="timed chunks")
    ap.add_argument("--warmup", type=int, default=2, help="untimed chunks before them")
    ap.add_argument("--workload", type=int, default=2, help="index of the synthetic workload preset")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--tau-floor", type=float, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gate-off", action="store_true")
    ap.add_argument("--no-alt-tau", action="store_true", help="skip the extra gate-on run at tau_floor 0.95")
    ap.add_argument("--no-stress", action="store_true", help="skip the gate-stress stream run")
    ap.add_argument("--force-every", type=int, default=0,
                    help="also run the gate-on stream with every P-th generation computed in full and report "
                         "the per-chunk skip fractions (the paper's periodic refresh cadence)")
    ap.add_argument("--ablations", action="store_true",
                    help="instead of the benchmark line, print one line of gate ablations on the same stream: "
                         "step-0 modes, anchors, staleness bound, refresh mode and a tau_floor sweep (skip rate "
                         "and mean chunk latency of each; --steps timed chunks after --warmup)")
    ap.add_argument("--rope", action="store_true",
                    help="model with the 3-D rotary embedding of the self-attention queries and keys")
    ap.add_argument("--cond-len", type=int, default=0,
                    help="model with a cross-attention layer over this many condition tokens")
    ap.add_argument("--phase", choices=["full", "skip", "gate-cold"], default=None,
                    help="run one phase alone and print its own JSON line (for profiling): 'full' = the gate-off "
                         "stream (every block computed), 'skip' = the skip path (every gated block skipped), "
                         "'gate-cold' = the gate comparison reading its input, in-stream and after a cache flush")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="copy a buffer of this many MiB once (calibrates rocprofv3 FETCH_SIZE/WRITE_SIZE)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the cached chunk forward of one rollout runs on a single device "
              "(several GPUs would each run their own rollout); run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2604_20289_amd import xcache as xcp
    global xcp_force_full
    xcp_force_full = xcp.XC_FORCE_FULL

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    w = synth.workload(args.workload)
    if args.tau_floor is not None:
        w = synth.with_gate(w, tau_floor=args.tau_floor)
    if args.rope or args.cond_len:
        w = synth.with_model(w, rope=int(args.rope), cond_len=args.cond_len)
        w = synth.Workload(w.name + ("-rope" if args.rope else "") +
                           (f"-cross{args.cond_len}" if args.cond_len else ""), w.model, w.gate, w.stream)
    m = w.model
    n_chunks = args.warmup + args.steps
    log(f"workload {w.name}: L={m.tokens} blocks={m.n_blocks} chunks={n_chunks}")
    t0 = time.time()
    weights = synth.make_weights(m, args.seed)
    eps_host = list(synth.latent_stream(m, w.stream, args.seed, n_chunks))
    actions = list(synth.action_stream(m, w.stream, args.seed, n_chunks))
    eps_dev = [torch.from_numpy(e).cuda() for e in eps_host]
    del eps_host
    log(f"inputs ready in {time.time() - t0:.1f} s")
    stream = torch.cuda.current_stream().cuda_stream
    cond = synth.condition_tokens(m, args.seed) if m.cond_len > 0 else None

    def make_xc(gate):
        xc = xcp.XCache(m, gate, weights, stream)
        if cond is not None:
            xc.set_condition(cond)
        return xc
    make_xc.weights, make_xc.stream, make_xc.cond = weights, stream, cond

    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.mul(src, 1.0, out=dst)  # one elementwise kernel: reads and writes exactly n*4 bytes
        torch.cuda.synchronize()
        log(f"calibration copy of {args.calib_copy_mib} MiB done")
        del src, dst

    if args.ablations:
        print(json.dumps(ablations(w, m, weights, eps_dev, actions, make_xc, args, torch)), flush=True)
        return
    if args.phase == "full":
        xc = make_xc(synth.with_gate(w, enabled=0).gate)
        ms = [v[0] for v in run_stream(xc, m, eps_dev, actions, args.warmup, args.steps, torch)]
        xc.close()
        print(json.dumps({"phase": "full", "workload": w.name, "warmup": args.warmup, "steps": args.steps,
                          "chunk_ms": [round(v, 3) for v in ms]}), flush=True)
        return
    if args.phase == "skip":
        print(json.dumps({"phase": "skip", "workload": w.name,
                          **skip_path(w, m, eps_dev, actions, make_xc, max(1, min(args.steps, n_chunks - 2)), torch,
                                      xcp)}), flush=True)
        return
    if args.phase == "gate-cold":
        print(json.dumps({"phase": "gate-cold", "workload": w.name,
                          **cold_gate(w, m, eps_dev, actions, make_xc, torch, xcp)}), flush=True)
        return

    def timed_rate(st0, st):
        """Skip rate over the timed chunks' denoising block evaluations."""
        return (st["skips"] - st0["skips"]) / max(1, st["evals_post_warmup"] - st0["evals_post_warmup"])

    # 1. gate on
    xc = make_xc(w.gate)
    st0 = {}
    on_split = run_stream(xc, m, eps_dev, actions, args.warmup, args.steps, torch,
                          at_timed=lambda h: st0.update(h.stats()))
    on_ms = [v[0] for v in on_split]
    st = xc.stats()
    xc.close()
    log(f"gate on: mean {statistics.mean(on_ms):.2f} ms/chunk, timed skips {st['skips'] - st0['skips']} / "
        f"{st['evals_post_warmup'] - st0['evals_post_warmup']}")

    # 3. the skip path alone, and the gate comparison that reads its input, in-stream and cold
    skp = skip_path(w, m, eps_dev, actions, make_xc, min(2, n_chunks - 2), torch, xcp)
    log(f"skip path: {skp['per_skipped_block_us']} us per skipped block")
    cgate = cold_gate(w, m, eps_dev, actions, make_xc, torch, xcp)
    log(f"gate reading x: in-stream {cgate['in_stream']['avg_us']} us, cold {cgate['cold']['avg_us']} us")

    # 1b. the same stream at the other tau_floor the paper states (0.95 vs Table 1's 0.97)
    alt = None
    if args.tau_floor is None and not args.no_alt_tau:
        wa = synth.with_gate(w, tau_floor=0.95)
        xc = make_xc(wa.gate)
        sa0 = {}
        alt_ms = [v[0] for v in run_stream(xc, m, eps_dev, actions, args.warmup, args.steps, torch,
                                           at_timed=lambda h: sa0.update(h.stats()))]
        sa = xc.stats()
        xc.close()
        alt = {"tau_floor": 0.95, "value": round(statistics.mean(alt_ms), 3),
               "chunk_ms_median": round(statistics.median(alt_ms), 3),
               "skip_rate": round(timed_rate(sa0, sa), 4)}
        log(f"tau_floor 0.95: mean {alt['value']:.2f} ms/chunk, skip rate {alt['skip_rate']:.3f}")

    # 1c. periodic whole-generation refresh: skip fraction per chunk
    cadence = None
    if args.force_every > 0:
        xc = make_xc(w.gate)
        counts = []
        cad_ms = [v[0] for v in run_stream(xc, m, eps_dev, actions, 0, n_chunks, torch,
                                           force_every=args.force_every, per_chunk=counts)]
        xc.close()
        per = [c - p for c, p in zip(counts, [0] + counts[:-1])]
        denom = m.n_blocks * m.n_steps
        cadence = {"force_every": args.force_every, "chunk_skip_fraction": [round(c / denom, 4) for c in per],
                   "mean_ms_after_warmup": round(statistics.mean(cad_ms[args.warmup:]), 3)}
        log(f"force every {args.force_every}: skip fractions {cadence['chunk_skip_fraction']}")

    # 2. gate off: the chunk latency without kernel events, then the same
    # chunks again with an event pair around every launch for the kernel table
    # (the events cost a few microseconds per launch: visible on small models)
    off_ms, kt = None, {}
    if not args.no_gate_off:
        xc = make_xc(synth.with_gate(w, enabled=0).gate)
        off_ms = [v[0] for v in run_stream(xc, m, eps_dev, actions, args.warmup, args.steps, torch)]
        xc.reset()
        run_stream(xc, m, eps_dev, actions, args.warmup, args.steps, torch, profile=True)
        kt = kernel_table(xc, xcp)
        xc.close()
        log(f"gate off: mean {statistics.mean(off_ms):.2f} ms/chunk")

    # 4. the gate-stress stream on the same shapes (scene cut every 8th chunk, steering step every 5th)
    stress = None
    if args.workload == 2 and not args.rope and not args.cond_len and not args.no_stress:
        ws = synth.workload(4)
        n_s = args.warmup + args.steps
        e_s = [torch.from_numpy(e).cuda() for e in synth.latent_stream(m, ws.stream, args.seed, n_s)]
        a_s = list(synth.action_stream(m, ws.stream, args.seed, n_s))
        xc = make_xc(ws.gate)
        ss0 = {}
        s_ms = [v[0] for v in run_stream(xc, m, e_s, a_s, args.warmup, args.steps, torch,
                                         at_timed=lambda h: ss0.update(h.stats()))]
        ss = xc.stats()
        xc.close()
        del e_s
        stress = {"workload": ws.name, "value": round(statistics.mean(s_ms), 3),
                  "chunk_ms_median": round(statistics.median(s_ms), 3), "skip_rate": round(timed_rate(ss0, ss), 4),
                  "chunk_ms": [round(v, 2) for v in s_ms]}
        if off_ms:
            stress["speedup_vs_full_compute"] = round(statistics.mean(off_ms) / stress["value"], 3)
        log(f"gate stress: mean {stress['value']:.2f} ms/chunk, skip rate {stress['skip_rate']:.3f}")

    Lk = m.kv_window * m.tokens  # every timed chunk sees the full window (warmup >= window - 1)
    steady = args.warmup >= m.kv_window - 1
    fl_block = block_flops(m, Lk)
    B, S = m.n_blocks, m.n_steps
    # skip rate over the timed chunks' denoising block evaluations (warmup chunks excluded)
    skip_rate = timed_rate(st0, st)
    on_mean = statistics.mean(on_ms)
    res = {
        "metric": METRIC,
        "value": round(on_mean, 3),
        "unit": "ms/chunk",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(on_mean, 3),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "blocks": B, "hidden": m.hidden, "heads": m.n_heads,
                   "head_dim": m.head_dim, "mlp_hidden": m.mlp_hidden, "tokens_per_chunk": m.tokens,
                   "kv_window_chunks": m.kv_window, "keys": Lk, "denoising_steps": S,
                   "rope": m.rope, "cross_attention_tokens": m.cond_len,
                   "stream_rho": w.stream.rho, "gate": "Table 1 defaults" if args.tau_floor is None
                   else f"Table 1 with tau_floor={args.tau_floor}", "steady_state_window": steady},
        "chunk_ms_median": round(statistics.median(on_ms), 3),
        "chunk_ms": [round(v, 2) for v in on_ms],
        "passes_ms_mean": round(statistics.mean(v[1] for v in on_split), 3),
        "kv_update_ms_mean": round(statistics.mean(v[2] for v in on_split), 3),
        "skip_rate": round(skip_rate, 4),
        "skips_timed": st["skips"] - st0["skips"],
        "block_evals_timed": st["evals_post_warmup"] - st0["evals_post_warmup"],
        # per (denoising step t, block b): skips over the whole stream, and the
        # gate's running cosine average s-bar after the last chunk
        "skip_counts_tb": np.asarray(st["skip_counts"]).reshape(S, B).astype(int).tolist(),
        "ema_cos_tb": [[None if not np.isfinite(v) else round(float(v), 5) for v in row]
                       for row in np.asarray(st["ema"]).reshape(S, B)],
    }
    # How close the gate runs to its threshold: with the adaptive threshold on
    # its floor, a (t, b) whose running cosine lies within a relative 1e-3 of
    # the floor takes decisions of which either is correct (the parity band),
    # so `skip_rate` and `value` depend on rounding there; the alt_tau_floor
    # and gate_stress legs decide outside it.
    ema = np.asarray(st["ema"], dtype=np.float64)
    ema = ema[np.isfinite(ema)]
    if ema.size and w.gate.adaptive:
        floor = float(w.gate.tau_floor)
        res["ema_near_floor"] = {"tau_floor": floor, "within_1e-3": int(np.sum(np.abs(ema - floor) <= 1e-3 * floor)),
                                 "gated_tb": int(ema.size)}
    if alt:
        res["alt_tau_floor"] = alt
    if stress:
        res["gate_stress"] = stress
    res["skip_path"] = skp
    res["gate_reading_input"] = cgate
    if cadence:
        res["periodic_refresh"] = cadence
    if off_ms:
        off_mean = statistics.mean(off_ms)
        chunk_flops = fl_block * B * (S + 1)
        res["full_compute_ms"] = round(off_mean, 3)
        res["speedup_vs_full_compute"] = round(off_mean / on_mean, 3)
        res["block_tflops_effective"] = round(chunk_flops / (off_mean * 1e-3) / 1e12, 1)
        res["block_mfma_frac_effective"] = round(res["block_tflops_effective"] / PEAK_BF16_TFLOPS, 4)
        contraction_ms = sum(kt[k]["total_ms"] for k in ("attention", "gemm_qkv", "gemm_oproj", "gemm_up",
                                                         "gemm_down", "cross_q", "cross_attention", "cross_o")
                             if k in kt)
        n_blocks_timed = args.steps * B * (S + 1)
        if contraction_ms > 0:
            res["block_tflops_kernels"] = round(fl_block * n_blocks_timed / (contraction_ms * 1e-3) / 1e12, 1)
        if "attention" in kt:
            a = kt["attention"]
            af = attention_flops(m, Lk)
            ach = af / (a["avg_us"] * 1e-6) / 1e12
            res["roofline"] = {"kernel": "attention", "bound": "mfma", "achieved": round(ach, 1),
                               "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4),
                               "traffic": measured_traffic("attention", w.name), "flops_per_launch": af, "avg_launch_us": round(a["avg_us"], 1)}
        gem = {"gemm_qkv": 6.0, "gemm_oproj": 2.0, "gemm_up": 2.0 * m.mlp_hidden / m.hidden,
               "gemm_down": 2.0 * m.mlp_hidden / m.hidden}
        res["kernels_full_compute"] = {}
        for k, v in kt.items():
            e = {"launches": v["launches"], "avg_us": round(v["avg_us"], 2)}
            if k in gem:
                f = gem[k] * m.tokens * m.hidden * m.hidden
                e["tflops"] = round(f / (v["avg_us"] * 1e-6) / 1e12, 1)
            if k == "attention":
                e["tflops"] = res["roofline"]["achieved"]
            if k == "cross_attention":
                e["tflops"] = round(attention_flops(m, m.cond_len) / (v["avg_us"] * 1e-6) / 1e12, 1)
            if k == "cross_o":
                e["tflops"] = round(2.0 * m.tokens * m.hidden * m.hidden / (v["avg_us"] * 1e-6) / 1e12, 1)
            if k == "ln_mod":
                e["gbs"] = round(6.0 * m.tokens * m.hidden / (v["avg_us"] * 1e-6) / 1e9, 1)
            res["kernels_full_compute"][k] = e
    # the MFMA rate a register-only loop sustains on random bf16 operands: the
    # practical ceiling the contraction kernels above can be read against
    # (context only; roofline.peak stays the published dense figure)
    ceil32 = xcp.xc_mfma_rate(0, True, torch.cuda.current_stream().cuda_stream)
    ceil16 = xcp.xc_mfma_rate(1, True, torch.cuda.current_stream().cuda_stream)
    res["mfma_ceiling"] = {"unit": "TFLOP/s", "operands": "random bf16",
                           "mfma_32x32x16": round(ceil32, 1), "mfma_16x16x32": round(ceil16, 1)}
    # the same 32x32x16 loop at the attention kernel's occupancy under its
    # instruction mix, on independent data: + one 16-byte LDS operand read per
    # MFMA, + a 64-key softmax tile's VALU work per 32 MFMAs, both -- what the
    # mix allows before any dependency or barrier is paid
    mix = {name: xcp.xc_mfma_rate(shape, True, torch.cuda.current_stream().cuda_stream)
           for name, shape in (("lds_reads", 2), ("softmax_valu", 3), ("lds_reads_and_softmax_valu", 4))}
    res["mfma_ceiling"]["attention_mix_32x32x16"] = {k: round(v, 1) for k, v in mix.items()}
    if "roofline" in res and ceil32 > 0:
        res["mfma_ceiling"]["attention_frac_of_32x32x16"] = round(res["roofline"]["achieved"] / ceil32, 4)
        if mix["lds_reads_and_softmax_valu"] > 0:
            res["mfma_ceiling"]["attention_frac_of_its_mix"] = round(
                res["roofline"]["achieved"] / mix["lds_reads_and_softmax_valu"], 4)
    if "block_tflops_effective" in res and ceil32 > 0:
        res["mfma_ceiling"]["block_effective_frac_of_32x32x16"] = round(res["block_tflops_effective"] / ceil32, 4)
    log(f"mfma ceiling: {ceil32:.0f} TFLOP/s (32x32x16), {ceil16:.0f} TFLOP/s (16x16x32), random operands; "
        f"attention mix {res['mfma_ceiling']['attention_mix_32x32x16']}")
    # the global -> LDS request stream the GEMMs stage operands with, by the
    # row segment one request fetches (why the wide GEMM uses 64-deep stages)
    res["lds_dma_rate"] = {"unit": "TB/s", **{f"rows_{rb}B": round(xcp.xc_lds_dma_rate(rb, torch.cuda.current_stream().cuda_stream), 2)
                                             for rb in (64, 128, 256)}}
    log(f"global -> LDS stream: {res['lds_dma_rate']}")
    if not args.no_cpu_baseline:
        log("cpu baseline: one oracle block at full shape ...")
        res["cpu_baseline"] = cpu_baseline(w, weights, args.seed)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
