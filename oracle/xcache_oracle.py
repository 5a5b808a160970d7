"""CPU oracle of the X-Cache cached chunk forward -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or run this module.  The product path (the HIP library
and its Python binding) never does, and this module imports nothing from it:
the two share only the seeded input generators in ``synth``.

What it computes, with the paper passage each piece follows:

* the AR rollout structure -- per generation n, S denoising passes over B
  blocks with residual connections, then one KV-update pass on the clean
  latent whose keys/values enter a FIFO rolling cache (Section 2.1, Eq. 1-2);
* cross-chunk residual caching and additive reuse keyed by (t, b)
  (Section 2.2, Eq. 3-4) with a warmup of W generations (Section 2.2.3);
* the fingerprint: a 3-D grid subsample of the block input per view group,
  a per-camera token-mean global channel and the per-chunk action vector
  (Section 2.3.1-2.3.2);
* the dual-metric gate: min-cosine over all entries (Eq. 5), max token
  deviation over the spatial group entries (Eq. 6), the skip rule (Eq. 7);
* the adaptive threshold from a per-(t, b) EMA of the cosine (Eq. 8-9);
* safety mechanisms: step-0 protection, anchor blocks, KV-update protection
  and maximum staleness (Section 2.5).

The DiT block itself is not specified by the paper beyond adaLN-Zero
conditioning on timestep and action (Sections 1 and 2.3.2); the block below is
a standard adaLN DiT block (LayerNorm without affine, six-way modulation,
QK-RMSNorm, softmax self-attention over the rolling cache, tanh-GELU MLP).
Two optional extensions move it toward the WAN-style blocks of the paper's
model (built on WAN 2.2, Section 3.1): a 3-D rotary position embedding of the
self-attention queries and keys over the latent (frame, row, column) grid,
with absolute frame positions across chunks, applied before the keys enter the
cache; and a cross-attention layer between the self-attention and the MLP that
attends to a condition token sequence (the text / object / lane embeddings the
paper injects through cross-attention, Sections 2.1 and 2.3.2).

Precision.  Arithmetic is float64.  For a bf16 model (the paper runs its DiT in
BF16, Section 3.1.1) values are rounded to bf16 (round to nearest even) at the
points where the model stores them and where that rounding does not depend on
how a kernel tiles the work: the Linear weights, the modulated LayerNorm
outputs, q/k/v after the QK-norm (the KV cache), the attention output, the
GELU output and the stored residuals.  For a float32 model no rounding is
applied.

Pins (see ``tests/test_oracle_*.py``): textbook spot values for the
elementwise functions, brute-force attention on tiny inputs and its closed
forms, hand-computed fingerprint indices and metric values, the gate truth
table and EMA closed form, hand-worked multi-generation decision sequences
(the threshold read before the EMA update, the action channel, the staleness
reset on compute: ``tests/gate_sequences.py``), and whole-stream invariants (zero thresholds give
zero skips and the uncached output, KV-update passes never skip, a skipped
block adds exactly its cached residual, zero adaLN weights make every block
the identity, an evicted chunk has no influence).  Beyond those invariants and
sequences the cached path as a whole has no independent numeric reference in
the paper: its multi-chunk outputs are "parity unpinned" except through them.
"""
from __future__ import annotations

import math
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

import synth

FORCE_FULL = 1           # forward flag: compute every block, still refresh caches
STEP0_OFF, STEP0_FORCE, STEP0_STRICT = 0, 1, 2
FP_GRID3D, FP_LINSPACE1D = 0, 1
FP_REFRESH_EVERY, FP_REFRESH_ON_COMPUTE = 0, 1   # when phi_prev takes the current fingerprint

# decision codes reported per block and pass
DEC_COMPUTE = 0          # gate evaluated, test failed -> computed
DEC_SKIP = 1             # gate evaluated, test passed -> cached residual added
DEC_FORCED = 2           # not evaluated (anchor, warmup, forced, gate off, no cache)


# ---------------------------------------------------------------------------
# Rounding
# ---------------------------------------------------------------------------

def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bf16 value (ties to even), as float64.

    bf16 keeps float32's 8 exponent bits and 7 mantissa bits; here the float64
    mantissa (52 bits) is rounded to 7 bits directly, so there is a single
    rounding.  Values are assumed to lie inside the float32 normal range or be
    exactly zero (true for every tensor of this model).
    """
    a = np.ascontiguousarray(a, dtype=np.float64)
    bits = a.view(np.uint64)
    drop = np.uint64(45)
    lsb = (bits >> drop) & np.uint64(1)
    bias = np.uint64((1 << 44) - 1) + lsb
    out = ((bits + bias) >> drop) << drop
    return out.view(np.float64)


# ---------------------------------------------------------------------------
# Elementwise and normalisation pieces of the block
# ---------------------------------------------------------------------------

def silu(x):
    return x / (1.0 + np.exp(-x))


def gelu_tanh(x):
    """GELU, tanh form: 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x * x * x)))


def layer_norm(x, eps=1e-6):
    """Row LayerNorm without affine parameters, biased variance."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def rms_norm(x, gain, eps=1e-6):
    """RMSNorm over the last axis, times a per-channel gain."""
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps) * gain


def timestep_embedding(tau: float, dim: int) -> np.ndarray:
    """Sinusoidal embedding [cos(tau f_i), sin(tau f_i)], f_i = 10000^(-i/h), h = dim/2."""
    h = dim // 2
    f = np.exp(-math.log(10000.0) * np.arange(h, dtype=np.float64) / h)
    return np.concatenate([np.cos(tau * f), np.sin(tau * f)])


def rope_axis_dims(d: int) -> Tuple[int, int, int]:
    """Head dimensions given to the (frame, row, column) axes of the 3-D rotary
    embedding: the row and column axes get 2 floor(d/6) each, the frame axis
    the rest (the split of WAN-style 3-D RoPE)."""
    s = d // 6
    return d - 4 * s, 2 * s, 2 * s


def rope_pair_frequencies(d: int, theta: float) -> Tuple[np.ndarray, np.ndarray]:
    """For each of the d/2 rotated pairs (2j, 2j+1) of a head: the axis it
    follows (0 frame, 1 row, 2 column) and its angular frequency theta^(-2i/d_a),
    i the pair's index within its axis's d_a/2 pairs."""
    axes, omega = [], []
    for a, da in enumerate(rope_axis_dims(d)):
        for i in range(da // 2):
            axes.append(a)
            omega.append(theta ** (-2.0 * i / da))
    return np.asarray(axes, dtype=np.int64), np.asarray(omega, dtype=np.float64)


def token_positions(groups: Sequence[synth.ViewGroup], n: int) -> np.ndarray:
    """[L, 3] positions (n F + f, h, w) of generation n's tokens: camera-major,
    each camera's (f, h, w) grid row-major; the frame position is absolute
    across chunks (F frames per chunk), so keys cached from earlier chunks keep
    their own frame positions."""
    out = []
    for g in groups:
        for _v in range(g.views):
            for f in range(g.frames):
                for hh in range(g.height):
                    for ww in range(g.width):
                        out.append((n * g.frames + f, hh, ww))
    return np.asarray(out, dtype=np.float64)


def apply_rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate each pair (x[2j], x[2j+1]) of every head by the angle p_a omega_j,
    p_a the token's position on the pair's axis: x [L, H, d], pos [L, 3]."""
    axes, omega = rope_pair_frequencies(x.shape[-1], theta)
    ang = pos[:, axes] * omega
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    a, b = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2] = a * c - b * s
    out[..., 1::2] = a * s + b * c
    return out


def softmax_attention(q, k, v):
    """Plain softmax(q k^T / sqrt(d)) v for one head: q [Lq, d], k/v [Lk, d]."""
    d = q.shape[-1]
    s = (q @ k.T) / math.sqrt(d)
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    return (p @ v) / p.sum(axis=-1, keepdims=True)


# ---------------------------------------------------------------------------
# Fingerprint (Section 2.3.1-2.3.2)
# ---------------------------------------------------------------------------

def axis_counts(frames: int, height: int, width: int, budget: int) -> Tuple[int, int, int]:
    """Per-axis sample counts proportional to the grid's aspect ratio with
    product about ``budget``: each axis gets round(dim * s) clamped to
    [1, dim], where s = (budget / (F H W))^(1/3) is the common scale."""
    s = (budget / float(frames * height * width)) ** (1.0 / 3.0)
    out = []
    for dim in (frames, height, width):
        k = int(math.floor(dim * s + 0.5))
        out.append(min(max(k, 1), dim))
    return tuple(out)


def axis_indices(dim: int, k: int) -> List[int]:
    """k uniformly spaced indices over [0, dim-1], floored: floor(i (dim-1) / (k-1))."""
    if k <= 1:
        return [0]
    return [(i * (dim - 1)) // (k - 1) for i in range(k)]


def fingerprint_rows(groups: Sequence[synth.ViewGroup], budget: int,
                     mode: int = FP_GRID3D) -> List[np.ndarray]:
    """Global token rows sampled per view group, shape [V_g, K'_g] each.

    Tokens are camera-major; within a camera the (f, h, w) grid is row-major.
    A camera with no more than ``budget`` tokens keeps all of them.  In the
    3-D mode the sample is the Cartesian product of per-axis indices; the 1-D
    fallback takes ``min(budget, T)`` uniformly spaced tokens along the
    flattened axis.
    """
    out = []
    start = 0
    for g in groups:
        T = g.tokens_per_view
        if T <= budget:
            local = list(range(T))
        elif mode == FP_LINSPACE1D:
            local = axis_indices(T, min(budget, T))
        else:
            kf, kh, kw = axis_counts(g.frames, g.height, g.width, budget)
            local = [f * g.height * g.width + h * g.width + w
                     for f in axis_indices(g.frames, kf)
                     for h in axis_indices(g.height, kh)
                     for w in axis_indices(g.width, kw)]
        local = np.asarray(local, dtype=np.int64)
        rows = np.stack([start + v * T + local for v in range(g.views)])
        out.append(rows)
        start += g.tokens
    return out


def fingerprint(x: np.ndarray, groups: Sequence[synth.ViewGroup],
                rows: Sequence[np.ndarray]) -> List[Tuple[np.ndarray, np.ndarray]]:
    """Per view group: (spatial sample flattened [V K' C], global channel [V C]).

    The global channel is each camera's mean over its tokens (the
    per-view-group sequence mean, one vector per camera stacked along V).
    """
    out = []
    start = 0
    for g, r in zip(groups, rows):
        spatial = x[r.reshape(-1)].reshape(-1)
        blk = x[start:start + g.tokens].reshape(g.views, g.tokens_per_view, -1)
        glob = blk.mean(axis=1).reshape(-1)
        out.append((spatial, glob))
        start += g.tokens
    return out


def cosine(u: np.ndarray, v: np.ndarray) -> float:
    """Eq. 5 for one entry; a zero-norm entry gives 0 (never passes a positive threshold)."""
    den = float(np.linalg.norm(u) * np.linalg.norm(v))
    return float(np.dot(u, v)) / max(den, 1e-12)


def max_deviation(cur: np.ndarray, prev: np.ndarray, eps: float) -> float:
    """Eq. 6 for one group: max|cur - prev| / (mean|prev| + eps)."""
    return float(np.max(np.abs(cur - prev))) / (float(np.mean(np.abs(prev))) + eps)


def gate_metrics(fp, fp_prev, action, action_prev, eps):
    """(s, d): min cosine over every entry (spatial and global per group, plus
    the action channel), max deviation over the spatial group entries."""
    cos_terms = []
    dev_terms = []
    for (sp, gl), (sp0, gl0) in zip(fp, fp_prev):
        cos_terms.append(cosine(sp, sp0))
        cos_terms.append(cosine(gl, gl0))
        dev_terms.append(max_deviation(sp, sp0, eps))
    if action is not None and action_prev is not None:
        cos_terms.append(cosine(np.asarray(action, np.float64), np.asarray(action_prev, np.float64)))
    return min(cos_terms), max(dev_terms)


# ---------------------------------------------------------------------------
# Threshold and decision (Eq. 7-9, Section 2.5)
# ---------------------------------------------------------------------------

def cosine_threshold(g: synth.GateParams, ema: Optional[float], t: int) -> float:
    """tau_cos(t, b): max(tau_floor, ema - m) from the EMA *before* this
    evaluation's update (the floor alone on the first evaluation); the fixed
    threshold when adaptation is off; at t = 0 in strict step-0 mode at least
    tau_strict0."""
    if g.adaptive:
        tau = g.tau_floor if ema is None else max(g.tau_floor, ema - g.margin)
    else:
        tau = g.tau_cos_fixed
    if t == 0 and g.step0_mode == STEP0_STRICT:
        tau = max(tau, g.tau_strict0)
    return tau


def ema_update(g: synth.GateParams, ema: Optional[float], s: float) -> float:
    """Eq. 8: ema <- alpha s + (1 - alpha) ema, seeded with s on the first evaluation."""
    return s if ema is None else g.alpha * s + (1.0 - g.alpha) * ema


def skip_rule(g: synth.GateParams, s: float, d: float, tau: float, stale: int) -> bool:
    """Eq. 7 plus the staleness bound: skip iff s >= tau and d < tau_dev and
    (M off or fewer than M consecutive skips so far)."""
    return (s >= tau) and (d < g.tau_dev) and (g.max_stale == 0 or stale < g.max_stale)


# ---------------------------------------------------------------------------
# The DiT block
# ---------------------------------------------------------------------------

class BlockWeights:
    def __init__(self, m: synth.ModelShape, blob: np.ndarray, b: int, compute=np.float64):
        t = synth.split_block_weights(m, blob, b)
        lin = ("w_ada", "wq", "wk", "wv", "wo", "w1", "w2", "wq_c", "wk_c", "wv_c", "wo_c")
        self.p = {}
        for name, a in t.items():
            a = np.asarray(a, dtype=np.float64)
            if m.dtype == synth.BF16 and name in lin:
                a = bf16_round(a)
            self.p[name] = a.astype(compute)


class XCacheOracle:
    """Step-by-step CPU model of the cached rollout.

    API mirrors the library: ``forward_chunk`` (one denoising pass of the
    current generation), ``kv_update`` (the full clean pass that commits K/V
    and advances the generation), ``stats``.
    """

    def __init__(self, model: synth.ModelShape, gate: synth.GateParams,
                 weights: np.ndarray, compute=np.float64):
        self.m = model
        self.g = gate
        self.compute = compute
        self.bf16 = model.dtype == synth.BF16
        self.blocks = [BlockWeights(model, weights, b, compute) for b in range(model.n_blocks)]
        self.rows = fingerprint_rows(model.groups, gate.fp_budget, gate.fp_mode)
        self.cross_kv: Optional[List[Tuple[np.ndarray, np.ndarray]]] = None
        self.reset()

    def set_condition(self, cond: np.ndarray):
        """Condition tokens [n, C] (1 <= n <= cond_len) of the cross-attention
        layer; each block's keys and values of them are computed here once and
        used by every later pass until the next call."""
        m = self.m
        cond = np.asarray(cond, dtype=np.float64)
        assert m.cond_len > 0 and cond.ndim == 2 and 1 <= cond.shape[0] <= m.cond_len
        assert cond.shape[1] == m.hidden
        n, H, d = cond.shape[0], m.n_heads, m.head_dim
        cr = self._rnd(cond)
        self.cross_kv = []
        for b in range(m.n_blocks):
            p = self.blocks[b].p
            k = self._rnd(rms_norm((cr @ p["wk_c"].T + p["bk_c"]).reshape(n, H, d), p["gk_c"]))
            v = self._rnd((cr @ p["wv_c"].T + p["bv_c"]).reshape(n, H, d))
            self.cross_kv.append((np.ascontiguousarray(k.transpose(1, 0, 2)),
                                  np.ascontiguousarray(v.transpose(1, 0, 2))))

    # -- state ---------------------------------------------------------------
    def reset(self):
        S, B = self.m.n_steps, self.m.n_blocks
        self.n = 0
        self.ring: List[List[Tuple[np.ndarray, np.ndarray]]] = [[] for _ in range(B)]
        self.fp_prev: Dict[Tuple[int, int], list] = {}
        self.rhat: Dict[Tuple[int, int], np.ndarray] = {}
        self.ema: Dict[Tuple[int, int], float] = {}
        self.stale = np.zeros((S, B), dtype=np.int64)
        self.action_prev: Optional[np.ndarray] = None
        self.skip_counts = np.zeros((S, B), dtype=np.int64)
        self.evals_post_warmup = 0
        self.gated_evals = 0
        self.skips = 0
        self.kv_block_evals = 0
        self.last = None

    def _rnd(self, a):
        return bf16_round(a).astype(self.compute) if self.bf16 else a

    def gateable(self, b: int) -> bool:
        g = self.g
        return bool(g.enabled) and g.front_anchors <= b < self.m.n_blocks - g.back_anchors

    # -- the block -----------------------------------------------------------
    def block(self, b: int, x: np.ndarray, cond: np.ndarray, rows=None):
        """One DiT block on input x [L, C]; returns (y, (k, v)) with k/v [H, L, d].

        ``rows`` (token indices) restricts y to those rows: keys and values
        still come from every token, the queries and everything after the
        attention only from those rows (each output row depends on the other
        tokens only through the keys and values)."""
        m, p = self.m, self.blocks[b].p
        L, C, H, d = m.tokens, m.hidden, m.n_heads, m.head_dim
        mod = p["w_ada"] @ silu(cond) + p["b_ada"]
        sh1, sc1, g1, sh2, sc2, g2 = np.split(mod, 6)
        h = self._rnd(layer_norm(x) * (1.0 + sc1) + sh1)
        if rows is not None:
            x = x[rows]
            Lq = len(rows)
        else:
            Lq = L
        q = h[rows if rows is not None else slice(None)] @ p["wq"].T + p["bq"]
        k = h @ p["wk"].T + p["bk"]
        v = h @ p["wv"].T + p["bv"]
        q = rms_norm(q.reshape(Lq, H, d), p["gq"])
        k = rms_norm(k.reshape(L, H, d), p["gk"])
        if m.rope:
            pos = token_positions(m.groups, self.n)
            q = apply_rope(q, pos[rows] if rows is not None else pos, m.rope_theta)
            k = apply_rope(k, pos, m.rope_theta)
        q = self._rnd(q)
        k = self._rnd(k)
        v = self._rnd(v.reshape(L, H, d))
        kh = np.ascontiguousarray(k.transpose(1, 0, 2))
        vh = np.ascontiguousarray(v.transpose(1, 0, 2))
        kall = np.concatenate([pk for pk, _ in self.ring[b]] + [kh], axis=1)
        vall = np.concatenate([pv for _, pv in self.ring[b]] + [vh], axis=1)
        o = np.empty((Lq, H, d), dtype=self.compute)
        for hd in range(H):
            o[:, hd, :] = softmax_attention(q[:, hd, :], kall[hd], vall[hd])
        o = self._rnd(o.reshape(Lq, C))
        x1 = x + g1 * (o @ p["wo"].T + p["bo"])
        if m.cond_len > 0:
            x1 = self.cross_attention(b, x1)
        h2 = self._rnd(layer_norm(x1) * (1.0 + sc2) + sh2)
        u = self._rnd(gelu_tanh(h2 @ p["w1"].T + p["b1"]))
        y = x1 + g2 * (u @ p["w2"].T + p["b2"])
        return y, (kh, vh)

    def cross_attention(self, b: int, x1: np.ndarray) -> np.ndarray:
        """The cross-attention layer of block b on its rows x1 [Lq, C]: affine
        LayerNorm, q projection with RMSNorm, softmax attention over the
        condition's keys and values, output projection added to the stream
        (no adaLN gate)."""
        m, p = self.m, self.blocks[b].p
        assert self.cross_kv is not None, "set_condition() first"
        Lq, C, H, d = x1.shape[0], m.hidden, m.n_heads, m.head_dim
        kc, vc = self.cross_kv[b]
        hc = self._rnd(layer_norm(x1) * p["ln3_w"] + p["ln3_b"])
        qc = self._rnd(rms_norm((hc @ p["wq_c"].T + p["bq_c"]).reshape(Lq, H, d), p["gq_c"]))
        oc = np.empty((Lq, H, d), dtype=self.compute)
        for hd in range(H):
            oc[:, hd, :] = softmax_attention(qc[:, hd, :], kc[hd], vc[hd])
        oc = self._rnd(oc.reshape(Lq, C))
        return x1 + (oc @ p["wo_c"].T + p["bo_c"])

    def cond(self, tau: float, action: np.ndarray) -> np.ndarray:
        return np.concatenate([timestep_embedding(tau, self.m.temb_dim),
                               np.asarray(action, dtype=np.float64)]).astype(self.compute)

    # -- one denoising pass ----------------------------------------------------
    def forward_chunk(self, t: int, tau: float, action: np.ndarray, x: np.ndarray,
                      flags: int = 0,
                      decide: Optional[Callable[[int, dict], bool]] = None, rows=None) -> np.ndarray:
        """Denoising step t of generation n (Eq. 1) under the X-Cache gate.

        ``decide(b, info)`` may override the skip decision of an evaluated
        block (the tests use it to follow the device where a metric sits
        within the tolerance band of its threshold); ``info`` holds the
        oracle's own ``s``, ``d``, ``tau`` and ``skip``.

        ``rows`` (token indices) is a checking mode for large shapes: the last
        block's output is computed, and returned, for those rows only, and
        that block's cached residual is then left as it was (everything else,
        the gate included, proceeds in full).
        """
        m, g = self.m, self.g
        assert 0 <= t < m.n_steps
        x = np.asarray(x, dtype=self.compute).copy()
        c = self.cond(tau, action)
        forced_all = ((not g.enabled) or self.n < g.warmup or bool(flags & FORCE_FULL)
                      or (t == 0 and g.step0_mode == STEP0_FORCE))
        record = []
        for b in range(m.n_blocks):
            info = {"decision": DEC_FORCED, "s": math.nan, "d": math.nan, "tau": math.nan}
            skip = False
            key = (t, b)
            gate_b = self.gateable(b)
            fp = fingerprint(x, m.groups, self.rows) if gate_b else None
            if gate_b and not forced_all and key in self.fp_prev and key in self.rhat:
                s, dmax = gate_metrics(fp, self.fp_prev[key], action, self.action_prev, g.eps)
                tau_c = cosine_threshold(g, self.ema.get(key), t)
                if g.adaptive:
                    self.ema[key] = ema_update(g, self.ema.get(key), s)
                skip = skip_rule(g, s, dmax, tau_c, int(self.stale[t, b]))
                info.update(s=s, d=dmax, tau=tau_c, skip=skip)
                if decide is not None:
                    skip = bool(decide(b, info))
                info["decision"] = DEC_SKIP if skip else DEC_COMPUTE
                self.gated_evals += 1
            # Section 2.5 keeps the fingerprint cache refreshed; by default at
            # every evaluation of (t, b), alternatively only when it computes
            if gate_b and (g.fp_refresh == FP_REFRESH_EVERY or not skip):
                self.fp_prev[key] = fp
            restrict = rows is not None and b == m.n_blocks - 1
            if skip:
                x = x[rows] + self.rhat[key][rows] if restrict else x + self.rhat[key]
                self.stale[t, b] += 1
            else:
                y, _ = self.block(b, x, c, rows if restrict else None)
                if gate_b and not restrict:
                    self.rhat[key] = self._rnd(y - x)
                self.stale[t, b] = 0
                x = y
            if self.n >= g.warmup:
                self.evals_post_warmup += 1
                if skip:
                    self.skips += 1
                    self.skip_counts[t, b] += 1
            record.append(info)
        self.last = record
        return x

    # -- the KV-update pass ----------------------------------------------------
    def kv_update(self, tau: float, action: np.ndarray, x: np.ndarray, rows=None) -> np.ndarray:
        """Full pass on the clean latent, never gated; commits K/V FIFO (Section 2.1, 2.5).
        ``rows`` restricts the returned output to those token rows (the last
        block's keys and values still come from every token)."""
        m = self.m
        x = np.asarray(x, dtype=self.compute).copy()
        c = self.cond(tau, action)
        new_kv = []
        for b in range(m.n_blocks):
            x, kv = self.block(b, x, c, rows if b == m.n_blocks - 1 else None)
            new_kv.append(kv)
        for b in range(m.n_blocks):
            self.ring[b].append(new_kv[b])
            while len(self.ring[b]) > m.kv_window - 1:
                self.ring[b].pop(0)
        self.kv_block_evals += m.n_blocks
        self.action_prev = np.asarray(action, dtype=np.float64).copy()
        self.n += 1
        return x

    def stats(self) -> dict:
        return {"generations": self.n, "evals_post_warmup": self.evals_post_warmup,
                "gated_evals": self.gated_evals, "skips": self.skips,
                "kv_block_evals": self.kv_block_evals,
                "skip_counts": self.skip_counts.copy()}


def rollout(orc: XCacheOracle, eps_chunks, actions, n_chunks: int,
            forward_flags: Callable[[int, int], int] = lambda n, t: 0,
            on_pass: Optional[Callable] = None):
    """Drive the oracle through ``n_chunks`` generations with the harness sampler.

    x_0 = eps_n; after pass t, x_{t+1} = (1 - sigma_{t+1}) y_t + sigma_{t+1} eps_n;
    the clean latent y_{S-1} feeds the KV-update pass.  ``on_pass(n, t, y)`` is
    called after every pass (t == S for the KV-update pass).
    """
    m = orc.m
    taus = synth.timesteps(m)
    outs = []
    for n, eps, a in zip(range(n_chunks), eps_chunks, actions):
        eps = np.asarray(eps, dtype=np.float64)
        x = eps
        y = None
        for t in range(m.n_steps):
            y = orc.forward_chunk(t, taus[t], a, x, forward_flags(n, t))
            if on_pass:
                on_pass(n, t, y)
            if t + 1 < m.n_steps:
                sg = synth.sampler_sigma(m, t + 1)
                x = (1.0 - sg) * y + sg * eps
        yk = orc.kv_update(synth.KV_UPDATE_TIMESTEP, a, y)
        if on_pass:
            on_pass(n, m.n_steps, yk)
        outs.append(y)
    return outs
