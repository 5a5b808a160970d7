"""Seeded synthetic inputs shared by the oracle and the HIP path.

This module holds the workload presets and the random draws only: model
shapes, the flat weight blob, the AR(1) latent stream, the action random walk
and the denoising schedule that the rollout driver hands to both sides.  It
contains none of the caching method's arithmetic (no block, no fingerprint,
no gate), so importing it from the oracle and from the product path shares no
computation between them.

Stream recipe (the paper's workloads are internal multi-camera driving clips,
so these stand in for them with the same structure: per-chunk latent grids of
several cameras x 3 latent frames, 4 denoising steps, one action vector per
chunk, Section 3.1):

* weights: every Linear weight and bias ~ N(0, 0.02^2), drawn row-major
  [out, in] per block in the blob order below from ``default_rng(seed)``;
  QK-norm gains are 1; the cross-attention LayerNorm (models with a
  cross-attention layer) has scale 1 + N(0, 0.02^2) and shift N(0, 0.02^2).
* cross-attention condition (models that have one): [n_tokens, C] ~ N(0, 1)
  from ``default_rng(seed + 3)``.
* latent noise: eps_0 ~ N(0, I); eps_n = rho * eps_{n-1} + sqrt(1 - rho^2) z_n,
  from ``default_rng(seed + 1)``; optionally redrawn i.i.d. every ``cut_every``
  chunks (scene cut).
* actions: a_0 ~ N(0, I_A); a_n = a_{n-1} + sigma z'_n, from
  ``default_rng(seed + 2)``; optionally a step of ``big_sigma`` every
  ``big_every`` chunks (sharp steering).
* denoising schedule: sigma_t = 1 - t/S, timestep tau_t = 1000 sigma_t for the
  S denoising passes and tau = 0 for the KV-update pass; between passes the
  driver forms x_{t+1} = (1 - sigma_{t+1}) y_t + sigma_{t+1} eps_n (a plain
  few-step flow sampler; the paper does not state its sampler).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Iterator, List, Sequence, Tuple

import numpy as np

F32 = "f32"
BF16 = "bf16"


@dataclasses.dataclass(frozen=True)
class ViewGroup:
    """Cameras sharing one latent grid: ``views`` x (frames x height x width)."""
    views: int
    frames: int
    height: int
    width: int

    @property
    def tokens_per_view(self) -> int:
        return self.frames * self.height * self.width

    @property
    def tokens(self) -> int:
        return self.views * self.tokens_per_view


@dataclasses.dataclass(frozen=True)
class ModelShape:
    n_blocks: int
    hidden: int
    n_heads: int
    head_dim: int
    mlp_hidden: int
    temb_dim: int
    action_dim: int
    dtype: str
    n_steps: int
    kv_window: int          # chunks visible to attention, the current one included
    groups: Tuple[ViewGroup, ...]
    rope: int = 0           # 1: 3-D rotary position embedding on the self-attention q / k
    rope_theta: float = 10000.0
    cond_len: int = 0       # condition tokens of the cross-attention layer (0: no cross-attention)

    @property
    def tokens(self) -> int:
        return sum(g.tokens for g in self.groups)

    @property
    def cond_dim(self) -> int:
        return self.temb_dim + self.action_dim


@dataclasses.dataclass(frozen=True)
class GateParams:
    """Gate hyper-parameters (names follow Table 1 of the paper)."""
    enabled: int = 1
    fp_budget: int = 32           # K, tokens per fingerprint
    warmup: int = 1               # W
    front_anchors: int = 1        # F_n
    back_anchors: int = 0         # B_n
    adaptive: int = 1
    tau_floor: float = 0.97
    margin: float = 0.02          # m
    alpha: float = 0.30
    tau_cos_fixed: float = 0.95   # used when adaptive == 0
    tau_dev: float = 2.0
    eps: float = 1e-6
    max_stale: int = 0            # M, 0 = off
    step0_mode: int = 0           # 0 off, 1 force, 2 strict
    tau_strict0: float = 0.999
    kv_protect: int = 1
    fp_mode: int = 0              # 0 3-D grid, 1 1-D linspace fallback
    fp_refresh: int = 0           # 0 at every evaluation, 1 only when the block is computed


@dataclasses.dataclass(frozen=True)
class StreamParams:
    n_chunks: int
    rho: float
    action_sigma: float
    cut_every: int = 0            # scene cut period (0 = none)
    big_every: int = 0            # sharp steering period (0 = none)
    big_sigma: float = 1.0


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    gate: GateParams
    stream: StreamParams


def _workloads() -> List[Workload]:
    cfg0 = Workload(
        "tiny-fp32-dit-2blk-h128-L64",
        ModelShape(2, 128, 4, 32, 512, 64, 8, F32, 4, 2, (ViewGroup(1, 4, 4, 4),)),
        GateParams(adaptive=0, tau_cos_fixed=0.95, tau_dev=0.05),
        StreamParams(6, 0.95, 0.05),
    )
    cfg1 = Workload(
        "single-camera-bf16-dit-8blk-h512-L768",
        ModelShape(8, 512, 8, 64, 2048, 256, 16, BF16, 4, 4, (ViewGroup(1, 3, 16, 16),)),
        GateParams(),
        StreamParams(16, 0.95, 0.05),
    )
    cfg2 = Workload(
        "multi-camera-bf16-dit-20blk-h1536-L7020",
        ModelShape(20, 1536, 12, 128, 6144, 256, 16, BF16, 4, 3, (ViewGroup(6, 3, 15, 26),)),
        GateParams(),
        StreamParams(32, 0.97, 0.03),
    )
    cfg3 = Workload(
        "multi-camera-bf16-dit-30blk-h2048-L12096",
        ModelShape(30, 2048, 16, 128, 8192, 256, 16, BF16, 4, 4, (ViewGroup(7, 3, 18, 32),)),
        GateParams(),
        StreamParams(64, 0.97, 0.03),
    )
    cfg4 = Workload(
        "gate-stress-bf16-dit-20blk-h1536-L7020",
        cfg2.model,
        GateParams(),
        StreamParams(48, 0.98, 0.03, cut_every=8, big_every=5, big_sigma=1.0),
    )
    return [cfg0, cfg1, cfg2, cfg3, cfg4]


WORKLOADS: List[Workload] = _workloads()


def workload(i: int) -> Workload:
    return WORKLOADS[i]


def with_model(w: Workload, **kw) -> Workload:
    return dataclasses.replace(w, model=dataclasses.replace(w.model, **kw))


def with_gate(w: Workload, **kw) -> Workload:
    return dataclasses.replace(w, gate=dataclasses.replace(w.gate, **kw))


def with_stream(w: Workload, **kw) -> Workload:
    return dataclasses.replace(w, stream=dataclasses.replace(w.stream, **kw))


# ---------------------------------------------------------------------------
# Weight blob.  Per block, in this order, row-major [out, in]:
#   W_ada [6C, D_c], b_ada [6C], Wq [C, C], bq [C], Wk [C, C], bk [C],
#   Wv [C, C], bv [C], Wo [C, C], bo [C], W1 [D_m, C], b1 [D_m],
#   W2 [C, D_m], b2 [C], gq [d], gk [d]
# and, for a model with a cross-attention layer (cond_len > 0), then
#   ln3_w [C], ln3_b [C], Wq_c [C, C], bq_c [C], Wk_c [C, C], bk_c [C],
#   Wv_c [C, C], bv_c [C], Wo_c [C, C], bo_c [C], gq_c [d], gk_c [d]
# Blocks are concatenated; the blob is float32.
# ---------------------------------------------------------------------------

_GAINS = ("gq", "gk", "gq_c", "gk_c")


def block_tensor_shapes(m: ModelShape) -> List[Tuple[str, Tuple[int, ...]]]:
    C, Dc, Dm, d = m.hidden, m.cond_dim, m.mlp_hidden, m.head_dim
    shapes = [
        ("w_ada", (6 * C, Dc)), ("b_ada", (6 * C,)),
        ("wq", (C, C)), ("bq", (C,)),
        ("wk", (C, C)), ("bk", (C,)),
        ("wv", (C, C)), ("bv", (C,)),
        ("wo", (C, C)), ("bo", (C,)),
        ("w1", (Dm, C)), ("b1", (Dm,)),
        ("w2", (C, Dm)), ("b2", (C,)),
        ("gq", (d,)), ("gk", (d,)),
    ]
    if m.cond_len > 0:
        shapes += [
            ("ln3_w", (C,)), ("ln3_b", (C,)),
            ("wq_c", (C, C)), ("bq_c", (C,)),
            ("wk_c", (C, C)), ("bk_c", (C,)),
            ("wv_c", (C, C)), ("bv_c", (C,)),
            ("wo_c", (C, C)), ("bo_c", (C,)),
            ("gq_c", (d,)), ("gk_c", (d,)),
        ]
    return shapes


def block_numel(m: ModelShape) -> int:
    return sum(int(np.prod(s)) for _, s in block_tensor_shapes(m))


def weights_numel(m: ModelShape) -> int:
    return m.n_blocks * block_numel(m)


def make_weights(m: ModelShape, seed: int = 0, std: float = 0.02) -> np.ndarray:
    """Flat float32 blob: Linear weights and biases N(0, std^2), QK-norm gains 1,
    cross-attention LayerNorm scale 1 + N(0, std^2) and shift N(0, std^2)."""
    rng = np.random.default_rng(seed)
    out = np.empty(weights_numel(m), dtype=np.float32)
    off = 0
    for _ in range(m.n_blocks):
        for name, shape in block_tensor_shapes(m):
            n = int(np.prod(shape))
            if name in _GAINS:
                out[off:off + n] = 1.0
            elif name == "ln3_w":
                out[off:off + n] = (1.0 + rng.standard_normal(n) * std).astype(np.float32)
            else:
                out[off:off + n] = (rng.standard_normal(n) * std).astype(np.float32)
            off += n
    return out


def split_block_weights(m: ModelShape, blob: np.ndarray, b: int) -> dict:
    """Views of block ``b``'s tensors inside the flat blob (no copies)."""
    off = b * block_numel(m)
    out = {}
    for name, shape in block_tensor_shapes(m):
        n = int(np.prod(shape))
        out[name] = blob[off:off + n].reshape(shape)
        off += n
    return out


# ---------------------------------------------------------------------------
# Streams
# ---------------------------------------------------------------------------

def latent_stream(m: ModelShape, s: StreamParams, seed: int = 0,
                  n_chunks: int | None = None) -> Iterator[np.ndarray]:
    """Yields eps_n as float32 [L, C], camera-major, each camera (f, h, w) row-major."""
    rng = np.random.default_rng(seed + 1)
    n_chunks = s.n_chunks if n_chunks is None else n_chunks
    shape = (m.tokens, m.hidden)
    a = math.sqrt(max(0.0, 1.0 - s.rho * s.rho))
    eps = None
    for n in range(n_chunks):
        z = rng.standard_normal(shape)
        if eps is None or (s.cut_every and n % s.cut_every == 0):
            eps = z
        else:
            eps = s.rho * eps + a * z
        yield eps.astype(np.float32)


def action_stream(m: ModelShape, s: StreamParams, seed: int = 0,
                  n_chunks: int | None = None) -> Iterator[np.ndarray]:
    """Yields a_n as float32 [A]."""
    rng = np.random.default_rng(seed + 2)
    n_chunks = s.n_chunks if n_chunks is None else n_chunks
    a = None
    for n in range(n_chunks):
        z = rng.standard_normal(m.action_dim)
        if a is None:
            a = z
        else:
            step = s.big_sigma if (s.big_every and n % s.big_every == 0) else s.action_sigma
            a = a + step * z
        yield a.astype(np.float32)


def condition_tokens(m: ModelShape, seed: int = 0, n_tokens: int | None = None) -> np.ndarray:
    """The cross-attention condition: float32 [n_tokens, C] ~ N(0, 1) from
    ``default_rng(seed + 3)`` (stands in for the text / object / lane embeddings)."""
    n = m.cond_len if n_tokens is None else n_tokens
    rng = np.random.default_rng(seed + 3)
    return rng.standard_normal((n, m.hidden)).astype(np.float32)


def timesteps(m: ModelShape) -> List[float]:
    """tau_t for the S denoising passes (the KV-update pass uses tau = 0)."""
    return [1000.0 * (1.0 - t / m.n_steps) for t in range(m.n_steps)]


def sampler_sigma(m: ModelShape, t: int) -> float:
    """sigma_t = 1 - t/S; the driver forms x_{t+1} = (1-sigma) y_t + sigma eps."""
    return 1.0 - t / m.n_steps


KV_UPDATE_TIMESTEP = 0.0
