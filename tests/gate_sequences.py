"""Hand-built gate streams whose decisions, thresholds and EMA values are
worked out by hand from the paper's equations.

Every block of the model is the identity (all adaLN weights and biases zero
make both adaLN gates zero, so y = x exactly), so each block's input is the
chunk's latent x.  Every token row of generation n's latent is the same unit
vector r_n = (cos theta_n, sin theta_n, 0, ...), so the spatial fingerprint
and each camera's token mean are copies of r_n and the cross-chunk cosine of
both equals cos(theta_n - theta_{n-1}) (Eq. 5).  Consecutive latents are
rotated by arccos(s_n) for a chosen s_n.  Actions are unit vectors at chosen
angles in one plane, so the action channel's cosine is the cosine of the
angle between consecutive actions.  The deviation metric (Eq. 6) is switched
off with tau_dev = +inf, so the decision is the cosine test alone.

The expected values in each sequence below are the hand arithmetic of the
paper's rules, written out as literals:

* EMA: first evaluation of (t, b) uses tau_floor and seeds the EMA with s;
  later evaluations take tau = max(tau_floor, ema - m) from the EMA *before*
  this evaluation, then update ema <- alpha s + (1 - alpha) ema
  (Section 2.4, Eq. 8-9).
* ACTION: the action channel is one more cosine entry of the min (Section
  2.3.2 auxiliary channels, Eq. 5), taken against the previous generation's
  action.
* STALE: with a maximum staleness M, a block that has skipped M times in a row
  recomputes, and any recompute restarts the count (Section 2.5).

Generation 0 is the warmup (W = 1, Section 2.2.3): every block computes and
fills the caches.  Block 0 is the front anchor (F_n = 1); block 1 is gated.
There is one denoising step per generation (S = 1) so each generation
evaluates (t, b) = (0, 1) exactly once.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import numpy as np

import synth

NAN = math.nan
F, C, S = 2, 0, 1   # forced (not evaluated), compute, skip -- the library's decision codes


@dataclasses.dataclass(frozen=True)
class Sequence:
    name: str
    gate: synth.GateParams
    latent_cos: List[Optional[float]]     # s_n of the latent vs generation n-1 (None for n = 0)
    action_deg: List[float]               # action angle per generation, degrees
    decision: List[int]                   # expected decision of block 1 per generation
    s: List[float]                        # expected min-cosine (NaN where not evaluated)
    tau: List[float]                      # expected cosine threshold
    ema: List[float]                      # expected EMA after the evaluation (NaN if not adaptive)


def model() -> synth.ModelShape:
    """The tiny float32 model's shapes with one denoising step."""
    return dataclasses.replace(synth.workload(0).model, n_steps=1)


def identity_weights(m: synth.ModelShape) -> np.ndarray:
    blob = synth.make_weights(m)
    for b in range(m.n_blocks):
        t = synth.split_block_weights(m, blob, b)
        t["w_ada"][...] = 0.0
        t["b_ada"][...] = 0.0
    return blob


def latents(m: synth.ModelShape, seq: Sequence) -> List[np.ndarray]:
    theta = 0.3
    out = []
    for n, s in enumerate(seq.latent_cos):
        if n > 0:
            theta += math.acos(s)
        r = np.zeros(m.hidden, np.float64)
        r[0], r[1] = math.cos(theta), math.sin(theta)
        out.append(np.tile(r, (m.tokens, 1)).astype(np.float32))
    return out


def actions(m: synth.ModelShape, seq: Sequence) -> List[np.ndarray]:
    out = []
    for deg in seq.action_deg:
        a = np.zeros(m.action_dim, np.float64)
        a[0], a[1] = math.cos(math.radians(deg)), math.sin(math.radians(deg))
        out.append(a.astype(np.float32))
    return out


_INF = math.inf

EMA_ORDER = Sequence(
    "ema_order",
    synth.GateParams(adaptive=1, tau_floor=0.5, margin=0.02, alpha=0.3, tau_dev=_INF),
    latent_cos=[None, 0.99, 0.965, 0.964, 0.955],
    action_deg=[0.0] * 5,
    # e1: tau = floor 0.5, 0.99 passes; ema = 0.99
    # e2: tau = 0.99 - 0.02 = 0.97 > 0.965 -> compute; ema = 0.3*0.965 + 0.7*0.99 = 0.9825
    # e3: tau = 0.9825 - 0.02 = 0.9625 <= 0.964 -> skip; ema = 0.3*0.964 + 0.7*0.9825 = 0.97695
    # e4: tau = 0.97695 - 0.02 = 0.95695 > 0.955 -> compute; ema = 0.3*0.955 + 0.7*0.97695 = 0.970365
    decision=[F, S, C, S, C],
    s=[NAN, 0.99, 0.965, 0.964, 0.955],
    tau=[NAN, 0.5, 0.97, 0.9625, 0.95695],
    ema=[NAN, 0.99, 0.9825, 0.97695, 0.970365],
)

ACTION_CHANNEL = Sequence(
    "action_channel",
    synth.GateParams(adaptive=0, tau_cos_fixed=0.9, tau_dev=_INF),
    latent_cos=[None, 1.0, 1.0, 1.0, 0.95, 1.0],
    action_deg=[0.0, 0.0, 60.0, 60.0, 70.0, 100.0],
    # n1: identical latent and action -> s = 1, skip
    # n2: identical latent, action turned by 60 deg -> s = cos 60 = 0.5 < 0.9, compute
    # n3: action as in n2 (the comparison is with the previous generation) -> s = 1, skip
    # n4: latent cos 0.95, action turned by 10 deg (cos 0.98481) -> s = 0.95, skip
    # n5: identical latent, action turned by 30 deg -> s = cos 30 = 0.8660254 < 0.9, compute
    decision=[F, S, C, S, S, C],
    s=[NAN, 1.0, 0.5, 1.0, 0.95, 0.8660254037844387],
    tau=[NAN, 0.9, 0.9, 0.9, 0.9, 0.9],
    ema=[NAN] * 6,
)

STALE_M2 = Sequence(
    "stale_m2",
    synth.GateParams(adaptive=0, tau_cos_fixed=0.9, tau_dev=_INF, max_stale=2),
    latent_cos=[None, 0.99, 0.5, 0.99, 0.99, 0.99, 0.99, 0.99],
    action_deg=[0.0] * 8,
    # n1 skip (1 in a row); n2 s = 0.5 fails -> compute, count restarts at 0; n3 skip (1);
    # n4 skip (2); n5 two skips in a row = M -> compute (0); n6 skip (1); n7 skip (2)
    decision=[F, S, C, S, S, C, S, S],
    s=[NAN, 0.99, 0.5, 0.99, 0.99, 0.99, 0.99, 0.99],
    tau=[NAN] + [0.9] * 7,
    ema=[NAN] * 8,
)

STALE_M1 = Sequence(
    "stale_m1",
    synth.GateParams(adaptive=0, tau_cos_fixed=0.9, tau_dev=_INF, max_stale=1),
    latent_cos=[None, 0.99, 0.99, 0.99, 0.99, 0.99],
    action_deg=[0.0] * 6,
    # every cosine passes; M = 1 allows one skip after each compute
    decision=[F, S, C, S, C, S],
    s=[NAN] + [0.99] * 5,
    tau=[NAN] + [0.9] * 5,
    ema=[NAN] * 6,
)

ALL = [EMA_ORDER, ACTION_CHANNEL, STALE_M2, STALE_M1]
