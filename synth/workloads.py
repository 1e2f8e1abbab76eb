"""Shapes and seeded draws for the five benchmark workloads.

Workloads (names used everywhere in this repository):

``tiny_fp32``   2 layers, width 128, 4 heads x 32, MLP 512, H=8 slots of
                action dim 7, 32 prefix tokens, 4 FOP tokens (32-d obs), fp32,
                batch 1, 200 steps.
``small_bf16``  6 layers, width 512, 8 heads x 64, MLP 2048, H=16, action dim
                14, 256 prefix tokens, 8 FOP tokens (64-d obs), bf16, batch 1,
                500 steps, context swapped every 4 steps.
``pi_b1``       pi0.5-style expert: 18 layers, width 1024, 8 query heads and 1
                KV head of 256, MLP 4096, H=50, action dim 32, 816 prefix
                tokens (3x256 image-like + 48 text-like), 16 FOP tokens (256-d
                obs), bf16, batch 1, 1000 steps.
``pi_b64``      the same model at batch 64, per-env context refresh every 5
                steps (staggered), 1000 steps.
``large_b16``   24 layers, width 2048, 16 query / 4 KV heads of 128, MLP 8192,
                H=100, action dim 32, 2048 prefix tokens, 32 FOP tokens (512-d
                obs), bf16, batch 16, 500 steps, context swap every 3 steps.

Weights are N(0, 0.02) (biases, the adapter norm scale and the adapter gate
included), rounded to bf16 with round-to-nearest-even for the bf16 workloads.
Prefix K/V and observation vectors are N(0, 1).
"""

from __future__ import annotations

import dataclasses
import zlib
from typing import Dict, List, Tuple

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

F32 = 0
BF16 = 1

TRANSFORMER = 0
ANALYTIC_OT = 1
ANALYTIC_LINEAR = 2

# how the context-age offset enters the expert: an MLP of it added to the
# flow-time embedding, concatenated to every slot's action input, or (the
# DynamicVLA way) concatenated before the action-time MLP plus a gated residual
# adapter conditioned on its sinusoidal embedding
OFFSET_MLP = 0
OFFSET_CONCAT = 1
OFFSET_ADAPTER = 2


@dataclasses.dataclass(frozen=True)
class RavelShape:
    """Static shape of one action expert plus its rolling buffer."""

    layers: int
    width: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    mlp_dim: int
    horizon: int  # H: number of buffer slots
    action_dim: int
    prefix_len: int  # P: prefix (VLM context) tokens per layer
    n_fop: int  # FOP tokens per env
    fop_obs_dim: int
    fop_stride: int = 2  # adapter in layers l with l % stride == stride - 1
    dtype: int = BF16
    model_kind: int = TRANSFORMER
    delta_bias: float = 0.0
    rms_eps: float = 1e-6
    offset_mode: int = OFFSET_MLP
    # rotary position embedding of the buffer tokens' self-attention queries and
    # keys at positions P + i (0: none)
    rope_base: float = 0.0
    # workload (not model) fields
    batch: int = 1
    steps: int = 200
    context_period: int = 0  # 0: one context at t=0 only
    stagger: bool = False  # per-env refresh phase (s + e) % period == 0
    name: str = "custom"

    def replace(self, **kw) -> "RavelShape":
        return dataclasses.replace(self, **kw)

    @property
    def qkv_dim(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    def adapter_layers(self) -> List[int]:
        if self.fop_stride <= 0 or self.n_fop <= 0:
            return []
        s = self.fop_stride
        return [l for l in range(self.layers) if l % s == s - 1]

    def adapter_rank(self) -> int:
        """Bottleneck width of the offset adapter (OFFSET_ADAPTER): a quarter of the width."""
        return self.width // 4


CONFIGS: Dict[str, RavelShape] = {
    "tiny_fp32": RavelShape(
        layers=2, width=128, n_q_heads=4, n_kv_heads=4, head_dim=32, mlp_dim=512,
        horizon=8, action_dim=7, prefix_len=32, n_fop=4, fop_obs_dim=32,
        dtype=F32, batch=1, steps=200, context_period=0, name="tiny_fp32"),
    "small_bf16": RavelShape(
        layers=6, width=512, n_q_heads=8, n_kv_heads=8, head_dim=64, mlp_dim=2048,
        horizon=16, action_dim=14, prefix_len=256, n_fop=8, fop_obs_dim=64,
        dtype=BF16, batch=1, steps=500, context_period=4, name="small_bf16"),
    "pi_b1": RavelShape(
        layers=18, width=1024, n_q_heads=8, n_kv_heads=1, head_dim=256, mlp_dim=4096,
        horizon=50, action_dim=32, prefix_len=816, n_fop=16, fop_obs_dim=256,
        dtype=BF16, batch=1, steps=1000, context_period=0, name="pi_b1"),
    "pi_b64": RavelShape(
        layers=18, width=1024, n_q_heads=8, n_kv_heads=1, head_dim=256, mlp_dim=4096,
        horizon=50, action_dim=32, prefix_len=816, n_fop=16, fop_obs_dim=256,
        dtype=BF16, batch=64, steps=1000, context_period=5, stagger=True, name="pi_b64"),
    "large_b16": RavelShape(
        layers=24, width=2048, n_q_heads=16, n_kv_heads=4, head_dim=128, mlp_dim=8192,
        horizon=100, action_dim=32, prefix_len=2048, n_fop=32, fop_obs_dim=512,
        dtype=BF16, batch=16, steps=500, context_period=3, name="large_b16"),
}


def get_config(name: str) -> RavelShape:
    return CONFIGS[name]


def weight_shapes(s: RavelShape, with_fop_encoder: bool = True) -> List[Tuple[str, Tuple[int, ...]]]:
    """(name, shape) of every parameter, row-major [out, in] for linears."""
    w, da = s.width, s.action_dim
    if s.model_kind == ANALYTIC_OT:
        return [("analytic.target", (da,))]
    if s.model_kind == ANALYTIC_LINEAR:
        return [("analytic.lambda", (1,))]
    concat = s.offset_mode == OFFSET_CONCAT
    out: List[Tuple[str, Tuple[int, ...]]] = [
        ("in.w", (w, da + 1 if concat else da)), ("in.b", (w,)),
        ("time.w1", (w, w)), ("time.b1", (w,)),
        ("time.w2", (w, w)), ("time.b2", (w,)),
    ]
    if s.offset_mode == OFFSET_MLP:
        out += [("delta.w1", (w, 1)), ("delta.b1", (w,)), ("delta.w2", (w, w)), ("delta.b2", (w,))]
    if s.offset_mode == OFFSET_ADAPTER:
        r = s.adapter_rank()
        out += [("at.w1", (w, 2 * w + 1)), ("at.b1", (w,)), ("at.w2", (w, w)), ("at.b2", (w,)),
                ("ta.w1", (r, 2 * w)), ("ta.b1", (r,)), ("ta.w2", (w, r)), ("ta.alpha", (1,))]
    qd = s.n_q_heads * s.head_dim
    kvd = s.n_kv_heads * s.head_dim
    adapters = set(s.adapter_layers())
    for l in range(s.layers):
        p = f"layers.{l}."
        out += [
            (p + "mod.w", (6 * w, w)), (p + "mod.b", (6 * w,)),
            (p + "qkv.w", (qd + 2 * kvd, w)),
            (p + "o.w", (w, qd)),
            (p + "gate.w", (s.mlp_dim, w)), (p + "up.w", (s.mlp_dim, w)),
            (p + "down.w", (w, s.mlp_dim)),
        ]
        if l in adapters:
            out += [
                (p + "fop.gamma", (w,)),
                (p + "fop.q.w", (qd, w)),
                (p + "fop.kv.w", (2 * kvd, w)),
                (p + "fop.o.w", (w, qd)),
                (p + "fop.alpha", (1,)),
            ]
    out += [("final.mod.w", (3 * w, w)), ("final.mod.b", (3 * w,)),
            ("out.w", (da, w)), ("out.b", (da,))]
    if with_fop_encoder and s.n_fop > 0:
        out += [("fop.w1", (w, s.fop_obs_dim)), ("fop.b1", (w,)),
                ("fop.w2", (s.n_fop * w, w)), ("fop.b2", (s.n_fop * w,))]
    return out


def param_count(s: RavelShape, with_fop: bool) -> int:
    """Number of scalars in the expert (with or without FOP adapters/encoder)."""
    n = 0
    for name, shp in weight_shapes(s, with_fop_encoder=with_fop):
        if not with_fop and ".fop." in name:
            continue
        n += int(np.prod(shp))
    return n


def _rng(seed: int, *tags) -> np.random.Generator:
    key = tuple(zlib.crc32(t.encode()) if isinstance(t, str) else int(t) for t in tags)
    return np.random.default_rng(np.random.SeedSequence(entropy=int(seed), spawn_key=key))


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    r = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    out = ((u + r) & np.uint32(0xFFFF0000)).view(np.float32)
    return out


def _bf16_round_inplace(a: np.ndarray, chunk: int = 1 << 22) -> None:
    """bf16_round on a float32 array in place, a chunk at a time (no full-size temporaries)."""
    u = a.reshape(-1).view(np.uint32)
    for i in range(0, u.size, chunk):
        c = u[i:i + chunk]
        r = ((c >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
        c += r
        c &= np.uint32(0xFFFF0000)


def _draw_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    a = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return a


def draw_weights(s: RavelShape, seed: int = 0, stress: bool = False,
                 with_fop_encoder: bool = True, analytic_target_std: float = 1.0,
                 analytic_lambda: float = 0.5) -> Dict[str, np.ndarray]:
    """Draw every parameter as float32 (bf16-valued for bf16 workloads).

    ``stress``: N(0, 1/sqrt(fan_in)) weights, adapter gate alpha = 1 and +1 on
    the bias of both residual gates, so every sub-block moves the output well
    above the bf16 tolerance.
    """
    out: Dict[str, np.ndarray] = {}
    if s.model_kind == ANALYTIC_OT:
        out["analytic.target"] = _normal(_rng(seed, "analytic.target"), (s.action_dim,), analytic_target_std)
        return out
    if s.model_kind == ANALYTIC_LINEAR:
        out["analytic.lambda"] = np.array([analytic_lambda], dtype=np.float32)
        return out
    w = s.width

    def draw(item):
        name, shp = item
        std = 0.02
        if stress and len(shp) == 2:
            std = 1.0 / np.sqrt(shp[1])
        a = _normal(_rng(seed, name), shp, std)
        if stress:
            if name.endswith("alpha"):
                a[:] = 1.0
            if name.endswith(".mod.b") and not name.startswith("final"):
                a[2 * w:3 * w] += 1.0
                a[5 * w:6 * w] += 1.0
        if s.dtype == BF16:
            _bf16_round_inplace(a)
        return name, a

    # every tensor has its own seeded stream, so drawing them on several threads
    # (numpy's generators release the GIL) gives the same values in any order
    items = weight_shapes(s, with_fop_encoder)
    with ThreadPoolExecutor(max_workers=_draw_threads()) as ex:
        for name, a in ex.map(draw, items):
            out[name] = a
    return out


def draw_context(s: RavelShape, seed: int, env: int, refresh: int) -> Tuple[np.ndarray, np.ndarray]:
    """Prefix K and V for one env and one refresh: each [L, P, n_kv, hd], N(0,1)."""
    shp = (s.layers, s.prefix_len, s.n_kv_heads, s.head_dim)
    k = _normal(_rng(seed, "ctx.k", env, refresh), shp, 1.0)
    v = _normal(_rng(seed, "ctx.v", env, refresh), shp, 1.0)
    if s.dtype == BF16:
        k, v = bf16_round(k), bf16_round(v)
    return k, v


def draw_observation(s: RavelShape, seed: int, step: int, batch: int | None = None) -> np.ndarray:
    """FOP observation vectors [B, d_obs], N(0,1), one draw per control step."""
    b = s.batch if batch is None else batch
    return _normal(_rng(seed, "obs", step), (b, s.fop_obs_dim), 1.0)


def draw_fop_tokens(s: RavelShape, seed: int, step: int, scale: float = 1.0,
                    batch: int | None = None) -> np.ndarray:
    """Stand-in FOP tokens [B, n_fop, w] drawn directly (model-dtype valued)."""
    b = s.batch if batch is None else batch
    z = _normal(_rng(seed, "fop_tokens", step), (b, s.n_fop, s.width), scale)
    if s.dtype == BF16:
        z = bf16_round(z)
    return z


def context_schedule(s: RavelShape, steps: int | None = None):
    """(step, env, t_obs, refresh) publishes of the workload's refresh policy.

    Initial context: every env publishes refresh 0 with t_obs = 0 before step 0.
    A later refresh published before step ``st`` carries t_obs = st - period
    (the VLM latency equals the refresh period).
    """
    n = s.steps if steps is None else steps
    ev = [(0, e, 0, 0) for e in range(s.batch)]
    if s.context_period > 0:
        per = s.context_period
        cnt = [0] * s.batch
        for st in range(1, n):
            for e in range(s.batch):
                phase = (st + e) if s.stagger else st
                if phase % per == 0 and st - per >= 0:
                    cnt[e] += 1
                    ev.append((st, e, st - per, cnt[e]))
    return ev
