"""Shared drivers for the GPU parity tests: roll the HIP library and the CPU
oracle on the same seeded inputs and compare.

Error measure (per compared tensor): max|gpu - ref| / max|ref| (normwise
infinity), applied to every released action batch [B, D_a] and to the whole
ring state [B, H, D_a] at checkpoints.
"""

from __future__ import annotations

import numpy as np

import synth
from oracle.rolling import OracleRavel

TOL_F32 = 1e-4
TOL_BF16 = 2e-2


def have_gpu() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def rel_err(g, r) -> float:
    g = np.asarray(g, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    den = np.abs(r).max()
    return float(np.abs(g - r).max() / max(den, 1e-30))


def logical(X, t):
    """Physical ring [B, H, D] -> logical order at step t."""
    H = X.shape[1]
    return X[:, (t + np.arange(H)) % H]


class GpuRoll:
    """Drives libravel through the binding with torch-owned device memory."""

    def __init__(self, shape, weights, batch, seed, sync_context=True, use_graph=True):
        import torch

        from paper_2609_34170_amd import ravel
        self.torch = torch
        self.rv = ravel
        self.s = shape
        self.B = batch
        self.model = ravel.Model(shape, weights)
        self.buf = ravel.Buffer(self.model, batch, seed)
        self.buf.set_option(ravel.OPT_SYNC_CONTEXT, 1 if sync_context else 0)
        self.buf.set_option(ravel.OPT_USE_GRAPH, 1 if use_graph else 0)
        self.dev = torch.device("cuda:0")
        self.tdtype = torch.bfloat16 if shape.dtype == synth.workloads.BF16 else torch.float32
        self.action = torch.zeros((batch, shape.action_dim), dtype=torch.float32, device=self.dev)
        self.fop = None
        if shape.n_fop > 0:
            self.fop = torch.zeros((batch, shape.n_fop, shape.width), dtype=self.tdtype, device=self.dev)
        self._keep = []

    def to_dev(self, a):
        return self.torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(self.dev).to(self.tdtype)

    def set_context(self, env, k, v, t_obs):
        kd, vd = self.to_dev(k), self.to_dev(v)
        self._keep.append((kd, vd))
        self.buf.set_context(env, kd, vd, t_obs)

    def step(self, fop_tokens=None):
        if fop_tokens is not None:
            self.fop.copy_(self.to_dev(fop_tokens))
        self.buf.step(self.fop, self.action)
        out = self.action.cpu().numpy().copy()
        self._keep = self._keep[-4:]
        return out

    def state(self):
        return self.buf.debug_state()


def run_parity(shape, weights, batch, seed, steps, env_sample=None, fop_mode="tokens",
               oracle_dtype=np.float64, check_every=10, tol=None, use_graph=True, ctx_seed=0):
    """Roll both sides `steps` steps; returns (max action error, max state error, n_checked)."""
    if tol is None:
        tol = TOL_F32 if shape.dtype == synth.workloads.F32 else TOL_BF16
    envs = list(range(batch)) if env_sample is None else list(env_sample)
    g = GpuRoll(shape, weights, batch, seed, use_graph=use_graph)
    o = OracleRavel(shape, weights, batch=len(envs), seed=seed, dtype=oracle_dtype, env_ids=envs)
    o_env = {e: i for i, e in enumerate(envs)}
    sched = synth.context_schedule(shape.replace(batch=batch), steps) if shape.model_kind == 0 else []
    ctx_cache = {}
    worst_a = worst_x = 0.0
    n = 0
    for st in range(steps):
        for (s_, e, t_obs, ref) in sched:
            if s_ != st:
                continue
            key = (e, ref)
            if key not in ctx_cache:
                ctx_cache[key] = synth.draw_context(shape, ctx_seed, e, ref)
            k, v = ctx_cache.pop(key)
            g.set_context(e, k, v, t_obs)
            if e in o_env:
                o.set_context(o_env[e], k, v, t_obs)
        z = None
        if shape.n_fop > 0 and shape.model_kind == 0:
            z = synth.draw_fop_tokens(shape, ctx_seed, st, batch=batch)
        ga = g.step(z)
        oa = o.step(None if z is None else z[envs])
        err = rel_err(ga[envs], oa)
        worst_a = max(worst_a, err)
        assert err <= tol, f"step {st}: released-action error {err:.3e} > {tol:.1e}"
        if (st + 1) % check_every == 0 or st == steps - 1:
            X, t, _ = g.state()
            assert t == st + 1
            ex = rel_err(X[envs], o.X)
            worst_x = max(worst_x, ex)
            assert ex <= tol, f"step {st}: ring-state error {ex:.3e} > {tol:.1e}"
        n += 1
    return worst_a, worst_x, n
