"""Rolling flow denoising with asynchronous context reuse -- plain CPU definition.

Follows Sec. 3.1 (Eq. 1 and Eq. 3, and the release/append rule stated right
after Eq. 3), Sec. 3.2 (latest-available context reused across steps) and the
cold-start rule of App. A.1 (no extra initialisation: the first action gets a
single update, later ones progressively more, K in steady state).

Time convention (the paper's mirror image, identical trajectories): logical
slot i = 0 .. H-1 holds the action executed i+1 control steps from now at flow
time tau_i = (i+1)/H (tau = 1 is pure noise), and one expert pass moves every
slot by dt = 1/H towards 0: a_i <- a_i - dt * v_i.  In the paper's notation
(tau' = 1 - tau, v' = -v, K = H) this is exactly Eq. 3.

State per environment e: a ring X[e] of H action vectors (physical slot
(t + i) mod H holds logical slot i at step t), the step counter t shared by
all environments, and the active context (prefix K/V and the observation step
t_obs it was computed from).  One call of ``step``:

1. applies contexts published since the previous step (newest wins);
2. per env: p = t - t_obs, delta = p / H + delta_0 (Sec. 3.1 after Eq. 2;
   delta_0 is the lead bias of Sec. 4.4 / App. B.1);
3. per env: v = v_theta(logical slots, tau, context, delta, FOP tokens);
4. Euler update of every slot (Eq. 3);
5. releases logical slot 0 (now clean) as the action for this step and puts
   fresh noise for action index r = t + H into its physical slot;
6. t <- t + 1.

Relative actions (App. B.1 for pi0.5 on RoboTwin 2.0, App. B.3 for DynamicVLA): a
model that predicts actions relative to the robot state cannot reuse its buffer
as the state moves.  The paper keeps the clean targets absolute, converts them
relative to the latest state before each expert pass and back afterwards, and
leaves the paired noise in model coordinates.  Written on the buffer of noisy
actions (slot i = tau_i eps_i + (1 - tau_i) a_rel_i), re-expressing the clean
part against a new state s moves every slot by (1 - tau_i) (s_prev - s) on the
relative dimensions, where s_prev is the state the buffer was last expressed
against -- the same for every slot, since every slot is re-expressed each step
(a slot appended at tau = 1 carries no clean part).  With relative dimensions
set, ``step`` takes the state [B, D_a]: it shifts the buffer by
(1 - tau_i)(s_prev - s) (no shift at an env's first step: the cold-start noise is
taken relative to the first state), runs the ordinary update, and releases the
absolute action a_0 + s.  Readings: the state comes in the actions' normalised
units; dimensions outside the mask (e.g. a gripper command) stay absolute; for
the analytic OT field the target a* is absolute, so the field aims at
a* - s on the relative dimensions.

This is test infrastructure: only the tests, the smoke check and the bench's
CPU-baseline leg may import it.
"""

from __future__ import annotations

import numpy as np

from .expert import Expert
from .philox import ring_noise

TRANSFORMER = 0
ANALYTIC_OT = 1
ANALYTIC_LINEAR = 2


class OracleRavel:
    def __init__(self, shape, weights: dict, batch: int, seed: int, dtype=np.float64, env_ids=None):
        """env_ids: environment index of each row for its noise stream (default
        0..batch-1); lets a few sampled environments of a large batch be rolled."""
        self.s = shape
        self.env_ids = list(range(batch)) if env_ids is None else [int(e) for e in env_ids]
        assert len(self.env_ids) == batch
        self.B = batch
        self.seed = int(seed)
        self.dt = dtype
        self.H = shape.horizon
        self.kind = shape.model_kind
        if self.kind == TRANSFORMER:
            self.expert = Expert(shape, weights, dtype)
        else:
            self.params = {k: np.asarray(v, dtype=dtype) for k, v in weights.items()}
        H, D = self.H, shape.action_dim
        # Cold start: every slot holds pure noise; initial actions r = 0..H-1
        # sit at physical slot r mod H (App. A.1: no extra initialisation).
        self.X = np.zeros((batch, H, D), dtype=dtype)
        for e in range(batch):
            for r in range(H):
                self.X[e, r % H] = ring_noise(self.seed, self.env_ids[e], r, D)
        self.t = 0
        self.ctx = [None] * batch  # (K, V) per env
        self.t_obs = np.zeros(batch, dtype=np.int64)
        self.has_ctx = np.zeros(batch, dtype=bool)
        self.pending = {}
        self.log = []  # (env, t_apply, t_obs)
        self.rel = None  # [D_a] 1.0 on relative dimensions (None: absolute actions)
        self.s_prev = np.zeros((batch, D), dtype=dtype)
        self.has_prev = np.zeros(batch, dtype=bool)
        self.state = None

    def set_relative_dims(self, mask):
        """Mark the relative action dimensions (before the first step)."""
        assert self.t == 0
        self.rel = np.asarray(mask, dtype=self.dt)

    # -- context plane (Sec. 3.2) ----------------------------------------
    def set_context(self, env: int, k, v, t_obs: int):
        """Publish a context; it becomes active at the start of the next step."""
        if self.has_ctx[env] and t_obs < self.t_obs[env]:
            raise ValueError("t_obs must not decrease per env")
        self.pending[env] = (k, v, int(t_obs))

    def _apply_pending(self):
        for env in sorted(self.pending):
            k, v, t_obs = self.pending[env]
            self.ctx[env] = (k, v)
            self.t_obs[env] = t_obs
            self.has_ctx[env] = True
            self.log.append((env, self.t, t_obs))
        self.pending = {}

    # -- velocity ----------------------------------------------------------
    def _taus(self):
        H = self.H
        return (np.arange(H, dtype=self.dt) + self.dt(1)) / self.dt(H)

    def offset(self, env: int) -> float:
        """delta = p / H + delta_0 with p = t - t_obs (context age in control steps)."""
        p = self.t - int(self.t_obs[env])
        return p / self.H + self.s.delta_bias

    def velocity(self, env: int, a_logical, z=None, hooks=None):
        if self.kind == ANALYTIC_OT:
            # Conditional OT field towards a fixed target a*: v = (x - a*) / tau (a* absolute:
            # relative to the current state on relative dimensions).
            target = self.params["analytic.target"]
            if self.rel is not None:
                target = target - self.rel * self.state[env]
            return (a_logical - target[None, :]) / self._taus()[:, None]
        if self.kind == ANALYTIC_LINEAR:
            return self.params["analytic.lambda"][0] * a_logical
        k, v = self.ctx[env]
        zz = None if z is None else z[env]
        return self.expert.velocity(a_logical, k, v, self.offset(env), zz, hooks)

    # -- one control step ----------------------------------------------------
    def step(self, fop_tokens=None, hooks=None, state=None):
        """Advance every env by one control step; returns released actions [B, D_a].
        With relative dimensions, state [B, D_a] is the latest robot state."""
        self._apply_pending()
        H, t = self.H, self.t
        if self.kind == TRANSFORMER and not self.has_ctx.all():
            raise RuntimeError("every env needs a context before its first step")
        if (self.rel is None) != (state is None):
            raise ValueError("a state is given exactly when relative dimensions are set")
        dtau = self.dt(1) / self.dt(H)
        phys = (t + np.arange(H)) % H
        out = np.empty((self.B, self.s.action_dim), dtype=self.dt)
        if state is not None:
            self.state = np.asarray(state, dtype=self.dt)
            for e in range(self.B):
                if self.has_prev[e]:
                    # re-express every slot's clean part against the new state
                    shift = self.rel * (self.s_prev[e] - self.state[e])
                    self.X[e, phys] = self.X[e, phys] + (self.dt(1) - self._taus())[:, None] * shift[None, :]
                self.s_prev[e] = self.state[e]
                self.has_prev[e] = True
        for e in range(self.B):
            a = self.X[e, phys]
            vel = np.asarray(self.velocity(e, a, fop_tokens, hooks), dtype=self.dt)
            self.X[e, phys] = a - dtau * vel
            out[e] = self.X[e, t % H]
            if state is not None:
                out[e] = out[e] + self.rel * self.state[e]
            self.X[e, t % H] = ring_noise(self.seed, self.env_ids[e], t + H, self.s.action_dim)
        self.t += 1
        return out

    def logical_state(self):
        """Ring contents in logical order at the current t: [B, H, D_a]."""
        phys = (self.t + np.arange(self.H)) % self.H
        return self.X[:, phys].copy()
