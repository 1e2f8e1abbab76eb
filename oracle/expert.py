"""The flow-matching action expert v_theta(A, tau, c, delta) -- plain CPU definition.

Sec. 3.1, Eq. 3 defines one pass of the expert over the whole rolling buffer:
it returns one velocity per slot, conditioned on every slot's own flow time
tau_k, the VLM context c (layer-wise prefix key/value caches, Sec. 3.1 after
Eq. 1 and Eq. 2) and the temporal offset delta_p = p / K.  App. A.1 fixes how
delta enters the pi0.5-style expert: an MLP of delta is added to the flow-time
embedding, all slots share delta and keep their own tau.  Sec. 3.2 (Eq. 4)
adds FOP tokens through gated cross-attention adapters in selected layers.

The paper does not print the expert's layer equations.  The readings taken
here (fixed for the whole repository) are:

* conditioning: cond_i = silu(c_tau(i) + d), with
  c_tau(i) = W_t2 silu(W_t1 emb(tau_i) + b_t1) + b_t2 and
  d = W_d2 silu(W_d1 delta + b_d1) + b_d2 (the delta MLP added to the time
  embedding before the shared final silu); or, for the X-VLA way of App. A.1
  (offset_mode 1: delta concatenated to the noisy action at the action
  encoder, every slot the same delta), cond_i = silu(c_tau(i)) and the input
  projection takes [a_i ; delta]; or, for the DynamicVLA way of App. A.1
  (offset_mode 2), cond_i = silu(c_tau(i)) and the action encoder becomes
  e_i = W_in a_i + b_in, g_i = W_a2 silu(W_a1 [e_i ; emb(tau_i) ; delta] + b_a1)
  + b_a2 (the action-time MLP with delta concatenated to the action and
  flow-time embeddings), then a gated residual adapter conditioned on the
  offset's sinusoidal embedding: h_i = g_i + tanh(beta) W_r2 silu(W_r1 [g_i ;
  emb(delta)] + b_r1), with a bottleneck of w/4 and emb the same sinusoid as
  the flow time's;
* emb(tau) = [sin(1000 tau w_j), cos(1000 tau w_j)], w_j = 10000^(-j/(w/2)),
  j < w/2;
* every block: adaptive RMSNorm whose scale/shift/gate come from
  Linear(cond) per token (six chunks per layer, three for the final norm of
  which the third is unused); residual updates are gated x += g * f(.);
* attention: bidirectional over [prefix tokens ; buffer tokens], no mask, no
  positional encoding (optionally a rotary one on the buffer tokens, see
  rope_rotate), grouped-query heads (query head j uses KV head
  floor(j * n_kv / n_q)), scale 1/sqrt(hd), no biases on attention/MLP linears;
* MLP: gated GeLU (tanh form), down(gelu_tanh(gate y) * up y);
* FOP adapter in layers l with l % stride == stride - 1: rms(x) (1 + gamma) ->
  queries, FOP tokens -> keys/values (no norm), attention over FOP tokens only,
  x += tanh(alpha) * W_oa o;
* output head: v_i = W_out (rms(h) (1 + s_f) + b_f) + b_out;
* RMSNorm: x / sqrt(mean(x^2) + eps).

With these readings the pi-style workload without FOP has exactly the
431,150,112 trainable parameters the paper reports for its pi0.5 action
expert (App. B.1, table of training configurations: 431.15M).

This is test infrastructure: only the tests, the smoke check and the bench's
CPU-baseline leg may import it.
"""

from __future__ import annotations

import numpy as np


def silu(x):
    return x / (1.0 + np.exp(-x))


def gelu_tanh(x):
    c = np.sqrt(2.0 / np.pi)
    return 0.5 * x * (1.0 + np.tanh(c * (x + 0.044715 * x ** 3)))


def rms_normalize(x, eps):
    """x / sqrt(mean over the last axis of x^2 + eps)."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def flow_times(H: int) -> np.ndarray:
    """tau_i = (i + 1) / H for logical slot i = 0 .. H-1 (1 = pure noise, 0 = clean).

    This is the paper's profile tau_k = 1 - k/K (Sec. 3.1, after Eq. 1) written
    with the opposite time direction: tau_here = 1 - tau_paper and slot i = k - 1
    counts from the next action to execute.
    """
    return (np.arange(H, dtype=np.float64) + 1.0) / H


def time_embedding(tau, width: int) -> np.ndarray:
    """Sinusoidal embedding [len(tau), width], float64."""
    half = width // 2
    j = np.arange(half, dtype=np.float64)
    omega = 10000.0 ** (-j / half)
    arg = 1000.0 * np.asarray(tau, dtype=np.float64)[:, None] * omega[None, :]
    return np.concatenate([np.sin(arg), np.cos(arg)], axis=1)


def rope_rotate(x, pos, n_heads: int, hd: int, base: float):
    """Rotary position embedding, rotate-half pairing: in every head, the pair
    (x_d, x_{d + hd/2}), d < hd/2, turns by the angle pos * base^(-2d/hd).

    x: [T, n_heads * hd]; pos: [T] positions.  The paper uses no positional
    encoding of the buffer tokens; this optional variant places logical slot i at
    position P + i, after the P prefix tokens, whose cached keys are taken as
    already encoded by the VLM and are used as given.
    """
    half = hd // 2
    theta = np.asarray(base, dtype=np.float64) ** (-2.0 * np.arange(half, dtype=np.float64) / hd)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * theta[None, :]
    c, s_ = np.cos(ang).astype(x.dtype), np.sin(ang).astype(x.dtype)
    out = np.empty_like(x)
    for j in range(n_heads):
        a = x[:, j * hd:j * hd + half]
        b = x[:, j * hd + half:(j + 1) * hd]
        out[:, j * hd:j * hd + half] = a * c - b * s_
        out[:, j * hd + half:(j + 1) * hd] = b * c + a * s_
    return out


def linear(x, w, b=None):
    """y = x W^T + b, W [out, in].  The product is formed as (W x^T)^T: the same
    numbers, and for few rows of x the library matmul runs it several times faster."""
    y = (w @ x.T).T
    if b is not None:
        y = y + b
    return y


def attention(q, k, v, n_q: int, n_kv: int, hd: int):
    """Grouped-query softmax attention without a mask.

    q: [Tq, n_q*hd]; k, v: [Tk, n_kv*hd]. Returns [Tq, n_q*hd].
    """
    out = np.empty_like(q)
    scale = 1.0 / np.sqrt(hd)
    for j in range(n_q):
        g = (j * n_kv) // n_q
        qj = q[:, j * hd:(j + 1) * hd]
        kg = k[:, g * hd:(g + 1) * hd]
        vg = v[:, g * hd:(g + 1) * hd]
        s = (qj @ kg.T) * scale
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, j * hd:(j + 1) * hd] = p @ vg
    return out


class Expert:
    """Weights of one expert, cast once to the oracle's working precision."""

    def __init__(self, shape, weights: dict, dtype=np.float64):
        self.s = shape
        self.dt = dtype
        self.W = {k: np.asarray(v, dtype=dtype) for k, v in weights.items()}
        self._ctau = None

    # -- conditioning -----------------------------------------------------
    def tau_conditioning(self, taus=None) -> np.ndarray:
        """c_tau for every slot: [H, w].  Default: the rolling buffer's fixed
        profile tau_i = (i+1)/H; otherwise the given flow time of each slot."""
        W = self.W

        def ctau(t):
            emb = time_embedding(t, self.s.width).astype(self.dt)
            h = silu(linear(emb, W["time.w1"], W["time.b1"]))
            return linear(h, W["time.w2"], W["time.b2"])

        if taus is not None:
            return ctau(np.asarray(taus, dtype=np.float64))
        if self._ctau is None:
            self._ctau = ctau(flow_times(self.s.horizon))
        return self._ctau

    def delta_conditioning(self, delta: float) -> np.ndarray:
        """d = W_d2 silu(W_d1 delta + b_d1) + b_d2: [w]."""
        W = self.W
        dl = np.asarray([delta], dtype=self.dt)
        h = silu(W["delta.w1"][:, 0] * dl[0] + W["delta.b1"])
        return W["delta.w2"] @ h + W["delta.b2"]

    def concat_offset(self) -> bool:
        return getattr(self.s, "offset_mode", 0) == 1

    def adapter_offset(self) -> bool:
        return getattr(self.s, "offset_mode", 0) == 2

    def conditioning(self, delta: float, taus=None) -> np.ndarray:
        if self.concat_offset() or self.adapter_offset():  # the offset enters at the action encoder
            return silu(self.tau_conditioning(taus))
        return silu(self.tau_conditioning(taus) + self.delta_conditioning(delta)[None, :])

    def encode_actions(self, a, delta: float, taus=None) -> np.ndarray:
        """Action encoder: h_i = W_in a_i + b_in; with the offset concatenated (the X-VLA
        expert, App. A.1), h_i = W_in [a_i ; delta] + b_in for every slot i; in the
        DynamicVLA form (App. A.1) the action-time MLP over [e_i ; emb(tau_i) ; delta]
        followed by the offset-conditioned gated residual adapter."""
        W = self.W
        if self.concat_offset():
            a = np.concatenate([a, np.full((a.shape[0], 1), delta, dtype=a.dtype)], axis=1)
        h = linear(a, W["in.w"], W["in.b"])
        if not self.adapter_offset():
            return h
        n = h.shape[0]
        t = flow_times(self.s.horizon) if taus is None else np.asarray(taus, dtype=np.float64)
        # action-time MLP: action embedding, flow-time embedding and the offset side by side
        z = np.concatenate([h, time_embedding(t, self.s.width).astype(self.dt),
                            np.full((n, 1), delta, dtype=self.dt)], axis=1)
        g = linear(silu(linear(z, W["at.w1"], W["at.b1"])), W["at.w2"], W["at.b2"])
        # gated residual adapter on the action tokens, conditioned on emb(delta)
        ed = np.repeat(time_embedding([delta], self.s.width).astype(self.dt), n, axis=0)
        r = silu(linear(np.concatenate([g, ed], axis=1), W["ta.w1"], W["ta.b1"]))
        return g + np.tanh(W["ta.alpha"][0]) * linear(r, W["ta.w2"])

    # -- one pass ---------------------------------------------------------
    def velocity(self, a_slots, ctx_k, ctx_v, delta: float, z=None, hooks=None, taus=None,
                 pos0=None) -> np.ndarray:
        """Velocity of every slot.

        a_slots: [H, D_a] noisy actions in logical order (slot i has tau_i, the
        rolling profile, unless taus gives each slot's flow time).
        ctx_k, ctx_v: [L, P, n_kv, hd] prefix caches of the active context.
        z: [n_fop, w] FOP tokens (ignored when the expert has no adapters).
        hooks: optional set of sub-block names to switch off ("attn",
        "adapter", "mlp", "delta") for sensitivity checks.
        pos0: rotary position of slot 0 (default P, the prefix length).
        """
        s, W, dt = self.s, self.W, self.dt
        hooks = hooks or set()
        w, nq, nkv, hd = s.width, s.n_q_heads, s.n_kv_heads, s.head_dim
        qd, kvd = nq * hd, nkv * hd
        eps = s.rms_eps
        a = np.asarray(a_slots, dtype=dt)
        d_eff = 0.0 if "delta" in hooks else delta
        cond = self.conditioning(d_eff, taus)
        h = self.encode_actions(a, d_eff, taus)
        adapters = set(s.adapter_layers())
        for l in range(s.layers):
            p = f"layers.{l}."
            mod = linear(cond, W[p + "mod.w"], W[p + "mod.b"])
            s1, b1, g1, s2, b2, g2 = np.split(mod, 6, axis=1)
            # self-attention block over [prefix ; buffer]
            y = rms_normalize(h, eps) * (1.0 + s1) + b1
            qkv = linear(y, W[p + "qkv.w"])
            q, k, v = qkv[:, :qd], qkv[:, qd:qd + kvd], qkv[:, qd + kvd:]
            P = ctx_k.shape[1] if ctx_k is not None else 0
            if getattr(s, "rope_base", 0.0):
                pos = (P if pos0 is None else pos0) + np.arange(a.shape[0])
                q = rope_rotate(q, pos, nq, hd, s.rope_base)
                k = rope_rotate(k, pos, nkv, hd, s.rope_base)
            if P:
                kp = np.asarray(ctx_k[l], dtype=dt).reshape(P, kvd)
                vp = np.asarray(ctx_v[l], dtype=dt).reshape(P, kvd)
                kk, vv = np.concatenate([kp, k]), np.concatenate([vp, v])
            else:
                kk, vv = k, v
            o = attention(q, kk, vv, nq, nkv, hd)
            if "attn" not in hooks:
                h = h + g1 * linear(o, W[p + "o.w"])
            # FOP gated cross-attention adapter
            if l in adapters and z is not None and "adapter" not in hooks:
                ya = rms_normalize(h, eps) * (1.0 + W[p + "fop.gamma"])
                qa = linear(ya, W[p + "fop.q.w"])
                kva = linear(np.asarray(z, dtype=dt), W[p + "fop.kv.w"])
                oa = attention(qa, kva[:, :kvd], kva[:, kvd:], nq, nkv, hd)
                h = h + np.tanh(W[p + "fop.alpha"][0]) * linear(oa, W[p + "fop.o.w"])
            # gated-GeLU MLP block
            y2 = rms_normalize(h, eps) * (1.0 + s2) + b2
            u = gelu_tanh(linear(y2, W[p + "gate.w"])) * linear(y2, W[p + "up.w"])
            if "mlp" not in hooks:
                h = h + g2 * linear(u, W[p + "down.w"])
        fm = linear(cond, W["final.mod.w"], W["final.mod.b"])
        sf, bf = fm[:, :w], fm[:, w:2 * w]
        return linear(rms_normalize(h, eps) * (1.0 + sf) + bf, W["out.w"], W["out.b"])


def fop_encode(shape, weights: dict, obs, dtype=np.float64) -> np.ndarray:
    """FOP stand-in encoder z = F(o): [B, d_obs] -> [B, n_fop, w] (Sec. 3.2, Eq. 4).

    The paper's encoder (a ConvNeXt image encoder plus state projection) is
    replaced by a 2-layer MLP of an observation vector:
    z = reshape(W_f2 gelu_tanh(W_f1 obs + b_f1) + b_f2, [n_fop, w]).
    """
    W = {k: np.asarray(weights[k], dtype=dtype) for k in ("fop.w1", "fop.b1", "fop.w2", "fop.b2")}
    o = np.asarray(obs, dtype=dtype)
    h = gelu_tanh(linear(o, W["fop.w1"], W["fop.b1"]))
    z = linear(h, W["fop.w2"], W["fop.b2"])
    return z.reshape(o.shape[0], shape.n_fop, shape.width)
