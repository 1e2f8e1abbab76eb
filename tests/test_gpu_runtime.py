"""Runtime behaviour of the step on the GPU: hipGraph replay on both execution paths,
a failed launch of the layers' kernel made visible to the control loop, the
non-blocking context plane (Sec. 3.2: the latest available context is reused and a
refresh never blocks a step; Sec. 4.3: separate VLM and action-expert workers), and
publishing every env's context in one call."""

import ctypes
import threading
import time

import numpy as np
import pytest

import synth
from oracle.rolling import OracleRavel
from tests.harness import GpuRoll, have_gpu, rel_err

pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not have_gpu(), reason="needs a GPU")]

W = synth.workloads


def _tiny_bf16(batch=2):
    # B * H = 24 rows: the persistent kernel's path by default
    s = synth.RavelShape(layers=2, width=128, n_q_heads=4, n_kv_heads=2, head_dim=32, mlp_dim=256,
                         horizon=12, action_dim=6, prefix_len=40, n_fop=4, fop_obs_dim=16,
                         dtype=W.BF16, batch=batch, name="rt")
    return s, synth.draw_weights(s, seed=4, stress=True)


def _tiny_fp32(batch=2):
    s = synth.RavelShape(layers=2, width=64, n_q_heads=2, n_kv_heads=1, head_dim=32, mlp_dim=128,
                         horizon=6, action_dim=5, prefix_len=10, n_fop=3, fop_obs_dim=8,
                         dtype=W.F32, batch=batch, name="rt32")
    return s, synth.draw_weights(s, seed=9, stress=True)


def _start(g, s, batch):
    for e in range(batch):
        k, v = synth.draw_context(s, 0, e, 0)
        g.set_context(e, k, v, 0)


def _roll(g, s, steps, t0=0):
    return np.stack([g.step(synth.draw_fop_tokens(s, 0, st, batch=g.B)) for st in range(t0, t0 + steps)])


# ---------------------------------------------------------------------------
# hipGraph replay
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("persistent", [True, False])
def test_graph_replay_equals_eager_bitwise(persistent):
    from paper_2609_34170_amd import ravel
    s, wts = _tiny_bf16()
    rolls = []
    for graph in (True, False):
        g = GpuRoll(s, wts, 2, seed=7, use_graph=graph)
        g.buf.set_option(ravel.OPT_PERSISTENT, 1 if persistent else 0)
        assert g.buf.query(ravel.Q_PERSISTENT) == (1 if persistent else 0)
        _start(g, s, 2)
        rolls.append(_roll(g, s, 30))
        # one graph per pointer set: the harness reuses its FOP and action tensors
        assert g.buf.query(ravel.Q_GRAPHS) == (1 if graph else 0)
        assert g.buf.query(ravel.Q_STEPS) == 30
    assert np.array_equal(rolls[0], rolls[1])


def test_graph_follows_the_execution_path_switch():
    """Switching the execution path between steps captures a second graph and keeps
    the roll on the oracle's track."""
    from paper_2609_34170_amd import ravel
    s, wts = _tiny_bf16()
    g = GpuRoll(s, wts, 2, seed=3)
    _start(g, s, 2)
    o = OracleRavel(s, wts, batch=2, seed=3)
    for e in range(2):
        o.set_context(e, *synth.draw_context(s, 0, e, 0), 0)
    outs_g, outs_o = [], []
    for st in range(12):
        if st == 6:
            g.buf.set_option(ravel.OPT_PERSISTENT, 0)
        z = synth.draw_fop_tokens(s, 0, st, batch=2)
        outs_g.append(g.step(z))
        outs_o.append(o.step(z))
    assert g.buf.query(ravel.Q_GRAPHS) == 2
    assert rel_err(np.stack(outs_g), np.stack(outs_o)) < 2e-2


# ---------------------------------------------------------------------------
# a failed launch of the layers' kernel
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("graph", [True, False])
def test_failed_layers_launch_releases_nan_and_the_next_step_reports_it(graph):
    """The host marks the persistent kernel as failed (its error word set, as a grid
    barrier that timed out sets it; every kernel still runs to its end).  That step
    releases NaN actions and leaves the ring and t alone; the next step call returns
    E_HIP without a sync by the caller; the call after it continues from the unchanged
    state exactly as a buffer that never failed."""
    from paper_2609_34170_amd import ravel
    s, wts = _tiny_bf16()
    ref = GpuRoll(s, wts, 2, seed=5, use_graph=graph)
    _start(ref, s, 2)
    want = _roll(ref, s, 6)

    g = GpuRoll(s, wts, 2, seed=5, use_graph=graph)
    _start(g, s, 2)
    assert np.array_equal(_roll(g, s, 3), want[:3])
    X3, t3, _ = g.state()
    g.buf.set_option(ravel.OPT_FAIL_LAYERS, 1)
    bad = g.step(synth.draw_fop_tokens(s, 0, 3, batch=2))  # enqueued; the release writes NaN
    assert np.isnan(bad).all()
    with pytest.raises(ravel.RavelError, match="E_HIP"):
        g.step(synth.draw_fop_tokens(s, 0, 3, batch=2))
    X, t, _ = g.state()
    assert t == t3 == 3
    assert np.array_equal(X, X3)
    assert g.buf.query(ravel.Q_STEPS) == 3
    assert np.array_equal(_roll(g, s, 3, t0=3), want[3:])


def test_failure_hook_needs_the_persistent_kernel():
    from paper_2609_34170_amd import ravel
    s, wts = _tiny_fp32()
    g = GpuRoll(s, wts, 2, seed=0)
    with pytest.raises(ravel.RavelError, match="E_STATE"):
        g.buf.set_option(ravel.OPT_FAIL_LAYERS, 1)


def test_cooperative_launch_request_is_refused(monkeypatch):
    from paper_2609_34170_amd import ravel
    s, wts = _tiny_bf16()
    monkeypatch.setenv("RAVEL_COOPERATIVE", "1")
    with pytest.raises(ravel.RavelError, match="E_INVALID"):
        GpuRoll(s, wts, 2, seed=0)


# ---------------------------------------------------------------------------
# context plane
# ---------------------------------------------------------------------------
def _hip():
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipStreamWaitValue32.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint,
                                         ctypes.c_uint32]
    hip.hipHostGetDevicePointer.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_void_p, ctypes.c_uint]
    return hip


def _replay(s, wts, log, ctx_of, fops, B, seed, dtype=np.float64):
    """The oracle roll that applies each publish at the step the library logged it."""
    o = OracleRavel(s, wts, batch=B, seed=seed, dtype=dtype)
    outs = []
    for st, z in enumerate(fops):
        for (e, ta, tob) in log:
            if ta == st:
                o.set_context(e, *ctx_of(e, tob), tob)
        outs.append(o.step(z))
    return np.stack(outs)


def test_pending_copy_keeps_the_old_context_until_it_lands():
    """The producer stream is held on a host-set word while two steps run: the copy has
    not landed, so both steps use the old context with a growing age.  Released, the
    copy completes and the publish lands on the first step after it; the roll equals
    the oracle's replay of the publish log."""
    import torch
    s, wts = _tiny_bf16()
    g = GpuRoll(s, wts, 2, seed=0, sync_context=False)
    ctx = {(e, 0): synth.draw_context(s, 0, e, 0) for e in range(2)}
    ctx[(1, 2)] = synth.draw_context(s, 0, 1, 1)
    for e in range(2):
        g.set_context(e, *ctx[(e, 0)], 0)
    g.buf.sync()
    fops = [synth.draw_fop_tokens(s, 0, st, batch=2) for st in range(8)]
    outs = [g.step(fops[st]) for st in range(3)]
    hip = _hip()
    gate = torch.zeros(4, dtype=torch.int32, pin_memory=True)
    dptr = ctypes.c_void_p()
    assert hip.hipHostGetDevicePointer(ctypes.byref(dptr), ctypes.c_void_p(gate.data_ptr()), 0) == 0
    ps = torch.cuda.Stream()
    if hip.hipStreamWaitValue32(ctypes.c_void_p(ps.cuda_stream), dptr, 1, 0x1, 0xFFFFFFFF) != 0:
        pytest.skip("hipStreamWaitValue32 is not supported here")
    try:
        kd, vd = g.to_dev(ctx[(1, 2)][0]), g.to_dev(ctx[(1, 2)][1])
        g.buf.set_context(1, kd, vd, 2, stream=ps)
        n_before = len(g.buf.publish_log())
        outs += [g.step(fops[st]) for st in (3, 4)]
        assert len(g.buf.publish_log()) == n_before  # still pending: old context, p = 3, 4
    finally:
        gate[0] = 1
    ps.synchronize()
    outs += [g.step(fops[st]) for st in range(5, 8)]
    log = g.buf.publish_log()
    assert log[-1] == (1, 5, 2)
    want = _replay(s, wts, log, lambda e, tob: ctx[(e, tob)], fops, 2, seed=0)
    assert rel_err(np.stack(outs), want) < 2e-2


def test_set_context_from_a_second_thread_while_stepping():
    """A VLM worker thread publishes refreshes (t_obs = refresh index, increasing)
    while the control thread steps; afterwards the publish log is consistent and the
    roll equals the oracle's replay of it (fp32 model, 1e-4)."""
    import torch
    s, wts = _tiny_fp32()
    B, steps, n_ref = 2, 80, 30
    g = GpuRoll(s, wts, B, seed=1, sync_context=False)
    ctx = {(e, r): synth.draw_context(s, 0, e, r) for e in range(B) for r in range(n_ref + 1)}
    dev = {key: (g.to_dev(k), g.to_dev(v)) for key, (k, v) in ctx.items()}
    for e in range(B):
        g.buf.set_context(e, *dev[(e, 0)], 0)
    g.buf.sync()
    errors = []

    def worker():
        try:
            ps = torch.cuda.Stream()
            for r in range(1, n_ref + 1):
                e = r % B
                g.buf.set_context(e, *dev[(e, r)], r, stream=ps)
                time.sleep(0.002)
            ps.synchronize()
        except Exception as exc:  # reported by the main thread
            errors.append(exc)

    fops = [synth.draw_fop_tokens(s, 0, st, batch=B) for st in range(steps)]
    th = threading.Thread(target=worker)
    th.start()
    outs = []
    for st in range(steps):
        outs.append(g.step(fops[st]))
        if st == steps - 3:
            th.join()
        time.sleep(0.001)
    assert not errors, errors
    log = g.buf.publish_log()
    for e in range(B):
        tobs = [tob for (ee, _, tob) in log if ee == e]
        assert tobs == sorted(tobs) and len(set(tobs)) == len(tobs)
        assert tobs[-1] == max(r for r in range(n_ref + 1) if r % B == e or r == 0)
    assert all(0 <= ta < steps for (_, ta, _) in log)
    want = _replay(s, wts, log, lambda e, tob: ctx[(e, tob)], fops, B, seed=1)
    assert rel_err(np.stack(outs), want) < 1e-4


def test_set_context_for_all_envs_at_once():
    """env = -1 publishes [B, L, P, n_kv, hd] contexts in one call: the roll equals the
    one with per-env publishes bit for bit; a t_obs that would decrease for one env
    rejects the whole call."""
    import torch
    from paper_2609_34170_amd import ravel
    s, wts = _tiny_bf16(batch=3)
    B = 3
    ctx = [synth.draw_context(s, 0, e, 0) for e in range(B)]
    a = GpuRoll(s, wts, B, seed=2)
    for e in range(B):
        a.set_context(e, *ctx[e], 0)
    want = _roll(a, s, 5)
    b = GpuRoll(s, wts, B, seed=2)
    K = b.to_dev(np.stack([c[0] for c in ctx]))
    V = b.to_dev(np.stack([c[1] for c in ctx]))
    b.buf.set_context(-1, K, V, 0)
    got = _roll(b, s, 5)
    assert np.array_equal(got, want)
    b.buf.set_context(1, b.to_dev(ctx[1][0]), b.to_dev(ctx[1][1]), 4)
    with pytest.raises(ravel.RavelError, match="E_STATE"):
        b.buf.set_context(-1, K, V, 3)  # env 1 would go back from 4 to 3
    with pytest.raises(ravel.RavelError, match="E_INVALID"):
        b.buf.set_context(-1, None, None, 9)
    torch.cuda.synchronize()
