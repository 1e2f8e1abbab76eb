"""Benchmark of the rolling denoise step on one MI355X.

Default workload: the pi-style action expert at batch 1 (18 layers, width
1024, 8 query heads / 1 KV head of 256, gated-GeLU MLP 4096, H = 50 slots of
action dim 32, 816 prefix tokens per layer, 16 FOP tokens), bf16 weights and
activations with fp32 accumulation, one context published at t = 0.  The
same model at batch 64 (per-env contexts, staggered refresh every 5 steps)
is measured too and reported under "batch64".

One step = one ravel_step: the whole expert pass, Euler update, release and
noise append for every env (one hipGraph replay).  Inputs (weights, contexts,
FOP tokens) are resident in HBM before timing starts.

Prints ONE JSON line.  Extra measurements:
  * roofline   -- the dominant kernel class of the step (largest total time in
                  an eagerly profiled step, HIP events around each launch on
                  the step stream): algorithmic bytes (or flops) / time;
  * step_roofline -- the whole step: algorithmic bytes per step / step time;
  * cpu_baseline -- the numpy oracle (fp32) on a bounded sample of the same
                  workload on the host cores;
  * batch64.train_forward -- the streaming-aligned training objective (forward
                  and loss) over the batch of 64 with random context ages;
  * relative_actions -- the step with every action dimension relative to a
                  moving robot state (batch-1 workloads);
  * offset_forms -- the step with the offset fed the X-VLA way (concatenated to
                  the action input) and the DynamicVLA way (action-time MLP plus
                  offset-conditioned adapter), batch-1 workloads;
  * rotary_positions -- the step with rotary positions of the buffer tokens,
                  batch-1 workloads;
  * full_denoise -- the full-horizon synchronous baseline on the same kernels
                  (batch-1 workloads): ms per chunk of 10 and of H Euler steps
                  and its first-action time relative to one rolling step;
  * roofline.traffic -- HBM bytes per launch of the dominant kernel from
                  rocprofv3 FETCH_SIZE / WRITE_SIZE runs scaled by the same
                  counters on a plain copy of known size (profiles/traffic.json,
                  written from those runs); null unless the kernel's source
                  files still hash to the values recorded there.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "rolling denoise steps/s (batch-1 latency us, batch-64) + % HBM/MFMA roofline"
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=1000)
    p.add_argument("--warmup", type=int, default=50)
    p.add_argument("--workload", default="pi_b1", choices=["pi_b1", "pi_b64", "small_bf16", "large_b16", "tiny_fp32"])
    p.add_argument("--no-batch64", action="store_true", help="skip the batch-64 secondary measurement")
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--no-full", action="store_true", help="skip the full-horizon denoising baseline")
    p.add_argument("--cpu-seconds", type=float, default=15.0)
    p.add_argument("--profile-steps", type=int, default=3)
    p.add_argument("--no-configs", action="store_true",
                   help="skip the other workloads (tiny fp32, small bf16, large expert at batch 16)")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="first run 5 plain device copies of MIB MiB (counter calibration under rocprofv3)")
    return p.parse_args()


def traffic_of(kernel: str, workload: str):
    """HBM bytes per launch recorded for this kernel and workload, if its sources are unchanged."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    from paper_2609_34170_amd.profiling import sources_sha256
    digest = sources_sha256(kernel)
    for e in rec.get("entries", []):
        if e.get("kernel") == kernel and e.get("workload") == workload and e.get("sources_sha256") == digest:
            return e.get("bytes_per_launch")
    return None


def copy_calibration(mib: int):
    import torch
    n = mib << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"[copy calibration] 5 copies of {n} bytes (read {n}, write {n} per copy)")
    del src, dst


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(s, batch) -> float:
    """Bytes one step must move: every weight once plus each env's context and FOP tokens."""
    import synth
    elt = 2 if s.dtype == synth.workloads.BF16 else 4
    n = 0
    for name, shp in synth.weight_shapes(s, with_fop_encoder=False):
        if name.startswith("time."):
            continue  # flow-time conditioning is fixed per slot and precomputed
        cnt = int(np.prod(shp))
        if name == "final.mod.w":
            cnt = cnt * 2 // 3  # the gate chunk of the final modulation is unused
        if name == "final.mod.b":
            cnt = cnt * 2 // 3
        is_vec = len(shp) == 1 or name in ("delta.w1", "in.w")
        n += cnt * (4 if is_vec else elt)
    kvd = s.n_kv_heads * s.head_dim
    n += batch * s.layers * s.prefix_len * kvd * 2 * elt  # prefix K and V
    n += batch * s.n_fop * s.width * elt  # FOP tokens
    n += batch * s.horizon * s.action_dim * 4 * 2  # ring read + write
    return float(n)


def modulation_rows(s, batch) -> int:
    """Buffer rows whose modulation the step computes.  With more than 64 rows the
    modulation GEMMs run once per distinct offset conditioning (envs with equal
    context age share delta): at steady state the refresh policy leaves
    min(batch, period) distinct ages when staggered, one otherwise."""
    H = s.horizon
    if batch * H <= 64 or batch == 1:
        return batch * H
    groups = min(batch, s.context_period) if (s.stagger and s.context_period > 0) else 1
    return groups * H


def algorithmic_flops(s, batch, mod_rows=None) -> float:
    w, H, F = s.width, s.horizon, s.mlp_dim
    qd, kvd = s.n_q_heads * s.head_dim, s.n_kv_heads * s.head_dim
    M = batch * H
    Mm = modulation_rows(s, batch) if mod_rows is None else mod_rows
    f = 2.0 * batch * w * w  # offset MLP
    f += 2.0 * M * w * s.action_dim * 2  # in / out projections
    per_layer = 2.0 * Mm * w * 6 * w + 2.0 * M * w * (qd + 2 * kvd) + 2.0 * M * qd * w + 2.0 * M * w * 3 * F
    per_layer += 4.0 * batch * s.n_q_heads * H * (s.prefix_len + H) * s.head_dim
    f += s.layers * per_layer
    n_ad = len(s.adapter_layers())
    f += n_ad * (2.0 * M * w * qd * 2 + 2.0 * batch * s.n_fop * w * 2 * kvd
                 + 4.0 * batch * s.n_q_heads * H * s.n_fop * s.head_dim)
    f += 2.0 * Mm * w * 2 * w  # final modulation
    return f


class Workload:
    def __init__(self, name, weights=None, seed=0):
        import torch

        import synth
        from paper_2609_34170_amd import ravel
        self.torch = torch
        self.s = s = synth.get_config(name)
        self.B = s.batch
        t0 = time.time()
        self.W = weights if weights is not None else synth.draw_weights(s, seed=seed)
        log(f"[{name}] weights drawn in {time.time() - t0:.1f}s")
        self.model = ravel.Model(s, self.W)
        self.buf = ravel.Buffer(self.model, self.B, seed)
        dev = torch.device("cuda:0")
        tdt = torch.bfloat16 if s.dtype == synth.workloads.BF16 else torch.float32
        self.stream = torch.cuda.current_stream()
        # two context generations per env resident in HBM; refreshes alternate between them
        self.ctx = []
        for gen in range(2 if s.context_period > 0 else 1):
            k = torch.empty((self.B, s.layers, s.prefix_len, s.n_kv_heads, s.head_dim), dtype=tdt, device=dev)
            v = torch.empty_like(k)
            for e in range(self.B):
                kk, vv = synth.draw_context(s, seed, e, gen)
                k[e].copy_(torch.from_numpy(kk))
                v[e].copy_(torch.from_numpy(vv))
            self.ctx.append((k, v))
        self.fop = torch.from_numpy(synth.draw_fop_tokens(s, seed, 0)).to(dev).to(tdt).contiguous()
        self.action = torch.zeros((self.B, s.action_dim), dtype=torch.float32, device=dev)
        k, v = self.ctx[0]
        for e in range(self.B):
            self.buf.set_context(e, k[e], v[e], 0)
        # the initial contexts are in place before the first step (their copies are
        # asynchronous, and a step publishes only copies that have completed)
        self.buf.sync()
        self.t = 0
        self.gen = [0] * self.B
        # refreshes come from the VLM worker's own stream (the paper's separate VLM and
        # action-expert workers): their copies run beside the steps, and a step applies a
        # refresh once its copy has completed
        self.producer = torch.cuda.Stream()
        log(f"[{name}] ready in {time.time() - t0:.1f}s")

    def refresh(self):
        """Context refreshes of the workload's policy due before step self.t."""
        s = self.s
        if s.context_period <= 0 or self.t == 0:
            return
        for e in range(self.B):
            phase = (self.t + e) if s.stagger else self.t
            if phase % s.context_period == 0 and self.t >= s.context_period:
                self.gen[e] ^= 1
                k, v = self.ctx[self.gen[e]]
                self.buf.set_context(e, k[e], v[e], self.t - s.context_period, stream=self.producer)

    def step(self):
        self.refresh()
        self.buf.step(self.fop, self.action)
        self.t += 1

    def timed(self, steps, warmup):
        torch = self.torch
        for _ in range(warmup):
            self.step()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        w0 = time.perf_counter()
        e0.record(self.stream)
        for _ in range(steps):
            self.step()
        e1.record(self.stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        return e0.elapsed_time(e1) / steps, wall

    def full_denoise_timing(self, steps_list, reps=5):
        """Full-horizon synchronous baseline: ms per chunk (steps expert passes) for each
        step count, timed with HIP events after one untimed call (which also builds the
        step count's flow-time table)."""
        torch = self.torch
        s = self.s
        noise = torch.randn((self.B, s.horizon, s.action_dim), dtype=torch.float32, device="cuda",
                            generator=torch.Generator(device="cuda").manual_seed(0))
        chunk = torch.empty_like(noise)
        res = []
        for S in steps_list:
            self.buf.full_denoise(S, self.fop, noise, chunk)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(self.stream)
            for _ in range(reps):
                self.buf.full_denoise(S, self.fop, noise, chunk)
            e1.record(self.stream)
            torch.cuda.synchronize()
            res.append((S, e0.elapsed_time(e1) / reps))
        return res

    def train_timing(self, steps, warmup=3, max_age=10):
        """Streaming-aligned training forward + loss over the batch (random targets, noise
        and context ages 0 .. max_age-1): ms per batch."""
        torch = self.torch
        s = self.s
        g = torch.Generator(device="cuda").manual_seed(1)
        shape = (self.B, s.horizon, s.action_dim)
        target = torch.randn(shape, dtype=torch.float32, device="cuda", generator=g)
        noise = torch.randn(shape, dtype=torch.float32, device="cuda", generator=g)
        ages = torch.randint(0, max_age, (self.B,), dtype=torch.int64, device="cuda", generator=g)
        loss = torch.empty(self.B, dtype=torch.float32, device="cuda")
        for _ in range(warmup):
            self.buf.train_loss(target, noise, ages, self.fop, loss)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(self.stream)
        for _ in range(steps):
            self.buf.train_loss(target, noise, ages, self.fop, loss)
        e1.record(self.stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps, int(torch.unique(ages).numel())

    def relative_timing(self, steps, warmup=20):
        """Relative actions (every action dimension relative to a random-walk state): a
        second buffer on the same model and context, ms per step."""
        torch = self.torch
        from paper_2609_34170_amd import ravel
        s = self.s
        buf = ravel.Buffer(self.model, self.B, 1)
        buf.set_relative_dims(np.ones(s.action_dim, dtype=np.int32))
        k, v = self.ctx[0]
        for e in range(self.B):
            buf.set_context(e, k[e], v[e], 0)
        buf.sync()
        g = torch.Generator(device="cuda").manual_seed(2)
        walk = torch.cumsum(0.05 * torch.randn((steps + warmup, self.B, s.action_dim), dtype=torch.float32,
                                               device="cuda", generator=g), dim=0).contiguous()
        for i in range(warmup):
            buf.step_state(self.fop, walk[i], self.action)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(self.stream)
        for i in range(steps):
            buf.step_state(self.fop, walk[warmup + i], self.action)
        e1.record(self.stream)
        torch.cuda.synchronize()
        buf.close()
        return e0.elapsed_time(e1) / steps

    def offset_form_timing(self, mode, steps, warmup=20, rope_base=0.0):
        """The step with the offset fed the X-VLA way (mode 1: concatenated to the
        action input) or the DynamicVLA way (mode 2: in the action-time MLP plus the
        offset-conditioned adapter), or with rotary positions of the buffer tokens
        (rope_base > 0): a model of the same widths that shares every other weight,
        on the same context; ms per step."""
        torch = self.torch
        import synth
        from paper_2609_34170_amd import ravel
        WL = synth.workloads
        s = self.s.replace(offset_mode=mode, rope_base=rope_base)
        shapes = dict(WL.weight_shapes(s))
        W = {k: v for k, v in self.W.items() if k in shapes and tuple(v.shape) == tuple(shapes[k])}
        rng = np.random.default_rng(7 + mode)
        for k, shp in shapes.items():
            if k not in W:
                a = (0.02 * rng.standard_normal(shp)).astype(np.float32)
                W[k] = WL.bf16_round(a) if s.dtype == WL.BF16 else a
        model = ravel.Model(s, W)
        buf = ravel.Buffer(model, self.B, 1)
        k, v = self.ctx[0]
        for e in range(self.B):
            buf.set_context(e, k[e], v[e], 0)
        buf.sync()
        for _ in range(warmup):
            buf.step(self.fop, self.action)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(self.stream)
        for _ in range(steps):
            buf.step(self.fop, self.action)
        e1.record(self.stream)
        torch.cuda.synchronize()
        buf.close()
        model.close()
        return e0.elapsed_time(e1) / steps

    def fop_timing(self, n=200, warmup=10):
        """ms per ravel_fop_encode call (the FOP stand-in encoder over the batch's
        observation vectors), timed with HIP events; not part of the step."""
        import synth
        torch = self.torch
        obs = torch.from_numpy(synth.draw_observation(self.s, 0, 0, batch=self.B)).to("cuda:0").contiguous()
        z = torch.empty_like(self.fop)
        for _ in range(warmup):
            self.buf.fop_encode(obs, z)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(self.stream)
        for _ in range(n):
            self.buf.fop_encode(obs, z)
        e1.record(self.stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    def latencies(self, n):
        torch = self.torch
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        for a, b in ev:
            a.record(self.stream)
            self.step()
            b.record(self.stream)
        torch.cuda.synchronize()
        return np.array([a.elapsed_time(b) for a, b in ev])

    def profile(self, nsteps):
        """Per kernel class: [launches, bytes, flops, ms] summed over nsteps eager
        steps.  Phase records of the persistent kernel ("persistent/<class>")
        split its time and go to self.phases instead."""
        agg = {}
        self.phases = {}
        total = 0.0
        for _ in range(nsteps):
            self.refresh()
            recs = self.buf.profile_step(self.fop, self.action)
            self.t += 1
            for name, by, fl, ms in recs:
                if name.startswith("phase/"):
                    continue  # single phases of the persistent kernel (already in its classes)
                if name.startswith("persistent/"):
                    a = self.phases.setdefault(name.split("/", 1)[1], [0, 0.0, 0.0, 0.0])
                    a[0] += 1
                    a[1] += by
                    a[2] += fl
                    a[3] += ms
                    continue
                cls = name.split(":")[0]
                a = agg.setdefault(cls, [0, 0.0, 0.0, 0.0])
                a[0] += 1
                a[1] += by
                a[2] += fl
                a[3] += ms
                total += ms
        return agg, total / nsteps


def roofline_of(agg, bound, workload=None):
    dom = max(agg.items(), key=lambda kv: kv[1][3])
    name, (cnt, by, fl, ms) = dom
    if bound == "hbm":
        achieved = by / (ms * 1e-3) / 1e9
        peak, unit = HBM_PEAK_GBS, "GB/s"
    else:
        achieved = fl / (ms * 1e-3) / 1e12
        peak, unit = BF16_PEAK_TFLOPS, "TFLOP/s"
    return {"kernel": name, "bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "traffic": traffic_of(name, workload) if workload else None,
            "algorithmic_bytes_per_launch": round(by / cnt), "launches_per_step_x_steps": cnt,
            "avg_launch_us": round(ms * 1e3 / cnt, 2)}


def cpu_baseline(name, W, seconds):
    import synth
    from oracle.rolling import OracleRavel
    s = synth.get_config(name)
    envs = [0]
    o = OracleRavel(s, W, batch=1, seed=0, dtype=np.float32, env_ids=envs)
    k, v = synth.draw_context(s, 0, 0, 0)
    o.set_context(0, k, v, 0)
    z = synth.draw_fop_tokens(s, 0, 0)[:1]
    n = 0
    t0 = time.perf_counter()
    while True:
        o.step(z)
        n += 1
        el = time.perf_counter() - t0
        if el > seconds or n >= 1000:
            break
    env_steps_per_s = n / el
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        blas = max([i.get("num_threads", 1) for i in info] + [1])
    except Exception:
        blas = None
    cores = blas if blas else os.cpu_count()
    return {"value": round(env_steps_per_s / s.batch, 4), "unit": "steps/s", "cores": cores,
            "cpu_count": os.cpu_count(), "blas_threads": blas, "kind": "oracle",
            "sample": f"{n} steps of env 0 of {name} with the float32 numpy oracle in {el:.1f}s "
                      f"(steps/s = env-steps/s / batch {s.batch})"}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch

    import synth
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_calibration > 0:
        copy_calibration(args.copy_calibration)

    wl = Workload(args.workload)
    s = wl.s
    bound = "hbm" if wl.B == 1 else "mfma"
    ms, wall = wl.timed(args.steps, args.warmup)
    lat = wl.latencies(min(200, args.steps))
    agg, prof_ms = wl.profile(args.profile_steps)
    roof = roofline_of(agg, bound, s.name)
    abytes = algorithmic_bytes(s, wl.B)
    aflops = algorithmic_flops(s, wl.B)
    step_roof = {
        "bytes_per_step": abytes, "flops_per_step": aflops,
        "hbm_GBs": round(abytes / (ms * 1e-3) / 1e9, 1),
        "hbm_frac": round(abytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "mfma_TFLOPs": round(aflops / (ms * 1e-3) / 1e12, 1),
        "mfma_frac": round(aflops / (ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
    }
    out = {
        "metric": METRIC,
        "value": round(1000.0 / ms, 2),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "latency_us_p50": round(float(np.percentile(lat, 50)) * 1e3, 1),
        "latency_us_p95": round(float(np.percentile(lat, 95)) * 1e3, 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if s.dtype == synth.workloads.BF16 else "f32",
        "data": "synthetic (seeded N(0,0.02) weights, N(0,1) prefix KV and FOP tokens)",
        "config": {"workload": s.name, "batch": wl.B, "layers": s.layers, "width": s.width,
                   "heads": f"{s.n_q_heads}q/{s.n_kv_heads}kv x {s.head_dim}", "mlp": s.mlp_dim,
                   "slots": s.horizon, "action_dim": s.action_dim, "prefix_tokens": s.prefix_len,
                   "fop_tokens": s.n_fop, "parallelism": "single GPU"},
        "roofline": roof,
        "step_roofline": step_roof,
        "profiled_step_ms_eager": round(prof_ms, 4),
        "kernel_classes_ms_per_step": {k: round(v[3] / args.profile_steps, 4) for k, v in
                                       sorted(agg.items(), key=lambda kv: -kv[1][3])[:8]},
        "wall_s_timed": round(wall, 3),
    }
    if wl.phases:
        # per phase class of the persistent kernel: ms per step and achieved GB/s
        out["persistent_phases"] = {
            k: {"ms": round(v[3] / args.profile_steps, 4),
                "GBs": round(v[1] / (v[3] * 1e-3) / 1e9, 1) if v[3] > 0 else None}
            for k, v in sorted(wl.phases.items(), key=lambda kv: -kv[1][3])}
    log(f"[{s.name}] {1000.0 / ms:.1f} steps/s, {ms * 1e3:.1f} us/step")
    if not args.no_full and wl.B == 1:
        # relative actions (state conversion around each pass) on the same model
        rms = wl.relative_timing(max(20, min(200, args.steps // 2)))
        out["relative_actions"] = {"ms_per_step": round(rms, 4), "steps_per_s": round(1000.0 / rms, 2),
                                   "vs_absolute_step": round(rms / ms, 4)}
        log(f"[{s.name}] relative actions: {rms * 1e3:.1f} us/step")
        # the other two ways of feeding the offset (App. A.1) on models of the same widths
        out["offset_forms"] = {}
        for mode, key in ((1, "concat_xvla"), (2, "adapter_dynamicvla")):
            oms = wl.offset_form_timing(mode, max(20, min(200, args.steps // 2)))
            out["offset_forms"][key] = {"ms_per_step": round(oms, 4), "steps_per_s": round(1000.0 / oms, 2),
                                        "vs_mlp_step": round(oms / ms, 4)}
            log(f"[{s.name}] offset form {key}: {oms * 1e3:.1f} us/step")
        # rotary positions of the buffer tokens (a rotary phase after each QKV projection)
        rms2 = wl.offset_form_timing(0, max(20, min(200, args.steps // 2)), rope_base=10000.0)
        out["rotary_positions"] = {"ms_per_step": round(rms2, 4), "steps_per_s": round(1000.0 / rms2, 2),
                                   "vs_step": round(rms2 / ms, 4)}
        log(f"[{s.name}] rotary positions: {rms2 * 1e3:.1f} us/step")
        # the synchronous baseline on the same kernels: a chunk needs `steps` expert
        # passes before its first action, a rolling step one (Sec. 4.1 latency table)
        out["full_denoise"] = [
            {"steps": S, "ms_per_chunk": round(fm, 4), "ms_per_pass": round(fm / S, 4),
             "first_action_vs_rolling_step": round(fm / ms, 2)}
            for S, fm in wl.full_denoise_timing(sorted({10, s.horizon}))]
        log(f"[{s.name}] full denoise: " + ", ".join(f"{d['steps']} steps {d['ms_per_chunk']} ms"
                                                       for d in out["full_denoise"]))
    out["fop_encode"] = {"ms_per_call": round(wl.fop_timing(), 4), "batch": wl.B,
                         "note": "FOP stand-in encoder, separate from the step"}
    log(f"[{s.name}] FOP encoder {out['fop_encode']['ms_per_call'] * 1e3:.1f} us per call")
    W = wl.W
    if not args.no_configs and args.workload == "pi_b1":
        # the other workloads: tiny fp32 (latency-bound), small bf16 (its 81 MB of
        # weights and contexts stay in the 256 MB Infinity Cache, so its HBM fraction
        # is quoted with that caveat), the large expert at batch 16 (MFMA-bound)
        wl = None
        torch.cuda.synchronize()
        out["configs"] = {}
        for name, steps_c in (("tiny_fp32", 400), ("small_bf16", 400), ("large_b16", 30)):
            wc = Workload(name)
            sc = wc.s
            msc, _ = wc.timed(steps_c, 10)
            d = {"steps": steps_c, "us_per_step": round(msc * 1e3, 2), "steps_per_s": round(1000.0 / msc, 2),
                 "batch": wc.B}
            if name == "small_bf16":
                by = algorithmic_bytes(sc, wc.B)
                d["hbm_frac"] = round(by / (msc * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
                d["note"] = "bytes per step fit the 256 MB Infinity Cache: not an HBM-streaming figure"
            if name == "large_b16":
                fl = algorithmic_flops(sc, wc.B)
                d["mfma_TFLOPs"] = round(fl / (msc * 1e-3) / 1e12, 1)
                d["mfma_frac"] = round(fl / (msc * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4)
                d["env_steps_per_s"] = round(wc.B * 1000.0 / msc, 1)
            out["configs"][name] = d
            log(f"[{name}] {d['us_per_step']} us/step")
            del wc
            torch.cuda.synchronize()
    if not args.no_batch64 and args.workload == "pi_b1":
        wl = None
        torch.cuda.synchronize()
        w64 = Workload("pi_b64", weights=W)  # the same model at batch 64
        s64 = w64.s
        steps64 = max(10, min(200, args.steps // 5))
        ms64, _ = w64.timed(steps64, 10)
        agg64, _ = w64.profile(2)
        out["batch64"] = {
            "workload": "pi_b64", "steps": steps64, "ms_per_step": round(ms64, 4),
            "steps_per_s": round(1000.0 / ms64, 2), "env_steps_per_s": round(64 * 1000.0 / ms64, 1),
            "mfma_TFLOPs": round(algorithmic_flops(s64, 64) / (ms64 * 1e-3) / 1e12, 1),
            "mfma_frac": round(algorithmic_flops(s64, 64) / (ms64 * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4),
            "roofline": roofline_of(agg64, "mfma", "pi_b64"),
            # eager profile steps: ms per step and achieved TFLOP/s per kernel class
            "kernel_classes": {k: {"ms": round(v[3] / 2, 4),
                                   "TFs": round(v[2] / (v[3] * 1e-3) / 1e12, 1) if v[2] > 0 else None}
                               for k, v in sorted(agg64.items(), key=lambda kv: -kv[1][3])[:8]},
        }
        log(f"[pi_b64] {1000.0 / ms64:.1f} steps/s")
        # streaming-aligned training forward + loss on the same batch of 64 (Sec. 3.3)
        tms, n_ages = w64.train_timing(max(5, steps64 // 4))
        tfl = algorithmic_flops(s64, 64, mod_rows=n_ages * s64.horizon)
        out["batch64"]["train_forward"] = {
            "ms_per_batch": round(tms, 4), "samples_per_s": round(64 * 1000.0 / tms, 1),
            "distinct_context_ages": n_ages, "mfma_TFLOPs": round(tfl / (tms * 1e-3) / 1e12, 1),
            "mfma_frac": round(tfl / (tms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4)}
        log(f"[pi_b64] training forward + loss {tms:.3f} ms per batch of 64")
        del w64
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(args.workload, W, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
