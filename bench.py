"""Throughput of the environment-plus-policy step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 4]
                    [--no-cpu-baseline] [--no-secondary] [--no-graph] [--no-rollout]
                    [--mall-flush MB]

One step = im_policy_act (MLP forward + Gaussian sampling) followed by
im_env_step_fused (reference sampling, FK, reward, termination, masked reset,
observation) for every env.  The physics solver is outside this path: a
kinematic stand-in produces the sim state each step would see.  To keep the
stand-in out of the timed region the rollout is recorded first (stand-in sim
states of every step kept resident in HBM, distinct buffers per step), then
replayed from the same initial state: the timed loop holds exactly the two
calls per step, with every input already in device memory.

Prints ONE JSON line.  `value` = n_envs * steps / timed seconds.
`graph` times the same steps captured as one HIP graph and replayed (results
checked equal to the eager run).  `roofline` covers the policy MLP (the
dominant call, MFMA-bound),
`roofline_env` the fused env-step kernel (HBM-bound); both use algorithmic
work (FLOPs / bytes) over the mean duration measured with HIP events on the
launch stream during the timed loop.  `traffic` is the HBM bytes per launch
measured with the profiler's byte counters on the same kernels (null when the
kernel sources changed since).  `mall_flushed` repeats the timed calls with
the last-level cache flushed before each step.  `rollout` times a whole PPO
rollout of the workload (policy, value head and env step per step written in
place into the rollout storage, then GAE and the rollout summaries).  `cpu_baseline` times
the CPU oracle on a bounded sample of the same workload.
"""
import argparse
import hashlib
import json
import os
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "env-steps/s (ref FK+reward+obs+reset+MLP policy) at 4096 & 65536 envs"
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}

# Measured HBM traffic per launch: rocprofv3 --pmc FETCH_SIZE and --pmc WRITE_SIZE passes
# over this bench (KiB per dispatch, mean over the dispatches of each kernel), each scaled
# by what the same counter reads over a plain 512 MiB device copy (bench.py
# --calibrate-copy 512): FETCH_SIZE reported 262166 KiB for 524288 KiB read, WRITE_SIZE
# 524288 KiB for 524288 KiB written, so the factors are 2.0 and 1.0.  Each entry is keyed
# by a hash of the kernel's source file and the device headers it includes; once one of
# them changes the figure no longer describes the kernel and the bench reports null.
FETCH_SCALE, WRITE_SCALE = 2.0, 1.0
CSRC = os.path.join(ROOT, "paper_2609_09821_amd", "csrc")
SHARED_SOURCES = []
TRAFFIC_KIB = {
    # policy: one entry per launch of im_policy_act (a bf16 policy is one launch)
    "policy": {"sources": ["policy_kernels.hip", "device_math.h", "launch.h"], "sha": "057f2257ff61f4c1", "workloads": {
        4: {"fetch": [109680.0], "write": [35584.0]},
        5: {"fetch": [140414.0], "write": [58368.0]}}},
    "env": {"sources": ["env_kernels.hip", "device_math.h", "tables.h"], "sha": "eeed804b596bf8b3", "workloads": {
        4: {"fetch": [61765.5], "write": [169488.8]},
        5: {"fetch": [184002.8], "write": [413742.0]}}},
}


def source_sha(kind):
    s = hashlib.sha256()
    for f in [os.path.join(CSRC, x) for x in TRAFFIC_KIB[kind]["sources"]] + SHARED_SOURCES:
        with open(f, "rb") as fh:
            s.update(fh.read())
    return s.hexdigest()[:16]


def measured_traffic(kind, wid):
    """(total, read, write) HBM bytes per launch, or None when not measured on the
    current kernel sources."""
    e = TRAFFIC_KIB[kind]
    m = e["workloads"].get(wid)
    if m is None or source_sha(kind) != e["sha"]:
        return None
    rd = 1024.0 * FETCH_SCALE * sum(m["fetch"])
    wr = 1024.0 * WRITE_SCALE * sum(m["write"])
    return rd + wr, rd, wr


def algorithmic_env_bytes(B, D, n_envs, n_reset, A_prev=0):
    """HBM bytes one env step must move: sim state read (52 B per body), env
    state in and out (16 + 16), reward (4), flags (2), observation (4 D), the
    previous action read when the observation holds it (4 A_prev), and the
    reference sim state written for reset envs (52 B per body)."""
    return n_envs * (52 * B + 32 + 6 + 4 * D + 4 * A_prev) + n_reset * 52 * B


def mlp_flops(dims, n_envs):
    return 2.0 * n_envs * sum(dims[i] * dims[i + 1] for i in range(len(dims) - 1))


class _Roctx:
    """roctx ranges around the step's calls (visible to rocprofv3 --marker-trace);
    no-ops when the marker library is missing."""

    def __init__(self):
        self.lib = None
        for name in ("librocprofiler-sdk-roctx.so.1", "libroctx64.so.4"):
            try:
                import ctypes
                lib = ctypes.CDLL(os.path.join("/opt/rocm/lib", name))
                lib.roctxRangePushA.argtypes = [ctypes.c_char_p]
                lib.roctxRangePushA.restype = ctypes.c_int
                lib.roctxRangePop.restype = ctypes.c_int
                self.lib = lib
                break
            except OSError:
                continue

    def push(self, name):
        if self.lib is not None:
            self.lib.roctxRangePushA(name)

    def pop(self):
        if self.lib is not None:
            self.lib.roctxRangePop()


ROCTX = _Roctx()


def run_gpu(wid, steps, warmup, graph=True, flush_mb=0):
    import torch
    from paper_2609_09821_amd import binding, synth

    desc = synth.make_world(wid)
    N = desc["n_envs"]
    pol = desc["policy"]
    A = pol["dims"][-1]
    ctx = binding.Context(desc, max_envs=N)
    B, D = ctx.info.n_bodies, ctx.info.obs_dim
    bufs = ctx.buffers(N)
    stream = torch.cuda.current_stream()
    total = warmup + steps

    # ---- record: initial reset, then stand-in sim states of every step ----
    ctx.reset_envs(bufs)
    if bufs.prev_action is not None:
        bufs.prev_action.normal_()
    init = {k: getattr(bufs, k).clone() for k in binding.EnvBuffers.ENV + ("obs",)}
    rec = []
    resets = []
    for t in range(total):
        ctx.standin_physics(bufs, desc["sigma_joint"], desc["sigma_vel"])
        rec.append(tuple(getattr(bufs, k).clone() for k in binding.EnvBuffers.SIM))
        ctx.env_step_fused(bufs, with_ref_frame=False)
        resets.append((bufs.terminated | bufs.truncated).sum())
    n_reset = [int(r) for r in torch.stack(resets).cpu()]
    # the replays write reference states of reset envs into these buffers: keep
    # a pristine copy so that the graph replay sees the same inputs
    pristine = [tuple(x.clone() for x in r) for r in rec] if graph else None
    for k, v in init.items():
        getattr(bufs, k).copy_(v)
    torch.cuda.synchronize()

    mean = torch.empty((N, A), device="cuda")
    action = torch.empty((N, A), device="cuda")
    logp = torch.empty(N, device="cuda")
    A_prev = 0
    if bufs.prev_action is not None:
        # the observation's previous action is the action the policy just drew
        bufs.prev_action = action
        A_prev = A

    # flush_mb > 0: a write of that many MB between steps (outside the per-call
    # events) evicts the last-level cache, so each call starts cold
    scratch = torch.empty(flush_mb << 18, device="cuda") if flush_mb > 0 else None

    def step(t, ev=None):
        bufs.body_pos, bufs.body_quat, bufs.body_linvel, bufs.body_angvel = rec[t]
        if scratch is not None:
            scratch.fill_(float(t))
        if ev is not None:
            ev[0].record(stream)
        ROCTX.push(b"im_policy_act")
        ctx.policy_act(bufs.obs, bufs.env_n, N, mean, action, logp, stream=stream)
        ROCTX.pop()
        if ev is not None:
            ev[1].record(stream)
        ROCTX.push(b"im_env_step_fused")
        ctx.env_step_fused(bufs, stream=stream, with_ref_frame=False)
        ROCTX.pop()
        if ev is not None:
            ev[2].record(stream)

    for t in range(warmup):
        step(t)
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(steps):
        step(warmup + t, events[t])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    final_eager = {k: getattr(bufs, k).clone() for k in binding.EnvBuffers.ENV + ("obs",)}

    # The same timed steps captured as one HIP graph (policy_act and
    # env_step_fused per step, each step with its own recorded sim input) and
    # replayed from the post-warmup state: the launch cost the graph removes.
    graph_wall = None
    if graph:
        def restore_rec(first):
            for t in range(first, total):
                for dst, src in zip(rec[t], pristine[t]):
                    dst.copy_(src)

        restore_rec(0)
        for k, v in init.items():
            getattr(bufs, k).copy_(v)
        for t in range(warmup):
            step(t)
        torch.cuda.synchronize()
        post_warm = {k: getattr(bufs, k).clone() for k in binding.EnvBuffers.ENV + ("obs",)}
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            with torch.cuda.graph(g, stream=side):
                for t in range(steps):
                    bufs.body_pos, bufs.body_quat, bufs.body_linvel, bufs.body_angvel = rec[warmup + t]
                    ctx.policy_act(bufs.obs, bufs.env_n, N, mean, action, logp)
                    ctx.env_step_fused(bufs, with_ref_frame=False)
        torch.cuda.current_stream().wait_stream(side)
        for rep in range(2):                  # one warm replay, one timed
            for k, v in post_warm.items():
                getattr(bufs, k).copy_(v)
            restore_rec(warmup)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            g.replay()
            torch.cuda.synchronize()
            graph_wall = time.perf_counter() - t0
        for k, v in final_eager.items():
            if not torch.equal(getattr(bufs, k), v):
                raise RuntimeError("graph replay differs from the eager run in " + k)
        del g, pristine
    pol_ms = np.array([e[0].elapsed_time(e[1]) for e in events])
    env_ms = np.array([e[1].elapsed_time(e[2]) for e in events])
    rho = float(np.mean(n_reset[warmup:]) / N)
    env_bytes = np.mean([algorithmic_env_bytes(B, D, N, n_reset[warmup + t], A_prev)
                         for t in range(steps)])
    flops = mlp_flops(pol["dims"], N)
    prec = "bf16" if pol["bf16"] else "f32"
    ctx.close()
    return dict(
        desc=desc, N=N, B=B, D=D, wall=wall, pol_ms=float(pol_ms.mean()),
        env_ms=float(env_ms.mean()), rho=rho, env_bytes=float(env_bytes), flops=flops,
        prec=prec, value=N * steps / wall,
        graph_value=None if graph_wall is None else N * steps / graph_wall,
        graph_ms=None if graph_wall is None else graph_wall * 1e3 / steps,
    )


def run_rollout(wid, reps=2):
    """A whole PPO rollout of the workload (T = its step count) written in
    place into the rollout storage: per step policy_act_value (action, logp and
    value of the observation, one staging of it for both networks) and
    env_step_fused, then the value of the last observation, GAE with the
    rollout summaries and the copy of the last observation into slot 0 for the
    next rollout.  The stand-in physics is recorded beforehand and excluded,
    as in the step benchmark; each timed rollout starts from the same state."""
    import torch
    from paper_2609_09821_amd import binding, synth

    desc = synth.make_world(wid)
    N = desc["n_envs"]
    T = int(desc["spec"]["steps"])
    ctx = binding.Context(desc, max_envs=N)
    bufs = ctx.buffers(N)
    ro = binding.RolloutStorage(ctx, N, T)
    stream = torch.cuda.current_stream()
    bufs.obs = ro.obs[0]
    ctx.reset_envs(bufs)
    init = {k: getattr(bufs, k).clone() for k in binding.EnvBuffers.ENV}
    init_obs = ro.obs[0].clone()
    rec = []
    for t in range(T):
        ctx.standin_physics(bufs, desc["sigma_joint"], desc["sigma_vel"])
        rec.append(tuple(getattr(bufs, k).clone() for k in binding.EnvBuffers.SIM))
        ro.env_bufs(bufs, t)
        ctx.env_step_fused(bufs, with_ref_frame=False)
    pristine = [tuple(x.clone() for x in r) for r in rec]

    def restore():
        for k, v in init.items():
            getattr(bufs, k).copy_(v)
        ro.obs[0].copy_(init_obs)
        ro.ep_return.zero_()
        ro.ep_length.zero_()
        for r, p in zip(rec, pristine):
            for dst, src in zip(r, p):
                dst.copy_(src)
        torch.cuda.synchronize()

    def one(ev=None):
        for t in range(T):
            bufs.body_pos, bufs.body_quat, bufs.body_linvel, bufs.body_angvel = rec[t]
            if ev is not None:
                ev[t][0].record(stream)
            ctx.policy_act_value(ro.obs[t], bufs.env_n, N, ro.mean[t], ro.action[t],
                                 ro.logp[t], ro.value[t], stream=stream)
            if ev is not None:
                ev[t][1].record(stream)
            ro.env_bufs(bufs, t)
            ctx.env_step_fused(bufs, stream=stream, with_ref_frame=False)
            if ev is not None:
                ev[t][2].record(stream)
        ctx.value(ro.obs[T], N, ro.value[T], stream=stream)
        if ev is not None:
            ev[T][0].record(stream)
        ctx.gae(ro, synth.GAMMA, synth.LAMBDA, stream=stream)
        if ev is not None:
            ev[T][1].record(stream)
        ro.obs[0].copy_(ro.obs[T])

    restore()
    one()                                   # warm-up
    walls, polval, env, gae = [], [], [], []
    for _ in range(reps):
        restore()
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(T + 1)]
        t0 = time.perf_counter()
        one(ev)
        torch.cuda.synchronize()
        walls.append(time.perf_counter() - t0)
        polval.append(np.mean([ev[t][0].elapsed_time(ev[t][1]) for t in range(T)]))
        env.append(np.mean([ev[t][1].elapsed_time(ev[t][2]) for t in range(T)]))
        gae.append(ev[T][0].elapsed_time(ev[T][1]))
    summ = ro.summary.cpu().numpy()
    ppo = None
    if desc["policy"]["bf16"]:
        ppo = run_ppo_update(ctx, desc, ro)
    ctx.close()
    wall = float(np.min(walls))
    return {
        "workload": desc["spec"]["name"], "n_envs": N, "T": T,
        "value": N * T / wall, "unit": "env-steps/s", "ms_per_rollout": wall * 1e3,
        "policy_value_us_per_step": float(np.mean(polval)) * 1e3,
        "env_step_us_per_step": float(np.mean(env)) * 1e3,
        "gae_summary_us": float(np.mean(gae)) * 1e3,
        "episodes_ended": int(summ[3]), "mean_reward": float(summ[0] / (N * T)),
        "ppo_update": ppo,
        "note": "policy_act_value + env_step_fused per step into the rollout storage, value of "
                "the last observation, GAE + summaries, last observation to slot 0; stand-in "
                "physics excluded; best of %d rollouts" % reps,
    }


def ppo_flops_per_sample(dims):
    """Forward, input-gradient and weight-gradient products of one MLP:
    2 in out each, no input gradient for the first layer."""
    macs = [dims[i] * dims[i + 1] for i in range(len(dims) - 1)]
    return 2.0 * (3 * sum(macs) - macs[0])


def run_ppo_update(ctx, desc, ro, reps=2):
    """One PPO update (the configuration table's baseline: 5 learning epochs,
    here 4 minibatches) over the rollout storage just filled, timed with HIP
    events on the launch stream after one warm-up update."""
    import torch
    from paper_2609_09821_amd import binding

    N, T = ro.n_envs, ro.T
    p = dict(binding.PPO_DEFAULTS)
    n_chunks = T * N // 64
    mb = (n_chunks + p["minibatches"] - 1) // p["minibatches"] * 64
    ctx.ppo_setup(mb)
    rng = np.random.default_rng(0)
    perm = torch.from_numpy(np.stack([rng.permutation(n_chunks) for _ in range(p["epochs"])])
                            .astype(np.int32)).cuda()
    lr = torch.full((1,), 5e-4, device="cuda")
    stats = torch.zeros(len(binding.PPO_STATS), dtype=torch.float64, device="cuda")
    batch = binding.ppo_batch(ro, perm, lr, stats)
    params = binding.ppo_params(**p)
    stream = torch.cuda.current_stream()
    # the first update runs on the rollout's own (on-policy) data: its loss
    # statistics are the ones reported; the timed repeats reuse the same batch
    ctx.ppo_update(batch, params, stream=stream)
    st = stats.cpu().numpy()
    times = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        ctx.ppo_update(batch, params, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) * 1e-3)
    t = float(np.min(times))
    samples = p["epochs"] * T * N
    flops = samples * (ppo_flops_per_sample(desc["policy"]["dims"]) +
                       ppo_flops_per_sample(desc["critic"]["dims"]))
    return {
        "ms": t * 1e3, "samples_per_s": samples / t, "epochs": p["epochs"],
        "minibatches": p["minibatches"], "minibatch_samples": mb,
        "tflops": flops / t / 1e12, "frac_of_bf16_peak": flops / t / 1e12 / MFMA_PEAK_TFLOPS["bf16"],
        "mean_kl": float(st[2] / st[5]), "mean_clip_frac": float(st[3] / st[5]),
        "note": "forward, backward and Adam of actor and critic on MFMA; flops = 2 in out per "
                "layer for the forward, input and weight gradients (no input gradient for the "
                "first layer), per sample and epoch; mean_kl and mean_clip_frac from the first "
                "update, which runs on the rollout's own data (the timed repeats reuse it); with "
                "sigma = 0.05 and a random-init policy, Adam's first steps at the paper's rate "
                "move the mean by more than sigma, so both are large: a load figure, not a "
                "learning one",
    }


def calibrate_probes():
    """Measurement probes of the GPU itself (include/instantmimic_calib.h) and
    of the vendor GEMM on the policy's layer shapes: what the chip sustains for
    the instruction mixes the step's kernels use.  One JSON line; each figure
    is the best of 5 timed launches (HIP events on the launch stream)."""
    import torch
    import torch.nn.functional as F
    from paper_2609_09821_amd import binding

    props = torch.cuda.get_device_properties(torch.cuda.current_device())
    n_cu = props.multi_processor_count
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream

    def best_ms(launch, reps=5):
        launch()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            launch()
            e1.record(stream)
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        return min(ts)

    res = {"n_cu": n_cu, "clock_for_per_clock_figures_ghz": 2.4}
    blocks = 2 * n_cu               # two wavefronts per SIMD
    out = torch.empty(256 * blocks, device="cuda")
    for kind, name, flop, iters in ((binding.IM_CALIB_MFMA_BF16, "mfma_bf16_32x32x16", 32768, 20000),
                                    (binding.IM_CALIB_MFMA_F32, "mfma_f32_32x32x2", 4096, 10000)):
        ms = best_ms(lambda: binding.im_calib_mfma(kind, iters, blocks, out.data_ptr(), sp))
        res[name + "_tflops"] = 4 * blocks * iters * 8 * flop / (ms * 1e-3) / 1e12
    lds = {}
    outl = torch.empty(64 * 16 * n_cu, dtype=torch.int32, device="cuda")
    for width in (16, 8):
        for waves in (1, 2, 4, 8, 12, 16):
            iters = 2000
            ms = best_ms(lambda: binding.im_calib_lds(width, waves, iters, n_cu, outl.data_ptr(), sp))
            per_cu = waves * 64 * width * 16 * iters / (ms * 1e-3)
            lds["b%d_w%d" % (8 * width, waves)] = {"gbs_per_cu": per_cu / 1e9,
                                                  "bytes_per_clk_per_cu": per_cu / 2.4e9}
    res["lds_read"] = lds
    rd = {}
    outr = torch.empty(256 * 8 * n_cu, dtype=torch.int32, device="cuda")
    for label, mib, passes in (("hbm_1gib", 1024, 1), ("mall_128mib", 128, 8), ("l2_2mib", 2, 256)):
        buf = torch.ones((mib << 20) // 4, device="cuda")
        ms = best_ms(lambda: binding.im_calib_read(buf.data_ptr(), mib << 20, passes, 8 * n_cu,
                                                   outr.data_ptr(), sp))
        rd[label + "_tbs"] = passes * (mib << 20) / (ms * 1e-3) / 1e12
        del buf
    src = torch.ones(128 << 20, device="cuda")      # 512 MiB
    dst = torch.empty_like(src)
    ms = best_ms(lambda: dst.copy_(src))
    rd["copy_512mib_tbs"] = 2 * src.numel() * 4 / (ms * 1e-3) / 1e12
    del src, dst
    res["global_read"] = rd
    blas = {}
    N = 65536
    for K, M in ((384, 1024), (1024, 1024), (1024, 512), (512, 96)):
        x = torch.randn(N, K, device="cuda", dtype=torch.bfloat16)
        w = torch.randn(M, K, device="cuda", dtype=torch.bfloat16)
        b = torch.randn(M, device="cuda", dtype=torch.bfloat16)
        for label, f in (("linear", lambda: F.linear(x, w)),
                         ("linear_bias_relu", lambda: torch.relu(F.linear(x, w, b)))):
            ms = best_ms(f)
            blas["%s_%dx%dx%d" % (label, N, K, M)] = {"us": ms * 1e3,
                                                       "tflops": 2 * N * K * M / (ms * 1e-3) / 1e12}
        del x, w, b
    res["vendor_gemm_bf16"] = blas
    print(json.dumps({"calibration": res}), flush=True)


def cpu_model():
    """The host CPU's model name (lscpu, else /proc/cpuinfo)."""
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(wid, target_s=16.0):
    """The oracle, as it stands, on a bounded sample of workload `wid`."""
    import oracle
    from paper_2609_09821_amd import synth

    desc = synth.make_world(wid)
    w = oracle.World(desc)
    pol = desc["policy"]

    def env_part(n):
        st = w.state(n)
        w.reset_envs(st)
        w.standin(st, desc["sigma_joint"], desc["sigma_vel"])
        prev = np.zeros((n, w.A), np.float32) if desc["config"]["obs_prev_action"] else None
        t0 = time.perf_counter()
        w.env_step(st, prev_action=prev)
        return time.perf_counter() - t0, st

    def mlp_part(st, n):
        obs = np.ascontiguousarray(st.obs[:, :n])
        t0 = time.perf_counter()
        oracle.policy(pol, desc["config"]["seed"], obs, st.n[:n])
        return time.perf_counter() - t0

    n_env = 2048
    t_env, st = env_part(n_env)
    while t_env < target_s / 4 and n_env < desc["n_envs"]:
        n_env = min(desc["n_envs"], int(n_env * min(8.0, max(2.0, target_s / 2 / max(t_env, 1e-4)))))
        t_env, st = env_part(n_env)
    n_mlp = 64
    t_mlp = mlp_part(st, n_mlp)
    while t_mlp < target_s / 4 and n_mlp < n_env:
        n_mlp = min(n_env, int(n_mlp * min(8.0, max(2.0, target_s / 2 / max(t_mlp, 1e-4)))))
        t_mlp = mlp_part(st, n_mlp)
    per_env = t_env / n_env + t_mlp / n_mlp
    return {
        "value": 1.0 / per_env,
        "unit": "env-steps/s",
        "cores": oracle.num_threads(),
        "affinity_cpus": len(os.sched_getaffinity(0)),
        "cpu_model": cpu_model(),
        "kind": "oracle",
        "sample": "one step of the %d-env workload: oracle env step on %d envs (%.2f s), "
                  "oracle MLP+sampling on %d envs (%.2f s); per-env times summed"
                  % (desc["n_envs"], n_env, t_env, n_mlp, t_mlp),
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=32)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=4, choices=[1, 2, 3, 4, 5, 6])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true")
    ap.add_argument("--no-rollout", action="store_true")
    ap.add_argument("--mall-flush", type=int, default=512, metavar="MB",
                    help="also time the calls with the last-level cache flushed before each step "
                         "by a write of MB megabytes (0: skip)")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the HIP-graph replay of the timed steps")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MB",
                    help="only run a plain device copy of MB mebibytes (profiler calibration "
                         "of the HBM byte counters) and exit")
    ap.add_argument("--calibrate-probes", action="store_true",
                    help="only run the GPU measurement probes (MFMA, LDS, global reads, copy, "
                         "vendor GEMM on the policy's layer shapes), print them and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the env-plus-policy step shards over envs with no "
              "exchange, and this build runs on a single MI355X (use --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.calibrate_probes:
        calibrate_probes()
        return
    if args.calibrate_copy:
        n = args.calibrate_copy * (1 << 20) // 4
        src = torch.ones(n, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration_copy_bytes": 4 * n}), flush=True)
        return

    # the secondary workload first: right after the long bf16 runs its short
    # eager calls measured slower than alone (the graph replays did not)
    sec = None
    if not args.no_secondary and args.workload != 2:
        sec = run_gpu(2, args.steps, args.warmup, graph=not args.no_graph)
    r = run_gpu(args.workload, args.steps, args.warmup, graph=not args.no_graph)
    cold = None
    if args.mall_flush > 0:
        cold = run_gpu(args.workload, args.steps, args.warmup, graph=False, flush_mb=args.mall_flush)
    desc = r["desc"]
    spec = desc["spec"]
    mlp_tflops = r["flops"] / (r["pol_ms"] * 1e-3) / 1e12
    env_gbs = r["env_bytes"] / (r["env_ms"] * 1e-3) / 1e9
    peak = MFMA_PEAK_TFLOPS[r["prec"]]
    tr_pol = measured_traffic("policy", args.workload)
    tr_env = measured_traffic("env", args.workload)
    out = {
        "metric": METRIC,
        "value": r["value"],
        "unit": "env-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r["wall"] * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": r["prec"],
        "data": "synthetic",
        "config": {
            "workload": spec["name"],
            "n_envs": r["N"],
            "skeleton": spec["skeleton"],
            "mlp": "-".join(str(x) for x in spec["mlp"]),
            "precision": "env kernels fp32; MLP %s" % (
                "bf16 x bf16 -> fp32 accumulate" if r["prec"] == "bf16" else "fp32"),
            "reset_fraction_per_step": r["rho"],
            "parallelism": "single GPU",
        },
        "graph": None if r["graph_value"] is None else {
            "value": r["graph_value"], "ms_per_step": r["graph_ms"],
            "note": "same timed steps captured as one HIP graph and replayed; results "
                    "checked equal to the eager run"},
        "roofline": {
            "kernel": ("policy MLP (im_policy_act: policy_fused_bf16_kernel, every layer and "
                       "the sampling in one launch)" if r["prec"] == "bf16" else
                       "policy MLP (im_policy_act: one MFMA GEMM per layer)"),
            "bound": "mfma", "achieved": mlp_tflops, "peak": peak, "unit": "TFLOP/s",
            "frac": mlp_tflops / peak, "traffic": tr_pol and tr_pol[0],
            "traffic_unit": "HBM bytes per launch",
            "traffic_read_write": tr_pol and tr_pol[1:],
            "per_launch_ms": r["pol_ms"], "work_per_launch": r["flops"],
        },
        "roofline_env": {
            "kernel": "env_step_kernel (im_env_step_fused)",
            "bound": "hbm", "achieved": env_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": env_gbs / HBM_PEAK_GBS, "traffic": tr_env and tr_env[0],
            "traffic_unit": "HBM bytes per launch",
            "traffic_read_write": tr_env and tr_env[1:],
            "per_launch_ms": r["env_ms"], "work_per_launch": r["env_bytes"],
        },
    }
    if cold is not None:
        c_gbs = cold["env_bytes"] / (cold["env_ms"] * 1e-3) / 1e9
        c_tf = cold["flops"] / (cold["pol_ms"] * 1e-3) / 1e12
        out["mall_flushed"] = {
            "flush_mb": args.mall_flush,
            "policy_ms": cold["pol_ms"], "env_step_ms": cold["env_ms"],
            "env_steps_per_s_of_calls": cold["N"] / ((cold["pol_ms"] + cold["env_ms"]) * 1e-3),
            "policy_tflops": c_tf, "policy_frac": c_tf / peak,
            "env_gbs": c_gbs, "env_frac": c_gbs / HBM_PEAK_GBS,
            "note": "the same calls with the last-level cache (Infinity Cache) flushed by a "
                    "write before each step; throughput from the per-call events"}
    if sec is not None:
        s = sec
        out["also"] = [{
            "workload": s["desc"]["spec"]["name"], "n_envs": s["N"], "value": s["value"],
            "ms_per_step": s["wall"] * 1e3 / args.steps, "policy_ms": s["pol_ms"],
            "env_step_ms": s["env_ms"], "graph_value": s["graph_value"],
            "graph_ms_per_step": s["graph_ms"]}]
    if not args.no_rollout:
        out["rollout"] = run_rollout(args.workload)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.workload)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
