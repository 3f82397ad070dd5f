"""Benchmark of one STAR rescheduling round on one MI355X.

A step is one full pass of the hot path over one decode step of the
continuous-mode workload (1024 concurrent requests on 8 decode instances,
bf16 hidden states [1024, 4096] from an AR(1) process, head 4096 -> 512
(GELU) -> 64 length bins with EMA alpha 0.2, horizon 16384 steps in 64-step
buckets, all 1024 x 8 candidates scored, top-256 ranked):
    a prediction -> star_project_and_score (the load projection and the
    migration scoring and ranking in one call).
The reported mode (graph_pipelined) makes the predictions with
star_predict_overlap, one launch per round holding that round's head and the
next round's first-layer product; the eager and one-graph-per-round modes use
star_predict.
Inputs for 200 decode steps are staged in HBM before timing.  The metric is
requests predicted + scored per second (= 1024 / seconds per round) and
microseconds per round.

Prints ONE JSON line.  Usage:
    python bench.py [--gpus 1] [--steps 200] [--warmup 40] [--mode graph_pipelined|...]

``--path mlp4`` measures the paper's own predictor, the 4-layer ReLU
regression head 3584 -> 2048 -> 512 -> 64 -> 1 (random-initialised weights of
that shape): per step one star_predict_mlp4 call on a 1024-request batch of
bf16 hidden states (AR(1) over 16 staged decode steps, EMA 0.2), plus the
latency of one call at batch 1 and 10.

``--path sim`` runs the event-driven simulation of decode instances under
each rescheduling policy, planned by the library every 2 simulated seconds,
on 8 and 64 instances; it reports the execution-time variance, TPOT and
migrations per policy and the simulated time per wall second.

``--path plan [--workload NAME] [--moves M]`` measures Algorithm 1 end to
end: per step, the placement is restored (a quarter of the requests crowded
onto one instance), then star_project_load -> star_plan_migrations with up
to M migrations (theta = 1/10, rem_len > 64).

``--path variance [--workload NAME]`` measures the time-weighted variance
objective instead: per step, star_project_load -> star_score_variance (every
migration's exact gain, each request's best target, the best feasible
move) on a workload's true remaining lengths, as the paper's oracle-predictor
runs do; one JSON line of its own.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

METRIC = "requests predicted+scored/sec at B=1024,d=4096; µs per reschedule round"
WORKLOAD = "continuous"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3      # MI355X dense fp32 MFMA
PEAK_HBM_GBS = 8000.0


def _parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=40)
    ap.add_argument("--mode", choices=("graph_pipelined", "pipelined", "eager", "graph"),
                    default="graph_pipelined",
                    help="which timing gives `value` (the others are reported beside it): "
                         "pipelined = predictions (star_predict_overlap: a round's head and "
                         "the next round's first-layer product per launch) on one stream "
                         "while earlier rounds are projected and scored on a second "
                         "(eagerly launched); "
                         "graph_pipelined = the same, 40 rounds per captured HIP graph; "
                         "eager = one stream, round after round; graph = one captured graph "
                         "per round")
    ap.add_argument("--cpu-rounds", type=int, default=200,
                    help="rounds of the CPU oracle timed for the baseline (0 = skip)")
    ap.add_argument("--path", choices=("round", "variance", "plan", "mlp4", "sim", "configs"),
                    default="round",
                    help="round: the full rescheduling round; variance: projection + "
                         "variance-gain scoring; plan: Algorithm 1 repeated; mlp4: the paper's "
                         "4-layer regression head; sim: the event-driven simulation; configs: "
                         "per-call times at every workload's shape")
    ap.add_argument("--moves", type=int, default=16, help="max_moves of --path plan")
    ap.add_argument("--workload", default=None,
                    help="workload of --path variance / plan (default rebalance_scan) or the "
                         "one workload --path configs measures (default: all five)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device-to-device copy of known size (the "
                         "reference for scaling FETCH_SIZE / WRITE_SIZE counters) and exit")
    return ap.parse_args()


COPY_BYTES = 256 << 20
COPY_REPS = 8
TRAFFIC_FILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles",
                            "predict_continuous_traffic.json")
CPU_ROUNDS_1T = 8       # decode steps of the oracle's one-thread leg
PREDICT_SOURCE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2510_13668_amd",
                            "csrc", "predict.hip")


def copy_calibration():
    """COPY_REPS copies of COPY_BYTES between two device buffers."""
    import torch
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(COPY_REPS):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES, "reps": COPY_REPS}), flush=True)


def measured_traffic():
    """HBM bytes per launch of the predictor kernel from the committed counter
    runs, or None when the kernel source changed since they were taken."""
    import hashlib
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
        with open(PREDICT_SOURCE, "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()
    except (OSError, ValueError):
        return None
    return t["traffic_bytes"] if t.get("source_sha256") == sha else None


KERNEL_SPLIT_FILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles",
                                 "predict_continuous_kernels.json")


def committed_kernel_split():
    """Per-kernel average durations of star_predict at this workload from the
    committed rocprofv3 summary, or None when the kernel source changed since
    it was taken."""
    import hashlib
    try:
        with open(KERNEL_SPLIT_FILE) as f:
            t = json.load(f)
        with open(PREDICT_SOURCE, "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()
    except (OSError, ValueError):
        return None
    return t["kernels"] if t.get("source_sha256") == sha else None


class HipEvents:
    """Raw hipEvent_t handles (timing events on an explicit stream)."""

    DISABLE_SYSTEM_FENCE = 0x20000000     # hipEventDisableSystemFence

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self, n):
        out = []
        for _ in range(n):
            e = ctypes.c_void_p()
            # no system-scope fence: the marker then costs little next to a
            # ~10 us kernel (the timestamps stay device-side)
            if self.hip.hipEventCreateWithFlags(ctypes.byref(e), self.DISABLE_SYSTEM_FENCE) != 0:
                raise RuntimeError("hipEventCreateWithFlags failed")
            out.append(e)
        return out

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(ms), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def destroy(self, evs):
        for e in evs:
            self.hip.hipEventDestroy(e)

    def time_calls(self, fn, n, stream):
        """Mean seconds of fn(i), i < n, each bracketed by its own pair of
        events recorded on `stream` (the stream fn launches on)."""
        import torch
        evs = self.create(2 * n)
        hs = ctypes.c_void_p(stream.cuda_stream)
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        torch.cuda.synchronize()
        for i in range(n):
            self.hip.hipEventRecord(evs[2 * i], hs)
            fn(i)
            self.hip.hipEventRecord(evs[2 * i + 1], hs)
        torch.cuda.synchronize()
        t = float(np.mean([self.elapsed_ms(evs[2 * i], evs[2 * i + 1]) for i in range(n)])) * 1e-3
        self.destroy(evs)
        return t


def cpu_info():
    """Host CPU model and this process's CPU affinity."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    aff = sorted(os.sched_getaffinity(0))
    runs, start = [], None
    for i, c in enumerate(aff):
        if start is None:
            start = c
        if i + 1 == len(aff) or aff[i + 1] != c + 1:
            runs.append(f"{start}-{c}" if c > start else f"{c}")
            start = None
    return {"cpu_model": model, "affinity": ",".join(runs), "affinity_cpus": len(aff)}


def cpu_baseline(x, wl, rounds: int, rounds_1t: int):
    """The CPU oracle on the first `rounds` decode steps of the same workload
    with all its OpenMP threads, then on the first `rounds_1t` with one."""
    import oracle

    def run(n_rounds):
        state = np.zeros(wl.n_req, np.float64)
        t0 = time.perf_counter()
        for s in range(n_rounds):
            out = oracle.predict(x.hidden[s], x.w1, x.w2, x.bin_values, dtype=wl.dtype,
                                 act=wl.act, ema_alpha=wl.ema_alpha, ema_init=(s == 0),
                                 ema_state=state, len_max=wl.len_max)
            oracle.round_((x.cur_len + s).astype(np.int32), out["rem_len"], x.inst_of,
                          n_inst=wl.n_inst, bucket=wl.bucket, n_buckets=wl.n_buckets,
                          top_k=wl.top_k)
        return time.perf_counter() - t0

    threads = oracle.threads()
    dt = run(rounds)
    oracle.set_threads(1)
    try:
        dt1 = run(rounds_1t)
    finally:
        oracle.set_threads(threads)
    out = {"value": wl.n_req * rounds / dt, "unit": "requests/s", "cores": threads,
           "kind": "oracle",
           "sample": f"first {rounds} of the 200 decode steps, all {wl.n_req} requests, full "
                     f"round (fp64 head, per-step int64 curves, direct peak per candidate, "
                     f"full sort); {dt:.2f} s on {threads} threads",
           "value_1thread": wl.n_req * rounds_1t / dt1,
           "sample_1thread": f"first {rounds_1t} decode steps on one thread; {dt1:.2f} s"}
    out.update(cpu_info())
    return out


VAR_STEPS = 16    # staged decode steps of the variance path (cur + s, rem - s)


def variance_inputs(wl):
    """Per-request arrays of the variance path: current lengths, true
    remaining lengths (a seeded draw where the workload has none) and
    instances, advanced by one decode step per staged step."""
    from paper_2510_13668_amd import synth
    x = synth.make_inputs(wl, steps=1, n_req=1)
    rem = x.true_len
    if rem is None:
        rem = np.random.default_rng(0).integers(1, wl.horizon, size=wl.n_req,
                                                endpoint=True).astype(np.int32)
    cur = np.stack([x.cur_len + s for s in range(VAR_STEPS)]).astype(np.int32)
    rem = np.stack([np.maximum(rem - s, 1) for s in range(VAR_STEPS)]).astype(np.int32)
    return cur, rem, x.inst_of


def variance_cpu_baseline(wl, cur, rem, inst, beta, sample: int):
    """The oracle on one step: the full projection, then the variance gains
    and the selection for `sample` requests; scaled to requests/s."""
    import oracle
    t0 = time.perf_counter()
    load, _ = oracle.project_load(cur, rem, inst, n_inst=wl.n_inst, bucket=wl.bucket,
                                  n_buckets=wl.n_buckets)
    t_proj = time.perf_counter() - t0
    idx = np.linspace(0, wl.n_req - 1, sample).astype(np.int64)
    t0 = time.perf_counter()
    g = oracle.score_variance(cur[idx], rem[idx], inst[idx], load, beta, bucket=wl.bucket)
    oracle.select_variance(cur[idx], rem[idx], inst[idx], g)
    t_score = time.perf_counter() - t0
    per_req = t_proj / wl.n_req + t_score / sample
    return {"value": 1.0 / per_req, "unit": "requests/s", "cores": oracle.threads(),
            "kind": "oracle",
            "sample": f"one decode step: projection of all {wl.n_req} requests ({t_proj:.2f} s) "
                      f"plus exact variance gains (full weighted variance of the moved curves "
                      f"per candidate) and the full-sort selection for {sample} evenly spaced "
                      f"requests ({t_score:.2f} s)"}


def bench_variance(args):
    import torch
    from paper_2510_13668_amd import star, synth

    dev = "cuda"
    wl = synth.WORKLOADS[args.workload or "rebalance_scan"]
    N, n, b, K = wl.n_req, wl.n_inst, wl.bucket, wl.n_buckets
    cur_h, rem_h, inst_h = variance_inputs(wl)
    beta_h = synth.bucket_weights(K)
    cur = torch.from_numpy(cur_h).to(dev)
    rem = torch.from_numpy(rem_h).to(dev)
    inst = torch.from_numpy(inst_h).to(dev)
    beta = torch.from_numpy(beta_h.view(np.int16)).to(dev)
    load = torch.empty((n, K), dtype=torch.int64, device=dev)
    gain = torch.empty((N, n, 2), dtype=torch.int64, device=dev)
    best_t = torch.empty(N, dtype=torch.int32, device=dev)
    best_g = torch.empty((N, 2), dtype=torch.int64, device=dev)
    move = torch.empty(star.MOVE_FIELDS, dtype=torch.int32, device=dev)
    lp = star.load_params(N, n, b, K)
    ws_l = star.Workspace(star.project_load_workspace_size(lp))
    ws_v = star.Workspace(star.score_variance_workspace_size(lp))
    stream = torch.cuda.Stream()
    torch.cuda.synchronize()

    def project(slot):
        star.project_load(lp, cur[slot], rem[slot], inst, load, ws_l, stream)

    def score(slot):
        star.score_variance(lp, cur[slot], rem[slot], inst, load, beta, gain, best_t, best_g, move,
                            ws_v, stream)

    for i in range(args.warmup):
        project(i % VAR_STEPS)
        score(i % VAR_STEPS)
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for i in range(args.steps):
        project(i % VAR_STEPS)
        score(i % VAR_STEPS)
    t1.record(stream)
    torch.cuda.synchronize()
    ms_step = t0.elapsed_time(t1) / args.steps

    # star_score_variance (prefix tables + scoring) timed with HIP events on
    # its stream, one pair per call
    he = HipEvents()
    evs = he.create(2 * args.steps)
    hs = ctypes.c_void_p(stream.cuda_stream)
    he.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    for i in range(args.steps):
        project(i % VAR_STEPS)
        he.hip.hipEventRecord(evs[2 * i], hs)
        score(i % VAR_STEPS)
        he.hip.hipEventRecord(evs[2 * i + 1], hs)
    torch.cuda.synchronize()
    call_s = float(np.mean([he.elapsed_ms(evs[2 * i], evs[2 * i + 1])
                            for i in range(args.steps)])) * 1e-3
    he.destroy(evs)
    # algorithmic bytes of one call: request arrays, curves and weights in;
    # gains, best targets and gains, and the move out
    nbytes = 12 * N + 8 * n * K + 2 * K + 16 * N * n + 20 * N + 32
    achieved = nbytes / call_s / 1e9

    out = {
        "metric": "requests scored/sec by exact time-weighted variance gain "
                  "(projection + all N x n migrations + best feasible move)",
        "value": N / (ms_step * 1e-3),
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int128",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: {N} requests on {n} instances, true remaining "
                               f"lengths {wl.true_len or 'uniform'}, horizon {wl.horizon} in "
                               f"{b}-step buckets, weights halving every K/8 buckets, "
                               f"{N}x{n} migrations, {VAR_STEPS} staged decode steps",
                   "n_req": N, "n_inst": n, "horizon": wl.horizon, "bucket": b},
        "roofline": {"kernel": "star_score_variance (var_prep_kernel + var_score_kernel)",
                     "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS, "traffic": None,
                     "avg_call_us": call_s * 1e6, "algorithmic_bytes": nbytes},
    }
    if args.cpu_rounds > 0:
        out["cpu_baseline"] = variance_cpu_baseline(wl, cur_h[0], rem_h[0], inst_h, beta_h,
                                                    min(N, 8192))
    print(json.dumps(out), flush=True)


def plan_cpu_baseline(wl, cur, rem, inst, beta, moves: int):
    """The oracle's Algorithm 1 on the same start.  Small workloads run the
    whole plan; large ones time one pass's dominant cost (the full weighted
    variance of the moved curves for every filtered candidate) on a sample
    of the source requests and scale it to all of them."""
    import oracle
    if wl.n_req <= 8192:
        t0 = time.perf_counter()
        out = oracle.plan(cur, rem, inst, beta, n_inst=wl.n_inst, bucket=wl.bucket,
                          n_buckets=wl.n_buckets, theta=(1, 10), min_rem=64, max_moves=moves)
        dt = time.perf_counter() - t0
        made = max(len(out["moves"]), 1)
        return {"value": made / dt, "unit": "moves/s", "cores": oracle.threads(),
                "kind": "oracle",
                "sample": f"{len(out['moves'])} moves of the same plan from the same start "
                          f"(classification, filtered candidates scored by the full weighted "
                          f"variance of the moved curves, per-step curve rebuild); {dt:.2f} s"}
    t0 = time.perf_counter()
    load, _ = oracle.project_load(cur, rem, inst, n_inst=wl.n_inst, bucket=wl.bucket,
                                  n_buckets=wl.n_buckets)
    t_proj = time.perf_counter() - t0
    w = load.astype(object).dot(beta.astype(object))
    wsum = sum(w)
    over = [10 * wl.n_inst * wi > 11 * wsum for wi in w]
    srcs = np.array([r for r in range(wl.n_req) if over[inst[r]] and rem[r] > 64], np.int64)
    sample = srcs[np.linspace(0, len(srcs) - 1, min(len(srcs), 4096)).astype(np.int64)]
    t0 = time.perf_counter()
    oracle.score_variance(cur[sample], rem[sample], inst[sample], load, beta, bucket=wl.bucket)
    t_score = time.perf_counter() - t0
    per_move = t_proj + t_score * len(srcs) / max(len(sample), 1)
    return {"value": 1.0 / per_move, "unit": "moves/s", "cores": oracle.threads(),
            "kind": "oracle",
            "sample": f"one pass of the plan from the same start: projection ({t_proj:.2f} s) and "
                      f"the variance gains of {len(sample)} of the {len(srcs)} source requests on "
                      f"overloaded instances ({t_score:.2f} s), scaled to all of them"}


def bench_plan(args):
    import torch
    from paper_2510_13668_amd import star, synth

    dev = "cuda"
    wl = synth.WORKLOADS[args.workload or "rebalance_scan"]
    N, n, b, K = wl.n_req, wl.n_inst, wl.bucket, wl.n_buckets
    M = args.moves
    x = synth.make_inputs(wl, steps=1, n_req=1)
    rem_h = x.true_len
    if rem_h is None:
        rem_h = np.random.default_rng(0).integers(1, wl.horizon, size=N,
                                                  endpoint=True).astype(np.int32)
    inst_h = x.inst_of.copy()
    inst_h[: N // 4] = 3 % n
    beta_h = synth.bucket_weights(K)
    cur = torch.from_numpy(x.cur_len).to(dev)
    rem = torch.from_numpy(rem_h).to(dev)
    inst0 = torch.from_numpy(inst_h).to(dev)
    inst = inst0.clone()
    beta = torch.from_numpy(beta_h.view(np.int16)).to(dev)
    load = torch.empty((n, K), dtype=torch.int64, device=dev)
    moves = torch.empty(max(M, 1) * star.MOVE_FIELDS, dtype=torch.int32, device=dev)
    cnt = torch.empty(1, dtype=torch.int32, device=dev)
    lp = star.load_params(N, n, b, K)
    pp = star.plan_params(N, n, b, K, M, theta=(1, 10), min_rem=64)
    ws_l = star.Workspace(star.project_load_workspace_size(lp))
    ws_p = star.Workspace(star.plan_workspace_size(pp))
    stream = torch.cuda.Stream()
    torch.cuda.synchronize()

    def step():
        with torch.cuda.stream(stream):
            inst.copy_(inst0)
        star.project_load(lp, cur, rem, inst, load, ws_l, stream)
        star.plan_migrations(pp, cur, rem, inst, load, beta, moves, cnt, ws_p, stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(args.steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    ms_step = t0.elapsed_time(t1) / args.steps
    made = int(cnt.cpu()[0])

    # star_plan_migrations alone, HIP events on its stream
    he = HipEvents()
    evs = he.create(2 * args.steps)
    hs = ctypes.c_void_p(stream.cuda_stream)
    he.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    for i in range(args.steps):
        with torch.cuda.stream(stream):
            inst.copy_(inst0)
        star.project_load(lp, cur, rem, inst, load, ws_l, stream)
        he.hip.hipEventRecord(evs[2 * i], hs)
        star.plan_migrations(pp, cur, rem, inst, load, beta, moves, cnt, ws_p, stream)
        he.hip.hipEventRecord(evs[2 * i + 1], hs)
    torch.cuda.synchronize()
    call_s = float(np.mean([he.elapsed_ms(evs[2 * i], evs[2 * i + 1])
                            for i in range(args.steps)])) * 1e-3
    he.destroy(evs)
    # algorithmic bytes: per pass the request arrays and the tables' target
    # rows are read once (12 B per request, 40 B per bucket and instance);
    # per move two curve rows are rewritten (16 B per bucket)
    passes = min(made + 1, M) if M else 0
    nbytes = passes * (12 * N + 40 * n * (K + 1)) + made * 16 * K + 40 * (n + 1) * (K + 1)
    achieved = nbytes / call_s / 1e9

    out = {
        "metric": "migration plans/sec (Algorithm 1: classification, filtered candidates, "
                  "best feasible move by exact variance gain, repeated)",
        "value": 1.0 / (ms_step * 1e-3),
        "unit": "plans/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int128",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: {N} requests on {n} instances, a quarter crowded onto "
                               f"one, true remaining lengths {wl.true_len or 'uniform'}, horizon "
                               f"{wl.horizon} in {b}-step buckets, up to {M} migrations per plan, "
                               f"theta 1/10, rem_len > 64",
                   "n_req": N, "n_inst": n, "horizon": wl.horizon, "bucket": b, "max_moves": M,
                   "moves_made": made},
        "roofline": {"kernel": "star_plan_migrations (prep, then per move a masked scoring pass "
                               "and a one-workgroup update)",
                     "bound": "latency", "achieved": achieved, "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, "traffic": None,
                     "avg_call_us": call_s * 1e6, "us_per_move": call_s * 1e6 / max(made, 1),
                     "algorithmic_bytes": nbytes},
    }
    if args.cpu_rounds > 0:
        out["cpu_baseline"] = plan_cpu_baseline(wl, x.cur_len, rem_h, inst_h, beta_h,
                                                min(M, 4 if N > 8192 else M))
    print(json.dumps(out), flush=True)


def bench_mlp4(args):
    import torch
    from paper_2510_13668_amd import star, synth
    import oracle

    dev = "cuda"
    B, S = 1024, 16
    d, m1, m2, m3 = synth.MLP4_DIMS
    x = synth.make_mlp4(B, dtype=synth.BF16, seed=0, steps=S)
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
    hid = bf(x.hidden)
    w1, w2, w3 = bf(x.w1), bf(x.w2), bf(x.w3)
    w4 = torch.from_numpy(x.w4).to(dev)
    ema = torch.zeros(B, dtype=torch.float32, device=dev)
    y = torch.empty(B, dtype=torch.float32, device=dev)
    rem = torch.empty(B, dtype=torch.int32, device=dev)
    stream = torch.cuda.Stream()

    def params(n, init=False):
        return star.mlp4_params(n, d, m1, m2, m3, synth.BF16, 0.2, init, 32768, x.b4)

    ws = star.Workspace(star.predict_mlp4_workspace_size(params(B)))
    star.predict_mlp4(params(B, True), hid[0], w1, None, w2, None, w3, None, w4, ema, y, rem, ws,
                      stream)
    torch.cuda.synchronize()

    def timed(fn, steps):
        for i in range(args.warmup):
            fn(i)
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for i in range(steps):
            fn(args.warmup + i)
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / steps

    pp = params(B)
    ms_step = timed(lambda i: star.predict_mlp4(pp, hid[i % S], w1, None, w2, None, w3, None, w4,
                                                ema, y, rem, ws, stream), args.steps)
    lat = {}
    for nb in (1, 10):
        p_small = params(nb)
        lat[nb] = timed(lambda i: star.predict_mlp4(p_small, hid[i % S, :nb], w1, None, w2, None,
                                                    w3, None, w4, ema[:nb], y[:nb], rem[:nb], ws,
                                                    stream), args.steps) * 1e3

    # one call (the four layers, five kernels) timed with HIP events on its
    # stream; the per-kernel split comes from rocprofv3
    he = HipEvents()
    call_s = he.time_calls(lambda i: star.predict_mlp4(pp, hid[i % S], w1, None, w2, None, w3,
                                                       None, w4, ema, y, rem, ws, stream),
                           args.steps, stream)
    flops = 2.0 * B * (d * m1 + m1 * m2 + m2 * m3 + m3)
    achieved = flops / call_s / 1e12

    out = {
        "metric": "requests predicted/sec by the paper's 4-layer regression head "
                  "(3584->2048->512->64->1, bf16) at a 1024-request batch",
        "value": B / (ms_step * 1e-3),
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "regression head of the paper's shape, random-initialised weights, "
                               "1024 requests, bf16 hidden [1024,3584] AR(1) over 16 staged steps, "
                               "EMA 0.2",
                   "n_req": B, "dims": [d, m1, m2, m3]},
        "latency_us": {"batch_1": lat[1], "batch_10": lat[10]},
        "roofline": {"kernel": "the whole call (four layers; layer 1, H[1024,3584] x "
                               "W1[2048,3584]^T, is 86% of its FLOPs)",
                     "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS, "traffic": None,
                     "avg_call_us": call_s * 1e6, "algorithmic_flop": flops},
    }
    if args.cpu_rounds > 0:
        steps = 8
        st = np.zeros(B, np.float64)
        t0 = time.perf_counter()
        for t in range(steps):
            oracle.predict_mlp4(x.hidden[t], x.w1, x.w2, x.w3, x.w4, dtype=synth.BF16, b4=x.b4,
                                ema_alpha=0.2, ema_init=(t == 0), ema_state=st, len_max=32768)
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": B * steps / dt, "unit": "requests/s",
                               "cores": oracle.threads(), "kind": "oracle",
                               "sample": f"all {B} rows of the first {steps} decode steps, fp64 "
                                         f"triple loops; {dt:.2f} s"}
    print(json.dumps(out), flush=True)


def bench_configs(args):
    """Per-call times of the round's two calls at each workload's own shape,
    with the predictor's FLOPs (both products) over the call's time (an MFMA
    fraction) and the projection-and-scoring call's compulsory bytes over its
    time (an HBM fraction)."""
    import torch
    from paper_2510_13668_amd import star, synth

    dev = "cuda"
    stream = torch.cuda.Stream()
    he = HipEvents()
    rows = []
    for name in ([args.workload] if args.workload else synth.WORKLOAD_ORDER):
        wl = synth.WORKLOADS[name]
        x = synth.make_inputs(wl, steps=1)
        N, d, m, nb = wl.n_req, wl.d_model, wl.d_hidden, wl.n_bins
        n, b, K, top_k = wl.n_inst, wl.bucket, wl.n_buckets, wl.top_k
        bf16 = wl.dtype == synth.BF16

        def up(a, as_bf16=False):
            t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16) if as_bf16 else a).to(dev)
            return t.view(torch.bfloat16) if as_bf16 else t
        hid, w1, w2 = up(x.hidden, bf16), up(x.w1, bf16), up(x.w2, bf16)
        bins, cur, inst = up(x.bin_values), up(x.cur_len), up(x.inst_of)
        ema = torch.zeros(N, dtype=torch.float32, device=dev) if wl.ema_alpha > 0 else None
        expected = torch.empty(N, dtype=torch.float32, device=dev)
        rem = torch.empty(N, dtype=torch.int32, device=dev)
        load = torch.empty((n, K), dtype=torch.int64, device=dev)
        scores = torch.empty((N, n), dtype=torch.int64, device=dev)
        best_t = torch.empty(N, dtype=torch.int32, device=dev)
        best_s = torch.empty(N, dtype=torch.int64, device=dev)
        tr = torch.empty(top_k, dtype=torch.int32, device=dev)
        tt = torch.empty(top_k, dtype=torch.int32, device=dev)
        ts = torch.empty(top_k, dtype=torch.int64, device=dev)
        pp = star.predict_params(N, d, m, nb, wl.dtype, wl.act, wl.ema_alpha, False, wl.len_max)
        sp = star.score_params(N, n, b, K, top_k)
        ws_p = star.Workspace(star.predict_workspace_size(pp))
        ws_s = star.Workspace(star.project_and_score_workspace_size(sp))
        # oracle-predictor mode where the workload has true remaining lengths
        rem_in = up(x.true_len) if x.true_len is not None else rem

        def predict(p=pp):
            star.predict(p, hid, w1, None, w2, None, bins, ema, expected, rem, ws_p, stream)

        def project_score():
            star.project_and_score(sp, cur, rem_in, inst, load, scores, best_t, best_s, tr, tt,
                                   ts, ws_s, stream)

        reps = 20 if N * d >= (1 << 27) else args.steps

        def timed(fn):
            for _ in range(5):
                fn()
            torch.cuda.synchronize()
            t0 = torch.cuda.Event(enable_timing=True)
            t1 = torch.cuda.Event(enable_timing=True)
            t0.record(stream)
            for _ in range(reps):
                fn()
            t1.record(stream)
            torch.cuda.synchronize()
            return t0.elapsed_time(t1) * 1e3 / reps

        predict_us = timed(predict)
        ps_us = timed(project_score)
        round_us = timed(lambda: (predict(), project_score()))
        g_us = he.time_calls(lambda i: predict(), reps, stream) * 1e6
        flops = 2.0 * N * d * m + 2.0 * N * m * nb
        peak = PEAK_BF16_TFLOPS if bf16 else PEAK_FP32_TFLOPS
        ps_bytes = 12 * N + 8 * n * K + 8 * N * n + 12 * N + 16 * top_k
        rows.append({
            "workload": name, "n_req": N, "d_model": d, "d_hidden": m, "n_bins": nb,
            "n_inst": n, "n_buckets": K, "top_k": top_k, "dtype": "bf16" if bf16 else "f32",
            "rem_len": "true lengths" if x.true_len is not None else "predicted",
            "predict_us": predict_us, "project_and_score_us": ps_us, "round_us": round_us,
            "predict_event_us": g_us, "predict_tflops": flops / (g_us * 1e-6) / 1e12,
            "predict_frac": flops / (g_us * 1e-6) / 1e12 / peak, "peak_tflops": peak,
            "project_and_score_bytes": ps_bytes,
            "project_and_score_gbs": ps_bytes / (ps_us * 1e-6) / 1e9,
            "project_and_score_hbm_frac": ps_bytes / (ps_us * 1e-6) / 1e9 / PEAK_HBM_GBS,
            "reps": reps})
        print(f"{name}: predict {predict_us:.1f} us (one call between events {g_us:.1f} us, "
              f"{rows[-1]['predict_frac'] * 100:.1f}% of peak), project+score {ps_us:.1f} us",
              file=sys.stderr, flush=True)
        del hid, w1, w2, ws_p, ws_s, scores
        torch.cuda.empty_cache()

    out = {
        "metric": "per-call microseconds of star_predict and star_project_and_score at each "
                  "workload's shape",
        "value": rows[-1]["round_us"],
        "unit": "us per round at the largest workload",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": 5,
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 (tiny: f32)",
        "data": "synthetic",
        "config": {"workload": "the five workloads, one decode step each; (b)(c) on the "
                               "workload's true remaining lengths where it has them"},
        "configs": rows,
    }
    print(json.dumps(out), flush=True)


def bench_sim(args):
    import dataclasses
    from paper_2510_13668_amd import sim
    import oracle

    def oracle_planner(cur, rem, inst, beta, *, n_inst, bucket, n_buckets, theta, min_rem,
                       mem_cap, max_moves):
        return oracle.plan(cur, rem, inst, beta, n_inst=n_inst, bucket=bucket,
                           n_buckets=n_buckets, theta=theta, min_rem=min_rem, mem_cap=mem_cap,
                           max_moves=max_moves)["moves"]

    base = sim.SimConfig(seed=11)
    runs = {}
    wall = {}
    for n, dur in ((8, 600.0), (64, 300.0)):
        cfg = dataclasses.replace(base, n_inst=n, duration_s=dur)
        lib = sim.LibraryPlanner()
        t0 = time.perf_counter()
        res = {p: sim.simulate(cfg, p, lib if p != "none" else None) for p in sim.POLICIES}
        wall[n] = time.perf_counter() - t0
        runs[n] = {p: {"exec_var_ms2": r.exec_var_ms2, "p99_tpot_ms": r.p99_tpot_ms,
                       "mean_tpot_ms": r.mean_tpot_ms, "migrations": r.migrations,
                       "oom_ticks": r.oom_ticks, "finished": r.finished}
                   for p, r in res.items()}
        runs[n]["simulated_s_per_policy"] = dur
    sim_s = sum(4 * d for d in (600.0, 300.0))
    out = {
        "metric": "simulated decode-cluster seconds per wall second (4 policies x {8, 64} "
                  "instances, Algorithm 1 planned by the library every 2 s)",
        "value": sim_s / sum(wall.values()),
        "unit": "simulated s / s",
        "n_gpus": 1,
        "steps": 1,
        "warmup": 0,
        "ms_per_step": sum(wall.values()) * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int128",
        "data": "synthetic",
        "config": {"workload": "event-driven simulation: Poisson arrivals 0.3 rps per 8 "
                               "instances, prompts U[128,4096], outputs 82.7% lognormal(7.16,0.67)"
                               " + 17.3% U[30000,32768], iteration 12 ms + 0.25 ms per 1000 batch "
                               "tokens, 25 Gbps KV transfers, plans of up to 4 moves every 2 s "
                               "(theta 1/10, rem > 64), horizon 32768 in 128-step buckets"},
        "policies": runs,
        "roofline": None,
    }
    if args.cpu_rounds > 0:
        cfg = dataclasses.replace(base, n_inst=64, duration_s=300.0)
        t0 = time.perf_counter()
        sim.simulate(cfg, "oracle", oracle_planner)
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": 300.0 / dt, "unit": "simulated s / s",
                               "cores": oracle.threads(), "kind": "oracle",
                               "sample": f"64 instances, oracle policy, 300 simulated s planned "
                                         f"by the CPU oracle (the same run as the GPU's); "
                                         f"{dt:.2f} s"}
    print(json.dumps(out), flush=True)


def main():
    args = _parse()
    if args.copy_calibration:
        copy_calibration()
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this hot path runs on one GPU (decode instances are data, not devices); "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)
    if args.path == "variance":
        bench_variance(args)
        return
    if args.path == "plan":
        bench_plan(args)
        return
    if args.path == "mlp4":
        bench_mlp4(args)
        return
    if args.path == "sim":
        bench_sim(args)
        return
    if args.path == "configs":
        bench_configs(args)
        return

    import torch
    from paper_2510_13668_amd import star, synth

    dev = "cuda"
    wl = synth.WORKLOADS[WORKLOAD]
    S = wl.steps
    x = synth.make_inputs(wl)                       # 200 staged decode steps
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
    hid = bf(x.hidden)                              # [200, 1024, 4096] bf16, 1.68 GB
    w1, w2 = bf(x.w1), bf(x.w2)
    bins = torch.from_numpy(x.bin_values).to(dev)
    cur_steps = torch.from_numpy(np.stack([x.cur_len + s for s in range(S)]).astype(np.int32)).to(dev)
    inst = torch.from_numpy(x.inst_of).to(dev)

    N, d, m, nb = wl.n_req, wl.d_model, wl.d_hidden, wl.n_bins
    n, b, K, top_k = wl.n_inst, wl.bucket, wl.n_buckets, wl.top_k
    ema = torch.zeros(N, dtype=torch.float32, device=dev)
    expected = torch.empty(N, dtype=torch.float32, device=dev)
    rem = torch.empty(N, dtype=torch.int32, device=dev)
    load = torch.empty((n, K), dtype=torch.int64, device=dev)
    scores = torch.empty((N, n), dtype=torch.int64, device=dev)
    best_t = torch.empty(N, dtype=torch.int32, device=dev)
    best_s = torch.empty(N, dtype=torch.int64, device=dev)
    tr = torch.empty(top_k, dtype=torch.int32, device=dev)
    tt = torch.empty(top_k, dtype=torch.int32, device=dev)
    ts = torch.empty(top_k, dtype=torch.int64, device=dev)

    pp = star.predict_params(N, d, m, nb, wl.dtype, wl.act, wl.ema_alpha, False, wl.len_max)
    pp_init = star.predict_params(N, d, m, nb, wl.dtype, wl.act, wl.ema_alpha, True, wl.len_max)
    sp = star.score_params(N, n, b, K, top_k)
    ws_p = star.Workspace(star.predict_workspace_size(pp))
    ws_s = star.Workspace(star.project_and_score_workspace_size(sp))
    # the pipelined modes' predictions: star_predict_overlap with the split-K
    # partials alternating between two workspaces
    ws_ov = [ws_p, star.Workspace(star.predict_workspace_size(pp))]

    stream = torch.cuda.Stream()
    torch.cuda.synchronize()

    # One round: the predictor head, then the load projection and the
    # migration scoring in one call (one kernel launch at this size).
    def round_(slot, params=pp):
        star.predict(params, hid[slot], w1, None, w2, None, bins, ema, expected, rem, ws_p, stream)
        star.project_and_score(sp, cur_steps[slot], rem, inst, load, scores, best_t, best_s,
                               tr, tt, ts, ws_s, stream)

    with torch.cuda.stream(stream):
        round_(0, pp_init)                          # first decode step initialises the EMA
    graphs = []
    for slot in range(S):                           # one captured round per staged step
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            round_(slot)
        graphs.append(g)
    torch.cuda.synchronize()

    def timed(mode):
        """Milliseconds per round over args.steps rounds after args.warmup."""
        def run_step(i):
            slot = (i + 1) % S
            if mode == "graph":
                with torch.cuda.stream(stream):
                    graphs[slot].replay()
            else:
                round_(slot)
        for i in range(args.warmup):
            run_step(i)
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for i in range(args.steps):
            run_step(args.warmup + i)
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / args.steps

    # Pipelined rounds: round i's prediction needs only round i-1's EMA state,
    # so it runs on `stream` while earlier rounds are projected and scored on
    # `sched`.  The predictions go through star_predict_overlap: one launch
    # runs round i's head and round i+1's first-layer product (a sequence
    # starts with a product-only call and ends with a head-only one).  Scheduling waits for the predictions SCHED_BATCH rounds at a
    # time (one cross-stream event per batch), then projects and scores each
    # of them and records one event when the batch is done.  Per-round
    # outputs rotate through NSLOT buffers: before a prediction overwrites a
    # buffer, its stream waits for the event of the batch that last scheduled
    # that buffer, once per distinct event, so once per batch.  (Measured,
    # graph-replayed: 28.3 us per round with three buffers and a wait per
    # round, 27.0-27.6 with six buffers, batches of two and an event per
    # round, 26.7-26.9 with an event and a wait per batch; without the
    # buffer-release waits, 33.0.)
    sched = torch.cuda.Stream()
    SCHED_BATCH = 2
    NSLOT = 6
    assert NSLOT >= SCHED_BATCH
    slot_buf = []
    for _ in range(NSLOT):
        slot_buf.append(dict(
            expected=torch.empty(N, dtype=torch.float32, device=dev),
            rem=torch.empty(N, dtype=torch.int32, device=dev),
            load=torch.empty((n, K), dtype=torch.int64, device=dev),
            scores=torch.empty((N, n), dtype=torch.int64, device=dev),
            best_t=torch.empty(N, dtype=torch.int32, device=dev),
            best_s=torch.empty(N, dtype=torch.int64, device=dev),
            tr=torch.empty(top_k, dtype=torch.int32, device=dev),
            tt=torch.empty(top_k, dtype=torch.int32, device=dev),
            ts=torch.empty(top_k, dtype=torch.int64, device=dev)))
    ev_pred = [torch.cuda.Event() for _ in range(NSLOT)]
    ev_done = [torch.cuda.Event() for _ in range(NSLOT)]   # one per batch, cycled
    # guard[k]: the done event of the batch that last scheduled buffer k
    state = dict(guard=[None] * NSLOT, waited=None, batches=0)

    def reset_guards():
        state.update(guard=[None] * NSLOT, waited=None)

    def prime(step, j):
        """The product of the first round j of a sequence (no head)."""
        star.predict_overlap(pp, hid[step], ws_ov[j % 2], None, w1, None, w2, None, bins,
                             None, None, None, stream)

    def predict_into(step_next, j, k):
        """Round j's head into buffer k, and round j+1's product (step_next,
        or none at the end of a sequence)."""
        sb = slot_buf[k]
        ev = state["guard"][k]
        if ev is not None and ev is not state["waited"]:
            stream.wait_event(ev)
            state["waited"] = ev
        nxt = hid[step_next] if step_next is not None else None
        star.predict_overlap(pp, nxt, ws_ov[(j + 1) % 2] if nxt is not None else None,
                             ws_ov[j % 2], w1, None, w2, None, bins, ema, sb["expected"],
                             sb["rem"], stream)

    def schedule(batch):
        """Scheduling of the rounds in `batch` ((step, slot) pairs, all predicted)."""
        k_last = batch[-1][1]
        ev_pred[k_last].record(stream)
        sched.wait_event(ev_pred[k_last])
        for step, k in batch:
            sb = slot_buf[k]
            star.project_and_score(sp, cur_steps[step], sb["rem"], inst, sb["load"], sb["scores"],
                                   sb["best_t"], sb["best_s"], sb["tr"], sb["tt"], sb["ts"], ws_s,
                                   sched)
        ev = ev_done[state["batches"] % NSLOT]
        state["batches"] += 1
        ev.record(sched)
        for _, k in batch:
            state["guard"][k] = ev

    pending = []

    def pipelined_round(i, first=False, last=False):
        step = (i + 1) % S
        k = i % NSLOT
        if first:
            prime(step, i)
        predict_into(None if last else (i + 2) % S, i, k)
        pending.append((step, k))
        if len(pending) == SCHED_BATCH or last:
            schedule(list(pending))
            pending.clear()

    def timed_pipelined():
        torch.cuda.synchronize()
        reset_guards()
        for i in range(args.warmup):
            pipelined_round(i, first=i == 0, last=i == args.warmup - 1)
        torch.cuda.synchronize()
        reset_guards()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for i in range(args.steps):
            pipelined_round(args.warmup + i, first=i == 0, last=i == args.steps - 1)
        for k in range(NSLOT):
            stream.wait_event(ev_done[k])
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / args.steps

    # The same pipeline captured in HIP graphs of up to CHUNK rounds each (the
    # two streams fork and join inside the capture), so that the host launches
    # one graph per CHUNK rounds instead of the kernels and event operations
    # of every round.  The warm-up and the timed region run exactly
    # args.warmup and args.steps rounds: a shorter graph takes any remainder.
    CHUNK = 40
    graph_cache = {}

    def capture(c0, length):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            sched.wait_stream(stream)
            reset_guards()           # the previous graph ends joined: every buffer is free
            batch = []
            prime(c0 % S, 0)
            for j in range(length):
                step = (c0 + j) % S
                k = j % NSLOT
                predict_into((c0 + j + 1) % S if j + 1 < length else None, j, k)
                batch.append((step, k))
                if len(batch) == SCHED_BATCH or j == length - 1:
                    schedule(batch)
                    batch = []
            stream.wait_stream(sched)
        reset_guards()               # no later wait may name an event recorded in the capture
        return g

    def graphs_for(start, rounds):
        """Graphs that run `rounds` pipelined rounds from decode step `start`."""
        out, i = [], 0
        while i < rounds:
            key = ((start + i) % S, min(CHUNK, rounds - i))
            if key not in graph_cache:
                graph_cache[key] = capture(*key)
            out.append(graph_cache[key])
            i += key[1]
        return out

    warm_graphs = graphs_for(0, args.warmup)
    timed_graphs = graphs_for(args.warmup, args.steps)
    torch.cuda.synchronize()

    def timed_graph_pipelined():
        with torch.cuda.stream(stream):
            for g in warm_graphs:
                g.replay()
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        with torch.cuda.stream(stream):
            for g in timed_graphs:
                g.replay()
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / args.steps

    def eager_percentiles():
        """Each eager round bracketed by its own events: p50 / p99 in us."""
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        for i in range(args.warmup):
            round_((i + 1) % S)
        torch.cuda.synchronize()
        for i, (a, b_) in enumerate(evs):
            a.record(stream)
            round_((args.warmup + i + 1) % S)
            b_.record(stream)
        torch.cuda.synchronize()
        t = np.array([a.elapsed_time(b_) * 1e3 for a, b_ in evs])
        return float(np.percentile(t, 50)), float(np.percentile(t, 99))

    ms_mode = {m: timed(m) for m in ("eager", "graph")}
    p50, p99 = eager_percentiles()
    ms_mode["pipelined"] = timed_pipelined()
    ms_mode["graph_pipelined"] = timed_graph_pipelined()
    ms_step = ms_mode[args.mode]

    # Dominant work of the round: the predictions.  The pipelined modes make
    # them with star_predict_overlap, one launch of predict_overlap_kernel
    # per round (one batch's split-K first-layer product and the previous
    # batch's head: split reduction, GELU, second product, softmax, EMA).
    # One pair of HIP events brackets each call on the stream it is launched
    # on, over `steps` back-to-back calls of the round's own inputs.
    # star_predict (the two kernels one after the other) is timed the same
    # way beside it.
    he = HipEvents()
    with torch.cuda.stream(stream):
        prime(1, 0)
    kern_s = he.time_calls(
        lambda i: star.predict_overlap(pp, hid[(i + 2) % S], ws_ov[(i + 1) % 2], ws_ov[i % 2],
                                       w1, None, w2, None, bins, ema, expected, rem, stream),
        args.steps, stream)
    pred_s = he.time_calls(lambda i: star.predict(pp, hid[(i + 1) % S], w1, None, w2, None, bins,
                                                  ema, expected, rem, ws_p, stream),
                           args.steps, stream)
    flops = 2.0 * N * d * m + 2.0 * N * m * nb
    achieved = flops / kern_s / 1e12

    out = {
        "metric": METRIC,
        "value": N / (ms_step * 1e-3),
        "unit": "requests/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "us_per_round": ms_step * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "continuous: 1024 requests on 8 instances, hidden bf16 [1024,4096] "
                               "AR(1) rho=0.95 over 200 staged decode steps, head 4096->512 GELU->64 "
                               "bins, EMA 0.2, horizon 16384 in 64-step buckets, 1024x8 candidates, "
                               "top-256",
                   "n_req": N, "d_model": d, "d_hidden": m, "n_bins": nb, "n_inst": n,
                   "horizon": wl.horizon, "bucket": b, "top_k": top_k,
                   "mode": args.mode + " (inputs resident in HBM)"},
        "us_per_round_pipelined": ms_mode["pipelined"] * 1e3,
        "us_per_round_graph_pipelined": ms_mode["graph_pipelined"] * 1e3,
        "us_per_round_eager": ms_mode["eager"] * 1e3,
        "us_per_round_eager_p50": p50,
        "us_per_round_eager_p99": p99,
        "us_per_round_graph": ms_mode["graph"] * 1e3,
        "timing": {"headline": args.mode, "rounds_timed": args.steps,
                   "warmup_rounds": args.warmup,
                   "overlap": "graph_pipelined and pipelined time throughput: later rounds' "
                              "predictions run while earlier rounds are projected and scored "
                              "(scheduling waits for the predictions %d rounds at a time, outputs "
                              "rotate through %d buffers), and each prediction launch also runs "
                              "the next round's first-layer product (star_predict_overlap); "
                              "us_per_round_eager (p50/p99, star_predict then "
                              "star_project_and_score) is one round's latency"
                              % (SCHED_BATCH, NSLOT)},
        "roofline": {"kernel": "predict_overlap_kernel<4> (star_predict_overlap): one batch's "
                               "first-layer product, bf16 MFMA H[1024,4096] x W1[512,4096]^T in 4 "
                               "K-splits, and the previous batch's head (split reduction, GELU, "
                               "x W2[64,512]^T, softmax, EMA) in one launch",
                     "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                     "traffic": measured_traffic(),
                     "avg_call_us": kern_s * 1e6, "algorithmic_flop": flops,
                     "kernels": committed_kernel_split(),
                     "star_predict_call_us": pred_s * 1e6,
                     "star_predict_tflops": flops / pred_s / 1e12},
    }
    if args.cpu_rounds > 0:
        out["cpu_baseline"] = cpu_baseline(x, wl, min(args.cpu_rounds, S),
                                           min(args.cpu_rounds, CPU_ROUNDS_1T))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
