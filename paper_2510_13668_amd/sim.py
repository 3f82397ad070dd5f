"""Event-driven simulation of decode instances under STAR rescheduling.

Evaluation, large-scale simulation (Section 6): requests arrive at a fixed
rate, every decode instance runs iterations whose duration grows with the
tokens in its batch, and a scheduler periodically reschedules with
Algorithm 1.  A migrated request pauses for its KV-cache transfer, its KV
bytes over the link bandwidth (25 Gbps in the paper).  Here:

* Arrivals are a Poisson process, 0.3 requests/s per 8 instances by
  default.  Prompt lengths are uniform; output lengths follow the published
  shape of the paper's ShareGPT outputs (Section 2.2: many short, about a
  sixth near the 32K cap) as a seeded synthetic draw; the dataset is not
  used.
* New requests join the instance with the fewest tokens (ties: lowest
  index).
* One iteration of instance i takes iter_base_ms + iter_per_ktoken_ms * N_i
  / 1000 ms, where N_i is its current token count.  Each running request
  gains one token per iteration and leaves after its true output length.
* Every `interval_s` of simulated time the scheduler plans up to `max_moves`
  migrations.  The planner is a callable taking (cur_len, rem_len, inst_of,
  beta, n_inst, bucket, n_buckets, params).  It returns the moves (r, s, t)
  in order; in the library's case that is star_project_load followed by
  star_plan_migrations.
* Policies, as in Section 6:
  - "none": no rescheduling;
  - "current": Algorithm 1 on current loads only (one one-step bucket,
    every remaining length set to 1), like STAR without prediction;
  - "predicted": remaining lengths from a noisy predictor (true remaining
    times a lognormal factor, fixed per request);
  - "oracle": the true remaining lengths.
* Metrics:
  - the time-averaged variance, across instances, of the iteration time
    (Exec. Var.), sampled at every scheduling tick;
  - P99 over requests of the mean time per output token (TPOT);
  - migrations;
  - ticks on which some instance's KV tokens exceed its memory capacity
    (OOM ticks).

Everything is deterministic for a seed.  Given identical planners, two runs
are identical event for event; the tests use that to compare the library
with the oracle.
"""
from __future__ import annotations

import dataclasses
import heapq
from typing import Callable, List, Optional, Sequence, Tuple

import numpy as np

from . import synth

Move = Tuple[int, int, int]
Planner = Callable[..., Sequence[Move]]

POLICIES = ("none", "current", "predicted", "oracle")


@dataclasses.dataclass
class SimConfig:
    n_inst: int = 8
    rate_per_8: float = 0.3           # arrivals per second per 8 instances
    duration_s: float = 600.0
    iter_base_ms: float = 12.0
    iter_per_ktoken_ms: float = 0.25  # iteration time per 1000 tokens in the batch
    kv_bytes_per_token: int = 57344   # 28 layers x 2 x 4 KV heads x 128 x bf16 (7B class)
    link_gbps: float = 25.0
    interval_s: float = 2.0
    max_moves: int = 4
    theta: Tuple[int, int] = (1, 10)
    min_rem: int = 64
    mem_cap_tokens: int = 600_000     # KV capacity of one instance, in tokens
    bucket: int = 128
    n_buckets: int = 256              # horizon 32768 steps
    beta_halvings: float = 8.0
    prompt_lo: int = 128
    prompt_hi: int = 4096
    out_law: str = "long_output_stress"   # a synth length law (ShareGPT-like stand-in)
    out_cap: int = 32768
    pred_sigma: float = 0.5           # "predicted": lognormal error of the predictor
    seed: int = 0


@dataclasses.dataclass
class SimResult:
    policy: str
    exec_var_ms2: float
    p99_tpot_ms: float
    mean_tpot_ms: float
    migrations: int
    oom_ticks: int
    finished: int
    ticks: int
    moves: List[Tuple[float, int, int, int]]   # (time, request id, source, target)


def bucket_weights(n_buckets: int, halvings: float) -> np.ndarray:
    k = np.arange(n_buckets, dtype=np.float64)
    w = np.rint(65535.0 * np.exp2(-halvings * k / max(n_buckets, 1)))
    return np.maximum(w, 1.0).astype(np.uint16)


class _Req:
    __slots__ = ("rid", "cur", "left", "pred_factor", "inst", "epoch", "tokens", "busy_ms")

    def __init__(self, rid, cur, left, pred_factor):
        self.rid = rid
        self.cur = cur            # tokens held (prompt + generated)
        self.left = left          # true remaining output tokens
        self.pred_factor = pred_factor
        self.inst = -1            # instance, or the target while in transfer
        self.epoch = 0            # bumped on every placement
        self.tokens = 0           # output tokens generated
        self.busy_ms = 0.0        # decode and transfer time spent on them


def simulate(cfg: SimConfig, policy: str, planner: Optional[Planner]) -> SimResult:
    """Run one simulation; `planner` may be None for policy "none"."""
    if policy not in POLICIES:
        raise ValueError(f"unknown policy {policy!r}")
    if policy != "none" and planner is None:
        raise ValueError("a rescheduling policy needs a planner")
    rng = np.random.default_rng(cfg.seed)
    n = cfg.n_inst
    rate = cfg.rate_per_8 * n / 8.0
    end_ms = cfg.duration_s * 1000.0

    # arrivals, drawn up front so that every policy sees the same requests
    t, times = 0.0, []
    while True:
        t += rng.exponential(1000.0 / rate)
        if t >= end_ms:
            break
        times.append(t)
    m = len(times)
    prompts = rng.integers(cfg.prompt_lo, cfg.prompt_hi, endpoint=True, size=m)
    outs = synth.draw_true_len(rng, cfg.out_law, m, cfg.out_cap)
    noise = np.exp(rng.normal(0.0, cfg.pred_sigma, size=m))
    arrivals = [(times[q], int(prompts[q]), int(outs[q]), float(noise[q])) for q in range(m)]

    inst_reqs: List[List[_Req]] = [[] for _ in range(n)]   # placed on the instance
    inst_tokens = np.zeros(n, np.int64)
    batch: List[Optional[List[Tuple[_Req, int]]]] = [None] * n   # the iteration in progress
    batch_ms = [0.0] * n
    events: List[Tuple[float, int, int, int]] = []   # (time, kind, seq, payload)
    seq = 0
    KIND_ARRIVE, KIND_ITER, KIND_LAND, KIND_TICK = 0, 1, 2, 3

    def push(time, kind, payload):
        nonlocal seq
        heapq.heappush(events, (time, kind, seq, payload))
        seq += 1

    for i, a in enumerate(arrivals):
        push(a[0], KIND_ARRIVE, i)
    k = 1                       # ticks sample the metrics under every policy
    while k * cfg.interval_s * 1000.0 < end_ms:
        push(k * cfg.interval_s * 1000.0, KIND_TICK, 0)
        k += 1

    reqs: List[_Req] = []
    landing: dict = {}
    finished_tpot: List[float] = []
    var_samples: List[float] = []
    moves_log: List[Tuple[float, int, int, int]] = []
    oom_ticks = 0
    beta = bucket_weights(cfg.n_buckets, cfg.beta_halvings)
    ticks = 0

    def iter_ms(i):
        return cfg.iter_base_ms + cfg.iter_per_ktoken_ms * float(inst_tokens[i]) / 1000.0

    def start_iter(i, now):
        # an iteration decodes the requests present when it starts
        if batch[i] is None and inst_reqs[i]:
            batch[i] = [(r, r.epoch) for r in inst_reqs[i]]
            batch_ms[i] = iter_ms(i)
            push(now + batch_ms[i], KIND_ITER, i)

    def place(r, i, now):
        r.inst = i
        r.epoch += 1
        inst_reqs[i].append(r)
        inst_tokens[i] += r.cur
        start_iter(i, now)

    while events:
        now, kind, _, payload = heapq.heappop(events)
        if now >= end_ms:
            break
        if kind == KIND_ARRIVE:
            _, prompt, out, noise = arrivals[payload]
            r = _Req(len(reqs), prompt, out, noise)
            reqs.append(r)
            place(r, int(np.argmin(inst_tokens)), now)   # fewest tokens, lowest index on ties
        elif kind == KIND_ITER:
            i = payload
            done = False
            for r, ep in batch[i]:
                if r.inst != i or r.epoch != ep or r.rid in landing:
                    continue                       # migrated away during the iteration
                r.cur += 1
                r.left -= 1
                r.tokens += 1
                r.busy_ms += batch_ms[i]
                inst_tokens[i] += 1
                if r.left <= 0:
                    inst_tokens[i] -= r.cur
                    r.inst = -1
                    finished_tpot.append(r.busy_ms / r.tokens)
                    done = True
            if done:
                inst_reqs[i] = [r for r in inst_reqs[i] if r.inst == i]
            batch[i] = None
            start_iter(i, now)
        elif kind == KIND_LAND:
            r = landing.pop(payload)
            place(r, r.inst, now)
        elif kind == KIND_TICK:
            ticks += 1
            times = np.array([iter_ms(i) if inst_reqs[i] else 0.0 for i in range(n)])
            var_samples.append(float(times.var()))
            if (inst_tokens > cfg.mem_cap_tokens).any():
                oom_ticks += 1
            live = [r for i in range(n) for r in inst_reqs[i]]
            if policy == "none" or not live:
                continue
            cur = np.array([r.cur for r in live], np.int32)
            inst = np.array([r.inst for r in live], np.int32)
            if policy == "current":
                rem = np.ones(len(live), np.int32)
                b, K, w = 1, 1, np.ones(1, np.uint16)
            else:
                if policy == "oracle":
                    rem = np.array([r.left for r in live], np.int64)
                else:
                    rem = np.array([max(1, int(round(r.left * r.pred_factor))) for r in live],
                                   np.int64)
                rem = np.minimum(rem, cfg.out_cap).astype(np.int32)
                b, K, w = cfg.bucket, cfg.n_buckets, beta
            params = dict(theta=cfg.theta, min_rem=cfg.min_rem if policy != "current" else 0,
                          mem_cap=cfg.mem_cap_tokens, max_moves=cfg.max_moves)
            moves = planner(cur, rem, inst, w, n_inst=n, bucket=b, n_buckets=K, **params)
            for (ri, s, tgt) in moves:
                r = live[ri]
                if r.inst != s:
                    raise RuntimeError("planner moved a request from the wrong instance")
                if r.rid in landing:
                    # moved again by a later pass of the same plan: the
                    # transfer under way now ends on the new target
                    r.inst = tgt
                    moves_log.append((now, r.rid, s, tgt))
                    continue
                inst_reqs[s].remove(r)
                inst_tokens[s] -= r.cur
                transfer_ms = r.cur * cfg.kv_bytes_per_token * 8.0 / (cfg.link_gbps * 1e9) * 1e3
                r.inst = tgt
                r.epoch += 1
                r.busy_ms += transfer_ms           # the transfer counts against its TPOT
                landing[r.rid] = r
                push(now + transfer_ms, KIND_LAND, r.rid)
                moves_log.append((now, r.rid, s, tgt))

    tp = np.array(finished_tpot) if finished_tpot else np.zeros(1)
    return SimResult(policy=policy, exec_var_ms2=float(np.mean(var_samples)) if var_samples else 0.0,
                     p99_tpot_ms=float(np.percentile(tp, 99)), mean_tpot_ms=float(tp.mean()),
                     migrations=len(moves_log), oom_ticks=oom_ticks, finished=len(finished_tpot),
                     ticks=ticks, moves=moves_log)


class LibraryPlanner:
    """star_project_load -> star_plan_migrations on the GPU, per tick."""

    def __init__(self, device: str = "cuda"):
        import torch
        from . import star
        self.torch, self.star, self.dev = torch, star, device
        self.calls = 0

    def __call__(self, cur, rem, inst, beta, *, n_inst, bucket, n_buckets, theta, min_rem,
                 mem_cap, max_moves):
        torch, star = self.torch, self.star
        N = len(cur)
        lp = star.load_params(N, n_inst, bucket, n_buckets)
        pp = star.plan_params(N, n_inst, bucket, n_buckets, max_moves, theta=theta,
                              min_rem=min_rem, mem_cap=mem_cap)
        d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(self.dev)
        cur_d, rem_d, inst_d = d(cur), d(rem), d(inst)
        beta_d = d(np.ascontiguousarray(beta, np.uint16).view(np.int16))
        load = torch.empty((n_inst, n_buckets), dtype=torch.int64, device=self.dev)
        moves = torch.empty(max(max_moves, 1) * star.MOVE_FIELDS, dtype=torch.int32,
                            device=self.dev)
        cnt = torch.empty(1, dtype=torch.int32, device=self.dev)
        ws_l = star.Workspace(star.project_load_workspace_size(lp))
        ws_p = star.Workspace(star.plan_workspace_size(pp))
        star.project_load(lp, cur_d, rem_d, inst_d, load, ws_l)
        star.plan_migrations(pp, cur_d, rem_d, inst_d, load, beta_d, moves, cnt, ws_p)
        m = int(cnt.cpu()[0])
        mv = moves.cpu().numpy().reshape(-1, star.MOVE_FIELDS)[:m]
        self.calls += 1
        return [(int(x[0]), int(x[1]), int(x[2])) for x in mv]
