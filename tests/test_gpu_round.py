"""GPU parity of (b) load projection and (c) scoring/ranking against the
oracle: bit-exact load curves, scores, best targets and top-k triples, at the
five workloads' full sizes and on adversarial inputs; plus the chained round
(a) -> (b) -> (c), device-error reporting and HIP-graph replay.  Cases marked
`fused` run (b) and (c) as one star_project_and_score call."""
import zlib

import numpy as np
import pytest
import torch

import oracle
from paper_2510_13668_amd import star, synth
from gpu_util import Predictor, Rescheduler, assert_round_equal, to_dev

pytestmark = pytest.mark.gpu


def _gpu_round(cur, rem, inst, n, b, K, top_k, want_scores=True, fused=False):
    rs = Rescheduler(len(cur), n, b, K, top_k, want_scores, fused)
    rs.run(to_dev(cur), to_dev(rem), to_dev(inst))
    out = rs.result()
    out["error"] = rs.ws_load.read_device_error() | rs.ws_score.read_device_error()
    return out


def _check(cur, rem, inst, n, b, K, top_k, want_scores=True, fused=False):
    print(f"round N={len(cur)} n={n} b={b} K={K} top_k={top_k} fused={fused}", flush=True)
    gpu = _gpu_round(cur, rem, inst, n, b, K, top_k, want_scores, fused)
    ref = oracle.round_(cur, rem, inst, n_inst=n, bucket=b, n_buckets=K, top_k=top_k)
    assert_round_equal(gpu, ref)
    assert gpu["error"] == ref["flags"]
    return gpu, ref


@pytest.mark.parametrize("fused", [False, True], ids=["separate", "fused"])
@pytest.mark.parametrize("name", ["8b_batch", "32b_long_mix", "continuous", "rebalance_scan"])
def test_workload_true_lengths(name, fused):
    """Oracle-predictor mode: the workload's true remaining lengths."""
    wl = synth.WORKLOADS[name]
    x = synth.make_inputs(wl, steps=1, n_req=1)
    _check(x.cur_len, x.true_len, x.inst_of, wl.n_inst, wl.bucket, wl.n_buckets, wl.top_k,
           fused=fused)


def test_long_output_stress_mix():
    rng = np.random.default_rng(5)
    N, n = 4096, 16
    rem = synth.draw_true_len(rng, "long_output_stress", N, 32768)
    cur = rng.integers(1, 32768, size=N, endpoint=True).astype(np.int32)
    inst = rng.integers(0, n, size=N).astype(np.int32)
    _check(cur, rem, inst, n, 64, 512, 256)


def test_tiny_chained_from_gpu_prediction():
    """(a) -> (b) -> (c) on the tiny workload; the oracle's (b)(c) consume the
    GPU's integer rem_len, the bit-exact contract for chained rounds."""
    wl = synth.WORKLOADS["tiny"]
    x = synth.make_inputs(wl)
    pr = Predictor(x.w1, x.w2, x.bin_values, dtype=wl.dtype, act=wl.act, n_req=wl.n_req,
                   len_max=wl.len_max)
    pr.run(to_dev(x.hidden))
    rem_dev = pr.rem
    rs = Rescheduler(wl.n_req, wl.n_inst, wl.bucket, wl.n_buckets, min(256, wl.n_req * 3))
    cur_dev, inst_dev = to_dev(x.cur_len), to_dev(x.inst_of)
    rs.run(cur_dev, rem_dev, inst_dev)
    gpu = rs.result()
    rem = pr.rem.cpu().numpy()
    ref = oracle.round_(x.cur_len, rem, x.inst_of, n_inst=wl.n_inst, bucket=wl.bucket,
                        n_buckets=wl.n_buckets, top_k=min(256, wl.n_req * 3))
    assert_round_equal(gpu, ref)


def test_continuous_chained_steps():
    """Continuous mode: cur_len grows by one token per decode step; (b)(c) on
    the GPU's own predictions, ten steps."""
    wl = synth.WORKLOADS["continuous"]
    x = synth.make_inputs(wl, steps=10)
    pr = Predictor(x.w1, x.w2, x.bin_values, dtype=wl.dtype, act=wl.act, n_req=wl.n_req,
                   len_max=wl.len_max, ema_alpha=wl.ema_alpha)
    rs = Rescheduler(wl.n_req, wl.n_inst, wl.bucket, wl.n_buckets, wl.top_k)
    hid = to_dev(x.hidden, True)
    inst_dev = to_dev(x.inst_of)
    for s in range(10):
        cur = (x.cur_len + s).astype(np.int32)
        pr.run(hid[s], ema_init=(s == 0))
        rs.run(to_dev(cur), pr.rem, inst_dev)
        gpu = rs.result()
        ref = oracle.round_(cur, pr.rem.cpu().numpy(), x.inst_of, n_inst=wl.n_inst,
                            bucket=wl.bucket, n_buckets=wl.n_buckets, top_k=wl.top_k)
        assert_round_equal(gpu, ref)


ADVERSARIAL = [
    # (label, N, n, b, K, top_k, cur_hi, len_hi, contiguous, empty_inst)
    ("shuffled", 700, 8, 64, 256, 256, 8192, 20000, False, 0),
    ("uneven_empty", 300, 9, 16, 100, 64, 4000, 2500, False, 4),
    ("unit_buckets_long_K", 200, 4, 1, 4096, 256, 2048, 5000, False, 0),
    ("ragged_chunks", 150, 3, 1, 3000, 100, 500, 3500, False, 0),
    ("single_bucket", 400, 6, 7, 1, 512, 9000, 30, False, 0),
    ("unit_horizon", 128, 5, 1, 1, 77, 3000, 3, False, 0),
    ("one_instance", 50, 1, 4, 10, 8, 100, 60, True, 0),
    ("more_topk_than_candidates", 10, 3, 2, 5, 1000, 50, 12, False, 0),
    ("no_topk", 333, 7, 32, 64, 0, 5000, 3000, False, 0),
    ("topk_one", 333, 7, 32, 64, 1, 5000, 3000, False, 0),
    ("many_instances", 600, 300, 8, 40, 1024, 3000, 400, False, 0),
    ("big_bucket", 64, 4, 1000, 3, 16, 100000, 5000, True, 0),
    # many scoring workgroups with all curves in LDS, top-k over every migration
    ("multi_block_direct", 2000, 4, 16, 64, 256, 5000, 1200, False, 0),
    # separate scoring workgroups grown to 8 requests each (2049 of them,
    # the last one ragged); the top-k narrows the best keys by code
    ("grown_groups", 16390, 64, 16, 64, 256, 5000, 1200, False, 0),
]


@pytest.mark.parametrize("fused", [False, True], ids=["separate", "fused"])
@pytest.mark.parametrize("case", ADVERSARIAL, ids=[c[0] for c in ADVERSARIAL])
def test_adversarial(case, fused):
    label, N, n, b, K, top_k, cur_hi, len_hi, contiguous, empty = case
    rng = np.random.default_rng(zlib.crc32(label.encode()))
    cur, rem, inst = synth.random_requests(rng, N, n, cur_hi=cur_hi, len_hi=len_hi,
                                           contiguous=contiguous, empty_inst=empty)
    H = b * K
    # lengths at and around the horizon and bucket boundaries
    special = np.array([1, b, 2 * b, H - 1, H, H + 1, 3 * H], np.int64)
    m = min(len(special), N)
    rem[:m] = np.clip(special[:m], 1, 2 ** 31 - 1).astype(np.int32)
    _check(cur, rem, inst, n, b, K, top_k, fused=fused)


@pytest.mark.parametrize("fused", [False, True], ids=["separate", "fused"])
@pytest.mark.parametrize("N", [256, 6000, 20000])
def test_ties_from_duplicated_requests(N, fused):
    """Many equal scores; N = 6000 takes the two-stage (pruned) ranking with
    every best key in registers, N = 20000 narrows its first stage with the
    best-key code histogram (16 instances: 1250 scoring workgroups)."""
    rng = np.random.default_rng(3)
    n = 8 if N < 20000 else 16
    cur = np.full(N, 1000, np.int32)
    rem = np.full(N, 777, np.int32)
    inst = rng.integers(0, n, N).astype(np.int32)
    cur[::3] = 5
    rem[::5] = 64
    _check(cur, rem, inst, n, 64, 32, 300, fused=fused)


@pytest.mark.parametrize("fused", [False, True], ids=["separate", "fused"])
def test_crowded_best_code_takes_streamed_stage(fused):
    """Every request's best move is the same (all go to the one empty
    instance with equal lengths): the code that holds the k-th best key holds
    all 20000 of them, more than the top-k can gather, so its first stage
    selects over the streamed best keys."""
    rng = np.random.default_rng(8)
    N, n = 20000, 16
    cur = np.full(N, 1000, np.int32)
    rem = np.full(N, 777, np.int32)
    inst = rng.integers(0, n - 1, N).astype(np.int32)     # instance n - 1 stays empty
    _check(cur, rem, inst, n, 64, 32, 256, fused=fused)


# (N, n, b, K): the split projection (request slices met by a last arriver)
# at its boundaries -- the smallest stream, a ragged last slice with a tail
# of one request, the largest curve -- and the chunked kernel beyond them
# (one request fewer, more than 1024 buckets, more instances than arrival
# counters)
PROJECTION_REGIMES = [
    (8191, 5, 16, 700),
    (8192, 64, 64, 1024),
    (8193, 3, 16, 1024),
    (12001, 200, 8, 300),
    (9000, 7, 4, 1025),
    (9000, 1000, 2, 50),
    (40000, 2, 1, 1),
]


@pytest.mark.parametrize("fused", [False, True], ids=["separate", "fused"])
@pytest.mark.parametrize("N,n,b,K", PROJECTION_REGIMES)
def test_projection_regimes(N, n, b, K, fused):
    rng = np.random.default_rng(N * 7 + n)
    cur, rem, inst = synth.random_requests(rng, N, n, cur_hi=5000, len_hi=b * K + 7)
    _check(cur, rem, inst, n, b, K, 256, fused=fused)


def _key_bits(ref, inst, n):
    """Bits of the widest packed ranking key: score range, then r*n + t."""
    sc = ref["scores"]
    mask = np.ones(sc.shape, bool)
    mask[np.arange(len(inst)), inst] = False
    v = sc[mask]
    return int(v.max() - v.min()).bit_length() + int(sc.size - 1).bit_length()


@pytest.mark.parametrize("N,heavy,b,top_k", [(1024, 900, 16384, 256), (128, 100, 2 ** 18, 1024)])
def test_wide_keys_one_workgroup(N, heavy, b, top_k):
    """One heavily loaded instance of huge requests beside light ones: scores
    spread over > 2^54, so the ranking key needs more than 64 bits and the
    wide radix select runs (one-workgroup path); with top_k above the number
    of migrations every key wins and the ordering falls back to rank counts."""
    rng = np.random.default_rng(11)
    n, K = 8, 2
    inst = np.concatenate([np.zeros(heavy, np.int32),
                           rng.integers(1, n, size=N - heavy).astype(np.int32)])
    cur = np.concatenate([rng.integers(2 ** 30, 2 ** 31 - 1, size=heavy, endpoint=True),
                          rng.integers(1, 1000, size=N - heavy, endpoint=True)]).astype(np.int32)
    rem = rng.integers(1, 2 * b * K, size=N, endpoint=True).astype(np.int32)
    gpu, ref = _check(cur, rem, inst, n, b, K, top_k)
    assert _key_bits(ref, inst, n) > 64


def test_wide_keys_many_instances():
    """Two requests with huge buckets over 1024 instances: the best-move key
    ((score - min) << target bits | t) no longer fits 64 bits, so the
    two-step best-move reduction runs."""
    N, n, b, K = 2, 1024, 2 ** 28, 1
    cur = np.array([2 ** 31 - 1, 2 ** 31 - 1], np.int32)
    rem = np.array([b, b // 2 + 3], np.int32)
    inst = np.array([0, 5], np.int32)
    gpu, ref = _check(cur, rem, inst, n, b, K, 16)
    sc = ref["scores"]
    mask = np.ones(sc.shape, bool)
    mask[np.arange(N), inst] = False
    v = sc[mask]
    assert int(v.max() - v.min()).bit_length() + int(n - 1).bit_length() > 64


@pytest.mark.parametrize("fused", [False, True], ids=["separate", "fused"])
def test_invalid_requests_are_skipped_and_reported(fused):
    rng = np.random.default_rng(4)
    N, n = 500, 6
    cur, rem, inst = synth.random_requests(rng, N, n, cur_hi=3000, len_hi=3000)
    inst[10] = n          # out of range
    inst[11] = -1
    cur[20] = 0
    rem[30] = 0
    rem[31] = -5
    gpu, ref = _check(cur, rem, inst, n, 64, 64, 128, fused=fused)
    assert gpu["error"] == star.DEV_BAD_INST | star.DEV_BAD_CUR | star.DEV_BAD_REM
    assert (gpu["best_target"][[10, 11, 20, 30, 31]] == -1).all()


@pytest.mark.parametrize("fused", [False, True], ids=["separate", "fused"])
def test_empty_request_set(fused):
    gpu = _gpu_round(np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32),
                     4, 8, 16, 10, fused=fused)
    assert (gpu["load"] == 0).all()
    assert (gpu["topk_req"] == -1).all()


# (N, n, b, K, top_k): curves projected in every scoring group, at 32, 35
# and 188 groups; too many requests to project per group (the projection
# kernel runs first); no top-k; curves too large for LDS
FUSED_PATHS = [(1024, 8, 64, 256, 256), (700, 5, 16, 100, 64), (6000, 8, 64, 32, 300),
               (10000, 8, 16, 40, 512), (900, 6, 32, 50, 0), (300, 64, 8, 80, 100),
               (10000, 64, 8, 40, 256)]


def test_calls_of_every_path_share_a_workspace():
    """Rounds of every path, one after another on one workspace sized for
    the largest, with a predictor call on the same workspace before each
    (its split-K partials fill the scratch area): the ranking's code
    histogram lives in the workspace header, which no call uses as scratch,
    and every call must equal the oracle.  The last case gathers best keys
    by code in the workspace."""
    rng = np.random.default_rng(21)
    B, d, m, nb = 64, 512, 128, 32
    w1 = synth.f32_to_bf16_bits((rng.standard_normal((m, d)) / np.sqrt(d)).astype(np.float32))
    w2 = synth.f32_to_bf16_bits((rng.standard_normal((nb, m)) / np.sqrt(m)).astype(np.float32))
    hid = to_dev(synth.f32_to_bf16_bits(rng.standard_normal((B, d)).astype(np.float32)), True)
    pr = Predictor(w1, w2, synth.bin_values(nb, 1.0, 4096.0), dtype=synth.BF16,
                   act=synth.ACT_GELU, n_req=B, len_max=4096)
    ws = star.Workspace(max([star.project_and_score_workspace_size(star.score_params(*c))
                             for c in FUSED_PATHS] + [star.predict_workspace_size(pr.params(False))]))
    pr.ws = ws
    for rep in range(2):
        for N, n, b, K, top_k in FUSED_PATHS:
            print(f"fused rep={rep} N={N} n={n} b={b} K={K} top_k={top_k}", flush=True)
            pr.run(hid)
            cur, rem, inst = synth.random_requests(rng, N, n, cur_hi=4000, len_hi=b * K + 50)
            rs = Rescheduler(N, n, b, K, top_k, fused=True)
            rs.ws_load = rs.ws_score = ws
            rs.run(to_dev(cur), to_dev(rem), to_dev(inst))
            ref = oracle.round_(cur, rem, inst, n_inst=n, bucket=b, n_buckets=K, top_k=top_k)
            assert_round_equal(rs.result(), ref)
            assert ws.read_device_error() == ref["flags"]


def test_error_word_clears_after_read():
    rs = Rescheduler(4, 2, 1, 4, 2)
    bad = to_dev(np.array([0, 5, 1, 1], np.int32))
    ok = to_dev(np.array([1, 1, 1, 1], np.int32))
    rs.run(ok, ok, bad)
    assert rs.ws_load.read_device_error() == star.DEV_BAD_INST
    assert rs.ws_load.read_device_error() == 0
    rs.run(ok, ok, to_dev(np.array([0, 1, 1, 0], np.int32)))
    assert rs.ws_load.read_device_error() == 0


def test_graph_replay_matches_eager():
    """The continuous-mode round captured once as a HIP graph and replayed
    several times, with eager work and synchronisations in between; every
    replay equals the eager result."""
    wl = synth.WORKLOADS["continuous"]
    x = synth.make_inputs(wl, steps=3)
    hid = to_dev(x.hidden, True)
    pr = Predictor(x.w1, x.w2, x.bin_values, dtype=wl.dtype, act=wl.act, n_req=wl.n_req,
                   len_max=wl.len_max, ema_alpha=wl.ema_alpha)
    rs = Rescheduler(wl.n_req, wl.n_inst, wl.bucket, wl.n_buckets, wl.top_k)
    cur = to_dev(x.cur_len)
    inst = to_dev(x.inst_of)
    src = hid[1].clone()

    def step(s):
        pr.run(src, stream=s)
        rs.run(cur, pr.rem, inst, stream=s)

    # eager reference from a known EMA state
    pr.run(hid[0], ema_init=True)
    ema0 = pr.ema.clone()
    step(None)
    torch.cuda.synchronize()
    want = rs.result()
    want_ema = pr.ema.cpu().numpy().copy()

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        pr.ema.copy_(ema0)
        step(s)          # warm-up on the capture stream
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        step(s)
    for rep in range(4):
        pr.ema.copy_(ema0)
        rs.load.fill_(-7)
        rs.best_target.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = rs.result()
        assert_round_equal(got, want)
        np.testing.assert_array_equal(pr.ema.cpu().numpy(), want_ema)
        _ = torch.ones(1000, device="cuda").sum().item()    # unrelated eager work between replays


def test_pipelined_graph_rounds_match_eager():
    """Rounds pipelined on two streams, as the benchmark runs them: the
    predictions run on one stream (star_predict_overlap: one round's head
    and the next round's first-layer product per call) while earlier rounds
    are projected and scored on a second, which waits for the predictions
    two rounds at a time and records one event per batch of two.  The per-round outputs
    rotate through six buffers; before a prediction overwrites a buffer,
    its stream waits once for the event of the batch that last scheduled
    it.  The whole chunk is captured as one HIP graph.  Every replay (with
    eager work and synchronisations between replays) must leave the last
    six rounds' outputs (all in reused buffers) and the EMA state equal to
    twelve eager rounds run one after another.  The pipelined rounds use
    the fused projection-and-scoring call, the eager ones the two separate
    calls."""
    wl = synth.WORKLOADS["continuous"]
    R = 12
    NS = 6
    BATCH = 2
    x = synth.make_inputs(wl, steps=R + 1)
    hid = to_dev(x.hidden, True)
    N = wl.n_req
    pr = Predictor(x.w1, x.w2, x.bin_values, dtype=wl.dtype, act=wl.act, n_req=N,
                   len_max=wl.len_max, ema_alpha=wl.ema_alpha)
    inst = to_dev(x.inst_of)
    curs = [to_dev((x.cur_len + s).astype(np.int32)) for s in range(R + 1)]

    # eager reference: step 0 initialises the EMA, then rounds on steps 1..R
    pr.run(hid[0], ema_init=True)
    ema0 = pr.ema.clone()
    ref = Rescheduler(N, wl.n_inst, wl.bucket, wl.n_buckets, wl.top_k)
    want = []
    for j in range(R):
        pr.run(hid[j + 1])
        ref.run(curs[j + 1], pr.rem, inst)
        want.append(ref.result())
    want_ema = pr.ema.cpu().numpy().copy()

    P, S2 = torch.cuda.Stream(), torch.cuda.Stream()
    slots = [Rescheduler(N, wl.n_inst, wl.bucket, wl.n_buckets, wl.top_k, fused=True)
             for _ in range(NS)]
    rems = [torch.empty(N, dtype=torch.int32, device="cuda") for _ in range(NS)]
    exps = [torch.empty(N, dtype=torch.float32, device="cuda") for _ in range(NS)]
    ev_pred = [torch.cuda.Event() for _ in range(NS)]
    ev_done = [torch.cuda.Event() for _ in range(NS)]
    pp = pr.params(False)

    wsp = [pr.ws, star.Workspace(pr.ws.nbytes)]

    def chunk():
        S2.wait_stream(P)
        guard, waited, nbatch = [None] * NS, None, 0
        batch = []
        # round j's head and round j+1's product in one call
        star.predict_overlap(pp, hid[1], wsp[0], None, pr.w1, pr.b1, pr.w2, pr.b2, pr.bins,
                             None, None, None, P)
        for j in range(R):
            k = j % NS
            if guard[k] is not None and guard[k] is not waited:
                P.wait_event(guard[k])
                waited = guard[k]
            nxt = hid[j + 2] if j + 1 < R else None
            star.predict_overlap(pp, nxt, wsp[(j + 1) % 2] if nxt is not None else None,
                                 wsp[j % 2], pr.w1, pr.b1, pr.w2, pr.b2, pr.bins, pr.ema,
                                 exps[k], rems[k], P)
            batch.append((j, k))
            if len(batch) == BATCH or j == R - 1:
                ev_pred[k].record(P)
                S2.wait_event(ev_pred[k])
                for bj, bk in batch:
                    slots[bk].run(curs[bj + 1], rems[bk], inst, stream=S2)
                ev = ev_done[nbatch % NS]
                nbatch += 1
                ev.record(S2)
                for _, bk in batch:
                    guard[bk] = ev
                batch = []
        P.wait_stream(S2)

    torch.cuda.synchronize()
    with torch.cuda.stream(P):
        pr.ema.copy_(ema0)
    chunk()                      # warm-up, eager, on the capture streams
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=P):
        chunk()
    for rep in range(3):
        pr.ema.copy_(ema0)
        for sl in slots:
            sl.load.fill_(-7)
            sl.best_target.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for j in range(R - NS, R):
            assert_round_equal(slots[j % NS].result(), want[j])
        np.testing.assert_array_equal(pr.ema.cpu().numpy(), want_ema)
        _ = torch.ones(1000, device="cuda").sum().item()    # unrelated eager work between replays


def _random_round_case(rng, kind):
    """Sizes aimed at one ranking regime each, and requests that are either
    random or drawn from a few distinct (c, l) pairs (crowded key codes and
    many ties)."""
    if kind == 0:     # pruned top-k, best keys in registers
        N, n = int(rng.integers(2100, 8192)), int(rng.integers(3, 20))
    elif kind == 1:   # best keys narrowed by code, many instances
        N, n = int(rng.integers(8193, 30000)), int(rng.integers(16, 70))
    elif kind == 2:   # best keys narrowed by code, few instances
        N, n = int(rng.integers(8193, 40000)), int(rng.integers(4, 16))
    elif kind == 3:   # direct top-k, 16 keys per thread
        n = int(rng.integers(2, 8))
        N = int(rng.integers(8192 // n + 1, 16384 // n))
    elif kind == 4:   # the k requests' migrations streamed (k (n - 1) > 16384)
        N, n = int(rng.integers(9000, 20000)), int(rng.integers(70, 120))
    else:             # small rounds
        N, n = int(rng.integers(1, 3000)), int(rng.integers(1, 40))
    b = int(rng.choice([1, 4, 16, 64]))
    K = int(rng.integers(1, 300))
    top_k = int(rng.choice([1, 17, 256, 1000, 1024]))
    H = b * K
    if rng.random() < 0.5:
        d = int(rng.integers(1, 6))
        cv = rng.integers(1, 5000, size=d)
        lv = rng.integers(1, H + 10, size=d)
        pick = rng.integers(0, d, size=N)
        cur, rem = cv[pick].astype(np.int32), lv[pick].astype(np.int32)
        live = max(1, n - int(rng.integers(0, 2)))
        inst = rng.integers(0, live, size=N).astype(np.int32)
    else:
        cur, rem, inst = synth.random_requests(rng, N, n, cur_hi=int(rng.integers(1, 20000)),
                                               len_hi=int(rng.integers(1, 3 * H + 2)))
    return cur, rem, inst, n, b, K, top_k


def test_random_rounds_every_ranking_regime():
    """30 seeded random rounds over the ranking regimes (register, code-
    narrowed and streamed stages, direct top-k with 8 or 16 keys per thread,
    crowded boundary codes), each as two calls and as one; bit-exact."""
    rng = np.random.default_rng(2510)
    for c in range(30):
        cur, rem, inst, n, b, K, top_k = _random_round_case(rng, c % 6)
        for fused in (False, True):
            _check(cur, rem, inst, n, b, K, top_k, fused=fused)


def _wide_round_case(rng, kind):
    """Sizes beyond the ranking regimes: the split projection near its
    largest K, fewer requests than buckets (instance-major planes), the
    one-workgroup round, and broad mixes; top_k = 0 included."""
    if kind == 0:     # 8192+ requests, K up to 1024: the sliced projection
        N, n, K = int(rng.integers(8192, 40000)), int(rng.integers(1, 100)), int(rng.integers(200, 1025))
    elif kind == 1:   # fewer requests than buckets
        N, n, K = int(rng.integers(1, 2000)), int(rng.integers(2, 70)), int(rng.integers(1000, 4097))
    elif kind == 2:   # the whole round in one workgroup
        N, n = int(rng.integers(1, 1025)), int(rng.integers(1, 9))
        K = int(rng.integers(1, 2600 // n))
    else:
        N, n, K = int(rng.integers(1, 20000)), int(rng.integers(1, 129)), int(rng.integers(1, 1100))
    while N * n * K > 1.5e9:
        K = max(1, K // 2)
    b = int(rng.choice([1, 3, 16, 64]))
    top_k = int(rng.choice([0, 1, 17, 256, 1024]))
    H = b * K
    if rng.random() < 0.4:
        d = int(rng.integers(1, 6))
        cv = rng.integers(1, 5000, size=d)
        lv = rng.integers(1, H + 10, size=d)
        pick = rng.integers(0, d, size=N)
        cur, rem = cv[pick].astype(np.int32), lv[pick].astype(np.int32)
        live = max(1, n - int(rng.integers(0, 2)))
        inst = rng.integers(0, live, size=N).astype(np.int32)
    else:
        cur, rem, inst = synth.random_requests(rng, N, n, cur_hi=int(rng.integers(1, 30000)),
                                               len_hi=int(rng.integers(1, 3 * H + 2)))
    return cur, rem, inst, n, b, K, top_k


def test_random_rounds_wide_regimes():
    """40 seeded random rounds over the projection and scoring paths (sliced
    projection up to K = 1024, instance-major planes up to K = 4096, the
    one-workgroup round, broad mixes, with and without a top-k), each as two
    calls and as one; bit-exact."""
    rng = np.random.default_rng(13668)
    for c in range(40):
        cur, rem, inst, n, b, K, top_k = _wide_round_case(rng, c % 4)
        for fused in (False, True):
            _check(cur, rem, inst, n, b, K, top_k, fused=fused)


@pytest.mark.parametrize("N", [3, 4099, 8195])
def test_projection_of_misaligned_request_arrays(N):
    """Request arrays that start 4 bytes past a 16-byte boundary take the
    projection's int32 reads, aligned ones of 8192 requests and more its
    16-byte reads (with a ragged tail): all equal the oracle."""
    rng = np.random.default_rng(N)
    n, b, K = 7, 16, 90
    cur, rem, inst = synth.random_requests(rng, N, n, cur_hi=3000, len_hi=b * K + 40)
    ref = oracle.round_(cur, rem, inst, n_inst=n, bucket=b, n_buckets=K, top_k=0)
    lp = star.load_params(N, n, b, K)
    ws = star.Workspace(star.project_load_workspace_size(lp))
    for off in (0, 1):
        def place(a):
            t = torch.zeros(N + 4, dtype=torch.int32, device="cuda")
            t[off:off + N] = torch.from_numpy(a).cuda()
            return t[off:off + N]
        c, r, s = place(cur), place(rem), place(inst)
        assert (c.data_ptr() % 16 == 0) == (off == 0)
        load = torch.full((n, K), -1, dtype=torch.int64, device="cuda")
        star.project_load(lp, c, r, s, load, ws)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(load.cpu().numpy(), ref["load"], err_msg=f"offset {off}")
