"""Pins of the CPU oracle's time-weighted variance objective and of Algorithm 1.

Section 5.2 states the migration objective as the variance of the instances'
token loads now plus a beta-weighted sum of the variances of their predicted
loads at later steps (Eq. 3-4).  Algorithm 1 classifies instances by their
weighted load w_i, enumerates filtered candidates and executes the one that
lowers that objective most, if any does.

The oracle reports a migration's gain as (n/2) times the change of
Phi = sum_k beta_k Var_i(L_i[k]).  It is pinned here against:
* a hand-worked example (golden file);
* statistics.pvariance over exact fractions, on curves rebuilt from scratch
  in pure Python with the request reassigned;
* the two-instance closed form Var{x, y} = ((x - y) / 2)^2;
* a move that swaps two curves, which changes nothing;
* linearity in the weights;
* current-load balancing at a one-step horizon;
* a pure-Python Algorithm 1, written from the algorithm's three phases
  with fractions for theta.
"""
import json
import os
import statistics
from fractions import Fraction

import numpy as np
import pytest

from paper_2510_13668_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _example():
    return json.load(open(os.path.join(GOLDEN, "variance_worked_example.json")))


# --------------------------------------------------------------------------
# pure-Python restatements used as independent pins
# --------------------------------------------------------------------------
def _curves(cur, rem, inst, n, b, K):
    """Bucketed load curves by per-step summation, in Python integers."""
    L = [[0] * K for _ in range(n)]
    for c, l, i in zip(cur.tolist(), rem.tolist(), inst.tolist()):
        for t in range(min(l, b * K)):
            L[i][t // b] += c + t
    return L


def _phi(L, beta):
    """sum_k beta_k * population variance over instances, exactly."""
    n, K = len(L), len(L[0])
    return sum(Fraction(int(beta[k])) * statistics.pvariance([Fraction(L[i][k]) for i in range(n)])
               for k in range(K))


def _random_case(rng, N, n, b, K, cur_hi=60, empty_inst=0):
    cur, rem, inst = synth.random_requests(rng, N, n, cur_hi=cur_hi, len_hi=b * K + 3,
                                           empty_inst=empty_inst)
    beta = rng.integers(0, 65536, size=K).astype(np.uint16)
    return cur, rem, inst, beta


# --------------------------------------------------------------------------
# f1: gains
# --------------------------------------------------------------------------
def test_worked_example(oracle_mod):
    ex = _example()
    rq = ex["requests"]
    cur, rem, inst = (np.array(rq[k], np.int32) for k in ("cur_len", "rem_len", "inst_of"))
    beta = np.array(ex["beta"], np.uint16)
    load, _ = oracle_mod.project_load(cur, rem, inst, n_inst=ex["n_inst"], bucket=ex["bucket"],
                                      n_buckets=ex["n_buckets"])
    np.testing.assert_array_equal(load, ex["load"])
    gain = oracle_mod.score_variance(cur, rem, inst, load, beta, bucket=ex["bucket"])
    assert gain.tolist() == ex["gain"]
    sel = oracle_mod.select_variance(cur, rem, inst, gain)
    assert sel["best_target"].tolist() == ex["best_target"]
    assert sel["best_gain"].tolist() == ex["best_gain"]
    assert list(sel["move"]) == ex["move"] and sel["move_gain"] == ex["move_gain"]

    two = ex["two_instance"]
    c2, r2, i2 = (np.array(two[k], np.int32) for k in ("cur_len", "rem_len", "inst_of"))
    one = np.ones(1, np.uint16)
    l2, _ = oracle_mod.project_load(c2, r2, i2, n_inst=2, bucket=1, n_buckets=1)
    assert oracle_mod.score_variance(c2, r2, i2, l2, one, bucket=1).tolist() == two["gain"]


@pytest.mark.parametrize("seed,N,n,b,K", [(0, 7, 3, 1, 5), (1, 9, 4, 3, 4), (2, 6, 5, 2, 3),
                                          (3, 10, 2, 4, 2), (4, 5, 3, 1, 1)])
def test_gain_is_exact_variance_change_of_rebuilt_curves(oracle_mod, seed, N, n, b, K):
    """For every (r, t): gain == (n/2) (Phi(after) - Phi(before)) with the
    curves after the move rebuilt from all requests, Phi via pvariance."""
    rng = np.random.default_rng(seed)
    cur, rem, inst, beta = _random_case(rng, N, n, b, K, empty_inst=1 if n > 2 else 0)
    load, _ = oracle_mod.project_load(cur, rem, inst, n_inst=n, bucket=b, n_buckets=K)
    gain = oracle_mod.score_variance(cur, rem, inst, load, beta, bucket=b)
    before = _phi(_curves(cur, rem, inst, n, b, K), beta)
    for r in range(N):
        for t in range(n):
            moved = inst.copy()
            moved[r] = t
            after = _phi(_curves(cur, rem, moved, n, b, K), beta)
            assert Fraction(int(gain[r, t])) == Fraction(n, 2) * (after - before), (r, t)


def test_two_instance_closed_form(oracle_mod):
    """n = 2: Var{x, y} = ((x - y)/2)^2, so the gain is
    sum_k beta_k [((x' - y')/2)^2 - ((x - y)/2)^2]."""
    rng = np.random.default_rng(11)
    b, K, N = 2, 6, 8
    cur, rem, inst, beta = _random_case(rng, N, 2, b, K)
    load, _ = oracle_mod.project_load(cur, rem, inst, n_inst=2, bucket=b, n_buckets=K)
    gain = oracle_mod.score_variance(cur, rem, inst, load, beta, bucket=b)
    for r in range(N):
        s, t = int(inst[r]), 1 - int(inst[r])
        moved = inst.copy()
        moved[r] = t
        La = _curves(cur, rem, moved, 2, b, K)
        Lb = load.tolist()
        expect = sum(Fraction(int(beta[k])) * (Fraction(La[0][k] - La[1][k], 2) ** 2
                                              - Fraction(Lb[0][k] - Lb[1][k], 2) ** 2)
                     for k in range(K))
        assert gain[r, t] == expect and gain[r, s] == 0


def test_mirror_move_changes_nothing(oracle_mod):
    """s holds {r, q}, t holds a copy of q: moving r swaps the two curves."""
    cur = np.array([40, 17, 17, 5], np.int32)
    rem = np.array([9, 4, 4, 2], np.int32)
    inst = np.array([0, 0, 1, 2], np.int32)
    beta = synth.bucket_weights(4, 3.0)
    load, _ = oracle_mod.project_load(cur, rem, inst, n_inst=3, bucket=3, n_buckets=4)
    gain = oracle_mod.score_variance(cur, rem, inst, load, beta, bucket=3)
    assert gain[0, 1] == 0
    assert gain[0, 2] != 0


def test_linear_in_weights_and_zero_weights(oracle_mod):
    rng = np.random.default_rng(5)
    cur, rem, inst, beta = _random_case(rng, 12, 4, 2, 5)
    beta = (beta // 4).astype(np.uint16)
    load, _ = oracle_mod.project_load(cur, rem, inst, n_inst=4, bucket=2, n_buckets=5)
    g1 = oracle_mod.score_variance(cur, rem, inst, load, beta, bucket=2)
    g3 = oracle_mod.score_variance(cur, rem, inst, load, (beta * 3).astype(np.uint16), bucket=2)
    assert (g3 == 3 * g1).all()
    g0 = oracle_mod.score_variance(cur, rem, inst, load, np.zeros(5, np.uint16), bucket=2)
    assert (g0 == 0).all()
    # one bucket alone: beta = e_j keeps only bucket j's variance change
    parts = []
    for j in range(5):
        e = np.zeros(5, np.uint16)
        e[j] = 1
        parts.append(oracle_mod.score_variance(cur, rem, inst, load, e, bucket=2))
    assert (sum(int(beta[j]) * parts[j] for j in range(5)) == g1).all()


def test_unit_horizon_is_current_load_balancing(oracle_mod):
    """b = 1, K = 1: only current loads N_i count; the best target of every
    request is the least-loaded other instance (lowest index on ties)."""
    rng = np.random.default_rng(8)
    N, n = 40, 6
    cur, _, inst = synth.random_requests(rng, N, n, cur_hi=500, len_hi=3)
    rem = np.ones(N, np.int32)
    load, _ = oracle_mod.project_load(cur, rem, inst, n_inst=n, bucket=1, n_buckets=1)
    gain = oracle_mod.score_variance(cur, rem, inst, load, np.ones(1, np.uint16), bucket=1)
    sel = oracle_mod.select_variance(cur, rem, inst, gain)
    now = load[:, 0]
    for r in range(N):
        others = [t for t in range(n) if t != inst[r]]
        least = min(others, key=lambda t: (now[t], t))
        assert sel["best_target"][r] == least


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_selection_against_library_sort(oracle_mod, seed):
    rng = np.random.default_rng(100 + seed)
    N, n, b, K = 30, 5, 2, 4
    cur, rem, inst, beta = _random_case(rng, N, n, b, K, empty_inst=1)
    inst[3] = n + 2          # an invalid request takes no part
    load, _ = oracle_mod.project_load(cur, rem, inst, n_inst=n, bucket=b, n_buckets=K)
    gain = oracle_mod.score_variance(cur, rem, inst, load, beta, bucket=b)
    assert (gain[3] == 0).all()
    keys = sorted((int(gain[r, t]), r, t) for r in range(N) for t in range(n)
                  if r != 3 and t != inst[r])
    sel = oracle_mod.select_variance(cur, rem, inst, gain)
    for r in range(N):
        mine = [k for k in keys if k[1] == r]
        assert sel["best_target"][r] == (mine[0][2] if mine else -1)
        assert sel["best_gain"][r] == (mine[0][0] if mine else 0)
    g, r, t = keys[0]
    if g < 0:
        assert sel["move"] == (r, int(inst[r]), t) and sel["move_gain"] == g
    else:
        assert sel["move"] == (-1, -1, -1) and sel["move_gain"] == 0


def test_no_improving_move_gives_none(oracle_mod):
    """Identical instances: every move raises the variance."""
    cur = np.array([30, 30, 30], np.int32)
    rem = np.array([5, 5, 5], np.int32)
    inst = np.array([0, 1, 2], np.int32)
    load, _ = oracle_mod.project_load(cur, rem, inst, n_inst=3, bucket=2, n_buckets=3)
    gain = oracle_mod.score_variance(cur, rem, inst, load, synth.bucket_weights(3), bucket=2)
    sel = oracle_mod.select_variance(cur, rem, inst, gain)
    assert all(gain[r, t] > 0 for r in range(3) for t in range(3) if t != r)
    assert sel["move"] == (-1, -1, -1)


def test_out_of_range_values_are_refused(oracle_mod):
    cur = np.full(64, 2**31 - 1, np.int32)
    rem = np.full(64, 1 << 20, np.int32)
    inst = np.zeros(64, np.int32)
    K, b = 1 << 10, 1 << 10
    load = np.full((2, K), (1 << 62), np.int64)
    with pytest.raises(OverflowError):
        oracle_mod.score_variance(cur, rem, inst, load, np.full(K, 65535, np.uint16), bucket=b)


# --------------------------------------------------------------------------
# f2: Algorithm 1 end to end
# --------------------------------------------------------------------------
def test_plan_worked_example(oracle_mod):
    ex = _example()
    rq = ex["requests"]
    cur, rem, inst = (np.array(rq[k], np.int32) for k in ("cur_len", "rem_len", "inst_of"))
    beta = np.array(ex["beta"], np.uint16)
    for p in ex["plans"]:
        out = oracle_mod.plan(cur, rem, inst, beta, n_inst=ex["n_inst"], bucket=ex["bucket"],
                              n_buckets=ex["n_buckets"], theta=p["theta"], u_mode=p["u_mode"],
                              min_rem=p["min_rem"], mem_cap=p["mem_cap"], mem_mode=p["mem_mode"],
                              max_moves=4)
        assert [list(m) for m in out["moves"]] == p["moves"], p
        assert out["gains"] == p["gains"]
        assert out["inst_of"].tolist() == p["inst_of"]
        np.testing.assert_array_equal(out["load"], p["load"])
    two = ex["two_instance"]
    c2, r2, i2 = (np.array(two[k], np.int32) for k in ("cur_len", "rem_len", "inst_of"))
    out = oracle_mod.plan(c2, r2, i2, np.ones(1, np.uint16), n_inst=2, bucket=1, n_buckets=1,
                          max_moves=5)
    assert [list(m) for m in out["moves"]] == two["moves"] and out["gains"] == two["gains"]


def _plan_python(cur, rem, inst, beta, n, b, K, theta, u_mode, min_rem, mem_cap, mem_mode,
                 max_moves):
    """Algorithm 1 with exact fractions: classification, filtered candidate
    enumeration, best-feasible selection by the exact variance objective."""
    inst = [int(x) for x in inst]
    th = Fraction(theta[0], theta[1])
    moves, gains = [], []
    valid = [c >= 1 and l >= 1 and 0 <= i < n for c, l, i in zip(cur, rem, inst)]
    for _ in range(max_moves):
        L = _curves(cur[valid], rem[valid], np.array(inst)[valid], n, b, K)
        w = [sum(int(beta[k]) * L[i][k] for k in range(K)) for i in range(n)]
        wbar = Fraction(sum(w), n)
        now = [sum(int(cur[r]) for r in range(len(inst)) if valid[r] and inst[r] == i)
               for i in range(n)]
        over = [w[i] > (1 + th) * wbar for i in range(n)]
        if u_mode == 0:
            under = [now[i] < (1 + th) * wbar for i in range(n)]
        else:
            under = [w[i] < (1 - th) * wbar for i in range(n)]
        if not any(over):
            break
        base = _phi(L, beta)
        best = None
        for r in range(len(inst)):
            s = inst[r]
            if not valid[r] or not over[s] or rem[r] <= min_rem:
                continue
            for t in range(n):
                if t == s or not under[t]:
                    continue
                if now[t] + int(rem[r]) + (int(cur[r]) if mem_mode else 0) > mem_cap:
                    continue
                moved = list(inst)
                moved[r] = t
                La = _curves(cur[valid], rem[valid], np.array(moved)[valid], n, b, K)
                d = Fraction(n, 2) * (_phi(La, beta) - base)
                assert d.denominator == 1
                key = (int(d), r, t)
                if d < 0 and (best is None or key < best):
                    best = key
        if best is None:
            break
        g, r, t = best
        moves.append((r, inst[r], t))
        gains.append(g)
        inst[r] = t
    return moves, gains, inst


@pytest.mark.parametrize("seed,N,n,b,K,theta,u_mode,min_rem,mem_mode",
                         [(0, 12, 3, 1, 4, (0, 1), 0, 0, 0),
                          (1, 14, 4, 2, 3, (1, 5), 0, 2, 1),
                          (2, 10, 3, 3, 2, (1, 10), 1, 0, 0),
                          (3, 16, 5, 1, 3, (0, 1), 1, 1, 1),
                          (4, 9, 2, 2, 4, (1, 3), 0, 0, 0)])
def test_plan_matches_python_algorithm(oracle_mod, seed, N, n, b, K, theta, u_mode, min_rem,
                                       mem_mode):
    rng = np.random.default_rng(300 + seed)
    cur, rem, inst, beta = _random_case(rng, N, n, b, K, cur_hi=40)
    # crowd the first instance so that the plan has work to do
    inst[: N // 2] = 0
    if seed == 3:
        inst[5] = -1             # an invalid request stays put and counts nowhere
    mem_cap = int(cur.sum()) // 2 if mem_mode else (1 << 40)
    ref = _plan_python(cur, rem, inst, beta, n, b, K, theta, u_mode, min_rem, mem_cap, mem_mode, 6)
    out = oracle_mod.plan(cur, rem, inst, beta, n_inst=n, bucket=b, n_buckets=K, theta=theta,
                          u_mode=u_mode, min_rem=min_rem, mem_cap=mem_cap, mem_mode=mem_mode,
                          max_moves=6)
    assert out["moves"] == ref[0]
    assert out["gains"] == ref[1]
    assert out["inst_of"].tolist() == ref[2]
    assert len(ref[0]) >= 1


def test_plan_invariants(oracle_mod):
    """Every move lowers the exact objective by (2/n) x its gain; the final
    curves are those of the final placement; max_moves caps the plan."""
    rng = np.random.default_rng(21)
    N, n, b, K = 24, 4, 2, 5
    cur, rem, inst, beta = _random_case(rng, N, n, b, K, cur_hi=80)
    inst[: 3 * N // 4] = 1
    out = oracle_mod.plan(cur, rem, inst, beta, n_inst=n, bucket=b, n_buckets=K, max_moves=8)
    assert len(out["moves"]) >= 2
    place = inst.copy()
    phi = _phi(_curves(cur, rem, place, n, b, K), beta)
    for (r, s, t), g in zip(out["moves"], out["gains"]):
        assert place[r] == s and s != t and g < 0
        place[r] = t
        nphi = _phi(_curves(cur, rem, place, n, b, K), beta)
        assert nphi - phi == Fraction(2, n) * g
        phi = nphi
    assert place.tolist() == out["inst_of"].tolist()
    assert out["load"].tolist() == _curves(cur, rem, place, n, b, K)
    capped = oracle_mod.plan(cur, rem, inst, beta, n_inst=n, bucket=b, n_buckets=K, max_moves=1)
    assert capped["moves"] == out["moves"][:1]


def test_plan_balanced_start_moves_nothing(oracle_mod):
    cur = np.array([30, 8, 30, 8, 30, 8], np.int32)
    rem = np.array([6, 2, 6, 2, 6, 2], np.int32)
    inst = np.array([0, 0, 1, 1, 2, 2], np.int32)
    out = oracle_mod.plan(cur, rem, inst, synth.bucket_weights(4), n_inst=3, bucket=2,
                          n_buckets=4, max_moves=5)
    assert out["moves"] == [] and out["inst_of"].tolist() == inst.tolist()


def test_neutral_best_move_is_not_taken(oracle_mod):
    """Three identical requests, two on instance 0: every migration out of 0
    swaps the two curves (gain 0), so there is no move that lowers the
    objective and neither the selection nor the plan takes one."""
    cur = np.array([25, 25, 25], np.int32)
    rem = np.array([7, 7, 7], np.int32)
    inst = np.array([0, 0, 1], np.int32)
    beta = synth.bucket_weights(4)
    load, _ = oracle_mod.project_load(cur, rem, inst, n_inst=2, bucket=2, n_buckets=4)
    gain = oracle_mod.score_variance(cur, rem, inst, load, beta, bucket=2)
    assert gain[0, 1] == 0 and gain[1, 1] == 0 and gain[2, 0] > 0
    sel = oracle_mod.select_variance(cur, rem, inst, gain)
    assert sel["best_gain"].tolist() == [0, 0, gain[2, 0]]
    assert sel["move"] == (-1, -1, -1) and sel["move_gain"] == 0
    out = oracle_mod.plan(cur, rem, inst, beta, n_inst=2, bucket=2, n_buckets=4, max_moves=3)
    assert out["moves"] == []


def test_plan_current_loads_gate_targets(oracle_mod):
    """b = 1, K = 1, beta = 1: w_i is the current load N_i.  Loads [20, 10, 0]
    with theta = 0 give mean 10, O = {0} and U = {2} (10 is not below 10),
    so the first move goes to instance 2 although instance 1 is also
    lighter.  With the memory filter N_t + rem_r <= 12 and instance 2
    pre-loaded to 9, only the request with rem_r <= 3 may go there."""
    one = np.ones(1, np.uint16)
    cur = np.array([12, 8, 10], np.int32)
    rem = np.array([1, 1, 1], np.int32)
    inst = np.array([0, 0, 1], np.int32)
    out = oracle_mod.plan(cur, rem, inst, one, n_inst=3, bucket=1, n_buckets=1, max_moves=1)
    assert [m[2] for m in out["moves"]] == [2]
    # the printed U rule uses current tokens, not remaining lengths
    cur = np.array([12, 8, 10, 9], np.int32)
    rem = np.array([5, 3, 1, 30], np.int32)
    inst = np.array([0, 0, 1, 2], np.int32)
    # loads [20, 10, 9]: mean 13, O = {0}, U = {1, 2}; N_2 + rem: 9+5, 9+3
    out = oracle_mod.plan(cur, rem, inst, one, n_inst=3, bucket=1, n_buckets=1, max_moves=1,
                          mem_cap=12)
    assert out["moves"] == [(1, 0, 2)]
    out = oracle_mod.plan(cur, rem, inst, one, n_inst=3, bucket=1, n_buckets=1, max_moves=1,
                          mem_cap=12, mem_mode=1)
    assert out["moves"] == []        # 9 + 8 + 3 and 10 + 12 + 5 both exceed 12


def test_plan_lower_threshold_is_strict():
    """U = {w_i < (1 - theta) mean w}: loads [20, 5, 5], theta = 1/2 put both
    light instances exactly at the threshold, so there is no target."""
    import oracle as oracle_mod
    one = np.ones(1, np.uint16)
    cur = np.array([12, 8, 5, 5], np.int32)
    rem = np.ones(4, np.int32)
    inst = np.array([0, 0, 1, 2], np.int32)
    out = oracle_mod.plan(cur, rem, inst, one, n_inst=3, bucket=1, n_buckets=1, max_moves=2,
                          theta=(1, 2), u_mode=1)
    assert out["moves"] == []
    out = oracle_mod.plan(cur, rem, inst, one, n_inst=3, bucket=1, n_buckets=1, max_moves=1,
                          theta=(1, 3), u_mode=1)
    # threshold 20/3: both light ones qualify; moving c = 8 to instance 1
    # gives 8 (8 + 5 - 20) = -56, moving c = 12 gives 12 (12 + 5 - 20) = -36
    assert out["moves"] == [(1, 0, 1)]
