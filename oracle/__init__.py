"""CPU oracle for the STAR decode-rescheduling hot path -- TEST INFRASTRUCTURE.

A plain, slow, obviously-correct restatement (fp64 predictor, int64 per-step
load curves, direct per-candidate maxima, full sort) used only by the test
suite, the smoke check and the benchmark's CPU-baseline leg.  Nothing in the
product path imports this package, and this package imports nothing from the
HIP path.  The C source is ``star_oracle.c``; ``python -m oracle.build``
compiles it.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

from .build import LIB, build

F32, BF16 = 0, 1
RELU, GELU = 0, 1
BAD_INST, BAD_CUR, BAD_REM = 1, 2, 4

_lib = None
_P = ctypes.c_void_p
_I64 = ctypes.c_int64


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        lib = ctypes.CDLL(LIB)
        lib.star_oracle_predict.argtypes = [_I64, _I64, _I64, _I64, ctypes.c_int, ctypes.c_int,
                                            _P, _P, _P, _P, _P, _P, ctypes.c_double, ctypes.c_int,
                                            _P, _I64, _P, _P, _P, _P]
        lib.star_oracle_project_load.argtypes = [_I64, _I64, _I64, _I64, _P, _P, _P, _P, _P]
        lib.star_oracle_score.argtypes = [_I64, _I64, _I64, _I64, _P, _P, _P, _P, _P]
        lib.star_oracle_rank.argtypes = [_I64, _I64, _P, _P, _P, _P, _I64, _P, _P, _P, _P, _P]
        lib.star_oracle_score_variance.argtypes = [_I64, _I64, _I64, _I64, _P, _P, _P, _P, _P, _P]
        lib.star_oracle_select_variance.argtypes = [_I64, _I64, _P, _P, _P, _P, _P, _P, _P, _P]
        lib.star_oracle_plan.argtypes = [_I64, _I64, _I64, _I64, _P, _P, _P, _P, _P, _I64, _I64,
                                         ctypes.c_int, _I64, _I64, ctypes.c_int, _I64, _P, _P, _P]
        lib.star_oracle_predict_mlp4.argtypes = [_I64, _I64, _I64, _I64, _I64, ctypes.c_int,
                                                 _P, _P, _P, _P, _P, _P, _P, _P,
                                                 ctypes.c_double, _P, _I64, ctypes.c_double,
                                                 ctypes.c_int, _P, _I64, _P, _P, _P]
        for f in ("star_oracle_predict_mlp4", "star_oracle_predict", "star_oracle_project_load",
                  "star_oracle_score",
                  "star_oracle_rank", "star_oracle_score_variance",
                  "star_oracle_select_variance", "star_oracle_plan"):
            getattr(lib, f).restype = ctypes.c_int
        _lib = lib
    return _lib


def threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(_load().star_oracle_threads())


def set_threads(n: int) -> None:
    """Threads of later parallel loops (timing only; results do not depend on it)."""
    lib = _load()
    lib.star_oracle_set_threads.argtypes = [ctypes.c_int]
    lib.star_oracle_set_threads(int(n))


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def predict(hidden, w1, w2, bin_values, *, dtype: int, act: int, b1=None, b2=None,
            ema_alpha: float = 0.0, ema_init: bool = False,
            ema_state: Optional[np.ndarray] = None, len_max: int = 1 << 30,
            want_stages: bool = False):
    """fp64 predictor.  bf16 operands are uint16 bit arrays.

    Returns dict(expected [B] f64, rem_len [B] i32[, z1 [B,m], z2 [B,nb]]).
    ``ema_state`` (fp64 [B]) is updated in place when ``ema_alpha > 0``.
    """
    et = np.uint16 if dtype == BF16 else np.float32
    hidden = _c(hidden, et)
    w1 = _c(w1, et)
    w2 = _c(w2, et)
    B, d = hidden.shape
    m = w1.shape[0]
    nb = w2.shape[0]
    assert w1.shape == (m, d) and w2.shape == (nb, m)
    b1 = _c(b1, np.float32)
    b2 = _c(b2, np.float32)
    v = _c(bin_values, np.float32)
    assert v.shape == (nb,)
    if ema_alpha > 0.0:
        assert ema_state is not None and ema_state.dtype == np.float64 and ema_state.shape == (B,)
        assert ema_state.flags.c_contiguous
    expected = np.empty(B, np.float64)
    rem = np.empty(B, np.int32)
    z1 = np.empty((B, m), np.float64) if want_stages else None
    z2 = np.empty((B, nb), np.float64) if want_stages else None
    rc = _load().star_oracle_predict(B, d, m, nb, dtype, act, _ptr(hidden), _ptr(w1), _ptr(b1),
                                     _ptr(w2), _ptr(b2), _ptr(v), float(ema_alpha),
                                     int(bool(ema_init)), _ptr(ema_state), int(len_max),
                                     _ptr(expected), _ptr(rem), _ptr(z1), _ptr(z2))
    if rc != 0:
        raise ValueError("star_oracle_predict: malformed arguments")
    out = {"expected": expected, "rem_len": rem}
    if want_stages:
        out["z1"] = z1
        out["z2"] = z2
    return out


def predict_mlp4(hidden, w1, w2, w3, w4, *, dtype: int, b1=None, b2=None, b3=None, b4=0.0,
                 rows=None, ema_alpha: float = 0.0, ema_init: bool = False,
                 ema_state: Optional[np.ndarray] = None, len_max: int = 1 << 30):
    """fp64 4-layer ReLU regression head on the listed rows (all if None).

    Returns dict(expected, rem_len, scale) indexed like `rows`.  ``ema_state``
    (fp64, one per listed row) is updated in place when ``ema_alpha > 0``.
    """
    et = np.uint16 if dtype == BF16 else np.float32
    hidden, w1, w2, w3 = (_c(a, et) for a in (hidden, w1, w2, w3))
    B, d = hidden.shape
    m1, m2, m3 = w1.shape[0], w2.shape[0], w3.shape[0]
    assert w1.shape == (m1, d) and w2.shape == (m2, m1) and w3.shape == (m3, m2)
    w4 = _c(w4, np.float32)
    assert w4.shape == (m3,)
    b1, b2, b3 = (_c(b, np.float32) for b in (b1, b2, b3))
    rows = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    R = B if rows is None else rows.shape[0]
    if ema_alpha > 0.0:
        assert ema_state is not None and ema_state.dtype == np.float64 and ema_state.shape == (R,)
    expected = np.empty(R, np.float64)
    rem = np.empty(R, np.int32)
    scale = np.empty(R, np.float64)
    rc = _load().star_oracle_predict_mlp4(B, d, m1, m2, m3, dtype, _ptr(hidden), _ptr(w1),
                                          _ptr(b1), _ptr(w2), _ptr(b2), _ptr(w3), _ptr(b3),
                                          _ptr(w4), float(b4), _ptr(rows), R, float(ema_alpha),
                                          int(bool(ema_init)), _ptr(ema_state), int(len_max),
                                          _ptr(expected), _ptr(rem), _ptr(scale))
    if rc != 0:
        raise ValueError("star_oracle_predict_mlp4: malformed arguments")
    return {"expected": expected, "rem_len": rem, "scale": scale}


def project_load(cur_len, rem_len, inst_of, *, n_inst: int, bucket: int, n_buckets: int):
    """int64 load curves [n, K] by per-step summation; returns (load, flags)."""
    cur = _c(cur_len, np.int32)
    rem = _c(rem_len, np.int32)
    inst = _c(inst_of, np.int32)
    N = cur.shape[0]
    assert rem.shape == (N,) and inst.shape == (N,)
    load = np.empty((n_inst, n_buckets), np.int64)
    flags = np.zeros(1, np.int32)
    rc = _load().star_oracle_project_load(N, n_inst, bucket, n_buckets, _ptr(cur), _ptr(rem),
                                          _ptr(inst), _ptr(load), _ptr(flags))
    if rc != 0:
        raise ValueError("star_oracle_project_load: malformed arguments")
    return load, int(flags[0])


def score(cur_len, rem_len, inst_of, load, *, bucket: int):
    """int64 candidate scores [N, n] by a direct maximum over all buckets."""
    cur = _c(cur_len, np.int32)
    rem = _c(rem_len, np.int32)
    inst = _c(inst_of, np.int32)
    load = _c(load, np.int64)
    n, K = load.shape
    N = cur.shape[0]
    scores = np.empty((N, n), np.int64)
    rc = _load().star_oracle_score(N, n, bucket, K, _ptr(cur), _ptr(rem), _ptr(inst),
                                   _ptr(load), _ptr(scores))
    if rc != 0:
        raise ValueError("star_oracle_score: malformed arguments")
    return scores


def rank(cur_len, rem_len, inst_of, scores, *, top_k: int):
    """Full-sort ranking; returns dict(best_target, best_score, topk_req, topk_tgt, topk_score)."""
    cur = _c(cur_len, np.int32)
    rem = _c(rem_len, np.int32)
    inst = _c(inst_of, np.int32)
    scores = _c(scores, np.int64)
    N, n = scores.shape
    bt = np.empty(N, np.int32)
    bs = np.empty(N, np.int64)
    tr = np.empty(max(top_k, 1), np.int32)
    tt = np.empty(max(top_k, 1), np.int32)
    ts = np.empty(max(top_k, 1), np.int64)
    rc = _load().star_oracle_rank(N, n, _ptr(cur), _ptr(rem), _ptr(inst), _ptr(scores), top_k,
                                  _ptr(bt), _ptr(bs), _ptr(tr), _ptr(tt), _ptr(ts))
    if rc != 0:
        raise ValueError("star_oracle_rank: malformed arguments")
    return {"best_target": bt, "best_score": bs, "topk_req": tr[:top_k],
            "topk_tgt": tt[:top_k], "topk_score": ts[:top_k]}


def round_(cur_len, rem_len, inst_of, *, n_inst: int, bucket: int, n_buckets: int, top_k: int):
    """Projection, scoring and ranking of one rescheduling round."""
    load, flags = project_load(cur_len, rem_len, inst_of, n_inst=n_inst, bucket=bucket,
                               n_buckets=n_buckets)
    scores = score(cur_len, rem_len, inst_of, load, bucket=bucket)
    out = rank(cur_len, rem_len, inst_of, scores, top_k=top_k)
    out.update(load=load, scores=scores, flags=flags)
    return out


# --------------------------------------------------------------------------
# time-weighted variance objective and Algorithm 1 end to end
# --------------------------------------------------------------------------
def i128_values(pairs: np.ndarray) -> np.ndarray:
    """(low, high) int64 pairs of 128-bit two's complement values -> Python ints."""
    pairs = np.asarray(pairs, dtype=np.int64)
    lo = pairs[..., 0].astype(np.uint64).astype(object)
    hi = pairs[..., 1].astype(object)
    return hi * (1 << 64) + lo


def score_variance(cur_len, rem_len, inst_of, load, beta, *, bucket: int):
    """Exact gains [N, n] (Python ints): (n/2) x the change of sum_k beta_k Var_k."""
    cur = _c(cur_len, np.int32)
    rem = _c(rem_len, np.int32)
    inst = _c(inst_of, np.int32)
    load = _c(load, np.int64)
    beta = _c(beta, np.uint16)
    n, K = load.shape
    N = cur.shape[0]
    assert beta.shape == (K,)
    gain = np.empty((N, n, 2), np.int64)
    rc = _load().star_oracle_score_variance(N, n, bucket, K, _ptr(cur), _ptr(rem), _ptr(inst),
                                            _ptr(load), _ptr(beta), _ptr(gain))
    if rc == -2:
        raise OverflowError("star_oracle_score_variance: values beyond the exact range")
    if rc != 0:
        raise ValueError(f"star_oracle_score_variance failed ({rc})")
    return i128_values(gain)


def select_variance(cur_len, rem_len, inst_of, gain):
    """Full-sort selection over exact gains [N, n] (Python ints).

    Returns dict(best_target [N] i32, best_gain [N] object, move (r, s, t),
    move_gain int).
    """
    cur = _c(cur_len, np.int32)
    rem = _c(rem_len, np.int32)
    inst = _c(inst_of, np.int32)
    g = np.asarray(gain, dtype=object)
    N, n = g.shape
    pairs = np.empty((N, n, 2), np.int64)
    flat = g.reshape(-1)
    pv = pairs.reshape(-1, 2)
    for e, v in enumerate(flat):
        u = int(v) & ((1 << 128) - 1)
        lo, hi = u & ((1 << 64) - 1), u >> 64
        pv[e, 0] = lo - (1 << 64) if lo >= (1 << 63) else lo
        pv[e, 1] = hi - (1 << 64) if hi >= (1 << 63) else hi
    bt = np.empty(N, np.int32)
    bg = np.empty((N, 2), np.int64)
    mv = np.empty(3, np.int32)
    mg = np.empty(2, np.int64)
    rc = _load().star_oracle_select_variance(N, n, _ptr(cur), _ptr(rem), _ptr(inst), _ptr(pairs),
                                             _ptr(bt), _ptr(bg), _ptr(mv), _ptr(mg))
    if rc != 0:
        raise ValueError("star_oracle_select_variance: malformed arguments")
    return {"best_target": bt, "best_gain": i128_values(bg), "move": tuple(int(x) for x in mv),
            "move_gain": int(i128_values(mg))}


def plan(cur_len, rem_len, inst_of, beta, *, n_inst: int, bucket: int, n_buckets: int,
         theta=(0, 1), u_mode: int = 0, min_rem: int = 0, mem_cap: int = (1 << 62),
         mem_mode: int = 0, max_moves: int = 1):
    """Algorithm 1 repeated up to ``max_moves`` times.

    Returns dict(moves [(r, s, t)], gains [int], inst_of (final), load (final)).
    """
    cur = _c(cur_len, np.int32)
    rem = _c(rem_len, np.int32)
    inst = np.array(inst_of, dtype=np.int32, copy=True)
    beta = _c(beta, np.uint16)
    N = cur.shape[0]
    load = np.empty((n_inst, n_buckets), np.int64)
    moves = np.empty((max(max_moves, 1), 3), np.int32)
    gains = np.empty((max(max_moves, 1), 2), np.int64)
    cnt = np.zeros(1, np.int64)
    rc = _load().star_oracle_plan(N, n_inst, bucket, n_buckets, _ptr(cur), _ptr(rem), _ptr(inst),
                                  _ptr(load), _ptr(beta), int(theta[0]), int(theta[1]),
                                  int(u_mode), int(min_rem), int(mem_cap), int(mem_mode),
                                  int(max_moves), _ptr(moves), _ptr(gains), _ptr(cnt))
    if rc == -2:
        raise OverflowError("star_oracle_plan: values beyond the exact range")
    if rc != 0:
        raise ValueError(f"star_oracle_plan failed ({rc})")
    m = int(cnt[0])
    return {"moves": [tuple(int(x) for x in moves[q]) for q in range(m)],
            "gains": [int(v) for v in i128_values(gains[:m])] if m else [],
            "inst_of": inst, "load": load}
