"""Seeded synthetic inputs for the STAR rescheduling hot path.

This module is the only code shared by the HIP path's callers and the CPU
oracle's callers.  It draws random numbers and shapes them into the arrays a
rescheduling round consumes; it holds none of the method's arithmetic (no
predictor, no load projection, no scoring).

Five decode-batch workloads: a tiny fp32 case; an 8B-class batch; a
32B-class long-reasoning mix; continuous mode over 200 decode steps; a
64-instance rebalancing scan.  The
paper's own workloads are ShareGPT / Alpaca outputs of DeepSeek-R1-Distill
(Section 6.1, Table 2); those datasets and models are not used: lognormal,
lognormal-mixture and Pareto draws of the remaining length stand in for them.

Conventions
-----------
* One child stream of ``SeedSequence(seed)`` per array, spawned in the fixed
  order ``hidden, w1, w2, b1, b2, cur_len, true_len, ar_innovations``.
* bf16 arrays are carried as ``uint16`` bit patterns, rounded from fp32 by
  round-to-nearest-even, so that every consumer sees identical bits.
* Instances are contiguous blocks of ``n_req // n_inst`` requests.
* Lognormal(mu, sigma) = exp(N(mu, sigma^2)); Pareto(alpha, x_min) is the
  type-I law ``x_min * U**(-1/alpha)`` with U uniform on (0, 1].  Every length
  draw is clipped to its cap, rounded half-to-even and raised to at least 1.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

STREAMS = ("hidden", "w1", "w2", "b1", "b2", "cur_len", "true_len", "ar_innovations")

F32 = 0
BF16 = 1
ACT_RELU = 0
ACT_GELU = 1


# --------------------------------------------------------------------------
# bf16 bit helpers (input preparation only)
# --------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); return uint16 bits.

    Inputs are finite; NaN/Inf payloads are not special-cased.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# --------------------------------------------------------------------------
# configurations
# --------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n_req: int          # B = N
    d_model: int        # d
    d_hidden: int       # m
    n_bins: int         # nb
    bin_lo: float
    bin_hi: float
    dtype: int          # F32 or BF16 (hidden, w1, w2)
    act: int            # ACT_RELU or ACT_GELU
    n_inst: int         # n
    horizon: int        # H
    bucket: int         # b
    cur_lo: int
    cur_hi: int
    true_len: Optional[str]   # law of the true remaining length, or None
    true_cap: int
    steps: int = 1            # decode steps (continuous mode)
    ar_rho: float = 0.0       # AR(1) correlation of hidden states across steps
    ema_alpha: float = 0.0
    top_k: int = 256

    @property
    def n_buckets(self) -> int:
        return self.horizon // self.bucket

    @property
    def len_max(self) -> int:
        return int(round(self.bin_hi))


WORKLOADS = {
    "tiny": Workload("tiny", 64, 1024, 256, 32, 1.0, 4096.0, F32, ACT_RELU,
                     4, 4096, 1, 1, 2048, None, 4096),
    "8b_batch": Workload("8b_batch", 512, 4096, 512, 64, 1.0, 16384.0, BF16, ACT_GELU,
                         8, 16384, 64, 128, 8192, "lognormal(7,1)", 16384),
    "32b_long_mix": Workload("32b_long_mix", 4096, 5120, 512, 64, 1.0, 32768.0, BF16, ACT_GELU,
                             16, 32768, 64, 256, 16384,
                             "0.7*lognormal(6,0.8)+0.3*lognormal(9,0.5)", 32768),
    "continuous": Workload("continuous", 1024, 4096, 512, 64, 1.0, 16384.0, BF16, ACT_GELU,
                           8, 16384, 64, 128, 8192, "lognormal(7,1)", 16384,
                           steps=200, ar_rho=0.95, ema_alpha=0.2),
    "rebalance_scan": Workload("rebalance_scan", 32768, 8192, 1024, 128, 1.0, 65536.0, BF16,
                               ACT_GELU, 64, 65536, 64, 1, 32768, "pareto(1.5,64)", 65536),
}
# the five workloads in the order they are listed for this hot path
WORKLOAD_ORDER = ("tiny", "8b_batch", "32b_long_mix", "continuous", "rebalance_scan")


def bin_values(n_bins: int, lo: float, hi: float) -> np.ndarray:
    """Log-spaced representative lengths v_0..v_{nb-1} from lo to hi (fp32).

    v_k = lo * (hi/lo)**(k/(nb-1)) evaluated in fp64, rounded to fp32, with
    both endpoints set exactly.
    """
    if n_bins == 1:
        return np.array([lo], dtype=np.float32)
    k = np.arange(n_bins, dtype=np.float64)
    v = lo * (hi / lo) ** (k / (n_bins - 1))
    v = v.astype(np.float32)
    v[0] = np.float32(lo)
    v[-1] = np.float32(hi)
    return v


def bucket_weights(n_buckets: int, halvings: float = 8.0) -> np.ndarray:
    """Bucket weights beta_k for the time-weighted variance objective (uint16).

    beta_k = max(1, round(65535 * 2**(-halvings * k / K))): full weight now,
    halving every K/halvings buckets, so the far horizon still counts.
    """
    k = np.arange(n_buckets, dtype=np.float64)
    w = np.rint(65535.0 * np.exp2(-halvings * k / max(n_buckets, 1)))
    return np.maximum(w, 1.0).astype(np.uint16)


def _streams(seed: int):
    children = np.random.SeedSequence(seed).spawn(len(STREAMS))
    return {name: np.random.default_rng(c) for name, c in zip(STREAMS, children)}


def _finish_lengths(x: np.ndarray, cap: int) -> np.ndarray:
    x = np.clip(x, 1.0, float(cap))
    return np.maximum(np.rint(x), 1).astype(np.int32)


def draw_true_len(rng: np.random.Generator, law: str, n: int, cap: int) -> np.ndarray:
    if law == "lognormal(7,1)":
        x = rng.lognormal(7.0, 1.0, size=n)
    elif law == "0.7*lognormal(6,0.8)+0.3*lognormal(9,0.5)":
        pick = rng.random(size=n) < 0.7
        a = rng.lognormal(6.0, 0.8, size=n)
        b = rng.lognormal(9.0, 0.5, size=n)
        x = np.where(pick, a, b)
    elif law == "pareto(1.5,64)":
        u = 1.0 - rng.random(size=n)            # (0, 1]
        x = 64.0 * u ** (-1.0 / 1.5)
    elif law == "long_output_stress":
        # Shape taken from published output-length statistics only: a light
        # lognormal body plus a block of near-cap outputs (Section 2.2 and Table 2).
        pick = rng.random(size=n) < 0.827
        a = rng.lognormal(7.16, 0.67, size=n)
        b = rng.uniform(30000.0, 32768.0, size=n)
        x = np.where(pick, a, b)
    else:
        raise ValueError(f"unknown length law {law!r}")
    return _finish_lengths(x, cap)


def _weights(rng, shape, fan_in, dtype):
    w = (rng.standard_normal(size=shape, dtype=np.float32) * np.float32(1.0 / np.sqrt(fan_in)))
    return f32_to_bf16_bits(w) if dtype == BF16 else w.astype(np.float32)


def _hidden_f32(rng, shape):
    return rng.standard_normal(size=shape, dtype=np.float32)


@dataclasses.dataclass
class Inputs:
    wl: Workload
    hidden: np.ndarray             # [B, d] (steps==1) or [S, B, d]; uint16 bits or float32
    w1: np.ndarray                 # [m, d]
    w2: np.ndarray                 # [nb, m]
    b1: Optional[np.ndarray]       # [m] float32 or None
    b2: Optional[np.ndarray]       # [nb] float32 or None
    bin_values: np.ndarray         # [nb] float32
    cur_len: np.ndarray            # [N] int32 (at step 0)
    true_len: Optional[np.ndarray] # [N] int32 or None
    inst_of: np.ndarray            # [N] int32


def make_inputs(wl: Workload, seed: int = 0, *, with_bias: bool = False,
                steps: Optional[int] = None, n_req: Optional[int] = None,
                w2_scale: float = 1.0) -> Inputs:
    """Draw one workload's inputs.

    ``steps`` overrides the number of decode steps staged for continuous
    mode; ``n_req`` draws only the first rows of the hidden states (the
    per-request arrays keep the full batch).  ``w2_scale`` multiplies the
    second-layer weights before rounding (peaky-softmax stress).
    """
    rs = _streams(seed)
    B, d, m, nb = wl.n_req, wl.d_model, wl.d_hidden, wl.n_bins
    rows = B if n_req is None else n_req
    S = wl.steps if steps is None else steps

    h_rng = rs["hidden"]
    if wl.ar_rho > 0.0 and S > 1:
        hidden = np.empty((S, rows, d), dtype=np.uint16 if wl.dtype == BF16 else np.float32)
        state = _hidden_f32(h_rng, (rows, d))
        eps_rng = rs["ar_innovations"]
        rho = np.float32(wl.ar_rho)
        sig = np.float32(np.sqrt(1.0 - wl.ar_rho ** 2))
        for s in range(S):
            if s > 0:
                state = rho * state + sig * _hidden_f32(eps_rng, (rows, d))
            hidden[s] = f32_to_bf16_bits(state) if wl.dtype == BF16 else state
    else:
        h = _hidden_f32(h_rng, (rows, d))
        hidden = f32_to_bf16_bits(h) if wl.dtype == BF16 else h

    w1 = _weights(rs["w1"], (m, d), d, wl.dtype)
    w2f = rs["w2"].standard_normal(size=(nb, m), dtype=np.float32) * np.float32(w2_scale / np.sqrt(m))
    w2 = f32_to_bf16_bits(w2f) if wl.dtype == BF16 else w2f.astype(np.float32)
    b1 = b2 = None
    if with_bias:
        b1 = (rs["b1"].standard_normal(size=m, dtype=np.float32) * np.float32(0.1)).astype(np.float32)
        b2 = (rs["b2"].standard_normal(size=nb, dtype=np.float32) * np.float32(0.1)).astype(np.float32)

    cur = rs["cur_len"].integers(wl.cur_lo, wl.cur_hi, endpoint=True, size=B).astype(np.int32)
    true = None
    if wl.true_len is not None:
        true = draw_true_len(rs["true_len"], wl.true_len, B, wl.true_cap)
    inst = (np.arange(B, dtype=np.int64) // (B // wl.n_inst)).astype(np.int32)
    return Inputs(wl, hidden, w1, w2, b1, b2, bin_values(nb, wl.bin_lo, wl.bin_hi),
                  cur, true, inst)


@dataclasses.dataclass
class Mlp4Inputs:
    hidden: np.ndarray             # [B, d] or [S, B, d]; uint16 bits (bf16) or float32
    w1: np.ndarray                 # [m1, d]
    w2: np.ndarray                 # [m2, m1]
    w3: np.ndarray                 # [m3, m2]
    w4: np.ndarray                 # [m3] float32
    b1: Optional[np.ndarray]
    b2: Optional[np.ndarray]
    b3: Optional[np.ndarray]
    b4: float


MLP4_DIMS = (3584, 2048, 512, 64)   # d and the three widths of the paper's head (Section 4.2)


def make_mlp4(n_req: int, dims=MLP4_DIMS, *, dtype: int = BF16, seed: int = 0, steps: int = 1,
              ar_rho: float = 0.95, with_bias: bool = False, y_mean: float = 1100.0,
              y_spread: float = 400.0) -> Mlp4Inputs:
    """Random-initialised regression head of the paper's shape and hidden
    states for it.  W1..W3 ~ N(0, 2/fan_in) (ReLU-preserving scale); w4 ~
    N(0, (y_spread)^2 / m3) and b4 = y_mean put the outputs at realistic
    remaining lengths.  Hidden states: N(0,1), an AR(1) chain over `steps`
    decode steps (as the continuous workload)."""
    d, m1, m2, m3 = dims
    children = np.random.SeedSequence(seed).spawn(9)
    rs = [np.random.default_rng(c) for c in children]

    def mat(rng, shape, fan_in):
        w = rng.standard_normal(size=shape, dtype=np.float32) * np.float32(np.sqrt(2.0 / fan_in))
        return f32_to_bf16_bits(w) if dtype == BF16 else w

    if steps > 1:
        hidden = np.empty((steps, n_req, d), dtype=np.uint16 if dtype == BF16 else np.float32)
        state = rs[0].standard_normal(size=(n_req, d), dtype=np.float32)
        sig = np.float32(np.sqrt(1.0 - ar_rho ** 2))
        for t in range(steps):
            if t > 0:
                state = np.float32(ar_rho) * state + sig * rs[1].standard_normal(
                    size=(n_req, d), dtype=np.float32)
            hidden[t] = f32_to_bf16_bits(state) if dtype == BF16 else state
    else:
        h = rs[0].standard_normal(size=(n_req, d), dtype=np.float32)
        hidden = f32_to_bf16_bits(h) if dtype == BF16 else h
    w1, w2, w3 = mat(rs[2], (m1, d), d), mat(rs[3], (m2, m1), m1), mat(rs[4], (m3, m2), m2)
    w4 = (rs[5].standard_normal(size=m3) * (y_spread / np.sqrt(m3))).astype(np.float32)
    b1 = b2 = b3 = None
    if with_bias:
        b1 = (rs[6].standard_normal(size=m1) * 0.1).astype(np.float32)
        b2 = (rs[7].standard_normal(size=m2) * 0.1).astype(np.float32)
        b3 = (rs[8].standard_normal(size=m3) * 0.1).astype(np.float32)
    return Mlp4Inputs(hidden, w1, w2, w3, w4, b1, b2, b3, float(y_mean))


def random_requests(rng: np.random.Generator, n_req: int, n_inst: int, *, cur_hi: int,
                    len_hi: int, contiguous: bool = False, empty_inst: int = 0):
    """Small random (cur_len, rem_len, inst_of) triples for parity and pin tests.

    ``empty_inst`` instances at the top of the range receive no requests.
    """
    cur = rng.integers(1, cur_hi, endpoint=True, size=n_req).astype(np.int32)
    rem = rng.integers(1, len_hi, endpoint=True, size=n_req).astype(np.int32)
    live = max(1, n_inst - empty_inst)
    if contiguous:
        inst = (np.arange(n_req) * live // max(n_req, 1)).astype(np.int32)
    else:
        inst = rng.integers(0, live, size=n_req).astype(np.int32)
    return cur, rem, inst
