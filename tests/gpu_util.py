"""Shared helpers of the GPU parity tests: device staging and one-call runners
for libstar's three entry points (through the C-ABI binding)."""
from __future__ import annotations

import numpy as np
import torch

from paper_2510_13668_amd import star, synth

DEV = "cuda"
E_RTOL = 2e-2        # predicted-length tolerance (relative): the contract
# A sharper bound the arithmetic supports: with bf16-exact operands (exact
# fp32 products), fp32 accumulation and a1 carried as a bf16 hi/lo pair
# (about 2^-16 relative), a logit's error is at most sum_j |w2_j| |da1_j|,
# about rms(W2) sqrt(m) max|da1|; since d log p_k / dz = e_k - p, E's
# relative error is at most twice the largest absolute logit error.  E_TIGHT
# applies at unit weight scale (W2 ~ N(0, 1/m)); tests scale it by the norm
# they use.
E_TIGHT = 1e-3


def w2_scale(w2, dtype) -> float:
    """rms(W2) sqrt(m): 1 for W2 ~ N(0, 1/m)."""
    w = synth.bf16_bits_to_f32(w2) if dtype == synth.BF16 else np.asarray(w2, np.float32)
    return float(np.sqrt(np.mean(np.square(w.astype(np.float64)))) * np.sqrt(w.shape[1]))


def to_dev(a: np.ndarray, bf16: bool = False) -> torch.Tensor:
    if bf16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def opt_dev(a):
    return None if a is None else to_dev(a)


class Predictor:
    """Device copies of one head's weights plus its workspace."""

    def __init__(self, w1, w2, bins, *, dtype, act, b1=None, b2=None, n_req, len_max,
                 ema_alpha=0.0):
        bf = dtype == synth.BF16
        self.w1 = to_dev(w1, bf)
        self.w2 = to_dev(w2, bf)
        self.b1 = opt_dev(b1)
        self.b2 = opt_dev(b2)
        self.bins = to_dev(bins)
        self.m, self.d = w1.shape
        self.nb = w2.shape[0]
        self.dtype, self.act, self.len_max, self.alpha = dtype, act, len_max, ema_alpha
        self.n_req = n_req
        p = self.params(False)
        self.ws = star.Workspace(star.predict_workspace_size(p))
        self.ema = torch.zeros(n_req, dtype=torch.float32, device=DEV)
        self.expected = torch.empty(n_req, dtype=torch.float32, device=DEV)
        self.rem = torch.empty(n_req, dtype=torch.int32, device=DEV)

    def params(self, ema_init):
        return star.predict_params(self.n_req, self.d, self.m, self.nb, self.dtype, self.act,
                                   self.alpha, ema_init, self.len_max)

    def run(self, hidden_dev: torch.Tensor, ema_init=False, stream=None):
        star.predict(self.params(ema_init), hidden_dev, self.w1, self.b1, self.w2, self.b2,
                     self.bins, self.ema if self.alpha > 0 else None, self.expected, self.rem,
                     self.ws, stream)


class Rescheduler:
    """Buffers and workspaces for (b) and (c) at fixed sizes.  fused: one
    star_project_and_score call per round (one workspace) instead of
    star_project_load then star_score_migrations."""

    def __init__(self, n_req, n_inst, bucket, n_buckets, top_k, want_scores=True, fused=False):
        self.lp = star.load_params(n_req, n_inst, bucket, n_buckets)
        self.sp = star.score_params(n_req, n_inst, bucket, n_buckets, top_k)
        self.fused = fused
        if fused:
            self.ws_load = self.ws_score = star.Workspace(
                star.project_and_score_workspace_size(self.sp))
        else:
            self.ws_load = star.Workspace(star.project_load_workspace_size(self.lp))
            self.ws_score = star.Workspace(star.score_workspace_size(self.sp))
        self.load = torch.empty((n_inst, n_buckets), dtype=torch.int64, device=DEV)
        self.scores = (torch.empty((n_req, n_inst), dtype=torch.int64, device=DEV)
                       if want_scores else None)
        self.best_target = torch.empty(n_req, dtype=torch.int32, device=DEV)
        self.best_score = torch.empty(n_req, dtype=torch.int64, device=DEV)
        k = max(top_k, 1)
        self.top_k = top_k
        self.tr = torch.empty(k, dtype=torch.int32, device=DEV) if top_k else None
        self.tt = torch.empty(k, dtype=torch.int32, device=DEV) if top_k else None
        self.ts = torch.empty(k, dtype=torch.int64, device=DEV) if top_k else None

    def run(self, cur, rem, inst, stream=None):
        if self.fused:
            star.project_and_score(self.sp, cur, rem, inst, self.load, self.scores,
                                   self.best_target, self.best_score, self.tr, self.tt, self.ts,
                                   self.ws_score, stream)
            return
        star.project_load(self.lp, cur, rem, inst, self.load, self.ws_load, stream)
        star.score_migrations(self.sp, cur, rem, inst, self.load, self.scores, self.best_target,
                              self.best_score, self.tr, self.tt, self.ts, self.ws_score, stream)

    def result(self):
        torch.cuda.synchronize()
        out = {"load": self.load.cpu().numpy(), "best_target": self.best_target.cpu().numpy(),
               "best_score": self.best_score.cpu().numpy()}
        if self.scores is not None:
            out["scores"] = self.scores.cpu().numpy()
        if self.top_k:
            out["topk_req"] = self.tr.cpu().numpy()[: self.top_k]
            out["topk_tgt"] = self.tt.cpu().numpy()[: self.top_k]
            out["topk_score"] = self.ts.cpu().numpy()[: self.top_k]
        return out


def assert_round_equal(gpu: dict, ref: dict):
    for k in ("load", "scores", "best_target", "best_score", "topk_req", "topk_tgt", "topk_score"):
        if k in gpu:
            np.testing.assert_array_equal(gpu[k], ref[k], err_msg=k)


def assert_lengths_close(e_gpu, e_ref, rtol=E_RTOL, what="expected length"):
    e_gpu = np.asarray(e_gpu, np.float64)
    rel = np.abs(e_gpu - e_ref) / np.abs(e_ref)
    assert np.all(np.isfinite(e_gpu)), what
    assert rel.max() <= rtol, f"{what}: max rel err {rel.max():.3e} at {int(rel.argmax())}"
    return float(rel.max())
