"""star_predict_noalloc (the predictor without a workspace: its scratch is
the library's fixed device array) against star_predict on the same inputs,
through the C ABI: bit-identical outputs (same plan, same kernels, both
deterministic) and within the 2e-2 contract of the fp64 oracle, on several
calls in a row, the second smaller than the first, and a third that takes
the fused one-slice kernel (whose counters live in the array's header)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2510_13668_amd import star, synth
from gpu_util import assert_lengths_close, to_dev

pytestmark = pytest.mark.gpu


def _inputs(B, d, m, nb, seed):
    rng = np.random.default_rng(seed)
    h = synth.f32_to_bf16_bits(rng.standard_normal((B, d)).astype(np.float32))
    w1 = synth.f32_to_bf16_bits((rng.standard_normal((m, d)) / np.sqrt(d)).astype(np.float32))
    w2 = synth.f32_to_bf16_bits((rng.standard_normal((nb, m)) * 4 / np.sqrt(m)).astype(np.float32))
    b1 = (rng.standard_normal(m) * 0.1).astype(np.float32)
    b2 = (rng.standard_normal(nb) * 0.1).astype(np.float32)
    ema0 = rng.uniform(100.0, 5000.0, B).astype(np.float32)
    return h, w1, w2, b1, b2, synth.bin_values(nb, 1.0, 16384.0), ema0


def _run_both(B, d, m, nb, seed):
    h, w1, w2, b1, b2, bins, ema0 = _inputs(B, d, m, nb, seed)
    dev = lambda a: torch.from_numpy(a).cuda()
    H, W1, W2 = to_dev(h, True), to_dev(w1, True), to_dev(w2, True)
    B1, B2, BINS = dev(b1), dev(b2), dev(bins)
    p = star.predict_params(B, d, m, nb, synth.BF16, synth.ACT_GELU, 0.2, False, 16384)
    outs = []
    for noalloc in (False, True):
        ema = dev(ema0.copy())
        e = torch.empty(B, dtype=torch.float32, device="cuda")
        r = torch.empty(B, dtype=torch.int32, device="cuda")
        if noalloc:
            star.predict_noalloc(p, H, W1, B1, W2, B2, BINS, ema, e, r)
        else:
            ws = star.Workspace(star.predict_workspace_size(p))
            star.predict(p, H, W1, B1, W2, B2, BINS, ema, e, r, ws)
        torch.cuda.synchronize()
        outs.append((e.cpu().numpy(), ema.cpu().numpy(), r.cpu().numpy()))
    for a, b in zip(*outs):
        np.testing.assert_array_equal(a, b)
    rows = np.unique(np.concatenate([np.arange(min(B, 40)), np.arange(max(0, B - 40), B)]))
    state = ema0[rows].astype(np.float64)
    ref = oracle.predict(h[rows], w1, w2, bins, dtype=synth.BF16, act=synth.ACT_GELU, b1=b1,
                         b2=b2, ema_alpha=0.2, ema_init=False, ema_state=state, len_max=16384)
    assert_lengths_close(outs[1][0][rows], ref["expected"])
    assert_lengths_close(outs[1][1][rows], state, what="ema")


def test_noalloc_matches_predict_on_successive_calls():
    for c, (B, d, m, nb) in enumerate([(1024, 4096, 512, 64),    # 4 K-splits: partial planes
                                       (200, 512, 256, 40),      # smaller, after a larger one
                                       (8192, 512, 512, 64)]):   # one K-slice: fused kernel
        print(f"noalloc call {c}: B={B} d={d} m={m} nb={nb}", flush=True)
        _run_both(B, d, m, nb, seed=c)


def test_noalloc_refuses_sizes_beyond_its_scratch():
    # 32768 rows at m = 1024 need 128 MiB of partials: refused before any launch
    L = star.lib()
    p = star.predict_params(32768, 8192, 1024, 128, synth.BF16, synth.ACT_GELU, 0.0, False, 65536)
    t = torch.empty(16, dtype=torch.float32, device="cuda")
    st = L.star_predict_noalloc(star.ctypes.byref(p), star._ptr(t), star._ptr(t), None,
                                star._ptr(t), None, star._ptr(t), None, star._ptr(t), None, None)
    assert st == star.STAR_ERR_SCRATCH_LIMIT
