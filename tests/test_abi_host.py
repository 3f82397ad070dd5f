"""Host-side contract of libstar.so: symbols and synchronous validation.

No test here launches a kernel: every call below is rejected by the scalar
checks that run before anything is enqueued, so the suite runs without a GPU.
"""
import ctypes
import os
import re

import pytest

from paper_2510_13668_amd import star

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "star.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(star.LIB_PATH):
        from paper_2510_13668_amd import build
        build.build()
    return star.lib()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(star_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(L):
    names = _declared_functions()
    assert {"star_predict", "star_project_load", "star_score_migrations"} <= set(names)
    for n in names:
        assert hasattr(L, n), n


def test_abi_version_and_status_strings(L):
    assert L.star_abi_version() == 2
    for s in (0, -1, -2, -3, -4, -5, -6, -7):
        assert L.star_status_string(s).decode().startswith("STAR_")
    assert b"unknown" in L.star_status_string(-99)


def _pp(**kw):
    base = dict(n_req=1024, d_model=4096, d_hidden=512, n_bins=64, dtype=star.BF16,
                act=star.ACT_GELU, ema_alpha=0.2, ema_init=False, len_max=16384)
    base.update(kw)
    return star.predict_params(**base)


FAKE = ctypes.c_void_p(1 << 20)   # never dereferenced: validation fails first


def _predict(L, p, ws_bytes=1 << 30, ws=FAKE, **ptrs):
    args = {k: FAKE for k in ("hidden", "w1", "w2", "bins", "ema", "expected")}
    args["b1"] = None
    args.update(ptrs)
    return L.star_predict(ctypes.byref(p) if p is not None else None, args["hidden"], args["w1"],
                          args["b1"], args["w2"], None, args["bins"], args["ema"],
                          args["expected"], None, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(n_req=-1), -1), (dict(d_model=0), -1), (dict(d_hidden=0), -1), (dict(n_bins=0), -1),
    (dict(dtype=7), -1), (dict(act=3), -1), (dict(ema_alpha=1.5), -1),
    (dict(ema_alpha=float("nan")), -1), (dict(len_max=0), -1),
    (dict(d_model=4100), -2), (dict(d_hidden=3000), -2), (dict(n_bins=300), -2),
    (dict(d_hidden=516), -2),
])
def test_predict_rejects_bad_scalars(L, kw, status):
    assert _predict(L, _pp(**kw)) == status


def test_predict_rejects_null_pointers_and_workspace(L):
    assert _predict(L, None) == -1
    assert _predict(L, _pp(), hidden=None) == -1
    assert _predict(L, _pp(ema_alpha=0.2), ema=None) == -1
    assert _predict(L, _pp(), hidden=ctypes.c_void_p((1 << 20) + 2)) == -2   # misaligned
    # b1 is read 16 bytes at a time: a bias view at a 4-byte offset is refused
    assert _predict(L, _pp(), b1=ctypes.c_void_p((1 << 20) + 4)) == -2
    p = _pp()
    need = star.predict_workspace_size(p)
    # 64 x 64 tiles, 4 K-splits: the split-K product writes 4 fp32 partial
    # planes of [1024, 512] for the head kernel, plus the header
    assert need == star.STAR_WS_HEADER_BYTES + 4 * 1024 * 512 * 4
    # one K-slice (8192 x 512 x 4096, 128 x 128 tiles, 4 column tiles): the
    # fused kernel's logit shares [64 row blocks][4][128 x 64] fp32
    big = _pp(n_req=8192)
    assert star.predict_workspace_size(big) == star.STAR_WS_HEADER_BYTES + 4 * 8192 * 64 * 4
    assert _predict(L, p, ws_bytes=need - 1) == -4
    assert _predict(L, p, ws=None) == -4
    assert _predict(L, p, ws=ctypes.c_void_p((1 << 20) + 64)) == -4   # not 256-aligned


def _overlap(L, p, hidden=FAKE, ws_next=FAKE, ws_prev=ctypes.c_void_p((1 << 20) + (1 << 26)),
             ws_bytes=1 << 24, **ptrs):
    args = {k: FAKE for k in ("w1", "w2", "bins", "ema", "expected")}
    args.update(ptrs)
    return L.star_predict_overlap(ctypes.byref(p) if p is not None else None, hidden, ws_next,
                                  ws_prev, args["w1"], None, args["w2"], None, args["bins"],
                                  args["ema"], args["expected"], None, ws_bytes, None)


def test_predict_overlap_validation(L):
    """The two-batch predictor call validates each side it is given, before
    launching anything.  Its workspace is star_predict's, except for
    one-slice products, which it runs as a product and a head (one fp32
    partial plane) instead of the fused kernel (logit shares)."""
    p = _pp()
    need = star.predict_overlap_workspace_size(p)
    assert need == star.predict_workspace_size(p)
    one = _pp(n_req=8192)                                            # one K-slice
    assert star.predict_overlap_workspace_size(one) == star.STAR_WS_HEADER_BYTES + 8192 * 512 * 4
    assert star.predict_overlap_workspace_size(one) > star.predict_workspace_size(one)
    assert _overlap(L, one, ws_bytes=star.predict_workspace_size(one)) == -4
    assert star.predict_overlap_workspace_size(_pp(n_req=-1)) == 0
    assert _overlap(L, None) == -1
    assert _overlap(L, p, hidden=None, ws_prev=None) == -1          # neither side
    assert _overlap(L, p, ws_bytes=need - 1) == -4
    assert _overlap(L, p, ws_next=None) == -4                        # product without a workspace
    assert _overlap(L, p, ws_prev=ctypes.c_void_p((1 << 20) + (1 << 26) + 64)) == -4
    assert _overlap(L, p, ws_prev=ctypes.c_void_p((1 << 20) + 256), ws_bytes=need) == -1
    assert _overlap(L, p, w1=None) == -1                              # product needs w1
    assert _overlap(L, p, hidden=None, w1=None, expected=None) == -1  # head needs its outputs
    assert _overlap(L, p, ema=None) == -1                             # EMA on, no state
    assert _overlap(L, p, hidden=ctypes.c_void_p((1 << 20) + 2)) == -2


def test_predict_noalloc_validation_and_scratch_limit(L):
    """The allocation-free predictor validates like star_predict and refuses,
    before launching anything, sizes whose scratch exceeds its fixed array
    (32768 rows at m = 1024 need 128 MiB of split-K partials)."""
    def call(p, **ptrs):
        a = {k: FAKE for k in ("hidden", "w1", "w2", "bins", "ema", "expected")}
        a.update(ptrs)
        return L.star_predict_noalloc(ctypes.byref(p) if p is not None else None, a["hidden"],
                                      a["w1"], None, a["w2"], None, a["bins"], a["ema"],
                                      a["expected"], None, None)
    assert call(None) == -1
    assert call(_pp(n_bins=0)) == -1
    assert call(_pp(), hidden=None) == -1
    assert call(_pp(), w1=ctypes.c_void_p((1 << 20) + 8)) == -2
    big = _pp(n_req=32768, d_model=8192, d_hidden=1024, n_bins=128)
    assert call(big) == star.STAR_ERR_SCRATCH_LIMIT == -7
    assert L.star_status_string(-7).decode().startswith("STAR_ERR_SCRATCH_LIMIT")


def test_load_and_score_validation(L):
    lp = star.load_params(1024, 8, 64, 256)
    assert star.project_load_workspace_size(lp) == star.STAR_WS_HEADER_BYTES
    # long streams (8192+ requests, at most 1024 buckets, at most 960
    # instances) keep one histogram triple per (instance, request slice):
    # 32768 requests on 64 instances take 4 slices of 8192
    H = star.STAR_WS_HEADER_BYTES
    big_lp = star.load_params(32768, 64, 64, 1024)
    assert star.project_load_workspace_size(big_lp) == H + 64 * 4 * 3 * 1026 * 8
    assert star.project_load_workspace_size(star.load_params(32768, 64, 64, 1025)) == H
    assert star.project_load_workspace_size(star.load_params(32768, 961, 64, 1024)) == H
    assert star.project_load_workspace_size(star.load_params(8191, 64, 64, 1024)) == H
    # 16384 requests on 16 instances: 8 slices of 2048
    assert star.project_load_workspace_size(star.load_params(16384, 16, 64, 512)) == (
        H + 16 * 8 * 3 * 514 * 8)
    assert L.star_project_load(ctypes.byref(big_lp), f := FAKE, f, f, f, f,
                               H + 64 * 4 * 3 * 1026 * 8 - 1, None) == -4
    f = FAKE
    assert L.star_project_load(ctypes.byref(star.load_params(1, 0, 1, 1)), f, f, f, f, f, 256, None) == -1
    assert L.star_project_load(ctypes.byref(star.load_params(1, 1, 0, 1)), f, f, f, f, f, 256, None) == -1
    assert L.star_project_load(ctypes.byref(lp), None, f, f, f, f, 256, None) == -1
    assert L.star_project_load(ctypes.byref(lp), f, f, f, None, f, 256, None) == -1
    assert L.star_project_load(ctypes.byref(lp), f, f, f, f, f, 255, None) == -4
    # horizon above 2^30 steps
    assert L.star_project_load(ctypes.byref(star.load_params(1, 1, 1 << 16, 1 << 15)), f, f, f, f, f,
                               256, None) == -2
    # (N+1) b (2^31 + H) >= 2^62
    big = star.load_params(1 << 26, 8, 64, 256)
    assert L.star_project_load(ctypes.byref(big), f, f, f, f, f, 256, None) == -3

    # ranking keeps per-workgroup sorted keys (or scores and best moves, and
    # the curve planes for large curve sets) in the workspace; a round that
    # one workgroup takes whole (up to 1024 requests on up to 8 instances,
    # curves in LDS) needs only the header
    H = star.STAR_WS_HEADER_BYTES
    assert star.score_workspace_size(star.score_params(1024, 8, 64, 256, 0)) == H
    assert star.score_workspace_size(star.score_params(1024, 8, 64, 256, 256)) == H
    assert star.score_workspace_size(star.score_params(1025, 8, 64, 256, 256)) > H
    assert star.score_workspace_size(star.score_params(1024, 9, 64, 256, 256)) > H
    sp = star.score_params(4096, 16, 64, 512, 256)
    need = star.score_workspace_size(sp)
    assert need > H
    args = [f] * 10
    assert L.star_score_migrations(ctypes.byref(sp), *args, f, need - 1, None) == -4
    nk = star.score_params(1024, 8, 64, 256, 0)
    # top-k outputs must be NULL iff top_k == 0
    assert L.star_score_migrations(ctypes.byref(nk), *args, f, 1 << 30, None) == -1
    assert L.star_score_migrations(ctypes.byref(sp), *args[:7], None, f, f, f, 1 << 30, None) == -1
    assert L.star_score_migrations(ctypes.byref(star.score_params(4, 2, 1, 1, 2000)), *args, f,
                                   1 << 30, None) == -1
    assert L.star_score_migrations(ctypes.byref(star.score_params(4, 5000, 1, 1, 1)), *args, f,
                                   1 << 30, None) == -2


def test_project_and_score_validation(L):
    f = FAKE
    sp = star.score_params(1024, 8, 64, 256, 256)
    need = star.project_and_score_workspace_size(sp)
    # the same workspace layout as scoring alone
    assert need == star.score_workspace_size(sp)
    # with the split projection, its histograms follow the scoring's scratch
    big = star.score_params(32768, 64, 64, 1024, 256)
    assert star.project_and_score_workspace_size(big) == (
        star.score_workspace_size(big) + 64 * 4 * 3 * 1026 * 8)
    args = [f] * 10
    assert L.star_project_and_score(None, *args, f, need, None) == -1
    assert L.star_project_and_score(ctypes.byref(sp), *args, f, need - 1, None) == -4
    assert L.star_project_and_score(ctypes.byref(sp), *args, None, need, None) == -4
    # load is an output here and may not be NULL
    assert L.star_project_and_score(ctypes.byref(sp), f, f, f, None, *args[4:], f, need,
                                    None) == -1
    # top-k outputs must be NULL iff top_k == 0
    nk = star.score_params(1024, 8, 64, 256, 0)
    assert L.star_project_and_score(ctypes.byref(nk), *args, f, 1 << 30, None) == -1
    assert L.star_project_and_score(ctypes.byref(sp), *args[:7], None, f, f, f, 1 << 30,
                                    None) == -1
    assert L.star_project_and_score(ctypes.byref(star.score_params(4, 5000, 1, 1, 1)), *args, f,
                                    1 << 30, None) == -2


def test_score_variance_validation(L):
    f = FAKE
    lp = star.load_params(1024, 8, 64, 256)
    need = star.score_variance_workspace_size(lp)
    # 128-bit prefix tables: two per instance and one for the weights, K + 1 each
    assert need >= star.STAR_WS_HEADER_BYTES + (2 * 8 + 3) * 257 * 16
    args = [f] * 9            # cur, rem, inst, load, beta, gain, best_target, best_gain, move
    assert L.star_score_variance(ctypes.byref(lp), *args, f, need - 1, None) == -4
    assert L.star_score_variance(ctypes.byref(lp), *args[:4], None, *args[5:], f, need, None) == -1
    assert L.star_score_variance(ctypes.byref(lp), *args[:3], None, *args[4:], f, need, None) == -1
    odd = ctypes.c_void_p((1 << 20) + 8)
    assert L.star_score_variance(ctypes.byref(lp), *args[:5], odd, *args[6:], f, need, None) == -2
    assert L.star_score_variance(None, *args, f, need, None) == -1
    # gains that could reach 2^126: refused although int64 curves would fit
    big = star.load_params(1 << 18, 8, 1 << 10, 1 << 20)
    assert L.star_project_load(ctypes.byref(big), f, f, f, f, f, 256, None) != -3
    assert L.star_score_variance(ctypes.byref(big), *args, f, 1 << 40, None) == -3
    assert star.score_variance_workspace_size(big) == 0
    # the largest rebalancing scan (32768 requests, 64 instances, 1024 buckets of 64) fits
    assert star.score_variance_workspace_size(star.load_params(32768, 64, 64, 1024)) > 0


def test_plan_validation(L):
    f = FAKE
    pp = star.plan_params(1024, 8, 64, 256, 16)
    need = star.plan_workspace_size(pp)
    assert need >= star.score_variance_workspace_size(star.load_params(1024, 8, 64, 256)) + 64
    args = [f] * 7            # cur, rem, inst, load, beta, moves, n_moves
    assert L.star_plan_migrations(ctypes.byref(pp), *args, f, need - 1, None) == -4
    assert L.star_plan_migrations(ctypes.byref(pp), *args[:4], None, *args[5:], f, need, None) == -1
    assert L.star_plan_migrations(ctypes.byref(pp), *args[:6], None, f, need, None) == -1
    assert L.star_plan_migrations(ctypes.byref(pp), *args[:5], None, f, f, need, None) == -1
    for bad in (dict(max_moves=-1), dict(max_moves=5000), dict(theta=(0, 0)),
                dict(theta=(-1, 1)), dict(theta=(1 << 21, 1)), dict(u_rule=2), dict(mem_rule=-1),
                dict(mem_cap=-5)):
        kw = dict(max_moves=4)
        kw.update(bad)
        bp = star.plan_params(100, 4, 8, 16, **kw)
        assert L.star_plan_migrations(ctypes.byref(bp), *args, f, 1 << 30, None) == -1, bad
    # more instances than a workgroup classifies in LDS
    assert star.plan_workspace_size(star.plan_params(100, 1025, 1, 4, 1)) == 0
    assert star.plan_workspace_size(star.plan_params(1 << 18, 8, 1 << 10, 1 << 20, 1)) == 0


def test_mlp4_validation(L):
    f = FAKE
    mp = star.mlp4_params(1024, 3584, 2048, 512, 64, star.BF16)
    need = star.predict_mlp4_workspace_size(mp)
    # split-K partials of both layers plus the first layer's bf16 output
    assert need >= star.STAR_WS_HEADER_BYTES + 1024 * 2048 * (4 + 2) + 1024 * 512 * 4
    args = [f] * 11           # hidden, w1, b1, w2, b2, w3, b3, w4, ema, expected, rem
    args[2] = args[4] = args[6] = None
    assert L.star_predict_mlp4(ctypes.byref(mp), *args, f, need - 1, None) == -4
    bad = list(args)
    bad[7] = None             # w4
    assert L.star_predict_mlp4(ctypes.byref(mp), *bad, f, need, None) == -1
    for kw in (dict(m2=4096), dict(m3=300), dict(d_model=3583)):
        base = dict(n_req=8, d_model=3584, m1=2048, m2=512, m3=64, dtype=star.BF16)
        base.update(kw)
        assert L.star_predict_mlp4(ctypes.byref(star.mlp4_params(**base)), *args, f, 1 << 30,
                                   None) == -2, kw
    assert L.star_predict_mlp4(ctypes.byref(star.mlp4_params(8, 64, 64, 64, 8, 7)), *args, f,
                               1 << 30, None) == -1
    assert L.star_predict_mlp4(ctypes.byref(star.mlp4_params(8, 64, 64, 64, 8, star.BF16,
                                                             ema_alpha=1.5)), *args, f,
                               1 << 30, None) == -1
    odd = ctypes.c_void_p((1 << 20) + 4)
    bad = list(args)
    bad[2] = odd              # b1 not 16-byte aligned
    assert L.star_predict_mlp4(ctypes.byref(mp), *bad, f, need, None) == -2


def test_read_device_error_rejects_bad_args(L):
    code = ctypes.c_int32(0)
    assert L.star_read_device_error(FAKE, None, None) == -1
    assert L.star_read_device_error(None, None, ctypes.byref(code)) == -4
    assert L.star_workspace_init(FAKE, 100, None) == -4
