"""The router GEMM with softmax and top-K fused into its epilogue (E a multiple
of 8, E <= 256, K <= 8), against the two-launch path and the oracle.

Three routings of the same inputs, through the C ABI:
  fused     moe_route (the default where the shapes fuse);
  separate  moe_route with MOE_ROUTE_SEPARATE_TOPK (router GEMM, then the
            softmax/top-K kernel on the logits);
  rerun     moe_route with MOE_ROUTE_SCORES_IN on the fused path's scores.
The logits of fused and separate agree bit for bit (the same k-loop), the
scores up to the rounding of the softmax sum, and both match the oracle's
logits and S_full.  Given the same scores, fused and rerun must agree exactly
on everything derived from them: top-K indices and weights, membership words,
counts and the transposed scores.
"""
import numpy as np
import pytest

import oracle
from dense_reference import rel_err
from paper_2512_14080_amd import workloads as W

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def routings(cfg, seed, T=None, bias=None, edit_x=None):
    torch = _torch()
    from paper_2512_14080_amd import binding as B
    from paper_2512_14080_amd.layer import to_device_bf16
    inp = W.make_inputs(cfg, seed, T=T)
    if bias is not None:
        inp.bias = np.asarray(bias, np.float32)
    if edit_x is not None:
        inp.X = inp.X.copy()
        edit_x(inp.X)
    T = inp.X.shape[0]
    D = B.dims(T, cfg.d, cfg.n, cfg.E, cfg.K)
    X, Wr = to_device_bf16(inp.X, "cuda"), to_device_bf16(inp.Wr, "cuda")
    bias_d = None if inp.bias is None else torch.from_numpy(inp.bias).cuda()
    keep = B.MOE_ROUTING_LOGITS | B.MOE_ROUTING_SCORES_T
    out, launches = {}, {}
    flags = B.MOE_ROUTE_WRITE_LOGITS | B.MOE_ROUTE_WRITE_SCORES_T
    for name, extra in (("fused", 0), ("separate", B.MOE_ROUTE_SEPARATE_TOPK)):
        r = B.Routing(D, T * cfg.K, keep)
        B.moe_prof_select("router_topk")
        B.moe_route(D, X, Wr, bias_d, flags | extra, r)
        torch.cuda.synchronize()
        launches[name] = B.moe_prof_read()[1]
        B.moe_prof_select(-1)
        out[name] = {k: v.cpu().numpy() for k, v in r.arrays().items() if v is not None}
    r = B.Routing(D, T * cfg.K, B.MOE_ROUTING_SCORES_T)
    r.arrays()["scores"].copy_(torch.from_numpy(out["fused"]["scores"]))
    B.moe_route(D, None, None, None, B.MOE_ROUTE_SCORES_IN | B.MOE_ROUTE_WRITE_SCORES_T, r)
    torch.cuda.synchronize()
    out["rerun"] = {k: v.cpu().numpy() for k, v in r.arrays().items() if v is not None}
    assert launches == {"fused": 1, "separate": 0}, launches
    return inp, out


def check(cfg, seed, T=None, bias=None):
    inp, o = routings(cfg, seed, T, bias)
    f, s, r = o["fused"], o["separate"], o["rerun"]
    L = oracle.router_logits(inp.f32("X"), inp.f32("Wr"), inp.bias, np.float32)
    S = oracle.softmax_scores(L).astype(np.float32)
    np.testing.assert_array_equal(f["logits"], s["logits"])
    assert rel_err(f["logits"], L) <= 1e-4
    assert rel_err(f["scores"], S) <= 1e-4
    np.testing.assert_allclose(f["scores"], s["scores"], rtol=4e-6, atol=1e-30)
    np.testing.assert_array_equal(f["scores_t"], f["scores"].T)
    for k in ("topk_idx", "topk_w", "mask", "counts", "scores_t", "mask_prefix", "offsets", "row_token",
              "row_w", "tok_offsets", "tok_rows"):
        if k in f:
            np.testing.assert_array_equal(f[k], r[k], err_msg=k)
    assert f["counts"].sum() == f["topk_idx"].shape[0] * cfg.K
    np.testing.assert_array_equal(f["counts"], np.bincount(f["topk_idx"].ravel(), minlength=cfg.E))
    # the two launch paths select the same experts wherever their scores agree
    same = np.all(f["scores"] == s["scores"], axis=1)
    np.testing.assert_array_equal(f["topk_idx"][same], s["topk_idx"][same])
    return o


@pytest.mark.parametrize("cfg,T", [
    (W.CONFIGS["tiny"], None),                                               # E = 8, K = 2 (128 x 64 tiles)
    (W.MoEConfig("e16", T=3000, d=512, n=64, E=16, K=4, m_tile=128), None),  # ragged last tile
    (W.MoEConfig("e64", T=700, d=256, n=64, E=64, K=8, m_tile=128), None),
    (W.MoEConfig("e128", T=1000, d=384, n=64, E=128, K=8, m_tile=128), None),
    (W.MoEConfig("e8k1", T=130, d=128, n=64, E=8, K=1, m_tile=16), None),
    (W.MoEConfig("e128t1", T=1, d=128, n=64, E=128, K=8, m_tile=128), None),
    (W.MoEConfig("e104k5", T=250, d=256, n=64, E=104, K=5, m_tile=16), None),  # 24 idle columns
    (W.MoEConfig("e256", T=1000, d=256, n=64, E=256, K=8, m_tile=128), None),   # 128 x 256 tiles, two row blocks
    (W.MoEConfig("e200k6", T=700, d=128, n=64, E=200, K=6, m_tile=64), None),  # 56 idle columns
])
def test_fused_router_topk(cfg, T):
    check(cfg, seed=31, T=T)


def test_fused_router_topk_with_bias_and_ties():
    """A router bias, and the Zipf-skewed bias of the sparse workloads: a hot
    expert chosen by every token and many near-equal scores."""
    cfg = W.MoEConfig("e96", T=900, d=256, n=64, E=96, K=6, m_tile=64, zipf_s=1.1)
    check(cfg, seed=32)
    bias = np.zeros(cfg.E, np.float32)
    bias[5] = 60.0
    o = check(cfg, seed=33, bias=bias)
    assert np.all(o["fused"]["topk_idx"][:, 0] == 5)


def test_fused_router_topk_several_tiles_per_workgroup():
    """More 128-row tiles than workgroups: each workgroup runs the epilogue of
    one tile while the next tile's operands load, reusing its LDS."""
    check(W.MoEConfig("e128big", T=70000, d=128, n=64, E=128, K=8, m_tile=128), seed=34)


def test_fused_router_topk_7b_full_size():
    """The 7B routing shape (T=32768, d=1536, E=128, K=8)."""
    check(W.CONFIGS["7b"], seed=0)


@pytest.mark.parametrize("name", ["1b", "coarse"])
def test_fused_router_topk_other_full_sizes(name):
    """The 1B (E=64, K=8: 128 x 64 tiles, every column an expert) and coarse
    (d=4096, E=8, K=2: 56 idle columns of a 128 x 64 tile) routing shapes."""
    check(W.CONFIGS[name], seed=0)


def test_fused_router_topk_nonfinite_logits():
    """X rows holding NaN, +-Inf or values whose logits overflow give NaN and
    infinite logits.  Every token still gets K distinct experts in [0, E)
    (the exact (score, expert) order is total, NaN included), and the selection,
    weights and bitmap equal those of the top-K kernel run on the fused
    path's own scores."""
    cfg = W.MoEConfig("e128nf", T=600, d=256, n=64, E=128, K=8, m_tile=128)
    nan, pinf, ninf = np.uint16(0x7FC0), np.uint16(0x7F80), np.uint16(0xFF80)

    def edit(X):
        X[3, 7] = nan                  # a whole logit row of NaN
        X[10, 0] = pinf                # +-Inf logits (and NaN where they cancel)
        X[11, 5] = ninf
        X[20, :] = np.uint16(0x7E00)   # about 4e37 everywhere: logits overflow
        X[599, 1] = nan                # the ragged last tile
    inp, o = routings(cfg, 35, edit_x=edit)
    f, r = o["fused"], o["rerun"]
    idx = f["topk_idx"]
    assert ((idx >= 0) & (idx < cfg.E)).all()
    assert all(len(set(row)) == cfg.K for row in idx)
    assert np.isnan(f["logits"][3]).all() and not np.isfinite(f["logits"][10]).all()
    for k in ("topk_idx", "topk_w", "mask", "counts", "scores_t"):
        np.testing.assert_array_equal(f[k], r[k], err_msg=k)
    np.testing.assert_array_equal(f["counts"], np.bincount(idx.ravel(), minlength=cfg.E))
    # rows with finite inputs are untouched by the others
    ok = np.isfinite(f["logits"]).all(axis=1)
    assert ok.sum() >= cfg.T - 5
    L = oracle.router_logits(inp.f32("X")[ok], inp.f32("Wr"), inp.bias, np.float32)
    assert rel_err(f["logits"][ok], L) <= 1e-4


def test_fused_router_topk_sparse_full_size():
    """The high-sparsity routing shape (T=32768, d=2048, E=256, K=8, Zipf-skewed
    router bias): 128 x 256 tiles."""
    check(W.CONFIGS["sparse"], seed=0)
