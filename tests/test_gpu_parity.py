"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Routing contract: the oracle computes the fp32 scores S_full from the seeded
inputs and the device consumes them (MOE_ROUTE_SCORES_IN), so every integer
routing result -- top-K, mask, counts, offsets, row order, token-major lists,
rounding decisions -- must match bit for bit.  Outputs and gradients must
match the fp32 oracle within max|gpu - ref| / max|ref| <= 2e-2.  The device's
own router (GEMM + softmax) is checked against the oracle's logits/scores
within the same tolerance, and its top-K is checked for validity against its
own scores.
"""
import numpy as np
import pytest

import oracle
from dense_reference import rel_err, rel_fro
from paper_2512_14080_amd import workloads as W

pytestmark = pytest.mark.gpu

TOL = 2e-2


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def oracle_scores(inp):
    L = oracle.router_logits(inp.f32("X"), inp.f32("Wr"), inp.bias, np.float32)
    return L, oracle.softmax_scores(L).astype(np.float32)


def oracle_routing(S, K, round_mode=None, m_tile=None, u=None):
    idx = oracle.topk_select(S, K)
    member = oracle.tc_membership(idx, S.shape[1])
    rdir = None
    if round_mode:
        member, _, rdir = oracle.round_tokens(S, member, m_tile, mode=round_mode, u=u)
    return idx, rdir, oracle.routing_from_membership(member, S, np.float32)


def mask_bits(member):
    """Oracle membership -> the device's [E, ceil(T/64)] uint64 bitmap."""
    T, E = member.shape
    Wd = (T + 63) // 64
    bits = np.zeros((E, Wd * 64), np.uint64)
    bits[:, :T] = member.T.astype(np.uint64)
    weights = np.left_shift(np.uint64(1), np.arange(64, dtype=np.uint64))
    return (bits.reshape(E, Wd, 64) * weights).sum(axis=2, dtype=np.uint64)


def check_routing(layer, R, idx=None, rdir=None):
    a = {k: (v.cpu().numpy() if v is not None else None) for k, v in layer.routing.arrays().items()}
    P = R.P
    np.testing.assert_array_equal(a["counts"], R.counts)
    np.testing.assert_array_equal(a["offsets"], R.offsets)
    np.testing.assert_array_equal(a["row_token"][:P], R.row_token)
    np.testing.assert_array_equal(a["row_expert"][:P], R.row_expert)
    np.testing.assert_array_equal(a["tok_offsets"], R.tok_offsets)
    np.testing.assert_array_equal(a["tok_rows"][:P], R.tok_rows)
    np.testing.assert_array_equal(a["mask"].view(np.uint64), mask_bits(R.member))
    # same fp32 operations in the same order: the weights agree exactly
    np.testing.assert_array_equal(a["row_w"][:P], R.row_w)
    if idx is not None:
        tc = {k: v.cpu().numpy() for k, v in layer.tc.arrays().items() if v is not None}
        np.testing.assert_array_equal(tc["topk_idx"], idx)
    if rdir is not None:
        np.testing.assert_array_equal(a["round_dir"], rdir)
    # the metadata kernels found a consistent selection
    assert int(a["status"][0]) == 0


def expert_biases(cfg, seed, scale=0.01):
    """Seeded fp32 expert biases b1 [E,2n], b2 [E,d] ~ N(0, scale)."""
    rng = np.random.default_rng(1000 + seed)
    b1 = (rng.standard_normal((cfg.E, 2 * cfg.n)) * scale).astype(np.float32)
    b2 = (rng.standard_normal((cfg.E, cfg.d)) * scale).astype(np.float32)
    return b1, b2


def run_layer(cfg, seed=0, T=None, round_mode=None, u=None, router_grad=True, bias=None, eb=None):
    torch = _torch()
    from paper_2512_14080_amd.layer import DeviceLayer
    inp = W.make_inputs(cfg, seed, T=T)
    if bias is not None:
        inp.bias = np.asarray(bias, np.float32)
    _, S = oracle_scores(inp)
    b1, b2 = eb if eb is not None else (None, None)
    layer = DeviceLayer(inp, round_mode=round_mode, scores_in=S, u=u, router_grad=router_grad, b1=b1, b2=b2)
    layer.step()
    torch.cuda.synchronize()
    return inp, S, layer


def check_layer(cfg, seed=0, T=None, round_mode=None, u=None, bias=None, eb=None):
    inp, S, layer = run_layer(cfg, seed, T, round_mode, u, bias=bias, eb=eb)
    idx, rdir, R = oracle_routing(S, cfg.K, round_mode, cfg.m_tile, u)
    check_routing(layer, R, idx, rdir)
    X, W1, W2, Wr, dO = (inp.f32(k) for k in ("X", "W1", "W2", "Wr", "dO"))
    b1, b2 = eb if eb is not None else (None, None)
    fw = oracle.forward(X, W1, W2, R, b1=b1, b2=b2)
    bw = oracle.backward(dO, X, fw["H"], W1, W2, Wr, R, b2=b2)
    P = R.P
    got = {
        "O": layer.O.float().cpu().numpy(), "H": layer.H[:P].float().cpu().numpy(),
        "dX": layer.dX.float().cpu().numpy(), "dW1": layer.dW1.float().cpu().numpy(),
        "dW2": layer.dW2.float().cpu().numpy(), "dWr": layer.dWr.cpu().numpy(),
        "dbias": layer.dbias.cpu().numpy(), "dS": layer.dS[:P].cpu().numpy(),
    }
    ref = {"O": fw["O"], "H": fw["H"], "dX": bw["dX"], "dW1": bw["dW1"], "dW2": bw["dW2"],
           "dWr": bw["dWr"], "dbias": bw["dbias"], "dS": bw["dS"]}
    if eb is not None:
        got["db1"], got["db2"] = layer.db1.cpu().numpy(), layer.db2.cpu().numpy()
        ref["db1"], ref["db2"] = bw["db1"], bw["db2"]
    errs = {k: rel_err(got[k], ref[k]) for k in ref}
    fro = {k: rel_fro(got[k], ref[k]) for k in ref}
    print(cfg.name, T, round_mode, "max-normalised", {k: f"{v:.2e}" for k, v in errs.items()},
          "Frobenius", {k: f"{v:.2e}" for k, v in fro.items()}, flush=True)
    for k, v in errs.items():
        assert v <= TOL, (k, v, errs)
    return layer, R


TINY = W.CONFIGS["tiny"]


def test_tiny_token_choice():
    check_layer(TINY)


@pytest.mark.parametrize("mode", ["nearest", "up", "down", "balance", "stochastic"])
def test_tiny_token_rounding(mode):
    u = np.random.default_rng(5).random(TINY.E).astype(np.float32) if mode == "stochastic" else None
    check_layer(TINY, seed=1, round_mode=mode, u=u)


# several tiles per expert with a ragged tail; T not a multiple of 64
MID = W.MoEConfig("mid", T=3000, d=512, n=256, E=16, K=4, m_tile=128)
# d not a multiple of 256 (128-wide tiles), n = 192 (dS reduced over three N tiles)
ODD = W.MoEConfig("odd", T=1000, d=384, n=192, E=24, K=3, m_tile=32)
# n = 512: dS over two 256-wide N tiles
WIDE = W.MoEConfig("wide", T=700, d=256, n=512, E=8, K=2, m_tile=64)
# many experts, Zipf-skewed popularity: empty and tiny experts
SKEW = W.MoEConfig("skew", T=700, d=256, n=128, E=256, K=8, m_tile=128, zipf_s=1.1)


@pytest.mark.parametrize("cfg,mode", [(MID, None), (MID, "nearest"), (ODD, None), (ODD, "up"), (WIDE, None),
                                      (SKEW, None), (SKEW, "nearest")])
def test_shapes(cfg, mode):
    check_layer(cfg, seed=2, round_mode=mode)


def test_k_equals_e_and_k_one():
    check_layer(W.MoEConfig("kE", T=300, d=128, n=64, E=8, K=8, m_tile=16, router="w_std"), seed=3)
    check_layer(W.MoEConfig("k1", T=300, d=128, n=64, E=8, K=1, m_tile=16), seed=4)


def test_wave_per_token_topk_shapes():
    """E > 256 takes the wave-per-token top-K (here with K = 3 and K = 12);
    K in (8, 16] at E <= 256 takes the lane-per-token kernel's 16-slot form
    (K = 10, and K = E = 16).  The routing and the layer still match."""
    check_layer(W.MoEConfig("e264", T=300, d=128, n=64, E=264, K=3, m_tile=16), seed=13)
    check_layer(W.MoEConfig("e264k12", T=300, d=128, n=64, E=264, K=12, m_tile=16), seed=16, round_mode="nearest")
    check_layer(W.MoEConfig("k10", T=300, d=128, n=64, E=16, K=10, m_tile=16), seed=14, round_mode="nearest")
    check_layer(W.MoEConfig("k16", T=300, d=128, n=64, E=16, K=16, m_tile=16), seed=17)


def test_weight_gradients_over_row_chunks():
    """An expert that holds far more rows than the rest (every token picks it)
    has its weight-gradient reductions cut into row chunks whose fp32 partials
    are summed in chunk order; dW1 and dW2 still match the oracle."""
    cfg = W.MoEConfig("hot", T=12000, d=256, n=128, E=16, K=2, m_tile=128)
    bias = np.zeros(cfg.E, np.float32)
    bias[3] = 60.0
    layer, R = check_layer(cfg, seed=15, round_mode="nearest", bias=bias)
    # the chunk length is at least 2048 rows: the hot expert is split
    assert R.counts[3] > 2 * 2048


def test_weight_gradients_short_k_loops():
    """Experts with 0, 12, 42, 80, 119, 134, 191 and 222 rows: the weight
    gradients' 256 x 256 tiles (d = 512, n = 256) then run k loops of 0 to 4
    steps of 64 rows, the cases where the two-stage pipeline has no stage, no
    second stage or no stage after next to prefetch, and an odd step count.
    dW1 and dW2 (and the empty expert's zero rows) match the oracle."""
    cfg = W.MoEConfig("kshort", T=400, d=512, n=256, E=8, K=2, m_tile=128)
    bias = np.array([-40, 0, 0.6, 1.0, 1.3, 1.5, 1.7, 2.0], np.float32)
    layer, R = check_layer(cfg, seed=21, bias=bias)
    steps = sorted(set(int(-(-c // 64)) for c in R.counts))
    assert steps == [0, 1, 2, 3, 4], (R.counts, steps)


def test_split_ring_short_k_loops():
    """d a multiple of 256 with n = 64: the down projection (k = n = 64) and
    dX~ (k = 2n = 128) run one- and two-step k loops on the split LDS ring
    (A rows two steps ahead), with token choice and with rounding."""
    cfg = W.MoEConfig("ring", T=600, d=256, n=64, E=8, K=2, m_tile=64)
    check_layer(cfg, seed=22)
    check_layer(cfg, seed=23, round_mode="nearest")


def test_single_token_and_one_hot_expert():
    check_layer(TINY, seed=5, T=1)
    check_layer(TINY, seed=6, T=65, round_mode="nearest")
    # expert 3 outranks every other expert for every token: it takes all T rows
    bias = np.zeros(TINY.E, np.float32)
    bias[3] = 60.0
    layer, R = check_layer(TINY, seed=7, T=200, bias=bias)
    assert R.counts[3] == 200


@pytest.mark.parametrize("T,mode", [(1, "nearest"), (10, "down")])
def test_rounding_that_drops_every_row(T, mode):
    """Token rounding can leave no rows at all (T below M_tile: every expert's
    ceiling exceeds T, so every expert is rounded down to zero).  The layer
    then runs on an empty routing: O, dX, the weight gradients and the router
    gradients are exactly zero (every output is written), with the routing
    itself matching the oracle."""
    inp, S, layer = run_layer(TINY, 8, T, mode, eb=expert_biases(TINY, 8))
    idx, rdir, R = oracle_routing(S, TINY.K, mode, TINY.m_tile)
    assert R.P == 0
    check_routing(layer, R, idx, rdir)
    for name in ("O", "dX", "dW1", "dW2", "dWr", "dbias", "db1", "db2"):
        v = getattr(layer, name).float().cpu().numpy()
        assert np.all(v == 0), (name, float(np.abs(v).max()))


def test_device_router_matches_oracle_scores():
    torch = _torch()
    from paper_2512_14080_amd.layer import DeviceLayer
    for cfg, seed in ((TINY, 0), (MID, 1), (SKEW, 2)):
        inp = W.make_inputs(cfg, seed)
        L, S = oracle_scores(inp)
        layer = DeviceLayer(inp)
        layer.route()
        torch.cuda.synchronize()
        a = {k: v.cpu().numpy() for k, v in layer.tc.arrays().items() if v is not None}
        assert rel_err(a["logits"], L) <= 1e-4, rel_err(a["logits"], L)
        assert rel_err(a["scores"], S) <= 1e-4
        # the device's top-K is a valid stable top-K of the device's own scores
        Sg, idx = a["scores"], a["topk_idx"]
        for t in range(0, cfg.T, max(1, cfg.T // 200)):
            sel = list(idx[t])
            assert len(set(sel)) == cfg.K
            worst = min(Sg[t, e] for e in sel)
            for e in range(cfg.E):
                if e not in sel:
                    assert Sg[t, e] < worst or (Sg[t, e] == worst and e > max(x for x in sel if Sg[t, x] == worst))
        assert a["counts"].sum() == cfg.T * cfg.K
        np.testing.assert_array_equal(a["counts"], np.bincount(idx.ravel(), minlength=cfg.E))


def test_deterministic_bitwise():
    torch = _torch()
    inp, S, layer = run_layer(MID, seed=8, round_mode="nearest")
    first = [t.clone() for t in (layer.O, layer.H, layer.dX, layer.dW1, layer.dW2, layer.dWr, layer.dS)]
    layer.step()
    torch.cuda.synchronize()
    for a, b in zip(first, (layer.O, layer.H, layer.dX, layer.dW1, layer.dW2, layer.dWr, layer.dS)):
        assert torch.equal(a, b)


def test_no_router_grad_path():
    torch = _torch()
    inp, S, layer = run_layer(TINY, seed=9, router_grad=False)
    idx, rdir, R = oracle_routing(S, TINY.K)
    X, W1, W2, dO = (inp.f32(k) for k in ("X", "W1", "W2", "dO"))
    fw = oracle.forward(X, W1, W2, R)
    bw = oracle.backward(dO, X, fw["H"], W1, W2, None, R)
    assert rel_err(layer.dX.float().cpu().numpy(), bw["dX"]) <= TOL


ROUTE_ONLY = W.MoEConfig("route", T=3000, d=128, n=128, E=16, K=4, m_tile=128)


@pytest.mark.parametrize("T", [3000, 9000, 20000, 40000])
@pytest.mark.parametrize("quantised", [False, True])
def test_rounding_selection_sizes_and_ties(T, quantised):
    """Token sizes spanning the two-level rounding selection (one and two
    32-key slot groups per lane in the second level), with real-valued scores
    and with scores on a coarse grid, where most candidates tie on the
    threshold and the token-order tie break decides."""
    torch = _torch()
    from paper_2512_14080_amd.layer import DeviceLayer
    inp = W.make_inputs(ROUTE_ONLY, 11, T=T)
    _, S = oracle_scores(inp)
    if quantised:
        S = (np.round(S * 16.0) / 16.0).astype(np.float32)
    for mode in ("up", "down", "nearest"):
        layer = DeviceLayer(inp, round_mode=mode, scores_in=S)
        layer.route()
        torch.cuda.synchronize()
        idx, rdir, R = oracle_routing(S, ROUTE_ONLY.K, mode, ROUTE_ONLY.m_tile)
        check_routing(layer, R, idx, rdir)


@pytest.mark.parametrize("T,m_tile", [(5000, 8), (20000, 256), (40000, 256), (65536, 128), (65537, 128)])
@pytest.mark.parametrize("quantised", [False, True])
def test_rounding_selection_tiles(T, m_tile, quantised):
    """The smallest and largest M_tile: selection in two levels with one and
    two slot groups in the final one (T = 5000 / 20000), and with a reduce
    level between them where the chunks' picks exceed what the final wave
    holds (T = 40000 at M_tile = 256).  At M_tile = 128, T = 65536 is the
    largest row without a reduce level (4096 picks) and T = 65537 the smallest
    with one, and the first whose mask row takes two LDS passes."""
    torch = _torch()
    from paper_2512_14080_amd.layer import DeviceLayer
    cfg = W.MoEConfig("tiles", T=T, d=128, n=128, E=16, K=4, m_tile=m_tile)
    inp = W.make_inputs(cfg, 12)
    _, S = oracle_scores(inp)
    if quantised:
        S = (np.round(S * 16.0) / 16.0).astype(np.float32)
    for mode in ("up", "down", "nearest"):
        layer = DeviceLayer(inp, round_mode=mode, scores_in=S)
        layer.route()
        torch.cuda.synchronize()
        idx, rdir, R = oracle_routing(S, cfg.K, mode, m_tile)
        check_routing(layer, R, idx, rdir)


def test_routing_with_nonfinite_scores():
    """Scores holding NaN and +-Inf (a diverged router, or caller-supplied
    scores) still give every token K distinct experts in [0, E), consistent
    counts/offsets/rows, and a rounded routing within capacity; the layer then
    runs on it.  Selection follows the total order of the fp32 bit patterns,
    which is the float order wherever both operands are numbers."""
    torch = _torch()
    from paper_2512_14080_amd.layer import DeviceLayer
    cfg = W.MoEConfig("nonfinite", T=700, d=128, n=128, E=64, K=6, m_tile=64)
    inp = W.make_inputs(cfg, 12)
    _, S = oracle_scores(inp)
    rng = np.random.default_rng(5)
    S = S.copy()
    flat = S.reshape(-1)
    pick = rng.choice(flat.size, flat.size // 20, replace=False)
    flat[pick[0::3]] = np.nan
    flat[pick[1::3]] = np.inf
    flat[pick[2::3]] = -np.inf
    S[3, :] = np.nan  # a token whose every score is NaN
    for mode in (None, "nearest"):
        layer = DeviceLayer(inp, round_mode=mode, scores_in=S)
        layer.step()
        torch.cuda.synchronize()
        tc = {k: v.cpu().numpy() for k, v in layer.tc.arrays().items() if v is not None}
        idx = tc["topk_idx"]
        assert idx.shape == (cfg.T, cfg.K)
        assert ((idx >= 0) & (idx < cfg.E)).all()
        assert all(len(set(r)) == cfg.K for r in idx)
        np.testing.assert_array_equal(tc["counts"], np.bincount(idx.ravel(), minlength=cfg.E))
        # finite-score tokens keep the oracle's choice
        ok = np.isfinite(S).all(axis=1)
        ref = oracle.topk_select(S[ok], cfg.K)
        np.testing.assert_array_equal(idx[ok], ref)
        a = {k: (v.cpu().numpy() if v is not None else None) for k, v in layer.routing.arrays().items()}
        P = int(a["offsets"][-1])
        assert P == int(a["counts"].sum()) <= layer.routing.capacity
        assert (np.diff(a["offsets"]) == a["counts"]).all()
        rt, re_ = a["row_token"][:P], a["row_expert"][:P]
        assert ((rt >= 0) & (rt < cfg.T)).all() and ((re_ >= 0) & (re_ < cfg.E)).all()
        assert sorted(a["tok_rows"][:P].tolist()) == list(range(P))


# Shapes at the limits the ABI accepts (E <= 4096, K <= 16) and the
# wave-per-token top-K instantiations behind them: values per lane EPL =
# ceil(E / 64) of 4 (E = 256), 16 (E = 1024), 64 (E = 2056 and 4096: lane
# values 32 .. 63 exercise the upper half of the selection mask).
@pytest.mark.parametrize("E,K", [(256, 16), (1024, 8), (2056, 16), (4096, 16)])
def test_wide_expert_counts_route(E, K):
    torch = _torch()
    from paper_2512_14080_amd.layer import DeviceLayer
    cfg = W.MoEConfig(f"e{E}k{K}", T=700, d=128, n=64, E=E, K=K, m_tile=16)
    inp = W.make_inputs(cfg, 21)
    _, S = oracle_scores(inp)
    for mode in (None, "nearest"):
        layer = DeviceLayer(inp, round_mode=mode, scores_in=S)
        layer.route()
        torch.cuda.synchronize()
        idx, rdir, R = oracle_routing(S, K, mode, cfg.m_tile)
        check_routing(layer, R, idx, rdir)


@pytest.mark.parametrize("E,K", [(256, 16), (1024, 8)])
def test_wide_expert_counts_layer(E, K):
    """The whole layer on the K = 16 / E = 256 shape of the paper's finest
    30B and 120B benchmark layers, and at E = 1024, at reduced T and d."""
    check_layer(W.MoEConfig(f"l{E}k{K}", T=600, d=128, n=64, E=E, K=K, m_tile=16), seed=22)
    check_layer(W.MoEConfig(f"l{E}k{K}", T=600, d=128, n=64, E=E, K=K, m_tile=16), seed=23, round_mode="nearest")


@pytest.mark.parametrize("mode", ["balance", "stochastic"])
def test_sequential_rounding_modes_many_experts(mode):
    """Balance-f carries its running residual over all experts in order; SR-f
    draws per expert.  Both at E = 128 and T = 32768 (the 7B routing shape),
    route only, bit-exact."""
    torch = _torch()
    from paper_2512_14080_amd.layer import DeviceLayer
    cfg = W.MoEConfig("seq", T=32768, d=128, n=64, E=128, K=8, m_tile=128)
    inp = W.make_inputs(cfg, 24)
    _, S = oracle_scores(inp)
    u = np.random.default_rng(25).random(cfg.E).astype(np.float32) if mode == "stochastic" else None
    layer = DeviceLayer(inp, round_mode=mode, scores_in=S, u=u)
    layer.route()
    torch.cuda.synchronize()
    idx, rdir, R = oracle_routing(S, cfg.K, mode, cfg.m_tile, u)
    check_routing(layer, R, idx, rdir)
    assert (R.counts % cfg.m_tile == 0).all()


def test_routing_beyond_word_scan_limit():
    """T > 262144 (more than 4096 bitmap words): the rounded routing's
    placement takes its word bases from a separate scan kernel."""
    torch = _torch()
    from paper_2512_14080_amd.layer import DeviceLayer
    cfg = W.MoEConfig("long", T=270000, d=128, n=64, E=8, K=2, m_tile=128)
    inp = W.make_inputs(cfg, 26)
    _, S = oracle_scores(inp)
    for mode in (None, "nearest"):
        layer = DeviceLayer(inp, round_mode=mode, scores_in=S)
        layer.route()
        torch.cuda.synchronize()
        idx, rdir, R = oracle_routing(S, cfg.K, mode, cfg.m_tile)
        check_routing(layer, R, idx, rdir)


@pytest.mark.parametrize("cfg,mode", [(TINY, None), (TINY, "nearest"), (MID, "nearest"), (ODD, None), (WIDE, None)])
def test_expert_biases(cfg, mode):
    """Expert biases b1 (up-projection) and b2 (down-projection): H, O, dS
    with its <dO_t, b2_e> term, every gradient and db1, db2 against the
    oracle; WIDE (n = 512) has dS summed over two N tiles."""
    check_layer(cfg, seed=31, round_mode=mode, eb=expert_biases(cfg, 31))


@pytest.mark.parametrize("cfg,mode", [(MID, "nearest"), (ODD, None), (SKEW, None)])
def test_aggregation_strategy_ablation(cfg, mode):
    """The expert-aggregation strategies of the ablation entry point: the
    scatter-fused store + contiguous sum gives O bit for bit equal to
    gather-and-sum (same bf16 Y rows, same order); fp32 atomics agree with the
    oracle within the tolerance (their rounding depends on arrival order)."""
    torch = _torch()
    from paper_2512_14080_amd import binding as B
    from paper_2512_14080_amd.layer import _aligned_empty
    inp, S, layer = run_layer(cfg, seed=41, round_mode=mode)
    idx, rdir, R = oracle_routing(S, cfg.K, mode, cfg.m_tile)
    X, W1, W2 = (inp.f32(k) for k in ("X", "W1", "W2"))
    ref = oracle.forward(X, W1, W2, R)["O"]
    ws = _aligned_empty(B.moe_workspace_bytes(layer.D, layer.routing.capacity, B.MOE_WS_FWD_AGG_ABLATION))
    outs = {}
    for name in ("gather_sum", "scatter_sum", "atomic_f32"):
        O = torch.empty_like(layer.O)
        B.moe_fwd_aggregation_ablation(layer.D, layer.X, layer.W1, layer.W2, layer.routing, layer.H, O, name, ws)
        torch.cuda.synchronize()
        outs[name] = O
        err = rel_err(O.float().cpu().numpy(), ref)
        print(cfg.name, name, f"{err:.2e}", flush=True)
        assert err <= TOL, (name, err)
    assert torch.equal(outs["gather_sum"], layer.O)
    assert torch.equal(outs["scatter_sum"], outs["gather_sum"])
