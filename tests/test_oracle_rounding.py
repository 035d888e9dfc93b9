"""Pins of the oracle's token rounding: a hand-worked example, brute force and invariants."""
import os

import numpy as np
import pytest

import oracle
from oracle.routing import ROUND_MODES

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tr_worked_example_m4.txt")


def load_golden():
    g = {"S": {}, "TOPK": {}, "F_TR": {}, "DIR": {}, "MEMBERS": {}, "U": {}, "W": []}
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        k, *v = line.split()
        if k == "S":
            g["S"][int(v[0])] = [float(x) for x in v[1:]]
        elif k == "TOPK":
            g["TOPK"][int(v[0])] = [int(x) for x in v[1:]]
        elif k == "COUNTS_TC":
            g["COUNTS_TC"] = [int(x) for x in v]
        elif k in ("F_TR", "DIR"):
            g[k][v[0]] = [int(x) for x in v[1:]]
        elif k == "MEMBERS":
            g["MEMBERS"].setdefault(v[0], {})[int(v[1])] = [int(x) for x in v[2:]]
        elif k == "U":
            g["U"][v[0]] = [float(x) for x in v[1:]]
        elif k in ("OFFSETS", "TOK_OFFSETS", "TOK_ROWS"):
            g[k] = [int(x) for x in v[1:]]
        elif k == "W":
            g["W"].append((v[0], int(v[1]), int(v[2]), float(v[3])))
    return g


def test_golden_worked_example():
    g = load_golden()
    T = len(g["S"])
    S = np.array([g["S"][t] for t in range(T)], np.float32)
    E = S.shape[1]
    idx = oracle.topk_select(S, 2)
    np.testing.assert_array_equal(idx, [g["TOPK"][t] for t in range(T)])
    tc = oracle.tc_membership(idx, E)
    np.testing.assert_array_equal(tc.sum(0), g["COUNTS_TC"])
    for mode in g["F_TR"]:
        u = np.array(g["U"][mode], np.float32) if mode in g["U"] else None
        mem, f_tr, rdir = oracle.round_tokens(S, tc, 4, mode=mode, u=u)
        np.testing.assert_array_equal(f_tr, g["F_TR"][mode], err_msg=mode)
        if mode in g["DIR"]:
            np.testing.assert_array_equal(rdir, g["DIR"][mode])
        for e, toks in g["MEMBERS"].get(mode, {}).items():
            assert np.flatnonzero(mem[:, e]).tolist() == toks, (mode, e)
    mem, _, _ = oracle.round_tokens(S, tc, 4, mode="nearest")
    R = oracle.routing_from_membership(mem, S, dtype=np.float64)
    np.testing.assert_array_equal(R.offsets, g["OFFSETS"])
    np.testing.assert_array_equal(R.tok_offsets, g["TOK_OFFSETS"])
    np.testing.assert_array_equal(R.tok_rows, g["TOK_ROWS"])
    for mode, t, e, w in g["W"]:
        assert abs(R.weights[t, e] - w) < 1e-6


def _brute_round(S, tc, M, f_tr):
    """Per expert: sort all tokens with Python's sort on (not TC, -score, t) and keep f_tr."""
    T, E = S.shape
    mem = np.zeros((T, E), bool)
    for e in range(E):
        order = sorted(range(T), key=lambda t: (not tc[t, e], -float(S[t, e]), t))
        for t in order[: f_tr[e]]:
            mem[t, e] = True
    return mem


def _random_case(seed, T, E, K, quant=None):
    rng = np.random.default_rng(seed)
    L = rng.standard_normal((T, E)) * 1.5 + rng.standard_normal(E) * 1.0
    S = oracle.softmax_scores(L).astype(np.float32)
    if quant:
        S = (np.round(S * quant) / quant).astype(np.float32)
    tc = oracle.tc_membership(oracle.topk_select(S, K), E)
    return S, tc


@pytest.mark.parametrize("mode", ROUND_MODES)
@pytest.mark.parametrize("seed,T,E,K,M,quant", [(0, 200, 8, 2, 16, None), (1, 300, 16, 4, 8, 64),
                                                (2, 64, 4, 1, 32, None), (3, 500, 32, 8, 16, 16)])
def test_rounding_invariants(mode, seed, T, E, K, M, quant):
    S, tc = _random_case(seed, T, E, K, quant)
    u = np.random.default_rng(seed + 99).random(E).astype(np.float32)
    mem, f_tr, rdir = oracle.round_tokens(S, tc, M, mode=mode, u=u)
    f = tc.sum(0)
    lo, hi = (f // M) * M, -(-f // M) * M
    np.testing.assert_array_equal(mem.sum(0), f_tr)
    assert np.all(f_tr % M == 0)
    assert np.all(np.abs(f_tr - f) < M)
    assert np.all((f_tr == lo) | (f_tr == hi))
    np.testing.assert_array_equal(rdir, np.sign(f_tr - f))
    if mode == "nearest":
        exp = np.where((hi - f) < (f - lo), hi, lo)
        exp = np.where(hi > T, lo, exp)
        np.testing.assert_array_equal(f_tr, exp)
    if mode == "up":
        np.testing.assert_array_equal(f_tr, np.where(hi > T, lo, hi))
    if mode == "down":
        np.testing.assert_array_equal(f_tr, lo)
    if mode == "stochastic":
        np.testing.assert_array_equal(f_tr, np.where((u * M < (f - lo)) & (hi <= T), hi, lo))
    np.testing.assert_array_equal(mem, _brute_round(S, tc, M, f_tr))
    # kept TC tokens are the best-scored TC tokens; pads are the best non-TC tokens
    for e in range(E):
        kept = mem[:, e] & tc[:, e]
        dropped = tc[:, e] & ~mem[:, e]
        padded = mem[:, e] & ~tc[:, e]
        if dropped.any():
            assert not padded.any()
            assert S[kept, e].min(initial=np.inf) >= S[dropped, e].max()
        if padded.any():
            assert kept.sum() == f[e]
            rest = ~tc[:, e] & ~mem[:, e]
            assert S[padded, e].min() >= S[rest, e].max(initial=-np.inf)


def test_rounding_order_between_modes_and_token_drop():
    S, tc = _random_case(7, 800, 32, 4)
    M = 16
    tot = {m: oracle.round_tokens(S, tc, M, mode=m)[1].sum() for m in ("down", "nearest", "up")}
    assert tot["down"] <= tot["nearest"] <= tot["up"]
    # DOWN == TC token dropping: capacity floor(f/M)*M, drop the lowest-scored tokens
    mem, f_tr, _ = oracle.round_tokens(S, tc, M, mode="down")
    for e in range(S.shape[1]):
        toks = np.flatnonzero(tc[:, e])
        keep = sorted(toks, key=lambda t: (-float(S[t, e]), t))[: f_tr[e]]
        assert sorted(keep) == np.flatnonzero(mem[:, e]).tolist()


@pytest.mark.parametrize("seed", range(6))
def test_balance_bounds(seed):
    S, tc = _random_case(seed, 2000, 64, 4)
    M = 32
    _, f_tr, _ = oracle.round_tokens(S, tc, M, mode="balance")
    f = tc.sum(0)
    # The running residual z stays within M/2 after every expert (the two
    # candidates z + r_up and z + r_down differ by exactly M and the smaller
    # magnitude is taken), so every prefix sum of deviations -- and the total --
    # is bounded by M/2.  The per-expert bound also printed with the algorithm
    # does not follow from it: z = M/2 - 1 with f - lo = M - 1 rounds down by
    # M - 1.  Only deviations below M per expert hold there.
    prefix = np.cumsum(f_tr.astype(np.int64) - f)
    assert np.max(np.abs(prefix)) <= M / 2
    assert abs(int(f_tr.sum()) - int(f.sum())) <= M / 2
    assert np.max(np.abs(f_tr - f)) < M


def test_balance_per_expert_counterexample():
    # f = (17, 31), M = 32: e0 |15| < |-17| pads, z = 15; e1 |1+15| < |-31+15|
    # is a tie, so it drops by 31 = M - 1 (the per-expert M/2 claim fails).
    T, E, M = 200, 2, 32
    tc = np.zeros((T, E), bool)
    tc[:17, 0] = True
    tc[:31, 1] = True
    S = np.random.default_rng(3).random((T, E)).astype(np.float32)
    _, f_tr, _ = oracle.round_tokens(S, tc, M, mode="balance")
    np.testing.assert_array_equal(f_tr, [32, 0])


def test_rounding_degenerate_cases():
    # counts already multiples of M: nothing moves, in every mode
    T, E, M = 64, 4, 8
    tc = np.zeros((T, E), bool)
    for e in range(E):
        tc[e * 8:(e + 2) * 8, e] = True
    S = np.random.default_rng(0).random((T, E)).astype(np.float32)
    for mode in ROUND_MODES:
        mem, f_tr, rdir = oracle.round_tokens(S, tc, M, mode=mode, u=np.zeros(E, np.float32))
        np.testing.assert_array_equal(mem, tc)
        assert np.all(rdir == 0)
    # an expert whose ceil exceeds T cannot be padded
    T, E, M = 10, 2, 16
    tc = np.zeros((T, E), bool)
    tc[:9, 0] = True
    tc[9, 1] = True
    S = np.random.default_rng(1).random((T, E)).astype(np.float32)
    _, f_tr, _ = oracle.round_tokens(S, tc, M, mode="up")
    np.testing.assert_array_equal(f_tr, [0, 0])
    # midpoint rounds down under NR-f
    T, E, M = 40, 1, 8
    tc = np.zeros((T, E), bool)
    tc[:12, 0] = True
    S = np.random.default_rng(2).random((T, E)).astype(np.float32)
    assert oracle.round_tokens(S, tc, M)[1][0] == 8
    tc[12, 0] = True
    assert oracle.round_tokens(S, tc, M)[1][0] == 16
