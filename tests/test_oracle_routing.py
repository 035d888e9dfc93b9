"""Pins of the oracle's routing steps against brute force, closed forms and invariants."""
import numpy as np
import pytest

import oracle
from oracle.routing import Routing


def _brute_topk(S, K):
    T, E = S.shape
    out = []
    for t in range(T):
        order = sorted(range(E), key=lambda e: (-float(S[t, e]), e))
        out.append(order[:K])
    return np.array(out, np.int32)


@pytest.mark.parametrize("T,E,K,quant", [(37, 8, 2, None), (50, 16, 4, 4), (20, 5, 5, 3), (9, 64, 16, 2), (12, 7, 1, None)])
def test_topk_brute_force(T, E, K, quant):
    rng = np.random.default_rng(T * 100 + E)
    S = rng.random((T, E)).astype(np.float32)
    if quant:  # many exact ties
        S = (np.floor(S * quant) / quant).astype(np.float32)
    np.testing.assert_array_equal(oracle.topk_select(S, K), _brute_topk(S, K))


def test_topk_invariants_and_signed_zero():
    rng = np.random.default_rng(1)
    S = rng.standard_normal((64, 32)).astype(np.float32)
    S[3, :] = 0.0
    S[3, 5] = -0.0  # -0 == +0: ties broken by index
    K = 6
    idx = oracle.topk_select(S, K)
    for t in range(S.shape[0]):
        sel = set(idx[t].tolist())
        assert len(sel) == K
        worst = min(S[t, e] for e in sel)
        for e in range(S.shape[1]):
            if e not in sel:
                assert S[t, e] <= worst
                if S[t, e] == worst:
                    assert e > max(x for x in sel if S[t, x] == worst)
    assert idx[3].tolist() == list(range(K))


def test_softmax_closed_forms():
    rng = np.random.default_rng(2)
    L = rng.standard_normal((16, 12)) * 3
    S = oracle.softmax_scores(L)
    np.testing.assert_allclose(S.sum(axis=1), 1.0, rtol=1e-12)
    # ratio of two scores is exp of the logit difference
    np.testing.assert_allclose(S[:, 3] / S[:, 7], np.exp(L[:, 3] - L[:, 7]), rtol=1e-12)
    # invariant to a per-row shift (large shift would overflow without max subtraction)
    np.testing.assert_allclose(oracle.softmax_scores(L + 800.0), S, rtol=1e-12)
    # uniform logits give 1/E
    np.testing.assert_allclose(oracle.softmax_scores(np.zeros((2, 5))), 0.2, rtol=1e-15)


def test_router_logits_bias():
    X = np.array([[1.0, 2.0]])
    Wr = np.array([[1.0, 0.0, -1.0], [0.5, 1.0, 2.0]])
    L = oracle.router_logits(X, Wr, bias=np.array([0.0, 1.0, -1.0]), dtype=np.float64)
    np.testing.assert_allclose(L, [[2.0, 3.0, 2.0]])


def _brute_metadata(member):
    T, E = member.shape
    row_token, row_expert = [], []
    for e in range(E):
        for t in range(T):
            if member[t, e]:
                row_token.append(t)
                row_expert.append(e)
    tok_rows = []
    for t in range(T):
        for e in range(E):
            if member[t, e]:
                tok_rows.append(next(r for r in range(len(row_token)) if row_token[r] == t and row_expert[r] == e))
    return np.array(row_token), np.array(row_expert), np.array(tok_rows)


def test_metadata_brute_force_and_invariants():
    rng = np.random.default_rng(3)
    T, E, K = 40, 6, 3
    S = rng.random((T, E)).astype(np.float32)
    idx = oracle.topk_select(S, K)
    member = oracle.tc_membership(idx, E)
    R = oracle.routing_from_membership(member, S)
    rt, re, tr = _brute_metadata(member)
    np.testing.assert_array_equal(R.row_token, rt)
    np.testing.assert_array_equal(R.row_expert, re)
    np.testing.assert_array_equal(R.tok_rows, tr)
    assert R.counts.sum() == T * K
    assert np.all(np.diff(R.offsets) >= 0) and R.offsets[0] == 0 and R.offsets[-1] == T * K
    np.testing.assert_array_equal(R.tok_offsets, np.arange(T + 1) * K)
    for e in range(E):
        seg = R.row_token[R.offsets[e]:R.offsets[e + 1]]
        assert np.all(np.diff(seg) > 0)
    for t in range(T):
        rows = R.tok_rows[R.tok_offsets[t]:R.tok_offsets[t + 1]]
        assert np.all(R.row_token[rows] == t)
        assert np.all(np.diff(R.row_expert[rows]) > 0)
        assert set(R.row_expert[rows].tolist()) == set(idx[t].tolist())


def test_weights_are_softmax_over_selected_logits():
    rng = np.random.default_rng(4)
    T, E, K, d = 30, 10, 4, 16
    X = rng.standard_normal((T, d))
    Wr = rng.standard_normal((d, E)) * 0.3
    S, idx, R = oracle.route(X, Wr, K, dtype=np.float64)
    L = X @ Wr
    for t in range(T):
        sel = idx[t]
        z = np.exp(L[t, sel] - L[t, sel].max())
        np.testing.assert_allclose(R.weights[t, sel], z / z.sum(), rtol=1e-12)
        rows = R.tok_rows[R.tok_offsets[t]:R.tok_offsets[t + 1]]
        np.testing.assert_allclose(R.row_w[rows].sum(), 1.0, rtol=1e-12)


def test_empty_token_and_empty_expert():
    member = np.zeros((4, 3), bool)
    member[0, 2] = True
    member[2, 2] = True
    member[2, 0] = True
    S = np.full((4, 3), 1.0 / 3, np.float32)
    R = oracle.routing_from_membership(member, S)
    np.testing.assert_array_equal(R.counts, [1, 0, 2])
    np.testing.assert_array_equal(R.offsets, [0, 1, 1, 3])
    np.testing.assert_array_equal(R.row_token, [2, 0, 2])
    np.testing.assert_array_equal(R.tok_offsets, [0, 1, 1, 3, 3])
    np.testing.assert_array_equal(R.tok_rows, [1, 0, 2])
    assert np.all(R.weights[1] == 0) and np.all(R.weights[3] == 0)
    np.testing.assert_allclose(R.row_w, [0.5, 1.0, 0.5])
