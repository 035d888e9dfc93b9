"""Pins of the oracle's forward and backward.

* dense masked evaluation (every expert on every token) with torch fp64 autograd,
* central finite differences with the routing frozen,
* the dS identity <dA', A> = <dO, Y> computed both ways,
* closed-form special cases (K = E with a zero router, E = K = 1),
* the cached-activation byte count.
"""
import numpy as np
import pytest

import oracle
from dense_reference import dense_moe, dense_ffn, rel_err

F64 = np.float64


def _case(seed, T, d, n, E, K, router_std=0.5, bias=False):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((T, d)) * 0.5
    Wr = rng.standard_normal((d, E)) * router_std
    W1 = rng.standard_normal((E, d, 2 * n)) * 0.3
    W2 = rng.standard_normal((E, n, d)) * 0.3
    dO = rng.standard_normal((T, d))
    b = rng.standard_normal(E) if bias else None
    return X, Wr, W1, W2, dO, b


def _run_oracle(X, Wr, W1, W2, dO, b, K, round_mode=None, M=4):
    S, idx, R = oracle.route(X, Wr, K, bias=b, dtype=F64)
    member = R.member
    if round_mode is not None:
        member, _, _ = oracle.round_tokens(S, member, M, mode=round_mode)
        R = oracle.routing_from_membership(member, S, dtype=F64)
    fw = oracle.forward(X, W1, W2, R, dtype=F64)
    bw = oracle.backward(dO, X, fw["H"], W1, W2, Wr, R, dtype=F64)
    return R, fw, bw


@pytest.mark.parametrize("seed,T,d,n,E,K,bias,round_mode", [
    (0, 24, 8, 4, 4, 2, False, None),
    (1, 33, 16, 8, 6, 3, True, None),
    (2, 40, 8, 4, 8, 1, False, None),
    (3, 48, 8, 6, 5, 2, False, "nearest"),
    (4, 48, 8, 6, 5, 3, True, "up"),
    (5, 30, 8, 4, 4, 2, False, "down"),
])
def test_against_dense_autograd(seed, T, d, n, E, K, bias, round_mode):
    X, Wr, W1, W2, dO, b = _case(seed, T, d, n, E, K, bias=bias)
    R, fw, bw = _run_oracle(X, Wr, W1, W2, dO, b, K, round_mode)
    ref = dense_moe(X, Wr, W1, W2, R.member, dO, bias=b)
    def close(a, r):
        # relative to the tensor's scale; K = 1 has an identically-zero router
        # gradient, where torch leaves ~1e-17 of rounding
        return np.abs(a - r).max() <= 1e-10 * max(np.abs(r).max(), 1e-6)
    for k in ("O",):
        assert close(fw[k], ref[k]), k
    for k in ("dX", "dW1", "dW2", "dWr", "dbias"):
        assert close(bw[k], ref[k]), k
    # dS of each routed pair equals d loss / d s_{t,e}
    assert close(bw["dS"], ref["dS"][R.row_token, R.row_expert])
    np.testing.assert_allclose(R.weights, ref["w"], rtol=1e-12, atol=1e-15)


def test_finite_differences_routing_frozen():
    X, Wr, W1, W2, dO, b = _case(11, 16, 8, 4, 4, 2, bias=True)
    K = 2
    S, idx, R = oracle.route(X, Wr, K, bias=b, dtype=F64)
    member = R.member

    def loss(X_, Wr_, W1_, W2_, b_):
        S_ = oracle.softmax_scores(oracle.router_logits(X_, Wr_, b_, F64))
        R_ = oracle.routing_from_membership(member, S_, dtype=F64)
        return float((oracle.forward(X_, W1_, W2_, R_, dtype=F64)["O"] * dO).sum())

    fw = oracle.forward(X, W1, W2, R, dtype=F64)
    bw = oracle.backward(dO, X, fw["H"], W1, W2, Wr, R, dtype=F64)
    h = 1e-6
    rng = np.random.default_rng(0)
    params = {"X": X, "Wr": Wr, "W1": W1, "W2": W2, "b": b}
    grads = {"X": bw["dX"], "Wr": bw["dWr"], "W1": bw["dW1"], "W2": bw["dW2"], "b": bw["dbias"]}
    for name, P in params.items():
        for _ in range(6):
            i = tuple(rng.integers(0, s) for s in P.shape)
            Pp, Pm = P.copy(), P.copy()
            Pp[i] += h
            Pm[i] -= h
            args_p = {**params, name: Pp}
            args_m = {**params, name: Pm}
            fd = (loss(args_p["X"], args_p["Wr"], args_p["W1"], args_p["W2"], args_p["b"])
                  - loss(args_m["X"], args_m["Wr"], args_m["W1"], args_m["W2"], args_m["b"])) / (2 * h)
            assert abs(fd - grads[name][i]) < 1e-6 * max(1.0, abs(fd)), (name, i, fd, grads[name][i])


def test_dS_identity_both_ways():
    X, Wr, W1, W2, dO, b = _case(21, 50, 16, 8, 8, 3)
    R, fw, bw = _run_oracle(X, Wr, W1, W2, dO, b, 3)
    # <dO_t, Y_{e,t}> from the forward's Y versus <dA', A> from the backward
    via_Y = (dO[R.row_token] * fw["Y"]).sum(axis=1)
    np.testing.assert_allclose(bw["dS"], via_Y, rtol=1e-10, atol=1e-12)
    # dW2 = A'^T dO_e = A^T (s dO_e)
    for e in range(W1.shape[0]):
        r0, r1 = R.offsets[e], R.offsets[e + 1]
        dY = R.row_w[r0:r1, None] * dO[R.row_token[r0:r1]]
        np.testing.assert_allclose(bw["dW2"][e], fw["A"][r0:r1].T @ dY, rtol=1e-10, atol=1e-12)


def test_K_equals_E_zero_router_is_mean_ffn():
    T, d, n, E = 20, 8, 4, 4
    X, _, W1, W2, dO, _ = _case(31, T, d, n, E, E)
    Wr = np.zeros((d, E))
    R, fw, _ = _run_oracle(X, Wr, W1, W2, dO, None, E)
    mean = sum(dense_ffn(X, W1[e], W2[e]) for e in range(E)) / E
    np.testing.assert_allclose(fw["O"], mean, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(R.row_w, 1.0 / E, rtol=1e-14)


def test_single_expert_is_dense_ffn():
    T, d, n = 17, 8, 4
    X, Wr, W1, W2, dO, _ = _case(41, T, d, n, 1, 1)
    R, fw, bw = _run_oracle(X, Wr, W1, W2, dO, None, 1)
    np.testing.assert_allclose(fw["O"], dense_ffn(X, W1[0], W2[0]), rtol=1e-12, atol=1e-14)
    # one expert: weight 1 and no router gradient
    assert np.all(bw["dWr"] == 0)


def test_sampled_variants_match_dense():
    X, Wr, W1, W2, dO, b = _case(51, 30, 8, 4, 6, 2)
    S, idx, R = oracle.route(X, Wr, 2, dtype=F64)
    member, _, _ = oracle.round_tokens(S, R.member, 4)
    R = oracle.routing_from_membership(member, S, dtype=F64)
    ref = dense_moe(X, Wr, W1, W2, R.member, dO)
    toks = [0, 3, 7, 29]
    O = oracle.forward_tokens(X, W1, W2, R, toks, dtype=F64)
    np.testing.assert_allclose(O, ref["O"][toks], rtol=1e-10, atol=1e-12)
    dX, rows, dS, dl = oracle.backward_tokens(dO, X, W1, W2, Wr, R, toks, dtype=F64)
    np.testing.assert_allclose(dX, ref["dX"][toks], rtol=1e-10, atol=1e-12)
    for t, rr, ds in zip(toks, rows, dS):
        np.testing.assert_allclose(ds, ref["dS"][t, R.row_expert[rr]], rtol=1e-10, atol=1e-12)


def test_fp32_oracle_close_to_fp64():
    X, Wr, W1, W2, dO, b = _case(61, 64, 32, 16, 8, 2)
    S, idx, R64 = oracle.route(X, Wr, 2, dtype=F64)
    R32 = oracle.routing_from_membership(R64.member, S.astype(np.float32), dtype=np.float32)
    f64 = oracle.forward(X, W1, W2, R64, dtype=F64)
    f32 = oracle.forward(X, W1, W2, R32, dtype=np.float32)
    assert f32["O"].dtype == np.float32
    assert rel_err(f32["O"], f64["O"]) < 1e-5


def test_cached_bytes_equals_the_arrays_backward_consumes():
    """The bytes are those of the activations the oracle's backward takes
    (X and the forward's H), stored as bf16 (2-byte) arrays: measured with
    nbytes on the arrays themselves, not from a formula."""
    X, Wr, W1, W2, dO, b = _case(71, 40, 16, 8, 6, 3)
    R, fw, _ = _run_oracle(X, Wr, W1, W2, dO, b, 3)
    as_bf16 = lambda a: np.zeros(a.shape, np.uint16)  # noqa: E731  (2 bytes per element)
    T, d = X.shape
    n = W2.shape[1]
    assert oracle.cached_bytes(T, d, n, R.P) == as_bf16(X).nbytes + as_bf16(fw["H"]).nbytes


def test_cached_bytes_is_a_dense_models_and_granularity_free():
    """Section 3.2: the cache equals a dense SwiGLU FFN's with the same
    activated parameters (intermediate width nK: X [T,d] and H [T,2nK] in
    bf16) and so does not change with granularity at fixed nK.  At the 7B
    shape (T=32768, d=1536, n=256, K=8) that is 100663296 + 268435456 bytes."""
    T, d = 32768, 1536
    dense = np.zeros((T, d), np.uint16).nbytes + np.zeros((T, 2 * 2048), np.uint16).nbytes
    for n, K in ((256, 8), (512, 4), (1024, 2), (128, 16)):
        assert oracle.cached_bytes(T, d, n, T * K) == dense
    assert dense == 100663296 + 268435456


@pytest.mark.parametrize("seed,round_mode", [(81, None), (82, "nearest")])
def test_expert_biases_against_dense_autograd(seed, round_mode):
    """Expert biases b1 (up-projection) and b2 (down-projection): O, every
    gradient, db1, db2 and dS (now <dA', A> + <dO, b2_e>) equal the dense
    masked autograd reference."""
    X, Wr, W1, W2, dO, b = _case(seed, 36, 8, 4, 5, 2, bias=True)
    rng = np.random.default_rng(seed + 100)
    b1 = rng.standard_normal((5, 8)) * 0.4
    b2 = rng.standard_normal((5, 8)) * 0.4
    S, idx, R = oracle.route(X, Wr, 2, bias=b, dtype=F64)
    if round_mode:
        member, _, _ = oracle.round_tokens(S, R.member, 4, mode=round_mode)
        R = oracle.routing_from_membership(member, S, dtype=F64)
    fw = oracle.forward(X, W1, W2, R, dtype=F64, b1=b1, b2=b2)
    bw = oracle.backward(dO, X, fw["H"], W1, W2, Wr, R, dtype=F64, b2=b2)
    ref = dense_moe(X, Wr, W1, W2, R.member, dO, bias=b, b1=b1, b2=b2)
    for k, got in (("O", fw["O"]), ("dX", bw["dX"]), ("dW1", bw["dW1"]), ("dW2", bw["dW2"]),
                   ("dWr", bw["dWr"]), ("dbias", bw["dbias"]), ("db1", bw["db1"]), ("db2", bw["db2"])):
        np.testing.assert_allclose(got, ref[k], rtol=1e-10, atol=1e-12, err_msg=k)
    np.testing.assert_allclose(bw["dS"], ref["dS"][R.row_token, R.row_expert], rtol=1e-10, atol=1e-12)
    # the identity extended: dS = <dO_t, Y_{e,t}> with the biased Y
    np.testing.assert_allclose(bw["dS"], (dO[R.row_token] * fw["Y"]).sum(axis=1), rtol=1e-10, atol=1e-12)
    # without b2 in the backward the bias term is missing: the pin sees it
    bw0 = oracle.backward(dO, X, fw["H"], W1, W2, Wr, R, dtype=F64)
    assert np.abs(bw0["dS"] - bw["dS"]).max() > 1e-3


def test_expert_bias_finite_differences():
    X, Wr, W1, W2, dO, b = _case(91, 16, 8, 4, 4, 2, bias=True)
    rng = np.random.default_rng(5)
    b1 = rng.standard_normal((4, 8)) * 0.4
    b2 = rng.standard_normal((4, 8)) * 0.4
    S, idx, R = oracle.route(X, Wr, 2, bias=b, dtype=F64)
    member = R.member

    def loss(b1_, b2_, Wr_):
        S_ = oracle.softmax_scores(oracle.router_logits(X, Wr_, b, F64))
        R_ = oracle.routing_from_membership(member, S_, dtype=F64)
        return float((oracle.forward(X, W1, W2, R_, dtype=F64, b1=b1_, b2=b2_)["O"] * dO).sum())

    fw = oracle.forward(X, W1, W2, R, dtype=F64, b1=b1, b2=b2)
    bw = oracle.backward(dO, X, fw["H"], W1, W2, Wr, R, dtype=F64, b2=b2)
    h = 1e-6
    for name in ("b1", "b2", "Wr"):
        P = {"b1": b1, "b2": b2, "Wr": Wr}[name]
        g = {"b1": bw["db1"], "b2": bw["db2"], "Wr": bw["dWr"]}[name]
        for i in [tuple(rng.integers(0, s) for s in P.shape) for _ in range(6)]:
            args_p = {"b1_": b1, "b2_": b2, "Wr_": Wr}
            args_m = dict(args_p)
            Pp, Pm = P.copy(), P.copy()
            Pp[i] += h
            Pm[i] -= h
            args_p[name + "_"] = Pp
            args_m[name + "_"] = Pm
            fd = (loss(**args_p) - loss(**args_m)) / (2 * h)
            assert abs(fd - g[i]) < 1e-6 * max(1.0, abs(fd)), (name, i, fd, g[i])


def test_weight_grad_columns_match_dense_autograd():
    """The column-restricted weight gradients equal the dense masked autograd
    reference (not the oracle's own full backward) for every expert and a mix
    of columns, under token rounding."""
    X, Wr, W1, W2, dO, b = _case(61, 36, 8, 6, 5, 2)
    S, idx, R = oracle.route(X, Wr, 2, dtype=F64)
    member, _, _ = oracle.round_tokens(S, R.member, 4)
    R = oracle.routing_from_membership(member, S, dtype=F64)
    ref = dense_moe(X, Wr, W1, W2, R.member, dO)
    n = 6
    cols = [0, 2, 5]
    for e in range(5):
        dW1c, dW2r = oracle.weight_grad_columns(dO, X, W1, W2, R, e, cols, dtype=F64)
        for i, j in enumerate(cols):
            np.testing.assert_allclose(dW1c[:, 0, i], ref["dW1"][e][:, j], rtol=1e-10, atol=1e-12)
            np.testing.assert_allclose(dW1c[:, 1, i], ref["dW1"][e][:, n + j], rtol=1e-10, atol=1e-12)
            np.testing.assert_allclose(dW2r[i], ref["dW2"][e][j, :], rtol=1e-10, atol=1e-12)
