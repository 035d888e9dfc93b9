"""Oracle of the MoE layer forward and backward -- TEST INFRASTRUCTURE ONLY.

Per routed pair (t,e) -- one "row" of the expert-major layout -- the layer
computes (Section 2.2 and the forward algorithm of Section 3):

    h = x_t W1_e                 (length 2n; gate = first n columns, up = last n)
    a = SwiGLU(h) = SiLU(h_gate) * h_up,   SiLU(z) = z / (1 + exp(-z))
    y = a W2_e
    O_t = sum over the rows of token t of s_{t,e} * y

Optional expert biases (the footnote of the "Gradient computation" appendix):
b1_e [2n] is added to h and b2_e [d] to y.  Then dS_{t,e} = <dO_t, y> gains
<dO_t, b2_e> next to <dA', a>, and db1_e = sum of dH over the expert's rows,
db2_e = sum of s * dO_t over them.  (The footnote prints the extra term with
a garbled second operand; the down-projection bias is the one that makes
<dO_t, y> differ from <dA', a>.)

The backward follows the "Gradient computation" appendix: with
dA' = dO_t W2_e^T, dS_{t,e} = <dA', a> (boxed identity), dA = s * dA',
dH = dSwiGLU(dA, h), A' = s * a, dW2_e = A'^T dO_e, dX~ = dH W1_e^T,
dW1_e = X_e^T dH, dX_t = sum of dX~ over the token's rows (up-projection
backward algorithm of Appendix E), plus the router's own gradient.

Every step is a per-expert dense matmul (a library primitive) or an
elementwise map; nothing is blocked, fused or reordered.
"""
from __future__ import annotations

import numpy as np


def _sigmoid(z):
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-z))


def swiglu(H):
    """A = SiLU(H[:, :n]) * H[:, n:] (gate columns first, up columns last)."""
    n = H.shape[1] // 2
    g, u = H[:, :n], H[:, n:]
    return g * _sigmoid(g) * u


def dswiglu(dA, H):
    """Gradient of SwiGLU w.r.t. its input H given dA (dH = dSwiGLU(dA, H)).

    With sigma = sigmoid(g): d/dg [g sigma(g)] = sigma (1 + g (1 - sigma)), so
    dH_gate = dA * u * sigma * (1 + g (1 - sigma)) and dH_up = dA * g * sigma.
    """
    n = H.shape[1] // 2
    g, u = H[:, :n], H[:, n:]
    s = _sigmoid(g)
    dg = dA * u * s * (1.0 + g * (1.0 - s))
    du = dA * g * s
    return np.concatenate([dg, du], axis=1)


def forward(X, W1, W2, R, dtype=np.float32, b1=None, b2=None):
    """MoE forward over routing ``R`` (up-proj A kernel, down-proj Y kernel,
    expert aggregation O kernel of the forward algorithm, Section 3).

    b1 [E,2n] and b2 [E,d] are optional expert biases of the up- and
    down-projection.  Returns dict with O [T,d] and the per-row
    intermediates H [P,2n], A [P,n], Y [P,d] (the layer caches only X and H,
    Section 3.2).
    """
    X = np.asarray(X, dtype)
    W1 = np.asarray(W1, dtype)
    W2 = np.asarray(W2, dtype)
    b1 = None if b1 is None else np.asarray(b1, dtype)
    b2 = None if b2 is None else np.asarray(b2, dtype)
    T, d = X.shape
    E, _, n2 = W1.shape
    P = R.P
    H = np.zeros((P, n2), dtype)
    A = np.zeros((P, n2 // 2), dtype)
    Y = np.zeros((P, d), dtype)
    for e in range(E):
        r0, r1 = int(R.offsets[e]), int(R.offsets[e + 1])
        if r0 == r1:
            continue
        Xe = X[R.row_token[r0:r1]]           # gather
        He = Xe @ W1[e]
        if b1 is not None:
            He = He + b1[e]
        Ae = swiglu(He)
        H[r0:r1] = He
        A[r0:r1] = Ae
        Ye = Ae @ W2[e]
        if b2 is not None:
            Ye = Ye + b2[e]
        Y[r0:r1] = Ye
    O = np.zeros((T, d), dtype)
    # O_t = sum_e pi_{t,e} s_{t,e} Y_{e,t}; np.add.at accumulates rows in
    # row order, i.e. expert-ascending per token
    np.add.at(O, R.row_token, R.row_w.astype(dtype)[:, None] * Y)
    return {"O": O, "H": H, "A": A, "Y": Y}


def backward(dO, X, H, W1, W2, Wr, R, dtype=np.float32, b2=None):
    """MoE backward over routing ``R`` given the cached H.

    Expert part: the dH and dW2 kernels of the down-projection backward
    (Section 3), the dX~, dW1 and dX kernels of the up-projection backward
    (Appendix E), with dS, dA and A' as in the "Gradient computation" appendix.
    With a down-projection bias b2 [E,d], dS of a row gains <dO_t, b2_e>.
    The expert-bias gradients db1 [E,2n] (column sums of the expert's dH rows)
    and db2 [E,d] (column sums of its s * dO_t rows) are always returned.

    Router part (the paper leaves the router to the caller): the weights are a
    softmax over the token's selected logits, so for a selected expert j
    dl_j = s_j (dS_j - sum_k s_k dS_k) and 0 elsewhere; then
    dW_r = X^T dL, db = column sums of dL and dX += dL W_r^T.  Routing and
    rounding decisions are piecewise constant and carry no gradient.
    """
    dO = np.asarray(dO, dtype)
    X = np.asarray(X, dtype)
    H = np.asarray(H, dtype)
    W1 = np.asarray(W1, dtype)
    W2 = np.asarray(W2, dtype)
    T, d = X.shape
    E, _, n2 = W1.shape
    n = n2 // 2
    P = R.P
    w = R.row_w.astype(dtype)
    dS = np.zeros(P, dtype)
    dH = np.zeros((P, n2), dtype)
    Ap = np.zeros((P, n), dtype)
    dXt = np.zeros((P, d), dtype)
    dW1 = np.zeros_like(W1)
    dW2 = np.zeros_like(W2)
    db1 = np.zeros((E, n2), dtype)
    db2 = np.zeros((E, d), dtype)
    b2 = None if b2 is None else np.asarray(b2, dtype)
    for e in range(E):
        r0, r1 = int(R.offsets[e]), int(R.offsets[e + 1])
        if r0 == r1:
            continue
        tok = R.row_token[r0:r1]
        dOe = dO[tok]                         # gather dO
        He = H[r0:r1]
        dAp = dOe @ W2[e].T                   # dA' = dO_e W2_e^T
        Ae = swiglu(He)                       # recompute A from H
        dS[r0:r1] = (dAp * Ae).sum(axis=1)    # dS = <dA', A>
        if b2 is not None:
            dS[r0:r1] += dOe @ b2[e]          # + <dO_t, b2_e>
        dA = w[r0:r1, None] * dAp             # dA = s dA'
        dHe = dswiglu(dA, He)
        Ape = w[r0:r1, None] * Ae             # A' = s A
        dH[r0:r1] = dHe
        Ap[r0:r1] = Ape
        db1[e] = dHe.sum(axis=0)              # db1 = column sums of dH_e
        db2[e] = (w[r0:r1, None] * dOe).sum(axis=0)  # db2 = column sums of s dO_e
        dW2[e] = Ape.T @ dOe                  # dW2 = A'^T dO_e
        dW1[e] = X[tok].T @ dHe               # dW1 = X_e^T dH
        dXt[r0:r1] = dHe @ W1[e].T            # dX~ = dH W1_e^T
    dX = np.zeros((T, d), dtype)
    np.add.at(dX, R.row_token, dXt)           # dX_t = sum over rows of t
    # router backward
    g = np.zeros(T, dtype)
    np.add.at(g, R.row_token, w * dS)
    dl = w * (dS - g[R.row_token])
    dL = np.zeros((T, E), dtype)
    dL[R.row_token, R.row_expert] = dl
    out = {"dX_experts": dX.copy(), "dW1": dW1, "dW2": dW2, "dS": dS, "dH": dH,
           "Ap": Ap, "dXt": dXt, "dL": dL, "db1": db1, "db2": db2}
    if Wr is not None:
        Wr = np.asarray(Wr, dtype)
        out["dWr"] = X.T @ dL
        out["dbias"] = dL.sum(axis=0)
        dX = dX + dL @ Wr.T
    out["dX"] = dX
    return out


def _row_values(x, W1e, W2e, dtype):
    h = x @ W1e
    a = swiglu(h[None, :])[0]
    return h, a, a @ W2e


def forward_tokens(X, W1, W2, R, tokens, dtype=np.float32):
    """O_t for the listed tokens only, computed row by row (for sampled checks)."""
    X = np.asarray(X, dtype)
    d = X.shape[1]
    out = np.zeros((len(tokens), d), dtype)
    for i, t in enumerate(tokens):
        for j in range(int(R.tok_offsets[t]), int(R.tok_offsets[t + 1])):
            r = int(R.tok_rows[j])
            e = int(R.row_expert[r])
            _, _, y = _row_values(X[t], np.asarray(W1[e], dtype), np.asarray(W2[e], dtype), dtype)
            out[i] += dtype(R.row_w[r]) * y
    return out


def backward_tokens(dO, X, W1, W2, Wr, R, tokens, dtype=np.float32):
    """dX_t (expert part + router part), and dS / dl of the token's rows,
    for the listed tokens only, row by row from the definitions above."""
    X = np.asarray(X, dtype)
    dO = np.asarray(dO, dtype)
    d = X.shape[1]
    dX = np.zeros((len(tokens), d), dtype)
    rows_out, dS_out, dl_out = [], [], []
    for i, t in enumerate(tokens):
        rows = [int(R.tok_rows[j]) for j in range(int(R.tok_offsets[t]), int(R.tok_offsets[t + 1]))]
        dS = []
        for r in rows:
            e = int(R.row_expert[r])
            W1e = np.asarray(W1[e], dtype)
            W2e = np.asarray(W2[e], dtype)
            h, a, _ = _row_values(X[t], W1e, W2e, dtype)
            dAp = W2e @ dO[t]
            dS.append(dtype(np.dot(dAp, a)))
            s = dtype(R.row_w[r])
            dh = dswiglu((s * dAp)[None, :], h[None, :])[0]
            dX[i] += W1e @ dh
        w = np.array([R.row_w[r] for r in rows], dtype)
        dS = np.array(dS, dtype)
        dl = w * (dS - np.dot(w, dS)) if rows else np.zeros(0, dtype)
        if Wr is not None:
            for r, v in zip(rows, dl):
                dX[i] += v * np.asarray(Wr, dtype)[:, int(R.row_expert[r])]
        rows_out.append(rows)
        dS_out.append(dS)
        dl_out.append(dl)
    return dX, rows_out, dS_out, dl_out


def weight_grad_columns(dO, X, W1, W2, R, e, cols, dtype=np.float32):
    """Columns of expert e's weight gradients from its routed rows only (for
    sampled checks at sizes where the full backward is too slow).

    For each j in cols (0 <= j < n), over the expert's rows (token t, score s):
    h = [x_t W1_e[:, j], x_t W1_e[:, n+j]] (gate, up), a = SwiGLU(h),
    dA'_j = dO_t W2_e[j, :]^T, dH = dSwiGLU(s dA'_j, h) -- the down-projection
    backward of Section 3 and the up-projection backward of Appendix E
    restricted to one column pair -- then
    dW1_e[:, j] = X_e^T dH_gate, dW1_e[:, n+j] = X_e^T dH_up and
    dW2_e[j, :] = (s a)^T dO_e.
    Returns (dW1 columns [d, 2, len(cols)] as gate/up, dW2 rows [len(cols), d]).
    """
    X = np.asarray(X, dtype)
    dO = np.asarray(dO, dtype)
    n = W2.shape[1]
    lo, hi = int(R.offsets[e]), int(R.offsets[e + 1])
    tok = np.asarray(R.row_token[lo:hi], np.int64)
    s = np.asarray(R.row_w[lo:hi], dtype)[:, None]
    Xe, dOe = X[tok], dO[tok]
    W1e, W2e = np.asarray(W1[e], dtype), np.asarray(W2[e], dtype)
    d = X.shape[1]
    dW1c = np.zeros((d, 2, len(cols)), dtype)
    dW2r = np.zeros((len(cols), d), dtype)
    for i, j in enumerate(cols):
        H = np.stack([Xe @ W1e[:, j], Xe @ W1e[:, n + j]], axis=1)  # [rows, 2]: n = 1 column pair
        a = swiglu(H)                                                # [rows, 1]
        dAp = (dOe @ W2e[j, :])[:, None]
        dH = dswiglu(s * dAp, H)
        dW1c[:, 0, i] = Xe.T @ dH[:, 0]
        dW1c[:, 1, i] = Xe.T @ dH[:, 1]
        dW2r[i] = ((s * a)[:, 0]) @ dOe
    return dW1c, dW2r


def cached_bytes(T, d, n, P):
    """Activation bytes kept from forward to backward in bf16: X and H,
    2Td + 4Pn (Section 3.2; P = TK under TC)."""
    return 2 * T * d + 4 * P * n
