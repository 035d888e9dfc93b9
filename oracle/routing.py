"""Oracle of the MoE routing steps -- TEST INFRASTRUCTURE ONLY.

Router scores, token-choice (TC) top-K selection, the routing metadata that the
grouped GEMMs and the aggregation consume, and token rounding (TR).

Routing is defined on one fp32 tensor, the full softmax score matrix
S_full[T,E]; every integer result (selected experts, counts, offsets, row
order, rounding decisions and membership) is a deterministic function of it.
"""
from __future__ import annotations

import dataclasses
import numpy as np


def router_logits(X, Wr, bias=None, dtype=np.float32):
    """Router logits L = X W_r (+ b).

    The router is a linear map of the token embeddings to one score per expert
    (Section 2.3, token-choice routing on expert scores S_{t,e}); the optional
    per-expert bias b is added to every token's logits.
    """
    L = np.asarray(X, dtype) @ np.asarray(Wr, dtype)
    if bias is not None:
        L = L + np.asarray(bias, dtype)[None, :]
    return L


def softmax_scores(L):
    """S_full[t,:] = softmax over all E experts of the logits of token t.

    The row maximum is subtracted before exponentiation (Section 2.3; the
    throughput experiments of Section 6.2 use a TC top-K router with softmax
    scores).
    """
    L = np.asarray(L)
    m = L.max(axis=1, keepdims=True)
    z = np.exp(L - m)
    return z / z.sum(axis=1, keepdims=True)


def topk_select(S, K):
    """Token-choice top-K: TopK_e(S_{t,e}, K) for every token (Section 2.3).

    The selection uses the total order (score descending, expert index
    ascending), so equal scores go to the lower expert index -- the stable
    result that the paper's top-K kernel guarantees (Appendix D).  Returns
    int32 [T,K] in that order.
    """
    S = np.asarray(S)
    T, E = S.shape
    eidx = np.broadcast_to(np.arange(E), (T, E))
    # np.lexsort sorts by the last key first: -S ascending == S descending,
    # then the expert index ascending.
    order = np.lexsort((eidx, -S), axis=1)
    return order[:, :K].astype(np.int32)


def tc_membership(topk_idx, E):
    """Binary routing matrix pi in {0,1}^{T x E} (Appendix A) from the TC selection."""
    topk_idx = np.asarray(topk_idx)
    T = topk_idx.shape[0]
    pi = np.zeros((T, E), dtype=bool)
    pi[np.arange(T)[:, None], topk_idx] = True
    return pi


@dataclasses.dataclass
class Routing:
    """Routing metadata for one routing matrix pi.

    Expert-major rows are ordered by (expert ascending, token ascending);
    the token-major view lists each token's rows by expert ascending.
    """
    member: np.ndarray      # bool [T,E]   pi
    weights: np.ndarray     # [T,E]        s_{t,e} (0 where pi = 0)
    counts: np.ndarray      # int32 [E]    f_e
    offsets: np.ndarray     # int32 [E+1]  exclusive scan of f_e
    row_token: np.ndarray   # int32 [P]    token of each expert-major row
    row_expert: np.ndarray  # int32 [P]    expert of each row
    row_w: np.ndarray       # [P]          weight of each row
    tok_offsets: np.ndarray  # int32 [T+1]
    tok_rows: np.ndarray    # int32 [P]    rows of each token, expert ascending
    row_of: np.ndarray      # int32 [T,E]  row index of pair (t,e), -1 if absent

    @property
    def P(self):
        return int(self.offsets[-1])


def routing_from_membership(member, S, dtype=np.float32):
    """Metadata for routing matrix ``member`` with scores ``S``.

    The weight of a routed pair is its softmax score renormalised over the
    token's selected experts, s_{t,e} = S_{t,e} / sum_{e' in sel(t)} S_{t,e'}
    (softmax over the selected logits: the top-K kernel of Appendix D fuses a
    softmax over the top-K values, and Section 6.3.1 trains TR with softmax
    renormalisation).  The denominator is accumulated over
    experts in ascending order.  A token with no expert gets no weight.
    """
    member = np.asarray(member, dtype=bool)
    S = np.asarray(S, dtype)
    T, E = member.shape
    counts = member.sum(axis=0).astype(np.int32)
    offsets = np.zeros(E + 1, np.int32)
    offsets[1:] = np.cumsum(counts)
    P = int(offsets[-1])
    # expert-major enumeration: nonzero of pi^T walks (e asc, t asc)
    es, ts = np.nonzero(member.T)
    row_token = ts.astype(np.int32)
    row_expert = es.astype(np.int32)
    row_of = np.full((T, E), -1, np.int32)
    row_of[ts, es] = np.arange(P, dtype=np.int32)
    # renormalisation denominators, summed over experts in ascending order
    denom = np.zeros(T, dtype)
    for e in range(E):
        denom = denom + np.where(member[:, e], S[:, e], dtype(0))
    weights = np.zeros((T, E), dtype)
    nz = denom > 0
    weights[nz] = np.where(member[nz], S[nz] / denom[nz, None], dtype(0))
    row_w = weights[ts, es]
    tok_counts = member.sum(axis=1)
    tok_offsets = np.zeros(T + 1, np.int32)
    tok_offsets[1:] = np.cumsum(tok_counts)
    # boolean indexing walks (t asc, e asc): token-major, expert ascending
    tok_rows = row_of[member].astype(np.int32)
    return Routing(member, weights, counts, offsets, row_token, row_expert, row_w,
                   tok_offsets, tok_rows, row_of)


ROUND_MODES = ("nearest", "up", "down", "balance", "stochastic")


def round_tokens(S, tc_member, m_tile, mode="nearest", u=None):
    """Token rounding (Section 5.2; rounding subroutines in the appendix ablation).

    Per expert e with TC frequency f_e, lo = floor(f_e/M)*M and
    hi = ceil(f_e/M)*M.  The rounding subroutine picks f^TR_e in {lo, hi}:

    * "nearest" (NR-f, the default): hi iff hi - f_e < f_e - lo (strict, so
      the exact midpoint rounds down);
    * "up" / "down": always hi / always lo (DOWN is TC token dropping);
    * "balance" (Balance-f): a running residual z over experts in index
      order; hi iff |hi - f_e + z| < |lo - f_e + z|, then z += chosen - f_e;
    * "stochastic" (SR-f): hi iff u_e * M < f_e - lo, with u_e ~ U[0,1)
      passed in (fp32), i.e. Bernoulli((f_e - lo)/M).

    If hi exceeds T the expert cannot be padded and takes lo.

    Membership follows the two-step sort: each expert orders all T tokens by
    (TC first, score descending, token ascending) and keeps the first f^TR_e,
    so rounding drops the lowest-scored TC tokens or pads the highest-scored
    non-TC tokens and only touches the expert's last tile.

    Returns (member_tr bool[T,E], f_tr int32[E], round_dir int32[E]).
    """
    S = np.asarray(S)
    tc_member = np.asarray(tc_member, dtype=bool)
    T, E = S.shape
    M = int(m_tile)
    f = tc_member.sum(axis=0).astype(np.int64)
    lo = (f // M) * M
    hi = ((f + M - 1) // M) * M
    can_pad = hi <= T
    if mode == "nearest":
        pad = (hi - f) < (f - lo)
    elif mode == "up":
        pad = hi > f
    elif mode == "down":
        pad = np.zeros(E, bool)
    elif mode == "stochastic":
        if u is None:
            raise ValueError("stochastic rounding needs the uniforms u[E]")
        u = np.asarray(u, np.float32)
        pad = (u * np.float32(M)) < (f - lo).astype(np.float32)
    elif mode == "balance":
        pad = np.zeros(E, bool)
        z = 0
        for e in range(E):
            r_up = int(hi[e] - f[e])
            r_dn = int(lo[e] - f[e])
            if abs(r_up + z) < abs(r_dn + z) and can_pad[e]:
                pad[e] = True
                z += r_up
            else:
                z += r_dn
    else:
        raise ValueError(f"unknown rounding mode {mode!r}")
    pad = pad & can_pad
    f_tr = np.where(pad, hi, lo)
    member = np.zeros((T, E), dtype=bool)
    tok = np.arange(T)
    for e in range(E):
        # primary key last: not-TC ascending (TC first), -S ascending, t ascending
        order = np.lexsort((tok, -S[:, e], ~tc_member[:, e]))
        member[order[: f_tr[e]], e] = True
    round_dir = np.sign(f_tr - f).astype(np.int32)
    return member, f_tr.astype(np.int32), round_dir


def route(X, Wr, K, bias=None, dtype=np.float32, S=None):
    """TC routing of a batch: logits -> S_full -> top-K -> metadata.

    If ``S`` is given it is used as the fp32 score matrix (the routing contract
    is defined on S_full, so parity of the integer results is checked given the
    same scores).
    """
    if S is None:
        S = softmax_scores(router_logits(X, Wr, bias, dtype))
    idx = topk_select(S, K)
    member = tc_membership(idx, S.shape[1])
    return S, idx, routing_from_membership(member, S, dtype)
