"""Independent dense reference used to pin the oracle (CPU, torch fp64 autograd).

Every expert is applied to every token and the outputs are masked by the routing
matrix and weighted by the renormalised softmax scores; gradients come from
torch autograd, not from any hand-derived backward.  It shares no code with the
oracle (it does not import it) or with the HIP path.
"""
from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as F


def dense_moe(X, Wr, W1, W2, member, dO, bias=None, b1=None, b2=None):
    """Return dict of numpy fp64 arrays: O, dX, dWr, dW1, dW2, dbias, dS[T,E], w[T,E]
    (and db1 [E,2n], db2 [E,d] when the expert biases b1, b2 are given)."""
    f64 = torch.float64
    X = torch.tensor(np.asarray(X, np.float64), dtype=f64, requires_grad=True)
    Wr = torch.tensor(np.asarray(Wr, np.float64), dtype=f64, requires_grad=True)
    W1 = torch.tensor(np.asarray(W1, np.float64), dtype=f64, requires_grad=True)
    W2 = torch.tensor(np.asarray(W2, np.float64), dtype=f64, requires_grad=True)
    b = torch.zeros(Wr.shape[1], dtype=f64) if bias is None else torch.tensor(np.asarray(bias, np.float64))
    b.requires_grad_(True)
    B1 = None if b1 is None else torch.tensor(np.asarray(b1, np.float64), dtype=f64, requires_grad=True)
    B2 = None if b2 is None else torch.tensor(np.asarray(b2, np.float64), dtype=f64, requires_grad=True)
    m = torch.tensor(np.asarray(member, np.float64))
    dOt = torch.tensor(np.asarray(dO, np.float64))
    logits = X @ Wr + b
    S = torch.softmax(logits, dim=1)
    Sm = S * m
    den = Sm.sum(dim=1, keepdim=True)
    w = torch.where(den > 0, Sm / torch.where(den > 0, den, torch.ones_like(den)), torch.zeros_like(Sm))
    w.retain_grad()
    E = W1.shape[0]
    n = W1.shape[2] // 2
    O = torch.zeros(X.shape[0], W2.shape[2], dtype=f64)
    for e in range(E):
        h = X @ W1[e]
        if B1 is not None:
            h = h + B1[e]
        a = F.silu(h[:, :n]) * h[:, n:]
        y = a @ W2[e]
        if B2 is not None:
            y = y + B2[e]
        O = O + w[:, e:e + 1] * y
    (O * dOt).sum().backward()
    out = {
        "O": O.detach().numpy(), "dX": X.grad.numpy(), "dWr": Wr.grad.numpy(),
        "dW1": W1.grad.numpy(), "dW2": W2.grad.numpy(), "dbias": b.grad.numpy(),
        "dS": w.grad.numpy(), "w": w.detach().numpy(),
    }
    if B1 is not None:
        out["db1"] = B1.grad.numpy()
    if B2 is not None:
        out["db2"] = B2.grad.numpy()
    return out


def dense_ffn(X, W1e, W2e):
    """A single SwiGLU FFN, silu(x W_gate) * (x W_up) W2, via torch ops (fp64)."""
    X = torch.tensor(np.asarray(X, np.float64))
    W1e = torch.tensor(np.asarray(W1e, np.float64))
    W2e = torch.tensor(np.asarray(W2e, np.float64))
    n = W1e.shape[1] // 2
    return (F.silu(X @ W1e[:, :n]) * (X @ W1e[:, n:]) @ W2e).numpy()


def rel_err(a, ref):
    """max |a - ref| / max |ref| over the tensor (the parity metric)."""
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.abs(ref).max()
    num = np.abs(a - ref).max()
    if den == 0:
        return float(num)
    return float(num / den)


def rel_fro(a, ref):
    """||a - ref||_F / ||ref||_F over the tensor (reported next to rel_err)."""
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref.ravel())
    num = np.linalg.norm((a - ref).ravel())
    if den == 0:
        return float(num)
    return float(num / den)
