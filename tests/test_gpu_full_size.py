"""Parity at the full 7B layer shape (T=32768, d=1536, n=256, E=128, K=8,
token rounding with M_tile=128, nearest rounding): the sizes and kernel
launch configurations the benchmark times.  Routing is fed the oracle's fp32
scores and must match bit for bit; every output and gradient element is
compared with the fp32 oracle (max|gpu - ref| / max|ref| <= 2e-2).  The
device's own router is checked against the oracle's logits at the same size.
"""
import time

import numpy as np
import pytest

import oracle
from dense_reference import rel_err, rel_fro
from paper_2512_14080_amd import workloads as W
from test_gpu_parity import TOL, check_routing, expert_biases, oracle_routing, oracle_scores

pytestmark = pytest.mark.gpu


def _full_size(name, mode="nearest", biases=False):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2512_14080_amd.layer import DeviceLayer
    cfg = W.CONFIGS[name]
    t0 = time.time()
    inp = W.make_inputs(cfg, 0)
    L, S = oracle_scores(inp)
    b1, b2 = expert_biases(cfg, 0) if biases else (None, None)
    layer = DeviceLayer(inp, round_mode=mode, scores_in=S, b1=b1, b2=b2)
    layer.step()
    torch.cuda.synchronize()
    print(f"{name}: device step done after {time.time() - t0:.1f}s", flush=True)

    idx, rdir, R = oracle_routing(S, cfg.K, mode, cfg.m_tile)
    check_routing(layer, R, idx, rdir)
    if mode:
        assert (R.counts % cfg.m_tile == 0).all()
    print(f"{name}: routing exact (P={R.P}) after {time.time() - t0:.1f}s", flush=True)

    X, W1, W2, Wr, dO = (inp.f32(k) for k in ("X", "W1", "W2", "Wr", "dO"))
    fw = oracle.forward(X, W1, W2, R, b1=b1, b2=b2)
    P = R.P
    errs, fro = {}, {}

    def cmp(k, got, ref):
        errs[k] = rel_err(got, ref)
        fro[k] = rel_fro(got, ref)

    cmp("O", layer.O.float().cpu().numpy(), fw["O"])
    cmp("H", layer.H[:P].float().cpu().numpy(), fw["H"])
    bw = oracle.backward(dO, X, fw["H"], W1, W2, Wr, R, b2=b2)
    del fw
    if biases:
        cmp("db1", layer.db1.cpu().numpy(), bw["db1"])
        cmp("db2", layer.db2.cpu().numpy(), bw["db2"])
    cmp("dX", layer.dX.float().cpu().numpy(), bw["dX"])
    cmp("dW1", layer.dW1.float().cpu().numpy(), bw["dW1"])
    cmp("dW2", layer.dW2.float().cpu().numpy(), bw["dW2"])
    cmp("dWr", layer.dWr.cpu().numpy(), bw["dWr"])
    cmp("dS", layer.dS[:P].cpu().numpy(), bw["dS"])
    cmp("dbias", layer.dbias.cpu().numpy(), bw["dbias"])
    print(f"{name} {mode} full-size errors, max-normalised", {k: f"{v:.2e}" for k, v in errs.items()},
          "Frobenius", {k: f"{v:.2e}" for k, v in fro.items()}, f"after {time.time() - t0:.1f}s", flush=True)
    for k, v in errs.items():
        assert v <= TOL, (k, v, errs)
    return inp, L, S


def test_7b_token_rounding_full_size():
    import torch
    from paper_2512_14080_amd.layer import DeviceLayer
    inp, L, S = _full_size("7b")
    # the device router (GEMM + softmax) at full size
    dev = DeviceLayer(inp, round_mode="nearest")
    dev.route()
    torch.cuda.synchronize()
    a = {k: v.cpu().numpy() for k, v in dev.tc.arrays().items() if v is not None}
    assert rel_err(a["logits"], L) <= 1e-4
    assert rel_err(a["scores"], S) <= 1e-4


@pytest.mark.parametrize("name", ["1b", "sparse"])
def test_other_configs_full_size(name):
    """The 1B shape (T=16384, d=1024, n=256, E=64, K=8) and the high-sparsity
    shape (T=32768, d=2048, n=128, E=256, K=8, Zipf(1.1) expert popularity),
    token rounding with M_tile=128, every element against the oracle."""
    _full_size(name)


@pytest.mark.parametrize("name", ["1b", "7b"])
def test_token_choice_full_size(name):
    """Token-choice routing without rounding (ragged expert counts) at the
    full 1B and 7B shapes, every element against the oracle."""
    _full_size(name, mode=None)


def test_7b_expert_biases_full_size():
    """The 7B shape with expert biases on both projections (token rounding),
    every element, db1 and db2 included, against the oracle."""
    _full_size("7b", biases=True)


@pytest.mark.parametrize("name", ["coarse", "paper-30b-e256k16", "paper-1.4b-e32k2", "paper-7b-e128k8",
                                  "paper-120b-e64k4", "tr-d1536n256k8-e512"])
def test_sampled_large_shapes(name):
    """Shapes where the full oracle is too slow: the coarse layer (T=16384,
    d=4096, n=14336, E=8, K=2); from the paper's benchmark sweep the finest 30B
    layer (T=32768, d=4096, n=256, E=256, K=16, the wave-per-token top-K), the
    coarsest 1.4B layer (T=40960, d=768, n=1024, E=32, K=2), the 7B layer at
    its T=24576 and the coarsest 120B layer (d=4096, n=2048, E=64, K=4); and
    the E=512 point of the token-rounding sweep (T=16384, d=1536, n=256, K=8).
    All with token rounding M_tile=128.  Routing is compared exactly and
    outputs on samples the oracle computes one by one -- O and dX of sampled
    tokens, dS of their rows, H of sampled rows, and whole columns of dW1 /
    rows of dW2 of two experts."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2512_14080_amd.layer import DeviceLayer
    cfg = W.CONFIGS[name]
    t0 = time.time()
    inp = W.make_inputs(cfg, 0)
    _, S = oracle_scores(inp)
    layer = DeviceLayer(inp, round_mode="nearest", scores_in=S)
    layer.step()
    torch.cuda.synchronize()
    idx, rdir, R = oracle_routing(S, cfg.K, "nearest", cfg.m_tile)
    check_routing(layer, R, idx, rdir)
    print(f"{name}: routing exact (P={R.P}) after {time.time() - t0:.1f}s", flush=True)
    X, W1, W2, Wr, dO = (inp.f32(k) for k in ("X", "W1", "W2", "Wr", "dO"))
    rng = np.random.default_rng(3)
    toks = sorted(rng.choice(cfg.T, 8, replace=False).tolist()) + [0, cfg.T - 1]
    n = cfg.n
    O = oracle.forward_tokens(X, W1, W2, R, toks)
    dX, rows, dS, _ = oracle.backward_tokens(dO, X, W1, W2, Wr, R, toks)
    got_dS = layer.dS.cpu().numpy()
    rs = [r for rr in rows for r in rr]
    H_ref = np.stack([X[R.row_token[r]] @ W1[R.row_expert[r]] for r in rs[:6]])
    errs = {
        "O": rel_err(layer.O[toks].float().cpu().numpy(), O),
        "dX": rel_err(layer.dX[toks].float().cpu().numpy(), dX),
        "dS": rel_err(np.array([got_dS[r] for r in rs]), np.concatenate(dS)),
        "H": rel_err(layer.H[rs[:6]].float().cpu().numpy(), H_ref),
    }
    dW1 = layer.dW1.float().cpu().numpy()
    dW2 = layer.dW2.float().cpu().numpy()
    cols = sorted({0, min(4099, n // 2 + 3), n - 1})
    for e in (0, cfg.E - 1):
        c1, r2 = oracle.weight_grad_columns(dO, X, W1, W2, R, e, cols)
        errs[f"dW1[{e}]"] = rel_err(np.stack([dW1[e][:, cols], dW1[e][:, [n + j for j in cols]]], axis=1), c1)
        errs[f"dW2[{e}]"] = rel_err(dW2[e][cols, :], r2)
    print(f"{name} sampled errors", {k: f"{v:.2e}" for k, v in errs.items()}, f"after {time.time() - t0:.1f}s",
          flush=True)
    for k, v in errs.items():
        assert v <= TOL, (k, v, errs)
