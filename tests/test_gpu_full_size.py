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
from dense_reference import rel_err
from paper_2512_14080_amd import workloads as W
from test_gpu_parity import TOL, check_routing, oracle_routing, oracle_scores

pytestmark = pytest.mark.gpu


def test_7b_token_rounding_full_size():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2512_14080_amd.layer import DeviceLayer
    cfg = W.CONFIGS["7b"]
    t0 = time.time()
    inp = W.make_inputs(cfg, 0)
    L, S = oracle_scores(inp)
    layer = DeviceLayer(inp, round_mode="nearest", scores_in=S)
    layer.step()
    torch.cuda.synchronize()
    print(f"device step done after {time.time() - t0:.1f}s", flush=True)

    idx, rdir, R = oracle_routing(S, cfg.K, "nearest", cfg.m_tile)
    check_routing(layer, R, idx, rdir)
    assert (R.counts % cfg.m_tile == 0).all()
    print(f"routing exact (P={R.P}) after {time.time() - t0:.1f}s", flush=True)

    X, W1, W2, Wr, dO = (inp.f32(k) for k in ("X", "W1", "W2", "Wr", "dO"))
    fw = oracle.forward(X, W1, W2, R)
    P = R.P
    errs = {"O": rel_err(layer.O.float().cpu().numpy(), fw["O"]),
            "H": rel_err(layer.H[:P].float().cpu().numpy(), fw["H"])}
    print(f"forward compared after {time.time() - t0:.1f}s", flush=True)
    bw = oracle.backward(dO, X, fw["H"], W1, W2, Wr, R)
    del fw
    errs.update({
        "dX": rel_err(layer.dX.float().cpu().numpy(), bw["dX"]),
        "dW1": rel_err(layer.dW1.float().cpu().numpy(), bw["dW1"]),
        "dW2": rel_err(layer.dW2.float().cpu().numpy(), bw["dW2"]),
        "dWr": rel_err(layer.dWr.cpu().numpy(), bw["dWr"]),
        "dS": rel_err(layer.dS[:P].cpu().numpy(), bw["dS"]),
        "dbias": rel_err(layer.dbias.cpu().numpy(), bw["dbias"]),
    })
    print("7b full-size errors", {k: f"{v:.2e}" for k, v in errs.items()}, f"after {time.time() - t0:.1f}s", flush=True)
    for k, v in errs.items():
        assert v <= TOL, (k, v, errs)

    # the device router (GEMM + softmax) at full size
    dev = DeviceLayer(inp, round_mode="nearest")
    dev.route()
    torch.cuda.synchronize()
    a = {k: v.cpu().numpy() for k, v in dev.tc.arrays().items() if v is not None}
    assert rel_err(a["logits"], L) <= 1e-4
    assert rel_err(a["scores"], S) <= 1e-4
