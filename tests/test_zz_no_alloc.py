"""The forward entry point that allocates nothing (moe_fwd_static: its
workspace is the library's static device array) against moe_fwd with a
caller workspace, through the C ABI, on two calls in a row, the second with
a smaller layer.  Same kernels, so the outputs must agree bit for bit."""
import numpy as np
import pytest

from paper_2512_14080_amd import workloads as W

pytestmark = pytest.mark.gpu


def _layer(cfg, seed, mode):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import oracle
    from paper_2512_14080_amd.layer import DeviceLayer
    inp = W.make_inputs(cfg, seed)
    S = oracle.softmax_scores(oracle.router_logits(inp.f32("X"), inp.f32("Wr"), inp.bias, np.float32))
    layer = DeviceLayer(inp, round_mode=mode, scores_in=S.astype(np.float32))
    layer.route()
    return layer


def test_static_forward_matches_moe_fwd_twice():
    import torch
    from paper_2512_14080_amd import binding as B
    big = W.MoEConfig("mid", T=3000, d=512, n=256, E=16, K=4, m_tile=128)
    small = W.MoEConfig("tiny", T=512, d=128, n=64, E=8, K=2, m_tile=16, router="w_std")
    for cfg, seed, mode in ((big, 51, "nearest"), (small, 52, None)):
        layer = _layer(cfg, seed, mode)
        need = B.moe_workspace_bytes(layer.D, layer.routing.capacity, B.MOE_WS_FWD)
        assert need <= B.lib().moe_fwd_static_max_bytes()
        layer.forward()
        torch.cuda.synchronize()
        H_ref, O_ref = layer.H.clone(), layer.O.clone()
        layer.H.fill_(0)
        layer.O.fill_(0)
        B.moe_fwd_static(layer.D, layer.X, layer.W1, layer.W2, layer.routing, layer.H, layer.O)
        torch.cuda.synchronize()
        P = layer.rows()
        assert torch.equal(layer.O, O_ref), cfg.name
        assert torch.equal(layer.H[:P], H_ref[:P]), cfg.name
        print(cfg.name, "P =", P, "static forward bit-identical", flush=True)
