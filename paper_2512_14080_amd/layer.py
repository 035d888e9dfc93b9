"""Device buffers for one MoE layer and the call sequence route -> round -> fwd -> bwd.

Allocation (torch) and argument marshalling only; the work happens in the
library's kernels through the C ABI.
"""
from __future__ import annotations

import numpy as np

from . import binding as B


def _aligned_empty(nbytes: int, device="cuda"):
    import torch
    buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    off = (-buf.data_ptr()) % 256
    return buf[off:off + nbytes]


def to_device_bf16(bits: np.ndarray, device="cuda"):
    """Raw bf16 bits (uint16 numpy) -> torch.bfloat16 device tensor with the same bits."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)
    return t.to(device)


def bf16_bits(t) -> np.ndarray:
    """torch bfloat16 tensor -> raw uint16 bits (numpy, host)."""
    import torch
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def bf16_to_f32(t) -> np.ndarray:
    return t.detach().float().cpu().numpy()


class DeviceLayer:
    """All device tensors of one layer invocation.

    ``round_mode`` None runs token-choice routing only; otherwise the layer is
    run on the token-rounded routing with tile ``m_tile``.
    """

    def __init__(self, inputs, round_mode=None, m_tile=None, scores_in=None, u=None, device="cuda",
                 router_grad=True, b1=None, b2=None, keep_logits=True):
        import torch
        cfg = inputs.cfg
        T, d, n, E, K = inputs.X.shape[0], cfg.d, cfg.n, cfg.E, cfg.K
        self.D = B.dims(T, d, n, E, K)
        self.T, self.d, self.n, self.E, self.K = T, d, n, E, K
        self.X = to_device_bf16(inputs.X, device)
        self.Wr = to_device_bf16(inputs.Wr, device)
        self.W1 = to_device_bf16(inputs.W1, device)
        self.W2 = to_device_bf16(inputs.W2, device)
        self.dO = to_device_bf16(inputs.dO, device)
        self.bias = None if inputs.bias is None else torch.from_numpy(inputs.bias).to(device)
        self.round_mode = round_mode
        self.m_tile = m_tile if m_tile is not None else cfg.m_tile
        flags = (B.MOE_ROUTING_LOGITS if keep_logits else 0) | (B.MOE_ROUTING_SCORES_T if round_mode else 0)
        self.tc = B.Routing(self.D, T * K, flags, device)
        self.tr = None
        if round_mode:
            self.tr = B.Routing(self.D, B.moe_round_capacity(self.D, self.m_tile), 0, device)
        # token rounding builds its own metadata: the token-choice routing
        # only needs its mask, counts and transposed scores
        for_round = (B.MOE_ROUTE_WRITE_SCORES_T | B.MOE_ROUTE_COUNTS_ONLY) if round_mode else 0
        self.route_flags = (B.MOE_ROUTE_WRITE_LOGITS if keep_logits else 0) | for_round
        if scores_in is not None:
            self.tc.arrays()["scores"].copy_(torch.from_numpy(np.ascontiguousarray(scores_in, np.float32)))
            self.route_flags = B.MOE_ROUTE_SCORES_IN | for_round
        self.u = None if u is None else torch.from_numpy(np.asarray(u, np.float32)).to(device)
        cap = self.routing.capacity
        self.H = torch.empty((cap, 2 * n), dtype=torch.bfloat16, device=device)
        self.O = torch.empty((T, d), dtype=torch.bfloat16, device=device)
        self.ws_f = _aligned_empty(B.moe_workspace_bytes(self.D, cap, B.MOE_WS_FWD), device)
        self.ws_b = _aligned_empty(B.moe_workspace_bytes(self.D, cap, B.MOE_WS_BWD), device)
        self.dX = torch.empty((T, d), dtype=torch.bfloat16, device=device)
        self.dW1 = torch.empty((E, d, 2 * n), dtype=torch.bfloat16, device=device)
        self.dW2 = torch.empty((E, n, d), dtype=torch.bfloat16, device=device)
        self.router_grad = router_grad
        self.dWr = torch.empty((d, E), dtype=torch.float32, device=device) if router_grad else None
        self.dbias = torch.empty((E,), dtype=torch.float32, device=device) if router_grad else None
        self.dS = torch.empty((cap,), dtype=torch.float32, device=device)
        # optional expert biases (fp32 [E,2n] and [E,d]) and their gradients
        f32 = torch.float32
        self.b1 = None if b1 is None else torch.from_numpy(np.ascontiguousarray(b1, np.float32)).to(device)
        self.b2 = None if b2 is None else torch.from_numpy(np.ascontiguousarray(b2, np.float32)).to(device)
        self.db1 = torch.empty((E, 2 * n), dtype=f32, device=device) if b1 is not None else None
        self.db2 = torch.empty((E, d), dtype=f32, device=device) if b2 is not None else None
        self.eb = B.expert_bias(self.b1, self.b2, self.db1, self.db2)

    @property
    def routing(self):
        return self.tr if self.round_mode else self.tc

    def route(self, stream=None):
        B.moe_route(self.D, self.X, self.Wr, self.bias, self.route_flags, self.tc, stream)
        if self.round_mode:
            B.moe_round_tokens(self.D, self.m_tile, self.round_mode, self.u, self.tc, self.tr, stream)

    def forward(self, stream=None):
        B.moe_fwd(self.D, self.X, self.W1, self.W2, self.routing, self.H, self.O, self.ws_f, stream, eb=self.eb)

    def backward(self, stream=None):
        B.moe_bwd(self.D, self.dO, self.X, self.H, self.W1, self.W2, self.Wr if self.router_grad else None,
                  self.routing, self.dX, self.dW1, self.dW2, self.dWr, self.dbias, self.dS, self.ws_b, stream,
                  eb=self.eb)

    def step(self, stream=None):
        self.route(stream)
        self.forward(stream)
        self.backward(stream)

    def rows(self) -> int:
        """P, the number of routed rows (reads the device offsets)."""
        return int(self.routing.arrays()["offsets"][-1].item())
