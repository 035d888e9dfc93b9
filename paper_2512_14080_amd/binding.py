"""ctypes binding of libsonicmoe.so (include/sonicmoe.h).

Argument marshalling only: every step of the layer runs in the library's HIP
kernels.  torch supplies device memory (tensor data pointers) and the stream.
Loading fails loudly if the built library is missing.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsonicmoe.so")

MOE_OK = 0
MOE_ERR_INVALID_ARG = -1
MOE_ERR_UNSUPPORTED = -2
MOE_ERR_CAPACITY = -3
MOE_ERR_WORKSPACE = -4
MOE_ERR_HIP = -5

MOE_ROUTING_LOGITS = 1
MOE_ROUTING_SCORES_T = 2

MOE_ROUTE_SCORES_IN = 1
MOE_ROUTE_WRITE_LOGITS = 2
MOE_ROUTE_WRITE_SCORES_T = 4
MOE_ROUTE_COUNTS_ONLY = 8
MOE_ROUTE_SEPARATE_TOPK = 16

MOE_ROUTING_STATE_EMPTY = 0
MOE_ROUTING_STATE_COUNTS = 1
MOE_ROUTING_STATE_BUILT = 2

MOE_STATUS_DUPLICATE_EXPERT = 1

ROUND_MODES = {"nearest": 0, "up": 1, "down": 2, "balance": 3, "stochastic": 4}

MOE_WS_FWD = 1
MOE_WS_BWD = 2
MOE_WS_FWD_AGG_ABLATION = 3

AGG_STRATEGIES = {"gather_sum": 0, "scatter_sum": 1, "atomic_f32": 2}

KERNEL_CLASSES = ["router_gemm", "topk", "routing_meta", "token_round", "up_proj", "down_proj", "aggregate_O",
                  "dH", "dW2", "dXtilde", "dW1", "aggregate_dX", "dWr", "router_topk"]

EXPORTS = ["moe_routing_bytes", "moe_routing_init", "moe_round_capacity", "moe_route", "moe_round_tokens",
           "moe_workspace_bytes", "moe_fwd", "moe_bwd", "moe_strerror", "moe_last_error", "moe_prof_select",
           "moe_prof_read", "moe_kernel_class_name", "moe_fwd_aggregation_ablation", "moe_fwd_static",
           "moe_fwd_static_max_bytes"]


class MoeDims(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("d", ctypes.c_int32), ("n", ctypes.c_int32),
                ("E", ctypes.c_int32), ("K", ctypes.c_int32)]


_P = ctypes.c_void_p


class MoeRouting(ctypes.Structure):
    _fields_ = [("capacity", ctypes.c_int32), ("words", ctypes.c_int32),
                ("state", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("logits", _P), ("scores", _P), ("scores_t", _P), ("topk_idx", _P), ("topk_w", _P),
                ("mask", _P), ("mask_prefix", _P), ("counts", _P), ("offsets", _P), ("row_token", _P),
                ("row_expert", _P), ("row_w", _P), ("tok_offsets", _P), ("tok_rows", _P), ("tok_count", _P),
                ("tok_denom", _P), ("round_dir", _P), ("scratch", _P), ("status", _P)]

    @classmethod
    def pointer_fields(cls):
        return [name for name, typ in cls._fields_ if typ is _P]


class MoeExpertBias(ctypes.Structure):
    _fields_ = [("b1", _P), ("b2", _P), ("db1", _P), ("db2", _P)]


class MoEError(RuntimeError):
    def __init__(self, fn, code, detail):
        super().__init__(f"{fn} failed with {code}: {detail}")
        self.code = code


_lib = None


def lib():
    """Load libsonicmoe.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with paper_2512_14080_amd.build.build()")
    L = ctypes.CDLL(LIB_PATH)
    sz, i32, vp = ctypes.c_size_t, ctypes.c_int32, ctypes.c_void_p
    D, R, EB = MoeDims, ctypes.POINTER(MoeRouting), ctypes.POINTER(MoeExpertBias)
    sig = {
        "moe_routing_bytes": (sz, [D, i32, ctypes.c_int]),
        "moe_routing_init": (ctypes.c_int, [D, i32, ctypes.c_int, vp, sz, R]),
        "moe_round_capacity": (i32, [D, i32]),
        "moe_route": (ctypes.c_int, [D, vp, vp, vp, ctypes.c_int, R, vp]),
        "moe_round_tokens": (ctypes.c_int, [D, i32, ctypes.c_int, vp, R, R, vp]),
        "moe_workspace_bytes": (sz, [D, i32, ctypes.c_int]),
        "moe_fwd": (ctypes.c_int, [D, vp, vp, vp, EB, R, vp, vp, vp, sz, vp]),
        "moe_bwd": (ctypes.c_int, [D, vp, vp, vp, vp, vp, EB, vp, R, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "moe_fwd_aggregation_ablation": (ctypes.c_int, [D, vp, vp, vp, R, vp, vp, ctypes.c_int, vp, sz, vp]),
        "moe_fwd_static": (ctypes.c_int, [D, vp, vp, vp, EB, R, vp, vp, vp]),
        "moe_fwd_static_max_bytes": (sz, []),
        "moe_strerror": (ctypes.c_char_p, [ctypes.c_int]),
        "moe_last_error": (ctypes.c_char_p, []),
        "moe_prof_select": (ctypes.c_int, [ctypes.c_int]),
        "moe_prof_read": (ctypes.c_int, [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i32)]),
        "moe_kernel_class_name": (ctypes.c_char_p, [ctypes.c_int]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def _check(fn, rc):
    if rc != MOE_OK:
        raise MoEError(fn, rc, lib().moe_last_error().decode())
    return rc


def dims(T, d, n, E, K) -> MoeDims:
    return MoeDims(T, d, n, E, K)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


# ------------------------------------------------------------------ entry points
def moe_routing_bytes(D, capacity, flags=0) -> int:
    return lib().moe_routing_bytes(D, capacity, flags)


def moe_round_capacity(D, m_tile) -> int:
    return lib().moe_round_capacity(D, m_tile)


def moe_workspace_bytes(D, capacity, which) -> int:
    return lib().moe_workspace_bytes(D, capacity, which)


def moe_strerror(code) -> str:
    return lib().moe_strerror(code).decode()


def moe_last_error() -> str:
    return lib().moe_last_error().decode()


class Routing:
    """A device routing buffer plus its moe_routing struct and typed views."""

    def __init__(self, D: MoeDims, capacity: int, flags: int = 0, device="cuda"):
        import torch
        self.D = D
        nbytes = moe_routing_bytes(D, capacity, flags)
        if nbytes == 0:
            _check("moe_routing_bytes", MOE_ERR_INVALID_ARG)
        self.buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        base = self.buf.data_ptr()
        self.off = (-base) % 256
        self.struct = MoeRouting()
        _check("moe_routing_init", lib().moe_routing_init(D, capacity, flags, ctypes.c_void_p(base + self.off),
                                                          nbytes, ctypes.byref(self.struct)))

    @property
    def capacity(self):
        return self.struct.capacity

    def view(self, field: str, dtype, shape):
        import torch
        ptr = getattr(self.struct, field)
        if not ptr:
            return None
        n = 1
        for s in shape:
            n *= s
        esize = torch.empty(0, dtype=dtype).element_size()
        start = ptr - self.buf.data_ptr()
        return self.buf[start:start + n * esize].view(dtype).view(*shape)

    # typed views of every array
    def arrays(self):
        import torch
        D = self.D
        T, E, K, W, cap = D.T, D.E, D.K, self.struct.words, self.capacity
        f32, i32 = torch.float32, torch.int32
        return {
            "logits": self.view("logits", f32, (T, E)), "scores": self.view("scores", f32, (T, E)),
            "scores_t": self.view("scores_t", f32, (E, T)), "topk_idx": self.view("topk_idx", i32, (T, K)),
            "topk_w": self.view("topk_w", f32, (T, K)), "mask": self.view("mask", torch.int64, (E, W)),
            "counts": self.view("counts", i32, (E,)), "offsets": self.view("offsets", i32, (E + 1,)),
            "row_token": self.view("row_token", i32, (cap,)), "row_expert": self.view("row_expert", i32, (cap,)),
            "row_w": self.view("row_w", f32, (cap,)), "tok_offsets": self.view("tok_offsets", i32, (T + 1,)),
            "tok_rows": self.view("tok_rows", i32, (cap,)), "round_dir": self.view("round_dir", i32, (E,)),
            "tok_count": self.view("tok_count", i32, (T,)), "status": self.view("status", i32, (1,)),
        }


def moe_route(D, X, Wr, bias, flags, r: Routing, stream=None):
    _check("moe_route", lib().moe_route(D, _ptr(X), _ptr(Wr), _ptr(bias), flags, ctypes.byref(r.struct),
                                        _stream(stream)))


def moe_round_tokens(D, m_tile, mode, u, tc: Routing, tr: Routing, stream=None):
    if isinstance(mode, str):
        mode = ROUND_MODES[mode]
    _check("moe_round_tokens", lib().moe_round_tokens(D, m_tile, mode, _ptr(u), ctypes.byref(tc.struct),
                                                      ctypes.byref(tr.struct), _stream(stream)))


def expert_bias(b1=None, b2=None, db1=None, db2=None):
    """A moe_expert_bias struct from device tensors (or None), or None if all are None."""
    if b1 is None and b2 is None and db1 is None and db2 is None:
        return None
    return MoeExpertBias(*(None if t is None else t.data_ptr() for t in (b1, b2, db1, db2)))


def _eb(eb):
    return None if eb is None else ctypes.byref(eb)


def moe_fwd(D, X, W1, W2, r: Routing, H, O, ws, stream=None, eb=None):
    _check("moe_fwd", lib().moe_fwd(D, _ptr(X), _ptr(W1), _ptr(W2), _eb(eb), ctypes.byref(r.struct), _ptr(H),
                                    _ptr(O), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def moe_bwd(D, dO, X, H, W1, W2, Wr, r: Routing, dX, dW1, dW2, dWr, dbias, dS, ws, stream=None, eb=None):
    _check("moe_bwd", lib().moe_bwd(D, _ptr(dO), _ptr(X), _ptr(H), _ptr(W1), _ptr(W2), _eb(eb), _ptr(Wr),
                                    ctypes.byref(r.struct), _ptr(dX), _ptr(dW1), _ptr(dW2), _ptr(dWr), _ptr(dbias),
                                    _ptr(dS), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))
def moe_fwd_static(D, X, W1, W2, r: Routing, H, O, stream=None, eb=None):
    _check("moe_fwd_static", lib().moe_fwd_static(D, _ptr(X), _ptr(W1), _ptr(W2), _eb(eb), ctypes.byref(r.struct),
                                                  _ptr(H), _ptr(O), _stream(stream)))


def moe_fwd_aggregation_ablation(D, X, W1, W2, r: Routing, H, O, strategy, ws, stream=None):
    if isinstance(strategy, str):
        strategy = AGG_STRATEGIES[strategy]
    _check("moe_fwd_aggregation_ablation",
           lib().moe_fwd_aggregation_ablation(D, _ptr(X), _ptr(W1), _ptr(W2), ctypes.byref(r.struct), _ptr(H),
                                              _ptr(O), strategy, _ptr(ws), ws.numel() * ws.element_size(),
                                              _stream(stream)))


def moe_prof_select(kernel_class):
    if isinstance(kernel_class, str):
        kernel_class = KERNEL_CLASSES.index(kernel_class)
    _check("moe_prof_select", lib().moe_prof_select(kernel_class))


def moe_prof_read():
    ms = ctypes.c_double()
    n = ctypes.c_int32()
    _check("moe_prof_read", lib().moe_prof_read(ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value
