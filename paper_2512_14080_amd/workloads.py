"""Seeded synthetic MoE-layer workloads.

This module holds the layer shapes that are exercised and the seeded input
generator that both the HIP path's tests/benchmark and the CPU oracle consume.
It contains none of the method's arithmetic: only random draws, the fp32 -> bf16
round-to-nearest-even conversion used to materialise bf16 inputs, and the
per-expert router bias that skews expert popularity.

Shapes follow the paper's problem statement (Appendix A, notation table):
X[T,d], router W_r[d,E], expert up-projection W1[E,d,2n] (gate columns first,
then up columns), down-projection W2[E,n,d], top-K routing.
"""
from __future__ import annotations

import dataclasses
import concurrent.futures
import os

import numpy as np


@dataclasses.dataclass(frozen=True)
class MoEConfig:
    name: str
    T: int
    d: int
    n: int
    E: int
    K: int
    m_tile: int
    # std of X, W1, W2 draws
    w_std: float = 0.02
    # "std1": router weights scaled so logits are ~N(0,1); "w_std": same std as weights
    router: str = "std1"
    # Zipf exponent of the per-expert bias (0 = no bias)
    zipf_s: float = 0.0

    @property
    def P(self) -> int:
        return self.T * self.K

    def model_flops(self, rows: int | None = None) -> float:
        """Model FLOPs of fwd+bwd: 18 * d * n * (sum of expert row counts)."""
        r = self.T * self.K if rows is None else rows
        return 18.0 * self.d * self.n * r


CONFIGS = {
    # Tiny correctness layer: everything ~N(0, 0.02), softmax top-2 router.
    "tiny": MoEConfig("tiny", T=512, d=128, n=64, E=8, K=2, m_tile=16, router="w_std"),
    # Fine-grained 1B-shaped layer, roughly balanced std-1 router logits.
    "1b": MoEConfig("1b", T=16384, d=1024, n=256, E=64, K=8, m_tile=128),
    # Fine-grained 7B-shaped layer (the headline workload).
    "7b": MoEConfig("7b", T=32768, d=1536, n=256, E=128, K=8, m_tile=128),
    # High-sparsity layer with a Zipf(1.1) per-expert bias on the logits.
    "sparse": MoEConfig("sparse", T=32768, d=2048, n=128, E=256, K=8, m_tile=128, zipf_s=1.1),
    # Coarse-grained layer (large GEMMs).
    "coarse": MoEConfig("coarse", T=16384, d=4096, n=14336, E=8, K=2, m_tile=128),
}

# The paper's benchmark layers (Appendix H, the H100 table): four model sizes,
# each at three granularities with equal FLOPs (n * K fixed).
PAPER_SHAPES = [
    ("1.4b", 40960, 768, [(256, 128, 8), (512, 64, 4), (1024, 32, 2)]),
    ("7b", 24576, 1536, [(256, 128, 8), (512, 64, 4), (1024, 32, 2)]),
    ("30b", 32768, 4096, [(256, 256, 16), (512, 128, 8), (1024, 64, 4)]),
    ("120b", 32768, 4096, [(512, 256, 16), (1024, 128, 8), (2048, 64, 4)]),
]
for _size, _T, _d, _rows in PAPER_SHAPES:
    for _n, _E, _K in _rows:
        _name = f"paper-{_size}-e{_E}k{_K}"
        CONFIGS[_name] = MoEConfig(_name, T=_T, d=_d, n=_n, E=_E, K=_K, m_tile=128)
# The paper's token-rounding speed sweeps (Appendix H): four (T, d, n, K)
# families, each over a range of E, with M_tile = 128.
TR_SWEEPS = [
    (16384, 1536, 256, 8, [64, 128, 256, 512]),
    (16384, 1536, 1024, 2, [16, 32, 64, 128]),
    (16384, 4096, 512, 8, [64, 128, 256, 512]),
    (16384, 4096, 1024, 4, [32, 64, 128, 256]),
]
for _T, _d, _n, _K, _Es in TR_SWEEPS:
    for _E in _Es:
        _name = f"tr-d{_d}n{_n}k{_K}-e{_E}"
        CONFIGS[_name] = MoEConfig(_name, T=_T, d=_d, n=_n, E=_E, K=_K, m_tile=128)
SWEEPS = {"paper": [k for k in CONFIGS if k.startswith("paper-")],
          "tr": [k for k in CONFIGS if k.startswith("tr-")]}


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round finite fp32 values to bf16 (round-to-nearest-even) and return raw
    uint16 bits.  The uint32 sum cannot wrap for finite inputs (largest bit
    pattern 0xFF7FFFFF + 0x8000 < 2^32)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32)
    r = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def f32_from_bf16_bits(u: np.ndarray) -> np.ndarray:
    """Exact upcast of raw bf16 bits to fp32."""
    return (np.ascontiguousarray(u, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass
class MoEInputs:
    cfg: MoEConfig
    seed: int
    # raw bf16 bits (uint16) -- what the device consumes
    X: np.ndarray
    Wr: np.ndarray
    W1: np.ndarray
    W2: np.ndarray
    dO: np.ndarray
    # fp32 per-expert logit bias, or None
    bias: np.ndarray | None

    def f32(self, name: str) -> np.ndarray:
        return f32_from_bf16_bits(getattr(self, name))


_ROW_BLOCK = 2048  # rows (tokens) or experts per independent normal stream


def _normal_blocks(ss: np.random.SeedSequence, shape, scale: float, block: int) -> np.ndarray:
    """Standard normals * scale, rounded to bf16 bits, drawn block by block along
    axis 0: block i of ``block`` leading indices uses its own Philox stream
    seeded by the child SeedSequence (entropy of ``ss``, spawn key + (i,)).
    Blocks are filled on a thread pool; the values do not depend on it, and a
    prefix along axis 0 reproduces the first blocks exactly."""
    out = np.empty(shape, np.uint16)
    nb = (shape[0] + block - 1) // block

    def fill(i):
        child = np.random.SeedSequence(ss.entropy, spawn_key=tuple(ss.spawn_key) + (i,))
        g = np.random.Generator(np.random.Philox(child))
        lo, hi = i * block, min(shape[0], (i + 1) * block)
        x = g.standard_normal((hi - lo,) + tuple(shape[1:]), dtype=np.float32)
        x *= np.float32(scale)
        out[lo:hi] = bf16_bits_from_f32(x)

    workers = max(1, min(16, os.cpu_count() or 1, nb))
    if workers == 1:
        for i in range(nb):
            fill(i)
    else:
        with concurrent.futures.ThreadPoolExecutor(workers) as ex:
            list(ex.map(fill, range(nb)))
    return out


def make_inputs(cfg: MoEConfig, seed: int = 0, T: int | None = None) -> MoEInputs:
    """Draw the layer's inputs from a fixed seed.

    Streams are spawned from one SeedSequence in the fixed order
    [X, W_r, W1, W2, dO, bias-permutation]; X and dO are drawn in blocks of
    2048 tokens and W1/W2 in blocks of 2048 experts' leading index (one child
    stream per block, see _normal_blocks).  Draws are fp32, then rounded to
    bf16.  ``T`` overrides the token count (the first T rows of X and dO are
    the same as for the full config, so a sample is a prefix).
    """
    T = cfg.T if T is None else T
    ss = np.random.SeedSequence(seed)
    sx, sr, s1, s2, sd, sb = ss.spawn(6)
    d, n, E = cfg.d, cfg.n, cfg.E
    r_std = cfg.w_std if cfg.router == "w_std" else 1.0 / (cfg.w_std * np.sqrt(d))
    X = _normal_blocks(sx, (T, d), cfg.w_std, _ROW_BLOCK)
    Wr = _normal_blocks(sr, (d, E), r_std, d)
    W1 = _normal_blocks(s1, (E, d, 2 * n), cfg.w_std, 1)
    W2 = _normal_blocks(s2, (E, n, d), cfg.w_std, 1)
    dO = _normal_blocks(sd, (T, d), 1.0, _ROW_BLOCK)
    bias = None
    if cfg.zipf_s > 0:
        gb = np.random.Generator(np.random.Philox(sb))
        rank = gb.permutation(E) + 1  # expert e gets popularity rank rank[e]
        bias = (-cfg.zipf_s * np.log(rank.astype(np.float64))).astype(np.float32)
    return MoEInputs(cfg, seed, X, Wr, W1, W2, dO, bias)


def scaled(cfg: MoEConfig, **kw) -> MoEConfig:
    """A copy of ``cfg`` with some fields replaced (for reduced parity shapes)."""
    return dataclasses.replace(cfg, **kw)
