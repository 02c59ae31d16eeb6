"""Seeded synthetic inputs for the slice -> token mix -> deslice path.

This module only draws random numbers and rounds them to the storage dtype. It holds none of
the method's arithmetic, so both the fp64 oracle (test side) and the HIP path (product side)
can consume what it produces without sharing any code with each other.

Every tensor comes from its own sub-stream ``numpy.random.default_rng([SEED, cfg_id, k])``
so that adding a tensor never shifts another one. Values are drawn in fp32 and, for bf16
storage, rounded to the nearest bf16 (ties to even) and kept as exactly representable fp32.

Workloads (shapes and value distributions of the paper's 3D-flow layers; the temperature and
W_s choices open in the text are the ``tau_mode`` / ``ws_mode`` fields below):

=========  ======  =====  =========  ==  ==  ====  =====================================
name       dtype   B      N          H   D   G     mix / special structure
=========  ======  =====  =========  ==  ==  ====  =====================================
tiny       f32     1      4096       8   16  32    fixed G x G matrix A ~ N(0, 1/G)
surface    f32     1      32768      8   32  32    single-head G x G token self-attention
volume     bf16    1      1048576    8   32  64    fixed G x G matrix
stressG    bf16    1      262144     8   32  G     per-head tau ~ U[0.3, 1.0]; W_s with
                                                   pre-temperature logit std 3; G in
                                                   {128, 256, 512, 1024}
stack      f32     4      131072     8   32  64    fixed G x G matrix (one layer's path)
infer      bf16    1      2^24       8   32  64    fixed G x G matrix; forward only; the
                                                   points are 16 copies of one seeded
                                                   2^20-point block
surface_   f32     1      32768      8   32  32    as surface, untied: the deslice has its
untied                                             own projection, bias and temperature
volume_    bf16    1      2^20       8   32  64    LinearNO: untied, slice weights
linearno                                           softmaxed over the points, per-token
                                                   channel map
attn1024   bf16    1      2^18       8   32  1024  single-head token self-attention over
                                                   1024 tokens; as stress1024 otherwise
=========  ======  =====  =========  ==  ==  ====  =====================================

A workload with ``block_N`` set draws only ``block_N`` points; the full point set is that block
repeated ``N / block_N`` times along N (done by whoever uploads it). The sums over points are
then exactly ``N / block_N`` times the block's sums, which lets the oracle check the full size
from the block alone.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional

import numpy as np

SEED = 20261202

MIX_IDENTITY, MIX_LINEAR_G, MIX_LINEAR_C, MIX_ATTN = 0, 1, 2, 3

# sub-stream ids, one per tensor
_K_X, _K_F, _K_WS, _K_B, _K_TAU, _K_A, _K_WC, _K_WQ, _K_WK, _K_WV, _K_DO = range(11)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int
    dtype: str            # "f32" or "bf16": storage of x, fx, out, dout, dx, dfx
    B: int
    N: int
    H: int
    D: int
    V: int
    G: int
    mix: int
    eps: float = 1e-5
    tau_mode: str = "const"     # "const" (tau = 0.5 for every head) or "uniform" (U[0.3, 1])
    ws_mode: str = "xavier"     # "xavier" or "std3" (pre-temperature logit std 3)
    ws_per_head: bool = False
    a_per_head: bool = False
    block_N: int = 0            # > 0: draw this many points, repeated N / block_N times
    forward_only: bool = False  # inference: no backward, no saved lse
    variant: str = "tied"       # "tied", "untied" or "linearno"

    @property
    def repeat(self) -> int:
        return self.N // self.block_N if self.block_N else 1

    def scaled(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    @property
    def points(self) -> int:
        return self.B * self.N


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", 0, "f32", 1, 4096, 8, 16, 16, 32, MIX_LINEAR_G),
    "surface": Workload("surface", 1, "f32", 1, 32768, 8, 32, 32, 32, MIX_ATTN),
    "volume": Workload("volume", 2, "bf16", 1, 1 << 20, 8, 32, 32, 64, MIX_LINEAR_G),
    "stack": Workload("stack", 4, "f32", 4, 1 << 17, 8, 32, 32, 64, MIX_LINEAR_G),
}
WORKLOADS["infer"] = Workload("infer", 5, "bf16", 1, 1 << 24, 8, 32, 32, 64, MIX_LINEAR_G,
                             block_N=1 << 20, forward_only=True)
WORKLOADS["surface_untied"] = Workload("surface_untied", 6, "f32", 1, 32768, 8, 32, 32, 32,
                                      MIX_ATTN, variant="untied")
WORKLOADS["volume_linearno"] = Workload("volume_linearno", 7, "bf16", 1, 1 << 20, 8, 32, 32, 64,
                                       MIX_LINEAR_C, variant="linearno")
WORKLOADS["attn1024"] = Workload("attn1024", 8, "bf16", 1, 1 << 18, 8, 32, 32, 1024, MIX_ATTN,
                                 tau_mode="uniform", ws_mode="std3")
for _g in (128, 256, 512, 1024):
    WORKLOADS[f"stress{_g}"] = Workload(f"stress{_g}", 3, "bf16", 1, 1 << 18, 8, 32, 32, _g,
                                        MIX_LINEAR_G, tau_mode="uniform", ws_mode="std3")


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Nearest bf16 value of each fp32 entry (ties to even), returned as fp32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32)
    # bits + 0x7FFF + lsb stays below 2^32 for every non-NaN value (largest: -inf, 0xFF800000)
    rounded = (bits >> 16) & np.uint32(1)
    rounded += bits
    rounded += np.uint32(0x7FFF)
    rounded &= np.uint32(0xFFFF0000)
    out = rounded.view(np.float32)
    nan = np.isnan(a)
    if nan.any():
        out = out.copy()
        out[nan] = np.float32("nan")
    return out


def _rng(w: Workload, k: int) -> np.random.Generator:
    return np.random.default_rng([SEED, w.cfg_id, k, w.G])


def _store(w: Workload, a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    return round_to_bf16(a) if w.dtype == "bf16" else a


def _normal(rng, shape, std=1.0) -> np.ndarray:
    out = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        out *= np.float32(std)
    return out


def _xavier(rng, shape, fan_in, fan_out) -> np.ndarray:
    lim = math.sqrt(6.0 / (fan_in + fan_out))
    return rng.uniform(-lim, lim, size=shape).astype(np.float32)


def make_inputs(w: Workload, with_grad: bool = True) -> Dict[str, Optional[np.ndarray]]:
    """All inputs of one forward + backward as fp32 numpy arrays (exact stored values).

    Keys: x (B,N,H,D), fx (B,N,H,V) (N = block_N when set), Ws (D,G) or (H,D,G), b (G) or (H,G), tau (H),
    A (G,G) or (H,G,G) for the fixed token matrix, Wc (V,V), Wq/Wk/Wv (V,V), scale, dout.
    """
    B, N, H, D, V, G = w.B, w.N, w.H, w.D, w.V, w.G
    if w.block_N:
        if N % w.block_N:
            raise ValueError("N must be a multiple of block_N")
        N = w.block_N
    x = _store(w, _normal(_rng(w, _K_X), (B, N, H, D)))
    fx = _store(w, _normal(_rng(w, _K_F), (B, N, H, V)))
    ws_shape = (H, D, G) if w.ws_per_head else (D, G)
    if w.ws_mode == "xavier":
        Ws = _xavier(_rng(w, _K_WS), ws_shape, D, G)
    else:  # pre-temperature logit std 3 for unit-variance x: W_s ~ N(0, 9/D)
        Ws = _normal(_rng(w, _K_WS), ws_shape, 3.0 / math.sqrt(D))
    b = np.zeros((H, G) if w.ws_per_head else (G,), dtype=np.float32)
    if w.tau_mode == "const":
        tau = np.full((H,), 0.5, dtype=np.float32)
    else:
        tau = _rng(w, _K_TAU).uniform(0.3, 1.0, size=(H,)).astype(np.float32)
    out = dict(x=x, fx=fx, Ws=Ws, b=b, tau=tau, A=None, Wc=None, Wq=None, Wk=None, Wv=None,
               scale=np.float32(1.0 / math.sqrt(V)), dout=None)
    if w.mix == MIX_LINEAR_G:
        out["A"] = _normal(_rng(w, _K_A), (H, G, G) if w.a_per_head else (G, G),
                           1.0 / math.sqrt(G))
    elif w.mix == MIX_LINEAR_C:
        out["Wc"] = _xavier(_rng(w, _K_WC), (V, V), V, V)
    elif w.mix == MIX_ATTN:
        out["Wq"] = _xavier(_rng(w, _K_WQ), (V, V), V, V)
        out["Wk"] = _xavier(_rng(w, _K_WK), (V, V), V, V)
        out["Wv"] = _xavier(_rng(w, _K_WV), (V, V), V, V)
    if with_grad:
        out["dout"] = _store(w, _normal(_rng(w, _K_DO), (B, N, H, V)))
    return out


_K_WD, _K_BD, _K_TAUD = 20, 21, 22


def untied_params(w: Workload) -> Dict[str, np.ndarray]:
    """The deslice's own projection, bias and temperature for the untied variant: W_d drawn
    like W_s (own sub-stream), b_d ~ N(0, 0.1^2), tau_d ~ U[0.4, 1.0] per head."""
    D, G, H = w.D, w.G, w.H
    ws_shape = (H, D, G) if w.ws_per_head else (D, G)
    if w.ws_mode == "xavier":
        Wd = _xavier(_rng(w, _K_WD), ws_shape, D, G)
    else:
        Wd = _normal(_rng(w, _K_WD), ws_shape, 3.0 / math.sqrt(D))
    bd = _normal(_rng(w, _K_BD), (H, G) if w.ws_per_head else (G,), 0.1)
    taud = _rng(w, _K_TAUD).uniform(0.4, 1.0, size=(H,)).astype(np.float32)
    return dict(Wd=Wd, bd=bd, taud=taud)


def random_like(w: Workload, seed_k: int, shape, std=1.0) -> np.ndarray:
    """Extra seeded N(0, std^2) tensor (for tests that need more random data)."""
    rng = np.random.default_rng([SEED, w.cfg_id, 1000 + seed_k, w.G])
    return _normal(rng, shape, std)


# The full 8-layer slicing stack (each layer: LayerNorm -> projections -> slice, constant
# G x G mix, deslice -> output projection -> residual -> GELU MLP at width 4C -> residual),
# fp32, trained with the loss sum(out * R): the input features h and R, each (B, N, C), drawn
# i.i.d. N(0, 1); the layer weights come from torch's seeded initialisation.
STACKS = {"stack8": dict(L=8, B=4, N=1 << 17, C=256, H=8, G=64, cfg_id=9)}


def make_stack_inputs(name: str, B: Optional[int] = None, N: Optional[int] = None):
    """(h, R) of a stack workload as fp32 numpy arrays (B, N, C); B and N may be cut down
    (the leading samples and points of the full draw are not reproduced: a cut is a draw of
    its own, from the same streams)."""
    spec = STACKS[name]
    B = spec["B"] if B is None else B
    N = spec["N"] if N is None else N
    C = spec["C"]
    h = np.random.default_rng([SEED, spec["cfg_id"], 1, C]).standard_normal((B, N, C), dtype=np.float32)
    R = np.random.default_rng([SEED, spec["cfg_id"], 2, C]).standard_normal((B, N, C), dtype=np.float32)
    return h, R
