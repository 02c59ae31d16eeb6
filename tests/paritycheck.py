"""How the GPU parity tests compare a result with the fp64 oracle (imported by the tests).

Every output tensor is judged by two measures:

* normwise:     ||gpu - ref||_2 / ||ref||_2                                  <= TOL
* element-wise: max_i |gpu_i - ref_i| / max(|ref_i|, KAPPA * rms(ref))       <= ELEM_TOL

The element-wise measure is a relative error per element, with a floor at KAPPA times the
tensor's root-mean-square value for elements whose reference lies near zero (an output that
is a sum of terms of either sign carries an absolute rounding error on the scale of its
terms, not of its own value). One wrong element (a point of a bad chunk seam, a bad ragged
tail tile, a misnumbered workgroup, a corrupted store lane) then fails the comparison even
where it hardly moves the norm of a tensor with 2^28 elements.

Normwise tolerances: 1e-5 for fp32 storage and 2e-2 for bf16 storage (fp32 accumulation in
both). Element-wise: fp32 1e-5 with KAPPA 4; bf16 4e-2 with KAPPA 16. These come from the
largest element-wise errors of correct results over the parity cases: fp32 up to 5.6e-6 at
KAPPA 4 (sums of thousands of products round at ~1e-6 of the rms); bf16 up to 2.4e-2 at
KAPPA 16, on elements of peaky outputs (LinearNO's weights over the points, G = 1024 logits
with std 3 and small temperatures) whose magnitude is ten or more times the rms, with
bf16-rounded MFMA operands (unit roundoff 2^-9) and a bf16-rounded result. The bf16 gate
still rejects any element off by more than 0.64 rms or 4% of its own magnitude.

For fp32 the paper's acceptance rule (App. F.2, "Precision modes and acceptance criteria")
admits an error up to 1.25 times that of evaluating the same definition in plain fp32 (3
times where that plain-fp32 error exceeds 1e-4). That rule is applied only to the
(case, output) pairs listed in FP32_EAGER_GATED, each for a stated reason, and to the two
tests that exist to measure it (peaky logits, and the 8-layer stack); every other fp32
output is held to 1e-5.
"""
from __future__ import annotations

import sys
from typing import Callable, Dict, Iterable, Optional, Tuple

import numpy as np

TOL = {"f32": 1e-5, "bf16": 2e-2}
ELEM_TOL = {"f32": 1e-5, "bf16": 4e-2}
KAPPA = {"f32": 4.0, "bf16": 16.0}

# (case, output) pairs that take the paper's plain-fp32 acceptance rule in fp32 instead of
# the fixed 1e-5, with the reason. The deslice weights of the untied variant and LinearNO
# see the mixed tokens only through how they differ from one another; where an attention mix
# over few tokens makes them nearly equal, the fp32 rounding of the tokens alone costs more
# than 1e-5 of those gradients (plain fp32 evaluation of the same definition loses more).
FP32_EAGER_GATED = {
    ("untied/f32_D32_G32_attn", "dWd"): "deslice weights' gradient through near-equal tokens",
    ("untied/f32_D32_G32_attn", "dbd"): "deslice weights' gradient through near-equal tokens",
    ("untied/f32_D32_G32_attn", "dtaud"): "deslice weights' gradient through near-equal tokens",
    ("untied/surface_untied", "dWd"): "deslice weights' gradient through near-equal tokens",
    ("untied/surface_untied", "dbd"): "deslice weights' gradient through near-equal tokens",
    ("untied/surface_untied", "dtaud"): "deslice weights' gradient through near-equal tokens",
    ("linearno/f32_D32_G64_attn", "dWd"): "deslice weights' gradient through near-equal tokens",
    ("linearno/f32_D32_G64_attn", "dbd"): "deslice weights' gradient through near-equal tokens",
    ("linearno/f32_D32_G64_attn", "dtaud"): "deslice weights' gradient through near-equal tokens",
    ("untied/f32_D32_G1024_lin", "db"): "slice bias gradient: per-point terms that cancel over "
                                        "1024 slots (plain fp32 loses 2e-5 already at 512)",
}


def measures(got, ref, kappa: float, floor: float = 0.0) -> Tuple[float, float]:
    """(normwise, element-wise) errors of got against ref (see the module docstring).

    floor: an absolute per-element scale below which the reference does not set the
    denominator (for outputs that vanish in exact arithmetic; 0 otherwise)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if got.shape != ref.shape:
        raise AssertionError(f"shape {got.shape} != reference {ref.shape}")
    if ref.size == 0:
        return 0.0, 0.0
    if not np.isfinite(got).all():
        return float("inf"), float("inf")
    d = np.abs(got - ref)
    nr = float(np.linalg.norm(ref))
    rms = nr / np.sqrt(ref.size)
    scale = max(kappa * rms, floor)
    nd = float(np.linalg.norm(d))
    if nr == 0.0 and floor == 0.0:
        return nd, float(d.max())
    norm = nd / max(nr, floor * np.sqrt(ref.size))
    den = np.maximum(np.abs(ref), scale)
    return norm, float((d / den).max())


def announce(msg: str) -> None:
    print(f"\n[case] {msg}", flush=True)
    sys.stdout.flush()


class Checker:
    """Collects the comparisons of one test case and asserts them at the end."""

    def __init__(self, case: str, dtype: str, tol: Optional[float] = None):
        self.case = case
        self.dtype = dtype
        self.tol = TOL[dtype] if tol is None else tol
        self.etol = ELEM_TOL[dtype] if tol is None else max(tol, ELEM_TOL[dtype])
        self.kappa = KAPPA[dtype]
        self.rows: Dict[str, Tuple[float, float]] = {}
        self.refs: Dict[str, np.ndarray] = {}
        self.gots: Dict[str, np.ndarray] = {}
        self.floors: Dict[str, float] = {}

    def add(self, key: str, got, ref, floor: float = 0.0, keep: bool = True) -> None:
        self.rows[key] = measures(got, ref, self.kappa, floor)
        self.floors[key] = floor
        if keep:
            self.refs[key], self.gots[key] = ref, got

    def failures(self) -> Dict[str, Tuple[float, float]]:
        return {k: v for k, v in self.rows.items()
                if not (v[0] <= self.tol and v[1] <= self.etol)}

    def finish(self, eager: Optional[Callable[[], Dict[str, np.ndarray]]] = None) -> None:
        """Prints every measure; asserts them. eager, called only when a listed (case,
        output) pair missed 1e-5 in fp32, returns the plain-fp32 evaluation of the same
        definition, whose errors set that pair's gate (App. F.2)."""
        print("  errors (norm / elem):",
              {k: f"{a:.2e}/{b:.2e}" for k, (a, b) in self.rows.items()}, flush=True)
        bad = self.failures()
        if bad and self.dtype == "f32" and eager is not None:
            gated = [k for k in bad if (self.case, k) in FP32_EAGER_GATED]
            if gated:
                ev = eager()
                for k in gated:
                    e_norm, e_elem = measures(ev[k], self.refs[k], self.kappa, self.floors[k])
                    gn = max(self.tol, eager_gate(e_norm))
                    ge = max(self.etol, eager_gate(e_elem))
                    a, b = bad[k]
                    print(f"  {k}: plain-fp32 gate ({FP32_EAGER_GATED[(self.case, k)]}): "
                          f"norm {a:.2e} <= {gn:.2e}, elem {b:.2e} <= {ge:.2e}", flush=True)
                    if a <= gn and b <= ge:
                        del bad[k]
        assert not bad, (f"{self.case}: above {self.tol:g} normwise or {self.etol:g} "
                         f"element-wise: {bad}")


def eager_gate(e: float) -> float:
    """The paper's fp32 acceptance gate for a plain-fp32 error e (App. F.2): 1.25 e, or 3 e
    where e exceeds 1e-4."""
    return (3.0 if e > 1e-4 else 1.25) * e


# ---- the oracle over many (sample, head) pairs at once -----------------------------------------
PAIR_SUM_KEYS = ("dWs", "db", "dtau", "dA", "dWc", "dWq", "dWk", "dWv")


def _pair_inputs(inp: Dict, b: int, h: int) -> Dict:
    """The inputs of one (sample, head) pair as a problem with B = H = 1 (views and slices;
    per-head parameters cut to the head)."""
    out = dict(inp)
    for k in ("x", "fx", "dout"):
        if inp.get(k) is not None:
            out[k] = inp[k][b:b + 1, :, h:h + 1, :]
    out["tau"] = np.asarray(inp["tau"])[h:h + 1]
    Ws, bias = np.asarray(inp["Ws"]), np.asarray(inp["b"])
    out["Ws"] = Ws[h:h + 1] if Ws.ndim == 3 else Ws
    out["b"] = bias[h:h + 1] if bias.ndim == 2 else bias
    if inp.get("A") is not None and np.asarray(inp["A"]).ndim == 3:
        out["A"] = np.asarray(inp["A"])[h:h + 1]
    return out


def oracle_pairs(O, inp: Dict, kind: int, eps: float, pairs: Optional[Iterable] = None,
                 backward: bool = True):
    """The unchanged fp64 oracle (O.run_inputs) on each listed (sample, head) pair in turn, as a
    problem of its own with B = H = 1, merged into full-size results: per-pair tensors at
    their place, parameter gradients summed over the pairs in pair order (the order the
    oracle sums them in). Returns (fwd, bwd) like O.run_inputs; entries of pairs not listed
    stay zero. The pairs run one after another: concurrent BLAS calls from several threads of
    one process gave wrong products at the full sizes."""
    x = inp["x"]
    B, N, H, D = x.shape
    V = inp["fx"].shape[3]
    G = np.asarray(inp["Ws"]).shape[-1]
    pairs = [(b, h) for b in range(B) for h in range(H)] if pairs is None else list(pairs)

    def one(p):
        return O.run_inputs(_pair_inputs(inp, *p), kind, eps, backward_too=backward)

    fwd = {k: np.zeros(sh) for k, sh in dict(
        z=(B, H, G, V), s=(B, H, G), zmix=(B, H, G, V), lse=(B, H, N),
        out=(B, N, H, V)).items()}
    fwd["P"] = np.zeros((B, H, G, G)) if kind == 3 else None
    bwd = None
    if backward:
        Ws, bias = np.asarray(inp["Ws"]), np.asarray(inp["b"])
        bwd = dict(dx=np.zeros((B, N, H, D)), dfx=np.zeros((B, N, H, V)),
                   dWs=np.zeros(Ws.shape), db=np.zeros(bias.shape), dtau=np.zeros(H),
                   dzmix=np.zeros((B, H, G, V)), dz=np.zeros((B, H, G, V)))
    for b, h in pairs:
        f, g = one((b, h))
        for k in ("z", "s", "zmix", "lse"):
            fwd[k][b, h] = f[k][0, 0]
        if f.get("P") is not None:
            fwd["P"][b, h] = f["P"][0, 0]
        fwd["out"][b, :, h, :] = f["out"][0, :, 0, :]
        if g is None:
            continue
        bwd["dx"][b, :, h, :] = g["dx"][0, :, 0, :]
        bwd["dfx"][b, :, h, :] = g["dfx"][0, :, 0, :]
        bwd["dzmix"][b, h], bwd["dz"][b, h] = g["dzmix"][0, 0], g["dz"][0, 0]
        bwd["dtau"][h] += g["dtau"][0]
        if Ws.ndim == 3:            # per-head projection: the pair's head only
            bwd["dWs"][h] += g["dWs"][0]
        else:
            bwd["dWs"] += g["dWs"]
        if bias.ndim == 2:
            bwd["db"][h] += g["db"][0]
        else:
            bwd["db"] += g["db"]
        for k in ("dA", "dWc", "dWq", "dWk", "dWv"):
            if k not in g:
                continue
            if k == "dA" and np.asarray(inp["A"]).ndim == 3:
                bwd.setdefault(k, np.zeros(np.asarray(inp["A"]).shape))[h] += g[k][0]
            else:
                bwd.setdefault(k, np.zeros_like(g[k]))
                bwd[k] += g[k]
    return fwd, bwd
