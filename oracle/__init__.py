"""fp64 CPU oracle of the fused slice -> token mix -> deslice path, forward and backward.

TEST INFRASTRUCTURE ONLY. Nothing on the product path imports this package: only the tests,
the smoke check and the benchmark's CPU-baseline leg call it. It shares no code with the HIP
library (no kernels, helpers, tables or constants); both sides only consume the seeded arrays
that ``workloads`` draws.

It is the plain definition written out, one (sample, head) at a time, with the N x G slice
weights materialised in fp64 (the fused kernels never store them). Library matmuls serve as
steps; nothing is blocked, fused or reordered.

What it computes (paper: Sec. 2 "The Transolver layer"; Eq. (1); App. F.1 "Kernel design"):

* logits   a = (X W_s + b) / tau_h                         X: (N, D) projected features
* weights  w[n, :] = softmax over the G slices of a[n, :]  (a partition of unity per point)
* slice    s = sum_n w[n, :],  U = w^T F,  z = U / (s + eps)   (eps as in App. F.1)
* mix      z' = Mix(z): identity, a fixed G x G matrix A (Eq. (1) with constant core,
           z'_g = sum_h A[g, h] z_h), a per-token channel map z' = z W_c (the attention-free
           variant of Sec. 2), or single-head softmax self-attention among the G tokens
* deslice  O = w z'                                         (Sec. 2, u_i = sum_g w_ig z'_g)

Two variants of the ablation suite (Sec. 2) are here as well: the untied one (the deslice
with its own projection, bias and temperature) and LinearNO (untied, with the slice weights
normalised by a softmax over the points of each slot; App. E).

The backward is derived from these definitions (the paper prints only the temperature
gradient and the per-point cancellation, App. F.2 "Temperature gradients"):

* dz' = w^T dO;  dz = Mix^T(dz') and the mix-parameter gradients
* dU = dz / (s + eps);  ds_g = -sum_v dz[g, v] z[g, v] / (s_g + eps)
* dw = dO z'^T + F dU^T + 1 ds^T;  c_n = sum_g w[n, g] dw[n, g];  da = w * (dw - c)
* dF = w dU;  dX = da W_s^T / tau;  dW_s = X^T da / tau;  db = 1^T da / tau;
  dtau = -(1 / tau) sum_{n, g} da[n, g] a[n, g]

Gradients of parameters shared by heads (W_s, b, A, W_c, W_q, W_k, W_v) are summed over
samples and heads; per-head parameters get per-head gradients.

Parity: every function here is pinned by the CPU tests (partition of unity, the G = 1 mean,
the zero-logit / averaging-operator reduction of App. A.2, hard-assignment limit against a
group-by mean, brute-force loops on tiny inputs, invariances, the per-point cancellation of
App. F.2, and central finite differences of the backward). The value of eps, the sharing of
W_s across heads and the attention details are readings of under-specified text (eps is an
argument, W_s may be shared or per head, the attention is one head over the V channels with
scale 1/sqrt(V)); within those readings no function is unpinned.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np

MIX_IDENTITY, MIX_LINEAR_G, MIX_LINEAR_C, MIX_ATTN = 0, 1, 2, 3

f64 = np.float64


# ----------------------------------------------------------------------------------------
# forward steps, one (sample, head) at a time
# ----------------------------------------------------------------------------------------
def logits(X, Ws, b, tau):
    """Slice logits a = (X W_s + b) / tau (Sec. 2; App. F.1, single-tile equation)."""
    return (X @ Ws + b[None, :]) / tau


def slot_softmax(a):
    """Per-point softmax over the slices, with its log-sum-exp (App. F.1, G-blocked kernels:
    m_n = max_g a, l_n = sum_g exp(a - m_n), w = exp(a - m_n) / l_n)."""
    m = a.max(axis=1, keepdims=True)
    e = np.exp(a - m)
    l = e.sum(axis=1, keepdims=True)
    return e / l, (m + np.log(l))[:, 0]


def slice_tokens(w, F, eps):
    """Token numerators, weight sums and normalised tokens z_g = U_g / (s_g + eps) (App. F.1)."""
    s = w.sum(axis=0)
    U = w.T @ F
    return s, U, U / (s + eps)[:, None]


def _row_softmax(S):
    m = S.max(axis=1, keepdims=True)
    e = np.exp(S - m)
    return e / e.sum(axis=1, keepdims=True)


def mix_forward(kind, z, p):
    """Token mix z' = Mix(z). Returns (z', P) with P the attention probabilities (or None).

    p holds the (per-head selected) parameters: A (G, G), Wc (V, V), Wq/Wk/Wv (V, V), scale.
    """
    if kind == MIX_IDENTITY:
        return z.copy(), None
    if kind == MIX_LINEAR_G:   # constant core of Eq. (1): z'_g = sum_h A[g, h] z_h
        return p["A"] @ z, None
    if kind == MIX_LINEAR_C:   # per-token channel map (attention-free variant, Sec. 2)
        return z @ p["Wc"], None
    if kind == MIX_ATTN:       # single-head self-attention among the G tokens
        q, k, v = z @ p["Wq"], z @ p["Wk"], z @ p["Wv"]
        P = _row_softmax(p["scale"] * (q @ k.T))
        return P @ v, P
    raise ValueError(f"unknown mix kind {kind}")


def deslice(w, zm):
    """Deslice O = w z' (Sec. 2, u_i = sum_g w_ig z'_g)."""
    return w @ zm


# ----------------------------------------------------------------------------------------
# backward steps
# ----------------------------------------------------------------------------------------
def mix_backward(kind, z, P, dzm, p):
    """dz = Mix^T(dz') and the mix-parameter gradients of this (sample, head)."""
    if kind == MIX_IDENTITY:
        return dzm.copy(), {}
    if kind == MIX_LINEAR_G:
        return p["A"].T @ dzm, {"dA": dzm @ z.T}
    if kind == MIX_LINEAR_C:
        return dzm @ p["Wc"].T, {"dWc": z.T @ dzm}
    if kind == MIX_ATTN:
        q, k, v = z @ p["Wq"], z @ p["Wk"], z @ p["Wv"]
        dv = P.T @ dzm
        dP = dzm @ v.T
        dS = P * (dP - (dP * P).sum(axis=1, keepdims=True))
        dq = p["scale"] * (dS @ k)
        dk = p["scale"] * (dS.T @ q)
        dz = dq @ p["Wq"].T + dk @ p["Wk"].T + dv @ p["Wv"].T
        return dz, {"dWq": z.T @ dq, "dWk": z.T @ dk, "dWv": z.T @ dv}
    raise ValueError(f"unknown mix kind {kind}")


def token_backward(dz, z, s, eps):
    """Through z = U / (s + eps): dU = dz / (s + eps), ds_g = -sum_v dz z / (s_g + eps)."""
    inv = 1.0 / (s + eps)
    return dz * inv[:, None], -(dz * z).sum(axis=1) * inv


def weight_grad(dO, zm, F, dU, ds):
    """Gradient with respect to the slice weights: w enters O = w z', U = w^T F and s = w^T 1."""
    return dO @ zm.T + F @ dU.T + ds[None, :]


def softmax_backward(w, dw):
    """da = w * (dw - sum_g w dw): the per-point softmax Jacobian (so sum_g da = 0)."""
    return w * (dw - (w * dw).sum(axis=1, keepdims=True))


def logit_backward(da, X, Ws, a, tau):
    """Through a = (X W_s + b) / tau (App. F.2 for the temperature)."""
    dX = da @ Ws.T / tau
    dWs = X.T @ da / tau
    db = da.sum(axis=0) / tau
    dtau = -(da * a).sum() / tau
    return dX, dWs, db, dtau


# ----------------------------------------------------------------------------------------
# whole path
# ----------------------------------------------------------------------------------------
def _head_params(kind, prm, h, ct=f64):
    p = {"scale": ct(prm.get("scale") if prm.get("scale") is not None else 1.0)}
    if kind == MIX_LINEAR_G:
        A = np.asarray(prm["A"], dtype=ct)
        p["A"] = A[h] if A.ndim == 3 else A
    elif kind == MIX_LINEAR_C:
        p["Wc"] = np.asarray(prm["Wc"], dtype=ct)
    elif kind == MIX_ATTN:
        for k in ("Wq", "Wk", "Wv"):
            p[k] = np.asarray(prm[k], dtype=ct)
    return p


def _ws_b(Ws, b, h, ct=f64):
    Ws = np.asarray(Ws, dtype=ct)
    b = np.asarray(b, dtype=ct)
    return (Ws[h] if Ws.ndim == 3 else Ws), (b[h] if b.ndim == 2 else b)


def _pairs(B, H, pairs):
    return [(bb, h) for bb in range(B) for h in range(H)] if pairs is None else list(pairs)


def forward(x, fx, Ws, b, tau, kind, prm: Optional[Dict] = None, eps=1e-5,
            keep_weights=False, pairs=None, dtype=f64) -> Dict[str, np.ndarray]:
    """Forward of the path over all samples and heads (or only the (sample, head) pairs
    listed in ``pairs``; entries of the other pairs are left at zero). ``dtype`` is the
    arithmetic type (fp64; fp32 only to measure what plain fp32 evaluation of the same
    definition loses, the yardstick of the acceptance rule in App. F.2).

    x (B, N, H, D), fx (B, N, H, V), Ws (D, G) or (H, D, G), b (G) or (H, G), tau (H).
    Returns z, s (B, H, G[, V]), zmix (B, H, G, V), P (B, H, G, G) for attention,
    lse (B, H, N), out (B, N, H, V); with keep_weights also a and w (B, H, N, G).
    """
    prm = prm or {}
    B, N, H, D = x.shape
    V = fx.shape[3]
    G = np.asarray(Ws).shape[-1]
    res = {k: np.zeros(sh) for k, sh in dict(
        z=(B, H, G, V), s=(B, H, G), zmix=(B, H, G, V), lse=(B, H, N),
        out=(B, N, H, V)).items()}
    res["P"] = np.zeros((B, H, G, G)) if kind == MIX_ATTN else None
    if keep_weights:
        res["a"] = np.zeros((B, H, N, G))
        res["w"] = np.zeros((B, H, N, G))
    ct = np.dtype(dtype).type
    for bb, h in _pairs(B, H, pairs):
        X = np.asarray(x[bb, :, h, :], dtype=ct)
        F = np.asarray(fx[bb, :, h, :], dtype=ct)
        Wsh, bh = _ws_b(Ws, b, h, ct)
        a = logits(X, Wsh, bh, ct(tau[h]))
        w, lse = slot_softmax(a)
        s, U, z = slice_tokens(w, F, ct(eps))
        zm, P = mix_forward(kind, z, _head_params(kind, prm, h, ct))
        res["z"][bb, h], res["s"][bb, h], res["zmix"][bb, h] = z, s, zm
        res["lse"][bb, h] = lse
        if P is not None:
            res["P"][bb, h] = P
        res["out"][bb, :, h, :] = deslice(w, zm)
        if keep_weights:
            res["a"][bb, h], res["w"][bb, h] = a, w
    return res


def forward_repeated(x, fx, Ws, b, tau, kind, prm: Optional[Dict], eps, repeat, points,
                     pairs=None) -> Dict[str, np.ndarray]:
    """Forward over the point set made of ``repeat`` back-to-back copies of the given block of
    points (full N = repeat * block), evaluated from the block alone: each copy contributes
    the same terms to s = sum_n w[n, :] and U = w^T F, so both are ``repeat`` times the
    block's sums, and a point's weights, lse and output depend only on its own row.

    points: full-size point indices (copy k of block point n is point k * block + n).
    Returns z, s, zmix (B, H, G[, V]), P, and lse (B, H, len(points)), out (B, len(points),
    H, V) at those points; entries of pairs not listed stay zero.
    """
    prm = prm or {}
    B, Nb, H, D = x.shape
    V = fx.shape[3]
    G = np.asarray(Ws).shape[-1]
    idx = np.asarray(points, dtype=np.int64) % Nb
    res = {k: np.zeros(sh) for k, sh in dict(
        z=(B, H, G, V), s=(B, H, G), zmix=(B, H, G, V), lse=(B, H, len(idx)),
        out=(B, len(idx), H, V)).items()}
    res["P"] = np.zeros((B, H, G, G)) if kind == MIX_ATTN else None
    for bb, h in _pairs(B, H, pairs):
        X = np.asarray(x[bb, :, h, :], dtype=f64)
        F = np.asarray(fx[bb, :, h, :], dtype=f64)
        Wsh, bh = _ws_b(Ws, b, h)
        w, lse = slot_softmax(logits(X, Wsh, bh, f64(tau[h])))
        s, U, z = slice_tokens(f64(repeat) * w, F, f64(eps))
        zm, P = mix_forward(kind, z, _head_params(kind, prm, h))
        res["z"][bb, h], res["s"][bb, h], res["zmix"][bb, h] = z, s, zm
        if P is not None:
            res["P"][bb, h] = P
        res["lse"][bb, h] = lse[idx]
        res["out"][bb, :, h, :] = deslice(w[idx], zm)
    return res


def backward(x, fx, Ws, b, tau, kind, prm: Optional[Dict], dout, eps=1e-5,
             fwd: Optional[Dict] = None, pairs=None, dtype=f64) -> Dict[str, np.ndarray]:
    """Backward of the path for the upstream gradient dout (B, N, H, V) (over all samples and
    heads, or only the listed pairs: then parameter gradients sum those pairs only).

    Returns dx, dfx (point gradients), dWs, db (shaped like Ws, b), dtau (H), dzmix and dz
    (B, H, G, V), and the mix-parameter gradients (dA, dWc or dWq/dWk/dWv).
    """
    prm = prm or {}
    B, N, H, D = x.shape
    V = fx.shape[3]
    Ws_arr = np.asarray(Ws, dtype=f64)
    b_arr = np.asarray(b, dtype=f64)
    G = Ws_arr.shape[-1]
    if fwd is None:
        fwd = forward(x, fx, Ws, b, tau, kind, prm, eps, pairs=pairs, dtype=dtype)
    ct = np.dtype(dtype).type
    res = dict(dx=np.zeros((B, N, H, D)), dfx=np.zeros((B, N, H, V)),
               dWs=np.zeros_like(Ws_arr), db=np.zeros_like(b_arr), dtau=np.zeros(H),
               dzmix=np.zeros((B, H, G, V)), dz=np.zeros((B, H, G, V)))
    for bb, h in _pairs(B, H, pairs):
        X = np.asarray(x[bb, :, h, :], dtype=ct)
        F = np.asarray(fx[bb, :, h, :], dtype=ct)
        dO = np.asarray(dout[bb, :, h, :], dtype=ct)
        Wsh, bh = _ws_b(Ws, b, h, ct)
        t = ct(tau[h])
        a = logits(X, Wsh, bh, t)
        w, _ = slot_softmax(a)
        z, s, zm = (fwd["z"][bb, h].astype(ct), fwd["s"][bb, h].astype(ct),
                    fwd["zmix"][bb, h].astype(ct))
        P = fwd["P"][bb, h].astype(ct) if fwd.get("P") is not None else None
        dzm = w.T @ dO
        dz, dprm = mix_backward(kind, z, P, dzm, _head_params(kind, prm, h, ct))
        dU, ds = token_backward(dz, z, s, ct(eps))
        dw = weight_grad(dO, zm, F, dU, ds)
        da = softmax_backward(w, dw)
        dX, dWs, db, dtau = logit_backward(da, X, Wsh, a, t)
        res["dx"][bb, :, h, :] = dX
        res["dfx"][bb, :, h, :] = w @ dU
        res["dzmix"][bb, h], res["dz"][bb, h] = dzm, dz
        res["dtau"][h] += dtau
        if Ws_arr.ndim == 3:
            res["dWs"][h] += dWs
        else:
            res["dWs"] += dWs
        if b_arr.ndim == 2:
            res["db"][h] += db
        else:
            res["db"] += db
        for k, v in dprm.items():
            if k == "dA" and np.asarray(prm["A"]).ndim == 3:
                res.setdefault(k, np.zeros((H, G, G)))[h] += v
            else:
                res.setdefault(k, np.zeros_like(v))
                res[k] += v
    return res


# ----------------------------------------------------------------------------------------
# untied variant (Sec. 2 ablation suite): the deslice has its own projection W_d, bias b_d
# and temperature tau_d, so its weights w_d = softmax_g((X W_d + b_d) / tau_d) differ from
# the slice weights w
# ----------------------------------------------------------------------------------------
def untied_forward(x, fx, Ws, b, tau, Wd, bd, taud, kind, prm: Optional[Dict] = None,
                   eps=1e-5, pairs=None, dtype=f64) -> Dict[str, np.ndarray]:
    """Slice with (W_s, b, tau), mix, deslice with (W_d, b_d, tau_d). Returns z, s, zmix,
    P, lse (slice normaliser), lse_d (deslice normaliser) and out. ``dtype`` as in
    forward."""
    prm = prm or {}
    B, N, H, D = x.shape
    V = fx.shape[3]
    G = np.asarray(Ws).shape[-1]
    res = {k: np.zeros(sh) for k, sh in dict(
        z=(B, H, G, V), s=(B, H, G), zmix=(B, H, G, V), lse=(B, H, N), lse_d=(B, H, N),
        out=(B, N, H, V)).items()}
    res["P"] = np.zeros((B, H, G, G)) if kind == MIX_ATTN else None
    ct = np.dtype(dtype).type
    for bb, h in _pairs(B, H, pairs):
        X = np.asarray(x[bb, :, h, :], dtype=ct)
        F = np.asarray(fx[bb, :, h, :], dtype=ct)
        Wsh, bh = _ws_b(Ws, b, h, ct)
        Wdh, bdh = _ws_b(Wd, bd, h, ct)
        w, lse = slot_softmax(logits(X, Wsh, bh, ct(tau[h])))
        s, U, z = slice_tokens(w, F, ct(eps))
        zm, P = mix_forward(kind, z, _head_params(kind, prm, h, ct))
        wd, lse_d = slot_softmax(logits(X, Wdh, bdh, ct(taud[h])))
        res["z"][bb, h], res["s"][bb, h], res["zmix"][bb, h] = z, s, zm
        res["lse"][bb, h], res["lse_d"][bb, h] = lse, lse_d
        if P is not None:
            res["P"][bb, h] = P
        res["out"][bb, :, h, :] = deslice(wd, zm)
    return res


def untied_backward(x, fx, Ws, b, tau, Wd, bd, taud, kind, prm: Optional[Dict], dout,
                    eps=1e-5, fwd: Optional[Dict] = None, pairs=None,
                    dtype=f64) -> Dict[str, np.ndarray]:
    """Backward of the untied path. The deslice weights receive dw_d = dO z'^T only; the
    slice weights receive dw = F dU^T + 1 ds^T only; each goes through its own softmax
    Jacobian and its own projection. Returns dx, dfx, dWs, db, dtau, dWd, dbd, dtaud,
    dzmix, dz and the mix-parameter gradients."""
    prm = prm or {}
    B, N, H, D = x.shape
    V = fx.shape[3]
    Ws_arr, b_arr = np.asarray(Ws, dtype=f64), np.asarray(b, dtype=f64)
    Wd_arr, bd_arr = np.asarray(Wd, dtype=f64), np.asarray(bd, dtype=f64)
    G = Ws_arr.shape[-1]
    if fwd is None:
        fwd = untied_forward(x, fx, Ws, b, tau, Wd, bd, taud, kind, prm, eps, pairs=pairs,
                             dtype=dtype)
    ct = np.dtype(dtype).type
    res = dict(dx=np.zeros((B, N, H, D)), dfx=np.zeros((B, N, H, V)),
               dWs=np.zeros_like(Ws_arr), db=np.zeros_like(b_arr), dtau=np.zeros(H),
               dWd=np.zeros_like(Wd_arr), dbd=np.zeros_like(bd_arr), dtaud=np.zeros(H),
               dzmix=np.zeros((B, H, G, V)), dz=np.zeros((B, H, G, V)))
    for bb, h in _pairs(B, H, pairs):
        X = np.asarray(x[bb, :, h, :], dtype=ct)
        F = np.asarray(fx[bb, :, h, :], dtype=ct)
        dO = np.asarray(dout[bb, :, h, :], dtype=ct)
        Wsh, bh = _ws_b(Ws, b, h, ct)
        Wdh, bdh = _ws_b(Wd, bd, h, ct)
        t, td = ct(tau[h]), ct(taud[h])
        a = logits(X, Wsh, bh, t)
        w, _ = slot_softmax(a)
        ad = logits(X, Wdh, bdh, td)
        wd, _ = slot_softmax(ad)
        z, s, zm = (fwd["z"][bb, h].astype(ct), fwd["s"][bb, h].astype(ct),
                    fwd["zmix"][bb, h].astype(ct))
        P = fwd["P"][bb, h].astype(ct) if fwd.get("P") is not None else None
        dzm = wd.T @ dO
        dz, dprm = mix_backward(kind, z, P, dzm, _head_params(kind, prm, h, ct))
        dU, ds = token_backward(dz, z, s, ct(eps))
        da = softmax_backward(w, F @ dU.T + ds[None, :])
        dad = softmax_backward(wd, dO @ zm.T)
        dX, dWs, db, dtau = logit_backward(da, X, Wsh, a, t)
        dXd, dWd, dbd, dtaud = logit_backward(dad, X, Wdh, ad, td)
        res["dx"][bb, :, h, :] = dX + dXd
        res["dfx"][bb, :, h, :] = w @ dU
        res["dzmix"][bb, h], res["dz"][bb, h] = dzm, dz
        res["dtau"][h] += dtau
        res["dtaud"][h] += dtaud
        for key, arr, val in (("dWs", Ws_arr, dWs), ("db", b_arr, db), ("dWd", Wd_arr, dWd),
                              ("dbd", bd_arr, dbd)):
            per_head = arr.ndim == (3 if key in ("dWs", "dWd") else 2)
            if per_head:
                res[key][h] += val
            else:
                res[key] += val
        for k, v in dprm.items():
            if k == "dA" and np.asarray(prm["A"]).ndim == 3:
                res.setdefault(k, np.zeros((H, G, G)))[h] += v
            else:
                res.setdefault(k, np.zeros_like(v))
                res[k] += v
    return res


# ----------------------------------------------------------------------------------------
# LinearNO (the Untied-LN variant of Sec. 2 and App. E): the slice weights are normalised by
# a softmax over the N points of each slot, k[:, g] = softmax_n(a[:, g]), so the tokens are
# z_g = sum_n k[n, g] F[n] with no division by a weight sum; the deslice has its own
# projection, bias and temperature with the usual softmax over the slots
# ----------------------------------------------------------------------------------------
def point_softmax(a):
    """Softmax of each slot's logits over the points, with its log-sum-exp per slot
    (natural log); an empty point set gives no weights and lse = -inf."""
    if a.shape[0] == 0:
        return a.copy(), np.full(a.shape[1], -np.inf)
    m = a.max(axis=0, keepdims=True)
    e = np.exp(a - m)
    l = e.sum(axis=0, keepdims=True)
    return e / l, (m + np.log(l))[0]


def point_softmax_backward(k, dk):
    """da = k * (dk - sum_n k dk), per slot (so sum_n da[:, g] = 0)."""
    return k * (dk - (k * dk).sum(axis=0, keepdims=True))


def linearno_forward(x, fx, Ws, b, tau, Wd, bd, taud, kind, prm: Optional[Dict] = None,
                     pairs=None, dtype=f64) -> Dict[str, np.ndarray]:
    """Returns z (B,H,G,V), clse (B,H,G) (the slots' log normalisers over the points,
    natural log), zmix, P, lse_d (B,H,N) and out."""
    prm = prm or {}
    B, N, H, D = x.shape
    V = fx.shape[3]
    G = np.asarray(Ws).shape[-1]
    res = {k: np.zeros(sh) for k, sh in dict(
        z=(B, H, G, V), clse=(B, H, G), zmix=(B, H, G, V), lse_d=(B, H, N),
        out=(B, N, H, V)).items()}
    res["P"] = np.zeros((B, H, G, G)) if kind == MIX_ATTN else None
    ct = np.dtype(dtype).type
    for bb, h in _pairs(B, H, pairs):
        X = np.asarray(x[bb, :, h, :], dtype=ct)
        F = np.asarray(fx[bb, :, h, :], dtype=ct)
        Wsh, bh = _ws_b(Ws, b, h, ct)
        Wdh, bdh = _ws_b(Wd, bd, h, ct)
        k, clse = point_softmax(logits(X, Wsh, bh, ct(tau[h])))
        z = k.T @ F
        zm, P = mix_forward(kind, z, _head_params(kind, prm, h, ct))
        wd, lse_d = slot_softmax(logits(X, Wdh, bdh, ct(taud[h])))
        res["z"][bb, h], res["clse"][bb, h], res["zmix"][bb, h] = z, clse, zm
        res["lse_d"][bb, h] = lse_d
        if P is not None:
            res["P"][bb, h] = P
        res["out"][bb, :, h, :] = deslice(wd, zm)
    return res


def linearno_backward(x, fx, Ws, b, tau, Wd, bd, taud, kind, prm: Optional[Dict], dout,
                      fwd: Optional[Dict] = None, pairs=None,
                      dtype=f64) -> Dict[str, np.ndarray]:
    """Backward of LinearNO: the deslice part as in untied_backward; the slice weights get
    dk = F dz^T through the softmax over the points. Returns dx, dfx, dWs, db, dtau, dWd,
    dbd, dtaud, dzmix, dz and the mix-parameter gradients."""
    prm = prm or {}
    B, N, H, D = x.shape
    V = fx.shape[3]
    Ws_arr, b_arr = np.asarray(Ws, dtype=f64), np.asarray(b, dtype=f64)
    Wd_arr, bd_arr = np.asarray(Wd, dtype=f64), np.asarray(bd, dtype=f64)
    G = Ws_arr.shape[-1]
    if fwd is None:
        fwd = linearno_forward(x, fx, Ws, b, tau, Wd, bd, taud, kind, prm, pairs=pairs,
                               dtype=dtype)
    ct = np.dtype(dtype).type
    res = dict(dx=np.zeros((B, N, H, D)), dfx=np.zeros((B, N, H, V)),
               dWs=np.zeros_like(Ws_arr), db=np.zeros_like(b_arr), dtau=np.zeros(H),
               dWd=np.zeros_like(Wd_arr), dbd=np.zeros_like(bd_arr), dtaud=np.zeros(H),
               dzmix=np.zeros((B, H, G, V)), dz=np.zeros((B, H, G, V)))
    for bb, h in _pairs(B, H, pairs):
        X = np.asarray(x[bb, :, h, :], dtype=ct)
        F = np.asarray(fx[bb, :, h, :], dtype=ct)
        dO = np.asarray(dout[bb, :, h, :], dtype=ct)
        Wsh, bh = _ws_b(Ws, b, h, ct)
        Wdh, bdh = _ws_b(Wd, bd, h, ct)
        t, td = ct(tau[h]), ct(taud[h])
        a = logits(X, Wsh, bh, t)
        k, _ = point_softmax(a)
        ad = logits(X, Wdh, bdh, td)
        wd, _ = slot_softmax(ad)
        z, zm = fwd["z"][bb, h].astype(ct), fwd["zmix"][bb, h].astype(ct)
        P = fwd["P"][bb, h].astype(ct) if fwd.get("P") is not None else None
        dzm = wd.T @ dO
        dz, dprm = mix_backward(kind, z, P, dzm, _head_params(kind, prm, h, ct))
        da = point_softmax_backward(k, F @ dz.T)
        dad = softmax_backward(wd, dO @ zm.T)
        dX, dWs, db, dtau = logit_backward(da, X, Wsh, a, t)
        dXd, dWd, dbd, dtaud = logit_backward(dad, X, Wdh, ad, td)
        res["dx"][bb, :, h, :] = dX + dXd
        res["dfx"][bb, :, h, :] = k @ dz
        res["dzmix"][bb, h], res["dz"][bb, h] = dzm, dz
        res["dtau"][h] += dtau
        res["dtaud"][h] += dtaud
        for key, arr, val in (("dWs", Ws_arr, dWs), ("db", b_arr, db), ("dWd", Wd_arr, dWd),
                              ("dbd", bd_arr, dbd)):
            per_head = arr.ndim == (3 if key in ("dWs", "dWd") else 2)
            if per_head:
                res[key][h] += val
            else:
                res[key] += val
        for kk, v in dprm.items():
            if kk == "dA" and np.asarray(prm["A"]).ndim == 3:
                res.setdefault(kk, np.zeros((H, G, G)))[h] += v
            else:
                res.setdefault(kk, np.zeros_like(v))
                res[kk] += v
    return res


def run_inputs(inp: Dict, kind: int, eps: float = 1e-5, backward_too: bool = True,
               pairs=None, dtype=f64):
    """Convenience: forward (+ backward) on a ``workloads.make_inputs`` dictionary."""
    prm = {k: inp.get(k) for k in ("A", "Wc", "Wq", "Wk", "Wv", "scale")}
    fwd = forward(inp["x"], inp["fx"], inp["Ws"], inp["b"], inp["tau"], kind, prm, eps,
                  pairs=pairs, dtype=dtype)
    if not backward_too:
        return fwd, None
    bwd = backward(inp["x"], inp["fx"], inp["Ws"], inp["b"], inp["tau"], kind, prm,
                   inp["dout"], eps, fwd=fwd, pairs=pairs, dtype=dtype)
    return fwd, bwd
