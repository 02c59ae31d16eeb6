"""Pins of the fp64 oracle against what the paper and the mathematics fix (CPU only).

Each ``check_*`` takes the oracle module and raises AssertionError on a violation. The tests
run every check on the real oracle; ``test_planted_mistakes`` plants plausible mistakes in a
copy of the oracle (a dropped term, a wrong sign, a transposed operand, ...) and asserts that
at least one check fails for each, which shows the checks are not vacuous.
"""
import itertools
import types

import numpy as np
import pytest

import oracle as O

RNG = np.random.default_rng(12345)
MIXES = [O.MIX_IDENTITY, O.MIX_LINEAR_G, O.MIX_LINEAR_C, O.MIX_ATTN]


def _rand(*shape, std=1.0, rng=None):
    return (rng or RNG).standard_normal(shape) * std


def _prm(kind, G, V, rng, H=None):
    p = {"scale": 1.0 / np.sqrt(V)}
    if kind == O.MIX_LINEAR_G:
        p["A"] = _rand(*((H, G, G) if H else (G, G)), std=1 / np.sqrt(G), rng=rng)
    elif kind == O.MIX_LINEAR_C:
        p["Wc"] = _rand(V, V, std=0.5, rng=rng)
    elif kind == O.MIX_ATTN:
        for k in ("Wq", "Wk", "Wv"):
            p[k] = _rand(V, V, std=0.7, rng=rng)
    return p


def _problem(B=2, N=7, H=2, D=3, V=2, G=4, seed=0, per_head=False, bias=True):
    rng = np.random.default_rng(seed)
    x = _rand(B, N, H, D, rng=rng)
    fx = _rand(B, N, H, V, rng=rng)
    Ws = _rand(*((H, D, G) if per_head else (D, G)), rng=rng)
    b = _rand(*((H, G) if per_head else (G,)), rng=rng) * (1.0 if bias else 0.0)
    tau = rng.uniform(0.4, 1.5, size=H)
    return x, fx, Ws, b, tau, rng


# ----------------------------------------------------------------------------------------
# forward pins
# ----------------------------------------------------------------------------------------
def check_partition_of_unity(o):
    """I1: slice weights are non-negative and sum to one over the slices (Sec. 2)."""
    x, fx, Ws, b, tau, rng = _problem(N=50, G=6)
    r = o.forward(x, fx, Ws, b, tau, o.MIX_IDENTITY, {}, keep_weights=True)
    w = r["w"]
    assert (w >= 0).all()
    np.testing.assert_allclose(w.sum(-1), 1.0, rtol=0, atol=1e-13)
    # lse is the log of the softmax normaliser: w = exp(a - lse)
    np.testing.assert_allclose(w, np.exp(r["a"] - r["lse"][..., None]), rtol=1e-12, atol=1e-15)


def check_single_slice_mean(o):
    """I2: with G = 1 every weight is 1, so z = sum_n F_n / (N + eps)."""
    eps = 0.37
    x, fx, Ws, b, tau, rng = _problem(N=9, G=1)
    r = o.forward(x, fx, Ws, b, tau, o.MIX_IDENTITY, {}, eps=eps)
    want = fx.sum(axis=1).transpose(0, 1, 2)[:, :, None, :] / (x.shape[1] + eps)  # (B,H,1,V)
    np.testing.assert_allclose(r["z"], want, rtol=1e-13)
    np.testing.assert_allclose(r["s"], x.shape[1], rtol=1e-13)
    # deslice of the single token broadcasts it to every point
    np.testing.assert_allclose(r["out"], np.broadcast_to(want[:, None, :, 0, :], r["out"].shape),
                               rtol=1e-13)


def check_identical_points(o):
    """I3: identical points give z_g = f N w_g / (N w_g + eps) for every slot."""
    eps = 1e-3
    B, N, H, D, V, G = 1, 11, 2, 3, 4, 5
    rng = np.random.default_rng(3)
    x = np.broadcast_to(_rand(1, 1, H, D, rng=rng), (B, N, H, D)).copy()
    f = _rand(1, 1, H, V, rng=rng)
    fx = np.broadcast_to(f, (B, N, H, V)).copy()
    Ws, b, tau = _rand(D, G, rng=rng), _rand(G, rng=rng), np.array([0.7, 1.3])
    r = o.forward(x, fx, Ws, b, tau, o.MIX_IDENTITY, {}, eps=eps, keep_weights=True)
    w0 = r["w"][0, :, 0, :]                                      # (H, G) weights of one point
    want = f[0, 0][:, None, :] * (N * w0 / (N * w0 + eps))[:, :, None]
    np.testing.assert_allclose(r["z"][0], want, rtol=1e-12)


def check_constant_tokens(o):
    """I4: if every mixed token equals the same vector c, the deslice gives c at every point
    (the weights are a partition of unity). A = ones/G makes z'_g = mean_h z_h for all g."""
    x, fx, Ws, b, tau, rng = _problem(N=13, G=5, V=3)
    G = 5
    prm = {"A": np.full((G, G), 1.0 / G)}
    r = o.forward(x, fx, Ws, b, tau, o.MIX_LINEAR_G, prm)
    c = r["z"].mean(axis=2)                                      # (B, H, V)
    np.testing.assert_allclose(r["zmix"], np.broadcast_to(c[:, :, None, :], r["zmix"].shape),
                               rtol=1e-12)
    np.testing.assert_allclose(r["out"], np.broadcast_to(c[:, None, :, :], r["out"].shape),
                               rtol=1e-12, atol=1e-14)


def check_zero_logits(o):
    """I5/I6: zero logits make every weight 1/G, every token the global mean (times
    N / (N + G eps)), and with a constant core normalised so that sum_{g,h} A_gh / G = 1 the
    layer reduces to the averaging operator O_n = mean (App. A.2, proof of Proposition 1)."""
    eps = 0.05
    x, fx, Ws, b, tau, rng = _problem(N=17, G=6, V=3)
    N, G = 17, 6
    Ws0, b0 = np.zeros_like(Ws), np.zeros_like(b)
    A = rng.uniform(0.1, 1.0, size=(G, G))
    A *= G / A.sum()
    r = o.forward(x, fx, Ws0, b0, tau, o.MIX_LINEAR_G, {"A": A}, eps=eps)
    mean = fx.sum(axis=1) / (N + G * eps)                        # (B, H, V)
    np.testing.assert_allclose(r["z"], np.broadcast_to(mean[:, :, None, :], r["z"].shape),
                               rtol=1e-13)
    np.testing.assert_allclose(r["lse"], np.log(G), rtol=1e-13)
    np.testing.assert_allclose(r["out"], np.broadcast_to(mean[:, None, :, :], r["out"].shape),
                               rtol=1e-12)


def check_hard_assignment(o):
    """At a tiny temperature the weights become the one-hot argmax of the logits, the slice
    becomes a group-by mean (k-means style) and the deslice a table look-up."""
    eps = 1e-5
    B, N, H, D, V, G = 1, 60, 1, 4, 3, 5
    rng = np.random.default_rng(11)
    x, fx = _rand(B, N, H, D, rng=rng), _rand(B, N, H, V, rng=rng)
    Ws, b = _rand(D, G, rng=rng), _rand(G, rng=rng)
    raw = x[0, :, 0, :] @ Ws + b
    srt = np.sort(raw, axis=1)
    keep = (srt[:, -1] - srt[:, -2]) > 0.05                      # drop near-ties
    x, fx = x[:, keep], fx[:, keep]
    raw = raw[keep]
    tau = np.array([1e-4])
    prm = {"Wc": _rand(V, V, rng=rng)}
    r = o.forward(x, fx, Ws, b, tau, o.MIX_LINEAR_C, prm, eps=eps)
    lab = raw.argmax(axis=1)
    F = fx[0, :, 0, :]
    cnt = np.bincount(lab, minlength=G).astype(float)
    sums = np.zeros((G, F.shape[1]))
    np.add.at(sums, lab, F)
    z = sums / (cnt + eps)[:, None]
    np.testing.assert_allclose(r["s"][0, 0], cnt, atol=1e-12)
    np.testing.assert_allclose(r["z"][0, 0], z, rtol=1e-10, atol=1e-12)
    zm = z @ prm["Wc"]
    np.testing.assert_allclose(r["out"][0, :, 0, :], zm[lab], rtol=1e-10, atol=1e-12)


def _brute_forward(x, fx, Ws, b, tau, kind, prm, eps):
    """Naive loops over every index (tiny inputs only)."""
    B, N, H, D = x.shape
    V, G = fx.shape[3], Ws.shape[-1]
    out = np.zeros((B, N, H, V))
    zs = np.zeros((B, H, G, V))
    for bb, h in itertools.product(range(B), range(H)):
        w = np.zeros((N, G))
        for n in range(N):
            row = [sum(x[bb, n, h, d] * Ws[d, g] for d in range(D)) + b[g] for g in range(G)]
            row = [r / tau[h] for r in row]
            mx = max(row)
            ex = [np.exp(r - mx) for r in row]
            tot = sum(ex)
            for g in range(G):
                w[n, g] = ex[g] / tot
        z = np.zeros((G, V))
        for g in range(G):
            sg = sum(w[n, g] for n in range(N))
            for v in range(V):
                z[g, v] = sum(w[n, g] * fx[bb, n, h, v] for n in range(N)) / (sg + eps)
        zm = np.zeros((G, V))
        if kind == O.MIX_LINEAR_G:
            for g, v in itertools.product(range(G), range(V)):
                zm[g, v] = sum(prm["A"][g, k] * z[k, v] for k in range(G))
        elif kind == O.MIX_ATTN:
            q = [[sum(z[g, c] * prm["Wq"][c, e] for c in range(V)) for e in range(V)] for g in range(G)]
            k_ = [[sum(z[g, c] * prm["Wk"][c, e] for c in range(V)) for e in range(V)] for g in range(G)]
            v_ = [[sum(z[g, c] * prm["Wv"][c, e] for c in range(V)) for e in range(V)] for g in range(G)]
            for g in range(G):
                sc = [prm["scale"] * sum(q[g][e] * k_[t][e] for e in range(V)) for t in range(G)]
                mx = max(sc)
                ex = [np.exp(c - mx) for c in sc]
                tot = sum(ex)
                for v in range(V):
                    zm[g, v] = sum(ex[t] / tot * v_[t][v] for t in range(G))
        else:
            raise ValueError
        zs[bb, h] = zm
        for n, v in itertools.product(range(N), range(V)):
            out[bb, n, h, v] = sum(w[n, g] * zm[g, v] for g in range(G))
    return zs, out


def check_bruteforce(o):
    """Naive index loops agree with the oracle on tiny inputs (fixed matrix and attention)."""
    eps = 0.02
    for kind in (O.MIX_LINEAR_G, O.MIX_ATTN):
        x, fx, Ws, b, tau, rng = _problem(B=1, N=5, H=2, D=3, V=2, G=4, seed=kind)
        prm = _prm(kind, 4, 2, rng)
        r = o.forward(x, fx, Ws, b, tau, kind, prm, eps=eps)
        zs, out = _brute_forward(x, fx, Ws, b, tau, kind, prm, eps)
        np.testing.assert_allclose(r["zmix"], zs, rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(r["out"], out, rtol=1e-12, atol=1e-14)


def check_invariances(o):
    """I7: point permutation, slot permutation, positive rescaling of (W_s, b, tau),
    shifts of all logits of a point, and linearity of the output in F."""
    eps = 1e-3
    x, fx, Ws, b, tau, rng = _problem(B=1, N=12, H=2, D=3, V=2, G=5)
    G = 5
    prm = _prm(O.MIX_LINEAR_G, G, 2, rng)
    base = o.forward(x, fx, Ws, b, tau, O.MIX_LINEAR_G, prm, eps=eps)
    # points
    perm = rng.permutation(12)
    r = o.forward(x[:, perm], fx[:, perm], Ws, b, tau, O.MIX_LINEAR_G, prm, eps=eps)
    np.testing.assert_allclose(r["z"], base["z"], rtol=1e-12)
    np.testing.assert_allclose(r["out"], base["out"][:, perm], rtol=1e-12, atol=1e-14)
    # slots (W_s columns, b, A -> Pi A Pi^T)
    sp = rng.permutation(G)
    A2 = prm["A"][np.ix_(sp, sp)]
    r = o.forward(x, fx, Ws[:, sp], b[sp], tau, O.MIX_LINEAR_G, {"A": A2}, eps=eps)
    np.testing.assert_allclose(r["out"], base["out"], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(r["z"], base["z"][:, :, sp], rtol=1e-12)
    # scale (W_s, b, tau) by c > 0
    r = o.forward(x, fx, 2.5 * Ws, 2.5 * b, 2.5 * tau, O.MIX_LINEAR_G, prm, eps=eps)
    np.testing.assert_allclose(r["out"], base["out"], rtol=1e-12, atol=1e-14)
    # add a constant vector to every column of W_s and a constant to b
    cvec = rng.standard_normal((3, 1))
    r = o.forward(x, fx, Ws + cvec, b + 0.7, tau, O.MIX_LINEAR_G, prm, eps=eps)
    np.testing.assert_allclose(r["out"], base["out"], rtol=1e-11, atol=1e-13)
    # linear in F
    fx2 = rng.standard_normal(fx.shape)
    r2 = o.forward(x, fx2, Ws, b, tau, O.MIX_LINEAR_G, prm, eps=eps)
    r3 = o.forward(x, 2.0 * fx - 3.0 * fx2, Ws, b, tau, O.MIX_LINEAR_G, prm, eps=eps)
    np.testing.assert_allclose(r3["out"], 2.0 * base["out"] - 3.0 * r2["out"], rtol=1e-11,
                               atol=1e-12)


def check_mix_closed_forms(o):
    """I11: identity maps, uniform attention for W_q = 0, attention rows sum to one, and the
    one-hot limit of a very large attention scale."""
    rng = np.random.default_rng(5)
    G, V = 6, 3
    z = rng.standard_normal((G, V))
    zm, _ = o.mix_forward(o.MIX_IDENTITY, z, {})
    np.testing.assert_array_equal(zm, z)
    zm, _ = o.mix_forward(o.MIX_LINEAR_G, z, {"A": np.eye(G)})
    np.testing.assert_allclose(zm, z, rtol=0, atol=0)
    zm, _ = o.mix_forward(o.MIX_LINEAR_C, z, {"Wc": np.eye(V)})
    np.testing.assert_allclose(zm, z, rtol=0, atol=0)
    Wv = rng.standard_normal((V, V))
    p = {"Wq": np.zeros((V, V)), "Wk": rng.standard_normal((V, V)), "Wv": Wv, "scale": 0.6}
    zm, P = o.mix_forward(o.MIX_ATTN, z, p)
    np.testing.assert_allclose(P, 1.0 / G, rtol=1e-14)
    np.testing.assert_allclose(zm, np.broadcast_to(z.mean(0) @ Wv, (G, V)), rtol=1e-12)
    p = {"Wq": rng.standard_normal((V, V)), "Wk": rng.standard_normal((V, V)), "Wv": Wv,
         "scale": 0.6}
    zm, P = o.mix_forward(o.MIX_ATTN, z, p)
    np.testing.assert_allclose(P.sum(1), 1.0, rtol=1e-14)
    S = (z @ p["Wq"]) @ (z @ p["Wk"]).T
    p["scale"] = 1e6
    zm, P = o.mix_forward(o.MIX_ATTN, z, p)
    np.testing.assert_allclose(zm, (z @ Wv)[S.argmax(1)], rtol=1e-9, atol=1e-12)


# ----------------------------------------------------------------------------------------
# backward pins
# ----------------------------------------------------------------------------------------
def _loss_and_grads(o, x, fx, Ws, b, tau, kind, prm, R, eps):
    fwd = o.forward(x, fx, Ws, b, tau, kind, prm, eps=eps)
    g = o.backward(x, fx, Ws, b, tau, kind, prm, R, eps=eps, fwd=fwd)
    return (fwd["out"] * R).sum(), g


def check_finite_differences(o, kinds=tuple(MIXES), per_head=False):
    """I12: central differences of L = sum(O * R) in fp64 match every analytic gradient."""
    eps = 0.3   # large, so that a dropped eps term shows
    for kind in kinds:
        x, fx, Ws, b, tau, rng = _problem(B=2, N=6, H=2, D=3, V=2, G=4, seed=20 + kind,
                                          per_head=per_head)
        prm = _prm(kind, 4, 2, rng, H=2 if per_head else None)
        R = rng.standard_normal((2, 6, 2, 2))
        _, g = _loss_and_grads(o, x, fx, Ws, b, tau, kind, prm, R, eps)
        tensors = {"dx": x, "dfx": fx, "dWs": Ws, "db": b, "dtau": tau}
        for k in ("A", "Wc", "Wq", "Wk", "Wv"):
            if prm.get(k) is not None:
                tensors["d" + k] = prm[k]
        step = 1e-6
        for gname, arr in tensors.items():
            num = np.zeros_like(arr)
            for idx in np.ndindex(arr.shape):
                old = arr[idx]
                arr[idx] = old + step
                lp = (o.forward(x, fx, Ws, b, tau, kind, prm, eps=eps)["out"] * R).sum()
                arr[idx] = old - step
                lm = (o.forward(x, fx, Ws, b, tau, kind, prm, eps=eps)["out"] * R).sum()
                arr[idx] = old
                num[idx] = (lp - lm) / (2 * step)
            ana = g[gname]
            scale = max(np.abs(num).max(), 1e-3)
            err = np.abs(ana - num).max() / scale
            assert err < 2e-7, (kind, gname, err)


def check_cancellation(o):
    """I8 (App. F.2): sum_g da[n, g] = 0 per point, hence sum_g db_g = 0 and
    sum_g dW_s[d, g] = 0 for every d."""
    x, fx, Ws, b, tau, rng = _problem(B=2, N=30, H=3, D=4, V=3, G=7, seed=9)
    prm = _prm(O.MIX_LINEAR_G, 7, 3, rng)
    R = rng.standard_normal(fx.shape)
    _, g = _loss_and_grads(o, x, fx, Ws, b, tau, O.MIX_LINEAR_G, prm, R, 1e-3)
    assert abs(g["db"].sum()) < 1e-12 * np.abs(g["db"]).sum() + 1e-14
    np.testing.assert_allclose(g["dWs"].sum(axis=1), 0.0, atol=1e-12 * np.abs(g["dWs"]).sum())
    assert np.abs(g["db"]).max() > 1e-3   # and the gradients are not trivially zero


def check_temperature_identity(o):
    """I9/I10: with per-head W_s, b, scale invariance of the logits gives
    tau_h dtau_h = -(<W_s^h, dW_s^h> + <b^h, db^h>), an identity independent of the direct
    sum -(1/tau) sum da a of App. F.2."""
    x, fx, Ws, b, tau, rng = _problem(B=2, N=25, H=3, D=4, V=3, G=6, seed=13, per_head=True)
    prm = _prm(O.MIX_ATTN, 6, 3, rng)
    R = rng.standard_normal(fx.shape)
    _, g = _loss_and_grads(o, x, fx, Ws, b, tau, O.MIX_ATTN, prm, R, 1e-2)
    lhs = tau * g["dtau"]
    rhs = -((Ws * g["dWs"]).sum(axis=(1, 2)) + (b * g["db"]).sum(axis=1))
    np.testing.assert_allclose(lhs, rhs, rtol=1e-10, atol=1e-13)
    assert np.abs(lhs).max() > 1e-4


def check_repeated_block(o):
    """forward_repeated (the full-size forward of a point set built from repeated copies of
    one block, evaluated from the block) against the plain forward on the explicitly tiled
    point set, at every point, for every mix."""
    for kind in MIXES:
        x, fx, Ws, b, tau, rng = _problem(B=2, N=11, H=2, D=4, V=3, G=5, seed=21 + kind)
        prm = _prm(kind, 5, 3, rng)
        rep = 3
        full = o.forward(np.tile(x, (1, rep, 1, 1)), np.tile(fx, (1, rep, 1, 1)), Ws, b, tau,
                         kind, prm, eps=0.05)
        pts = np.arange(11 * rep)
        r = o.forward_repeated(x, fx, Ws, b, tau, kind, prm, 0.05, rep, pts)
        for k in ("z", "s", "zmix", "lse", "out"):
            np.testing.assert_allclose(r[k], full[k], rtol=1e-12, atol=1e-13, err_msg=k)
        if kind == o.MIX_ATTN:
            np.testing.assert_allclose(r["P"], full["P"], rtol=1e-12, atol=1e-13)


def _untied_problem(seed, per_head=False, **kw):
    x, fx, Ws, b, tau, rng = _problem(seed=seed, per_head=per_head, **kw)
    Wd = rng.standard_normal(Ws.shape)
    bd = rng.standard_normal(b.shape)
    taud = rng.uniform(0.4, 1.5, size=tau.shape)
    return x, fx, Ws, b, tau, Wd, bd, taud, rng


def check_untied_finite_differences(o, kinds=tuple(MIXES)):
    """Untied variant: central differences of L = sum(O * R) in fp64 match every analytic
    gradient, both projections' included."""
    eps = 0.3
    for kind in kinds:
        x, fx, Ws, b, tau, Wd, bd, taud, rng = _untied_problem(
            40 + kind, B=2, N=5, H=2, D=3, V=2, G=4)
        prm = _prm(kind, 4, 2, rng)
        R = rng.standard_normal((2, 5, 2, 2))
        fwd = o.untied_forward(x, fx, Ws, b, tau, Wd, bd, taud, kind, prm, eps=eps)
        g = o.untied_backward(x, fx, Ws, b, tau, Wd, bd, taud, kind, prm, R, eps=eps, fwd=fwd)
        tensors = {"dx": x, "dfx": fx, "dWs": Ws, "db": b, "dtau": tau, "dWd": Wd, "dbd": bd,
                   "dtaud": taud}
        for k in ("A", "Wc", "Wq", "Wk", "Wv"):
            if prm.get(k) is not None:
                tensors["d" + k] = prm[k]
        step = 1e-6
        for gname, arr in tensors.items():
            num = np.zeros_like(arr)
            for idx in np.ndindex(arr.shape):
                old = arr[idx]
                vals = []
                for sgn in (1, -1):
                    arr[idx] = old + sgn * step
                    vals.append((o.untied_forward(x, fx, Ws, b, tau, Wd, bd, taud, kind, prm,
                                                  eps=eps)["out"] * R).sum())
                arr[idx] = old
                num[idx] = (vals[0] - vals[1]) / (2 * step)
            scale = max(np.abs(num).max(), 1e-3)
            err = np.abs(g[gname] - num).max() / scale
            assert err < 2e-7, (kind, gname, err)


def check_untied_reduces_to_tied(o):
    """With the deslice projection, bias and temperature equal to the slice's, the untied
    forward is the tied one, and each shared-parameter gradient of the tied path is the sum
    of its two untied parts (the parameter feeds both weight sets)."""
    for kind in (o.MIX_LINEAR_G, o.MIX_ATTN):
        x, fx, Ws, b, tau, rng = _problem(B=2, N=9, H=2, D=3, V=3, G=5, seed=60 + kind)
        prm = _prm(kind, 5, 3, rng)
        R = rng.standard_normal(fx.shape)
        ut = o.untied_forward(x, fx, Ws, b, tau, Ws, b, tau, kind, prm, eps=0.1)
        t = o.forward(x, fx, Ws, b, tau, kind, prm, eps=0.1)
        for k in ("z", "s", "zmix", "lse", "out"):
            np.testing.assert_allclose(ut[k], t[k], rtol=1e-12, atol=1e-14, err_msg=k)
        np.testing.assert_allclose(ut["lse_d"], t["lse"], rtol=1e-12, atol=1e-14)
        gu = o.untied_backward(x, fx, Ws, b, tau, Ws, b, tau, kind, prm, R, eps=0.1, fwd=ut)
        gt = o.backward(x, fx, Ws, b, tau, kind, prm, R, eps=0.1, fwd=t)
        for k in ("dx", "dfx", "dzmix"):
            np.testing.assert_allclose(gu[k], gt[k], rtol=1e-11, atol=1e-13, err_msg=k)
        for k, kd in (("dWs", "dWd"), ("db", "dbd"), ("dtau", "dtaud")):
            np.testing.assert_allclose(gu[k] + gu[kd], gt[k], rtol=1e-11, atol=1e-13, err_msg=k)
            # and the split is not trivial: both parts carry gradient
            assert np.abs(gu[k]).max() > 1e-6 and np.abs(gu[kd]).max() > 1e-6


def check_untied_cancellation_and_temperature(o):
    """Each weight set's logit gradient cancels over the slots (sum_g db = sum_g db_d = 0,
    likewise the projection rows), and the scale invariance of each logit set gives
    tau dtau = -(<W, dW> + <b, db>) per head for both (App. F.2)."""
    x, fx, Ws, b, tau, Wd, bd, taud, rng = _untied_problem(
        70, per_head=True, B=2, N=20, H=3, D=4, V=3, G=6)
    prm = _prm(o.MIX_LINEAR_C, 6, 3, rng)
    R = rng.standard_normal(fx.shape)
    g = o.untied_backward(x, fx, Ws, b, tau, Wd, bd, taud, o.MIX_LINEAR_C, prm, R, eps=1e-2)
    for kW, kb, W_, b_, t_, kt in (("dWs", "db", Ws, b, tau, "dtau"),
                                   ("dWd", "dbd", Wd, bd, taud, "dtaud")):
        np.testing.assert_allclose(g[kb].sum(axis=-1), 0.0, atol=1e-12 * np.abs(g[kb]).sum())
        np.testing.assert_allclose(g[kW].sum(axis=-1), 0.0, atol=1e-12 * np.abs(g[kW]).sum())
        lhs = t_ * g[kt]
        rhs = -((W_ * g[kW]).sum(axis=(1, 2)) + (b_ * g[kb]).sum(axis=1))
        np.testing.assert_allclose(lhs, rhs, rtol=1e-10, atol=1e-13)
        assert np.abs(lhs).max() > 1e-5


def check_linearno_finite_differences(o, kinds=(MIXES[1], MIXES[2], MIXES[3])):
    """LinearNO: central differences of L = sum(O * R) in fp64 match every analytic
    gradient."""
    for kind in kinds:
        x, fx, Ws, b, tau, Wd, bd, taud, rng = _untied_problem(
            80 + kind, B=2, N=5, H=2, D=3, V=2, G=4)
        prm = _prm(kind, 4, 2, rng)
        R = rng.standard_normal((2, 5, 2, 2))
        fwd = o.linearno_forward(x, fx, Ws, b, tau, Wd, bd, taud, kind, prm)
        g = o.linearno_backward(x, fx, Ws, b, tau, Wd, bd, taud, kind, prm, R, fwd=fwd)
        tensors = {"dx": x, "dfx": fx, "dWs": Ws, "db": b, "dtau": tau, "dWd": Wd, "dbd": bd,
                   "dtaud": taud}
        for k in ("A", "Wc", "Wq", "Wk", "Wv"):
            if prm.get(k) is not None:
                tensors["d" + k] = prm[k]
        step = 1e-6
        for gname, arr in tensors.items():
            num = np.zeros_like(arr)
            for idx in np.ndindex(arr.shape):
                old = arr[idx]
                vals = []
                for sgn in (1, -1):
                    arr[idx] = old + sgn * step
                    vals.append((o.linearno_forward(x, fx, Ws, b, tau, Wd, bd, taud, kind,
                                                    prm)["out"] * R).sum())
                arr[idx] = old
                num[idx] = (vals[0] - vals[1]) / (2 * step)
            # the slice bias gradient is identically zero here: gate it by rounding noise
            scale = max(np.abs(num).max(), 1e-2)
            err = np.abs(g[gname] - num).max() / scale
            assert err < 2e-7, (kind, gname, err)


def check_linearno_closed_forms(o):
    """LinearNO's slice weights are a partition of unity over the points of each slot: they
    sum to one per slot, zero logits give every slot the plain mean of F, one dominant point
    per slot (hard assignment) gives that point's F, and a constant added to one slot's
    logits changes nothing (so the slice bias gets no gradient)."""
    x, fx, Ws, b, tau, Wd, bd, taud, rng = _untied_problem(90, B=2, N=12, H=2, D=3, V=2, G=4)
    kind = o.MIX_IDENTITY
    a = rng.standard_normal((12, 4)) * 3
    k, lse = o.point_softmax(a)
    np.testing.assert_allclose(k.sum(axis=0), 1.0, atol=1e-13)
    np.testing.assert_allclose(k, np.exp(a - lse[None, :]), rtol=1e-12)
    r = o.linearno_forward(x, fx, np.zeros_like(Ws), np.zeros_like(b), tau, Wd, bd, taud, kind)
    np.testing.assert_allclose(r["z"], np.broadcast_to(fx.mean(axis=1)[:, :, None, :],
                                                       r["z"].shape), rtol=1e-12, atol=1e-14)
    # hard assignment: slot g's logit is huge only at point g (D = G, X = identity rows)
    X = np.zeros((1, 12, 1, 4))
    for g in range(4):
        X[0, 3 * g, 0, g] = 1.0
    F = rng.standard_normal((1, 12, 1, 2))
    r = o.linearno_forward(X, F, 200.0 * np.eye(4), np.zeros(4), np.ones(1), np.eye(4),
                           np.zeros(4), np.ones(1), kind)
    np.testing.assert_allclose(r["z"][0, 0], F[0, [0, 3, 6, 9], 0], rtol=1e-10)
    # per-slot constant shift of the logits: no change, hence db = 0
    r1 = o.linearno_forward(x, fx, Ws, b, tau, Wd, bd, taud, kind)
    r2 = o.linearno_forward(x, fx, Ws, b + np.arange(4.0), tau, Wd, bd, taud, kind)
    np.testing.assert_allclose(r1["out"], r2["out"], rtol=1e-12, atol=1e-14)
    R = rng.standard_normal(fx.shape)
    gr = o.linearno_backward(x, fx, Ws, b, tau, Wd, bd, taud, o.MIX_LINEAR_C,
                             _prm(o.MIX_LINEAR_C, 4, 2, rng), R)
    assert np.abs(gr["db"]).max() < 1e-12 * max(1.0, np.abs(gr["dWs"]).max())
    assert np.abs(gr["dWs"]).max() > 1e-4
    # temperature identity (scale invariance of the slice logits), summed over the heads
    # that share W_s and b: sum_h tau_h dtau_h = -(<W_s, dW_s> + <b, db>)
    lhs = (tau * gr["dtau"]).sum()
    np.testing.assert_allclose(lhs, -((Ws * gr["dWs"]).sum() + (b * gr["db"]).sum()),
                               rtol=1e-10, atol=1e-13)
    assert abs(lhs) > 1e-5


ALL_CHECKS = [check_partition_of_unity, check_single_slice_mean, check_identical_points,
              check_constant_tokens, check_zero_logits, check_hard_assignment,
              check_bruteforce, check_invariances, check_mix_closed_forms,
              check_finite_differences, check_cancellation, check_temperature_identity,
              check_repeated_block, check_untied_finite_differences,
              check_untied_reduces_to_tied, check_untied_cancellation_and_temperature,
              check_linearno_finite_differences, check_linearno_closed_forms]


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda c: c.__name__)
def test_pin(check):
    check(O)


def test_finite_differences_per_head():
    check_finite_differences(O, kinds=(O.MIX_LINEAR_G,), per_head=True)


# ----------------------------------------------------------------------------------------
# planted mistakes: each must make at least one check fail
# ----------------------------------------------------------------------------------------
def _mutant(**overrides):
    m = types.ModuleType("oracle_mutant")
    m.__dict__.update({k: v for k, v in O.__dict__.items() if not k.startswith("__")})
    m.__dict__.update(overrides)
    # re-bind the module-level drivers so they call the planted functions
    for name in ("forward", "backward", "untied_forward", "untied_backward",
                 "forward_repeated", "linearno_forward", "linearno_backward"):
        f = O.__dict__[name]
        m.__dict__[name] = types.FunctionType(f.__code__, m.__dict__, name, f.__defaults__)
    return m


def _mut_no_eps(w, F, eps):
    s = w.sum(axis=0)
    U = w.T @ F
    return s, U, U / s[:, None]


def _mut_bias_outside(X, Ws, b, tau):
    return X @ Ws / tau + b[None, :]


def _mut_AT(kind, z, p):
    if kind == O.MIX_LINEAR_G:
        return p["A"].T @ z, None
    return O.mix_forward(kind, z, p)


def _mut_no_scale(kind, z, p):
    if kind == O.MIX_ATTN:
        p = dict(p, scale=1.0)
    return O.mix_forward(kind, z, p)


def _mut_point_softmax(a):   # normalise over points instead of slices
    e = np.exp(a - a.max(axis=0, keepdims=True))
    w = e / e.sum(axis=0, keepdims=True)
    return w, np.log(np.exp(a).sum(axis=1))


def _mut_no_ds(dO, zm, F, dU, ds):
    return dO @ zm.T + F @ dU.T


def _mut_softmax_sign(w, dw):
    return w * (dw + (w * dw).sum(axis=1, keepdims=True))


def _mut_dtau_sign(da, X, Ws, a, tau):
    dX, dWs, db, dtau = O.logit_backward(da, X, Ws, a, tau)
    return dX, dWs, db, -dtau


def _mut_dX_no_tau(da, X, Ws, a, tau):
    dX, dWs, db, dtau = O.logit_backward(da, X, Ws, a, tau)
    return dX * tau, dWs, db, dtau


def _mut_mixbwd_A(kind, z, P, dzm, p):
    if kind == O.MIX_LINEAR_G:
        return p["A"] @ dzm, {"dA": dzm @ z.T}
    return O.mix_backward(kind, z, P, dzm, p)


def _mut_token_bwd_sign(dz, z, s, eps):
    inv = 1.0 / (s + eps)
    return dz * inv[:, None], (dz * z).sum(axis=1) * inv


def _mut_deslice_unmixed(w, zm):
    return w @ (zm * 0.5 + 0.5 * zm[::-1])   # mixes the wrong tokens


def _mut_point_softmax_bwd(k, dk):   # the per-slot correction dropped
    return k * dk


def _mut_point_softmax_slots(a):     # LinearNO weights normalised over the slots instead
    return O.slot_softmax(a)


MUTANTS = {
    "dropped eps": dict(slice_tokens=_mut_no_eps),
    "bias not divided by tau": dict(logits=_mut_bias_outside),
    "transposed fixed token matrix": dict(mix_forward=_mut_AT),
    "attention scale dropped": dict(mix_forward=_mut_no_scale),
    "softmax over points": dict(slot_softmax=_mut_point_softmax),
    "weight-sum gradient dropped": dict(weight_grad=_mut_no_ds),
    "softmax backward sign": dict(softmax_backward=_mut_softmax_sign),
    "temperature gradient sign": dict(logit_backward=_mut_dtau_sign),
    "dX missing 1/tau": dict(logit_backward=_mut_dX_no_tau),
    "mix backward not transposed": dict(mix_backward=_mut_mixbwd_A),
    "token backward sign": dict(token_backward=_mut_token_bwd_sign),
    "deslice of the wrong tokens": dict(deslice=_mut_deslice_unmixed),
    "LinearNO slice correction dropped": dict(point_softmax_backward=_mut_point_softmax_bwd),
    "LinearNO weights over the slots": dict(point_softmax=_mut_point_softmax_slots),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes(name):
    m = _mutant(**MUTANTS[name])
    failed = []
    for check in ALL_CHECKS:
        try:
            if check is check_finite_differences:
                check(m, kinds=(O.MIX_LINEAR_G, O.MIX_ATTN))
            else:
                check(m)
        except (AssertionError, ValueError, FloatingPointError):
            failed.append(check.__name__)
    assert failed, f"no pin caught the planted mistake: {name}"
