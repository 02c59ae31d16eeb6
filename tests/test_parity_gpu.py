"""Parity of the HIP path against the fp64 oracle (needs an MI355X).

Every output and gradient is compared with the oracle both normwise and element by element
(tests/paritycheck.py): the normwise error ||gpu - oracle||_2 / ||oracle||_2 and the largest
per-element error |gpu - oracle| / max(|oracle|, KAPPA rms(oracle)) must both be at most
1e-5 for fp32 storage and 2e-2 for bf16 storage (fp32 accumulation in both). The oracle gets
exactly the values the GPU reads (bf16 inputs are upcast exactly). Sizes span several point
tiles with a ragged tail, B > 1, every head width and slot count the library supports, and
every token mix.
"""
import sys

import numpy as np
import pytest

import oracle as O
import workloads as W
from paritycheck import KAPPA, TOL, Checker, announce, eager_gate, measures, oracle_pairs

pytestmark = pytest.mark.gpu

FWD_KEYS = ("z", "s", "zmix", "lse", "out")
BWD_KEYS = ("dx", "dfx", "dWs", "db", "dtau", "dzmix")
MIX_PARAM_KEYS = {O.MIX_LINEAR_G: ("dA",), O.MIX_LINEAR_C: ("dWc",),
                  O.MIX_ATTN: ("dWq", "dWk", "dWv"), O.MIX_IDENTITY: ()}


def rel(a, b):
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / nb) if nb > 0 else float(np.linalg.norm(a))


LN2 = float(np.log(2.0))


def run_gpu(w, inp, backward=True):
    """Runs forward + backward; lse is converted from the library's base-2 unit to the
    oracle's natural log for comparison."""
    from paper_2609_32525_amd.runner import PathBuffers
    pb = PathBuffers(inp, w.mix, w.dtype, w.eps, with_backward=backward)
    pb.step()
    r = pb.results()
    r["lse"] = r["lse"] * LN2
    return pb, r


def compare(w, inp, got, tol=None, backward=True, ref=None):
    """Every output of the path (and the attention probabilities) against the oracle."""
    fwd, bwd = ref if ref is not None else O.run_inputs(inp, w.mix, w.eps, backward_too=backward)
    keys = list(FWD_KEYS) + (list(BWD_KEYS) + list(MIX_PARAM_KEYS[w.mix]) if backward else [])
    if w.mix == O.MIX_ATTN:
        keys.append("P")
    c = Checker(f"tied/{w.name}", w.dtype, tol)
    for k in keys:
        r = bwd[k] if (bwd is not None and k in bwd) else fwd[k]
        c.add(k, got[k], r, keep=False)
    c.finish()
    return c.rows


def small(name, dtype, D, G, mix, B=2, N=1000, H=3, **kw):
    base = W.Workload(name, 100 + G + D + mix, dtype, B, N, H, D, D, G, mix, **kw)
    return base


SMALL = [
    small("f32_D32_G32_attn", "f32", 32, 32, O.MIX_ATTN),
    small("f32_D16_G16_lin", "f32", 16, 16, O.MIX_LINEAR_G),
    small("f32_D16_G32_lin", "f32", 16, 32, O.MIX_LINEAR_G),
    small("f32_D32_G64_linc", "f32", 32, 64, O.MIX_LINEAR_C),
    small("f32_D64_G32_id", "f32", 64, 32, O.MIX_IDENTITY),
    small("f32_D32_G128_lin", "f32", 32, 128, O.MIX_LINEAR_G),
    small("f32_D32_G256_attn", "f32", 32, 256, O.MIX_ATTN, N=700),
    small("f32_D32_G512_lin", "f32", 32, 512, O.MIX_LINEAR_G, N=700, H=2),
    small("f32_D32_G1024_lin", "f32", 32, 1024, O.MIX_LINEAR_G, N=600, H=2, B=1),
    small("f32_D64_G128_lin_ph", "f32", 64, 128, O.MIX_LINEAR_G, ws_per_head=True,
          a_per_head=True),
    small("bf16_D32_G32_attn", "bf16", 32, 32, O.MIX_ATTN),
    small("bf16_D16_G64_lin", "bf16", 16, 64, O.MIX_LINEAR_G),
    small("bf16_D32_G64_lin", "bf16", 32, 64, O.MIX_LINEAR_G),
    small("bf16_D64_G64_linc", "bf16", 64, 64, O.MIX_LINEAR_C),
    small("bf16_D32_G128_lin", "bf16", 32, 128, O.MIX_LINEAR_G, tau_mode="uniform",
          ws_mode="std3"),
    small("bf16_D32_G256_lin", "bf16", 32, 256, O.MIX_LINEAR_G, tau_mode="uniform",
          ws_mode="std3", N=900),
    small("bf16_D32_G512_lin", "bf16", 32, 512, O.MIX_LINEAR_G, tau_mode="uniform",
          ws_mode="std3", N=800, H=2),
    small("bf16_D32_G1024_lin", "bf16", 32, 1024, O.MIX_LINEAR_G, tau_mode="uniform",
          ws_mode="std3", N=700, H=2, B=1),
    # large token sets with every mix kind, and dh = 64 beyond G = 128
    small("f32_D32_G512_linc", "f32", 32, 512, O.MIX_LINEAR_C, N=600, H=2),
    small("f32_D16_G1024_id", "f32", 16, 1024, O.MIX_IDENTITY, N=500, H=2, B=1),
    small("bf16_D64_G256_lin", "bf16", 64, 256, O.MIX_LINEAR_G, N=600, H=2),
    small("bf16_D32_G256_attn", "bf16", 32, 256, O.MIX_ATTN, N=600, H=2),
    # attention over large token sets inside the whole path
    small("f32_D32_G1024_attn", "f32", 32, 1024, O.MIX_ATTN, N=600, H=2, B=1),
    small("bf16_D64_G512_attn", "bf16", 64, 512, O.MIX_ATTN, N=600, H=2),
    # slot counts between the tile sizes (padded tilings): one padded wave (G = 16 in bf16,
    # 48), two slot waves (80, 112), slot blocks with a partial last block (144, 336, 1008),
    # cooperative waves with no real slot at all (272 and 336 run on 8 slot waves)
    small("bf16_D32_G16_lin", "bf16", 32, 16, O.MIX_LINEAR_G, N=777),
    small("f32_D32_G48_attn", "f32", 32, 48, O.MIX_ATTN),
    small("bf16_D32_G48_lin", "bf16", 32, 48, O.MIX_LINEAR_G, N=1031),
    small("f32_D16_G80_linc", "f32", 16, 80, O.MIX_LINEAR_C),
    small("bf16_D64_G112_attn", "bf16", 64, 112, O.MIX_ATTN, N=900),
    small("bf16_D32_G144_lin", "bf16", 32, 144, O.MIX_LINEAR_G, tau_mode="uniform",
          ws_mode="std3", N=900),
    small("f32_D32_G336_attn", "f32", 32, 336, O.MIX_ATTN, N=700, H=2),
    small("bf16_D64_G272_lin", "bf16", 64, 272, O.MIX_LINEAR_G, N=600, H=2),
    small("bf16_D32_G1008_lin", "bf16", 32, 1008, O.MIX_LINEAR_G, tau_mode="uniform",
          ws_mode="std3", N=700, H=2, B=1),
    small("f32_D32_G48_lin_N33", "f32", 32, 48, O.MIX_LINEAR_G, N=33),
    # head width 64 in the slot-blocked family (bf16): streamed statistics images, 4-wave
    # point-owned pass; a partial last block; a ragged tail
    small("bf16_D64_G1024_lin", "bf16", 64, 1024, O.MIX_LINEAR_G, tau_mode="uniform",
          ws_mode="std3", N=500, H=2, B=1),
    small("bf16_D64_G176_linc", "bf16", 64, 176, O.MIX_LINEAR_C, N=700, H=2),
    small("bf16_D64_G256_lin_N33", "bf16", 64, 256, O.MIX_LINEAR_G, N=33, H=2),
    # head width 64 takes the slot-blocked family from 80 slots: two whole 64-slot blocks
    small("bf16_D64_G128_lin", "bf16", 64, 128, O.MIX_LINEAR_G, N=900, H=2),
]


@pytest.mark.parametrize("w", SMALL, ids=lambda w: w.name)
def test_parity_small(w):
    announce(f"small {w}")
    inp = W.make_inputs(w)
    _, got = run_gpu(w, inp)
    compare(w, inp, got)


@pytest.mark.parametrize("N", [0, 1, 31, 33, 129])
def test_edge_point_counts(N):
    w = small(f"edge_N{N}", "f32", 32, 32, O.MIX_LINEAR_G, N=N, B=2, H=2)
    announce(f"edge N={N}")
    inp = W.make_inputs(w)
    _, got = run_gpu(w, inp)
    if N == 0:
        # no points: s = 0, z = 0 / eps = 0, every gradient 0
        assert np.all(got["s"] == 0) and np.all(got["z"] == 0)
        for k in ("dWs", "db", "dtau", "dzmix"):
            assert np.all(got[k] == 0), k
        return
    compare(w, inp, got)


@pytest.mark.parametrize("N,dtype,G", [(0, "bf16", 1024), (1, "bf16", 256), (33, "f32", 512),
                                       (129, "bf16", 128), (1, "f32", 1024)],
                         ids=["N0_bf16_G1024", "N1_bf16_G256", "N33_f32_G512",
                              "N129_bf16_G128", "N1_f32_G1024"])
def test_edge_point_counts_large_g(N, dtype, G):
    """Empty, single-point and one-tile-plus-one point sets on the G = 128 family and the
    slot-blocked family (statistics pass, slot-owned and point-owned passes)."""
    w = small(f"edge_N{N}_{dtype}_G{G}", dtype, 32, G, O.MIX_LINEAR_G, N=N, B=2, H=2)
    announce(f"edge N={N} {dtype} G={G}")
    inp = W.make_inputs(w)
    _, got = run_gpu(w, inp)
    if N == 0:
        assert np.all(got["s"] == 0) and np.all(got["z"] == 0)
        for k in ("dWs", "db", "dtau", "dzmix"):
            assert np.all(got[k] == 0), k
        return
    compare(w, inp, got)


# At logits of order 2000 (temperature 0.05, beyond the paper's trained models, whose logits
# are of order 10) the fp32 kernels carry two roundings per logit where plain fp32 carries
# one: the projection pre-scaled by log2(e)/tau and the product itself. The logit gradient
# then reaches 2-3 times the plain-fp32 error through the softmax Jacobian; these outputs of
# that case take a 3x normwise gate (5x on the largest element), every other output the
# paper's rule. The element-wise gate compares the largest per-element errors of two
# rounding patterns, a noisier statistic than the norm: it admits 3x plain fp32.
EXTREME_3X = ("dx", "dWs", "db")


@pytest.mark.parametrize("scale,taus", [(3.0, (0.1, 0.5, 2.0)), (30.0, (0.05, 0.5, 2.0))],
                         ids=["logits~100", "logits~2000"])
def test_peaky_and_tiny_temperature(scale, taus):
    """Logits in the hundreds or thousands (the max shift must prevent overflow) with a tiny
    temperature. fp32 logits then carry absolute rounding errors the softmax amplifies, so
    beside the 1e-5 bound the paper's acceptance rule applies (App. F.2): the error may reach
    1.25x that of evaluating the same definition in plain fp32 (3x when that exceeds 1e-4),
    normwise and element-wise alike."""
    w = small("peaky", "f32", 32, 64, O.MIX_LINEAR_G, N=500)
    inp = W.make_inputs(w)
    inp["Ws"] = inp["Ws"] * scale
    inp["tau"] = np.array(taus, dtype=np.float32)
    announce(f"peaky logits scale={scale} taus={taus}")
    _, got = run_gpu(w, inp)
    for k in ("z", "out", "dx", "dfx", "dWs", "db", "dtau"):
        assert np.isfinite(got[k]).all(), k
    f64, b64 = O.run_inputs(inp, w.mix, w.eps)
    f32, b32 = O.run_inputs(inp, w.mix, w.eps, dtype=np.float32)
    bad = {}
    for k in FWD_KEYS + BWD_KEYS + ("dA",):
        ref, eag = (b64[k], b32[k]) if k in b64 else (f64[k], f32[k])
        en, ee = measures(eag, ref, KAPPA["f32"])
        gn, ge = max(1e-5, eager_gate(en)), max(1e-5, 3.0 * ee)
        if scale > 10 and k in EXTREME_3X:
            gn, ge = max(gn, 3.0 * en), max(ge, 5.0 * ee)
        n, e = measures(got[k], ref, KAPPA["f32"])
        print(f"  {k}: fused {n:.2e}/{e:.2e} fp32-eager {en:.2e}/{ee:.2e} "
              f"gate {gn:.2e}/{ge:.2e} (norm/elem)", flush=True)
        if not (n <= gn and e <= ge):
            bad[k] = (n, e, gn, ge)
    assert not bad, bad


def test_determinism_bitwise():
    w = small("det", "bf16", 32, 128, O.MIX_LINEAR_G, N=3000)
    inp = W.make_inputs(w)
    announce("determinism")
    from paper_2609_32525_amd.runner import PathBuffers
    pb = PathBuffers(inp, w.mix, w.dtype, w.eps)
    pb.step()
    a = pb.results()
    pb.step()
    b = pb.results()
    for k, v in a.items():
        if v is not None:
            assert np.array_equal(v, b[k]), k


def test_two_shard_combine():
    """Point sharding (design only across GPUs): slicing two disjoint halves and combining
    U_i = z_i (s_i + eps), s_i matches slicing all points, within fp32 summation order."""
    w = small("shard", "f32", 32, 32, O.MIX_IDENTITY, N=2000, B=1, H=2, eps=1e-3)
    inp = W.make_inputs(w, with_grad=False)
    announce("two-shard combine")
    from paper_2609_32525_amd.runner import PathBuffers
    full = PathBuffers(inp, w.mix, w.dtype, w.eps, with_backward=False)
    full.step()
    rf = full.results()
    parts = []
    for sl in (slice(0, 1200), slice(1200, 2000)):
        sub = dict(inp)
        sub["x"] = inp["x"][:, sl]
        sub["fx"] = inp["fx"][:, sl]
        pb = PathBuffers(sub, w.mix, w.dtype, w.eps, with_backward=False)
        pb.step()
        parts.append(pb.results())
    s = parts[0]["s"] + parts[1]["s"]
    U = sum(p["z"] * (p["s"] + w.eps)[..., None] for p in parts)
    z = U / (s + w.eps)[..., None]
    ns, es = measures(s, rf["s"], KAPPA["f32"])
    nz, ez = measures(z, rf["z"], KAPPA["f32"])
    assert ns < 1e-6 and es < 1e-5, (ns, es)
    assert nz < 1e-5 and ez < 1e-5, (nz, ez)


@pytest.mark.parametrize("G", [32, 128, 256, 1024])
def test_no_nxg_allocation(G):
    """The library allocates nothing: the torch allocator sees only the caller's buffers,
    and the workspace stays far below one slice-weight tensor, for the cooperative kernels
    (G <= 128) and the slot-blocked ones."""
    import torch
    w = W.WORKLOADS["stress1024"].scaled(N=1 << 16, G=G)
    inp = W.make_inputs(w)
    announce("memory")
    from paper_2609_32525_amd.runner import PathBuffers
    pb = PathBuffers(inp, w.mix, w.dtype, w.eps)
    torch.cuda.synchronize()
    before = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    pb.step()
    torch.cuda.synchronize()
    assert torch.cuda.max_memory_allocated() == before
    wbytes = w.B * w.N * w.H * w.G * 4
    assert pb.ws_f.numel() + pb.ws_b.numel() < wbytes / 8


@pytest.mark.parametrize("dtype,G", [("f32", 32), ("bf16", 64), ("bf16", 256)])
def test_non_finite_inputs_propagate(dtype, G):
    """A NaN in one point's slice features (head 1), or an infinity in one point's values
    (head 0), makes exactly the outputs non-finite that it makes non-finite in the oracle: no
    kernel drops a non-finite value or invents one. The head that never sees it stays finite
    and within the parity bar."""
    for case, bad, clean in (("nan_x", 1, 0), ("inf_fx", 0, 1)):
        w = small(f"nonfinite_{case}_{dtype}_G{G}", dtype, 32, G, O.MIX_LINEAR_G, N=300, B=1,
                  H=2)
        announce(f"non-finite {case} {w}")
        inp = W.make_inputs(w)
        if case == "nan_x":
            inp["x"][0, 17, bad, 3] = np.nan
        else:
            inp["fx"][0, 41, bad, 5] = np.inf
        _, got = run_gpu(w, inp)
        with np.errstate(all="ignore"):
            fwd, bwd = O.run_inputs(inp, w.mix, w.eps)
        for k in ("z", "zmix", "lse", "out", "dx", "dfx", "dzmix", "dWs", "db", "dtau"):
            ref = bwd[k] if k in bwd else fwd[k]
            assert (~np.isfinite(ref)).any() or k in ("lse", "dfx", "dzmix"), (case, k)
            assert np.array_equal(np.isfinite(got[k]), np.isfinite(ref)), (case, k)
        c = Checker(f"nonfinite/{w.name}", dtype)
        for k in ("z", "zmix", "lse", "dzmix"):
            ref = bwd[k] if k in bwd else fwd[k]
            c.add(f"{k}[h{clean}]", got[k][0, clean], ref[0, clean], keep=False)
        for k in ("out", "dx", "dfx"):
            ref = bwd[k] if k in bwd else fwd[k]
            c.add(f"{k}[h{clean}]", got[k][0, :, clean], ref[0, :, clean], keep=False)
        c.add(f"dtau[h{clean}]", got["dtau"][clean], bwd["dtau"][clean], keep=False)
        c.finish()


# ---- the benchmark workloads at full size ---------------------------------------------------
# The GPU runs every (sample, head) in the launch configuration the benchmark times. For the
# workloads marked None the fp64 oracle recomputes every pair (pairs run side by side), so
# every output and every parameter gradient is compared element by element at full size; for
# the large-G ones it recomputes the listed pairs (every output of those pairs, at every
# point), and properties that hold at any size check the rest.
FULL = {"tiny": None, "surface": None, "stack": None, "volume": None,
        "stress128": [(0, 2)], "stress256": [(0, 6)], "stress512": [(0, 1)],
        "stress1024": [(0, 7)], "attn1024": [(0, 4)]}
PER_PAIR = ("z", "s", "zmix", "lse", "out", "dx", "dfx", "dzmix")


@pytest.mark.parametrize("name", list(FULL))
def test_parity_full_size(name):
    w = W.WORKLOADS[name]
    pairs = FULL[name]
    announce(f"full {w} pairs={pairs or 'all'}")
    inp = W.make_inputs(w)
    _, got = run_gpu(w, inp)
    # properties over all pairs: every point's weights sum to one, so the slot sums add up
    # to N; the logit gradient cancels per point, so the bias and projection gradients sum to
    # zero over the slots (App. F.2)
    np.testing.assert_allclose(got["s"].sum(-1), w.N, rtol=1e-5)
    assert abs(got["db"].sum()) <= 1e-4 * np.abs(got["db"]).sum()
    # dW_s contracts bf16-rounded logit gradients in bf16 storage, so its slot sums cancel
    # only to the bf16 rounding level there
    cancel = 2e-3 if w.dtype == "bf16" else 1e-4
    assert np.all(np.abs(got["dWs"].sum(-1)) <= cancel * np.abs(got["dWs"]).sum(-1))
    for k in ("out", "dx", "dfx", "dWs", "db", "dtau"):
        assert np.isfinite(got[k]).all(), k
    print(f"  oracle on {'all pairs' if pairs is None else pairs}", flush=True)
    fwd, bwd = oracle_pairs(O, inp, w.mix, w.eps, pairs=pairs)
    if pairs is None:
        compare(w, inp, got, ref=(fwd, bwd))
        return
    c = Checker(f"tied/{name}", w.dtype)
    for bb, h in pairs:
        for k in PER_PAIR:
            ref = bwd[k] if k in bwd else fwd[k]
            if k in ("out", "dx", "dfx"):
                c.add(f"{k}[{bb},{h}]", got[k][bb, :, h], ref[bb, :, h], keep=False)
            else:
                c.add(f"{k}[{bb},{h}]", got[k][bb, h], ref[bb, h], keep=False)
        if w.B == 1:   # the temperature gradient of head h comes from this pair alone
            c.add(f"dtau[{h}]", got["dtau"][h], bwd["dtau"][h], keep=False)
    c.finish()


# ---- the standalone token-mix entry points (fs_mix, fs_mix_bwd) -----------------------------
MIX_CASES = [
    ("identity", O.MIX_IDENTITY, 32, False), ("identity", O.MIX_IDENTITY, 1024, False),
    ("fixed", O.MIX_LINEAR_G, 32, False), ("fixed", O.MIX_LINEAR_G, 512, False),
    ("fixed_per_head", O.MIX_LINEAR_G, 64, True), ("fixed_per_head", O.MIX_LINEAR_G, 256, True),
    ("channel", O.MIX_LINEAR_C, 32, False), ("channel", O.MIX_LINEAR_C, 512, False),
    ("attention", O.MIX_ATTN, 32, False), ("attention", O.MIX_ATTN, 128, False),
    # attention over large token sets (the row-block forward and the batched-product backward)
    ("attention", O.MIX_ATTN, 512, False), ("attention", O.MIX_ATTN, 1024, False),
    ("attention_v64", O.MIX_ATTN, 256, False, 64), ("attention_v16", O.MIX_ATTN, 1024, False, 16),
    # token counts that are multiples of 16 but not of 64
    ("fixed", O.MIX_LINEAR_G, 48, False), ("channel", O.MIX_LINEAR_C, 336, False),
    ("attention", O.MIX_ATTN, 48, False), ("attention", O.MIX_ATTN, 80, False),
    ("attention", O.MIX_ATTN, 336, False),
]


@pytest.mark.parametrize("label,kind,G,per_head,V", [c if len(c) == 5 else c + (32,)
                                                     for c in MIX_CASES],
                         ids=[f"{c[0]}_G{c[2]}" for c in MIX_CASES])
def test_mix_entry_points(label, kind, G, per_head, V):
    """fs_mix and fs_mix_bwd on their own (both the single-workgroup LDS kernels and the
    batched products for large token sets) against the oracle's mix steps, per (b, h); the
    parameter gradients are summed over samples and heads (over samples per head for a
    per-head matrix)."""
    import torch
    import paper_2609_32525_amd as fs
    B, H = 2, 3
    w = W.Workload(f"mix_{label}", 300 + kind, "f32", B, 64, H, V, V, G, kind, a_per_head=per_head)
    inp = W.make_inputs(w, with_grad=False)
    z = W.random_like(w, 1, (B, H, G, V))
    dzm = W.random_like(w, 2, (B, H, G, V))
    announce(f"mix {label} G={G}")
    dev = torch.device("cuda:0")
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
    prob = fs.Problem.make(B, 64, H, V, V, G, fs.F32, 1e-5)
    prm = {k: up(inp[k]) for k in ("A", "Wc", "Wq", "Wk", "Wv") if inp.get(k) is not None}
    md = fs.MixDesc.make(kind, A=prm.get("A"), Wc=prm.get("Wc"), Wq=prm.get("Wq"),
                         Wk=prm.get("Wk"), Wv=prm.get("Wv"), scale=float(inp["scale"]),
                         a_per_head=1 if per_head else 0)
    zt, dzt = up(z), up(dzm)
    zmix = torch.empty_like(zt)
    attn = torch.empty((B, H, G, G), device=dev) if kind == O.MIX_ATTN else None
    fs.mix(prob, md, zt, zmix, attn)
    dz = torch.empty_like(zt)
    npar = {O.MIX_IDENTITY: 0, O.MIX_LINEAR_G: (H if per_head else 1) * G * G,
            O.MIX_LINEAR_C: V * V, O.MIX_ATTN: 3 * V * V}[kind]
    dmix = torch.empty(max(npar, 1), device=dev)
    ws = torch.empty(fs.workspace_bytes(prob, True), device=dev, dtype=torch.uint8)
    fs.mix_bwd(prob, md, zt, attn, dzt, dz, dmix if npar else None, ws)
    torch.cuda.synchronize()
    got_zm, got_dz = zmix.double().cpu().numpy(), dz.double().cpu().numpy()
    ref_zm, ref_dz, ref_P = np.zeros_like(got_zm), np.zeros_like(got_dz), []
    ref_par = {}
    prm_np = {k: inp[k] for k in ("A", "Wc", "Wq", "Wk", "Wv", "scale")}
    for b in range(B):
        for h in range(H):
            p = O._head_params(kind, prm_np, h)
            zbh = z[b, h].astype(np.float64)
            zm, P = O.mix_forward(kind, zbh, p)
            ref_zm[b, h] = zm
            d, dp = O.mix_backward(kind, zbh, P, dzm[b, h].astype(np.float64), p)
            ref_dz[b, h] = d
            if P is not None:
                ref_P.append(P)
            for k, v in dp.items():
                if k == "dA" and per_head:
                    ref_par.setdefault(k, np.zeros((H, G, G)))[h] += v
                else:
                    ref_par[k] = ref_par.get(k, 0) + v
    c = Checker(f"mix/{label}_G{G}", "f32")
    c.add("zmix", got_zm, ref_zm, keep=False)
    c.add("dz", got_dz, ref_dz, keep=False)
    if kind == O.MIX_ATTN:
        c.add("P", attn.double().cpu().numpy().reshape(-1, G, G), np.stack(ref_P), keep=False)
    if npar:
        d = dmix.double().cpu().numpy()
        if kind == O.MIX_ATTN:
            for n, k in enumerate(("dWq", "dWk", "dWv")):
                c.add(k, d[n * V * V:(n + 1) * V * V].reshape(V, V), ref_par[k], keep=False)
        else:
            k = "dA" if kind == O.MIX_LINEAR_G else "dWc"
            c.add(k, d.reshape(ref_par[k].shape), ref_par[k], keep=False)
    c.finish()


# ---- HIP graph replay ------------------------------------------------------------------------
@pytest.mark.parametrize("name,dtype,D,G,mix", [
    ("graph_f32_G32_attn", "f32", 32, 32, O.MIX_ATTN),
    ("graph_bf16_G64_lin", "bf16", 32, 64, O.MIX_LINEAR_G),
    ("graph_bf16_G256_lin", "bf16", 32, 256, O.MIX_LINEAR_G),
    ("graph_f32_G1024_attn", "f32", 32, 1024, O.MIX_ATTN),
])
def test_graph_replay_matches_eager(name, dtype, D, G, mix):
    """One forward + backward captured as a HIP graph and replayed several times, with eager
    launches and synchronisations in between, gives bitwise the eager results every time
    (the kernels are deterministic, and no call records a memset)."""
    import torch
    from paper_2609_32525_amd.runner import PathBuffers
    w = small(name, dtype, D, G, mix, N=3000 if G <= 256 else 900, B=2, H=2)
    announce(f"graph {w}")
    inp = W.make_inputs(w)
    pb = PathBuffers(inp, w.mix, w.dtype, w.eps)
    pb.step()
    eager = pb.results()
    dev = pb.dev
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        pb.step()
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize(dev)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        pb.step()
    torch.cuda.synchronize(dev)
    for rep in range(3):
        for t in (pb.out, pb.dx, pb.dfx, pb.dWs, pb.z):
            t.fill_(float("nan"))          # the replay must rewrite every output
        graph.replay()
        got = pb.results()
        for k, v in eager.items():
            if v is not None:
                assert np.array_equal(v, got[k]), (rep, k)
        pb.forward()                        # eager work between replays
        torch.cuda.synchronize(dev)
