"""Parity of the forward-only (inference) path against the fp64 oracle (needs an MI355X).

The forward-only path saves no normaliser: fs_slice_fwd runs with lse = NULL and the deslice
recomputes every point's softmax statistics from its logits (fs_deslice_fwd with lse = NULL,
or fs_deslice_stats_fwd, which also writes lse). Outputs are compared normwise and element by
element (tests/paritycheck.py), 1e-5 for fp32 storage and 2e-2 for bf16 storage, as in the
forward + backward parity tests.
"""
import sys

import numpy as np
import pytest

import oracle as O
import workloads as W
from paritycheck import ELEM_TOL, KAPPA, TOL, Checker, announce, measures

pytestmark = pytest.mark.gpu

LN2 = float(np.log(2.0))


def case(name, dtype, D, G, mix, B=2, N=1000, H=3, **kw):
    return W.Workload(name, 300 + G + D + mix, dtype, B, N, H, D, D, G, mix, **kw)


# every head width, the single-wave deslice (G <= 64) and the cooperative one with 2, 4 and
# 16 slot waves (G = 128, 256, 1024), every mix kind, peaky logits, ragged point tails
CASES = [
    case("f32_D32_G32_attn", "f32", 32, 32, O.MIX_ATTN),
    case("f32_D16_G16_lin", "f32", 16, 16, O.MIX_LINEAR_G, N=777),
    case("f32_D64_G32_id", "f32", 64, 32, O.MIX_IDENTITY),
    case("f32_D32_G64_linc", "f32", 32, 64, O.MIX_LINEAR_C, N=1031),
    case("f32_D32_G128_lin", "f32", 32, 128, O.MIX_LINEAR_G),
    case("f32_D32_G256_attn", "f32", 32, 256, O.MIX_ATTN, N=700),
    case("f32_D32_G1024_lin", "f32", 32, 1024, O.MIX_LINEAR_G, N=600, H=2, B=1),
    case("bf16_D32_G64_lin", "bf16", 32, 64, O.MIX_LINEAR_G),
    case("bf16_D64_G64_linc", "bf16", 64, 64, O.MIX_LINEAR_C),
    case("bf16_D16_G128_lin", "bf16", 16, 128, O.MIX_LINEAR_G, tau_mode="uniform",
         ws_mode="std3"),
    case("bf16_D32_G256_lin", "bf16", 32, 256, O.MIX_LINEAR_G, tau_mode="uniform",
         ws_mode="std3", N=900),
    case("bf16_D64_G256_lin", "bf16", 64, 256, O.MIX_LINEAR_G, N=600, H=2),
    case("bf16_D32_G1024_lin", "bf16", 32, 1024, O.MIX_LINEAR_G, tau_mode="uniform",
         ws_mode="std3", N=700, H=2, B=1),
    case("f32_D32_G64_lin_N1", "f32", 32, 64, O.MIX_LINEAR_G, N=1),
    case("f32_D32_G256_lin_N33", "f32", 32, 256, O.MIX_LINEAR_G, N=33),
]


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_forward_only(w):
    import torch
    import paper_2609_32525_amd as fs
    from paper_2609_32525_amd.runner import PathBuffers
    announce(f"forward-only {w}")
    inp = W.make_inputs(w, with_grad=False)
    pb = PathBuffers(inp, w.mix, w.dtype, w.eps, with_backward=False, keep_lse=False)
    pb.forward()
    got = pb.results()
    ref, _ = O.run_inputs(inp, w.mix, w.eps, backward_too=False)
    c = Checker(f"forward/{w.name}", w.dtype)
    for k in ("z", "s", "zmix", "out"):
        c.add(k, got[k], ref[k], keep=False)
    # the same deslice writing its statistics: lse in the base-2 unit of the library
    lse = torch.full((w.B, w.H, w.N), float("nan"), device=pb.dev)
    out2 = torch.empty_like(pb.out)
    fs.deslice_stats_fwd(pb.prob, pb.x, pb.Ws, pb.b, pb.tau, pb.zmix, lse, out2)
    torch.cuda.synchronize()
    lse_h = lse.double().cpu().numpy() * LN2
    out2_h = out2.float().cpu().numpy().astype(np.float64)
    c.add("lse", lse_h, ref["lse"], keep=False)
    c.add("out(stats)", out2_h, ref["out"], keep=False)
    c.finish()
    # writing lse changes nothing else: both calls run the same arithmetic
    assert np.array_equal(out2_h, got["out"])
    # the saved-normaliser deslice, fed the recomputed lse, agrees with the recomputing one
    out3 = torch.empty_like(pb.out)
    fs.deslice_fwd(pb.prob, pb.x, pb.Ws, pb.b, pb.tau, pb.zmix, lse, out3)
    torch.cuda.synchronize()
    out3_h = out3.float().cpu().numpy().astype(np.float64)
    n3, e3 = measures(out3_h, got["out"], KAPPA[w.dtype])
    assert n3 <= TOL[w.dtype] and e3 <= ELEM_TOL[w.dtype], (n3, e3)


def test_forward_only_empty_point_set():
    """N = 0: nothing to deslice; the call succeeds and the tokens are zero."""
    import paper_2609_32525_amd as fs
    from paper_2609_32525_amd.runner import PathBuffers
    w = case("f32_N0", "f32", 32, 256, O.MIX_LINEAR_G, N=0, B=2, H=2)
    announce("forward-only N=0")
    inp = W.make_inputs(w, with_grad=False)
    pb = PathBuffers(inp, w.mix, w.dtype, w.eps, with_backward=False, keep_lse=False)
    pb.forward()
    fs.deslice_stats_fwd(pb.prob, pb.x, pb.Ws, pb.b, pb.tau, pb.zmix, None, pb.out)
    got = pb.results()
    assert np.all(got["s"] == 0) and np.all(got["z"] == 0)


def test_forward_only_full_size_infer():
    """The inference workload at its full size (bf16, N = 2^24 points from 16 copies of one
    seeded 2^20-point block, H = 8, dh = 32, G = 64), in the launch configuration the
    benchmark times. The oracle evaluates the full-size sums from the block (forward_repeated)
    for two heads, and the outputs and normalisers at sampled points, among them both ends,
    the block seams and the 2^22-point boundaries."""
    import torch
    import paper_2609_32525_amd as fs
    from paper_2609_32525_amd.runner import PathBuffers
    w = W.WORKLOADS["infer"]
    announce(f"forward-only full size {w}")
    inp = W.make_inputs(w, with_grad=False)
    pb = PathBuffers(inp, w.mix, w.dtype, w.eps, with_backward=False, repeat=w.repeat,
                     keep_lse=False)
    pb.forward()
    torch.cuda.synchronize()
    N = w.N
    rng = np.random.default_rng(7)
    special = [0, 1, N - 1, N - 2]
    for k in range(1, w.repeat):
        special += [k * w.block_N - 1, k * w.block_N]
    for k in range(1, 4):
        special += [k * (1 << 22) - 1, k * (1 << 22)]
    pts = np.unique(np.concatenate([rng.integers(0, N, 4096), np.array(special)]))
    idx = torch.from_numpy(pts).to(pb.dev)
    out_s = pb.out.index_select(1, idx).float().cpu().numpy().astype(np.float64)
    z = pb.z.double().cpu().numpy()
    s = pb.s.double().cpu().numpy()
    zmix = pb.zmix.double().cpu().numpy()
    # every head: the weights of each point sum to one, so the slot sums add up to N
    np.testing.assert_allclose(s.sum(-1), N, rtol=1e-5)
    assert np.isfinite(out_s).all()
    # the recomputing deslice with its lse output, at full size
    lse = torch.empty((w.B, w.H, N), device=pb.dev)
    out2 = torch.empty_like(pb.out)
    fs.deslice_stats_fwd(pb.prob, pb.x, pb.Ws, pb.b, pb.tau, pb.zmix, lse, out2)
    torch.cuda.synchronize()
    out2_s = out2.index_select(1, idx).float().cpu().numpy().astype(np.float64)
    lse_s = lse.index_select(2, idx).double().cpu().numpy() * LN2
    del out2, lse
    assert np.array_equal(out2_s, out_s)
    pairs = [(0, 0), (0, 5)]
    print(f"  oracle on pairs {pairs} from the {w.block_N}-point block", flush=True)
    prm = {k: inp.get(k) for k in ("A", "Wc", "Wq", "Wk", "Wv", "scale")}
    ref = O.forward_repeated(inp["x"], inp["fx"], inp["Ws"], inp["b"], inp["tau"], w.mix, prm,
                             w.eps, w.repeat, pts, pairs=pairs)
    c = Checker("forward/infer", w.dtype)
    for bb, h in pairs:
        for k, g in (("z", z), ("s", s), ("zmix", zmix)):
            c.add(f"{k}[{h}]", g[bb, h], ref[k][bb, h], keep=False)
        c.add(f"out[{h}]", out_s[bb, :, h], ref["out"][bb, :, h], keep=False)
        c.add(f"lse[{h}]", lse_s[bb, h], ref["lse"][bb, h], keep=False)
    c.finish()
