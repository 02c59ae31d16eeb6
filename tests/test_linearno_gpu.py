"""Parity of the LinearNO variant (untied, slice weights softmaxed over the points of each
slot) against the fp64 oracle (needs an MI355X).

Forward: fs_linearno_slice_fwd (z, clse), fs_mix, fs_deslice_stats_fwd with the deslice's own
projection (lse_d); backward: fs_linearno_bwd. Every output is compared normwise and element
by element (tests/paritycheck.py), at most 1e-5 for fp32 storage and 2e-2 for bf16 storage;
the (case, output) pairs listed in paritycheck.FP32_EAGER_GATED take the paper's plain-fp32
acceptance rule instead (App. F.2). The slice bias gradient is zero in exact arithmetic (a
constant added to one slot's logits changes nothing), so it is compared with zero on the
scale of the slice projection gradient.
"""
import sys

import numpy as np
import pytest

import oracle as O
import workloads as W
from paritycheck import Checker, announce

pytestmark = pytest.mark.gpu

LN2 = float(np.log(2.0))


def rms(a):
    a = np.asarray(a, dtype=np.float64)
    return float(np.sqrt(np.mean(a * a))) if a.size else 0.0


def case(name, dtype, D, G, mix, B=2, N=1000, H=3, **kw):
    return W.Workload(name, 700 + G + D + mix, dtype, B, N, H, D, D, G, mix, **kw)


# the paper's layer uses the channel map; the other mixes, every head width, single-wave and
# cooperative tilings (G = 128, 256), per-head projections, peaky logits, ragged tails, N = 1
CASES = [
    case("f32_D32_G32_linc", "f32", 32, 32, O.MIX_LINEAR_C),
    case("f32_D16_G16_linc", "f32", 16, 16, O.MIX_LINEAR_C, N=777),
    case("f32_D64_G64_lin", "f32", 64, 64, O.MIX_LINEAR_G),
    case("f32_D32_G64_attn", "f32", 32, 64, O.MIX_ATTN, N=1031),
    case("f32_D32_G128_id", "f32", 32, 128, O.MIX_IDENTITY),
    case("f32_D32_G256_linc_ph", "f32", 32, 256, O.MIX_LINEAR_C, N=600, H=2, ws_per_head=True),
    case("f32_D32_G32_linc_N1", "f32", 32, 32, O.MIX_LINEAR_C, N=1),
    case("bf16_D32_G64_linc", "bf16", 32, 64, O.MIX_LINEAR_C),
    case("bf16_D64_G32_lin", "bf16", 64, 32, O.MIX_LINEAR_G),
    case("bf16_D16_G128_linc", "bf16", 16, 128, O.MIX_LINEAR_C, tau_mode="uniform",
         ws_mode="std3"),
    case("bf16_D32_G256_linc", "bf16", 32, 256, O.MIX_LINEAR_C, N=700, H=2),
    # one-tile-plus-one point sets (ragged tails only)
    case("bf16_D32_G64_linc_N33", "bf16", 32, 64, O.MIX_LINEAR_C, N=33),
    case("f32_D32_G256_linc_N33", "f32", 32, 256, O.MIX_LINEAR_C, N=33, H=2),
    # padded tilings: one wave (48), two waves (80), four waves with a partial one (208)
    case("f32_D32_G48_linc", "f32", 32, 48, O.MIX_LINEAR_C),
    case("bf16_D32_G80_linc", "bf16", 32, 80, O.MIX_LINEAR_C, N=900),
    case("f32_D32_G208_linc", "f32", 32, 208, O.MIX_LINEAR_C, N=600, H=2),
    # slot-blocked family at G = 1024 and with a partial last block; head width 64 stays on
    # the cooperative form
    case("bf16_D32_G1024_linc", "bf16", 32, 1024, O.MIX_LINEAR_C, N=600, H=2, B=1),
    case("f32_D32_G336_lin", "f32", 32, 336, O.MIX_LINEAR_G, N=500, H=2),
    case("f32_D64_G256_linc", "f32", 64, 256, O.MIX_LINEAR_C, N=500, H=2),
]


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_linearno(w):
    from paper_2609_32525_amd.runner import PathBuffers
    announce(f"linearno {w}")
    inp = W.make_inputs(w)
    ut = W.untied_params(w)
    pb = PathBuffers(inp, w.mix, w.dtype, w.eps, untied=ut, linearno=True)
    pb.step()
    got = pb.results()
    got["clse"] = got["clse"] * LN2
    got["lse_d"] = got["lse_d"] * LN2
    prm = {k: inp.get(k) for k in ("A", "Wc", "Wq", "Wk", "Wv", "scale")}
    args = (inp["x"], inp["fx"], inp["Ws"], inp["b"], inp["tau"], ut["Wd"], ut["bd"],
            ut["taud"], w.mix, prm)
    fwd = O.linearno_forward(*args)
    bwd = O.linearno_backward(*args, inp["dout"], fwd=fwd)
    keys_f = ["z", "clse", "zmix", "lse_d", "out"] + (["P"] if w.mix == O.MIX_ATTN else [])
    keys_b = ["dx", "dfx", "dWs", "dtau", "dWd", "dbd", "dtaud", "dzmix"]
    c = Checker(f"linearno/{w.name}", w.dtype)
    for k in keys_f:
        c.add(k, got[k], fwd[k])
    # one point: every slot's weight over the points is 1 and the tokens all equal that
    # point's fx, so both logit gradients vanish exactly; they are compared on the scale of
    # the nonzero fx gradient instead
    vanish = ("dx", "dWs", "dtau", "dWd", "dbd", "dtaud") if w.N == 1 else ()
    for k in keys_b:
        c.add(k, got[k], bwd[k], floor=rms(bwd["dfx"]) if k in vanish else 0.0)
    d = pb.dmix.double().cpu().numpy() if pb.dmix is not None else None
    V = w.V
    if w.mix == O.MIX_ATTN:
        for n, k in enumerate(("dWq", "dWk", "dWv")):
            c.add(k, d[n * V * V:(n + 1) * V * V].reshape(V, V), bwd[k])
    elif w.mix == O.MIX_LINEAR_G:
        c.add("dA", d.reshape(bwd["dA"].shape), bwd["dA"])
    elif w.mix == O.MIX_LINEAR_C:
        c.add("dWc", d.reshape(V, V), bwd["dWc"])
    # the slice bias gradient vanishes: rounding only, on the scale of the projection gradient
    c.add("db", got["db"], np.zeros_like(got["db"]),
          floor=max(rms(bwd["dWs"]), rms(bwd["dfx"]) if w.N == 1 else 0.0))

    def eager():
        f32 = O.linearno_forward(*args, dtype=np.float32)
        b32 = O.linearno_backward(*args, inp["dout"], fwd=f32, dtype=np.float32)
        return {**f32, **b32}

    c.finish(eager)


def test_linearno_full_size_volume():
    """The LinearNO workload at its full size (bf16, N = 2^20, H = 8, G = 64, channel map), in
    the launch configuration the benchmark times. The oracle recomputes one (sample, head)
    pair (every output of it at every point, and that head's two temperature gradients);
    over all heads every output is finite and the slice bias gradient vanishes."""
    from paper_2609_32525_amd.runner import PathBuffers
    w = W.WORKLOADS["volume_linearno"]
    print(f"\n[case] linearno full size {w}", flush=True)
    inp = W.make_inputs(w)
    ut = W.untied_params(w)
    pb = PathBuffers(inp, w.mix, w.dtype, w.eps, untied=ut, linearno=True)
    pb.step()
    got = pb.results()
    for k in ("z", "clse", "zmix", "out", "dx", "dfx", "dWs", "db", "dtau", "dWd", "dbd",
              "dtaud"):
        assert np.isfinite(got[k]).all(), k
    assert np.linalg.norm(got["db"]) <= 2e-2 * np.linalg.norm(got["dWs"])
    pairs = [(0, 3)]
    prm = {k: inp.get(k) for k in ("A", "Wc", "Wq", "Wk", "Wv", "scale")}
    args = (inp["x"], inp["fx"], inp["Ws"], inp["b"], inp["tau"], ut["Wd"], ut["bd"],
            ut["taud"], w.mix, prm)
    print(f"  oracle on pairs {pairs}", flush=True)
    fwd = O.linearno_forward(*args, pairs=pairs)
    bwd = O.linearno_backward(*args, inp["dout"], fwd=fwd, pairs=pairs)
    c = Checker("linearno/volume_linearno", w.dtype)
    for bb, h in pairs:
        for k in ("z", "zmix", "dzmix"):
            c.add(f"{k}[{h}]", got[k][bb, h], (bwd if k in bwd else fwd)[k][bb, h], keep=False)
        c.add(f"clse[{h}]", got["clse"][bb, h] * LN2, fwd["clse"][bb, h], keep=False)
        c.add(f"lse_d[{h}]", got["lse_d"][bb, h] * LN2, fwd["lse_d"][bb, h], keep=False)
        for k in ("out", "dx", "dfx"):
            c.add(f"{k}[{h}]", got[k][bb, :, h], (bwd if k in bwd else fwd)[k][bb, :, h],
                  keep=False)
        for k in ("dtau", "dtaud"):
            c.add(f"{k}[{h}]", got[k][h], bwd[k][h], keep=False)
    c.finish()
