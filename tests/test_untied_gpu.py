"""Parity of the untied variant (the deslice with its own projection, bias and temperature)
against the fp64 oracle (needs an MI355X).

Forward: fs_slice_fwd with (W_s, b, tau), fs_mix, fs_deslice_stats_fwd with (W_d, b_d, tau_d)
saving lse_d; backward: fs_untied_bwd. Every output and gradient is compared normwise and
element by element (tests/paritycheck.py), at most 1e-5 for fp32 storage and 2e-2 for bf16
storage. The (case, output) pairs listed in paritycheck.FP32_EAGER_GATED take the paper's
plain-fp32 acceptance rule instead (App. F.2): the deslice weights' gradients see zmix only
through how its tokens differ from one another, and where the tokens are close (an attention
mix over few tokens averages them) the fp32 rounding of zmix alone exceeds 1e-5 of those
gradients.
"""
import sys

import numpy as np
import pytest

import oracle as O
import workloads as W
from paritycheck import Checker, announce

pytestmark = pytest.mark.gpu

LN2 = float(np.log(2.0))


def case(name, dtype, D, G, mix, B=2, N=1000, H=3, **kw):
    return W.Workload(name, 500 + G + D + mix, dtype, B, N, H, D, D, G, mix, **kw)


# single-wave and cooperative tilings (G = 128: two slot waves; G = 256: four), every head
# width, every mix kind, per-head projections, peaky logits, ragged tails
CASES = [
    case("f32_D32_G32_attn", "f32", 32, 32, O.MIX_ATTN),
    case("f32_D16_G16_lin", "f32", 16, 16, O.MIX_LINEAR_G, N=777),
    case("f32_D64_G32_linc", "f32", 64, 32, O.MIX_LINEAR_C),
    case("f32_D32_G64_id", "f32", 32, 64, O.MIX_IDENTITY, N=1031),
    case("f32_D32_G128_lin", "f32", 32, 128, O.MIX_LINEAR_G),
    case("f32_D32_G256_lin_ph", "f32", 32, 256, O.MIX_LINEAR_G, N=600, H=2, ws_per_head=True),
    case("bf16_D32_G64_lin", "bf16", 32, 64, O.MIX_LINEAR_G),
    case("bf16_D64_G64_linc", "bf16", 64, 64, O.MIX_LINEAR_C),
    case("bf16_D16_G128_lin", "bf16", 16, 128, O.MIX_LINEAR_G, tau_mode="uniform",
         ws_mode="std3"),
    case("bf16_D32_G256_attn", "bf16", 32, 256, O.MIX_ATTN, N=700, H=2),
    # single-point and one-tile-plus-one point sets (ragged tails only)
    case("f32_D32_G32_lin_N1", "f32", 32, 32, O.MIX_LINEAR_G, N=1),
    case("bf16_D32_G64_linc_N33", "bf16", 32, 64, O.MIX_LINEAR_C, N=33),
    case("f32_D32_G256_lin_N33", "f32", 32, 256, O.MIX_LINEAR_G, N=33, H=2),
    # padded tilings: one wave (48), two waves (80), 8 waves of which 3 hold no real slot (272)
    case("f32_D32_G48_lin", "f32", 32, 48, O.MIX_LINEAR_G),
    case("bf16_D32_G80_attn", "bf16", 32, 80, O.MIX_ATTN, N=900),
    case("f32_D32_G272_lin", "f32", 32, 272, O.MIX_LINEAR_G, N=600, H=2),
    # slot-blocked family (point-owned pass and parameter pass per weight set) at G = 1024;
    # the cooperative form beyond 128 slots remains for head width 64
    case("f32_D32_G1024_lin", "f32", 32, 1024, O.MIX_LINEAR_G, N=500, H=2, B=1),
    case("bf16_D16_G512_attn", "bf16", 16, 512, O.MIX_ATTN, N=600, H=2, B=1),
    case("f32_D64_G256_lin", "f32", 64, 256, O.MIX_LINEAR_G, N=500, H=2),
]


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_untied(w):
    from paper_2609_32525_amd.runner import PathBuffers
    announce(f"untied {w}")
    inp = W.make_inputs(w)
    ut = W.untied_params(w)
    pb = PathBuffers(inp, w.mix, w.dtype, w.eps, untied=ut)
    pb.step()
    got = pb.results()
    got["lse"] = got["lse"] * LN2
    got["lse_d"] = got["lse_d"] * LN2
    prm = {k: inp.get(k) for k in ("A", "Wc", "Wq", "Wk", "Wv", "scale")}
    args = (inp["x"], inp["fx"], inp["Ws"], inp["b"], inp["tau"], ut["Wd"], ut["bd"],
            ut["taud"], w.mix, prm)
    fwd = O.untied_forward(*args, eps=w.eps)
    bwd = O.untied_backward(*args, inp["dout"], eps=w.eps, fwd=fwd)
    keys_f = ["z", "s", "zmix", "lse", "lse_d", "out"] + (["P"] if w.mix == O.MIX_ATTN else [])
    keys_b = ["dx", "dfx", "dWs", "db", "dtau", "dWd", "dbd", "dtaud", "dzmix"]
    c = Checker(f"untied/{w.name}", w.dtype)
    for k in keys_f:
        c.add(k, got[k], fwd[k])
    for k in keys_b:
        c.add(k, got[k], bwd[k])
    d = pb.dmix.double().cpu().numpy() if pb.dmix is not None else None
    V = w.V
    if w.mix == O.MIX_ATTN:
        for n, k in enumerate(("dWq", "dWk", "dWv")):
            c.add(k, d[n * V * V:(n + 1) * V * V].reshape(V, V), bwd[k])
    elif w.mix == O.MIX_LINEAR_G:
        c.add("dA", d.reshape(bwd["dA"].shape), bwd["dA"])
    elif w.mix == O.MIX_LINEAR_C:
        c.add("dWc", d.reshape(V, V), bwd["dWc"])

    def eager():
        f32 = O.untied_forward(*args, eps=w.eps, dtype=np.float32)
        b32 = O.untied_backward(*args, inp["dout"], eps=w.eps, fwd=f32, dtype=np.float32)
        return {**f32, **b32}

    c.finish(eager)


def test_untied_full_size_surface():
    """The untied workload at its full size (fp32, N = 32768, H = 8, G = 32, attention mix),
    in the launch configuration the benchmark times, against the oracle on every head."""
    w = W.WORKLOADS["surface_untied"]
    test_untied(w)
