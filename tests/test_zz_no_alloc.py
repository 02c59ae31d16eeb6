"""fs_slice_fwd_noalloc (the slice with the library's static per-device scratch instead of a
caller workspace) against fs_slice_fwd on the same inputs, through the C ABI (needs an
MI355X): two calls in a row, the second with a smaller problem, each bitwise equal to the
workspace entry point (the same kernels run) and within the parity bar of the fp64
oracle."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from paritycheck import Checker, announce

pytestmark = pytest.mark.gpu

LN2 = float(np.log(2.0))


def _slice_both(w):
    import torch
    import paper_2609_32525_amd as fs
    from paper_2609_32525_amd.runner import PathBuffers
    inp = W.make_inputs(w, with_grad=False)
    pb = PathBuffers(inp, w.mix, w.dtype, w.eps, with_backward=False)
    B, N, H, D, V, G = pb.shape
    dev = pb.dev
    z1, s1, l1 = pb.z, pb.s, pb.lse
    fs.slice_fwd(pb.prob, pb.x, pb.fx, pb.Ws, pb.b, pb.tau, z1, s1, l1, pb.ws_f)
    z2 = torch.full_like(z1, float("nan"))
    s2 = torch.full_like(s1, float("nan"))
    l2 = torch.full_like(l1, float("nan"))
    fs.slice_fwd_noalloc(pb.prob, pb.x, pb.fx, pb.Ws, pb.b, pb.tau, z2, s2, l2)
    torch.cuda.synchronize(dev)
    h = lambda t: t.double().cpu().numpy()
    return inp, (h(z1), h(s1), h(l1)), (h(z2), h(s2), h(l2))


@pytest.mark.parametrize("first,second", [
    (("bf16", 64, 1 << 16, 8), ("bf16", 64, 4097, 2)),
    (("f32", 1024, 20000, 4), ("f32", 256, 333, 2)),
], ids=["cooperative", "slot_blocked"])
def test_noalloc_slice_matches_workspace_entry(first, second):
    for k, (dtype, G, N, H) in enumerate((first, second)):
        w = W.Workload(f"noalloc{k}_{dtype}_G{G}", 950 + k, dtype, 2, N, H, 32, 32, G,
                       O.MIX_LINEAR_G)
        announce(f"noalloc call {k + 1}: {w}")
        inp, ws_out, st_out = _slice_both(w)
        for name, a, b in zip(("z", "s", "lse"), ws_out, st_out):
            assert np.array_equal(a, b), (k, name)
        ref, _ = O.run_inputs(inp, w.mix, w.eps, backward_too=False)
        c = Checker(f"noalloc/{w.name}", dtype)
        c.add("z", st_out[0], ref["z"], keep=False)
        c.add("s", st_out[1], ref["s"], keep=False)
        c.add("lse", st_out[2] * LN2, ref["lse"], keep=False)
        c.finish()
