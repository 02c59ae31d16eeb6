"""The CPU reference of the layer stack (CPU): its oracle-backed path node is consistent with
its own forward (central finite differences through the whole stack, float64), and the
stack's wiring is the one the GPU stack uses (same parameter names and shapes)."""
import numpy as np
import torch

from oracle.stack import RefStack, reference_step


def test_reference_stack_gradients_by_finite_differences():
    torch.manual_seed(3)
    L, B, N, C, H, G = 2, 2, 5, 8, 2, 3
    ref = RefStack(L, C, H, G, eps=1e-3).double()
    with torch.no_grad():
        for name, p in ref.named_parameters():
            if name.endswith(("Ws", "A")):
                p.normal_(0, 0.7)
            elif name.endswith("tau"):
                p.uniform_(0.4, 1.2)
            elif name.endswith(".b"):
                p.normal_(0, 0.3)
    h = torch.randn(B, N, C, dtype=torch.float64, requires_grad=True)
    R = torch.randn(B, N, C, dtype=torch.float64)
    params = [p for p in ref.parameters()]

    def f(hh, *ps):
        with torch.no_grad():
            for p, v in zip(params, ps):
                p.copy_(v)
        return (ref(hh) * R).sum()

    loss = (ref(h) * R).sum()
    grads = torch.autograd.grad(loss, [h] + params)
    # central differences along random directions, for the input and every parameter
    rng = np.random.default_rng(5)
    base = [p.detach().clone() for p in params]
    for k, t in enumerate([h] + params):
        d = torch.from_numpy(rng.standard_normal(tuple(t.shape)))
        step = 1e-6
        args_p = [h.detach().clone()] + [b.clone() for b in base]
        args_m = [h.detach().clone()] + [b.clone() for b in base]
        args_p[k] = args_p[k] + step * d
        args_m[k] = args_m[k] - step * d
        fd = (f(*args_p) - f(*args_m)).item() / (2 * step)
        an = float((grads[k] * d).sum())
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (k, fd, an)
    with torch.no_grad():
        for p, b in zip(params, base):
            p.copy_(b)


def test_reference_stack_matches_library_parameter_layout():
    from paper_2609_32525_amd.layer import SliceStack
    torch.manual_seed(0)
    gpu_side = SliceStack(2, 16, 2, 4)
    ref = RefStack(2, 16, 2, 4)
    a = {k: tuple(v.shape) for k, v in gpu_side.state_dict().items()}
    b = {k: tuple(v.shape) for k, v in ref.state_dict().items()}
    assert a == b
    h = np.random.default_rng(1).standard_normal((1, 6, 16)).astype(np.float32)
    R = np.random.default_rng(2).standard_normal((1, 6, 16)).astype(np.float32)
    l64, _, g64 = reference_step(gpu_side.state_dict(), 2, 16, 2, 4, h, R)
    l32, _, g32 = reference_step(gpu_side.state_dict(), 2, 16, 2, 4, h, R, torch.float32)
    assert abs(l64 - l32) <= 1e-4 * max(1.0, abs(l64))
    assert set(g64) == set(a) | {"h"}
