"""Reference of the 8-layer slicing stack on the CPU (paper: Sec. 2, "The Transolver layer").

TEST INFRASTRUCTURE ONLY, like the rest of this package: the tests and the benchmark's
CPU-baseline leg use it; nothing on the product path does.

Each layer: pre-LayerNorm; input projections C -> C for the slice features x and the values
fx (H heads of width C / H); the physics-attention path with a constant G x G token matrix,
computed by this package's oracle (its forward, and its derived backward for the gradients);
an output projection C -> C; residual; pre-LayerNorm; MLP C -> 4C -> C with the exact (erf)
GELU; residual. LayerNorm, the projections and the MLP are plain torch CPU modules, in
float64 (or float32, the plain-fp32 yardstick of the paper's acceptance rule).
"""
from __future__ import annotations

import numpy as np
import torch
from torch import nn

from . import MIX_LINEAR_G, backward as _backward, forward as _forward


class OraclePath(torch.autograd.Function):
    """The oracle's path (constant G x G token matrix A, shared W_s, b) as an autograd node:
    forward with O.forward, gradients with O.backward, in the tensors' dtype."""

    @staticmethod
    def forward(ctx, x, fx, Ws, b, tau, A, eps):
        dt = x.dtype
        npd = np.float64 if dt == torch.float64 else np.float32
        a = [t.detach().numpy() for t in (x, fx, Ws, b, tau, A)]
        prm = {"A": a[5]}
        f = _forward(a[0], a[1], a[2], a[3], a[4], MIX_LINEAR_G, prm, eps, dtype=npd)
        ctx.save_for_backward(x, fx, Ws, b, tau, A)
        ctx.fwd, ctx.eps = f, eps
        return torch.from_numpy(f["out"].astype(npd))

    @staticmethod
    def backward(ctx, dout):
        x, fx, Ws, b, tau, A = ctx.saved_tensors
        dt = x.dtype
        npd = np.float64 if dt == torch.float64 else np.float32
        a = [t.detach().numpy() for t in (x, fx, Ws, b, tau, A)]
        g = _backward(a[0], a[1], a[2], a[3], a[4], MIX_LINEAR_G, {"A": a[5]},
                       dout.detach().numpy(), ctx.eps, fwd=ctx.fwd, dtype=npd)
        t = lambda k: torch.from_numpy(np.asarray(g[k], dtype=npd))
        return t("dx"), t("dfx"), t("dWs"), t("db"), t("dtau"), t("dA"), None


class RefAttention(nn.Module):
    def __init__(self, C, H, G, eps):
        super().__init__()
        self.H, self.D, self.eps = H, C // H, eps
        self.in_x, self.in_fx, self.out = nn.Linear(C, C), nn.Linear(C, C), nn.Linear(C, C)
        self.Ws = nn.Parameter(torch.zeros(self.D, G))
        self.b = nn.Parameter(torch.zeros(G))
        self.tau = nn.Parameter(torch.ones(H))
        self.A = nn.Parameter(torch.zeros(G, G))

    def forward(self, h):
        B, N, C = h.shape
        x = self.in_x(h).reshape(B, N, self.H, self.D)
        fx = self.in_fx(h).reshape(B, N, self.H, self.D)
        o = OraclePath.apply(x, fx, self.Ws, self.b, self.tau, self.A, self.eps)
        return self.out(o.reshape(B, N, C))


class RefBlock(nn.Module):
    def __init__(self, C, H, G, eps):
        super().__init__()
        self.ln1 = nn.LayerNorm(C)
        self.attn = RefAttention(C, H, G, eps)
        self.ln2 = nn.LayerNorm(C)
        self.mlp = nn.Sequential(nn.Linear(C, 4 * C), nn.GELU(), nn.Linear(4 * C, C))

    def forward(self, h):
        h = h + self.attn(self.ln1(h))
        return h + self.mlp(self.ln2(h))


class RefStack(nn.Module):
    def __init__(self, L, C, H, G, eps=1e-5):
        super().__init__()
        self.blocks = nn.ModuleList([RefBlock(C, H, G, eps) for _ in range(L)])

    def forward(self, h):
        for blk in self.blocks:
            h = blk(h)
        return h


def reference_step(state_dict, L, C, H, G, h, R, dtype=torch.float64, eps=1e-5):
    """Loss sum(out * R), the output, and the gradients of every parameter and of h, from the
    given parameter values (a state dict), in dtype on the CPU."""
    ref = RefStack(L, C, H, G, eps).to(dtype)
    ref.load_state_dict({k: v.detach().cpu().to(dtype) for k, v in state_dict.items()})
    hh = torch.as_tensor(h, dtype=dtype).clone().requires_grad_(True)
    out = ref(hh)
    loss = (out * torch.as_tensor(R, dtype=dtype)).sum()
    loss.backward()
    grads = {k: p.grad.detach().double().numpy() for k, p in ref.named_parameters()}
    grads["h"] = hh.grad.double().numpy()
    return float(loss.detach()), out.detach().double().numpy(), grads
