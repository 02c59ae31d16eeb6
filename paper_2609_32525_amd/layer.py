"""A stack of Transolver-style layers whose physics-attention core runs through the C ABI.

Each layer (paper: Sec. 2, "The Transolver layer"): pre-LayerNorm; two input projections
C -> C giving the slice features x and the values fx, each viewed as H heads of width
D = C / H; the fused slice -> constant G x G token mix -> deslice path of this library
(PathFunction, forward and backward through libflashslice); an output projection C -> C;
residual; pre-LayerNorm; an MLP C -> 4C -> C with the exact (erf) GELU; residual.

Only the path is this library's work. LayerNorm, the projections and the MLP are plain torch
modules (hipBLASLt GEMMs on the GPU), as the paper keeps them outside its fused kernels
(App. F.1: input projections remain separate GEMMs). Storage is fp32.
"""
from __future__ import annotations

import math
from typing import Callable, List, Optional

import torch
from torch import nn

from . import (F32, MIX_LINEAR_G, MixDesc, Problem, deslice_fwd, mix, slice_deslice_bwd,
               slice_fwd, workspace_bytes)


class PathFunction(torch.autograd.Function):
    """out = deslice(Mix(slice(x, fx))) for x, fx (B, N, H, D) fp32 on the GPU, with the
    slice parameters W_s (D, G), b (G), tau (H) shared by the heads and the constant token
    matrix A (G, G). Forward: fs_slice_fwd, fs_mix, fs_deslice_fwd. Backward:
    fs_slice_deslice_bwd, which also returns the gradients of W_s, b, tau and A. Launches go
    to torch's current stream; workspaces come from the caller's PathWorkspace."""

    @staticmethod
    def forward(ctx, x, fx, Ws, b, tau, A, space: "PathWorkspace"):
        B, N, H, D = x.shape
        G = Ws.shape[1]
        prob = space.problem(B, N, H, D, G)
        md = MixDesc.make(MIX_LINEAR_G, A=A)
        f32 = dict(device=x.device, dtype=torch.float32)
        z = torch.empty((B, H, G, D), **f32)
        s = torch.empty((B, H, G), **f32)
        zmix = torch.empty_like(z)
        lse = torch.empty((B, H, N), **f32)
        out = torch.empty_like(fx)
        space.mark(0)
        slice_fwd(prob, x, fx, Ws, b, tau, z, s, lse, space.buffer(prob, 0, x.device))
        mix(prob, md, z, zmix, None)
        deslice_fwd(prob, x, Ws, b, tau, zmix, lse, out)
        space.mark(1)
        ctx.save_for_backward(x, fx, Ws, b, tau, A, z, s, zmix, lse)
        ctx.space = space
        return out

    @staticmethod
    def backward(ctx, dout):
        x, fx, Ws, b, tau, A, z, s, zmix, lse = ctx.saved_tensors
        space = ctx.space
        B, N, H, D = x.shape
        G = Ws.shape[1]
        prob = space.problem(B, N, H, D, G)
        md = MixDesc.make(MIX_LINEAR_G, A=A)
        dout = dout.contiguous()
        dx, dfx = torch.empty_like(x), torch.empty_like(fx)
        dWs, db, dtau, dA = (torch.empty_like(Ws), torch.empty_like(b), torch.empty_like(tau),
                             torch.empty_like(A))
        space.mark(0)
        slice_deslice_bwd(prob, md, x, fx, Ws, b, tau, z, s, zmix, None, lse, dout, dx, dfx,
                          dWs, db, dtau, dA, None, space.buffer(prob, 1, x.device))
        space.mark(1)
        return dx, dfx, dWs, db, dtau, dA, None


class PathWorkspace:
    """Device workspaces of the path calls, grown on demand and reused by every layer (the
    calls of one step run in order on one stream). With ``events`` set (a list), a pair of
    CUDA events is appended around every forward and backward path call, for timing."""

    def __init__(self, eps: float = 1e-5):
        self.eps = eps
        self.ws = {0: None, 1: None}
        self.events: Optional[List] = None
        self._open = None

    def problem(self, B, N, H, D, G) -> Problem:
        return Problem.make(B, N, H, D, D, G, F32, self.eps)

    def buffer(self, prob: Problem, code: int, device) -> torch.Tensor:
        need = max(1, workspace_bytes(prob, code))
        t = self.ws[code]
        if t is None or t.numel() < need or t.device != device:
            t = torch.empty(need, dtype=torch.uint8, device=device)
            self.ws[code] = t
        return t

    def mark(self, which: int) -> None:
        if self.events is None:
            return
        ev = torch.cuda.Event(enable_timing=True)
        ev.record()
        if which == 0:
            self._open = ev
        else:
            self.events.append((self._open, ev))


class PhysicsAttention(nn.Module):
    """Input projections, the fused path over H heads with G slices, output projection."""

    def __init__(self, C: int, H: int, G: int, space: PathWorkspace):
        super().__init__()
        if C % H:
            raise ValueError("C must be a multiple of H")
        self.C, self.H, self.D, self.G = C, H, C // H, G
        self.space = space
        self.in_x = nn.Linear(C, C)
        self.in_fx = nn.Linear(C, C)
        self.out = nn.Linear(C, C)
        lim = math.sqrt(6.0 / (self.D + G))
        self.Ws = nn.Parameter(torch.empty(self.D, G).uniform_(-lim, lim))
        self.b = nn.Parameter(torch.zeros(G))
        self.tau = nn.Parameter(torch.full((H,), 0.5))
        self.A = nn.Parameter(torch.randn(G, G) / math.sqrt(G))

    def forward(self, h):
        B, N, C = h.shape
        x = self.in_x(h).view(B, N, self.H, self.D)
        fx = self.in_fx(h).view(B, N, self.H, self.D)
        o = PathFunction.apply(x.contiguous(), fx.contiguous(), self.Ws, self.b, self.tau,
                               self.A, self.space)
        return self.out(o.reshape(B, N, C))


class Block(nn.Module):
    def __init__(self, C: int, H: int, G: int, space: PathWorkspace):
        super().__init__()
        self.ln1 = nn.LayerNorm(C)
        self.attn = PhysicsAttention(C, H, G, space)
        self.ln2 = nn.LayerNorm(C)
        self.mlp = nn.Sequential(nn.Linear(C, 4 * C), nn.GELU(), nn.Linear(4 * C, C))

    def forward(self, h):
        h = h + self.attn(self.ln1(h))
        return h + self.mlp(self.ln2(h))


class SliceStack(nn.Module):
    """L layers of width C with H heads and G slices (fp32)."""

    def __init__(self, L: int, C: int, H: int, G: int, eps: float = 1e-5):
        super().__init__()
        self.space = PathWorkspace(eps)
        self.blocks = nn.ModuleList([Block(C, H, G, self.space) for _ in range(L)])

    def forward(self, h):
        for blk in self.blocks:
            h = blk(h)
        return h


def training_step(model: SliceStack, h: torch.Tensor, R: torch.Tensor, lr: float = 0.0,
                  hook: Optional[Callable[[], None]] = None) -> torch.Tensor:
    """One training step: forward, the loss sum(out * R) (so d loss / d out = R), backward,
    and a plain SGD update of every parameter by lr (lr = 0 leaves the weights as they are
    but still runs the update). Returns the loss (a device scalar)."""
    for p in model.parameters():
        p.grad = None
    out = model(h)
    loss = (out * R).sum()
    loss.backward()
    if hook is not None:
        hook()
    with torch.no_grad():
        params = [p for p in model.parameters() if p.grad is not None]
        torch._foreach_add_(params, [p.grad for p in params], alpha=-lr)
    return loss
