"""Seeded synthetic inputs for the Mamba-3 SSM hot path.

This module only draws random tensors with the distributions of the five
workloads (sequence lengths, head counts, state size, MIMO rank, chunk), in
the memory layout the library takes.  It holds none of the recurrence's
arithmetic; both the HIP path and the CPU oracle consume what it returns.

Distributions (per workload; none is printed in the paper, which only fixes
the parameter roles, Sec. 3.1 Prop. "Exponential-Trapezoidal Discretization"
and Sec. 3.2, and the block layout of App. "MIMO for Mamba-3"):

* x, B, C ~ N(0, 1).  B and C are RMS-normalised over the state axis N for
  every (token, head, rank column), eps 1e-6, no weight (the BCNorm of
  Sec. 3.4), then rounded to the I/O dtype.
* dt = softplus(z + inv_softplus(u)), z ~ N(0, 1) per (batch, token, head),
  u ~ U[1e-3, 0.1] per head (the dt bias).
* A = -exp(U[0, ln 16]) per head (strided so the library sees a per-head A).
* lambda = sigmoid(N(0, 1)) per (batch, token, head) (App. on the lambda
  parameterisation).
* theta = dt * omega with omega ~ U[0, pi] per (head, rotation pair); theta
  is the per-step rotation angle handed to the library as is.
* D ~ N(0, 1) per head.

Draw order is fixed: x, B, C, z, u, A, lambda, omega, D.  Workload k uses
seed 1000 + k; decode step s draws its fresh token inputs with seed 4000 + s.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch

# Workload table.  "io" is the dtype of x, B, C, y and the decode carry;
# dt, lambda, theta, A, D and every state are fp32.
WORKLOADS = {
    0: dict(name="tiny-siso-fp32", batch=1, seqlen=256, nheads=2, headdim=16,
            dstate=16, rank=1, chunk=64, io="f32"),
    1: dict(name="siso-bf16-prefill", batch=4, seqlen=2048, nheads=16,
            headdim=64, dstate=128, rank=1, chunk=64, io="bf16"),
    2: dict(name="mimo4-bf16-prefill", batch=8, seqlen=4096, nheads=32,
            headdim=64, dstate=128, rank=4, chunk=64, io="bf16"),
    3: dict(name="long-mimo4-prefill", batch=1, seqlen=65536, nheads=32,
            headdim=64, dstate=128, rank=4, chunk=128, io="bf16"),
    # Decode loop: state from a 1024-token prefill with these shapes, then
    # 1024 single-token steps.
    4: dict(name="decode-b256", batch=256, seqlen=1024, nheads=32, headdim=64,
            dstate=128, rank=4, chunk=64, io="bf16", steps=1024),
}

TORCH_IO = {"f32": torch.float32, "bf16": torch.bfloat16}


@dataclass
class ScanInputs:
    """Tensors in the library layout (see include/m3.h)."""
    x: torch.Tensor        # [B, L, H, R, P]  io dtype
    Bm: torch.Tensor       # [B, L, H, R, N]  io dtype
    Cm: torch.Tensor       # [B, L, H, R, N]  io dtype
    dt: torch.Tensor       # [B, L, H]        fp32
    A: torch.Tensor        # [H]              fp32 (per-head decay rate < 0)
    lam: torch.Tensor      # [B, L, H]        fp32
    theta: torch.Tensor    # [B, L, H, N/2]   fp32 per-step angle
    D: torch.Tensor        # [H]              fp32
    # layer parameters kept so that decode steps draw from the same layer
    dt_bias: torch.Tensor = field(default=None)   # [H]
    omega: torch.Tensor = field(default=None)     # [H, N/2]
    chunk: int = 64


def _rms_normalise(v: torch.Tensor, eps: float = 1e-6) -> torch.Tensor:
    return v * torch.rsqrt(v.pow(2).mean(dim=-1, keepdim=True) + eps)


def _inv_softplus(u: torch.Tensor) -> torch.Tensor:
    return torch.log(torch.expm1(u))


def make_scan_inputs(batch, seqlen, nheads, headdim, dstate, rank, io="bf16",
                     seed=0, device="cpu", chunk=64) -> ScanInputs:
    """Draw one prefill batch with the workload distributions."""
    if dstate % 2:
        raise ValueError("dstate must be even")
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    f32 = dict(device=device, dtype=torch.float32, generator=g)
    iod = TORCH_IO[io]
    x = torch.randn((batch, seqlen, nheads, rank, headdim), **f32)
    Bm = torch.randn((batch, seqlen, nheads, rank, dstate), **f32)
    Cm = torch.randn((batch, seqlen, nheads, rank, dstate), **f32)
    z = torch.randn((batch, seqlen, nheads), **f32)
    u = torch.rand((nheads,), **f32) * (0.1 - 1e-3) + 1e-3
    A = -torch.exp(torch.rand((nheads,), **f32) * math.log(16.0))
    lam = torch.sigmoid(torch.randn((batch, seqlen, nheads), **f32))
    omega = torch.rand((nheads, dstate // 2), **f32) * math.pi
    D = torch.randn((nheads,), **f32)
    dt_bias = _inv_softplus(u)
    dt = torch.nn.functional.softplus(z + dt_bias)
    theta = dt.unsqueeze(-1) * omega
    return ScanInputs(
        x=x.to(iod).contiguous(),
        Bm=_rms_normalise(Bm).to(iod).contiguous(),
        Cm=_rms_normalise(Cm).to(iod).contiguous(),
        dt=dt.contiguous(), A=A.contiguous(), lam=lam.contiguous(),
        theta=theta.contiguous(), D=D.contiguous(),
        dt_bias=dt_bias, omega=omega, chunk=chunk)


@dataclass
class StepInputs:
    x: torch.Tensor        # [B, H, R, P]
    Bm: torch.Tensor       # [B, H, R, N]
    Cm: torch.Tensor       # [B, H, R, N]
    dt: torch.Tensor       # [B, H]
    lam: torch.Tensor      # [B, H]
    theta: torch.Tensor    # [B, H, N/2]


def make_step_inputs(layer: ScanInputs, step: int, device=None) -> StepInputs:
    """Fresh token inputs for decode step `step` of the layer `layer`.

    Per-head parameters (dt bias, omega; A and D are read from `layer` by the
    caller) stay those of the layer, so the decode loop continues the same
    sequence model.  Draw order: x, B, C, z, lambda; seed 4000 + step.
    """
    device = device or layer.x.device
    batch, _, nheads, rank, headdim = layer.x.shape
    dstate = layer.Bm.shape[-1]
    g = torch.Generator(device=device)
    g.manual_seed(4000 + int(step))
    f32 = dict(device=device, dtype=torch.float32, generator=g)
    iod = layer.x.dtype
    x = torch.randn((batch, nheads, rank, headdim), **f32)
    Bm = torch.randn((batch, nheads, rank, dstate), **f32)
    Cm = torch.randn((batch, nheads, rank, dstate), **f32)
    z = torch.randn((batch, nheads), **f32)
    lam = torch.sigmoid(torch.randn((batch, nheads), **f32))
    dt = torch.nn.functional.softplus(z + layer.dt_bias.to(device))
    theta = dt.unsqueeze(-1) * layer.omega.to(device)
    return StepInputs(
        x=x.to(iod).contiguous(), Bm=_rms_normalise(Bm).to(iod).contiguous(),
        Cm=_rms_normalise(Cm).to(iod).contiguous(), dt=dt.contiguous(),
        lam=lam.contiguous(), theta=theta.contiguous())


def workload_inputs(k: int, device="cpu", **override) -> ScanInputs:
    """Inputs of workload k (seed 1000 + k), optionally with fields overridden
    (e.g. a shorter seqlen for a bounded sample)."""
    w = dict(WORKLOADS[k])
    w.update(override)
    return make_scan_inputs(w["batch"], w["seqlen"], w["nheads"], w["headdim"],
                            w["dstate"], w["rank"], io=w["io"],
                            seed=w.get("seed", 1000 + k), device=device,
                            chunk=w["chunk"])


def make_gate_input(like: torch.Tensor, seed: int) -> torch.Tensor:
    """Output-gate input z shaped and typed like `like` (x of a scan, or x_t
    of a step): N(0, 1) pre-activations, own seed 5000 + seed."""
    g = torch.Generator(device=like.device)
    g.manual_seed(5000 + int(seed))
    z = torch.randn(tuple(like.shape), device=like.device, dtype=torch.float32, generator=g)
    return z.to(like.dtype).contiguous()


@dataclass
class PrologueInputs:
    """Raw projection outputs and block parameters for the fused prologue
    (BCNorm, B/C biases, structured MIMO input and gate)."""
    Bp: torch.Tensor       # [B, L, H, R, N] io dtype: B before the norm
    Cp: torch.Tensor       # [B, L, H, R, N] io dtype
    xp: torch.Tensor       # [B, L, H, P]    io dtype: X' (one vector per token and head)
    zp: torch.Tensor       # [B, L, H, P]    io dtype: Z'
    gB: torch.Tensor       # [H, R, N] fp32 norm gains
    gC: torch.Tensor
    bB: torch.Tensor       # [H, R, N] fp32 biases
    bC: torch.Tensor
    wx: torch.Tensor       # [H, R, P] fp32 structured-input weights
    wz: torch.Tensor


def make_prologue_inputs(batch, seqlen, nheads, headdim, dstate, rank, io="bf16", seed=0,
                         device="cpu") -> PrologueInputs:
    """Draw the prologue's inputs (own seed 6000 + seed).  Draw order: B', C'
    (N(0, 1) times a scale U[0.25, 4] per token, head and rank column, like
    projection outputs of varying size), X', Z' (N(0, 1)), gains U[0.5, 1.5],
    biases 1 + 0.25 N(0, 1) (the all-ones initialisation of App. "B, C Bias
    Parameterization", perturbed), W_X, W_Z (N(0, 1))."""
    g = torch.Generator(device=device)
    g.manual_seed(6000 + int(seed))
    f32 = dict(device=device, dtype=torch.float32, generator=g)
    iod = TORCH_IO[io]
    col = (batch, seqlen, nheads, rank, 1)
    Bp = torch.randn((batch, seqlen, nheads, rank, dstate), **f32) * (torch.rand(col, **f32) * 3.75 + 0.25)
    Cp = torch.randn((batch, seqlen, nheads, rank, dstate), **f32) * (torch.rand(col, **f32) * 3.75 + 0.25)
    xp = torch.randn((batch, seqlen, nheads, headdim), **f32)
    zp = torch.randn((batch, seqlen, nheads, headdim), **f32)
    gB = torch.rand((nheads, rank, dstate), **f32) + 0.5
    gC = torch.rand((nheads, rank, dstate), **f32) + 0.5
    bB = 1.0 + 0.25 * torch.randn((nheads, rank, dstate), **f32)
    bC = 1.0 + 0.25 * torch.randn((nheads, rank, dstate), **f32)
    wx = torch.randn((nheads, rank, headdim), **f32)
    wz = torch.randn((nheads, rank, headdim), **f32)
    return PrologueInputs(Bp=Bp.to(iod).contiguous(), Cp=Cp.to(iod).contiguous(),
                          xp=xp.to(iod).contiguous(), zp=zp.to(iod).contiguous(),
                          gB=gB.contiguous(), gC=gC.contiguous(), bB=bB.contiguous(),
                          bC=bC.contiguous(), wx=wx.contiguous(), wz=wz.contiguous())


def make_prologue_step_inputs(pro: PrologueInputs, batch: int, step: int) -> PrologueInputs:
    """Fresh raw token inputs (B', C' [B,H,R,N], X', Z' [B,H,P]) for decode
    step `step` with the layer's prologue parameters; seed 7000 + step, draw
    order B', C', X', Z'."""
    device = pro.Bp.device
    _, _, nheads, rank, dstate = pro.Bp.shape
    headdim = pro.xp.shape[-1]
    g = torch.Generator(device=device)
    g.manual_seed(7000 + int(step))
    f32 = dict(device=device, dtype=torch.float32, generator=g)
    iod = pro.Bp.dtype
    col = (batch, nheads, rank, 1)
    Bp = torch.randn((batch, nheads, rank, dstate), **f32) * (torch.rand(col, **f32) * 3.75 + 0.25)
    Cp = torch.randn((batch, nheads, rank, dstate), **f32) * (torch.rand(col, **f32) * 3.75 + 0.25)
    xp = torch.randn((batch, nheads, headdim), **f32)
    zp = torch.randn((batch, nheads, headdim), **f32)
    return PrologueInputs(Bp=Bp.to(iod).contiguous(), Cp=Cp.to(iod).contiguous(),
                          xp=xp.to(iod).contiguous(), zp=zp.to(iod).contiguous(),
                          gB=pro.gB, gC=pro.gC, bB=pro.bB, bC=pro.bC, wx=pro.wx, wz=pro.wz)
