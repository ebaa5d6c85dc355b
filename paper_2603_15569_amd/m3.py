"""Python binding of libm3 (ctypes): argument marshalling only.

Every step of the path runs in the HIP kernels behind the C ABI declared in
include/m3.h; PyTorch supplies device memory and the current HIP stream.
There is no fallback: when libm3.so is missing or a call fails, an exception
is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libm3.so")

M3_OK, M3_ERR_NULL, M3_ERR_SHAPE, M3_ERR_DTYPE = 0, 1, 2, 3
M3_ERR_UNSUPPORTED, M3_ERR_ALIGN, M3_ERR_WORKSPACE, M3_ERR_HIP = 4, 5, 6, 7
M3_F32, M3_BF16 = 0, 1
M3_SCAN_SPLIT, M3_SCAN_PER_CHUNK, M3_THETA_PER_HEAD = 1, 2, 4
_IO = {torch.float32: M3_F32, torch.bfloat16: M3_BF16}


class M3Dims(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int64), ("seqlen", ctypes.c_int64),
                ("nheads", ctypes.c_int64), ("headdim", ctypes.c_int64),
                ("dstate", ctypes.c_int64), ("rank", ctypes.c_int64),
                ("chunk", ctypes.c_int64), ("io", ctypes.c_int32),
                ("flags", ctypes.c_int32), ("a_stride_b", ctypes.c_int64),
                ("a_stride_t", ctypes.c_int64), ("a_stride_h", ctypes.c_int64),
                ("seg_chunks", ctypes.c_int64)]


class M3Prologue(ctypes.Structure):
    """m3_prologue: the block prologue fused into the kernels' input loads,
    and the optional output norm fused into the y store."""
    _fields_ = [("bc_norm", ctypes.c_int32), ("eps", ctypes.c_float),
                ("norm_B", ctypes.c_void_p), ("norm_C", ctypes.c_void_p),
                ("bias_B", ctypes.c_void_p), ("bias_C", ctypes.c_void_p),
                ("w_x", ctypes.c_void_p), ("w_z", ctypes.c_void_p),
                ("out_norm", ctypes.c_int32), ("out_group", ctypes.c_int32),
                ("out_eps", ctypes.c_float), ("out_gain", ctypes.c_void_p)]


M3_OUT_NORM_NONE, M3_OUT_NORM_PRE_GATE, M3_OUT_NORM_POST_GATE = 0, 1, 2


class M3Error(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"libm3 status {status}: {msg}")
        self.status = status


EXPORTS = ("m3_scan_workspace_bytes", "m3_scan_fwd", "m3_scan_fwd_gated", "m3_scan_fwd_varlen",
           "m3_scan_varlen_workspace_bytes", "m3_scan_varlen_check",
           "m3_step", "m3_step_gated", "m3_scan_check", "m3_set_wait_limit", "m3_scan_fwd_noalloc",
           "m3_scan_fwd_pro", "m3_step_pro", "m3_scan_bwd", "m3_scan_bwd_workspace_bytes",
           "m3_status_string", "m3_last_hip_error")
SCRATCH_BYTES = 256 << 20   # M3_SCRATCH_BYTES: the allocation-free scan's fixed workspace
CTL_BYTES = 1280            # M3_CTL_BYTES: a scan workspace's control block (zero before first use)
_lib = None


def lib() -> ctypes.CDLL:
    """Load libm3.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -c 'import __graft_entry__ as g; g.build()'`")
        L = ctypes.CDLL(LIB_PATH)
        vp, dims_p = ctypes.c_void_p, ctypes.POINTER(M3Dims)
        L.m3_scan_workspace_bytes.argtypes = [dims_p]
        L.m3_scan_workspace_bytes.restype = ctypes.c_size_t
        L.m3_scan_fwd.argtypes = [dims_p] + [vp] * 15 + [vp, ctypes.c_size_t, vp]
        L.m3_scan_fwd.restype = ctypes.c_int
        L.m3_scan_fwd_gated.argtypes = [dims_p] + [vp] * 16 + [vp, ctypes.c_size_t, vp]
        L.m3_scan_fwd_gated.restype = ctypes.c_int
        L.m3_scan_fwd_varlen.argtypes = ([dims_p, ctypes.POINTER(ctypes.c_int64)] + [vp] * 16
                                         + [vp, ctypes.c_size_t, vp])
        L.m3_scan_fwd_varlen.restype = ctypes.c_int
        i64p = ctypes.POINTER(ctypes.c_int64)
        L.m3_scan_varlen_workspace_bytes.argtypes = [dims_p, i64p]
        L.m3_scan_varlen_workspace_bytes.restype = ctypes.c_size_t
        L.m3_scan_varlen_check.argtypes = [dims_p, i64p, vp, ctypes.c_size_t,
                                           ctypes.POINTER(ctypes.c_uint32), vp]
        L.m3_scan_varlen_check.restype = ctypes.c_int
        L.m3_step.argtypes = [dims_p] + [vp] * 12 + [vp]
        L.m3_step.restype = ctypes.c_int
        L.m3_step_gated.argtypes = [dims_p] + [vp] * 13 + [vp]
        L.m3_step_gated.restype = ctypes.c_int
        pro_p = ctypes.POINTER(M3Prologue)
        L.m3_scan_fwd_pro.argtypes = [dims_p, pro_p] + [vp] * 16 + [vp, ctypes.c_size_t, vp]
        L.m3_scan_fwd_pro.restype = ctypes.c_int
        L.m3_step_pro.argtypes = [dims_p, pro_p] + [vp] * 13 + [vp]
        L.m3_step_pro.restype = ctypes.c_int
        L.m3_scan_bwd_workspace_bytes.argtypes = [dims_p]
        L.m3_scan_bwd_workspace_bytes.restype = ctypes.c_size_t
        L.m3_scan_bwd.argtypes = [dims_p] + [vp] * 20 + [vp, ctypes.c_size_t, vp]
        L.m3_scan_bwd.restype = ctypes.c_int
        L.m3_scan_fwd_noalloc.argtypes = [dims_p] + [vp] * 15 + [vp]
        L.m3_scan_fwd_noalloc.restype = ctypes.c_int
        L.m3_scan_check.argtypes = [dims_p, vp, ctypes.c_size_t, ctypes.POINTER(ctypes.c_uint32), vp]
        L.m3_scan_check.restype = ctypes.c_int
        L.m3_set_wait_limit.argtypes = [ctypes.c_uint32]
        L.m3_set_wait_limit.restype = None
        L.m3_status_string.argtypes = [ctypes.c_int]
        L.m3_status_string.restype = ctypes.c_char_p
        L.m3_last_hip_error.argtypes = []
        L.m3_last_hip_error.restype = ctypes.c_int
        _lib = L
    return _lib


def _check(status: int):
    if status != M3_OK:
        msg = lib().m3_status_string(status).decode()
        if status == M3_ERR_HIP:
            msg += f" (hipError {lib().m3_last_hip_error()})"
        raise M3Error(status, msg)


def _p(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("libm3 takes contiguous tensors")
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _a_strides(A: torch.Tensor, batch: int, seqlen: int, nheads: int):
    """A is per head [H] or per token [B, L, H] (Mamba-3's data-dependent A)."""
    if A.dim() == 1 and A.shape[0] == nheads:
        return 0, 0, 1
    if A.dim() == 3 and tuple(A.shape) == (batch, seqlen, nheads):
        s = A.stride()
        return s[0], s[1], s[2]
    raise ValueError(f"A must be [H] or [B, L, H], got {tuple(A.shape)}")


def _theta_per_head(theta: Optional[torch.Tensor], nheads: int, dstate: int) -> bool:
    """theta given as per-head frequencies omega [H, N/2] (angle = dt * omega)
    rather than per-token angles."""
    return theta is not None and theta.dim() == 2 and tuple(theta.shape) == (nheads, dstate // 2)


def scan_dims(x: torch.Tensor, Bm: torch.Tensor, chunk: int, A: Optional[torch.Tensor] = None,
              split: bool = False, per_chunk: bool = False, seg: int = 0,
              theta_per_head: bool = False) -> M3Dims:
    batch, seqlen, nheads, rank, headdim = x.shape
    dstate = Bm.shape[-1]
    sb, st, sh = _a_strides(A, batch, seqlen, nheads) if A is not None else (0, 0, 1)
    flags = ((M3_SCAN_SPLIT if split else 0) | (M3_SCAN_PER_CHUNK if per_chunk else 0)
             | (M3_THETA_PER_HEAD if theta_per_head else 0))
    return M3Dims(batch, seqlen, nheads, headdim, dstate, rank, int(chunk),
                  _IO[x.dtype], flags, sb, st, sh, int(seg))


def workspace_bytes(dims: M3Dims) -> int:
    return int(lib().m3_scan_workspace_bytes(ctypes.byref(dims)))


class LookBackTimeout(RuntimeError):
    """A single-pass scan's look-back wait gave up: its y and final state are invalid."""


def scan_check(dims: M3Dims, workspace, stream=None) -> int:
    """m3_scan_check: the number of look-back waits that gave up in the last
    scan run with `dims` on `workspace` (synchronises the stream)."""
    n = ctypes.c_uint32(0)
    wsb = workspace.numel() if workspace is not None else 0
    _check(lib().m3_scan_check(ctypes.byref(dims), _p(workspace), wsb, ctypes.byref(n),
                               _stream(stream)))
    return int(n.value)


def set_wait_limit(polls: int) -> None:
    """m3_set_wait_limit: polls before a look-back wait gives up (0: default)."""
    lib().m3_set_wait_limit(int(polls))


def scan_fwd(x, Bm, Cm, dt, A, lam, theta, D, chunk: int,
             init_state=None, init_carry=None, out=None, workspace=None,
             stream=None, split: bool = False, per_chunk: bool = False, seg: int = 0,
             z=None, check: bool = False
             ) -> Tuple[torch.Tensor, torch.Tensor, Tuple[torch.Tensor, torch.Tensor]]:
    """m3_scan_fwd (m3_scan_fwd_gated when the gate input `z`, shaped like x,
    is given: y o SiLU(z)); `theta` is [B,L,H,N/2] per-token angles, or
    [H,N/2] per-head frequencies omega (M3_THETA_PER_HEAD: angle dt * omega).
    Returns y [B,L,H,R,P], final_state [B,H,N,P] fp32
    and the carry (B_{L-1} [B,H,R,N], X_{L-1} [B,H,R,P]).  `out` may supply
    (y, final_state, carryB, carryX) to write into.  Kernel choice: `split`
    (M3_SCAN_SPLIT, three kernels), `per_chunk` (M3_SCAN_PER_CHUNK, one chunk
    per workgroup), else the segmented kernel with `seg` chunks per
    workgroup (0: library choice).  With `check`, the call synchronises and
    raises LookBackTimeout when a look-back wait gave up (m3_scan_check)."""
    d = scan_dims(x, Bm, chunk, A, split, per_chunk, seg,
                  _theta_per_head(theta, x.shape[2], Bm.shape[-1]))
    batch, seqlen, nheads, rank, headdim = x.shape
    dstate = Bm.shape[-1]
    dev = x.device
    if out is None:
        y = torch.empty_like(x)
        fs = torch.empty((batch, nheads, dstate, headdim), dtype=torch.float32, device=dev)
        cB = torch.empty((batch, nheads, rank, dstate), dtype=x.dtype, device=dev)
        cX = torch.empty((batch, nheads, rank, headdim), dtype=x.dtype, device=dev)
    else:
        y, fs, cB, cX = out
    nbytes = workspace_bytes(d)
    if workspace is None and nbytes > 0:
        workspace = torch.zeros(nbytes, dtype=torch.uint8, device=dev)   # control block zero
    icB, icX = (None, None) if init_carry is None else init_carry
    wsb = workspace.numel() if workspace is not None else 0
    if z is None:
        _check(lib().m3_scan_fwd(ctypes.byref(d), _p(x), _p(Bm), _p(Cm), _p(dt), _p(A), _p(lam),
                                 _p(theta), _p(D), _p(init_state), _p(icB), _p(icX), _p(y),
                                 _p(fs), _p(cB), _p(cX), _p(workspace), wsb, _stream(stream)))
    else:
        if z.shape != x.shape or z.dtype != x.dtype:
            raise ValueError("z must have the shape and dtype of x")
        _check(lib().m3_scan_fwd_gated(ctypes.byref(d), _p(x), _p(Bm), _p(Cm), _p(dt), _p(A),
                                       _p(lam), _p(theta), _p(D), _p(z), _p(init_state), _p(icB),
                                       _p(icX), _p(y), _p(fs), _p(cB), _p(cX), _p(workspace), wsb,
                                       _stream(stream)))
    if check:
        n = scan_check(d, workspace, stream)
        if n:
            raise LookBackTimeout(f"{n} look-back wait(s) gave up: y and the final state are invalid")
    return y, fs, (cB, cX)


def scan_fwd_noalloc(x, Bm, Cm, dt, A, lam, theta, D, chunk: int, out,
                     init_state=None, init_carry=None, stream=None, split: bool = False,
                     per_chunk: bool = False, seg: int = 0):
    """m3_scan_fwd_noalloc: the scan with the library's fixed device scratch
    as its workspace (no allocation in the library).  `out` = (y,
    final_state, carryB, carryX) must be given (this call allocates nothing
    either); arguments otherwise as scan_fwd."""
    d = scan_dims(x, Bm, chunk, A, split, per_chunk, seg,
                  _theta_per_head(theta, x.shape[2], Bm.shape[-1]))
    y, fs, cB, cX = out
    icB, icX = (None, None) if init_carry is None else init_carry
    _check(lib().m3_scan_fwd_noalloc(ctypes.byref(d), _p(x), _p(Bm), _p(Cm), _p(dt), _p(A),
                                     _p(lam), _p(theta), _p(D), _p(init_state), _p(icB), _p(icX),
                                     _p(y), _p(fs), _p(cB), _p(cX), _stream(stream)))
    return y, fs, (cB, cX)


def varlen_dims(x, Bm, A, chunk: int, cu, split: bool = False, per_chunk: bool = False,
                seg: int = 0, theta=None) -> M3Dims:
    T, nheads, rank, headdim = x.shape
    dstate = Bm.shape[-1]
    S = len(cu) - 1
    if A.dim() == 1 and A.shape[0] == nheads:
        sb, st, sh = 0, 0, 1
    elif A.dim() == 2 and tuple(A.shape) == (T, nheads):
        sb, (st, sh) = 0, A.stride()
    else:
        raise ValueError(f"A must be [H] or [T, H], got {tuple(A.shape)}")
    ph = theta is not None and _theta_per_head(theta, nheads, dstate)
    flags = ((M3_SCAN_SPLIT if split else 0) | (M3_SCAN_PER_CHUNK if per_chunk else 0)
             | (M3_THETA_PER_HEAD if ph else 0))
    return M3Dims(S, T, nheads, headdim, dstate, rank, int(chunk), _IO[x.dtype], flags, sb, st, sh,
                  int(seg))


def _cu_list(cu_seqlens):
    return [int(v) for v in (cu_seqlens.tolist() if hasattr(cu_seqlens, "tolist") else cu_seqlens)]


def varlen_workspace_bytes(dims: M3Dims, cu_seqlens) -> int:
    """m3_scan_varlen_workspace_bytes: the workspace of the one-launch varlen
    scan (0: it does not apply)."""
    cu = _cu_list(cu_seqlens)
    return int(lib().m3_scan_varlen_workspace_bytes(ctypes.byref(dims), (ctypes.c_int64 * len(cu))(*cu)))


def varlen_check(dims: M3Dims, cu_seqlens, workspace, stream=None) -> int:
    """m3_scan_varlen_check: look-back timeouts of the last varlen call on
    `workspace` (synchronises the stream)."""
    cu = _cu_list(cu_seqlens)
    n = ctypes.c_uint32(0)
    wsb = workspace.numel() if workspace is not None else 0
    _check(lib().m3_scan_varlen_check(ctypes.byref(dims), (ctypes.c_int64 * len(cu))(*cu),
                                      _p(workspace), wsb, ctypes.byref(n), _stream(stream)))
    return int(n.value)


def scan_fwd_varlen(x, Bm, Cm, dt, A, lam, theta, D, chunk: int, cu_seqlens,
                    init_state=None, init_carry=None, z=None, workspace=None, stream=None,
                    split: bool = False, per_chunk: bool = False, seg: int = 0,
                    check: bool = False):
    """m3_scan_fwd_varlen: sequences packed along the token axis, x [T,H,R,P],
    Bm/Cm [T,H,R,N], dt/lam [T,H], theta [T,H,N/2] (or [H,N/2] frequencies),
    A [H] or [T,H]; `cu_seqlens` (S + 1 offsets, host list or tensor).  Returns
    y [T,H,R,P], final_state [S,H,N,P] and the carry ([S,H,R,N], [S,H,R,P]).
    Without a workspace one is allocated (zero-filled) for the one-launch
    scan where that applies, else for the largest sequence."""
    cu = [int(v) for v in (cu_seqlens.tolist() if hasattr(cu_seqlens, "tolist") else cu_seqlens)]
    T, nheads, rank, headdim = x.shape
    dstate = Bm.shape[-1]
    S = len(cu) - 1
    if A.dim() == 1 and A.shape[0] == nheads:
        sb, st, sh = 0, 0, 1
    elif A.dim() == 2 and tuple(A.shape) == (T, nheads):
        sb, (st, sh) = 0, A.stride()
    else:
        raise ValueError(f"A must be [H] or [T, H], got {tuple(A.shape)}")
    flags = ((M3_SCAN_SPLIT if split else 0) | (M3_SCAN_PER_CHUNK if per_chunk else 0)
             | (M3_THETA_PER_HEAD if _theta_per_head(theta, nheads, dstate) else 0))
    d = M3Dims(S, T, nheads, headdim, dstate, rank, int(chunk), _IO[x.dtype], flags, sb, st, sh,
               int(seg))
    dev = x.device
    y = torch.empty_like(x)
    fs = torch.empty((S, nheads, dstate, headdim), dtype=torch.float32, device=dev)
    cB = torch.empty((S, nheads, rank, dstate), dtype=x.dtype, device=dev)
    cX = torch.empty((S, nheads, rank, headdim), dtype=x.dtype, device=dev)
    if workspace is None:
        one = varlen_workspace_bytes(d, cu)
        if one == 0:
            longest = max([cu[i + 1] - cu[i] for i in range(S)] + [0])
            d1 = M3Dims(1, longest, nheads, headdim, dstate, rank, int(chunk), _IO[x.dtype], flags,
                        0, st, sh, int(seg))
            one = workspace_bytes(d1)
        workspace = torch.zeros(max(one, 16), dtype=torch.uint8, device=dev)
    icB, icX = (None, None) if init_carry is None else init_carry
    cu_arr = (ctypes.c_int64 * len(cu))(*cu)
    _check(lib().m3_scan_fwd_varlen(ctypes.byref(d), cu_arr, _p(x), _p(Bm), _p(Cm), _p(dt), _p(A),
                                    _p(lam), _p(theta), _p(D), _p(z), _p(init_state), _p(icB),
                                    _p(icX), _p(y), _p(fs), _p(cB), _p(cX), _p(workspace),
                                    workspace.numel(), _stream(stream)))
    if check:
        n = varlen_check(d, cu, workspace, stream)
        if n:
            raise LookBackTimeout(f"{n} look-back wait(s) gave up: y and the final state are invalid")
    return y, fs, (cB, cX)


def step_dims(x_t: torch.Tensor, B_t: torch.Tensor, A: torch.Tensor,
              theta_per_head: bool = False) -> M3Dims:
    batch, nheads, rank, headdim = x_t.shape
    dstate = B_t.shape[-1]
    if A.dim() == 1 and A.shape[0] == nheads:
        sb, sh = 0, 1
    elif A.dim() == 2 and tuple(A.shape) == (batch, nheads):
        sb, sh = A.stride()
    else:
        raise ValueError(f"A must be [H] or [B, H], got {tuple(A.shape)}")
    return M3Dims(batch, 1, nheads, headdim, dstate, rank, 1, _IO[x_t.dtype],
                  M3_THETA_PER_HEAD if theta_per_head else 0, sb, 0, sh, 0)


def step(state, carry, x_t, B_t, C_t, dt_t, A, lam_t, theta_t, D, y=None, stream=None, z=None):
    """m3_step (m3_step_gated when the gate input `z`, shaped like x_t, is
    given: y_t o SiLU(z_t); `theta_t` [B,H,N/2] angles or [H,N/2] frequencies
    omega, as in scan_fwd): advances `state` [B,H,N,P] and `carry`
    (B [B,H,R,N], X [B,H,R,P]) in place by one token; returns y_t [B,H,R,P]."""
    d = step_dims(x_t, B_t, A, _theta_per_head(theta_t, x_t.shape[1], B_t.shape[-1]))
    if y is None:
        y = torch.empty_like(x_t)
    cB, cX = carry
    if z is None:
        _check(lib().m3_step(ctypes.byref(d), _p(state), _p(cB), _p(cX), _p(x_t), _p(B_t),
                             _p(C_t), _p(dt_t), _p(A), _p(lam_t), _p(theta_t), _p(D), _p(y),
                             _stream(stream)))
    else:
        if z.shape != x_t.shape or z.dtype != x_t.dtype:
            raise ValueError("z must have the shape and dtype of x_t")
        _check(lib().m3_step_gated(ctypes.byref(d), _p(state), _p(cB), _p(cX), _p(x_t), _p(B_t),
                                   _p(C_t), _p(dt_t), _p(A), _p(lam_t), _p(theta_t), _p(D), _p(z),
                                   _p(y), _stream(stream)))
    return y


def prologue(bc_norm: bool = False, eps: float = 1e-6, norm_B=None, norm_C=None, bias_B=None,
             bias_C=None, w_x=None, w_z=None, out_norm: int = M3_OUT_NORM_NONE,
             out_group: int = 0, out_eps: float = 1e-6, out_gain=None) -> M3Prologue:
    """An m3_prologue over fp32 device tables: gains and biases [H,R,N],
    w_x / w_z [H,R,P] (None: not applied); the output norm (M3_OUT_NORM_*)
    over groups of out_group channels with gain out_gain [H,R,P] (None:
    ones)."""
    for t in (norm_B, norm_C, bias_B, bias_C, w_x, w_z, out_gain):
        if t is not None and t.dtype != torch.float32:
            raise ValueError("prologue tables are fp32")
    return M3Prologue(1 if bc_norm else 0, float(eps), _p(norm_B), _p(norm_C), _p(bias_B),
                      _p(bias_C), _p(w_x), _p(w_z), int(out_norm), int(out_group),
                      float(out_eps), _p(out_gain))


def scan_fwd_pro(x, Bm, Cm, dt, A, lam, theta, D, chunk: int, pro: M3Prologue, rank: int,
                 z=None, init_state=None, init_carry=None, out=None, workspace=None,
                 stream=None, check: bool = False, seg: int = 0):
    """m3_scan_fwd_pro: the scan with the block prologue `pro` applied to the
    raw B', C' [B,L,H,R,N] and to x (X' [B,L,H,P] when pro.w_x is set, else
    [B,L,H,R,P]) and z as they are read.  Returns y [B,L,H,R,P], the final
    state and the carry (the prologue's B_{L-1}, X_{L-1}).  `seg` is the
    dims' seg_chunks (0: chosen at launch; at least the chunk count: one
    segment per slice, the warp-specialised kernel where it is built)."""
    batch, seqlen, nheads = x.shape[:3]
    headdim, dstate = x.shape[-1], Bm.shape[-1]
    if tuple(Bm.shape) != (batch, seqlen, nheads, rank, dstate):
        raise ValueError("B must be [B, L, H, R, N]")
    sb, st, sh = _a_strides(A, batch, seqlen, nheads)
    flags = M3_THETA_PER_HEAD if _theta_per_head(theta, nheads, dstate) else 0
    d = M3Dims(batch, seqlen, nheads, headdim, dstate, rank, int(chunk), _IO[x.dtype], flags,
               sb, st, sh, int(seg))
    dev = x.device
    if out is None:
        y = torch.empty((batch, seqlen, nheads, rank, headdim), dtype=x.dtype, device=dev)
        fs = torch.empty((batch, nheads, dstate, headdim), dtype=torch.float32, device=dev)
        cB = torch.empty((batch, nheads, rank, dstate), dtype=x.dtype, device=dev)
        cX = torch.empty((batch, nheads, rank, headdim), dtype=x.dtype, device=dev)
    else:
        y, fs, cB, cX = out
    nbytes = workspace_bytes(d)
    if workspace is None and nbytes > 0:
        workspace = torch.zeros(nbytes, dtype=torch.uint8, device=dev)   # control block zero
    icB, icX = (None, None) if init_carry is None else init_carry
    wsb = workspace.numel() if workspace is not None else 0
    _check(lib().m3_scan_fwd_pro(ctypes.byref(d), ctypes.byref(pro), _p(x), _p(Bm), _p(Cm),
                                 _p(dt), _p(A), _p(lam), _p(theta), _p(D), _p(z),
                                 _p(init_state), _p(icB), _p(icX), _p(y), _p(fs), _p(cB), _p(cX),
                                 _p(workspace), wsb, _stream(stream)))
    if check:
        n = scan_check(d, workspace, stream)
        if n:
            raise LookBackTimeout(f"{n} look-back wait(s) gave up: y and the final state are invalid")
    return y, fs, (cB, cX)


def step_pro(state, carry, x_t, B_t, C_t, dt_t, A, lam_t, theta_t, D, pro: M3Prologue,
             z=None, y=None, stream=None):
    """m3_step_pro: one decode step with the block prologue; x_t (z) is
    [B,H,P] when pro.w_x (pro.w_z) is set.  Returns y_t [B,H,R,P]."""
    batch, nheads, rank, dstate = B_t.shape
    headdim = x_t.shape[-1]
    if A.dim() == 1 and A.shape[0] == nheads:
        sb, sh = 0, 1
    elif A.dim() == 2 and tuple(A.shape) == (batch, nheads):
        sb, sh = A.stride()
    else:
        raise ValueError(f"A must be [H] or [B, H], got {tuple(A.shape)}")
    flags = M3_THETA_PER_HEAD if _theta_per_head(theta_t, nheads, dstate) else 0
    d = M3Dims(batch, 1, nheads, headdim, dstate, rank, 1, _IO[x_t.dtype], flags, sb, 0, sh, 0)
    if y is None:
        y = torch.empty((batch, nheads, rank, headdim), dtype=x_t.dtype, device=x_t.device)
    cB, cX = carry
    _check(lib().m3_step_pro(ctypes.byref(d), ctypes.byref(pro), _p(state), _p(cB), _p(cX),
                             _p(x_t), _p(B_t), _p(C_t), _p(dt_t), _p(A), _p(lam_t), _p(theta_t),
                             _p(D), _p(z), _p(y), _stream(stream)))
    return y


def scan_bwd(x, Bm, Cm, dt, A, lam, theta, D, dy, chunk: int, dfinal=None, init_state=None,
             want_dinit: bool = False, workspace=None, stream=None):
    """m3_scan_bwd: gradients of J = <dy, y> + <dfinal, final_state> for the
    scan of these inputs.  Returns a dict: dx, dB, dC (io dtype), ddt, dlam,
    dtheta, dD, dA ([H] for a per-head A, [B,L,H] for a per-token A) and
    dinit (when `want_dinit`)."""
    d = scan_dims(x, Bm, chunk, A)
    batch, seqlen, nheads, rank, headdim = x.shape
    dstate = Bm.shape[-1]
    dev = x.device
    f32 = dict(dtype=torch.float32, device=dev)
    out = dict(dx=torch.empty_like(x), dB=torch.empty_like(Bm), dC=torch.empty_like(Cm),
               ddt=torch.empty((batch, seqlen, nheads), **f32),
               dlam=torch.empty((batch, seqlen, nheads), **f32),
               dtheta=torch.empty((batch, seqlen, nheads, dstate // 2), **f32),
               dD=torch.empty((nheads,), **f32),
               dA=torch.empty((nheads,) if A.dim() == 1 else (batch, seqlen, nheads), **f32))
    dinit = torch.empty((batch, nheads, dstate, headdim), **f32) if want_dinit else None
    if dinit is not None:
        out["dinit"] = dinit
    nbytes = int(lib().m3_scan_bwd_workspace_bytes(ctypes.byref(d)))
    if workspace is None:
        workspace = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=dev)
    _check(lib().m3_scan_bwd(ctypes.byref(d), _p(x), _p(Bm), _p(Cm), _p(dt), _p(A), _p(lam),
                             _p(theta), _p(D), _p(init_state), _p(dy), _p(dfinal),
                             _p(out["dx"]), _p(out["dB"]), _p(out["dC"]), _p(out["ddt"]),
                             _p(out["dA"]), _p(out["dlam"]), _p(out["dtheta"]), _p(out["dD"]),
                             _p(dinit), _p(workspace), workspace.numel(), _stream(stream)))
    return out
