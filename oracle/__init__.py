"""CPU oracle for the Mamba-3 SSM hot path (fp64, plain sequential recurrence).

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU
baseline may import it; the library and its Python binding never do.  It
shares no code with the HIP path.  The arithmetic lives in m3_oracle.c (see
its header for the equations and the readings of the paper it follows); this
module builds it with gcc, marshals arrays and extracts (batch, head) slices
from tensors in the library layout.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "m3_oracle.c")
_LIB = os.path.join(_HERE, "libm3_oracle.so")
_LIB_NATIVE = os.path.join(_HERE, "libm3_oracle_native.so")
_lib = None
_lib_path = _LIB
BUILD_FLAGS = ["-O3", "-fopenmp", "-shared", "-fPIC", "-std=c11"]


def build(force: bool = True, native: bool = False) -> str:
    """Compile the oracle with gcc -O3 (OpenMP over slices).  The default
    target ISA is the portable x86-64-v3, so the library built here runs on
    any AVX2 host; `native` builds a -march=native copy for the host it runs
    on (the CPU baseline's timing build, made where it is timed)."""
    out = _LIB_NATIVE if native else _LIB
    if force or not os.path.exists(out):
        tmp = out + f".tmp{os.getpid()}"
        march = "-march=native" if native else "-march=x86-64-v3"
        subprocess.run(["gcc", *BUILD_FLAGS, march, _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, out)
    return out


def use_native() -> str:
    """Build the -march=native copy on this host and route every later call
    through it; returns the gcc flags used."""
    global _lib, _lib_path
    build(force=True, native=True)
    _lib, _lib_path = None, _LIB_NATIVE
    return " ".join(["gcc", *BUILD_FLAGS, "-march=native"])


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_lib_path):
            build(native=_lib_path == _LIB_NATIVE)
        lib = ctypes.CDLL(_lib_path)
        i64, dp, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
        lib.m3o_scan.argtypes = [i64] * 5 + [dp] * 8 + [dp] * 3 + [dp] * 4 + [ci]
        lib.m3o_scan.restype = ci
        lib.m3o_step.argtypes = [i64] * 4 + [dp] * 3 + [dp] * 8 + [dp, ci]
        lib.m3o_step.restype = ci
        lib.m3o_scan_bwd.argtypes = [i64] * 5 + [dp] * 9 + [dp] * 2 + [dp] * 9 + [ci]
        lib.m3o_scan_bwd.restype = ci
        _lib = lib
    return _lib


def _f64(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a):
    return None if a is None else a.ctypes.data


def scan(x, B, C, dt, A, lam, theta, D, init_state=None, init_B=None,
         init_X=None, nthreads=0, return_threads=False):
    """Sequential scan over S independent slices.

    x [S,L,R,P], B/C [S,L,R,N], dt/A/lam [S,L], theta [S,L,N/2], D [S],
    optional init_state [S,N,P] and carry init_B [S,R,N], init_X [S,R,P].
    Returns y [S,L,R,P], state [S,N,P], carryB [S,R,N], carryX [S,R,P].
    """
    x, B, C = _f64(x), _f64(B), _f64(C)
    dt, A, lam, theta, D = _f64(dt), _f64(A), _f64(lam), _f64(theta), _f64(D)
    S, L, R, P = x.shape
    N = B.shape[-1]
    assert B.shape == (S, L, R, N) and C.shape == (S, L, R, N)
    assert dt.shape == (S, L) and A.shape == (S, L) and lam.shape == (S, L)
    assert theta.shape == (S, L, N // 2) and D.shape == (S,)
    if (init_B is None) != (init_X is None):
        raise ValueError("give both carry halves or neither")
    init_state = None if init_state is None else _f64(init_state)
    init_B = None if init_B is None else _f64(init_B)
    init_X = None if init_X is None else _f64(init_X)
    y = np.empty((S, L, R, P))
    state = np.empty((S, N, P))
    cB = np.empty((S, R, N))
    cX = np.empty((S, R, P))
    used = _load().m3o_scan(S, L, N, P, R, _ptr(x), _ptr(B), _ptr(C), _ptr(dt),
                            _ptr(A), _ptr(lam), _ptr(theta), _ptr(D),
                            _ptr(init_state), _ptr(init_B), _ptr(init_X),
                            _ptr(y), _ptr(state), _ptr(cB), _ptr(cX),
                            int(nthreads))
    out = (y, state, cB, cX)
    return (out, used) if return_threads else out


def scan_bwd(x, B, C, dt, A, lam, theta, D, dy, dfinal=None, init_state=None, nthreads=0):
    """Gradients of J = <dy, y> + <dfinal, final_state> for the scan on S
    slices (no initial carry), by reverse mode through the sequential
    recurrence (m3o_scan_bwd).  Shapes as scan(); dy like y, dfinal like the
    state.  Returns a dict: dx, dB, dC, ddt, dA (per token), dlam, dtheta,
    dD [S], dinit [S,N,P]."""
    x, B, C = _f64(x), _f64(B), _f64(C)
    dt, A, lam, theta, D, dy = _f64(dt), _f64(A), _f64(lam), _f64(theta), _f64(D), _f64(dy)
    S, L, R, P = x.shape
    N = B.shape[-1]
    assert dy.shape == x.shape and theta.shape == (S, L, N // 2)
    dfinal = None if dfinal is None else _f64(dfinal)
    init_state = None if init_state is None else _f64(init_state)
    out = dict(dx=np.empty_like(x), dB=np.empty_like(B), dC=np.empty_like(C),
               ddt=np.empty_like(dt), dA=np.empty_like(A), dlam=np.empty_like(lam),
               dtheta=np.empty_like(theta), dD=np.empty(S), dinit=np.empty((S, N, P)))
    _load().m3o_scan_bwd(S, L, N, P, R, _ptr(x), _ptr(B), _ptr(C), _ptr(dt), _ptr(A),
                         _ptr(lam), _ptr(theta), _ptr(D), _ptr(init_state), _ptr(dy),
                         _ptr(dfinal), _ptr(out["dx"]), _ptr(out["dB"]), _ptr(out["dC"]),
                         _ptr(out["ddt"]), _ptr(out["dA"]), _ptr(out["dlam"]),
                         _ptr(out["dtheta"]), _ptr(out["dD"]), _ptr(out["dinit"]),
                         int(nthreads))
    return out


def step(state, carryB, carryX, x, B, C, dt, A, lam, theta, D, nthreads=0):
    """One decode step on S slices.  Returns (y [S,R,P], state', carryB',
    carryX'); the inputs are not modified."""
    state, carryB, carryX = _f64(state).copy(), _f64(carryB).copy(), _f64(carryX).copy()
    x, B, C = _f64(x), _f64(B), _f64(C)
    dt, A, lam, theta, D = _f64(dt), _f64(A), _f64(lam), _f64(theta), _f64(D)
    S, R, P = x.shape
    N = B.shape[-1]
    assert state.shape == (S, N, P) and theta.shape == (S, N // 2)
    y = np.empty((S, R, P))
    _load().m3o_step(S, N, P, R, _ptr(state), _ptr(carryB), _ptr(carryX),
                     _ptr(x), _ptr(B), _ptr(C), _ptr(dt), _ptr(A), _ptr(lam),
                     _ptr(theta), _ptr(D), _ptr(y), int(nthreads))
    return y, state, carryB, carryX


# ---------------------------------------------------------------------------
# Output gate (App. "MIMO for Mamba-3", paragraph "Mamba with MIMO": the
# block's residual function phi(Y, Z) = Y o SiLU(Z), Z shaped like X).
# ---------------------------------------------------------------------------

def silu(z):
    """SiLU(z) = z / (1 + e^{-z}), elementwise, fp64 (exp overflow for very
    negative z gives the correct limit -0)."""
    z = _f64(z)
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def gate(y, z):
    """phi(Y, Z) = Y o SiLU(Z): the SSM output (D skip included, the Mamba
    order) times SiLU of the gate input, elementwise, fp64."""
    return _f64(y) * silu(z)


# ---------------------------------------------------------------------------
# Block prologue: the cheap per-token operations of the Mamba-3 block that
# produce the SSM's B, C, X (and the gate's Z) from the projections' outputs.
#   * BCNorm (Sec. 3.4, paragraph "BC / QK Normalization"): an RMS
#     normalisation of B and C after their projection, here over the state
#     axis N of every (token, head, rank-column), with an optional per-channel
#     gain;
#   * B, C biases (Sec. 3.4, paragraph "B, C Biases"; App. "B, C Bias
#     Parameterization"): head-specific, channel-wise, added after the norm;
#   * structured MIMO input (App. "MIMO for Mamba-3", paragraph "Mamba with
#     MIMO"): X_t = contract(PR, P -> PR)(W_X, X'_t), i.e. X_t[p, r] =
#     W_X[p, r] X'_t[p]; the gate input Z is formed the same way from Z'.
# All in fp64.
# ---------------------------------------------------------------------------

def rms_norm(v, gain=None, bias=None, eps=1e-6):
    """v [..., N] -> gain * v / sqrt(mean_N(v^2) + eps) + bias, the mean over
    the last (state) axis of each vector.  gain and bias broadcast against v
    (per head, rank and channel); None means ones / zeros."""
    v = _f64(v)
    out = v / np.sqrt(np.mean(v * v, axis=-1, keepdims=True) + eps)
    if gain is not None:
        out = out * _f64(gain)
    if bias is not None:
        out = out + _f64(bias)
    return out


def add_bias(v, bias):
    """The bias alone (no norm): v + bias, broadcast."""
    return _f64(v) if bias is None else _f64(v) + _f64(bias)


def structured_input(xp, w):
    """X_t[r, p] = W[r, p] X'_t[p] for every token: xp [S, L, P] (one P-vector
    per token and head), w [S, R, P] (the head's weights, one row per rank)
    -> [S, L, R, P]."""
    xp, w = _f64(xp), _f64(w)
    return w[:, None, :, :] * xp[:, :, None, :]


# ---------------------------------------------------------------------------
# Optional output norm of the block (Sec. 4, hybrid models; App. table of the
# norm type and placement ablation): a grouped RMS normalisation of the SSM
# output, either before the output gate (pre-gate: g o norm(Y) o SiLU(Z)) or
# after it (post-gate: g o norm(Y o SiLU(Z))).  Grouped: the mean of squares
# runs over `group` consecutive channels of one (token, head, rank) row of Y
# (the paper gives no group size: it is a parameter here, group = headdim
# being one RMS per row).  fp64.
# ---------------------------------------------------------------------------

def group_rms(v, group, eps):
    """v [..., P] -> v / sqrt(mean of squares over each run of `group`
    consecutive channels + eps), P a multiple of group."""
    v = _f64(v)
    P = v.shape[-1]
    if group <= 0 or P % group:
        raise ValueError("group must divide the channel count")
    g = v.reshape(v.shape[:-1] + (P // group, group))
    out = g / np.sqrt(np.mean(g * g, axis=-1, keepdims=True) + eps)
    return out.reshape(v.shape)


def out_norm(y, group, eps=1e-6, gain=None, z=None, pre_gate=True):
    """Output norm of the block: y [..., P] (the SSM output, D skip
    included), z like y or None (no output gate), gain broadcast against y
    (per head, rank and channel; None: ones).  pre_gate: gain o
    group_rms(y) o SiLU(z); else gain o group_rms(y o SiLU(z))."""
    y = _f64(y)
    if pre_gate:
        out = group_rms(y, group, eps)
        if gain is not None:
            out = out * _f64(gain)
        return out if z is None else out * silu(z)
    u = y if z is None else y * silu(z)
    out = group_rms(u, group, eps)
    return out if gain is None else out * _f64(gain)


# ---------------------------------------------------------------------------
# Slice extraction from tensors in the library layout.
# ---------------------------------------------------------------------------

def _np(t):
    """torch tensor (any device, any float dtype) or array -> fp64 numpy,
    exactly (bf16 values are representable in fp64)."""
    try:
        import torch
        if isinstance(t, torch.Tensor):
            return t.detach().to("cpu", torch.float64).numpy()
    except ImportError:  # pragma: no cover
        pass
    return np.asarray(t, dtype=np.float64)


def slices_of_scan(x, Bm, Cm, dt, A, lam, theta, D, slices, t0=0, t1=None):
    """Gather the oracle's per-slice arrays for (b, h) pairs in `slices` from
    library-layout tensors x [B,L,H,R,P], Bm/Cm [B,L,H,R,N], dt/lam [B,L,H],
    A [H] (per head), theta [B,L,H,N/2], D [H]; tokens t0..t1."""
    t1 = x.shape[1] if t1 is None else t1
    bs = [b for b, _ in slices]
    hs = [h for _, h in slices]

    def take(t):
        # stack of t[b, t0:t1, h, ...] over (b, h) in slices
        return np.stack([_np(t[b, t0:t1, h]) for b, h in zip(bs, hs)])

    xs, Bs, Cs = take(x), take(Bm), take(Cm)
    dts, lams, ths = take(dt), take(lam), take(theta)
    A_np, D_np = _np(A), _np(D)
    As = np.repeat(A_np[hs][:, None], dts.shape[1], axis=1)
    Ds = D_np[hs]
    return dict(x=xs, B=Bs, C=Cs, dt=dts, A=As, lam=lams, theta=ths, D=Ds)


def slices_of_state(t, slices):
    """state-like tensor [B,H,...] -> numpy [S,...] for the given (b, h)."""
    return np.stack([_np(t[b, h]) for b, h in slices])


def slices_of_step(x, Bm, Cm, dt, lam, theta, slices):
    """Per-step tensors x [B,H,R,P], Bm/Cm [B,H,R,N], dt/lam [B,H],
    theta [B,H,N/2] -> per-slice arrays."""
    return dict(x=slices_of_state(x, slices), B=slices_of_state(Bm, slices),
                C=slices_of_state(Cm, slices),
                dt=np.array([_np(dt[b, h]) for b, h in slices], dtype=np.float64).reshape(-1),
                lam=np.array([_np(lam[b, h]) for b, h in slices], dtype=np.float64).reshape(-1),
                theta=slices_of_state(theta, slices))


def rel_err(got, ref):
    """Infinity-norm relative error max|got - ref| / max|ref| (0 if both are
    zero).  Applied per slice by the parity tests."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.max(np.abs(ref)) if ref.size else 0.0
    num = np.max(np.abs(got - ref)) if ref.size else 0.0
    if den == 0.0:
        return float(num)
    return float(num / den)
