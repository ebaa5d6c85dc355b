"""Algorithmic FLOP and byte counts of the hot path and MI355X peaks.

Counts follow the paper's own accounting:
* decode arithmetic intensity, Tab. arith_intensity (SISO and MIMO, 2-byte
  data), Sec. 3.3 "Decoding Arithmetic Intensity";
* chunked-algorithm FLOPs, Sec. 3.3 "Chunked Algorithm for MIMO SSMs":
  intra-chunk 2 (T/C) (CR)^2 (N+P), inter-chunk 4 (T/C) N P (CR) + 2 (T/C) N P.
Bytes are algorithmic: every input read once, every output written once;
chunk-state round trips inside an implementation are not counted.
"""
from __future__ import annotations

# MI355X published peaks (dense).
HBM_BYTES_PER_S = 8.0e12
MFMA_BF16_FLOPS = 2.5e15
MFMA_FP32_FLOPS = 157.3e12
VALU_FP32_FLOPS = 157.3e12


def decode_ai_siso(N: int, P: int) -> float:
    """FLOPs / bytes of one SISO decode step, 2-byte data (Tab. arith_intensity (a))."""
    return (5 * N * P - P) / (2 * (1 + 2 * N + P + N * P))


def decode_ai_mimo(N: int, P: int, R: int) -> float:
    """FLOPs / bytes of one MIMO decode step, 2-byte data (Tab. arith_intensity (b))."""
    return (4 * N * P * R + N * P - P * R) / (2 * (1 + 2 * N * R + P * R + N * P))


def chunked_flops(T: int, N: int, P: int, R: int, C: int) -> float:
    """FLOPs of the chunked algorithm over T tokens of one head (Sec. 3.3)."""
    nch = T / C
    intra = 2 * nch * (C * R) ** 2 * (N + P)
    inter = 4 * nch * N * P * (C * R) + 2 * nch * N * P
    return intra + inter


def prefill_bytes(batch: int, L: int, H: int, N: int, P: int, R: int, io_bytes: int) -> int:
    """Algorithmic HBM bytes of one prefill scan: x, B, C read and y written in
    the io dtype; dt, lambda and theta (N/2 angles) read as fp32; the final
    fp32 state and the carry written once.  A and D (per head) are negligible
    and not counted."""
    per_token_head = R * (2 * N + 2 * P) * io_bytes + 4 + 4 + 4 * (N // 2)
    tail = batch * H * (N * P * 4 + R * (N + P) * io_bytes)
    return batch * L * H * per_token_head + tail


def decode_bytes_per_slice(N: int, P: int, R: int, io_bytes: int) -> int:
    """Algorithmic HBM bytes of one decode step per (batch, head): the fp32
    state read and written, the carry (B_{t-1}, X_{t-1}) read and rewritten,
    the step inputs x, B, C (io dtype), dt, lambda and N/2 angles (fp32), and
    y written."""
    state = 2 * N * P * 4
    carry = 2 * R * (N + P) * io_bytes
    inputs = R * (P + 2 * N) * io_bytes + 8 + 4 * (N // 2)
    out = R * P * io_bytes
    return state + carry + inputs + out


def decode_flops_per_slice(N: int, P: int, R: int) -> int:
    """FLOPs of one decode step per (batch, head) as the kernel computes it:
    two rank-R outer products (2 N P R each), the rotation and decay of the
    state (6 N P / 2 ... 3 N P), the rank-R output contraction (2 N P R), the
    skip term (2 P R)."""
    return 2 * N * P * R * 3 + 3 * N * P + 2 * P * R


def backward_bytes(batch: int, L: int, H: int, N: int, P: int, R: int, io_bytes: int) -> int:
    """Algorithmic HBM bytes of one backward scan: the forward's inputs x, B, C
    (io dtype), dt, lambda and N/2 angles (fp32) and dy (io dtype) read once;
    dx, dB, dC (io dtype), ddt, dlambda and the N/2 angle gradients (fp32)
    written once; dJ/d(final state) read once (fp32).  Per-head A, D and their
    gradients are negligible and not counted."""
    per_token_head_in = R * (2 * N + 2 * P) * io_bytes + 4 + 4 + 4 * (N // 2)
    per_token_head_out = R * (2 * N + P) * io_bytes + 4 + 4 + 4 * (N // 2)
    return batch * L * H * (per_token_head_in + per_token_head_out) + batch * H * N * P * 4


def backward_flops(T: int, N: int, P: int, R: int, C: int) -> float:
    """Matrix-product FLOPs of the chunked backward over T tokens of one head,
    counted like the forward's (Sec. 3.3): per chunk of CR rows, the two
    state-sized contractions of the recomputed forward aggregate and of the
    reverse state input (2 x 2 N P CR), the scores C^ B^T and the two
    orientations of dy x^T (2 (CR)^2 (N + 2P)), the three products with the
    masked scores (dx, dB^, dC^: 2 (CR)^2 (P + 2N)), and the four products with
    the state maps (B^ U, x U^T, dy S^T: 2 CR N P each, and the forward
    aggregate's second operand) — 2 (CR)^2 (3N + 3P) + 12 N P CR in all."""
    nch = T / C
    return nch * (2 * (C * R) ** 2 * (3 * N + 3 * P) + 12 * N * P * (C * R))


def prologue_prefill_bytes(batch: int, L: int, H: int, N: int, P: int, R: int, io_bytes: int) -> int:
    """Algorithmic HBM bytes of a prefill scan with the block prologue and the
    structured MIMO input: as prefill_bytes, but x is read as X' (P values per
    token and head instead of P x R); the raw B', C' have the size of B, C;
    the per-head tables are negligible."""
    return prefill_bytes(batch, L, H, N, P, R, io_bytes) - batch * L * H * (R - 1) * P * io_bytes
