"""Independent statements of the Mamba-3 SSM, used only to pin the oracle.

Each function restates one form the paper gives for the same layer, written
from that form and not from the oracle's step loop:

* masked_form   - the parallel (SSD) form Y = (L o C B^T) X with Mamba-3's
                  mask L = (1-semiseparable decay) x (2-band) (Sec. 3.1.2,
                  eq. mamba3-mask) and the rotary ("RoPE trick") rotation of
                  B and C by the cumulative angle (Sec. 3.2, Props.
                  "Data-Dependent RoPE Equivalence" and "Rotary Embedding
                  Equivalence with Exponential-Trapezoidal Discretization").
* complex_form  - the complex-valued state in C^{N/2} (App. proof of the
                  trapezoid/RoPE proposition, eq. trap-complex), with
                  B = B_re + i B_im, C = C_re - i C_im (Sec. 3.2, the real
                  projections [B; B_hat], [C; -C_hat]).
* euler_complex - the two-term exponential-Euler recurrence of Mamba-2 with
                  a rotating state (Sec. 3.1, eq. mamba2-recurrence), the
                  lambda = 1 case.
* mamba2_masked - Mamba-2's mask 1-SS(alpha) Diag(gamma) (Sec. 2.2,
                  eq. mamba2-mask), the lambda = 1, theta = 0 case.

All take one slice: x [L,R,P], B/C [L,R,N], dt/A/lam [L], theta [L,N/2],
D scalar, and return y [L,R,P].
"""
import numpy as np


def rotate_pairs(v, phi):
    """Apply the block rotation R(phi) to v [..., N] with pairs (i, i+N/2)."""
    h = v.shape[-1] // 2
    c, s = np.cos(phi), np.sin(phi)
    re, im = v[..., :h], v[..., h:]
    return np.concatenate([c * re - s * im, s * re + c * im], axis=-1)


def trapezoid_coeffs(dt, A, lam):
    alpha = np.exp(dt * A)
    return alpha, (1.0 - lam) * dt * alpha, lam * dt


def masked_form(x, B, C, dt, A, lam, theta, D):
    L = x.shape[0]
    alpha, beta, gamma = trapezoid_coeffs(dt, A, lam)
    # 1-semiseparable decay matrix: entry (t, j) = alpha_{t..j+1}, 1 on the diagonal
    L1 = np.zeros((L, L))
    for t in range(L):
        for j in range(t + 1):
            L1[t, j] = np.prod(alpha[j + 1:t + 1])
    # 2-band matrix: gamma on the diagonal, beta_t at (t, t-1)
    L2 = np.diag(gamma) + np.diag(beta[1:], -1)
    mask = L1 @ L2
    # RoPE trick: rotate B_t and C_t by the transpose of the cumulative product
    # R_0 ... R_t, i.e. by minus the cumulative angle.
    phi = np.cumsum(theta, axis=0)                      # [L, N/2]
    Bbar = rotate_pairs(B, -phi[:, None, :])            # [L, R, N]
    Cbar = rotate_pairs(C, -phi[:, None, :])
    G = np.einsum("tin,jrn->tijr", Cbar, Bbar)           # [L, R, L, R]
    y = np.einsum("tj,tijr,jrp->tip", mask, G, x)
    return y + D * x


def complex_form(x, B, C, dt, A, lam, theta, D):
    L, R, P = x.shape
    h2 = B.shape[-1] // 2
    Bc = B[..., :h2] + 1j * B[..., h2:]
    Cc = C[..., :h2] - 1j * C[..., h2:]
    alpha, beta, gamma = trapezoid_coeffs(dt, A, lam)
    h = np.zeros((h2, P), dtype=complex)
    prev = np.zeros((h2, P), dtype=complex)
    y = np.zeros((L, R, P))
    for t in range(L):
        rot = np.exp(1j * theta[t])[:, None]
        cur = sum(np.outer(Bc[t, r], x[t, r]) for r in range(R))
        h = alpha[t] * rot * h + beta[t] * rot * prev + gamma[t] * cur
        prev = cur
        for r in range(R):
            y[t, r] = np.real(Cc[t, r] @ h) + D * x[t, r]
    return y


def euler_complex(x, B, C, dt, A, theta, D):
    L, R, P = x.shape
    h2 = B.shape[-1] // 2
    Bc = B[..., :h2] + 1j * B[..., h2:]
    Cc = C[..., :h2] - 1j * C[..., h2:]
    h = np.zeros((h2, P), dtype=complex)
    y = np.zeros((L, R, P))
    for t in range(L):
        a = np.exp(dt[t] * A[t]) * np.exp(1j * theta[t])[:, None]
        h = a * h + dt[t] * sum(np.outer(Bc[t, r], x[t, r]) for r in range(R))
        for r in range(R):
            y[t, r] = np.real(Cc[t, r] @ h) + D * x[t, r]
    return y


def mamba2_masked(x, B, C, dt, A, D):
    L = x.shape[0]
    alpha = np.exp(dt * A)
    one_ss = np.zeros((L, L))
    for t in range(L):
        for j in range(t + 1):
            one_ss[t, j] = np.prod(alpha[j + 1:t + 1])
    mask = one_ss @ np.diag(dt)
    G = np.einsum("tin,jrn->tijr", C, B)
    return np.einsum("tj,tijr,jrp->tip", mask, G, x) + D * x


def tiny_slice(rng, L, N, P, R, theta_scale=1.0):
    """Random single-slice inputs for the pins (not a workload)."""
    return dict(
        x=rng.standard_normal((L, R, P)),
        B=rng.standard_normal((L, R, N)),
        C=rng.standard_normal((L, R, N)),
        dt=rng.uniform(0.01, 0.6, L),
        A=-rng.uniform(0.1, 2.0, L),
        lam=rng.uniform(0.0, 1.0, L),
        theta=theta_scale * rng.uniform(-1.0, 1.0, (L, N // 2)),
        D=float(rng.standard_normal()),
    )
