"""The chunked decomposition used by the HIP prefill, checked in fp64 on the CPU.

The chunked algorithm (Sec. 3.3, "Chunked Algorithm for MIMO SSMs") computes
the same recurrence as the oracle: a masked quadratic form inside each chunk of
Q tokens and a recurrence on the N x P state across chunks.  For Mamba-3 the
two-band mask means token j's weight inside its chunk is
    sigma_j = gamma_j + (1 - lambda_{j+1}) dt_{j+1}    (sigma_{L-1} = gamma_{L-1}),
so the last token of a chunk reads the next token's lambda and dt.  The state
passed between chunks is kept in the physical (unrotated) frame and already
holds the next token's previous-input term; decays and angles are prefix sums
local to the chunk.  This file restates that decomposition in numpy and checks
it against the oracle, so the GPU design is known to be exact before any
kernel runs.  It shares no code with the HIP path.
"""
import numpy as np
import pytest

import oracle
from tests.formulations import rotate_pairs, tiny_slice


def chunked(x, B, C, dt, A, lam, theta, D, Q, init_state=None, init_B=None, init_X=None):
    L, R, P = x.shape
    N = B.shape[-1]
    S = np.zeros((N, P)) if init_state is None else init_state.copy()
    if L == 0:
        return np.zeros((0, R, P)), S
    if init_B is not None:          # fold the carried previous input into S
        S = S + (1 - lam[0]) * dt[0] * (init_B.T @ init_X)
    gamma = lam * dt
    sigma = gamma.copy()
    sigma[:-1] += (1 - lam[1:]) * dt[1:]
    y = np.zeros((L, R, P))
    for c0 in range(0, L, Q):
        c1 = min(c0 + Q, L)
        cum = np.cumsum(dt[c0:c1] * A[c0:c1])                # chunk-local
        psi = np.cumsum(theta[c0:c1], axis=0)                # [q, N/2]
        Chat = rotate_pairs(C[c0:c1], -psi[:, None, :])      # [q, R, N]
        Bhat = rotate_pairs(B[c0:c1], -psi[:, None, :])
        q = c1 - c0
        W = np.zeros((q, q))
        for t in range(q):
            W[t, t] = gamma[c0 + t]
            for j in range(t):
                W[t, j] = np.exp(cum[t] - cum[j]) * sigma[c0 + j]
        G = np.einsum("tin,jrn->tijr", Chat, Bhat)
        y[c0:c1] = np.einsum("tj,tijr,jrp->tip", W, G, x[c0:c1])
        y[c0:c1] += np.exp(cum)[:, None, None] * np.einsum("tin,np->tip", Chat, S)
        y[c0:c1] += D * x[c0:c1]
        w = np.exp(cum[-1] - cum) * sigma[c0:c1]              # [q]
        M = np.einsum("j,jrn,jrp->np", w, Bhat, x[c0:c1])
        # S_c = R(psi_e) (e^{cum_e} S_{c-1} + M)
        S = rotate_pairs((np.exp(cum[-1]) * S + M).T, psi[-1]).T
    return y, S


@pytest.mark.parametrize("Q", [1, 2, 8, 16, 64, 128])
def test_chunked_equals_sequential(oracle_lib, Q):
    rng = np.random.default_rng(20 + Q)
    for L, N, P, R in [(250, 8, 3, 2), (64, 4, 2, 1), (37, 8, 1, 4)]:
        s = tiny_slice(rng, L, N, P, R)
        y, st, _, _ = oracle.scan(*(s[k][None] for k in ("x", "B", "C", "dt", "A", "lam", "theta")),
                                  np.array([s["D"]]))
        yc, Sc = chunked(**s, Q=Q)
        scale = np.max(np.abs(y[0]))
        assert np.max(np.abs(yc - y[0])) <= 1e-12 * scale
        assert np.max(np.abs(Sc - st[0])) <= 1e-12 * np.max(np.abs(st[0]))


def test_chunked_with_initial_state_and_carry(oracle_lib):
    rng = np.random.default_rng(31)
    L, N, P, R = 70, 8, 3, 2
    s = tiny_slice(rng, L, N, P, R)
    st0 = rng.standard_normal((N, P))
    cb0, cx0 = rng.standard_normal((R, N)), rng.standard_normal((R, P))
    y, st, _, _ = oracle.scan(*(s[k][None] for k in ("x", "B", "C", "dt", "A", "lam", "theta")),
                              np.array([s["D"]]), init_state=st0[None], init_B=cb0[None],
                              init_X=cx0[None])
    yc, Sc = chunked(**s, Q=16, init_state=st0, init_B=cb0, init_X=cx0)
    assert np.max(np.abs(yc - y[0])) <= 1e-12 * np.max(np.abs(y[0]))
    assert np.max(np.abs(Sc - st[0])) <= 1e-12 * np.max(np.abs(st[0]))
