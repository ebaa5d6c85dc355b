"""Pins of the fp64 CPU oracle against what the paper and the mathematics fix.

Every test here runs on the CPU.  Each one would fail for a plausible slip in
the oracle: a dropped beta term, beta using the previous step's lambda/dt, the
beta term left unrotated, the wrong rotation sign or pairing, a transposed
MIMO operand, or D applied inside the recurrence.
"""
import itertools
import math

import numpy as np
import pytest

import oracle
from tests.formulations import (complex_form, euler_complex, mamba2_masked,
                                masked_form, rotate_pairs, tiny_slice)


def run1(s, **kw):
    """Oracle on one slice dict (adds the slice axis)."""
    y, st, cb, cx = oracle.scan(s["x"][None], s["B"][None], s["C"][None],
                                s["dt"][None], s["A"][None], s["lam"][None],
                                s["theta"][None], np.array([s["D"]]), **kw)
    return y[0], st[0], cb[0], cx[0]


@pytest.mark.parametrize("N,P,R", list(itertools.product([2, 4, 8], [1, 3], [1, 2, 4])))
def test_p1_masked_form(oracle_lib, N, P, R):
    """Oracle = parallel masked form with the 2-band mask (eq. mamba3-mask)."""
    rng = np.random.default_rng(100 + N * 10 + P + R)
    for L in (1, 2, 17, 64):
        s = tiny_slice(rng, L, N, P, R)
        y, *_ = run1(s)
        ref = masked_form(**s)
        assert np.max(np.abs(y - ref)) <= 1e-12 * max(1.0, np.max(np.abs(ref)))


@pytest.mark.parametrize("N,P,R", [(2, 1, 1), (8, 3, 2), (16, 4, 4)])
def test_p2_complex_form(oracle_lib, N, P, R):
    """Oracle = complex-valued state (eq. trap-complex); pins the rotation
    direction and the [re; im] / [C; -C_hat] pairing."""
    rng = np.random.default_rng(7 + N)
    s = tiny_slice(rng, 40, N, P, R, theta_scale=2.0)
    y, *_ = run1(s)
    ref = complex_form(**s)
    assert np.max(np.abs(y - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_p3_lambda_one_is_exp_euler(oracle_lib):
    """lambda = 1 removes the previous-input term: Mamba-2's exponential-Euler
    recurrence with a rotating state."""
    rng = np.random.default_rng(3)
    s = tiny_slice(rng, 30, 8, 3, 2)
    s["lam"] = np.ones(30)
    y, *_ = run1(s)
    ref = euler_complex(s["x"], s["B"], s["C"], s["dt"], s["A"], s["theta"], s["D"])
    assert np.max(np.abs(y - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_p3_lambda_one_theta_zero_is_mamba2_mask(oracle_lib):
    """lambda = 1 and theta = 0: the mask collapses to 1-SS(alpha) Diag(dt)
    (eq. mamba2-mask)."""
    rng = np.random.default_rng(4)
    s = tiny_slice(rng, 25, 4, 2, 3)
    s["lam"] = np.ones(25)
    s["theta"] = np.zeros_like(s["theta"])
    y, *_ = run1(s)
    ref = mamba2_masked(s["x"], s["B"], s["C"], s["dt"], s["A"], s["D"])
    assert np.max(np.abs(y - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_p3_mimo_is_sum_of_siso(oracle_lib):
    """MIMO output column i = sum over input columns j of SISO SSMs with
    (B^(j), C^(i), x^(j)) sharing the recurrence (eqs. mamba3-mimo-siso-equiv)."""
    rng = np.random.default_rng(5)
    R = 3
    s = tiny_slice(rng, 33, 8, 5, R)
    y, *_ = run1(s)
    ref = np.zeros_like(y)
    for i in range(R):
        for j in range(R):
            sj = dict(s, x=s["x"][:, j:j + 1], B=s["B"][:, j:j + 1],
                      C=s["C"][:, i:i + 1], D=0.0)
            ref[:, i] += run1(sj)[0][:, 0]
        ref[:, i] += s["D"] * s["x"][:, i]
    assert np.max(np.abs(y - ref)) <= 1e-12 * np.max(np.abs(ref))


@pytest.mark.parametrize("omega", [0.0, 1.3])
def test_p3_discretisation_order(oracle_lib, omega):
    """The recurrence discretises dh/dt = (A + i omega) h + B x(t) (Sec. 3.1,
    Prop. trap; Sec. 3.2).  With x(t) = sin t, uniform steps and h(0) = 0, the
    exact solution is closed form.  lambda = 1/2 (classical trapezoid) must
    converge at second order and lambda = 1 (Euler) at first order; a wrong
    alpha/beta/gamma or an unrotated beta term breaks the second order."""
    A, T = -0.7, 3.0
    a = complex(A, omega)
    exact = ((-a * math.sin(T) - math.cos(T)) + np.exp(a * T)) / (a * a + 1)

    def err(lam, steps):
        d = T / steps
        tau = d * np.arange(1, steps + 1)          # right endpoints
        s = dict(x=np.sin(tau)[:, None, None],
                 B=np.tile([[1.0, 0.0]], (steps, 1))[:, None, :],
                 C=np.tile([[1.0, 0.0]], (steps, 1))[:, None, :],
                 dt=np.full(steps, d), A=np.full(steps, A),
                 lam=np.full(steps, lam), theta=np.full((steps, 1), d * omega),
                 D=0.0)
        _, st, *_ = run1(s)
        return abs(complex(st[0, 0], st[1, 0]) - exact)

    e2 = [err(0.5, n) for n in (200, 400, 800)]
    e1 = [err(1.0, n) for n in (200, 400, 800)]
    for k in range(2):
        assert 3.6 < e2[k] / e2[k + 1] < 4.4, e2
        assert 1.8 < e1[k] / e1[k + 1] < 2.2, e1


def test_p5_boundary_impulse(oracle_lib):
    """Only x_j nonzero, with j the last token of a 16-token chunk.  With
    gamma_j = 0 everything after j flows through beta_{j+1}: the single mask
    entry alpha_{t..j+2} beta_{j+1} C_t^T R(phi_t - phi_j) B_j x_j."""
    rng = np.random.default_rng(6)
    L, N, P, R, j = 48, 8, 3, 2, 15
    for lam_j in (0.0, 0.4):
        s = tiny_slice(rng, L, N, P, R)
        s["x"][:] = 0.0
        s["x"][j] = rng.standard_normal((R, P))
        s["lam"][j] = lam_j
        s["lam"][j + 1] = 0.3
        y, *_ = run1(s)
        alpha = np.exp(s["dt"] * s["A"])
        beta = (1 - s["lam"]) * s["dt"] * alpha
        gamma = s["lam"] * s["dt"]
        phi = np.cumsum(s["theta"], axis=0)
        ref = np.zeros_like(y)
        ref[j] = gamma[j] * np.einsum("in,rn,rp->ip", s["C"][j], s["B"][j], s["x"][j]) \
            + s["D"] * s["x"][j]
        for t in range(j + 1, L):
            w = np.prod(alpha[j + 2:t + 1]) * (gamma[j] * alpha[j + 1] + beta[j + 1])
            rb = rotate_pairs(s["B"][j], phi[t] - phi[j])
            ref[t] = w * np.einsum("in,rn,rp->ip", s["C"][t], rb, s["x"][j])
        assert np.max(np.abs(y[:j])) == 0.0
        if lam_j == 0.0:
            assert np.array_equal(y[j], s["D"] * s["x"][j])
        assert np.max(np.abs(y - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_p6_first_step_angle_and_decay_are_inert(oracle_lib):
    """h_{-1} = 0 and no previous input: theta_0 and A_0 only multiply zero."""
    rng = np.random.default_rng(8)
    s = tiny_slice(rng, 20, 8, 2, 2)
    y0, st0, *_ = run1(s)
    s2 = dict(s, theta=s["theta"].copy(), A=s["A"].copy())
    s2["theta"][0] += 2.0
    s2["A"][0] *= 5.0
    y1, st1, *_ = run1(s2)
    assert np.array_equal(y0, y1) and np.array_equal(st0, st1)


def test_p7_step_and_segment_resume(oracle_lib):
    """scan(L) then one step = scan(L+1) at t = L, same state and carry; and
    scan(0:L1) then scan(L1:L) from (state, carry) = scan(0:L)."""
    rng = np.random.default_rng(9)
    L, N, P, R = 37, 8, 3, 2
    s = tiny_slice(rng, L + 1, N, P, R)
    yf, stf, cbf, cxf = run1(s)
    pre = {k: (v[:L] if isinstance(v, np.ndarray) else v) for k, v in s.items()}
    _, st, cb, cx = run1(pre)
    ys, st2, cb2, cx2 = oracle.step(st[None], cb[None], cx[None], s["x"][L][None],
                                    s["B"][L][None], s["C"][L][None],
                                    s["dt"][L:L + 1], s["A"][L:L + 1],
                                    s["lam"][L:L + 1], s["theta"][L][None],
                                    np.array([s["D"]]))
    assert np.allclose(ys[0], yf[L], rtol=0, atol=1e-13)
    assert np.allclose(st2[0], stf, rtol=0, atol=1e-13)
    assert np.array_equal(cb2[0], cbf) and np.array_equal(cx2[0], cxf)
    L1 = 13
    a = {k: (v[:L1] if isinstance(v, np.ndarray) else v) for k, v in s.items()}
    b = {k: (v[L1:] if isinstance(v, np.ndarray) else v) for k, v in s.items()}
    ya, sta, cba, cxa = run1(a)
    yb, stb, _, _ = run1(b, init_state=sta[None], init_B=cba[None], init_X=cxa[None])
    assert np.allclose(np.concatenate([ya, yb]), yf, rtol=0, atol=1e-13)
    assert np.allclose(stb, stf, rtol=0, atol=1e-13)


def test_p8_lti_steady_state(oracle_lib):
    """Constant alpha, lambda, dt, theta, B, x: the state converges to
    (I - alpha R)^{-1} (alpha beta' R + gamma) B X^T with beta' = (1-lambda) dt
    (geometric series of the recurrence)."""
    rng = np.random.default_rng(10)
    L, N, P, R = 4000, 8, 3, 2
    dt, A, lam = 0.05, -0.5, 0.3
    th = rng.uniform(-0.5, 0.5, N // 2)
    Bv, Xv = rng.standard_normal((R, N)), rng.standard_normal((R, P))
    s = dict(x=np.broadcast_to(Xv, (L, R, P)).copy(),
             B=np.broadcast_to(Bv, (L, R, N)).copy(),
             C=rng.standard_normal((L, R, N)), dt=np.full(L, dt), A=np.full(L, A),
             lam=np.full(L, lam), theta=np.broadcast_to(th, (L, N // 2)).copy(), D=0.0)
    _, st, *_ = run1(s)
    alpha = math.exp(dt * A)
    Rm = np.zeros((N, N))
    h2 = N // 2
    for i in range(h2):
        c, sn = math.cos(th[i]), math.sin(th[i])
        Rm[i, i], Rm[i, i + h2], Rm[i + h2, i], Rm[i + h2, i + h2] = c, -sn, sn, c
    v = Bv.T @ Xv
    ref = np.linalg.solve(np.eye(N) - alpha * Rm, (alpha * (1 - lam) * dt * Rm + lam * dt * np.eye(N)) @ v)
    assert np.max(np.abs(st - ref)) <= 1e-10 * np.max(np.abs(ref))


def test_p9_parity_chain(oracle_lib):
    """alpha = 1, lambda = 1, an input only at t = 0 and theta_t = pi bit_t:
    Y_T = (-1)^{bit_1 + ... + bit_T} gamma_0 C_T^T B_0 x_0 (state-tracking by
    rotation, Sec. 3.2).  bit_0 only rotates h_{-1} = 0."""
    rng = np.random.default_rng(11)
    L, N, P = 3000, 4, 2
    bits = rng.integers(0, 2, L)
    x = np.zeros((L, 1, P))
    x[0, 0] = rng.standard_normal(P)
    B = np.zeros((L, 1, N))
    B[0, 0] = rng.standard_normal(N)
    C = rng.standard_normal((L, 1, N))
    s = dict(x=x, B=B, C=C, dt=np.full(L, 0.7), A=np.zeros(L), lam=np.ones(L),
             theta=np.pi * np.repeat(bits[:, None], N // 2, axis=1).astype(float), D=0.0)
    y, *_ = run1(s)
    sign = (-1.0) ** np.cumsum(np.concatenate([[0], bits[1:]]))
    ref = sign[:, None] * 0.7 * (C[:, 0] @ B[0, 0])[:, None] * x[0, 0][None, :]
    assert np.max(np.abs(y[:, 0] - ref)) <= 1e-11 * np.max(np.abs(ref))


def test_p10_linearity_and_common_rotation(oracle_lib):
    rng = np.random.default_rng(12)
    s = tiny_slice(rng, 29, 8, 3, 2)
    y, *_ = run1(s)
    y2, *_ = run1(dict(s, x=2.5 * s["x"]))
    assert np.allclose(y2, 2.5 * y, rtol=1e-13, atol=1e-13)
    C2 = rng.standard_normal(s["C"].shape)
    ya, *_ = run1(dict(s, C=C2, D=0.0))
    yb, *_ = run1(dict(s, C=s["C"] + C2, D=0.0))
    yc, *_ = run1(dict(s, D=0.0))
    assert np.allclose(yb, ya + yc, rtol=1e-12, atol=1e-12)
    phi0 = rng.uniform(-3, 3, 4)
    yr, *_ = run1(dict(s, B=rotate_pairs(s["B"], phi0), C=rotate_pairs(s["C"], phi0)))
    assert np.allclose(yr, y, rtol=1e-12, atol=1e-12)


def test_empty_sequence_returns_initial_state(oracle_lib):
    rng = np.random.default_rng(13)
    s = tiny_slice(rng, 0, 4, 2, 2)
    st0 = rng.standard_normal((1, 4, 2))
    cb0, cx0 = rng.standard_normal((1, 2, 4)), rng.standard_normal((1, 2, 2))
    y, st, cb, cx = run1(s, init_state=st0, init_B=cb0, init_X=cx0)
    assert y.shape == (0, 2, 2)
    assert np.array_equal(st, st0[0]) and np.array_equal(cb, cb0[0]) and np.array_equal(cx, cx0[0])


def test_gate_silu_closed_forms():
    """SiLU against textbook values of the logistic function: sigma(1) =
    1 / (1 + 1/e), sigma(-1) = 1 - sigma(1); SiLU(0) = 0; the odd-part
    identity SiLU(z) - SiLU(-z) = z; and the limits (identity for large z,
    zero for very negative z, where exp overflows)."""
    s1 = 0.7310585786300049          # logistic(1) = e / (1 + e)
    assert math.isclose(s1, math.e / (1.0 + math.e), rel_tol=0, abs_tol=1e-16)
    got = oracle.silu(np.array([0.0, 1.0, -1.0, 2.0, 40.0, -800.0]))
    assert got[0] == 0.0
    assert math.isclose(got[1], s1, rel_tol=1e-15)
    assert math.isclose(got[2], -(1.0 - s1), rel_tol=1e-15)
    assert math.isclose(got[3], 2.0 * math.e ** 2 / (1.0 + math.e ** 2), rel_tol=1e-15)
    assert got[4] == 40.0            # 1 + e^-40 rounds to 1
    assert got[5] == 0.0 and np.isfinite(got).all()
    z = np.random.default_rng(7).normal(scale=4.0, size=1000)
    assert np.max(np.abs(oracle.silu(z) - oracle.silu(-z) - z)) <= 1e-13


def test_gate_is_elementwise_product():
    """phi(Y, Z) = Y o SiLU(Z), elementwise: y z for a large gate (sigma = 1),
    zero for a zero gate, and for a gate pair z, -z the sum
    y (SiLU(z) + SiLU(-z)) = y z tanh(z / 2)."""
    rng = np.random.default_rng(8)
    y = rng.normal(size=(3, 5, 2, 4))
    np.testing.assert_array_equal(oracle.gate(y, np.full_like(y, 40.0)), y * 40.0)
    np.testing.assert_array_equal(oracle.gate(y, np.zeros_like(y)), np.zeros_like(y))
    z = rng.normal(size=y.shape)
    lhs = oracle.gate(y, z) + oracle.gate(y, -z)
    np.testing.assert_allclose(lhs, y * z * np.tanh(z / 2.0), rtol=1e-13, atol=1e-15)


def test_rel_err_definition():
    """The parity metric max|got - ref| / max|ref| (infinity norms over the
    whole array), on values worked out by hand: a slip that normalises by the
    other operand, drops an absolute value, takes a mean or a norm of another
    order changes at least one of these."""
    assert oracle.rel_err([1.0, 2.0], [1.0, 4.0]) == 0.5            # 2 / 4
    assert oracle.rel_err([1.0, 4.0], [1.0, 2.0]) == 1.0            # 2 / 2 (not 2 / 4)
    assert oracle.rel_err([-3.0, 0.0], [-1.0, 0.5]) == 2.0          # |-2| / |-1|
    assert oracle.rel_err([0.0, 0.0], [-2.0, 1.0]) == 1.0           # max|ref| is 2, not max(ref) = 1
    assert oracle.rel_err([1.0, 1.0, 1.0], [0.0, 0.0, 4.0]) == 0.75  # max error 3 over 4, not a mean
    assert oracle.rel_err([[0.5, -1.5], [2.0, 3.0]], [[1.0, -1.0], [2.0, 4.0]]) == 0.25
    assert oracle.rel_err([0.0, 0.0], [0.0, 0.0]) == 0.0            # both zero
    assert oracle.rel_err([0.0, 3.0], [0.0, 0.0]) == 3.0            # zero reference: absolute error
    assert oracle.rel_err([], []) == 0.0
    assert oracle.rel_err(np.full(5, 7.0), np.full(5, 7.0)) == 0.0


# ---------------------------------------------------------------------------
# Block prologue: BCNorm, B/C biases, structured MIMO input (Sec. 3.4; App.
# "MIMO for Mamba-3", paragraph "Mamba with MIMO").
# ---------------------------------------------------------------------------

def test_bcnorm_unit_rms_over_state_axis():
    """With eps = 0 and no gain or bias every (token, rank) column comes out
    with mean square exactly 1 over N, pointing the same way as its input.
    The columns are given scales 1e-3 .. 1e3, so a norm over another axis
    (ranks, tokens) or over all of them fails."""
    rng = np.random.default_rng(20)
    v = rng.standard_normal((3, 5, 4, 16)) * np.logspace(-3, 3, 4)[None, None, :, None]
    out = oracle.rms_norm(v, eps=0.0)
    np.testing.assert_allclose(np.mean(out * out, axis=-1), 1.0, rtol=1e-13)
    cos = np.sum(out * v, axis=-1) / np.sqrt(np.sum(out * out, axis=-1) * np.sum(v * v, axis=-1))
    np.testing.assert_allclose(cos, 1.0, rtol=1e-13)


def test_bcnorm_constant_vector_closed_form():
    """A constant vector c: c / sqrt(c^2 + eps) in every channel.  c = 0.5,
    eps = 0.25 gives 0.5 / sqrt(0.5) = 1 / sqrt(2); eps added outside the
    root (c / (|c| + eps) = 2/3) or to the root mean (c / (sqrt(c^2) + eps))
    would not."""
    out = oracle.rms_norm(np.full((1, 8), 0.5), eps=0.25)
    np.testing.assert_allclose(out, 1.0 / math.sqrt(2.0), rtol=1e-15)
    out = oracle.rms_norm(np.full((1, 8), -3.0), eps=0.0)
    np.testing.assert_array_equal(out, -1.0)


def test_bcnorm_scale_invariance_and_oddness():
    """Without eps the norm does not see the scale: f(k v) = f(v), k > 0, and
    f(-v) = -f(v)."""
    rng = np.random.default_rng(21)
    v = rng.standard_normal((6, 32))
    f = oracle.rms_norm(v, eps=0.0)
    np.testing.assert_allclose(oracle.rms_norm(7.25 * v, eps=0.0), f, rtol=1e-14)
    np.testing.assert_allclose(oracle.rms_norm(-v, eps=0.0), -f, rtol=1e-14)


def test_bcnorm_gain_then_bias_after_norm():
    """Gain multiplies the normalised channels and the bias is added after
    the norm: (out - bias) / gain has unit mean square whatever the bias (a
    bias added before the norm changes it), and a worked example: v = (3, 4)
    has RMS sqrt(12.5); gain (2, 1), bias (1, -1) give (2*3/sqrt(12.5) + 1,
    4/sqrt(12.5) - 1)."""
    rng = np.random.default_rng(22)
    v = rng.standard_normal((4, 2, 16))
    gain = rng.uniform(0.5, 2.0, (2, 16))
    bias = rng.standard_normal((2, 16)) + 1.0
    out = oracle.rms_norm(v, gain=gain, bias=bias, eps=0.0)
    np.testing.assert_allclose(np.mean(((out - bias) / gain) ** 2, axis=-1), 1.0, rtol=1e-13)
    got = oracle.rms_norm(np.array([3.0, 4.0]), gain=np.array([2.0, 1.0]),
                          bias=np.array([1.0, -1.0]), eps=0.0)
    r = math.sqrt(12.5)
    np.testing.assert_allclose(got, [6.0 / r + 1.0, 4.0 / r - 1.0], rtol=1e-15)
    np.testing.assert_array_equal(oracle.add_bias(v, bias), v + bias)


def test_structured_input_worked_example():
    """X_t[r, p] = W[r, p] X'_t[p]: W[2, 3] = 7 and X'_t[3] = 2 give 14 at
    (t, r=2, p=3) and W[0, 3] X'_t[3] at r = 0; R != P so a transposed W
    fails on shape or value."""
    S, L, R, P = 1, 2, 3, 5
    xp = np.zeros((S, L, P))
    xp[0, 1, 3] = 2.0
    xp[0, 0, 1] = -1.5
    w = np.arange(R * P, dtype=float).reshape(1, R, P)
    w[0, 2, 3] = 7.0
    X = oracle.structured_input(xp, w)
    assert X.shape == (S, L, R, P)
    assert X[0, 1, 2, 3] == 14.0
    assert X[0, 1, 0, 3] == 2.0 * 3.0          # W[0, 3] = 3
    assert X[0, 0, 1, 1] == -1.5 * 6.0         # W[1, 1] = 6
    assert np.count_nonzero(X[0, 1]) == R and np.count_nonzero(X[0, 0]) == R


def test_structured_input_feeds_rank_columns(oracle_lib):
    """With W rows c_r (constants per rank) the MIMO layer's input columns
    are c_r X': by linearity in X (Sec. 3.3), the output of the scan on the
    structured input equals sum_r c_r times the scan with X' in column r
    alone (D = 0)."""
    rng = np.random.default_rng(23)
    R, P = 3, 4
    s = tiny_slice(rng, 21, 8, P, R)
    s["D"] = 0.0
    xp = rng.standard_normal((1, 21, P))
    c = np.array([0.5, -2.0, 1.25])
    w = np.repeat(c[:, None], P, axis=1)[None]
    y, *_ = run1(dict(s, x=oracle.structured_input(xp, w)[0]))
    ref = np.zeros_like(y)
    for r in range(R):
        xr = np.zeros((21, R, P))
        xr[:, r, :] = xp[0]
        ref += c[r] * run1(dict(s, x=xr))[0]
    assert np.max(np.abs(y - ref)) <= 1e-12 * np.max(np.abs(ref))


# ---------------------------------------------------------------------------
# Output norm (Sec. 4 hybrid models; App. norm type / placement ablation):
# grouped RMS of the SSM output before or after the output gate.
# ---------------------------------------------------------------------------

def test_out_norm_worked_example():
    """y row [3, 4, 0, 2] in groups of two: the first group's RMS is
    sqrt(12.5), the second's sqrt(2); no gain, no gate, eps 0."""
    y = np.array([[3.0, 4.0, 0.0, 2.0]])
    got = oracle.out_norm(y, 2, eps=0.0)
    want = np.array([[3 / math.sqrt(12.5), 4 / math.sqrt(12.5), 0.0, 2 / math.sqrt(2.0)]])
    np.testing.assert_allclose(got, want, rtol=1e-15)


def test_out_norm_groups_are_independent_and_unit_rms():
    rng = np.random.default_rng(70)
    y = rng.standard_normal((3, 5, 64))
    a = oracle.out_norm(y, 16, eps=1e-12)
    # every group of 16 channels has unit RMS
    g = a.reshape(3, 5, 4, 16)
    np.testing.assert_allclose(np.sqrt(np.mean(g * g, axis=-1)), 1.0, rtol=1e-9)
    # scaling one group changes only that group (and not even it: scale invariance)
    y2 = y.copy()
    y2[..., 16:32] *= -7.5
    b = oracle.out_norm(y2, 16, eps=1e-12)
    np.testing.assert_allclose(b[..., :16], a[..., :16], rtol=1e-12)
    np.testing.assert_allclose(b[..., 32:], a[..., 32:], rtol=1e-12)
    np.testing.assert_allclose(b[..., 16:32], -a[..., 16:32], rtol=1e-9)


def test_out_norm_constant_group_closed_form():
    y = np.full((2, 32), 0.25)
    gain = np.linspace(0.5, 2.0, 32)
    got = oracle.out_norm(y, 8, eps=1e-3, gain=gain)
    np.testing.assert_allclose(got, np.broadcast_to(gain * 0.25 / math.sqrt(0.0625 + 1e-3), got.shape),
                               rtol=1e-14)


def test_out_norm_whole_row_group_is_bcnorm_form():
    """group = the row length: one RMS over the row, the same form as the
    (separately pinned) state-axis norm."""
    rng = np.random.default_rng(71)
    y = rng.standard_normal((4, 64))
    gain = rng.uniform(0.5, 1.5, 64)
    np.testing.assert_allclose(oracle.out_norm(y, 64, eps=1e-5, gain=gain),
                               oracle.rms_norm(y, gain=gain, eps=1e-5), rtol=1e-13)


def test_out_norm_pre_and_post_gate():
    """The gate enters after the norm (pre-gate) or inside it (post-gate): with
    SiLU(z) constant s over a group, post-gate = (pre-gate) / |s|
    (eps -> 0); with varying z the two differ; without z they agree."""
    rng = np.random.default_rng(72)
    y = rng.standard_normal((2, 3, 32))
    zc = np.repeat(rng.uniform(-3, 3, (2, 3, 4, 1)), 8, axis=-1).reshape(2, 3, 32)
    s = oracle.silu(zc)
    pre = oracle.out_norm(y, 8, eps=1e-14, z=zc, pre_gate=True)
    post = oracle.out_norm(y, 8, eps=1e-14, z=zc, pre_gate=False)
    np.testing.assert_allclose(post, pre / np.abs(s), rtol=1e-7)
    np.testing.assert_allclose(pre, oracle.group_rms(y, 8, 1e-14) * s, rtol=1e-14)
    z = rng.standard_normal((2, 3, 32))
    assert np.max(np.abs(oracle.out_norm(y, 8, z=z) - oracle.out_norm(y, 8, z=z, pre_gate=False))) > 0.1
    np.testing.assert_array_equal(oracle.out_norm(y, 8), oracle.out_norm(y, 8, pre_gate=False))
    with pytest.raises(ValueError):
        oracle.group_rms(y, 12, 1e-6)
