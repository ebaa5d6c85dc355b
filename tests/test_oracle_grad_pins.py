"""Pins of the oracle's reverse mode (oracle.scan_bwd) against what the
mathematics fixes, independently of its own code:

* central finite differences of the (separately pinned) forward oracle, for
  every input element, on tiny inputs;
* torch autograd (fp64) through an independent statement of the layer, the
  parallel masked form with Mamba-3's two-band mask and the rotary B, C
  (Sec. 3.1.2 eq. mamba3-mask; Sec. 3.2), written here in torch;
* adjoint identities: y and the final state are linear in x, in B, in C
  (zero initial state) and affine in the initial state, so <dx, x> etc.
  equal <dy, y> + <dfinal, h_L>;
* the first step's angle and decay only multiply the zero initial state
  (Sec. 3.1.2: the unrolled state starts at gamma_0 B_0 x_0), so their
  gradients are exactly zero.
A dropped beta-term chain, a sign slip in the rotation's derivative, the
wrong step's lambda or dt in beta, or a transposed MIMO operand fails at
least one of these.
"""
import numpy as np
import pytest
import torch

import oracle
from tests.formulations import tiny_slice


def stack(s):
    """One slice dict -> the oracle's [S=1, ...] arrays."""
    return dict(x=s["x"][None], B=s["B"][None], C=s["C"][None], dt=s["dt"][None],
                A=s["A"][None], lam=s["lam"][None], theta=s["theta"][None],
                D=np.array([s["D"]]))


def loss(a, dy, dfinal, init):
    y, st, _, _ = oracle.scan(**a, init_state=init)
    return float(np.sum(dy * y) + (0.0 if dfinal is None else np.sum(dfinal * st)))


@pytest.mark.parametrize("N,P,R", [(4, 3, 2), (2, 1, 1), (6, 2, 3)])
def test_bwd_central_differences(oracle_lib, N, P, R):
    rng = np.random.default_rng(40 + N + P + R)
    L = 11
    a = stack(tiny_slice(rng, L, N, P, R, theta_scale=1.5))
    dy = rng.standard_normal(a["x"].shape)
    dfinal = rng.standard_normal((1, N, P))
    init = rng.standard_normal((1, N, P))
    g = oracle.scan_bwd(**a, dy=dy, dfinal=dfinal, init_state=init)
    names = {"x": "dx", "B": "dB", "C": "dC", "dt": "ddt", "A": "dA", "lam": "dlam",
             "theta": "dtheta", "D": "dD"}
    h = 1e-6
    for key, gkey in names.items():
        base = a[key]
        fd = np.zeros_like(base)
        for idx in np.ndindex(base.shape):
            plus, minus = dict(a), dict(a)
            plus[key], minus[key] = base.copy(), base.copy()
            plus[key][idx] += h
            minus[key][idx] -= h
            fd[idx] = (loss(plus, dy, dfinal, init) - loss(minus, dy, dfinal, init)) / (2 * h)
        err = np.max(np.abs(fd - g[gkey])) / max(1.0, np.max(np.abs(fd)))
        assert err < 1e-7, f"{key}: {err:.3g}"
    fd = np.zeros_like(init)
    for idx in np.ndindex(init.shape):
        ip, im = init.copy(), init.copy()
        ip[idx] += h
        im[idx] -= h
        fd[idx] = (loss(a, dy, dfinal, ip) - loss(a, dy, dfinal, im)) / (2 * h)
    assert np.max(np.abs(fd - g["dinit"])) / max(1.0, np.max(np.abs(fd))) < 1e-7


def masked_form_torch(x, B, C, dt, A, lam, theta, D):
    """Y = (L o C^ B^T) X + D X with L = (1-semiseparable decay) @ (2-band
    trapezoid matrix) and C^, B^ rotated by minus the cumulative angle."""
    L_ = x.shape[0]
    alpha = torch.exp(dt * A)
    beta = (1 - lam) * dt * alpha
    gamma = lam * dt
    la = torch.log(alpha)
    cs = torch.cumsum(la, 0)
    diff = cs[:, None] - cs[None, :]
    causal = torch.tril(torch.ones(L_, L_, dtype=torch.bool))
    L1 = torch.where(causal, torch.exp(torch.where(causal, diff, torch.zeros_like(diff))),
                     torch.zeros_like(diff))
    L2 = torch.diag(gamma) + torch.diag(beta[1:], -1)
    mask = L1 @ L2
    phi = torch.cumsum(theta, 0)                          # [L, N/2]

    def rot(v, ang):                                      # v [L, R, N], angle [L, N/2]
        h = v.shape[-1] // 2
        c, s = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]
        re, im = v[..., :h], v[..., h:]
        return torch.cat([c * re - s * im, s * re + c * im], dim=-1)
    Bb, Cb = rot(B, -phi), rot(C, -phi)
    G = torch.einsum("tin,jrn->tijr", Cb, Bb)
    return torch.einsum("tj,tijr,jrp->tip", mask, G, x) + D * x


@pytest.mark.parametrize("N,P,R", [(4, 3, 2), (8, 2, 1), (4, 2, 4)])
def test_bwd_matches_autograd_of_masked_form(oracle_lib, N, P, R):
    rng = np.random.default_rng(50 + N * R + P)
    L = 19
    s = tiny_slice(rng, L, N, P, R, theta_scale=1.5)
    dy = rng.standard_normal((L, R, P))
    t = {k: torch.tensor(np.asarray(v, dtype=np.float64), requires_grad=True)
         for k, v in s.items()}
    y = masked_form_torch(t["x"], t["B"], t["C"], t["dt"], t["A"], t["lam"], t["theta"], t["D"])
    (y * torch.tensor(dy)).sum().backward()
    g = oracle.scan_bwd(**stack(s), dy=dy[None])
    pairs = {"x": "dx", "B": "dB", "C": "dC", "dt": "ddt", "A": "dA", "lam": "dlam",
             "theta": "dtheta"}
    for k, gk in pairs.items():
        ref = t[k].grad.numpy()
        assert np.max(np.abs(g[gk][0] - ref)) <= 1e-10 * max(1.0, np.max(np.abs(ref))), k
    assert abs(g["dD"][0] - float(t["D"].grad)) <= 1e-10 * max(1.0, abs(float(t["D"].grad)))


def test_bwd_adjoint_identities(oracle_lib):
    rng = np.random.default_rng(60)
    N, P, R, L = 6, 3, 2, 23
    a = stack(tiny_slice(rng, L, N, P, R))
    dy = rng.standard_normal(a["x"].shape)
    dfin = rng.standard_normal((1, N, P))
    y, st, _, _ = oracle.scan(**a)
    g = oracle.scan_bwd(**a, dy=dy, dfinal=dfin)
    J = np.sum(dy * y) + np.sum(dfin * st)
    Dx = a["D"][0] * a["x"]
    np.testing.assert_allclose(np.sum(g["dx"] * a["x"]), J, rtol=1e-12)
    np.testing.assert_allclose(np.sum(g["dB"] * a["B"]), J - np.sum(dy * Dx), rtol=1e-12)
    np.testing.assert_allclose(np.sum(g["dC"] * a["C"]), np.sum(dy * (y - Dx)), rtol=1e-12)
    np.testing.assert_allclose(g["dD"][0], np.sum(dy * a["x"]), rtol=1e-12)
    h0 = rng.standard_normal((1, N, P))
    y1, st1, _, _ = oracle.scan(**a, init_state=h0)
    g1 = oracle.scan_bwd(**a, dy=dy, dfinal=dfin, init_state=h0)
    np.testing.assert_allclose(np.sum(g1["dinit"] * h0),
                               np.sum(dy * (y1 - y)) + np.sum(dfin * (st1 - st)), rtol=1e-12)


def test_bwd_first_step_angle_and_decay_are_inert(oracle_lib):
    rng = np.random.default_rng(61)
    a = stack(tiny_slice(rng, 17, 4, 2, 2))
    dy = rng.standard_normal(a["x"].shape)
    g = oracle.scan_bwd(**a, dy=dy, dfinal=rng.standard_normal((1, 4, 2)))
    assert np.all(g["dtheta"][0, 0] == 0.0) and g["dA"][0, 0] == 0.0
    assert np.any(g["dtheta"][0, 1] != 0.0) and g["dA"][0, 1] != 0.0
    # with an initial state they act on it and are no longer inert
    g2 = oracle.scan_bwd(**a, dy=dy, init_state=rng.standard_normal((1, 4, 2)))
    assert np.any(g2["dtheta"][0, 0] != 0.0) and g2["dA"][0, 0] != 0.0
