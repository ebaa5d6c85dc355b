"""GPU parity of the fused block prologue (m3_scan_fwd_pro, m3_step_pro)
against the fp64 oracle: BCNorm over the state axis with gains, the B/C
biases after it (Sec. 3.4), the structured MIMO input X = W_X o X' and gate
input Z = W_Z o Z' (App. "MIMO for Mamba-3", paragraph "Mamba with MIMO").

The oracle applies the same prologue in fp64 (oracle.rms_norm, add_bias,
structured_input) to the exact raw inputs the GPU received and runs its
sequential recurrence.  Bars: y and the final state 2e-2 (bf16 inputs, as
for every bf16 scan); the carry, which now holds computed values (the
normalised B, the expanded X) rounded once to bf16, within 8e-3 (two bf16
half-ulps of the largest element).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2603_15569_amd import m3
from paper_2603_15569_amd.inputs import (WORKLOADS, make_prologue_inputs,
                                         make_prologue_step_inputs, make_scan_inputs,
                                         make_step_inputs, workload_inputs)

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 2e-2
TOL_CARRY = 8e-3
EPS = 1e-6


def say(msg):
    print(f"[gpu-case] {msg}", flush=True)


VARIANTS = {
    # name: (bc_norm, gains, biases, structured x, gate: None / "z" / "wz")
    "full": (True, True, True, True, None),
    "norm_only": (True, False, False, False, None),
    "bias_only": (False, False, True, False, None),
    "wx_only": (False, False, False, True, None),
    "gated_wz": (True, True, True, True, "wz"),
    "gated_z": (True, True, True, False, "z"),
}


def make_case(B, L, H, R, Q, seed):
    inp = make_scan_inputs(B, L, H, 64, 128, R, io="bf16", seed=seed, device=DEV, chunk=Q)
    pin = make_prologue_inputs(B, L, H, 64, 128, R, io="bf16", seed=seed, device=DEV)
    return inp, pin


def pro_of(pin, variant):
    norm, gains, biases, sx, gate = VARIANTS[variant]
    return m3.prologue(bc_norm=norm, eps=EPS, norm_B=pin.gB if gains else None,
                       norm_C=pin.gC if gains else None, bias_B=pin.bB if biases else None,
                       bias_C=pin.bC if biases else None, w_x=pin.wx if sx else None,
                       w_z=pin.wz if gate == "wz" else None)


def gpu_args(inp, pin, variant, zfull):
    """x and z as the library reads them for the variant."""
    _, _, _, sx, gate = VARIANTS[variant]
    x = pin.xp if sx else inp.x
    z = None if gate is None else (pin.zp if gate == "wz" else zfull)
    return x, z


def oracle_prologue(inp, pin, variant, slices, zfull=None, t0=0, t1=None):
    """Per-slice oracle inputs after the prologue (fp64) and the gate input."""
    norm, gains, biases, sx, gate = VARIANTS[variant]
    hs = [h for _, h in slices]
    x_arg = pin.xp if sx else inp.x
    ref = oracle.slices_of_scan(x_arg, pin.Bp, pin.Cp, inp.dt, inp.A, inp.lam, inp.theta, inp.D,
                                slices, t0, t1)
    g_b = oracle._np(pin.gB)[hs][:, None] if gains else None
    g_c = oracle._np(pin.gC)[hs][:, None] if gains else None
    b_b = oracle._np(pin.bB)[hs][:, None] if biases else None
    b_c = oracle._np(pin.bC)[hs][:, None] if biases else None
    if norm:
        ref["B"] = oracle.rms_norm(ref["B"], g_b, b_b, EPS)
        ref["C"] = oracle.rms_norm(ref["C"], g_c, b_c, EPS)
    else:
        ref["B"] = oracle.add_bias(ref["B"], b_b)
        ref["C"] = oracle.add_bias(ref["C"], b_c)
    if sx:
        ref["x"] = oracle.structured_input(ref["x"], oracle._np(pin.wx)[hs])
    zref = None
    t1 = pin.Bp.shape[1] if t1 is None else t1
    if gate == "wz":
        zs = np.stack([oracle._np(pin.zp[b, t0:t1, h]) for b, h in slices])
        zref = oracle.structured_input(zs, oracle._np(pin.wz)[hs])
    elif gate == "z":
        zref = np.stack([oracle._np(zfull[b, t0:t1, h]) for b, h in slices])
    return ref, zref


def run_pro(inp, pin, variant, Q, zfull=None, init_state=None, init_carry=None, t0=0, t1=None,
            seg=0):
    x, z = gpu_args(inp, pin, variant, zfull)
    sl = slice(t0, t1)

    def cut(t):
        return None if t is None else t[:, sl].contiguous()
    R = pin.Bp.shape[3]
    y, fs, (cB, cX) = m3.scan_fwd_pro(cut(x), cut(pin.Bp), cut(pin.Cp), cut(inp.dt), inp.A,
                                      cut(inp.lam), cut(inp.theta), inp.D, Q,
                                      pro_of(pin, variant), R, z=cut(z), init_state=init_state,
                                      init_carry=init_carry, check=True, seg=seg)
    torch.cuda.synchronize()
    return y, fs, cB, cX


def compare(y, fs, cB, cX, ref, zref, slices, label, kw=None):
    ry, rs, rb, rx = oracle.scan(**ref, **(kw or {}))
    if zref is not None:
        ry = oracle.gate(ry, zref)
    worst, worst_c = 0.0, 0.0
    for k, (b, h) in enumerate(slices):
        gy = y[b, :, h].double().cpu().numpy()
        gs = fs[b, h].double().cpu().numpy()
        assert np.all(np.isfinite(gy)) and np.all(np.isfinite(gs)), f"{label} non-finite {(b, h)}"
        e = max(oracle.rel_err(gy, ry[k]), oracle.rel_err(gs, rs[k]))
        ec = max(oracle.rel_err(cB[b, h].double().cpu().numpy(), rb[k]),
                 oracle.rel_err(cX[b, h].double().cpu().numpy(), rx[k]))
        worst, worst_c = max(worst, e), max(worst_c, ec)
        assert e <= TOL, f"{label} slice {(b, h)}: rel err {e:.3g}"
        assert ec <= TOL_CARRY, f"{label} slice {(b, h)}: carry rel err {ec:.3g}"
    say(f"{label}: worst rel err {worst:.3g}, carry {worst_c:.3g}, {len(slices)} slices")
    return worst


@pytest.mark.parametrize("variant", list(VARIANTS))
@pytest.mark.parametrize("R,Q,L", [(1, 64, 300), (4, 64, 200), (4, 128, 300), (2, 32, 77)])
def test_prologue_scan(R, Q, L, variant):
    say(f"prologue scan R={R} Q={Q} L={L} {variant}")
    inp, pin = make_case(2, L, 3, R, Q, seed=R * 100 + Q + L)
    zfull = torch.randn(inp.x.shape, device=DEV, generator=torch.Generator(DEV).manual_seed(9)
                        ).to(torch.bfloat16)
    y, fs, cB, cX = run_pro(inp, pin, variant, Q, zfull=zfull)
    slices = [(b, h) for b in range(2) for h in range(3)]
    ref, zref = oracle_prologue(inp, pin, variant, slices, zfull=zfull)
    compare(y, fs, cB, cX, ref, zref, slices, f"pro R={R} Q={Q} L={L} {variant}")


@pytest.mark.parametrize("R,Q", [(1, 64), (4, 128)])
def test_prologue_continuation(R, Q):
    """scan(0:L1) then scan(L1:L) from its state and carry (the prologue's B
    and X) = the oracle over 0:L."""
    say(f"prologue continuation R={R} Q={Q}")
    L, L1 = 333, 190
    inp, pin = make_case(1, L, 2, R, Q, seed=77 + R)
    ya, fa, cBa, cXa = run_pro(inp, pin, "full", Q, t0=0, t1=L1)
    yb, fb, cBb, cXb = run_pro(inp, pin, "full", Q, init_state=fa, init_carry=(cBa, cXa),
                               t0=L1, t1=L)
    y = torch.cat([ya, yb], dim=1)
    slices = [(0, 0), (0, 1)]
    ref, _ = oracle_prologue(inp, pin, "full", slices)
    compare(y, fb, cBb, cXb, ref, None, slices, f"pro continuation R={R} Q={Q}")


# One segment per slice (seg at least the chunk count) runs the
# warp-specialised kernel with the prologue (rank 4, chunk 64): every
# variant, a ragged last chunk, and a continuation from a state and carry.
WS = 1 << 20


@pytest.mark.parametrize("variant", list(VARIANTS))
@pytest.mark.parametrize("L", [200, 64, 1])
def test_prologue_scan_ws(L, variant):
    say(f"prologue scan warp-specialised R=4 Q=64 L={L} {variant}")
    inp, pin = make_case(2, L, 3, 4, 64, seed=400 + L)
    zfull = torch.randn(inp.x.shape, device=DEV, generator=torch.Generator(DEV).manual_seed(11)
                        ).to(torch.bfloat16)
    y, fs, cB, cX = run_pro(inp, pin, variant, 64, zfull=zfull, seg=WS)
    slices = [(b, h) for b in range(2) for h in range(3)]
    ref, zref = oracle_prologue(inp, pin, variant, slices, zfull=zfull)
    compare(y, fs, cB, cX, ref, zref, slices, f"pro ws L={L} {variant}")


def test_prologue_continuation_ws():
    say("prologue continuation warp-specialised R=4 Q=64")
    L, L1 = 333, 190
    inp, pin = make_case(1, L, 2, 4, 64, seed=81)
    ya, fa, cBa, cXa = run_pro(inp, pin, "full", 64, t0=0, t1=L1, seg=WS)
    yb, fb, cBb, cXb = run_pro(inp, pin, "full", 64, init_state=fa, init_carry=(cBa, cXa),
                               t0=L1, t1=L, seg=WS)
    y = torch.cat([ya, yb], dim=1)
    slices = [(0, 0), (0, 1)]
    ref, _ = oracle_prologue(inp, pin, "full", slices)
    compare(y, fb, cBb, cXb, ref, None, slices, "pro continuation ws")


@pytest.mark.parametrize("gated", [False, True])
@pytest.mark.parametrize("R", [1, 4])
def test_prologue_decode(R, gated):
    """prefill (pro) of L tokens, then steps (pro) with fresh raw inputs: every
    step's y and the final state against the oracle scan over all tokens."""
    say(f"prologue decode R={R} gated={gated}")
    B, H, L, steps = 4, 3, 100, 5
    variant = "gated_wz" if gated else "full"
    inp, pin = make_case(B, L, H, R, 64, seed=31 + R)
    _, fs, (cB, cX) = m3.scan_fwd_pro(pin.xp, pin.Bp, pin.Cp, inp.dt, inp.A, inp.lam,
                                      inp.theta, inp.D, 64, pro_of(pin, variant), R,
                                      z=pin.zp if gated else None)
    slices = [(b, h) for b in range(B) for h in range(H)]
    hs = [h for _, h in slices]
    ref, _ = oracle_prologue(inp, pin, variant, slices)
    _, rs, rb, rx = oracle.scan(**ref)
    for s in range(steps):
        st = make_step_inputs(inp, s)
        sp = make_prologue_step_inputs(pin, B, s)
        y = m3.step_pro(fs, (cB, cX), sp.xp, sp.Bp, sp.Cp, st.dt, inp.A, st.lam, st.theta,
                        inp.D, pro_of(pin, variant), z=sp.zp if gated else None)
        torch.cuda.synchronize()
        stp = oracle.slices_of_step(sp.xp, sp.Bp, sp.Cp, st.dt, st.lam, st.theta, slices)
        Bn = oracle.rms_norm(stp["B"], oracle._np(pin.gB)[hs], oracle._np(pin.bB)[hs], EPS)
        Cn = oracle.rms_norm(stp["C"], oracle._np(pin.gC)[hs], oracle._np(pin.bC)[hs], EPS)
        Xn = oracle._np(pin.wx)[hs] * stp["x"][:, None, :]
        ry, rs, rb, rx = oracle.step(rs, rb, rx, Xn, Bn, Cn, stp["dt"], ref["A"][:, 0],
                                     stp["lam"], stp["theta"], ref["D"])
        if gated:
            zs = np.stack([oracle._np(sp.zp[b, h]) for b, h in slices])
            ry = oracle.gate(ry, oracle._np(pin.wz)[hs] * zs[:, None, :])
        for k, (b, h) in enumerate(slices):
            e = oracle.rel_err(y[b, h].double().cpu().numpy(), ry[k])
            assert e <= TOL, f"step {s} slice {(b, h)}: y rel err {e:.3g}"
    for k, (b, h) in enumerate(slices):
        e = oracle.rel_err(fs[b, h].double().cpu().numpy(), rs[k])
        assert e <= TOL, f"final state slice {(b, h)}: rel err {e:.3g}"
        ec = max(oracle.rel_err(cB[b, h].double().cpu().numpy(), rb[k]),
                 oracle.rel_err(cX[b, h].double().cpu().numpy(), rx[k]))
        assert ec <= TOL_CARRY, f"carry slice {(b, h)}: rel err {ec:.3g}"
    say(f"prologue decode R={R} gated={gated}: ok")


def sample_slices(batch, nheads, count, seed):
    rng = np.random.default_rng(seed)
    allsl = [(b, h) for b in range(batch) for h in range(nheads)]
    if len(allsl) <= count:
        return allsl
    pick = {allsl[0], allsl[-1]}
    for i in rng.permutation(len(allsl)):
        if len(pick) >= count:
            break
        pick.add(allsl[i])
    return sorted(pick)


@pytest.mark.parametrize("k", [1, 2, 3])
def test_prologue_workloads(k):
    """The prefill workloads' shapes with the whole prologue (norm, gains,
    biases, structured input; raw B', C', X' drawn by make_prologue_inputs):
    the SISO B=4 L=2048 prefill on every slice, the rank-4 B=8 L=4096 and
    B=1 L=65536 prefills on 16 seeded slices plus the first and the last."""
    w = WORKLOADS[k]
    say(f"prologue workload {k}")
    inp = workload_inputs(k, device=DEV)
    pin = make_prologue_inputs(w["batch"], w["seqlen"], w["nheads"], w["headdim"], w["dstate"],
                               w["rank"], io="bf16", seed=k, device=DEV)
    del inp.x, inp.Bm, inp.Cm
    torch.cuda.empty_cache()
    y, fs, cB, cX = run_pro(inp, pin, "full", w["chunk"])
    slices = sample_slices(w["batch"], w["nheads"], 10**6 if k == 1 else 18, 60 + k)
    ref, _ = oracle_prologue(inp, pin, "full", slices)
    compare(y, fs, cB, cX, ref, None, slices, f"pro workload {k}")


# ---------------------------------------------------------------------------
# Output norm fused into the y store (Sec. 4 hybrid models; App. norm type /
# placement ablation): grouped RMS of y before or after the output gate.
# The kernel normalises y as the plain scan would store it (bf16); the oracle
# normalises its fp64 y.  The bar is y's own (|dy| <= d = 2e-2 of the
# slice's max |y|) carried through the norm: for n = u / r over a group, r =
# sqrt(mean(u^2) + eps) (1-Lipschitz in u: r' >= r - d_u), an error of at
# most d_u per element gives |n'_e - n_e| <= |du_e| / r' + |n_e| |r - r'| / r'
# <= (1 + |n_e|) d_u / (r - d_u) when r > d_u, and at most sqrt(group) +
# |n_e| in any case (unit-RMS vectors); u = y (pre-gate; the factor
# gain |SiLU(z)| follows, d_u = d) or u = y o SiLU(z) (post-gate, d_u =
# max_group |SiLU(z)| d); plus the bf16 rounding of the output (2^-8 of each
# element).  A flat relative bar on the output would not hold for small
# groups: their RMS can be far below the slice's max |y|, and the norm
# divides y's absolute error by it.
# ---------------------------------------------------------------------------

ONORM = {
    # name: (pre-gate, group, gate: None / "z" / "wz", gain)
    "pre16_z": (True, 16, "z", True),
    "post64_z": (False, 64, "z", True),
    "pre8_nogate": (True, 8, None, False),
    "post32_wz": (False, 32, "wz", True),
    "pre64_wz": (True, 64, "wz", False),
}
OEPS = 1e-5


def onorm_pro(pin, name, gain_t):
    pre, group, gate, gain = ONORM[name]
    variant = {"z": "gated_z", "wz": "gated_wz", None: "full"}[gate]
    base = pro_of(pin, variant)
    base.out_norm = m3.M3_OUT_NORM_PRE_GATE if pre else m3.M3_OUT_NORM_POST_GATE
    base.out_group = group
    base.out_eps = OEPS
    base.out_gain = m3._p(gain_t) if gain else None
    return base, variant


def gain_for(gain_t, hs, ry):
    """The heads' gains [S, R, P], with a token axis when y has one."""
    g = oracle._np(gain_t)[hs]
    return g[:, None] if ry.ndim == 4 else g


def onorm_reference(ry, zref, name, gain_t, hs):
    pre, group, gate, gain = ONORM[name]
    g = gain_for(gain_t, hs, ry) if gain else None
    return oracle.out_norm(ry, group, eps=OEPS, gain=g, z=zref, pre_gate=pre)


def onorm_bound(ry, zref, name, gain_t, hs):
    """Per-element bar of the normalised output (above), from the oracle's
    y [S, L, R, P] and gate input."""
    pre, group, gate, gain = ONORM[name]
    sg = np.ones_like(ry) if zref is None else np.abs(oracle.silu(zref))
    g = np.abs(gain_for(gain_t, hs, ry)) if gain else 1.0
    u = ry if pre else ry * (np.ones_like(ry) if zref is None else oracle.silu(zref))
    shp = u.shape[:-1] + (u.shape[-1] // group, group)
    rms = np.sqrt(np.mean(u.reshape(shp) ** 2, axis=-1, keepdims=True) + OEPS)
    n = np.abs(u.reshape(shp) / rms).reshape(u.shape)
    rms = np.broadcast_to(rms, shp).reshape(u.shape)
    smax = np.broadcast_to(np.max(sg.reshape(shp), axis=-1, keepdims=True), shp).reshape(u.shape)
    dy = TOL * np.max(np.abs(ry).reshape(ry.shape[0], -1), axis=1).reshape((-1,) + (1,) * (ry.ndim - 1))
    du = dy * (1.0 if pre else smax)
    fac = g * (sg if pre else 1.0)
    near = (1.0 + n) * du / np.maximum(rms - du, 1e-300)
    return fac * np.where(rms > du, np.minimum(near, np.sqrt(group) + n), np.sqrt(group) + n)


def check_onorm(got, want, bound, label):
    """|got - want| within the propagated bar plus the output rounding; the
    plain relative error is reported beside it."""
    err = np.abs(got - want)
    lim = bound + 2.0 ** -8 * np.abs(want) + 1e-30
    worst = float(np.max(err / lim))
    assert worst <= 1.0, f"{label}: error {worst:.3g} of the propagated bar"
    return worst, oracle.rel_err(got, want)


@pytest.mark.parametrize("name", list(ONORM))
@pytest.mark.parametrize("R,Q,L,seg", [(1, 64, 300, 0), (4, 64, 200, 0), (2, 32, 77, 0), (4, 128, 130, 0),
                                       (4, 64, 200, 1 << 20)])
def test_out_norm_scan(R, Q, L, seg, name):
    say(f"output norm scan R={R} Q={Q} L={L} seg={seg} {name}")
    B, H = 2, 3
    inp, pin = make_case(B, L, H, R, Q, seed=R * 50 + Q + L + 7)
    zfull = torch.randn(inp.x.shape, device=DEV, generator=torch.Generator(DEV).manual_seed(19)
                        ).to(torch.bfloat16)
    gain_t = 0.5 + torch.rand((H, R, 64), device=DEV, generator=torch.Generator(DEV).manual_seed(5))
    p, variant = onorm_pro(pin, name, gain_t)
    x, z = gpu_args(inp, pin, variant, zfull)
    y, fs, (cB, cX) = m3.scan_fwd_pro(x, pin.Bp, pin.Cp, inp.dt, inp.A, inp.lam, inp.theta, inp.D,
                                      Q, p, R, z=z, check=True, seg=seg)
    torch.cuda.synchronize()
    slices = [(b, h) for b in range(B) for h in range(H)]
    ref, zref = oracle_prologue(inp, pin, variant, slices, zfull=zfull)
    ry, rs, _, _ = oracle.scan(**ref)
    hs = [h for _, h in slices]
    want = onorm_reference(ry, zref, name, gain_t, hs)
    bound = onorm_bound(ry, zref, name, gain_t, hs)
    worst, worst_rel = 0.0, 0.0
    for k, (b, h) in enumerate(slices):
        gy = y[b, :, h].double().cpu().numpy()
        assert np.all(np.isfinite(gy)), (b, h)
        w, r = check_onorm(gy, want[k], bound[k], f"{name} slice {(b, h)}")
        worst, worst_rel = max(worst, w), max(worst_rel, r)
        e = oracle.rel_err(fs[b, h].double().cpu().numpy(), rs[k])
        assert e <= TOL, f"{name} slice {(b, h)}: final state rel err {e:.3g}"
    say(f"output norm scan R={R} Q={Q} L={L} {name}: {worst:.3g} of the bar "
        f"(plain rel err {worst_rel:.3g})")


@pytest.mark.parametrize("name", ["pre16_z", "post64_z", "pre8_nogate"])
@pytest.mark.parametrize("R", [1, 4])
def test_out_norm_decode(R, name):
    """Decode steps with the output norm after a prefill with it: each step's
    y against the oracle's step output normalised the same way."""
    say(f"output norm decode R={R} {name}")
    B, H, L, steps = 4, 3, 100, 3
    inp, pin = make_case(B, L, H, R, 64, seed=41 + R)
    gain_t = 0.5 + torch.rand((H, R, 64), device=DEV, generator=torch.Generator(DEV).manual_seed(6))
    p, variant = onorm_pro(pin, name, gain_t)
    gate = ONORM[name][2]
    zfull = torch.randn(inp.x.shape, device=DEV, generator=torch.Generator(DEV).manual_seed(20)
                        ).to(torch.bfloat16)
    x, z = gpu_args(inp, pin, variant, zfull)
    _, fs, (cB, cX) = m3.scan_fwd_pro(x, pin.Bp, pin.Cp, inp.dt, inp.A, inp.lam, inp.theta,
                                      inp.D, 64, p, R, z=z)
    slices = [(b, h) for b in range(B) for h in range(H)]
    hs = [h for _, h in slices]
    ref, _ = oracle_prologue(inp, pin, variant, slices, zfull=zfull)
    _, rs, rb, rx = oracle.scan(**ref)
    sx = VARIANTS[variant][3]
    for s in range(steps):
        st = make_step_inputs(inp, s)
        sp = make_prologue_step_inputs(pin, B, s)
        zs_full = torch.randn((B, H, R, 64), device=DEV,
                              generator=torch.Generator(DEV).manual_seed(100 + s)).to(torch.bfloat16)
        zt = None if gate is None else (sp.zp if gate == "wz" else zs_full)
        xt = sp.xp if sx else st.x
        y = m3.step_pro(fs, (cB, cX), xt, sp.Bp, sp.Cp, st.dt, inp.A, st.lam, st.theta,
                        inp.D, p, z=zt)
        torch.cuda.synchronize()
        stp = oracle.slices_of_step(xt, sp.Bp, sp.Cp, st.dt, st.lam, st.theta, slices)
        Bn = oracle.rms_norm(stp["B"], oracle._np(pin.gB)[hs], oracle._np(pin.bB)[hs], EPS)
        Cn = oracle.rms_norm(stp["C"], oracle._np(pin.gC)[hs], oracle._np(pin.bC)[hs], EPS)
        Xn = oracle._np(pin.wx)[hs] * stp["x"][:, None, :] if sx else stp["x"]
        ry, rs, rb, rx = oracle.step(rs, rb, rx, Xn, Bn, Cn, stp["dt"], ref["A"][:, 0],
                                     stp["lam"], stp["theta"], ref["D"])
        zref = None
        if gate == "wz":
            zref = oracle._np(pin.wz)[hs] * np.stack([oracle._np(sp.zp[b, h]) for b, h in slices])[:, None, :]
        elif gate == "z":
            zref = np.stack([oracle._np(zs_full[b, h]) for b, h in slices])
        want = onorm_reference(ry, zref, name, gain_t, hs)
        bound = onorm_bound(ry, zref, name, gain_t, hs)
        for k, (b, h) in enumerate(slices):
            check_onorm(y[b, h].double().cpu().numpy(), want[k], bound[k],
                        f"{name} step {s} slice {(b, h)}")
    say(f"output norm decode R={R} {name}: ok")
