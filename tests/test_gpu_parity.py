"""GPU parity: libm3 (through the C ABI) against the fp64 CPU oracle.

Metric: per (batch, head) slice, max|gpu - oracle| / max|oracle| (infinity
norm relative error), for y, the final state and (decode) every step's y.
Bars: 1e-5 for the fp32 build, 2e-2 for bf16 inputs.  The oracle reads the
exact (bf16-rounded) inputs the GPU received.  Integer-like results (the
carry, a copy of the last token's B and x) must match bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2603_15569_amd import m3
from paper_2603_15569_amd.inputs import (WORKLOADS, make_gate_input, make_scan_inputs,
                                         make_step_inputs, workload_inputs)

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}
DEV = "cuda:0"


def say(msg):
    print(f"[gpu-case] {msg}", flush=True)


MODES = ("seg", "per_chunk", "split")   # segmented single-pass (default), one chunk per WG, 3 kernels


def run_scan(inp, chunk, init_state=None, init_carry=None, nan_fill=True, mode="seg", seg=0,
             z=None):
    """Scan with every output pre-filled with NaN, so an unwritten element fails."""
    x = inp.x
    B_, L, H, R, P = x.shape
    N = inp.Bm.shape[-1]
    out = None
    if nan_fill:
        out = (torch.full_like(x, float("nan")),
               torch.full((B_, H, N, P), float("nan"), device=x.device),
               torch.full((B_, H, R, N), float("nan"), device=x.device, dtype=x.dtype),
               torch.full((B_, H, R, P), float("nan"), device=x.device, dtype=x.dtype))
    kw = dict(split=mode == "split", per_chunk=mode == "per_chunk", seg=seg)
    nbytes = m3.workspace_bytes(m3.scan_dims(x, inp.Bm, chunk, inp.A, **kw))
    # a single-pass kernel serves this shape iff its workspace differs from the split path's
    single_pass = mode != "split" and nbytes != m3.workspace_bytes(
        m3.scan_dims(x, inp.Bm, chunk, inp.A, split=True))
    ws = torch.zeros(max(nbytes, 16), dtype=torch.uint8, device=x.device)
    y, fs, (cB, cX) = m3.scan_fwd(x, inp.Bm, inp.Cm, inp.dt, inp.A, inp.lam, inp.theta, inp.D,
                                  chunk=chunk, init_state=init_state, init_carry=init_carry,
                                  out=out, workspace=ws, z=z, **kw)
    torch.cuda.synchronize()
    # no look-back wait gave up (m3_scan_check; zero without a device read
    # for the three-kernel path)
    assert m3.scan_check(m3.scan_dims(x, inp.Bm, chunk, inp.A, **kw), ws) == 0, "look-back wait timed out"
    if single_pass and L > 0:
        # the same read directly: after a clean call both timeout words of the
        # control block (words 1 and 3, for even and odd call epochs) are zero
        w = ws[:16].view(torch.int32).cpu().numpy()
        assert w[1] == 0 and w[3] == 0
    return y, fs, cB, cX


def check_slices(inp, y, fs, cB, cX, slices, tol, init_state=None, init_carry=None, label="",
                 z=None):
    ref = oracle.slices_of_scan(inp.x, inp.Bm, inp.Cm, inp.dt, inp.A, inp.lam, inp.theta,
                                inp.D, slices)
    kw = {}
    if init_state is not None:
        kw["init_state"] = oracle.slices_of_state(init_state, slices)
    if init_carry is not None:
        kw["init_B"] = oracle.slices_of_state(init_carry[0], slices)
        kw["init_X"] = oracle.slices_of_state(init_carry[1], slices)
    ry, rs, rb, rx = oracle.scan(**ref, **kw)
    if z is not None:   # the output gate y o SiLU(z)
        ry = oracle.gate(ry, np.stack([oracle._np(z[b, :, h]) for b, h in slices]))
    worst = 0.0
    for k, (b, h) in enumerate(slices):
        gy = y[b, :, h].double().cpu().numpy()
        gs = fs[b, h].double().cpu().numpy()
        assert np.all(np.isfinite(gy)) and np.all(np.isfinite(gs)), f"{label} non-finite {(b, h)}"
        e = max(oracle.rel_err(gy, ry[k]), oracle.rel_err(gs, rs[k]))
        worst = max(worst, e)
        assert e <= tol, f"{label} slice {(b, h)}: rel err {e:.3g} > {tol}"
        assert np.array_equal(cB[b, h].double().cpu().numpy(), rb[k]), f"{label} carry B {(b, h)}"
        assert np.array_equal(cX[b, h].double().cpu().numpy(), rx[k]), f"{label} carry X {(b, h)}"
    say(f"{label}: worst rel err {worst:.3g} over {len(slices)} slices")
    return worst


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


# ---------------------------------------------------------------------------
# Workloads
# ---------------------------------------------------------------------------

def test_workload0_tiny_siso_fp32():
    say("workload 0: tiny SISO fp32, full check")
    inp = workload_inputs(0, device=DEV)
    y, fs, cB, cX = run_scan(inp, WORKLOADS[0]["chunk"])
    check_slices(inp, y, fs, cB, cX, sample_slices(1, 2, 99, 0), TOL["f32"], label="w0")


def test_workload1_siso_bf16():
    say("workload 1: SISO bf16 prefill, all 64 slices")
    w = WORKLOADS[1]
    inp = workload_inputs(1, device=DEV)
    y, fs, cB, cX = run_scan(inp, w["chunk"])
    check_slices(inp, y, fs, cB, cX, sample_slices(w["batch"], w["nheads"], 10**6, 1),
                 TOL["bf16"], label="w1")


def test_workload2_mimo_bf16():
    say("workload 2: MIMO R=4 bf16 prefill, 18 sampled slices")
    w = WORKLOADS[2]
    inp = workload_inputs(2, device=DEV)
    y, fs, cB, cX = run_scan(inp, w["chunk"])
    check_slices(inp, y, fs, cB, cX, sample_slices(w["batch"], w["nheads"], 18, 2),
                 TOL["bf16"], label="w2")


def check_tail_chunks(inp, y, slices, chunk, nlast, tol, label):
    """The last `nlast` chunks of each slice checked on their own (error
    normalised by that chunk's largest output), so that drift late in a long
    sequence cannot hide under the slice-wide maximum."""
    L = y.shape[1]
    t0 = max(0, L - nlast * chunk)
    ref = oracle.slices_of_scan(inp.x, inp.Bm, inp.Cm, inp.dt, inp.A, inp.lam, inp.theta,
                                inp.D, slices)
    ry = oracle.scan(**ref)[0]
    worst = 0.0
    for k, (b, h) in enumerate(slices):
        gy = y[b, :, h].double().cpu().numpy()
        for c0 in range(t0, L, chunk):
            c1 = min(L, c0 + chunk)
            e = oracle.rel_err(gy[c0:c1], ry[k][c0:c1])
            worst = max(worst, e)
            assert e <= tol, f"{label} slice {(b, h)} tokens {c0}..{c1 - 1}: rel err {e:.3g}"
    say(f"{label}: worst per-chunk rel err {worst:.3g} over the last {nlast} chunks")


def test_workload3_long_mimo_bf16():
    w = WORKLOADS[3]
    slices = sample_slices(w["batch"], w["nheads"], 18, 3)   # 16 seeded + first and last
    assert (0, 0) in slices and (w["batch"] - 1, w["nheads"] - 1) in slices and len(slices) == 18
    say(f"workload 3: long-context MIMO prefill L=65536, {len(slices)} sampled slices")
    inp = workload_inputs(3, device=DEV)
    y, fs, cB, cX = run_scan(inp, w["chunk"])
    check_slices(inp, y, fs, cB, cX, slices, TOL["bf16"], label="w3")
    check_tail_chunks(inp, y, slices[:4] + slices[-2:], w["chunk"], 8, TOL["bf16"], label="w3 tail")


def test_workload4_decode_loop():
    """State from a 1024-token prefill (B=256, H=32, R=4), then 1024 decode
    steps with fresh inputs; every step's y and the final state checked on 18
    slices (16 seeded, the first and the last)."""
    w = WORKLOADS[4]
    slices = sample_slices(w["batch"], w["nheads"], 18, 4)   # 16 seeded + first and last
    assert (0, 0) in slices and (w["batch"] - 1, w["nheads"] - 1) in slices and len(slices) == 18
    say(f"workload 4: prefill B=256 L=1024 then 1024 steps, {len(slices)} sampled slices")
    inp = workload_inputs(4, device=DEV)
    y, fs, cB, cX = run_scan(inp, w["chunk"], nan_fill=False)
    ref = oracle.slices_of_scan(inp.x, inp.Bm, inp.Cm, inp.dt, inp.A, inp.lam, inp.theta,
                                inp.D, slices)
    ry, rs, rb, rx = oracle.scan(**ref)
    del y
    bi = torch.tensor([b for b, _ in slices], device=DEV)
    hi = torch.tensor([h for _, h in slices], device=DEV)
    A_s, D_s = ref["A"][:, 0], ref["D"]
    worst = 0.0
    for s in range(w["steps"]):
        st = make_step_inputs(inp, s)
        yt = m3.step(fs, (cB, cX), st.x, st.Bm, st.Cm, st.dt, inp.A, st.lam, st.theta, inp.D)
        g = lambda t: t[bi, hi].double().cpu().numpy()
        ryt, rs, rb, rx = oracle.step(rs, rb, rx, g(st.x), g(st.Bm), g(st.Cm), g(st.dt),
                                      A_s, g(st.lam), g(st.theta), D_s)
        gy = g(yt)
        for k in range(len(slices)):
            e = oracle.rel_err(gy[k], ryt[k])
            worst = max(worst, e)
            assert e <= TOL["bf16"], f"step {s} slice {slices[k]} rel err {e:.3g}"
    gs = fs[bi, hi].double().cpu().numpy()
    for k in range(len(slices)):
        e = oracle.rel_err(gs[k], rs[k])
        worst = max(worst, e)
        assert e <= TOL["bf16"], f"final state slice {slices[k]} rel err {e:.3g}"
    assert np.array_equal(cB[bi, hi].double().cpu().numpy(), rb)
    assert np.array_equal(cX[bi, hi].double().cpu().numpy(), rx)
    say(f"w4: worst rel err {worst:.3g}")


# ---------------------------------------------------------------------------
# Shapes, ragged lengths and edge cases
# ---------------------------------------------------------------------------

SHAPES = [  # io, N, P, R, Q
    ("f32", 16, 16, 1, 64), ("f32", 16, 16, 2, 32), ("f32", 16, 16, 4, 16),
    ("f32", 16, 16, 4, 64), ("f32", 128, 64, 2, 32), ("f32", 128, 64, 4, 16),
    ("f32", 128, 64, 4, 32),
    ("bf16", 128, 64, 1, 64), ("bf16", 128, 64, 1, 128), ("bf16", 128, 64, 2, 64),
    ("bf16", 128, 64, 4, 32), ("bf16", 128, 64, 4, 64), ("bf16", 128, 64, 4, 128),
    # smaller states (the paper's state-size sweep): the three-kernel path
    ("bf16", 64, 64, 1, 64), ("bf16", 64, 64, 2, 64), ("bf16", 64, 64, 4, 32),
    ("bf16", 32, 64, 1, 64), ("bf16", 32, 64, 4, 16),
]


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("io,N,P,R,Q", SHAPES)
def test_shapes_ragged(io, N, P, R, Q, mode):
    """Several chunks plus a ragged tail, two batch rows and three heads, on
    each prefill kernel (shapes a kernel is not built for fall back)."""
    L = 3 * Q + Q // 2 + 3
    say(f"shape io={io} N={N} P={P} R={R} Q={Q} L={L} mode={mode}")
    inp = make_scan_inputs(2, L, 3, P, N, R, io=io, seed=11 + N + R + Q, device=DEV, chunk=Q)
    y, fs, cB, cX = run_scan(inp, Q, mode=mode)
    check_slices(inp, y, fs, cB, cX, sample_slices(2, 3, 99, 5), TOL[io], label=f"{io}/{N}/{R}/{Q}")


@pytest.mark.parametrize("mode", ["seg", "per_chunk"])
@pytest.mark.parametrize("io", ["f32", "bf16"])
@pytest.mark.parametrize("L", [1, 2, 63, 64, 65])
def test_short_sequences(io, L, mode):
    N, P, R, Q = (128, 64, 2, 32) if io == "f32" else (128, 64, 4, 64)
    say(f"short io={io} L={L} mode={mode}")
    inp = make_scan_inputs(2, L, 2, P, N, R, io=io, seed=100 + L, device=DEV, chunk=Q)
    y, fs, cB, cX = run_scan(inp, Q, mode=mode)
    check_slices(inp, y, fs, cB, cX, sample_slices(2, 2, 99, 6), TOL[io], label=f"short{L}")


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_empty_sequence(io):
    N, P, R, Q = (16, 16, 2, 32) if io == "f32" else (128, 64, 2, 64)
    say(f"empty io={io}")
    dt = torch.float32 if io == "f32" else torch.bfloat16
    inp = make_scan_inputs(2, 0, 2, P, N, R, io=io, seed=3, device=DEV, chunk=Q)
    st0 = torch.randn(2, 2, N, P, device=DEV)
    c0 = (torch.randn(2, 2, R, N, device=DEV).to(dt), torch.randn(2, 2, R, P, device=DEV).to(dt))
    y, fs, cB, cX = run_scan(inp, Q, init_state=st0, init_carry=c0)
    assert y.numel() == 0
    assert torch.equal(fs, st0) and torch.equal(cB, c0[0]) and torch.equal(cX, c0[1])
    y, fs, cB, cX = run_scan(inp, Q)
    assert torch.count_nonzero(fs) == 0 and torch.count_nonzero(cB.float()) == 0


@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_segment_resume_and_decode_consistency(io):
    """scan(0:L1) -> (state, carry) -> scan(L1:L) equals scan(0:L); and
    scan(0:L) then one m3_step equals scan(0:L+1) at token L (the decode
    state is the physical-frame state plus the previous token's B and x)."""
    N, P, R, Q = (16, 16, 2, 32) if io == "f32" else (128, 64, 4, 64)
    L, L1 = 200, 77
    say(f"segment resume io={io}")
    inp = make_scan_inputs(2, L + 1, 2, P, N, R, io=io, seed=42, device=DEV, chunk=Q)

    def part(t0, t1):
        return type(inp)(x=inp.x[:, t0:t1].contiguous(), Bm=inp.Bm[:, t0:t1].contiguous(),
                         Cm=inp.Cm[:, t0:t1].contiguous(), dt=inp.dt[:, t0:t1].contiguous(),
                         A=inp.A, lam=inp.lam[:, t0:t1].contiguous(),
                         theta=inp.theta[:, t0:t1].contiguous(), D=inp.D, chunk=Q)
    yf, fsf, _, _ = run_scan(part(0, L + 1), Q)
    ya, fsa, cBa, cXa = run_scan(part(0, L1), Q)
    yb, fsb, cBb, cXb = run_scan(part(L1, L), Q, init_state=fsa, init_carry=(cBa, cXa))
    check_slices(part(L1, L), yb, fsb, cBb, cXb, sample_slices(2, 2, 99, 7), TOL[io],
                 init_state=fsa, init_carry=(cBa, cXa), label="resume")
    # decode consistency: one step from the state after L tokens
    yl, fsl, cBl, cXl = run_scan(part(0, L), Q)
    xt, Bt, Ct = inp.x[:, L].contiguous(), inp.Bm[:, L].contiguous(), inp.Cm[:, L].contiguous()
    yt = m3.step(fsl, (cBl, cXl), xt, Bt, Ct, inp.dt[:, L].contiguous(), inp.A,
                 inp.lam[:, L].contiguous(), inp.theta[:, L].contiguous(), inp.D)
    torch.cuda.synchronize()
    tol = TOL[io] if io == "bf16" else 1e-5
    for b in range(2):
        for h in range(2):
            assert oracle.rel_err(yt[b, h].double().cpu().numpy(),
                                  yf[b, L, h].double().cpu().numpy()) <= tol
            assert oracle.rel_err(fsl[b, h].cpu().numpy(), fsf[b, h].cpu().numpy()) <= tol


@pytest.mark.parametrize("mode,seg", [("seg", 1), ("seg", 2), ("seg", 0), ("per_chunk", 0)])
@pytest.mark.parametrize("io", ["f32", "bf16"])
def test_chunk_boundary_impulse(io, mode, seg):
    """Only x at the last token of a chunk is nonzero and lambda there is 0,
    so every later output flows through the cross-chunk previous-input term
    (sigma of that token reads the next chunk's lambda and dt); with one
    chunk per segment the boundary is also a segment boundary."""
    N, P, R, Q = (128, 64, 2, 32) if io == "f32" else (128, 64, 2, 64)
    L = 3 * Q
    say(f"boundary impulse io={io} mode={mode} seg={seg}")
    inp = make_scan_inputs(1, L, 2, P, N, R, io=io, seed=9, device=DEV, chunk=Q)
    j = Q - 1
    keep = inp.x[:, j].clone()
    inp.x.zero_()
    inp.x[:, j] = keep
    inp.lam[:, j] = 0.0
    y, fs, cB, cX = run_scan(inp, Q, mode=mode, seg=seg)
    assert torch.count_nonzero(y[:, :j].float()) == 0
    check_slices(inp, y, fs, cB, cX, [(0, 0), (0, 1)], TOL[io], label="impulse")
    # beyond the boundary the output is large (not a trivially small residue)
    assert y[:, j + 1:].float().abs().max() > 1e-3


SEG_SHAPES = [("f32", 128, 64, 2, 32), ("f32", 128, 64, 4, 16), ("bf16", 128, 64, 1, 64),
              ("bf16", 128, 64, 1, 128), ("bf16", 128, 64, 4, 64), ("bf16", 128, 64, 2, 32)]


@pytest.mark.parametrize("seg", [1, 2, 3, 8, 0])
@pytest.mark.parametrize("io,N,P,R,Q", SEG_SHAPES)
def test_segment_lengths(io, N, P, R, Q, seg):
    """Segmented kernel: eight chunks (the last ragged) split into segments of
    1, 2, 3 (uneven) or 8 chunks (no look-back), or the library's choice."""
    L = 7 * Q + Q // 2 + 1
    say(f"segments io={io} R={R} Q={Q} L={L} seg={seg}")
    inp = make_scan_inputs(2, L, 3, P, N, R, io=io, seed=70 + R + Q + seg, device=DEV, chunk=Q)
    y, fs, cB, cX = run_scan(inp, Q, seg=seg)
    check_slices(inp, y, fs, cB, cX, sample_slices(2, 3, 99, 8), TOL[io],
                 label=f"seg{seg}/{io}/{R}/{Q}")


@pytest.mark.parametrize("seg", [1, 3, 0])
def test_segment_lengths_with_initial_state(seg):
    """A continued sequence (initial state and carry) through every segment split."""
    N, P, R, Q = 128, 64, 4, 32
    L = 9 * Q + 5
    say(f"segments + init seg={seg}")
    inp = make_scan_inputs(2, L, 2, P, N, R, io="bf16", seed=90 + seg, device=DEV, chunk=Q)
    st0 = torch.randn(2, 2, N, P, device=DEV)
    c0 = (torch.randn(2, 2, R, N, device=DEV).to(torch.bfloat16),
          torch.randn(2, 2, R, P, device=DEV).to(torch.bfloat16))
    y, fs, cB, cX = run_scan(inp, Q, init_state=st0, init_carry=c0, seg=seg)
    check_slices(inp, y, fs, cB, cX, sample_slices(2, 2, 99, 9), TOL["bf16"], init_state=st0,
                 init_carry=c0, label=f"seg{seg}+init")


@pytest.mark.parametrize("L", [1, 37, 64, 64 * 5 + 17, 64 * 12])
def test_one_segment_per_slice(L):
    """Each slice scanned whole by one workgroup (R=4, chunk 64: the
    warp-specialised kernel): one token, one partial chunk, one full chunk,
    a ragged tail and whole chunks, continuing from an initial state and
    carry."""
    N, P, R, Q = 128, 64, 4, 64
    say(f"one segment per slice bf16 R={R} Q={Q} L={L}")
    inp = make_scan_inputs(2, L, 3, P, N, R, io="bf16", seed=400 + L, device=DEV, chunk=Q)
    st0 = torch.randn(2, 3, N, P, device=DEV)
    c0 = (torch.randn(2, 3, R, N, device=DEV).to(torch.bfloat16),
          torch.randn(2, 3, R, P, device=DEV).to(torch.bfloat16))
    y, fs, cB, cX = run_scan(inp, Q, init_state=st0, init_carry=c0, seg=1 << 20)
    check_slices(inp, y, fs, cB, cX, sample_slices(2, 3, 99, 3), TOL["bf16"], init_state=st0,
                 init_carry=c0, label=f"one segment L={L}")
    y0, fs0, _, _ = run_scan(inp, Q, seg=1 << 20)
    check_slices(inp, y0, fs0, cB, cX, sample_slices(2, 3, 99, 4), TOL["bf16"],
                 label=f"one segment L={L} zero state")


def test_chunk_size_invariance():
    """Results do not depend on the chunk length (Sec. 3.3)."""
    say("chunk invariance bf16 R=4 Q in {32, 64, 128}")
    inp = make_scan_inputs(2, 700, 2, 64, 128, 4, io="bf16", seed=5, device=DEV)
    ys = [run_scan(inp, Q) for Q in (32, 64, 128)]
    for y, fs, _, _ in ys[1:]:
        for b in range(2):
            for h in range(2):
                assert oracle.rel_err(y[b, :, h].double().cpu().numpy(),
                                      ys[0][0][b, :, h].double().cpu().numpy()) <= 2e-2
                assert oracle.rel_err(fs[b, h].cpu().numpy(), ys[0][1][b, h].cpu().numpy()) <= 2e-2


def test_per_token_A():
    """Mamba-3's data-dependent A_t passed as a [B, L, H] tensor."""
    say("per-token A fp32")
    inp = make_scan_inputs(2, 150, 2, 16, 16, 2, io="f32", seed=21, device=DEV, chunk=32)
    A_t = -torch.rand(2, 150, 2, device=DEV) * 4 - 0.1
    y, fs, (cB, cX) = m3.scan_fwd(inp.x, inp.Bm, inp.Cm, inp.dt, A_t, inp.lam, inp.theta, inp.D,
                                  chunk=32)
    torch.cuda.synchronize()
    sl = [(0, 0), (1, 1)]
    ref = oracle.slices_of_scan(inp.x, inp.Bm, inp.Cm, inp.dt, inp.A, inp.lam, inp.theta,
                                inp.D, sl)
    ref["A"] = np.stack([A_t[b, :, h].double().cpu().numpy() for b, h in sl])
    ry, rs, _, _ = oracle.scan(**ref)
    for k, (b, h) in enumerate(sl):
        assert oracle.rel_err(y[b, :, h].double().cpu().numpy(), ry[k]) <= 1e-5
        assert oracle.rel_err(fs[b, h].cpu().numpy(), rs[k]) <= 1e-5


@pytest.mark.parametrize("mode,seg", [("seg", 1 << 20), ("seg", 2), ("per_chunk", 0)])
def test_per_token_A_bf16_mimo(mode, seg):
    """Per-token A_t through the bf16 rank-4 kernels: one segment per slice
    (the warp-specialised kernel), two-chunk segments and one chunk per
    workgroup."""
    say(f"per-token A bf16 R=4 mode={mode} seg={seg}")
    L = 3 * 64 + 29
    inp = make_scan_inputs(2, L, 2, 64, 128, 4, io="bf16", seed=23, device=DEV, chunk=64)
    A_t = -torch.rand(2, L, 2, device=DEV) * 4 - 0.1
    kw = dict(per_chunk=mode == "per_chunk", seg=seg)
    y, fs, (cB, cX) = m3.scan_fwd(inp.x, inp.Bm, inp.Cm, inp.dt, A_t, inp.lam, inp.theta, inp.D,
                                  chunk=64, **kw)
    torch.cuda.synchronize()
    sl = [(0, 0), (1, 1)]
    ref = oracle.slices_of_scan(inp.x, inp.Bm, inp.Cm, inp.dt, inp.A, inp.lam, inp.theta,
                                inp.D, sl)
    ref["A"] = np.stack([A_t[b, :, h].double().cpu().numpy() for b, h in sl])
    ry, rs, _, _ = oracle.scan(**ref)
    for k, (b, h) in enumerate(sl):
        assert oracle.rel_err(y[b, :, h].double().cpu().numpy(), ry[k]) <= TOL["bf16"]
        assert oracle.rel_err(fs[b, h].cpu().numpy(), rs[k]) <= TOL["bf16"]


@pytest.mark.parametrize("mode,seg", [("seg", 0), ("seg", 1 << 20), ("seg", 2), ("per_chunk", 0)])
def test_determinism(mode, seg):
    """Two runs give bitwise-identical outputs (no atomics in reductions)."""
    say(f"determinism bf16 R=4 mode={mode} seg={seg}")
    inp = make_scan_inputs(2, 300, 4, 64, 128, 4, io="bf16", seed=8, device=DEV)
    a = run_scan(inp, 64, mode=mode, seg=seg)
    b = run_scan(inp, 64, mode=mode, seg=seg)
    for u, v in zip(a, b):
        assert torch.equal(u, v)


@pytest.mark.parametrize("io,N,P,R", [("f32", 16, 16, 1), ("f32", 128, 64, 4),
                                      ("bf16", 128, 64, 1), ("bf16", 128, 64, 4),
                                      ("bf16", 64, 64, 1), ("bf16", 64, 64, 4),
                                      ("bf16", 32, 64, 2)])
def test_decode_steps_small(io, N, P, R):
    """A few decode steps from a random state and carry, every output checked."""
    say(f"decode small io={io} N={N} R={R}")
    dt = torch.float32 if io == "f32" else torch.bfloat16
    inp = make_scan_inputs(3, 4, 5, P, N, R, io=io, seed=31, device=DEV)
    state = torch.randn(3, 5, N, P, device=DEV)
    cB = torch.randn(3, 5, R, N, device=DEV).to(dt)
    cX = torch.randn(3, 5, R, P, device=DEV).to(dt)
    sl = [(b, h) for b in range(3) for h in range(5)]
    rs = oracle.slices_of_state(state, sl)
    rb, rx = oracle.slices_of_state(cB, sl), oracle.slices_of_state(cX, sl)
    A_s = np.array([float(inp.A[h]) for _, h in sl])
    D_s = np.array([float(inp.D[h]) for _, h in sl])
    tol = TOL[io]
    for s in range(4):
        st = make_step_inputs(inp, s)
        y = torch.full_like(st.x, float("nan"))
        m3.step(state, (cB, cX), st.x, st.Bm, st.Cm, st.dt, inp.A, st.lam, st.theta, inp.D, y=y)
        torch.cuda.synchronize()
        p = oracle.slices_of_step(st.x, st.Bm, st.Cm, st.dt, st.lam, st.theta, sl)
        ry, rs, rb, rx = oracle.step(rs, rb, rx, p["x"], p["B"], p["C"], p["dt"], A_s, p["lam"],
                                     p["theta"], D_s)
        for k, (b, h) in enumerate(sl):
            assert oracle.rel_err(y[b, h].double().cpu().numpy(), ry[k]) <= tol
            assert oracle.rel_err(state[b, h].cpu().numpy(), rs[k]) <= tol
        assert np.array_equal(oracle.slices_of_state(cB, sl), rb)


# ---------------------------------------------------------------------------
# Output gate y o SiLU(z) (m3_scan_fwd_gated, m3_step_gated)
# ---------------------------------------------------------------------------

GATE_CASES = [  # io, N, P, R, Q, mode, seg
    ("f32", 16, 16, 1, 64, "seg", 0), ("f32", 16, 16, 1, 64, "per_chunk", 0),
    ("f32", 16, 16, 1, 64, "split", 0), ("f32", 128, 64, 4, 32, "seg", 2),
    ("bf16", 128, 64, 1, 64, "seg", 0), ("bf16", 128, 64, 1, 64, "seg", 1 << 20),
    ("bf16", 128, 64, 1, 64, "per_chunk", 0), ("bf16", 128, 64, 1, 64, "split", 0),
    ("bf16", 128, 64, 2, 32, "per_chunk", 0),
    ("bf16", 128, 64, 4, 64, "seg", 1 << 20), ("bf16", 128, 64, 4, 64, "seg", 2),
    ("bf16", 128, 64, 4, 64, "per_chunk", 0), ("bf16", 128, 64, 4, 128, "per_chunk", 0),
    ("bf16", 128, 64, 4, 128, "seg", 2),
]


@pytest.mark.parametrize("io,N,P,R,Q,mode,seg", GATE_CASES)
def test_gated_scan(io, N, P, R, Q, mode, seg):
    """Gated prefill on every kernel (several chunks and a ragged tail) against
    the oracle's y o SiLU(z); the final state and the carry are those of the
    ungated call, bit for bit (the gate acts on the output only)."""
    L = 3 * Q + Q // 2 + 3
    say(f"gated scan io={io} N={N} R={R} Q={Q} L={L} mode={mode} seg={seg}")
    inp = make_scan_inputs(2, L, 3, P, N, R, io=io, seed=71 + R + Q, device=DEV, chunk=Q)
    z = make_gate_input(inp.x, R + Q)
    y, fs, cB, cX = run_scan(inp, Q, mode=mode, seg=seg, z=z)
    check_slices(inp, y, fs, cB, cX, sample_slices(2, 3, 99, 6), TOL[io],
                 label=f"gated {io}/{R}/{Q}/{mode}", z=z)
    y0, fs0, cB0, cX0 = run_scan(inp, Q, mode=mode, seg=seg)
    assert torch.equal(fs, fs0) and torch.equal(cB, cB0) and torch.equal(cX, cX0)
    # the gate itself, against the ungated output of the same kernel
    ref = y0.double() * torch.nn.functional.silu(z.double())
    scale = ref.abs().max().item()
    assert (y.double() - ref).abs().max().item() <= (1e-6 if io == "f32" else 8e-3) * scale


def test_gated_workload1_siso():
    """Workload 1 (SISO bf16 prefill) gated, all 64 slices."""
    say("gated workload 1: all 64 slices")
    w = WORKLOADS[1]
    inp = workload_inputs(1, device=DEV)
    z = make_gate_input(inp.x, 1)
    y, fs, cB, cX = run_scan(inp, w["chunk"], z=z)
    check_slices(inp, y, fs, cB, cX, sample_slices(w["batch"], w["nheads"], 10**6, 1),
                 TOL["bf16"], label="gated w1", z=z)


@pytest.mark.parametrize("io,N,P,R", [("f32", 16, 16, 1), ("f32", 128, 64, 4),
                                      ("bf16", 128, 64, 1), ("bf16", 128, 64, 4),
                                      ("bf16", 64, 64, 4)])
def test_gated_decode_steps(io, N, P, R):
    """Gated decode steps: y_t o SiLU(z_t) against the oracle, state and
    carry advanced as by the ungated step."""
    say(f"gated decode io={io} N={N} R={R}")
    dt = torch.float32 if io == "f32" else torch.bfloat16
    inp = make_scan_inputs(3, 4, 5, P, N, R, io=io, seed=37, device=DEV)
    state = torch.randn(3, 5, N, P, device=DEV)
    cB = torch.randn(3, 5, R, N, device=DEV).to(dt)
    cX = torch.randn(3, 5, R, P, device=DEV).to(dt)
    state0, cB0, cX0 = state.clone(), cB.clone(), cX.clone()
    sl = [(b, h) for b in range(3) for h in range(5)]
    rs = oracle.slices_of_state(state, sl)
    rb, rx = oracle.slices_of_state(cB, sl), oracle.slices_of_state(cX, sl)
    A_s = np.array([float(inp.A[h]) for _, h in sl])
    D_s = np.array([float(inp.D[h]) for _, h in sl])
    for s in range(3):
        st = make_step_inputs(inp, s)
        z = make_gate_input(st.x, 100 + s)
        y = torch.full_like(st.x, float("nan"))
        m3.step(state, (cB, cX), st.x, st.Bm, st.Cm, st.dt, inp.A, st.lam, st.theta, inp.D, y=y, z=z)
        m3.step(state0, (cB0, cX0), st.x, st.Bm, st.Cm, st.dt, inp.A, st.lam, st.theta, inp.D)
        torch.cuda.synchronize()
        p = oracle.slices_of_step(st.x, st.Bm, st.Cm, st.dt, st.lam, st.theta, sl)
        ry, rs, rb, rx = oracle.step(rs, rb, rx, p["x"], p["B"], p["C"], p["dt"], A_s, p["lam"],
                                     p["theta"], D_s)
        ry = oracle.gate(ry, oracle.slices_of_state(z, sl))
        for k, (b, h) in enumerate(sl):
            assert oracle.rel_err(y[b, h].double().cpu().numpy(), ry[k]) <= TOL[io]
        assert torch.equal(state, state0) and torch.equal(cB, cB0) and torch.equal(cX, cX0)


# ---------------------------------------------------------------------------
# Maximum sizes: the single-pass kernels address a token's rows with a 24-bit
# stride multiply and a chunk's rows with 32-bit buffer offsets; the widest
# tokens they accept, and the first ones they hand to the three-kernel path
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("H,Q,L,mode", [
    (16383, 64, 70, "seg"),          # tokens of 2^24 - 1024 bytes: single pass, several chunks
    (16384, 64, 70, "seg"),          # 2^24 bytes: three-kernel path
    (16383, 128, 133, "seg"),        # a chunk's rows span 2^31 - 1.1 MB
    (16383, 128, 133, "per_chunk"),
])
def test_widest_tokens(H, Q, L, mode):
    """bf16, N=128, P=64, R=4: nheads * rank * dstate elements per token at and
    just past the single-pass kernels' 2^24-byte row stride (and a 128-token
    chunk whose rows reach within 1.1 MB of 2 GiB); three sampled heads plus
    the first and the last checked against the oracle."""
    say(f"widest tokens H={H} Q={Q} L={L} mode={mode}")
    inp = make_scan_inputs(1, L, H, 64, 128, 4, io="bf16", seed=91, device=DEV, chunk=Q)
    y, fs, cB, cX = run_scan(inp, Q, mode=mode)
    sl = [(0, 0), (0, 1), (0, H // 2), (0, H - 2), (0, H - 1)]
    check_slices(inp, y, fs, cB, cX, sl, TOL["bf16"], label=f"wide H={H} Q={Q} {mode}")
    del inp, y, fs, cB, cX
    torch.cuda.empty_cache()


# ---------------------------------------------------------------------------
# Per-head rotary frequencies (M3_THETA_PER_HEAD): theta given as omega [H, N/2],
# every angle dt * omega formed in the kernels
# ---------------------------------------------------------------------------

PH_CASES = [  # io, N, P, R, Q, mode, seg
    ("f32", 16, 16, 1, 64, "seg", 0), ("f32", 16, 16, 2, 32, "per_chunk", 0),
    ("f32", 128, 64, 4, 32, "split", 0), ("f32", 128, 64, 4, 32, "seg", 2),
    ("bf16", 128, 64, 1, 64, "seg", 0), ("bf16", 128, 64, 1, 64, "seg", 1 << 20),
    ("bf16", 128, 64, 1, 64, "split", 0), ("bf16", 128, 64, 4, 64, "seg", 1 << 20),
    ("bf16", 128, 64, 4, 64, "seg", 2), ("bf16", 128, 64, 4, 128, "per_chunk", 0),
    ("bf16", 128, 64, 2, 64, "per_chunk", 0),
]


@pytest.mark.parametrize("io,N,P,R,Q,mode,seg", PH_CASES)
def test_theta_per_head(io, N, P, R, Q, mode, seg):
    """Prefill with per-head frequencies on every kernel (several chunks and a
    ragged tail): against the oracle on the per-token angles theta = dt * omega
    that the input generator forms in fp32, and against the same kernel fed
    those angles."""
    L = 3 * Q + Q // 2 + 3
    say(f"theta per head io={io} N={N} R={R} Q={Q} L={L} mode={mode} seg={seg}")
    inp = make_scan_inputs(2, L, 3, P, N, R, io=io, seed=83 + R + Q, device=DEV, chunk=Q)
    per_tok = inp.theta
    inp.theta = inp.omega.contiguous()          # [H, N/2]
    y, fs, cB, cX = run_scan(inp, Q, mode=mode, seg=seg)
    inp.theta = per_tok
    check_slices(inp, y, fs, cB, cX, sample_slices(2, 3, 99, 8), TOL[io],
                 label=f"omega {io}/{R}/{Q}/{mode}")
    y0, fs0, cB0, cX0 = run_scan(inp, Q, mode=mode, seg=seg)
    for a, b0 in ((y, y0), (fs, fs0)):
        d = (a.double() - b0.double()).abs().max().item()
        assert d <= (1e-6 if io == "f32" else 1e-2) * b0.double().abs().max().item()
    assert torch.equal(cB, cB0) and torch.equal(cX, cX0)


@pytest.mark.parametrize("io,N,P,R", [("f32", 16, 16, 2), ("bf16", 128, 64, 4)])
def test_theta_per_head_decode(io, N, P, R):
    """Decode steps with per-head frequencies against the oracle on the
    per-step angles dt_t * omega."""
    say(f"theta per head decode io={io} N={N} R={R}")
    dt = torch.float32 if io == "f32" else torch.bfloat16
    inp = make_scan_inputs(3, 4, 5, P, N, R, io=io, seed=41, device=DEV)
    state = torch.randn(3, 5, N, P, device=DEV)
    cB = torch.randn(3, 5, R, N, device=DEV).to(dt)
    cX = torch.randn(3, 5, R, P, device=DEV).to(dt)
    sl = [(b, h) for b in range(3) for h in range(5)]
    rs = oracle.slices_of_state(state, sl)
    rb, rx = oracle.slices_of_state(cB, sl), oracle.slices_of_state(cX, sl)
    A_s = np.array([float(inp.A[h]) for _, h in sl])
    D_s = np.array([float(inp.D[h]) for _, h in sl])
    om = inp.omega.to(DEV).contiguous()
    for s in range(3):
        st = make_step_inputs(inp, s)
        y = torch.full_like(st.x, float("nan"))
        m3.step(state, (cB, cX), st.x, st.Bm, st.Cm, st.dt, inp.A, st.lam, om, inp.D, y=y)
        torch.cuda.synchronize()
        p = oracle.slices_of_step(st.x, st.Bm, st.Cm, st.dt, st.lam, st.theta, sl)
        ry, rs, rb, rx = oracle.step(rs, rb, rx, p["x"], p["B"], p["C"], p["dt"], A_s, p["lam"],
                                     p["theta"], D_s)
        for k, (b, h) in enumerate(sl):
            assert oracle.rel_err(y[b, h].double().cpu().numpy(), ry[k]) <= TOL[io]
            assert oracle.rel_err(state[b, h].cpu().numpy(), rs[k]) <= TOL[io]


# ---------------------------------------------------------------------------
# Varlen: sequences of different lengths packed along one token axis
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("io,N,P,R,Q,gated,per_head", [
    ("f32", 16, 16, 1, 64, False, False), ("bf16", 128, 64, 1, 64, False, False),
    ("bf16", 128, 64, 4, 64, True, False), ("bf16", 128, 64, 4, 128, False, True),
])
def test_varlen(io, N, P, R, Q, gated, per_head):
    """Packed sequences (lengths 70, 1, 0, 2Q + 9 and Q; the second with an
    initial state and carry) against the oracle per sequence, and against
    separate m3_scan_fwd calls on each sequence (the same launches: equal bit
    for bit)."""
    lens = [70, 1, 0, 2 * Q + 9, Q]
    cu = [0]
    for n in lens:
        cu.append(cu[-1] + n)
    T, H = cu[-1], 3
    say(f"varlen io={io} R={R} Q={Q} lens={lens} gated={gated} per_head={per_head}")
    inp = make_scan_inputs(1, T, H, P, N, R, io=io, seed=97 + R + Q, device=DEV, chunk=Q)
    flat = lambda t: t[0].contiguous()
    x, Bm, Cm, dt, lam, theta = (flat(inp.x), flat(inp.Bm), flat(inp.Cm), flat(inp.dt),
                                 flat(inp.lam), flat(inp.theta))
    th_in = inp.omega.contiguous() if per_head else theta
    z = make_gate_input(x, 3) if gated else None
    S = len(lens)
    iodt = x.dtype
    init = torch.randn(S, H, N, P, device=DEV)
    icB = torch.randn(S, H, R, N, device=DEV).to(iodt)
    icX = torch.randn(S, H, R, P, device=DEV).to(iodt)
    y, fs, (cB, cX) = m3.scan_fwd_varlen(x, Bm, Cm, dt, inp.A, lam, th_in, inp.D, Q, cu,
                                         init_state=init, init_carry=(icB, icX), z=z)
    torch.cuda.synchronize()
    for i in range(S):
        t0, t1 = cu[i], cu[i + 1]
        sl = [(0, h) for h in range(H)]
        if t1 > t0:
            ref = oracle.slices_of_scan(inp.x, inp.Bm, inp.Cm, inp.dt, inp.A, inp.lam, inp.theta,
                                        inp.D, sl, t0, t1)
        else:
            ref = dict(x=np.zeros((H, 0, R, P)), B=np.zeros((H, 0, R, N)), C=np.zeros((H, 0, R, N)),
                       dt=np.zeros((H, 0)), A=np.zeros((H, 0)), lam=np.zeros((H, 0)),
                       theta=np.zeros((H, 0, N // 2)), D=oracle._np(inp.D))
        ry, rs, rb, rx = oracle.scan(**ref, init_state=oracle._np(init[i]), init_B=oracle._np(icB[i]),
                                     init_X=oracle._np(icX[i]))
        for h in range(H):
            gy = y[t0:t1, h].double().cpu().numpy()
            ref_y = ry[h] if z is None else oracle.gate(ry[h], oracle._np(z[t0:t1, h]))
            if t1 > t0:
                assert oracle.rel_err(gy, ref_y) <= TOL[io], f"seq {i} head {h} y"
            assert oracle.rel_err(fs[i, h].cpu().numpy(), rs[h]) <= TOL[io], f"seq {i} head {h} state"
            assert np.array_equal(oracle._np(cB[i, h]), rb[h]) and np.array_equal(oracle._np(cX[i, h]), rx[h])
        # the same sequence on its own
        if t1 > t0:
            one = lambda t: t[None, t0:t1].contiguous()
            y1, fs1, (cB1, cX1) = m3.scan_fwd(one(x), one(Bm), one(Cm), one(dt), inp.A, one(lam),
                                              th_in if per_head else one(theta), inp.D, chunk=Q,
                                              init_state=init[i:i + 1].contiguous(),
                                              init_carry=(icB[i:i + 1].contiguous(), icX[i:i + 1].contiguous()),
                                              z=None if z is None else one(z))
            torch.cuda.synchronize()
            assert torch.equal(y1[0], y[t0:t1]) and torch.equal(fs1[0], fs[i])
            assert torch.equal(cB1[0], cB[i]) and torch.equal(cX1[0], cX[i])


@pytest.mark.parametrize("variant", ["plain", "per_token_A", "gated_per_head"])
def test_varlen_equal_length_runs(variant):
    """Runs of consecutive equal-length sequences (3 x 64, 2 x 10, 2 x 0, 33)
    with a workspace large enough to batch each run: every sequence against
    the oracle, from its own initial state; with per-token A [T, H] (the
    batched launch then strides A by the sequence length), and gated with
    per-head frequencies omega."""
    io, N, P, R, Q, H = "bf16", 128, 64, 4, 64, 3
    lens = [64, 64, 64, 10, 10, 0, 0, 33]
    cu = [0]
    for n in lens:
        cu.append(cu[-1] + n)
    T, S = cu[-1], len(lens)
    say(f"varlen runs lens={lens} variant={variant}")
    inp = make_scan_inputs(1, T, H, P, N, R, io=io, seed=131, device=DEV, chunk=Q)
    flat = lambda t: t[0].contiguous()
    init = torch.randn(S, H, N, P, device=DEV)
    A_in, A_ref = inp.A, None
    if variant == "per_token_A":
        A_in = (-torch.rand(T, H, device=DEV) * 4 - 0.1).contiguous()
        A_ref = A_in
    th_in = inp.omega.contiguous() if variant == "gated_per_head" else flat(inp.theta)
    z = make_gate_input(flat(inp.x), 5) if variant == "gated_per_head" else None
    st_t = 0 if A_ref is None else H
    ws = torch.zeros(m3.workspace_bytes(m3.M3Dims(S, 64, H, P, N, R, Q, 1, 0, 64 * st_t, st_t, 1, 0)),
                     dtype=torch.uint8, device=DEV)
    y, fs, (cB, cX) = m3.scan_fwd_varlen(flat(inp.x), flat(inp.Bm), flat(inp.Cm), flat(inp.dt),
                                         A_in, flat(inp.lam), th_in, inp.D, Q, cu,
                                         init_state=init, workspace=ws, z=z)
    torch.cuda.synchronize()
    for i in range(S):
        t0, t1 = cu[i], cu[i + 1]
        sl = [(0, h) for h in range(H)]
        if t1 == t0:
            assert torch.equal(fs[i], init[i]) and not cB[i].abs().any() and not cX[i].abs().any()
            continue
        ref = oracle.slices_of_scan(inp.x, inp.Bm, inp.Cm, inp.dt, inp.A, inp.lam, inp.theta,
                                    inp.D, sl, t0, t1)
        if A_ref is not None:
            ref["A"] = np.stack([A_ref[t0:t1, h].double().cpu().numpy() for h in range(H)])
        ry, rs, rb, rx = oracle.scan(**ref, init_state=oracle._np(init[i]))
        for h in range(H):
            ref_y = ry[h] if z is None else oracle.gate(ry[h], oracle._np(z[t0:t1, h]))
            assert oracle.rel_err(y[t0:t1, h].double().cpu().numpy(), ref_y) <= TOL[io], f"seq {i} y"
            assert oracle.rel_err(fs[i, h].cpu().numpy(), rs[h]) <= TOL[io], f"seq {i} state"
            assert np.array_equal(oracle._np(cB[i, h]), rb[h]) and np.array_equal(oracle._np(cX[i, h]), rx[h])


def varlen_oracle_check(inp, y, fs, cB, cX, cu, seqs, H, R, N, P, io, init=None, icB=None, icX=None,
                        z=None, A_tok=None, label=""):
    """Every listed sequence of a packed batch against the oracle from its own
    initial state and carry."""
    for i in seqs:
        t0, t1 = cu[i], cu[i + 1]
        sl = [(0, h) for h in range(H)]
        ref = oracle.slices_of_scan(inp.x, inp.Bm, inp.Cm, inp.dt, inp.A, inp.lam, inp.theta,
                                    inp.D, sl, t0, t1)
        if A_tok is not None:
            ref["A"] = np.stack([A_tok[t0:t1, h].double().cpu().numpy() for h in range(H)])
        kw = {}
        if init is not None:
            kw = dict(init_state=oracle._np(init[i]), init_B=oracle._np(icB[i]), init_X=oracle._np(icX[i]))
        ry, rs, rb, rx = oracle.scan(**ref, **kw)
        for h in range(H):
            ref_y = ry[h] if z is None else oracle.gate(ry[h], oracle._np(z[t0:t1, h]))
            e = oracle.rel_err(y[t0:t1, h].double().cpu().numpy(), ref_y)
            assert e <= TOL[io], f"{label} seq {i} head {h} y rel err {e:.3g}"
            e = oracle.rel_err(fs[i, h].cpu().numpy(), rs[h])
            assert e <= TOL[io], f"{label} seq {i} head {h} state rel err {e:.3g}"
            assert np.array_equal(oracle._np(cB[i, h]), rb[h]) and np.array_equal(oracle._np(cX[i, h]), rx[h])


@pytest.mark.parametrize("R,Q,gated,per_head,per_token_A", [
    (1, 64, False, False, False), (4, 128, True, False, False), (2, 32, False, True, False),
    (4, 64, False, False, True), (1, 128, True, True, False),
])
def test_varlen_one_launch(R, Q, gated, per_head, per_token_A):
    """29 packed sequences of ragged lengths (1 .. 5Q, some whole chunks) in
    one launch of the per-chunk kernel: every sequence against the oracle
    from its own initial state and carry; the same bits as each sequence
    scanned alone with the per-chunk kernel; a second call gives the same
    bits."""
    io, N, P, H = "bf16", 128, 64, 3
    rng = np.random.default_rng(200 + R + Q)
    lens = [int(v) for v in rng.integers(1, 5 * Q + 1, 29)]
    lens[3], lens[7], lens[11] = 1, Q, 2 * Q
    cu = [0]
    for n in lens:
        cu.append(cu[-1] + n)
    T, S = cu[-1], len(lens)
    say(f"varlen one launch R={R} Q={Q} T={T} gated={gated} per_head={per_head} A per token={per_token_A}")
    inp = make_scan_inputs(1, T, H, P, N, R, io=io, seed=211 + R + Q, device=DEV, chunk=Q)
    flat = lambda t: t[0].contiguous()
    x, Bm, Cm, dt, lam, theta = (flat(inp.x), flat(inp.Bm), flat(inp.Cm), flat(inp.dt),
                                 flat(inp.lam), flat(inp.theta))
    th_in = inp.omega.contiguous() if per_head else theta
    z = make_gate_input(x, 4) if gated else None
    A_in = (-torch.rand(T, H, device=DEV) * 4 - 0.1).contiguous() if per_token_A else inp.A
    init = torch.randn(S, H, N, P, device=DEV)
    icB = torch.randn(S, H, R, N, device=DEV).to(x.dtype)
    icX = torch.randn(S, H, R, P, device=DEV).to(x.dtype)
    d = m3.varlen_dims(x, Bm, A_in, Q, cu, theta=th_in)
    need = m3.varlen_workspace_bytes(d, cu)
    assert need > 0, "the one-launch scan applies"
    ws = torch.zeros(need, dtype=torch.uint8, device=DEV)
    args = (x, Bm, Cm, dt, A_in, lam, th_in, inp.D, Q, cu)
    kw = dict(init_state=init, init_carry=(icB, icX), z=z, workspace=ws, check=True)
    y, fs, (cB, cX) = m3.scan_fwd_varlen(*args, **kw)
    torch.cuda.synchronize()
    varlen_oracle_check(inp, y, fs, cB, cX, cu, range(S), H, R, N, P, io, init, icB, icX, z,
                        A_in if per_token_A else None, label="one launch")
    # each sequence alone, one chunk per workgroup: the same launches' arithmetic
    for i in sorted({0, 3, 7, 11, S - 1, int(rng.integers(0, S))}):
        t0, t1 = cu[i], cu[i + 1]
        one = lambda t: t[None, t0:t1].contiguous()
        A1 = A_in[t0:t1].contiguous()[None] if per_token_A else inp.A
        y1, fs1, (cB1, cX1) = m3.scan_fwd(one(x), one(Bm), one(Cm), one(dt), A1, one(lam),
                                          th_in if per_head else one(theta), inp.D, chunk=Q,
                                          init_state=init[i:i + 1].contiguous(),
                                          init_carry=(icB[i:i + 1].contiguous(), icX[i:i + 1].contiguous()),
                                          z=None if z is None else one(z), per_chunk=True)
        torch.cuda.synchronize()
        assert torch.equal(y1[0], y[t0:t1]) and torch.equal(fs1[0], fs[i]), f"seq {i}: not bit-identical"
        assert torch.equal(cB1[0], cB[i]) and torch.equal(cX1[0], cX[i])
    y2, fs2, _ = m3.scan_fwd_varlen(*args, **kw)
    torch.cuda.synchronize()
    assert torch.equal(y2, y) and torch.equal(fs2, fs), "second call differs"


def test_varlen_many_short_sequences():
    """600 packed sequences of 1 .. 40 tokens (SISO, chunk 64): one launch
    against the oracle on a sample of sequences (the first, the last and
    30 more), and against the sequence-by-sequence launches the same call
    makes with a workspace too small for one launch."""
    io, N, P, R, Q, H = "bf16", 128, 64, 1, 64, 4
    rng = np.random.default_rng(300)
    lens = [int(v) for v in rng.integers(1, 41, 600)]
    cu = [0]
    for n in lens:
        cu.append(cu[-1] + n)
    T, S = cu[-1], len(lens)
    say(f"varlen many short sequences S={S} T={T}")
    inp = make_scan_inputs(1, T, H, P, N, R, io=io, seed=301, device=DEV, chunk=Q)
    flat = lambda t: t[0].contiguous()
    args = (flat(inp.x), flat(inp.Bm), flat(inp.Cm), flat(inp.dt), inp.A, flat(inp.lam),
            flat(inp.theta), inp.D, Q, cu)
    d = m3.varlen_dims(args[0], args[1], inp.A, Q, cu)
    need = m3.varlen_workspace_bytes(d, cu)
    assert need > 0
    ws = torch.zeros(need, dtype=torch.uint8, device=DEV)
    y, fs, (cB, cX) = m3.scan_fwd_varlen(*args, workspace=ws, check=True)
    torch.cuda.synchronize()
    seqs = sorted({0, S - 1} | {int(v) for v in rng.integers(0, S, 30)})
    varlen_oracle_check(inp, y, fs, cB, cX, cu, seqs, H, R, N, P, io, label="many short")
    small = torch.zeros(m3.workspace_bytes(m3.M3Dims(1, 40, H, P, N, R, Q, 1, 0, 0, 0, 1, 0)),
                        dtype=torch.uint8, device=DEV)
    y2, fs2, (cB2, cX2) = m3.scan_fwd_varlen(*args, workspace=small, check=True)
    torch.cuda.synchronize()
    varlen_oracle_check(inp, y2, fs2, cB2, cX2, cu, seqs, H, R, N, P, io, label="per sequence")
    # timing of the two (reported, not asserted)
    for name, w in (("one launch", ws), ("per sequence", small)):
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(3):
            m3.scan_fwd_varlen(*args, workspace=w)
        e1.record()
        torch.cuda.synchronize()
        say(f"varlen {S} sequences, {name}: {e0.elapsed_time(e1) / 3:.3f} ms")


@pytest.mark.parametrize("mode,seg,R,Q", [("per_chunk", 0, 1, 64), ("per_chunk", 0, 4, 128),
                                          ("seg", 2, 4, 64), ("seg", 4, 1, 64)])
def test_determinism_many_items(mode, seg, R, Q):
    """Thousands of look-back items, three runs with other work in between:
    bitwise-identical outputs.  The entering state of a chunk (segment) is the
    forward fold from the sequence start whichever predecessors happened to
    be done when it looked back."""
    say(f"determinism many items mode={mode} seg={seg} R={R} Q={Q}")
    L = 2048 if R == 1 else 1024
    inp = make_scan_inputs(4, L, 16, 64, 128, R, io="bf16", seed=9 + R, device=DEV, chunk=Q)
    runs = []
    for k in range(3):
        runs.append(run_scan(inp, Q, mode=mode, seg=seg, nan_fill=False))
        if k == 1:   # shift the timing of the next run
            torch.randn(1 << 24, device=DEV).sum().item()
    for other in runs[1:]:
        for u, v in zip(runs[0], other):
            assert torch.equal(u, v)


# ---------------------------------------------------------------------------
# Look-back timeouts: reported through m3_scan_check, results NaN
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("mode,seg", [("per_chunk", 0), ("seg", 2)])
def test_lookback_timeout_reported(mode, seg):
    """With a wait limit of one poll, workgroups that find their predecessor
    unpublished give up at once (every kernel still exits normally): the
    scan's check count is non-zero and the invalid results are NaN, not
    plausible numbers; with the default limit restored the same scan is
    clean and matches the oracle.  Two slices of 256 chunks: every item of
    a slice is resident at once, so most find their predecessor still
    working (with many short slices whether any item waits at all depends
    on timing)."""
    R, Q = 1, 64
    say(f"look-back timeout mode={mode} seg={seg}")
    inp = make_scan_inputs(1, 16384, 2, 64, 128, R, io="bf16", seed=17, device=DEV, chunk=Q)
    kw = dict(per_chunk=mode == "per_chunk", seg=seg)
    d = m3.scan_dims(inp.x, inp.Bm, Q, inp.A, **kw)
    ws = torch.zeros(m3.workspace_bytes(d), dtype=torch.uint8, device=DEV)
    args = (inp.x, inp.Bm, inp.Cm, inp.dt, inp.A, inp.lam, inp.theta, inp.D)
    try:
        m3.set_wait_limit(1)
        y, fs, _ = m3.scan_fwd(*args, chunk=Q, workspace=ws, **kw)
        n = m3.scan_check(d, ws)
        with pytest.raises(m3.LookBackTimeout):
            m3.scan_fwd(*args, chunk=Q, workspace=ws, check=True, **kw)
    finally:
        m3.set_wait_limit(0)
    say(f"timeouts with a one-poll limit: {n}")
    assert n > 0
    assert torch.isnan(fs).any() and torch.isnan(y.float()).any()
    # a slice with a NaN final state has NaN outputs from some chunk on
    bad = torch.isnan(fs).flatten(2).any(-1).nonzero()
    b, h = (int(v) for v in bad[0])
    assert torch.isnan(y[b, -1, h].float()).all()
    y2, fs2, (cB2, cX2) = m3.scan_fwd(*args, chunk=Q, workspace=ws, check=True, **kw)
    assert m3.scan_check(d, ws) == 0
    check_slices(inp, y2, fs2, cB2, cX2, sample_slices(1, 2, 6, 12), TOL["bf16"], label="after timeout")


def ctl_words(ws):
    """The workspace's control block as int32 words (copied to the host)."""
    return ws[:m3.CTL_BYTES].view(torch.int32).cpu().numpy()


def test_workspace_shared_across_calls():
    """One zero-filled workspace serves scans of different kernels and shapes
    and a backward call in turn.  Each single-pass call's last workgroup
    resets the control block for the next call (no reset launch): after
    every call the work-item and timeout counters read zero and the call
    counter has advanced once per single-pass call; every result matches the
    oracle, and repeating the first scan later gives the same bits."""
    cases = [(1, 64, "per_chunk", 0, 700), (1, 64, "seg", 2, 700), (1, 64, "split", 0, 300),
             (4, 32, "per_chunk", 0, 333), (2, 64, "seg", 3, 900)]
    B_, H = 2, 4
    inps = [make_scan_inputs(B_, L, H, 64, 128, R, io="bf16", seed=2100 + k, device=DEV, chunk=Q)
            for k, (R, Q, mode, seg, L) in enumerate(cases)]
    kws = [dict(split=mode == "split", per_chunk=mode == "per_chunk", seg=seg)
           for (R, Q, mode, seg, L) in cases]
    need = [m3.workspace_bytes(m3.scan_dims(i.x, i.Bm, c[1], i.A, **kw))
            for i, c, kw in zip(inps, cases, kws)]
    binp = make_scan_inputs(1, 200, 3, 64, 128, 1, io="bf16", seed=2199, device=DEV, chunk=64)
    bd = m3.scan_dims(binp.x, binp.Bm, 64, binp.A)
    need.append(int(m3.lib().m3_scan_bwd_workspace_bytes(__import__("ctypes").byref(bd))))
    ws = torch.zeros(max(need), dtype=torch.uint8, device=DEV)
    groups = [32 * (y + 1) for y in range(8)]
    epoch = 0
    first = None
    for rep in range(2):
        for k, ((R, Q, mode, seg, L), inp, kw) in enumerate(zip(cases, inps, kws)):
            if rep == 1 and k > 0:
                break
            say(f"shared workspace: call R={R} Q={Q} mode={mode} seg={seg} L={L}")
            y, fs, (cB, cX) = m3.scan_fwd(inp.x, inp.Bm, inp.Cm, inp.dt, inp.A, inp.lam, inp.theta,
                                          inp.D, chunk=Q, workspace=ws, check=True, **kw)
            torch.cuda.synchronize()
            w = ctl_words(ws)
            epoch += 0 if mode == "split" else 1
            # both timeout words zero; every group's ticket counter at ticket 0
            # with the flags-cleared bit off and the epoch (the count of
            # single-pass calls) in its high word; the ready word at the last
            # call's epoch + 1
            assert w[1] == 0 and w[3] == 0, w[:8]
            assert all(w[g] == 0 and w[g + 1] == epoch for g in groups), \
                [(w[g], w[g + 1]) for g in groups]
            assert w[5] == epoch, (w[5], epoch)
            if rep == 0:
                check_slices(inp, y, fs, cB, cX, [(b, h) for b in range(B_) for h in range(H)],
                             TOL["bf16"], label=f"shared workspace {mode} R={R}")
                if k == 0:
                    first = (y.clone(), fs.clone())
            else:
                assert torch.equal(y, first[0]) and torch.equal(fs, first[1])
        if rep == 0:   # a backward call on the same workspace leaves the block alone
            say("shared workspace: backward call")
            g = torch.Generator(DEV).manual_seed(3)
            dy = torch.randn(binp.x.shape, device=DEV, generator=g).to(binp.x.dtype)
            before = ctl_words(ws)
            m3.scan_bwd(binp.x, binp.Bm, binp.Cm, binp.dt, binp.A, binp.lam, binp.theta, binp.D,
                        dy, 64, workspace=ws)
            torch.cuda.synchronize()
            assert np.array_equal(ctl_words(ws), before)
