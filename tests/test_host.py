"""CPU tests of the host side: the C-ABI library loads and exports every
symbol of include/m3.h, every argument error is caught on the host before a
launch, and the benchmark's accounting matches the paper's printed forms."""
import ctypes
import os
import re

import pytest

from paper_2603_15569_amd import m3, roofline

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def golden():
    vals = {}
    with open(os.path.join(ROOT, "tests", "golden", "paper_formulas.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                k, v = line.split()[:2]
                vals[k] = float(v)
    return vals


@pytest.fixture(scope="module")
def L():
    return m3.lib()


def test_exports_match_header(L):
    hdr = open(os.path.join(ROOT, "include", "m3.h")).read()
    declared = set(re.findall(r"^\S.*?\b(m3_\w+)\s*\(", hdr, flags=re.M))
    assert declared == set(m3.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name


def test_status_strings(L):
    for s in range(8):
        assert L.m3_status_string(s)
    assert L.m3_last_hip_error() == 0


FAKE = 0x100000  # 16-byte aligned fake device address; never dereferenced


def dims(**kw):
    d = dict(batch=1, seqlen=256, nheads=2, headdim=16, dstate=16, rank=1, chunk=64,
             io=m3.M3_F32, flags=0, a_stride_b=0, a_stride_t=0, a_stride_h=1, seg_chunks=0)
    d.update(kw)
    return m3.M3Dims(**d)


def scan_call(L, d, over=None, ws_bytes=None):
    ptrs = [FAKE] * 15
    for k, v in (over or {}).items():
        ptrs[k] = v
    # init_state / init carry default to NULL
    for k in (8, 9, 10):
        if not over or k not in over:
            ptrs[k] = None
    need = L.m3_scan_workspace_bytes(ctypes.byref(d)) if d is not None else 0
    ws = FAKE
    wsb = need if ws_bytes is None else ws_bytes
    return L.m3_scan_fwd(ctypes.byref(d) if d is not None else None, *ptrs, ws, wsb, None)


def test_scan_host_validation(L):
    assert scan_call(L, None) == m3.M3_ERR_NULL
    assert scan_call(L, dims(io=7)) == m3.M3_ERR_DTYPE
    assert scan_call(L, dims(dstate=15)) == m3.M3_ERR_SHAPE
    assert scan_call(L, dims(rank=0)) == m3.M3_ERR_SHAPE
    assert scan_call(L, dims(batch=0)) == m3.M3_ERR_SHAPE
    assert scan_call(L, dims(seqlen=-1)) == m3.M3_ERR_SHAPE
    assert scan_call(L, dims(chunk=0)) == m3.M3_ERR_SHAPE
    assert scan_call(L, dims(flags=8)) == m3.M3_ERR_SHAPE
    assert scan_call(L, dims(seg_chunks=-1)) == m3.M3_ERR_SHAPE
    assert scan_call(L, dims(dstate=64, headdim=64)) == m3.M3_ERR_UNSUPPORTED
    assert scan_call(L, dims(chunk=48)) == m3.M3_ERR_UNSUPPORTED
    assert scan_call(L, dims(io=m3.M3_BF16)) == m3.M3_ERR_UNSUPPORTED
    assert scan_call(L, dims(), {0: None}) == m3.M3_ERR_NULL
    assert scan_call(L, dims(), {14: None}) == m3.M3_ERR_NULL
    assert scan_call(L, dims(), {11: None}) == m3.M3_ERR_NULL       # y with seqlen > 0
    assert scan_call(L, dims(), {9: FAKE}) == m3.M3_ERR_NULL        # one carry half only
    assert scan_call(L, dims(), {0: FAKE + 4}) == m3.M3_ERR_ALIGN
    assert scan_call(L, dims(), {3: FAKE + 2}) == m3.M3_ERR_ALIGN
    assert scan_call(L, dims(), ws_bytes=0) == m3.M3_ERR_WORKSPACE
    need = L.m3_scan_workspace_bytes(ctypes.byref(dims()))
    assert scan_call(L, dims(), ws_bytes=need - 1) == m3.M3_ERR_WORKSPACE
    assert L.m3_last_hip_error() == 0


def test_workspace_bytes(L):
    assert L.m3_scan_workspace_bytes(None) == 0
    assert L.m3_scan_workspace_bytes(ctypes.byref(dims(dstate=64, headdim=64))) == 0
    d = dims(io=m3.M3_BF16, dstate=128, headdim=64, rank=4, chunk=64, seqlen=4096, batch=8,
             nheads=32)
    nb = L.m3_scan_workspace_bytes(ctypes.byref(d))
    per = 8 * 32 * 64
    # single-pass: flags, chunk totals, aggregate and inclusive fp32 states
    assert nb >= per * (4 + 65 * 4 + 2 * 128 * 64 * 4)
    assert nb % 256 == 0
    d.flags = m3.M3_SCAN_SPLIT
    nb = L.m3_scan_workspace_bytes(ctypes.byref(d))
    # three-kernel: the control block it leaves alone, per-chunk fp32
    # contributions, bf16 entering states, totals
    assert nb >= m3.CTL_BYTES + per * 128 * 64 * (4 + 2) + per * 65 * 4
    assert nb % 256 == 0


def test_control_block_size_matches_header():
    hdr = open(os.path.join(ROOT, "include", "m3.h")).read()
    m = re.search(r"#define M3_CTL_BYTES \(\(size_t\)(\d+)\)", hdr)
    assert m and int(m.group(1)) == m3.CTL_BYTES and m3.CTL_BYTES % 256 == 0


def test_step_host_validation(L):
    def call(d, over=None):
        ptrs = [FAKE] * 12
        for k, v in (over or {}).items():
            ptrs[k] = v
        return L.m3_step(ctypes.byref(d) if d is not None else None, *ptrs, None)
    assert call(None) == m3.M3_ERR_NULL
    assert call(dims(io=9)) == m3.M3_ERR_DTYPE
    assert call(dims(dstate=32, headdim=16)) == m3.M3_ERR_UNSUPPORTED
    assert call(dims(), {0: None}) == m3.M3_ERR_NULL
    assert call(dims(), {11: None}) == m3.M3_ERR_NULL
    assert call(dims(), {0: FAKE + 8}) == m3.M3_ERR_ALIGN
    assert call(dims(), {6: FAKE + 1}) == m3.M3_ERR_ALIGN


def test_accounting_against_paper():
    g = golden()
    # Tab. arith_intensity (a): about 2.5 for large N, P
    assert abs(roofline.decode_ai_siso(4096, 4096) - g["siso_decode_ai_approx"]) < 0.01
    assert 2.3 < roofline.decode_ai_siso(128, 64) < g["siso_decode_ai_approx"]
    # MIMO intensity grows linearly with R (Tab. arith_intensity (b))
    a1, a4 = roofline.decode_ai_mimo(128, 64, 1), roofline.decode_ai_mimo(128, 64, 4)
    assert 3.0 < a4 / a1 < 3.3
    assert abs(roofline.decode_ai_mimo(128, 64, 1) - roofline.decode_ai_siso(128, 64)) < 0.2
    # Sec. 3.3: C = P = N gives 8 T N^2 (ignoring the 2 (T/C) N P term)
    T, N = 4096, 64
    f = roofline.chunked_flops(T, N, N, 1, N)
    assert abs(f - g["chunked_siso_total_coeff"] * T * N * N) == 2 * T * N
    # Sec. 3.3: C R = N = P gives 8 T R N^2
    R = 4
    f = roofline.chunked_flops(T, N, N, R, N // R)
    assert abs(f - g["chunked_mimo_total_coeff"] * T * R * N * N) == 2 * (T * R // N) * N * N
    # intra-chunk FLOPs grow R^2, inter-chunk projections R times
    intra = lambda R: 2 * (T / 64) * (64 * R) ** 2 * (128 + 64)
    assert intra(4) / intra(1) == 4 ** g["mimo_intra_growth_power"]


def test_prefill_bytes_workloads():
    # SISO bf16 prefill (B=4, L=2048, H=16, N=128, P=64): 1032 B per token-head
    per = roofline.prefill_bytes(1, 1, 1, 128, 64, 1, 2) - (128 * 64 * 4 + (128 + 64) * 2)
    assert per == 1032
    # MIMO R=4: 3336 B per token-head
    per4 = roofline.prefill_bytes(1, 1, 1, 128, 64, 4, 2) - (128 * 64 * 4 + 4 * (128 + 64) * 2)
    assert per4 == 3336
    assert roofline.decode_bytes_per_slice(128, 64, 4, 2) == 71944


def test_gated_host_validation(L):
    """The gated entry points: z is required (a token array like x, 16-byte
    aligned); every other check is the ungated call's."""
    def scan(d, over=None):
        ptrs = [FAKE] * 16       # x B C dt A lam theta D z init icB icX y fs cB cX
        for k in (9, 10, 11):
            ptrs[k] = None
        for k, v in (over or {}).items():
            ptrs[k] = v
        wsb = L.m3_scan_workspace_bytes(ctypes.byref(d))
        return L.m3_scan_fwd_gated(ctypes.byref(d), *ptrs, FAKE, wsb, None)
    assert scan(dims(), {8: None}) == m3.M3_ERR_NULL
    assert scan(dims(), {8: FAKE + 2}) == m3.M3_ERR_ALIGN
    assert scan(dims(), {0: None}) == m3.M3_ERR_NULL
    assert scan(dims(chunk=48)) == m3.M3_ERR_UNSUPPORTED
    assert scan(dims(), {10: FAKE}) == m3.M3_ERR_NULL              # one carry half only

    def step(d, over=None):
        ptrs = [FAKE] * 13       # state cB cX x B C dt A lam theta D z y
        for k, v in (over or {}).items():
            ptrs[k] = v
        return L.m3_step_gated(ctypes.byref(d), *ptrs, None)
    assert step(dims(), {11: None}) == m3.M3_ERR_NULL
    assert step(dims(), {11: FAKE + 4}) == m3.M3_ERR_ALIGN
    assert step(dims(), {12: None}) == m3.M3_ERR_NULL
    assert step(dims(io=5)) == m3.M3_ERR_DTYPE
    assert L.m3_last_hip_error() == 0


def test_varlen_host_validation(L):
    """m3_scan_fwd_varlen: the offsets are checked on the host, and every
    sequence's arguments before the first launch."""
    def call(d, cu, over=None):
        ptrs = [FAKE] * 16       # x B C dt A lam theta D z init icB icX y fs cB cX
        for k in (8, 9, 10, 11):
            ptrs[k] = None
        for k, v in (over or {}).items():
            ptrs[k] = v
        arr = None if cu is None else (ctypes.c_int64 * len(cu))(*cu)
        return L.m3_scan_fwd_varlen(ctypes.byref(d), arr, *ptrs, FAKE, 1 << 30, None)
    d = dims(batch=3, seqlen=100)
    assert call(d, None) == m3.M3_ERR_NULL
    assert call(d, [1, 10, 50, 100]) == m3.M3_ERR_SHAPE           # must start at 0
    assert call(d, [0, 60, 50, 100]) == m3.M3_ERR_SHAPE           # decreasing
    assert call(d, [0, 10, 50, 99]) == m3.M3_ERR_SHAPE            # must end at seqlen
    assert call(dims(batch=3, seqlen=100, a_stride_b=5), [0, 10, 50, 100]) == m3.M3_ERR_SHAPE
    # the third sequence's misaligned token offset (fp32, P = 16: 64 B a token)
    # is fine; a misaligned base is caught before any launch
    assert call(d, [0, 10, 50, 100], {0: FAKE + 4}) == m3.M3_ERR_ALIGN
    assert call(d, [0, 10, 50, 100], {12: None}) == m3.M3_ERR_NULL   # y
    assert call(dims(batch=3, seqlen=100, chunk=48), [0, 10, 50, 100]) == m3.M3_ERR_UNSUPPORTED
    assert L.m3_last_hip_error() == 0


def test_varlen_one_launch_host(L):
    """m3_scan_varlen_workspace_bytes: the one-launch workspace (control block,
    a flag, the totals and two state maps per (sequence, head, chunk) slot,
    the tables) where the per-chunk kernel serves the shape and every
    sequence is non-empty, else 0; m3_scan_varlen_check's argument errors on
    the host."""
    bf = dict(io=m3.M3_BF16, headdim=64, dstate=128, rank=1, chunk=64, nheads=4)

    def nb(d, cu):
        return L.m3_scan_varlen_workspace_bytes(ctypes.byref(d), (ctypes.c_int64 * len(cu))(*cu))
    cu = [0, 100, 101, 357]
    d = dims(batch=3, seqlen=357, **bf)
    n = nb(d, cu)
    slots = 4 * (2 + 1 + 4)
    assert n >= m3.CTL_BYTES + slots * (4 + 65 * 4 + 2 * 128 * 64 * 4) and n % 256 == 0
    assert nb(dims(batch=3, seqlen=357, **dict(bf, rank=4, chunk=128)), cu) > 0
    assert nb(d, [0, 100, 100, 357]) == 0                                   # an empty sequence
    assert nb(d, [0, 100, 50, 357]) == 0                                    # bad offsets
    assert nb(dims(batch=3, seqlen=357, flags=m3.M3_SCAN_SPLIT, **bf), cu) == 0
    assert nb(dims(batch=3, seqlen=357, seg_chunks=2, **bf), cu) == 0
    assert nb(dims(batch=3, seqlen=357, **dict(bf, dstate=64)), cu) == 0    # three-kernel shape
    assert nb(dims(batch=3, seqlen=357), cu) == 0                          # fp32 16 x 16
    t = ctypes.c_uint32(7)
    arr = (ctypes.c_int64 * 4)(*cu)
    chk = L.m3_scan_varlen_check
    assert chk(ctypes.byref(d), None, FAKE, n, ctypes.byref(t), None) == m3.M3_ERR_NULL
    assert chk(ctypes.byref(d), arr, FAKE, n, None, None) == m3.M3_ERR_NULL
    bad = (ctypes.c_int64 * 4)(0, 100, 50, 357)
    assert chk(ctypes.byref(d), bad, FAKE, n, ctypes.byref(t), None) == m3.M3_ERR_SHAPE
    assert chk(ctypes.byref(d), arr, FAKE + 4, n, ctypes.byref(t), None) == m3.M3_ERR_ALIGN
    # too small for the one launch: the last sequence's launch is the one checked
    assert chk(ctypes.byref(d), arr, None, 0, ctypes.byref(t), None) == m3.M3_ERR_WORKSPACE
    assert L.m3_last_hip_error() == 0


def test_scan_check_host_validation(L):
    """m3_scan_check: argument errors on the host; the three-kernel path and
    the empty sequence report zero waits without touching the device."""
    n = ctypes.c_uint32(123)
    d = dims(io=m3.M3_BF16, headdim=64, dstate=128, rank=4, chunk=64, seqlen=300)
    need = L.m3_scan_workspace_bytes(ctypes.byref(d))
    assert need > 0
    assert L.m3_scan_check(None, FAKE, need, ctypes.byref(n), None) == m3.M3_ERR_NULL
    assert L.m3_scan_check(ctypes.byref(d), FAKE, need, None, None) == m3.M3_ERR_NULL
    assert L.m3_scan_check(ctypes.byref(dims(dstate=15)), FAKE, need, ctypes.byref(n), None) == m3.M3_ERR_SHAPE
    assert L.m3_scan_check(ctypes.byref(d), None, need, ctypes.byref(n), None) == m3.M3_ERR_WORKSPACE
    assert L.m3_scan_check(ctypes.byref(d), FAKE, need - 1, ctypes.byref(n), None) == m3.M3_ERR_WORKSPACE
    assert L.m3_scan_check(ctypes.byref(d), FAKE + 4, need, ctypes.byref(n), None) == m3.M3_ERR_ALIGN
    assert n.value == 123   # errors leave the output untouched
    ds = dims(io=m3.M3_BF16, headdim=64, dstate=128, rank=4, chunk=64, seqlen=300, flags=m3.M3_SCAN_SPLIT)
    assert L.m3_scan_check(ctypes.byref(ds), None, 0, ctypes.byref(n), None) == m3.M3_OK
    assert n.value == 0
    n.value = 5
    d0 = dims(io=m3.M3_BF16, headdim=64, dstate=128, rank=4, chunk=64, seqlen=0)
    assert L.m3_scan_check(ctypes.byref(d0), None, 0, ctypes.byref(n), None) == m3.M3_OK
    assert n.value == 0
    L.m3_set_wait_limit(0)   # restores the default; no device access


def test_noalloc_host_validation(L):
    """m3_scan_fwd_noalloc: the argument checks of m3_scan_fwd, and a scan
    whose workspace would exceed the fixed scratch is refused before any
    device call."""
    ptrs = [FAKE] * 15
    for k in (8, 9, 10):
        ptrs[k] = None
    assert L.m3_scan_fwd_noalloc(None, *ptrs, None) == m3.M3_ERR_NULL
    assert L.m3_scan_fwd_noalloc(ctypes.byref(dims(dstate=15)), *ptrs, None) == m3.M3_ERR_SHAPE
    bad = list(ptrs)
    bad[0] = FAKE + 2
    assert L.m3_scan_fwd_noalloc(ctypes.byref(dims()), *bad, None) == m3.M3_ERR_ALIGN
    big = dims(io=m3.M3_BF16, headdim=64, dstate=128, rank=1, chunk=64, batch=8, seqlen=4096, nheads=32)
    assert L.m3_scan_workspace_bytes(ctypes.byref(big)) > m3.SCRATCH_BYTES
    assert L.m3_scan_fwd_noalloc(ctypes.byref(big), *ptrs, None) == m3.M3_ERR_WORKSPACE


def test_prologue_host_validation(L):
    """m3_scan_fwd_pro / m3_step_pro: the prologue is checked on the host
    before any launch (eps > 0 with the norm, gains only with the norm, w_z
    only with z, aligned tables) and only the built shapes are accepted."""
    bf = dict(io=m3.M3_BF16, headdim=64, dstate=128, rank=4, chunk=64, seqlen=300)

    def pro(**kw):
        p = dict(bc_norm=1, eps=1e-6, norm_B=None, norm_C=None, bias_B=None, bias_C=None,
                 w_x=None, w_z=None)
        p.update(kw)
        return m3.M3Prologue(**p)

    def scan(d, p, over=None):
        ptrs = [FAKE] * 16       # x B C dt A lam theta D z init icB icX y fs cB cX
        for k in (8, 9, 10, 11):
            ptrs[k] = None
        for k, v in (over or {}).items():
            ptrs[k] = v
        wsb = L.m3_scan_workspace_bytes(ctypes.byref(d))
        return L.m3_scan_fwd_pro(ctypes.byref(d), None if p is None else ctypes.byref(p), *ptrs,
                                 FAKE, wsb, None)
    assert scan(dims(**bf), None) == m3.M3_ERR_NULL
    assert scan(dims(**bf), pro(eps=0.0)) == m3.M3_ERR_SHAPE
    assert scan(dims(**bf), pro(eps=float("nan"))) == m3.M3_ERR_SHAPE
    assert scan(dims(**bf), pro(bc_norm=0, norm_B=FAKE)) == m3.M3_ERR_SHAPE
    assert scan(dims(**bf), pro(w_z=FAKE)) == m3.M3_ERR_NULL          # no z
    assert scan(dims(**bf), pro(bias_C=FAKE + 4)) == m3.M3_ERR_ALIGN
    assert scan(dims(**bf), pro(w_x=FAKE + 8)) == m3.M3_ERR_ALIGN
    assert scan(dims(), pro()) == m3.M3_ERR_UNSUPPORTED                # fp32: not built
    assert scan(dims(**dict(bf, flags=m3.M3_SCAN_SPLIT)), pro()) == m3.M3_ERR_UNSUPPORTED
    assert scan(dims(**dict(bf, chunk=48)), pro()) == m3.M3_ERR_UNSUPPORTED
    assert scan(dims(**bf), pro(), {0: None}) == m3.M3_ERR_NULL
    # output norm: a known kind, eps > 0, a power-of-two group in [8, headdim],
    # a gain only with the norm, an aligned gain
    on = dict(out_norm=m3.M3_OUT_NORM_PRE_GATE, out_group=16, out_eps=1e-6)
    assert scan(dims(**bf), pro(out_norm=3, out_group=16, out_eps=1e-6)) == m3.M3_ERR_SHAPE
    assert scan(dims(**bf), pro(out_norm=-1)) == m3.M3_ERR_SHAPE
    assert scan(dims(**bf), pro(**dict(on, out_eps=0.0))) == m3.M3_ERR_SHAPE
    assert scan(dims(**bf), pro(**dict(on, out_eps=float("nan")))) == m3.M3_ERR_SHAPE
    for bad_group in (0, 4, 12, 128, -16):
        assert scan(dims(**bf), pro(**dict(on, out_group=bad_group))) == m3.M3_ERR_SHAPE
    assert scan(dims(**bf), pro(out_gain=FAKE)) == m3.M3_ERR_SHAPE     # gain without the norm
    assert scan(dims(**bf), pro(**dict(on, out_gain=FAKE + 4))) == m3.M3_ERR_ALIGN

    def step(d, p, over=None):
        ptrs = [FAKE] * 13       # state cB cX x B C dt A lam theta D z y
        ptrs[11] = None
        for k, v in (over or {}).items():
            ptrs[k] = v
        return L.m3_step_pro(ctypes.byref(d), None if p is None else ctypes.byref(p), *ptrs, None)
    assert step(dims(**bf), None) == m3.M3_ERR_NULL
    assert step(dims(**bf), pro(eps=-1.0)) == m3.M3_ERR_SHAPE
    assert step(dims(**bf), pro(out_norm=m3.M3_OUT_NORM_POST_GATE, out_group=128,
                                out_eps=1e-6)) == m3.M3_ERR_SHAPE
    assert step(dims(**bf), pro(w_z=FAKE)) == m3.M3_ERR_NULL
    assert step(dims(**bf), pro(norm_C=FAKE + 12)) == m3.M3_ERR_ALIGN
    assert step(dims(), pro()) == m3.M3_ERR_UNSUPPORTED
    assert step(dims(**bf), pro(), {0: None}) == m3.M3_ERR_NULL
    assert L.m3_last_hip_error() == 0


def test_backward_host_validation(L):
    """m3_scan_bwd: shapes, pointers, alignment and workspace are checked on
    the host before any launch; the workspace query agrees."""
    bf = dict(io=m3.M3_BF16, headdim=64, dstate=128, rank=1, chunk=64, seqlen=300)

    def call(d, over=None, ws_bytes=None):
        # x B C dt A lam theta D init dy dfinal dx dB dC ddt dA dlam dtheta dD dinit
        ptrs = [FAKE] * 20
        for k in (8, 10, 19):
            ptrs[k] = None
        for k, v in (over or {}).items():
            ptrs[k] = v
        need = L.m3_scan_bwd_workspace_bytes(ctypes.byref(d)) if ws_bytes is None else ws_bytes
        return L.m3_scan_bwd(ctypes.byref(d), *ptrs, FAKE, need, None)
    d = dims(**bf)
    need = L.m3_scan_bwd_workspace_bytes(ctypes.byref(d))
    nc = (300 + 63) // 64
    assert need >= 2 * nc * 3 * 128 * 64 * 4          # two fp32 and two bf16 N x P maps per chunk and slice
    assert call(dims(**dict(bf, rank=4, chunk=64))) == m3.M3_ERR_UNSUPPORTED   # chunk*rank 256
    assert L.m3_scan_bwd_workspace_bytes(ctypes.byref(dims(**dict(bf, rank=4, chunk=16)))) > 0
    assert call(dims()) == m3.M3_ERR_UNSUPPORTED                                  # fp32 not built
    assert call(dims(**dict(bf, flags=m3.M3_THETA_PER_HEAD))) == m3.M3_ERR_UNSUPPORTED
    assert call(dims(**dict(bf, a_stride_b=5, a_stride_t=0))) == m3.M3_ERR_UNSUPPORTED
    assert call(dims(**bf), {0: None}) == m3.M3_ERR_NULL
    assert call(dims(**bf), {9: None}) == m3.M3_ERR_NULL          # dy
    assert call(dims(**bf), {15: None}) == m3.M3_ERR_NULL         # dA
    assert call(dims(**bf), {9: FAKE + 2}) == m3.M3_ERR_ALIGN
    assert call(dims(**bf), {14: FAKE + 2}) == m3.M3_ERR_ALIGN    # ddt
    assert call(dims(**bf), ws_bytes=need - 1) == m3.M3_ERR_WORKSPACE
    assert L.m3_scan_bwd_workspace_bytes(ctypes.byref(dims())) == 0
    assert L.m3_last_hip_error() == 0
