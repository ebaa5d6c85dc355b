"""The allocation-free prefill entry point (m3_scan_fwd_noalloc, the
library's fixed device scratch as workspace) against m3_scan_fwd with a
caller workspace: the same kernels, so the same bits, on two calls in a row
(the second smaller and on another kernel, so it reuses the first call's
scratch contents), and within tolerance of the fp64 oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2603_15569_amd import m3
from paper_2603_15569_amd.inputs import make_scan_inputs

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def outputs(inp, fill):
    B_, L, H, R, P = inp.x.shape
    N = inp.Bm.shape[-1]
    return (torch.full_like(inp.x, fill), torch.full((B_, H, N, P), fill, device=DEV),
            torch.full((B_, H, R, N), fill, device=DEV, dtype=inp.x.dtype),
            torch.full((B_, H, R, P), fill, device=DEV, dtype=inp.x.dtype))


@pytest.mark.parametrize("case", [
    # batch, L, heads, R, chunk, chunks per segment: a linked-segment scan
    # (look-back across segments), then a smaller SISO scan on the
    # one-chunk-per-workgroup kernel
    ((2, 1000, 8, 4, 64, 0), (1, 300, 4, 1, 64, 0)),
    # a scan of one segment per slice (warp-specialised kernel), then a
    # smaller look-back scan
    ((2, 777, 3, 4, 64, 1 << 20), (1, 200, 2, 2, 32, 0)),
])
def test_noalloc_matches_workspace_call(case):
    for k, (Bb, L, H, R, Q, seg) in enumerate(case):
        print(f"[gpu-case] noalloc call {k}: B={Bb} L={L} H={H} R={R} Q={Q} seg={seg}", flush=True)
        inp = make_scan_inputs(Bb, L, H, 64, 128, R, io="bf16", seed=300 + 7 * k + R, device=DEV, chunk=Q)
        args = (inp.x, inp.Bm, inp.Cm, inp.dt, inp.A, inp.lam, inp.theta, inp.D)
        d = m3.scan_dims(inp.x, inp.Bm, Q, inp.A, seg=seg)
        assert 0 < m3.workspace_bytes(d) <= m3.SCRATCH_BYTES
        ref = m3.scan_fwd(*args, chunk=Q, out=outputs(inp, float("nan")), seg=seg)
        got = m3.scan_fwd_noalloc(*args, chunk=Q, out=outputs(inp, float("nan")), seg=seg)
        torch.cuda.synchronize()
        (ry, rs, (rb, rx)), (gy, gs, (gb, gx)) = ref, got
        for a, b in ((gy, ry), (gs, rs), (gb, rb), (gx, rx)):
            assert torch.equal(a, b)
        sl = [(0, 0), (Bb - 1, H - 1)]
        o = oracle.slices_of_scan(*args, sl)
        oy, os_, _, _ = oracle.scan(**o)
        for i, (b, h) in enumerate(sl):
            assert oracle.rel_err(gy[b, :, h].double().cpu().numpy(), oy[i]) <= 2e-2
            assert oracle.rel_err(gs[b, h].cpu().numpy(), os_[i]) <= 2e-2
