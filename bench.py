"""Benchmark of the Mamba-3 SSM hot path on one MI355X.

One timed step = one pass of the whole hot path:
  * one m3_scan_fwd over the long-context MIMO prefill (B=1, L=65536, H=32,
    P=64, N=128, R=4, chunk 128, bf16 inputs, fp32 state): the largest
    prefill that fits one GPU, where the chunked algorithm's intensity
    (~275 FLOP per algorithmic byte) makes bf16 MFMA the roof;
  * one m3_step over the decode batch (B=256, H=32, P=64, N=128, R=4, fp32
    state from a 1024-token prefill), each step with fresh seeded inputs.
`value` is the prefill's tokens/s; `decode_us_per_step` the decode step time.
Both come from HIP events recorded on the stream the kernels run on; inputs
are resident in HBM before timing starts.  After the timed loop the other
prefill workloads are timed on their own (rank-4 B=8 L=4096 chunk 64, the
SISO B=4 L=2048 chunk 64 with its gated and per-head-frequency variants,
and the decode state's B=256 L=1024 prefill).  The CPU oracle is timed on
the host over whole workloads (decode: a sample of slices, scaled).

Usage: python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "prefill scan tokens/s + decode step µs @B=256; % of MFMA/HBM roofline"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-extras", action="store_true",
                    help="only the timed loop (the long-context prefill and the decode step)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run 10 plain device copies of 1 GiB (reference for HBM byte counters)")
    ap.add_argument("--bwd-calls", type=int, default=None, metavar="K",
                    help="only run K m3_scan_bwd calls (after one warm-up call) on the SISO "
                         "prefill workload's shape and print their mean time")
    ap.add_argument("--scan-workload", type=int, default=None, metavar="K",
                    help="only run --steps m3_scan_fwd calls (after one warm-up call) on prefill "
                         "workload K (1-4; the scan of workload 4 is its decode-state prefill) and "
                         "print their mean time, for hardware-counter runs")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): this build uses a "
              "single GPU; every (batch, head) slice is independent, so more GPUs would only "
              "split the batch.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2603_15569_amd import m3, roofline
    from paper_2603_15569_amd.inputs import (WORKLOADS, make_gate_input, make_step_inputs,
                                             workload_inputs)

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    if args.calibrate_copy:
        # a plain copy kernel of known size: reads and writes 2^30 bytes per launch
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(10):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes_each_way": 1 << 30, "launches": 10}), flush=True)
        return

    if args.bwd_calls is not None:
        bw = BackwardCase(m3, torch, dev, WORKLOADS, workload_inputs)
        bw.call()
        ms = bw.time(stream, args.bwd_calls)
        print(json.dumps({"bwd_workload": 1, "calls": args.bwd_calls, "ms_per_call": round(ms, 5)}),
              flush=True)
        return

    if args.scan_workload is not None:
        k = args.scan_workload
        if k not in (1, 2, 3, 4):
            print("--scan-workload takes 1, 2, 3 or 4", file=sys.stderr)
            sys.exit(2)
        inp = workload_inputs(k, device=dev)
        ms = time_scan(m3, torch, stream, [inp], WORKLOADS[k]["chunk"], 1, args.steps)
        Bk, Lk, Hk, Rk, Pk = inp.x.shape
        Nk = inp.Bm.shape[-1]
        fl = Bk * Hk * roofline.chunked_flops(Lk, Nk, Pk, Rk, WORKLOADS[k]["chunk"])
        print(json.dumps({"scan_workload": k, "shape": [Bk, Lk, Hk, Rk, Pk, Nk],
                          "chunk": WORKLOADS[k]["chunk"], "calls": args.steps,
                          "ms_per_call": round(ms, 5), "alg_tflops": round(fl / ms / 1e9, 2)}),
              flush=True)
        return

    peak_gbs = roofline.HBM_BYTES_PER_S / 1e9
    peak_tfs = roofline.MFMA_BF16_FLOPS / 1e12

    # ---------------- headline prefill: long-context MIMO, B=1 L=65536 H=32 R=4 ----------------
    log("inputs: long-context prefill")
    w3 = WORKLOADS[3]
    Q3 = w3["chunk"]
    p3 = workload_inputs(3, device=dev)
    B3, L3, H3, R3, P3 = p3.x.shape
    N3 = p3.Bm.shape[-1]
    ws3 = torch.zeros(max(m3.workspace_bytes(m3.scan_dims(p3.x, p3.Bm, Q3, p3.A)), 16),
                      dtype=torch.uint8, device=dev)
    out3 = (torch.empty_like(p3.x), torch.empty(B3, H3, N3, P3, device=dev),
            torch.empty(B3, H3, R3, N3, device=dev, dtype=p3.x.dtype),
            torch.empty(B3, H3, R3, P3, device=dev, dtype=p3.x.dtype))

    def scan3(i):
        m3.scan_fwd(p3.x, p3.Bm, p3.Cm, p3.dt, p3.A, p3.lam, p3.theta, p3.D, chunk=Q3, out=out3,
                    workspace=ws3)

    # ---------------- decode workload (B=256, MIMO R=4) ----------------
    log("inputs: decode state prefill")
    wd = WORKLOADS[4]
    layer = workload_inputs(4, device=dev)
    pre_args = (layer.x, layer.Bm, layer.Cm, layer.dt, layer.A, layer.lam, layer.theta, layer.D)
    _, dstate, (dcB, dcX) = m3.scan_fwd(*pre_args, chunk=wd["chunk"])
    torch.cuda.synchronize()
    Bm_, Lm_, Hm_, Rm_, Pm_ = layer.x.shape
    Nm_ = layer.Bm.shape[-1]
    mimo_ms = None
    if not args.no_extras:
        # the same decode-state prefill (rank 4, 8192 slices), timed over a few
        # more calls writing the same state (the decode steps start from it)
        mimo_out = (torch.empty_like(layer.x), dstate, dcB, dcX)
        mimo_ms = time_scan(m3, torch, stream, [layer], wd["chunk"], 1, 3, out=mimo_out)
        del mimo_out
    del pre_args
    del layer.x, layer.Bm, layer.Cm, layer.theta, layer.lam, layer.dt  # free the prefill inputs
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    n_step_inputs = max(1, min(args.steps + args.warmup, wd["steps"]))
    step_in = [make_step_inputs(_LayerView(layer, wd), s, device=dev) for s in range(n_step_inputs)]
    yd = torch.empty_like(step_in[0].x)

    def dstep(i):
        st = step_in[i % n_step_inputs]
        m3.step(dstate, (dcB, dcX), st.x, st.Bm, st.Cm, st.dt, layer.A, st.lam, st.theta, layer.D,
                y=yd)

    # ---------------- timed loop ----------------
    log(f"timed loop: {args.warmup} warm-up + {args.steps} steps")
    for i in range(args.warmup):
        scan3(i)
        dstep(i)
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    for i in range(args.steps):
        ev[i][0].record(stream)
        scan3(i)
        ev[i][1].record(stream)
        dstep(args.warmup + i)
        ev[i][2].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    scan_ms = np.array([e[0].elapsed_time(e[1]) for e in ev])
    step_ms = np.array([e[1].elapsed_time(e[2]) for e in ev])
    tot_ms = np.array([e[0].elapsed_time(e[2]) for e in ev])
    assert m3.scan_check(m3.scan_dims(p3.x, p3.Bm, Q3, p3.A), ws3) == 0, "look-back wait timed out"

    tokens3 = B3 * L3
    pre_ms = float(scan_ms.mean())
    pre_bytes = roofline.prefill_bytes(B3, L3, H3, N3, P3, R3, 2)
    pre_flops = B3 * H3 * roofline.chunked_flops(L3, N3, P3, R3, Q3)
    pre_tfs = pre_flops / (pre_ms * 1e-3) / 1e12
    pre_gbs = pre_bytes / (pre_ms * 1e-3) / 1e9
    Bd, Hd, Rd, Pd = step_in[0].x.shape
    Nd = step_in[0].Bm.shape[-1]
    dec_us = float(step_ms.mean()) * 1e3
    dec_bytes = Bd * Hd * roofline.decode_bytes_per_slice(Nd, Pd, Rd, 2)
    dec_gbs = dec_bytes / (dec_us * 1e-6) / 1e9

    result = {
        "metric": METRIC,
        "value": round(tokens3 / (pre_ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(float(tot_ms.mean()), 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": (f"long-context MIMO prefill B={B3} L={L3} H={H3} P={P3} N={N3} R={R3} "
                         f"chunk={Q3} bf16 in, fp32 state + decode step B={Bd} H={Hd} P={Pd} "
                         f"N={Nd} R={Rd} fp32 state"),
            "prefill": {"batch": B3, "seqlen": L3, "nheads": H3, "headdim": P3, "dstate": N3,
                        "rank": R3, "chunk": Q3, "io": "bf16", "state": "fp32"},
            "decode": {"batch": Bd, "nheads": Hd, "headdim": Pd, "dstate": Nd, "rank": Rd,
                       "io": "bf16", "state": "fp32"},
        },
        "prefill_ms": round(pre_ms, 5),
        "prefill_ms_p10_p90": [round(float(np.percentile(scan_ms, 10)), 5),
                               round(float(np.percentile(scan_ms, 90)), 5)],
        "decode_us_per_step": round(dec_us, 3),
        "decode_us_p10_p90": [round(float(np.percentile(step_ms, 10)) * 1e3, 3),
                              round(float(np.percentile(step_ms, 90)) * 1e3, 3)],
        # the dominant kernel of the step: the long-context scan (one
        # m3_scan_fwd = one launch of the per-chunk kernel)
        "roofline": {
            "kernel": "m3_scan_fwd long-context MIMO prefill (k_scan_fused<bf16,128,4>)",
            "bound": "mfma", "achieved": round(pre_tfs, 2), "peak": peak_tfs, "unit": "TFLOP/s",
            "frac": round(pre_tfs / peak_tfs, 4),
            "traffic": measured_traffic("k_scan_fused_long"),
            "flops_per_launch": pre_flops,
            "hbm_achieved_gbs": round(pre_gbs, 1), "hbm_frac": round(pre_gbs / peak_gbs, 4),
            "bytes_per_launch": pre_bytes,
        },
        "roofline_decode": {
            "kernel": "k_step (m3_step, one launch per step)",
            "bound": "hbm", "achieved": round(dec_gbs, 1), "peak": peak_gbs, "unit": "GB/s",
            "frac": round(dec_gbs / peak_gbs, 4), "traffic": measured_traffic("k_step"),
            "bytes_per_launch": dec_bytes,
        },
        "wall_s_timed_loop": round(wall, 3),
    }
    if mimo_ms is not None:
        result["prefill_decode_state"] = prefill_figures(
            roofline, Bm_, Lm_, Hm_, Nm_, Pm_, Rm_, wd["chunk"], mimo_ms,
            "warp-specialised kernel, one workgroup per slice", measured_traffic("k_scan_ws_mimo"))

    if not args.no_extras:
        del ev
        # ---------------- rank-4 prefill, B=8 L=4096 H=32 ----------------
        log("extras: rank-4 prefill")
        w2 = WORKLOADS[2]
        p2 = workload_inputs(2, device=dev)
        ms2 = time_scan(m3, torch, stream, [p2], w2["chunk"], 3, 20)
        B2, L2, H2, R2, P2 = p2.x.shape
        result["prefill_mimo"] = prefill_figures(
            roofline, B2, L2, H2, p2.Bm.shape[-1], P2, R2, w2["chunk"], ms2,
            "warp-specialised kernel, one workgroup per slice", measured_traffic("k_scan_ws_w2"))
        del p2
        torch.cuda.empty_cache()
        # ---------------- SISO prefill B=4 L=2048 H=16, gated and per-head variants ----------------
        log("extras: SISO prefill")
        result.update(siso_figures(m3, roofline, torch, np, stream, dev, WORKLOADS[1],
                                   workload_inputs, make_gate_input, step_in, dstep, dstate,
                                   dcB, dcX, layer, yd, peak_gbs))

    if not args.no_extras:
        log("extras: block prologue")
        result["prologue"] = prologue_figures(m3, roofline, torch, stream, dev, WORKLOADS,
                                              workload_inputs, peak_gbs, peak_tfs)
        torch.cuda.empty_cache()
        log("extras: backward")
        bw = BackwardCase(m3, torch, dev, WORKLOADS, workload_inputs)
        for _ in range(3):
            bw.call()
        ms = bw.time(stream, 20)
        result["backward_siso"] = bw.figures(roofline, ms, peak_gbs, peak_tfs)
        result["backward_siso"]["traffic"] = measured_traffic("backward_siso")
        del bw
        torch.cuda.empty_cache()
        log("extras: backward at rank 4 and SISO, B=8 L=4096 H=32")
        result["backward_mimo"] = backward_mimo_figures(torch, stream, dev, WORKLOADS, workload_inputs,
                                                        m3, roofline, peak_gbs, peak_tfs)
        torch.cuda.empty_cache()
        log("extras: decode at state size 64")
        result["decode_state64"] = decode_state64_figures(m3, roofline, torch, stream, dev,
                                                          wd, dec_us, peak_gbs)
        torch.cuda.empty_cache()

    if not args.no_cpu:
        log("CPU baseline")
        result["cpu_baseline"] = cpu_baseline(p3, layer, step_in, WORKLOADS)
    print(json.dumps(result), flush=True)
    torch.cuda.synchronize()


def time_scan(m3, torch, stream, copies, chunk, warm, n, out=None, z=None, theta_per_head=False):
    """Mean ms of n m3_scan_fwd calls (after `warm` untimed ones), rotating
    over the input copies, one workspace."""
    c0 = copies[0]
    ws = torch.zeros(max(m3.workspace_bytes(m3.scan_dims(c0.x, c0.Bm, chunk, c0.A)), 16),
                     dtype=torch.uint8, device=c0.x.device)
    if out is None:
        Bb, Lb, Hb, Rb, Pb = c0.x.shape
        Nb = c0.Bm.shape[-1]
        out = (torch.empty_like(c0.x), torch.empty(Bb, Hb, Nb, Pb, device=c0.x.device),
               torch.empty(Bb, Hb, Rb, Nb, device=c0.x.device, dtype=c0.x.dtype),
               torch.empty(Bb, Hb, Rb, Pb, device=c0.x.device, dtype=c0.x.dtype))

    def call(i):
        c = copies[i % len(copies)]
        m3.scan_fwd(c.x, c.Bm, c.Cm, c.dt, c.A, c.lam, c.omega if theta_per_head else c.theta,
                    c.D, chunk=chunk, out=out, workspace=ws,
                    z=None if z is None else z[i % len(z)])

    for i in range(warm):
        call(i)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for i in range(n):
        call(warm + i)
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / max(1, n)


def prefill_figures(roofline, B, L, H, N, P, R, Q, ms, kernel, traffic):
    """Tokens/s and the algorithmic HBM and bf16 MFMA rates of one prefill."""
    nbytes = roofline.prefill_bytes(B, L, H, N, P, R, 2)
    flops = B * H * roofline.chunked_flops(L, N, P, R, Q)
    gbs = nbytes / (ms * 1e-3) / 1e9
    tfs = flops / (ms * 1e-3) / 1e12
    return {
        "workload": f"prefill B={B} L={L} H={H} P={P} N={N} R={R} chunk={Q} bf16",
        "kernel": kernel, "ms": round(ms, 4), "tokens_per_s": round(B * L / (ms * 1e-3), 1),
        "hbm_achieved_gbs": round(gbs, 1), "hbm_frac": round(gbs * 1e9 / roofline.HBM_BYTES_PER_S, 4),
        "bytes_per_launch": nbytes, "traffic": traffic,
        "mfma_tflops": round(tfs, 2), "mfma_frac": round(tfs * 1e12 / roofline.MFMA_BF16_FLOPS, 4),
        "flops_per_launch": flops,
    }


def siso_figures(m3, roofline, torch, np, stream, dev, wp, workload_inputs, make_gate_input,
                 step_in, dstep, dstate, dcB, dcX, layer, yd, peak_gbs):
    """The SISO bf16 prefill (B=4 L=2048 H=16, chunk 64; inputs rotated over
    four resident copies, 550 MB, so the 256 MB Infinity Cache cannot hold
    them), alternating with decode steps as in the timed loop; its fused
    output gate against the ungated scan and against the ungated scan
    followed by a separate torch gate pass; and the scan with per-head rotary
    frequencies (angles dt * omega formed in the kernels)."""
    base = workload_inputs(1, device=dev)
    copies = [base] + [type(base)(**{k: (v.clone() if isinstance(v, torch.Tensor) else v)
                                     for k, v in base.__dict__.items()}) for _ in range(3)]
    Bp, Lp, Hp, Rp, Pp = base.x.shape
    Np = base.Bm.shape[-1]
    Qp = wp["chunk"]
    ws = torch.zeros(max(m3.workspace_bytes(m3.scan_dims(base.x, base.Bm, Qp, base.A)), 16),
                     dtype=torch.uint8, device=dev)
    out = (torch.empty_like(base.x), torch.empty(Bp, Hp, Np, Pp, device=dev),
           torch.empty(Bp, Hp, Rp, Np, device=dev, dtype=base.x.dtype),
           torch.empty(Bp, Hp, Rp, Pp, device=dev, dtype=base.x.dtype))
    zs = [make_gate_input(c.x, i) for i, c in enumerate(copies)]
    zd = [make_gate_input(st.x, 100 + i) for i, st in enumerate(step_in[:4])]
    n_in = len(step_in)

    def scan(i, gated=False, per_head=False):
        c = copies[i % len(copies)]
        m3.scan_fwd(c.x, c.Bm, c.Cm, c.dt, c.A, c.lam, c.omega if per_head else c.theta, c.D,
                    chunk=Qp, out=out, workspace=ws, z=zs[i % len(zs)] if gated else None)

    def unfused(i):   # ungated scan, then the gate as a separate elementwise pass
        scan(i)
        out[0].mul_(torch.nn.functional.silu(zs[i % len(zs)]))

    def gstep(i):
        st = step_in[i % n_in]
        m3.step(dstate, (dcB, dcX), st.x, st.Bm, st.Cm, st.dt, layer.A, st.lam, st.theta, layer.D,
                y=yd, z=zd[i % len(zd)])

    def timed(pre, dec, n=100):
        for i in range(3):
            pre(i)
            dec(i)
        e = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n)]
        torch.cuda.synchronize()
        for i in range(n):
            e[i][0].record(stream)
            pre(i)
            e[i][1].record(stream)
            dec(i)
            e[i][2].record(stream)
        torch.cuda.synchronize()
        return (float(np.mean([x[0].elapsed_time(x[1]) for x in e])),
                float(np.mean([x[1].elapsed_time(x[2]) for x in e])))

    s_ms, d_ms = timed(scan, dstep)
    g_ms, gd_ms = timed(lambda i: scan(i, gated=True), gstep)
    u_ms, _ = timed(unfused, dstep)
    ph_ms, _ = timed(lambda i: scan(i, per_head=True), dstep)
    tokens = Bp * Lp
    pre_bytes = roofline.prefill_bytes(Bp, Lp, Hp, Np, Pp, Rp, 2)
    z_bytes = Bp * Lp * Hp * Rp * Pp * 2
    Bd, Hd, Rd, Pd = step_in[0].x.shape
    Nd = step_in[0].Bm.shape[-1]
    dec_bytes = Bd * Hd * roofline.decode_bytes_per_slice(Nd, Pd, Rd, 2)
    zd_bytes = Bd * Hd * Rd * Pd * 2
    ph_bytes = pre_bytes - Bp * Lp * Hp * (Np // 2) * 4 + Hp * (Np // 2) * 4
    siso = prefill_figures(roofline, Bp, Lp, Hp, Np, Pp, Rp, Qp, s_ms,
                           "one chunk per workgroup, look-back", measured_traffic("k_scan_fused_siso"))
    return {
        "prefill_siso": siso,
        "gate": {
            "prefill_ms": round(g_ms, 5), "prefill_tokens_per_s": round(tokens / (g_ms * 1e-3), 1),
            "prefill_achieved_gbs": round((pre_bytes + z_bytes) / (g_ms * 1e-3) / 1e9, 1),
            "prefill_bytes_per_launch": pre_bytes + z_bytes,
            "ungated_prefill_ms": round(s_ms, 5), "unfused_prefill_ms": round(u_ms, 5),
            "decode_us_per_step": round(gd_ms * 1e3, 3),
            "ungated_decode_us_per_step": round(d_ms * 1e3, 3),
            "decode_achieved_gbs": round((dec_bytes + zd_bytes) / (gd_ms * 1e-3) / 1e9, 1),
            "decode_frac": round((dec_bytes + zd_bytes) / (gd_ms * 1e-3) / 1e9 / peak_gbs, 4),
            "decode_bytes_per_launch": dec_bytes + zd_bytes,
        },
        "theta_per_head": {
            "prefill_ms": round(ph_ms, 5), "prefill_tokens_per_s": round(tokens / (ph_ms * 1e-3), 1),
            "per_token_theta_prefill_ms": round(s_ms, 5),
            "achieved_gbs": round(ph_bytes / (ph_ms * 1e-3) / 1e9, 1),
            "frac": round(ph_bytes / (ph_ms * 1e-3) / 1e9 / peak_gbs, 4), "bytes_per_launch": ph_bytes,
        },
    }


def prologue_figures(m3, roofline, torch, stream, dev, W, workload_inputs, peak_gbs, peak_tfs):
    """The prefill with the block prologue fused (BCNorm with gains, B/C
    biases, structured MIMO input X = W_X o X') on the three prefill
    workloads' shapes, against the plain scan of the same shape (the
    library's default kernel, and the one-chunk-per-workgroup kernel; the
    prologue scan runs in the warp-specialised kernel where the default
    choice is that kernel, the rank-4 B=8 L=4096 prefill, else in the
    one-chunk-per-workgroup kernel)."""
    from paper_2603_15569_amd.inputs import make_prologue_inputs
    out = {}
    for k in (1, 2, 3):
        w = W[k]
        inp = workload_inputs(k, device=dev)
        pin = make_prologue_inputs(w["batch"], w["seqlen"], w["nheads"], w["headdim"], w["dstate"],
                                   w["rank"], io="bf16", seed=k, device=dev)
        pro = m3.prologue(bc_norm=True, eps=1e-6, norm_B=pin.gB, norm_C=pin.gC, bias_B=pin.bB,
                          bias_C=pin.bC, w_x=pin.wx)
        B, L, H, R, P = inp.x.shape
        N = inp.Bm.shape[-1]
        Q = w["chunk"]
        d = m3.scan_dims(inp.x, inp.Bm, Q, inp.A)
        ws = torch.zeros(max(m3.workspace_bytes(d), 16), dtype=torch.uint8, device=dev)
        o = (torch.empty_like(inp.x), torch.empty((B, H, N, P), device=dev),
             torch.empty((B, H, R, N), device=dev, dtype=inp.x.dtype),
             torch.empty((B, H, R, P), device=dev, dtype=inp.x.dtype))

        def plain(per_chunk):
            return lambda: m3.scan_fwd(inp.x, inp.Bm, inp.Cm, inp.dt, inp.A, inp.lam, inp.theta,
                                       inp.D, chunk=Q, out=o, workspace=ws, per_chunk=per_chunk)

        def fused():
            m3.scan_fwd_pro(pin.xp, pin.Bp, pin.Cp, inp.dt, inp.A, inp.lam, inp.theta, inp.D, Q,
                            pro, R, out=o, workspace=ws)

        def timed(fn, n):
            for _ in range(2):
                fn()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record(stream)
            for _ in range(n):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / n
        n = 20 if k == 1 else 5
        t_pro, t_def, t_pc = timed(fused, n), timed(plain(False), n), timed(plain(True), n)
        nbytes = roofline.prologue_prefill_bytes(B, L, H, N, P, R, 2)
        flops = B * H * roofline.chunked_flops(L, N, P, R, Q)
        gbs = nbytes / (t_pro * 1e-3) / 1e9
        out[f"workload{k}"] = {
            "workload": f"prefill B={B} L={L} H={H} P={P} N={N} R={R} chunk={Q} bf16, BCNorm + gains + "
                        "biases + structured input",
            "ms": round(t_pro, 4), "tokens_per_s": round(B * L / (t_pro * 1e-3), 1),
            "bytes_per_launch": nbytes, "achieved_gbs": round(gbs, 1),
            "hbm_frac": round(gbs / peak_gbs, 4),
            "mfma_frac": round(flops / (t_pro * 1e-3) / 1e12 / peak_tfs, 4),
            "plain_default_ms": round(t_def, 4), "plain_per_chunk_ms": round(t_pc, 4),
            "plain_bytes_per_launch": roofline.prefill_bytes(B, L, H, N, P, R, 2),
        }
        del inp, pin, ws, o
        torch.cuda.empty_cache()
    return out


def decode_state64_figures(m3, roofline, torch, stream, dev, wd, dec_us_128, peak_gbs):
    """The decode workload's batch, heads and rank at state size 64 (the
    paper's MIMO state-size point): microseconds per step from a random fp32
    state and carry, seeded step inputs, against the state-128 step."""
    from paper_2603_15569_amd.inputs import make_scan_inputs, make_step_inputs
    B, H, R, P, N = wd["batch"], wd["nheads"], wd["rank"], wd["headdim"], 64
    layer = make_scan_inputs(B, 1, H, P, N, R, io="bf16", seed=4400, device=dev, chunk=64)
    g = torch.Generator(dev).manual_seed(4401)
    state = torch.randn((B, H, N, P), device=dev, generator=g) * 0.1
    cB = torch.randn((B, H, R, N), device=dev, generator=g).to(torch.bfloat16)
    cX = torch.randn((B, H, R, P), device=dev, generator=g).to(torch.bfloat16)
    steps = [make_step_inputs(layer, s, device=dev) for s in range(8)]
    y = torch.empty_like(steps[0].x)

    def step(i):
        st = steps[i % len(steps)]
        m3.step(state, (cB, cX), st.x, st.Bm, st.Cm, st.dt, layer.A, st.lam, st.theta, layer.D, y=y)
    for i in range(5):
        step(i)
    n = 100
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for i in range(n):
        step(i)
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / n * 1e3
    nbytes = B * H * roofline.decode_bytes_per_slice(N, P, R, 2)
    gbs = nbytes / (us * 1e-6) / 1e9
    return {"workload": f"decode step B={B} H={H} P={P} N={N} R={R} fp32 state",
            "us_per_step": round(us, 3), "achieved_gbs": round(gbs, 1),
            "hbm_frac": round(gbs / peak_gbs, 4), "bytes_per_launch": nbytes,
            "state128_us_per_step": round(dec_us_128, 3),
            "ratio_to_state128": round(us / dec_us_128, 3)}


class BackwardCase:
    """m3_scan_bwd on prefill workload k's shape (by default the SISO one:
    B=4, L=2048, H=16, P=64, N=128, chunk 64; `override` changes fields such
    as the rank and the chunk): inputs, dy, dJ/d(final state) and the
    outputs and workspace allocated once."""

    def __init__(self, m3, torch, dev, W, workload_inputs, k=1, **override):
        import ctypes
        self.m3, self.torch, self.ctypes = m3, torch, ctypes
        self.inp = inp = workload_inputs(k, device=dev, **override)
        self.chunk = override.get("chunk", W[k]["chunk"])
        g = torch.Generator(dev).manual_seed(77)
        B, L, H, R, P = inp.x.shape
        N = inp.Bm.shape[-1]
        self.shape = (B, L, H, R, P, N)
        self.dy = torch.randn(inp.x.shape, device=dev, generator=g).to(inp.x.dtype)
        self.dfin = torch.randn((B, H, N, P), device=dev, generator=g) * 0.1
        self.d = m3.scan_dims(inp.x, inp.Bm, self.chunk, inp.A)
        f32 = dict(dtype=torch.float32, device=dev)
        self.out = [torch.empty_like(inp.x), torch.empty_like(inp.Bm), torch.empty_like(inp.Cm),
                    torch.empty((B, L, H), **f32), torch.empty((H,), **f32),
                    torch.empty((B, L, H), **f32), torch.empty((B, L, H, N // 2), **f32),
                    torch.empty((H,), **f32)]
        nb = int(m3.lib().m3_scan_bwd_workspace_bytes(ctypes.byref(self.d)))
        self.ws = torch.empty(nb, dtype=torch.uint8, device=dev)

    def call(self):
        m3, i, o = self.m3, self.inp, self.out
        p = m3._p
        m3._check(m3.lib().m3_scan_bwd(
            self.ctypes.byref(self.d), p(i.x), p(i.Bm), p(i.Cm), p(i.dt), p(i.A), p(i.lam),
            p(i.theta), p(i.D), None, p(self.dy), p(self.dfin), p(o[0]), p(o[1]), p(o[2]),
            p(o[3]), p(o[4]), p(o[5]), p(o[6]), p(o[7]), None, p(self.ws), self.ws.numel(),
            m3._stream(None)))

    def time(self, stream, n):
        torch = self.torch
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(n):
            self.call()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    def figures(self, roofline, ms, peak_gbs, peak_tfs):
        B, L, H, R, P, N = self.shape
        nbytes = roofline.backward_bytes(B, L, H, N, P, R, 2)
        flops = B * H * roofline.backward_flops(L, N, P, R, self.chunk)
        gbs = nbytes / (ms * 1e-3) / 1e9
        return {"workload": f"backward B={B} L={L} H={H} P={P} N={N} R={R} chunk={self.chunk} bf16",
                "ms": round(ms, 5), "tokens_per_s": round(B * L / (ms * 1e-3), 1),
                "bound": "hbm", "achieved_gbs": round(gbs, 1), "frac": round(gbs / peak_gbs, 4),
                "bytes_per_launch": nbytes, "flops_per_launch": flops,
                "mfma_tflops": round(flops / (ms * 1e-3) / 1e12, 2)}


def backward_mimo_figures(torch, stream, dev, W, workload_inputs, m3, roofline, peak_gbs, peak_tfs):
    """The backward at rank 4 (chunk 16: 64 rows a chunk, the backward's
    tile) on the rank-4 prefill's batch, length and heads (B=8 L=4096 H=32),
    and the SISO backward
    (chunk 64) of the same batch, length and heads: the paper puts MIMO
    training at rank 4 about twice as slow as SISO (Sec. 3.3)."""
    out = {}
    for name, ov in (("mimo", dict(chunk=16)), ("siso", dict(rank=1, chunk=64))):
        bw = BackwardCase(m3, torch, dev, W, workload_inputs, k=2, **ov)
        for _ in range(2):
            bw.call()
        ms = bw.time(stream, 5)
        out[name] = bw.figures(roofline, ms, peak_gbs, peak_tfs)
        del bw
        torch.cuda.empty_cache()
    res = dict(out["mimo"])
    res["siso_same_shape_ms"] = out["siso"]["ms"]
    res["siso_same_shape_tokens_per_s"] = out["siso"]["tokens_per_s"]
    res["time_ratio_to_siso"] = round(out["mimo"]["ms"] / out["siso"]["ms"], 3)
    return res


def measured_traffic(key):
    """HBM bytes per launch measured with rocprofv3 counters (profiles/traffic.json),
    or None when the kernel source changed since the measurement."""
    import hashlib
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))[key]
        srcs = rec["sources"]
        blob = b"".join(open(os.path.join(ROOT, f), "rb").read() for f in srcs)
    except (OSError, KeyError, ValueError, TypeError):
        return None
    if hashlib.sha256(blob).hexdigest() != rec["src_sha256"]:
        return None
    return rec["read_bytes"] + rec["write_bytes"]


class _LayerView:
    """Shape/dtype view of the decode layer for the step-input generator."""

    def __init__(self, layer, w):
        import torch
        self.x = torch.empty((w["batch"], 1, w["nheads"], w["rank"], w["headdim"]),
                             dtype=torch.bfloat16, device=layer.A.device)
        self.Bm = torch.empty((w["batch"], 1, w["nheads"], w["rank"], w["dstate"]),
                              dtype=torch.bfloat16, device=layer.A.device)
        self.dt_bias = layer.dt_bias
        self.omega = layer.omega


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(p3, layer, step_in, W):
    """The fp64 oracle (-O3 -march=native, built here for this host) on the
    host cores: every slice of the long-context prefill (the headline; in
    two halves of 16 slices to bound host memory), every slice of the rank-4
    and of the SISO prefill batches, and one decode step on 64 of the 8192
    slices scaled to the batch."""
    import numpy as np
    import torch
    import oracle
    from paper_2603_15569_amd.inputs import workload_inputs
    flags = oracle.use_native()

    def run(inp, slices, L):
        ref = oracle.slices_of_scan(inp.x, inp.Bm, inp.Cm, inp.dt, inp.A, inp.lam, inp.theta,
                                    inp.D, slices, 0, L)
        t0 = time.perf_counter()
        _, used = oracle.scan(**ref, return_threads=True)
        return time.perf_counter() - t0, used

    w3 = W[3]
    t3, used = 0.0, 1
    all3 = [(b, h) for b in range(w3["batch"]) for h in range(w3["nheads"])]
    for half in (all3[:len(all3) // 2], all3[len(all3) // 2:]):
        dt_, used = run(p3, half, w3["seqlen"])
        t3 += dt_
    out = {"value": round(w3["batch"] * w3["seqlen"] / t3, 1), "unit": "tokens/s",
           "cores": int(used), "kind": "oracle"}
    detail = {"long_context_s": round(t3, 2)}
    for k, key in ((2, "mimo"), (1, "siso")):
        w = W[k]
        inp = workload_inputs(k, device=p3.x.device)
        dt_, _ = run(inp, [(b, h) for b in range(w["batch"]) for h in range(w["nheads"])], w["seqlen"])
        detail[f"{key}_s"] = round(dt_, 2)
        detail[f"{key}_tokens_per_s"] = round(w["batch"] * w["seqlen"] / dt_, 1)
        del inp
    wd = W[4]
    dsl = [(b, h) for b in range(0, wd["batch"], 4) for h in range(0, wd["nheads"], 8)][:64]
    st = step_in[0]
    p = oracle.slices_of_step(st.x, st.Bm, st.Cm, st.dt, st.lam, st.theta, dsl)
    N, P, R = wd["dstate"], wd["headdim"], wd["rank"]
    rng = np.random.default_rng(0)
    S = len(dsl)
    state = rng.standard_normal((S, N, P))
    cb, cx = rng.standard_normal((S, R, N)), rng.standard_normal((S, R, P))
    A_s = np.array([float(layer.A[h]) for _, h in dsl])
    D_s = np.array([float(layer.D[h]) for _, h in dsl])
    reps = 20
    t0 = time.perf_counter()
    for _ in range(reps):
        oracle.step(state, cb, cx, p["x"], p["B"], p["C"], p["dt"], A_s, p["lam"], p["theta"], D_s)
    ddt = (time.perf_counter() - t0) / reps
    detail["decode_us_per_step"] = round(ddt * (wd["batch"] * wd["nheads"] / S) * 1e6, 1)
    out["sample"] = (f"prefill: all {len(all3)} (batch, head) slices x {w3['seqlen']} tokens of the "
                     f"long-context batch in two halves, fp64, {t3:.1f} s (also every slice of the "
                     f"rank-4 and SISO batches, below); decode: one step on {S} of "
                     f"{wd['batch'] * wd['nheads']} slices x {reps} reps, scaled (extrapolated)")
    out.update(detail)
    out["cpu_model"] = cpu_model()
    out["nproc"] = os.cpu_count()
    out["build"] = flags
    del torch
    return out


if __name__ == "__main__":
    main()
