"""Benchmark of the Mamba-3 SSM hot path on one MI355X.

One timed step = one pass of the whole hot path:
  * one m3_scan_fwd over the SISO bf16 prefill batch (B=4, L=2048, H=16,
    P=64, N=128, R=1, chunk 64), inputs rotated over 4 resident copies so the
    256 MB Infinity Cache cannot hold them between steps;
  * one m3_step over the decode batch (B=256, H=32, P=64, N=128, R=4, fp32
    state from a 1024-token prefill), each step with fresh seeded inputs.
`value` is the prefill tokens/s; `decode_us_per_step` the decode step time.
Both come from HIP events recorded on the stream the kernels run on.  The
CPU oracle is timed on a bounded sample of the same workloads on the host.

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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run 10 plain device copies of 1 GiB (reference for HBM byte counters)")
    ap.add_argument("--scan-workload", type=int, default=None, metavar="K",
                    help="only run --steps m3_scan_fwd calls (after one warm-up call) on prefill "
                         "workload K (1-4; the scan of workload 4 is its decode-state prefill) and "
                         "print their mean time, for hardware-counter runs")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); every (batch, head) "
              "slice is independent, so more GPUs would only split the batch.", file=sys.stderr)
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

    if args.scan_workload is not None:
        k = args.scan_workload
        if k not in (1, 2, 3, 4):
            print("--scan-workload takes 1, 2, 3 or 4", file=sys.stderr)
            sys.exit(2)
        w = WORKLOADS[k]
        inp = workload_inputs(k, device=dev)
        Bk, Lk, Hk, Rk, Pk = inp.x.shape
        Nk = inp.Bm.shape[-1]
        dims = m3.scan_dims(inp.x, inp.Bm, w["chunk"], inp.A)
        ws = torch.zeros(m3.workspace_bytes(dims), dtype=torch.uint8, device=dev)
        args_k = (inp.x, inp.Bm, inp.Cm, inp.dt, inp.A, inp.lam, inp.theta, inp.D)
        m3.scan_fwd(*args_k, chunk=w["chunk"], workspace=ws)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            m3.scan_fwd(*args_k, chunk=w["chunk"], workspace=ws)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / max(1, args.steps)
        fl = Bk * Hk * roofline.chunked_flops(Lk, Nk, Pk, Rk, w["chunk"])
        print(json.dumps({"scan_workload": k, "shape": [Bk, Lk, Hk, Rk, Pk, Nk], "chunk": w["chunk"],
                          "calls": args.steps, "ms_per_call": round(ms, 5),
                          "alg_tflops": round(fl / ms / 1e9, 2)}), flush=True)
        return

    # ---------------- prefill workload (SISO bf16) ----------------
    wp = WORKLOADS[1]
    base = workload_inputs(1, device=dev)
    copies = [base] + [type(base)(**{k: (v.clone() if isinstance(v, torch.Tensor) else v)
                                     for k, v in base.__dict__.items()}) for _ in range(3)]
    Bp, Lp, Hp, Rp, Pp = base.x.shape
    Np = base.Bm.shape[-1]
    Qp = wp["chunk"]
    dims = m3.scan_dims(base.x, base.Bm, Qp, base.A)
    ws = torch.empty(max(m3.workspace_bytes(dims), 1), dtype=torch.uint8, device=dev)
    out = (torch.empty_like(base.x), torch.empty(Bp, Hp, Np, Pp, device=dev),
           torch.empty(Bp, Hp, Rp, Np, device=dev, dtype=base.x.dtype),
           torch.empty(Bp, Hp, Rp, Pp, device=dev, dtype=base.x.dtype))

    def scan(i):
        c = copies[i % len(copies)]
        m3.scan_fwd(c.x, c.Bm, c.Cm, c.dt, c.A, c.lam, c.theta, c.D, chunk=Qp, out=out,
                    workspace=ws)

    # ---------------- decode workload (B=256, MIMO R=4) ----------------
    wd = WORKLOADS[4]
    layer = workload_inputs(4, device=dev)
    pre_args = (layer.x, layer.Bm, layer.Cm, layer.dt, layer.A, layer.lam, layer.theta, layer.D)
    _, dstate, (dcB, dcX) = m3.scan_fwd(*pre_args, chunk=wd["chunk"])
    # The same MIMO prefill (rank 4, 8192 slices), timed: a few more calls
    # writing the same state (the decode steps start from it).
    mimo_out = (torch.empty_like(layer.x), dstate, dcB, dcX)
    mimo_ws = torch.empty(max(m3.workspace_bytes(m3.scan_dims(layer.x, layer.Bm, wd["chunk"], layer.A)), 1),
                          dtype=torch.uint8, device=dev)
    n_mimo = 3
    mimo_ev = [torch.cuda.Event(enable_timing=True) for _ in range(n_mimo + 1)]
    torch.cuda.synchronize()
    mimo_ev[0].record(stream)
    for i in range(n_mimo):
        m3.scan_fwd(*pre_args, chunk=wd["chunk"], out=mimo_out, workspace=mimo_ws)
        mimo_ev[i + 1].record(stream)
    torch.cuda.synchronize()
    mimo_ms = float(np.mean([mimo_ev[i].elapsed_time(mimo_ev[i + 1]) for i in range(n_mimo)]))
    Bm_, Lm_, Hm_, Rm_, Pm_ = layer.x.shape
    Nm_ = layer.Bm.shape[-1]
    del mimo_out, mimo_ws, pre_args
    del layer.x, layer.Bm, layer.Cm, layer.theta, layer.lam, layer.dt  # free the prefill inputs
    torch.cuda.synchronize()
    n_step_inputs = max(1, min(args.steps + args.warmup, wd["steps"]))
    step_in = []
    for s in range(n_step_inputs):
        step_in.append(make_step_inputs(_LayerView(layer, wd), s, device=dev))
    yd = torch.empty_like(step_in[0].x)

    def dstep(i):
        st = step_in[i % n_step_inputs]
        m3.step(dstate, (dcB, dcX), st.x, st.Bm, st.Cm, st.dt, layer.A, st.lam, st.theta, layer.D,
                y=yd)

    # ---------------- timed loop ----------------
    for i in range(args.warmup):
        scan(i)
        dstep(i)
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    for i in range(args.steps):
        ev[i][0].record(stream)
        scan(i)
        ev[i][1].record(stream)
        dstep(args.warmup + i)
        ev[i][2].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    scan_ms = np.array([e[0].elapsed_time(e[1]) for e in ev])
    step_ms = np.array([e[1].elapsed_time(e[2]) for e in ev])
    tot_ms = np.array([e[0].elapsed_time(e[2]) for e in ev])

    # ---------------- output gate y o SiLU(z) (after the timed loop) ----------------
    zs = [make_gate_input(c.x, i) for i, c in enumerate(copies)]
    zd = [make_gate_input(st.x, 100 + i) for i, st in enumerate(step_in[:4])]

    def gscan(i):
        c = copies[i % len(copies)]
        m3.scan_fwd(c.x, c.Bm, c.Cm, c.dt, c.A, c.lam, c.theta, c.D, chunk=Qp, out=out,
                    workspace=ws, z=zs[i % len(zs)])

    def unfused(i):   # ungated scan, then the gate as a separate elementwise pass
        scan(i)
        out[0].mul_(torch.nn.functional.silu(zs[i % len(zs)]))

    def gstep(i):
        st = step_in[i % n_step_inputs]
        m3.step(dstate, (dcB, dcX), st.x, st.Bm, st.Cm, st.dt, layer.A, st.lam, st.theta, layer.D,
                y=yd, z=zd[i % len(zd)])

    def timed(pre, dec, n):
        # the timed loop's pattern (a prefill, then a decode step), so that
        # the figures compare with its ungated ones call for call
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

    def pscan(i):   # per-head frequencies omega [H, N/2]: the kernels form dt * omega
        c = copies[i % len(copies)]
        m3.scan_fwd(c.x, c.Bm, c.Cm, c.dt, c.A, c.lam, c.omega, c.D, chunk=Qp, out=out,
                    workspace=ws)

    n_gate = max(10, min(args.steps, 100))
    g_scan_ms, g_step_ms = timed(gscan, gstep, n_gate)
    g_unfused_ms, _ = timed(unfused, dstep, n_gate)
    p_scan_ms, _ = timed(pscan, dstep, n_gate)

    tokens = Bp * Lp
    prefill_tok_s = tokens / (scan_ms.mean() * 1e-3)
    dec_us = step_ms.mean() * 1e3

    # rooflines (algorithmic bytes / FLOPs per launch, see roofline.py)
    Bd, Hd, Rd, Pd = step_in[0].x.shape
    Nd = step_in[0].Bm.shape[-1]
    dec_bytes = Bd * Hd * roofline.decode_bytes_per_slice(Nd, Pd, Rd, 2)
    dec_gbs = dec_bytes / (step_ms.mean() * 1e-3) / 1e9
    pre_bytes = roofline.prefill_bytes(Bp, Lp, Hp, Np, Pp, Rp, 2)
    pre_flops = Bp * Hp * roofline.chunked_flops(Lp, Np, Pp, Rp, Qp)
    pre_gbs = pre_bytes / (scan_ms.mean() * 1e-3) / 1e9
    pre_tfs = pre_flops / (scan_ms.mean() * 1e-3) / 1e12
    peak_gbs = roofline.HBM_BYTES_PER_S / 1e9

    result = {
        "metric": METRIC,
        "value": round(prefill_tok_s, 1),
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
            "workload": (f"prefill B={Bp} L={Lp} H={Hp} P={Pp} N={Np} R={Rp} chunk={Qp} bf16 "
                         f"+ decode step B={Bd} H={Hd} P={Pd} N={Nd} R={Rd} fp32 state"),
            "prefill": {"batch": Bp, "seqlen": Lp, "nheads": Hp, "headdim": Pp, "dstate": Np,
                        "rank": Rp, "chunk": Qp, "io": "bf16"},
            "decode": {"batch": Bd, "nheads": Hd, "headdim": Pd, "dstate": Nd, "rank": Rd,
                       "io": "bf16", "state": "fp32"},
        },
        "prefill_ms": round(float(scan_ms.mean()), 5),
        "prefill_ms_p10_p90": [round(float(np.percentile(scan_ms, 10)), 5),
                               round(float(np.percentile(scan_ms, 90)), 5)],
        "decode_us_per_step": round(dec_us, 3),
        "decode_us_p10_p90": [round(float(np.percentile(step_ms, 10)) * 1e3, 3),
                              round(float(np.percentile(step_ms, 90)) * 1e3, 3)],
        "roofline": {
            "kernel": "k_step (m3_step, one launch per step)",
            "bound": "hbm", "achieved": round(dec_gbs, 1), "peak": peak_gbs, "unit": "GB/s",
            "frac": round(dec_gbs / peak_gbs, 4), "traffic": measured_traffic("k_step"),
            "bytes_per_launch": dec_bytes,
        },
        "roofline_prefill": {
            "kernel": "m3_scan_fwd (all launches of one scan)",
            "bound": "hbm", "achieved": round(pre_gbs, 1), "peak": peak_gbs, "unit": "GB/s",
            "frac": round(pre_gbs / peak_gbs, 4), "traffic": measured_traffic("k_scan_fused_siso"),
            "bytes_per_launch": pre_bytes,
            "mfma_tflops": round(pre_tfs, 2),
            "mfma_frac": round(pre_tfs * 1e12 / roofline.MFMA_BF16_FLOPS, 4),
        },
        "gate": gate_figures(g_scan_ms, g_unfused_ms, g_step_ms, float(scan_ms.mean()),
                             float(step_ms.mean()), tokens, pre_bytes,
                             Bp * Lp * Hp * Rp * Pp * 2, dec_bytes, Bd * Hd * Rd * Pd * 2, peak_gbs),
        "theta_per_head": per_head_figures(p_scan_ms, float(scan_ms.mean()), tokens,
                                           pre_bytes - Bp * Lp * Hp * (Np // 2) * 4 + Hp * (Np // 2) * 4,
                                           peak_gbs),
        "roofline_prefill_mimo": mimo_roofline(Bm_, Lm_, Hm_, Nm_, Pm_, Rm_, wd["chunk"], mimo_ms,
                                               roofline, peak_gbs),
        "wall_s_timed_loop": round(wall, 3),
    }
    if not args.no_cpu:
        result["cpu_baseline"] = cpu_baseline(base, layer, step_in, wp, wd)
    print(json.dumps(result), flush=True)


def gate_figures(scan_ms, unfused_ms, step_ms, base_scan_ms, base_step_ms, tokens, pre_bytes,
                 z_bytes, dec_bytes, zd_bytes, peak_gbs):
    """The fused output gate y o SiLU(z) on the same two workloads, timed in
    the timed loop's pattern: the gated prefill (algorithmic bytes plus z)
    against the ungated one and against the ungated one followed by the gate
    as a separate elementwise pass (torch), the gated decode step against the
    ungated one (the ungated figures are the timed loop's)."""
    pre_gbs = (pre_bytes + z_bytes) / (scan_ms * 1e-3) / 1e9
    dec_gbs = (dec_bytes + zd_bytes) / (step_ms * 1e-3) / 1e9
    return {
        "prefill_ms": round(scan_ms, 5), "prefill_tokens_per_s": round(tokens / (scan_ms * 1e-3), 1),
        "prefill_bound": "hbm", "prefill_achieved_gbs": round(pre_gbs, 1),
        "prefill_frac": round(pre_gbs / peak_gbs, 4), "prefill_bytes_per_launch": pre_bytes + z_bytes,
        "ungated_prefill_ms": round(base_scan_ms, 5), "unfused_prefill_ms": round(unfused_ms, 5),
        "decode_us_per_step": round(step_ms * 1e3, 3),
        "ungated_decode_us_per_step": round(base_step_ms * 1e3, 3), "decode_bound": "hbm",
        "decode_achieved_gbs": round(dec_gbs, 1), "decode_frac": round(dec_gbs / peak_gbs, 4),
        "decode_bytes_per_launch": dec_bytes + zd_bytes,
    }


def per_head_figures(ms, theta_ms, tokens, nbytes, peak_gbs):
    """The SISO prefill with per-head rotary frequencies omega (angles dt *
    omega formed in the kernels, M3_THETA_PER_HEAD) in the timed loop's
    pattern, against the timed loop's per-token-angle prefill; bytes without
    the per-token angle array."""
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"prefill_ms": round(ms, 5), "prefill_tokens_per_s": round(tokens / (ms * 1e-3), 1),
            "per_token_theta_prefill_ms": round(theta_ms, 5), "bound": "hbm",
            "achieved_gbs": round(gbs, 1), "frac": round(gbs / peak_gbs, 4),
            "bytes_per_launch": nbytes}


def mimo_roofline(B, L, H, N, P, R, Q, ms, roofline, peak_gbs):
    """HBM and MFMA rates of the rank-4 prefill that builds the decode state
    (mean over a few calls; not part of the timed step)."""
    nbytes = roofline.prefill_bytes(B, L, H, N, P, R, 2)
    flops = B * H * roofline.chunked_flops(L, N, P, R, Q)
    gbs = nbytes / (ms * 1e-3) / 1e9
    tfs = flops / (ms * 1e-3) / 1e12
    return {
        "kernel": "m3_scan_fwd (warp-specialised kernel, one workgroup per slice)",
        "workload": f"prefill B={B} L={L} H={H} P={P} N={N} R={R} chunk={Q} bf16",
        "ms": round(ms, 4), "tokens_per_s": round(B * L / (ms * 1e-3), 1),
        "bound": "hbm", "achieved": round(gbs, 1), "peak": peak_gbs, "unit": "GB/s",
        "frac": round(gbs / peak_gbs, 4), "traffic": measured_traffic("k_scan_ws_mimo"),
        "bytes_per_launch": nbytes,
        "mfma_tflops": round(tfs, 2), "mfma_frac": round(tfs * 1e12 / roofline.MFMA_BF16_FLOPS, 4),
    }


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


def cpu_baseline(base, layer, step_in, wp, wd):
    """The fp64 oracle on the host: all 64 slices of the whole prefill batch
    (tokens/s), and one decode step on 64 of the 8192 slices (scaled to the
    whole batch)."""
    import numpy as np
    import oracle
    sl = [(b, h) for b in range(wp["batch"]) for h in range(wp["nheads"])]
    Ls = wp["seqlen"]
    ref = oracle.slices_of_scan(base.x, base.Bm, base.Cm, base.dt, base.A, base.lam, base.theta,
                                base.D, sl, 0, Ls)
    t0 = time.perf_counter()
    _, used = oracle.scan(**ref, return_threads=True)
    dt = time.perf_counter() - t0
    tok_s = wp["batch"] * Ls / dt
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
    dec_us = ddt * (wd["batch"] * wd["nheads"] / S) * 1e6
    return {"value": round(tok_s, 1), "unit": "tokens/s", "cores": int(used), "kind": "oracle",
            "sample": (f"prefill: all {len(sl)} (batch, head) slices of the SISO bf16 batch, "
                       f"first {Ls} of {wp['seqlen']} tokens, fp64, {dt:.2f} s; decode: one step "
                       f"on {S} of {wd['batch'] * wd['nheads']} slices x {reps} reps, scaled"),
            "decode_us_per_step": round(dec_us, 1)}


if __name__ == "__main__":
    main()
