// C-ABI front end of libm3: argument validation on the host (before any HIP
// call), workspace layout, dispatch to the shape-specialised kernels.
#include <limits.h>

#include <algorithm>
#include <atomic>
#include <vector>

#include "m3.h"
#include "m3_internal.h"

namespace m3 {

static thread_local int g_last_hip_error = 0;
// bound of the single-pass kernels' look-back waits (m3_set_wait_limit)
static std::atomic<uint32_t> g_spin_max{kSpinMaxDefault};

static size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }
static_assert(kCtlBytes == M3_CTL_BYTES, "control block size as documented");

ScanWorkspaceLayout scan_workspace_layout(int64_t BH, int64_t nchunks, int64_t N, int64_t P,
                                          int io_bytes, int acc_bytes, bool fused) {
    ScanWorkspaceLayout w = {};
    const size_t per = (size_t)BH * (size_t)nchunks;
    const size_t tot_bytes = per * (size_t)(N / 2 + 1) * (size_t)acc_bytes;
    const size_t state_bytes = per * (size_t)(N * P) * sizeof(float);
    // the control block of the single-pass paths comes first on every path,
    // so that a workspace shared by calls of either kind keeps it
    if (!fused) {
        w.off_M = kCtlBytes;
        w.off_Sin = align_up(w.off_M + state_bytes, 256);
        w.off_tot = align_up(w.off_Sin + per * (size_t)(N * P) * (size_t)io_bytes, 256);
        w.total = align_up(w.off_tot + tot_bytes, 256);
    } else {
        w.off_ctl = 0;
        w.off_flags = kCtlBytes;
        w.off_tot = align_up(w.off_flags + per * sizeof(uint32_t), 256);
        w.off_agg = align_up(w.off_tot + tot_bytes, 256);
        w.off_inc = align_up(w.off_agg + state_bytes, 256);
        w.total = align_up(w.off_inc + state_bytes, 256);
    }
    return w;
}

static bool aligned16(const void *p) { return p == nullptr || ((uintptr_t)p & 15u) == 0; }
static bool aligned4(const void *p) { return p == nullptr || ((uintptr_t)p & 3u) == 0; }

// Checks a block prologue and converts it (pro may be null: none).
static m3_status check_prologue(const m3_prologue *pro, bool have_z, int64_t headdim, Prologue *out) {
    *out = Prologue{};
    if (!pro) return M3_OK;
    if (pro->bc_norm && !(pro->eps > 0.f)) return M3_ERR_SHAPE;   // (also NaN)
    if (!pro->bc_norm && (pro->norm_B || pro->norm_C)) return M3_ERR_SHAPE;
    if (pro->out_norm < M3_OUT_NORM_NONE || pro->out_norm > M3_OUT_NORM_POST_GATE) return M3_ERR_SHAPE;
    if (pro->out_norm) {
        const int32_t gs = pro->out_group;
        if (!(pro->out_eps > 0.f) || gs < 8 || gs > headdim || (gs & (gs - 1))) return M3_ERR_SHAPE;
    } else if (pro->out_gain) {
        return M3_ERR_SHAPE;
    }
    if (pro->w_z && !have_z) return M3_ERR_NULL;
    const void *tabs[] = {pro->norm_B, pro->norm_C, pro->bias_B, pro->bias_C, pro->w_x, pro->w_z,
                          pro->out_gain};
    for (const void *p : tabs)
        if (!aligned16(p)) return M3_ERR_ALIGN;
    out->on = 1;
    out->bcnorm = pro->bc_norm ? 1 : 0;
    out->eps = pro->eps;
    out->gB = pro->norm_B; out->gC = pro->norm_C;
    out->bB = pro->bias_B; out->bC = pro->bias_C;
    out->wx = pro->w_x; out->wz = pro->w_z;
    out->onorm = pro->out_norm;
    out->ogroup = pro->out_norm ? pro->out_group : 0;
    out->oeps = pro->out_eps;
    out->og = pro->out_gain;
    return M3_OK;
}

static int io_bytes_of(int32_t io) { return io == M3_F32 ? 4 : io == M3_BF16 ? 2 : 0; }

// Sizes shared by both entry points.  Limits keep every element offset and
// the 1-D grid of one workgroup per (slice, chunk) inside 31/63-bit ranges.
static m3_status check_dims_common(const m3_dims *d) {
    if (!d) return M3_ERR_NULL;
    if (d->io != M3_F32 && d->io != M3_BF16) return M3_ERR_DTYPE;
    if (d->flags & ~(M3_SCAN_SPLIT | M3_SCAN_PER_CHUNK | M3_THETA_PER_HEAD)) return M3_ERR_SHAPE;
    if (d->batch < 1 || d->nheads < 1 || d->headdim < 1 || d->dstate < 2 || d->rank < 1)
        return M3_ERR_SHAPE;
    if (d->dstate % 2) return M3_ERR_SHAPE;
    if (d->batch > INT_MAX || d->nheads > INT_MAX || d->batch * d->nheads > INT_MAX / 16)
        return M3_ERR_SHAPE;
    return M3_OK;
}

}  // namespace m3

using namespace m3;

extern "C" const char *m3_status_string(m3_status s) {
    switch (s) {
    case M3_OK: return "ok";
    case M3_ERR_NULL: return "a required pointer is NULL";
    case M3_ERR_SHAPE: return "a size is out of range or inconsistent";
    case M3_ERR_DTYPE: return "unknown io dtype";
    case M3_ERR_UNSUPPORTED: return "no kernel is built for this shape";
    case M3_ERR_ALIGN: return "a pointer is misaligned";
    case M3_ERR_WORKSPACE: return "workspace missing or too small";
    case M3_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

extern "C" int m3_last_hip_error(void) { return g_last_hip_error; }

static m3_status check_scan_dims(const m3_dims *d, ScanImpl *impl, int64_t *nchunks) {
    m3_status s = check_dims_common(d);
    if (s != M3_OK) return s;
    if (d->seqlen < 0 || d->chunk < 1 || d->seg_chunks < 0) return M3_ERR_SHAPE;
    // element offsets of the largest tensors must fit in int64 comfortably
    const int64_t per_tok = d->nheads * d->rank * (d->dstate > d->headdim ? d->dstate : d->headdim);
    if (d->seqlen > (INT64_MAX / 4) / (d->batch * per_tok)) return M3_ERR_SHAPE;
    const int64_t nc = (d->seqlen + d->chunk - 1) / d->chunk;
    if (d->batch * d->nheads * nc > (int64_t)INT_MAX) return M3_ERR_SHAPE;
    *impl = find_scan_impl(d->io, d->dstate, d->headdim, d->rank, d->chunk);
    if (!impl->launch) return M3_ERR_UNSUPPORTED;
    // the single-pass kernels serve every shape they are built for, except
    // the empty sequence (handled by the three-kernel path's state kernel)
    // and per-token strides too wide for their 32-bit row offsets (24-bit
    // stride multiplies, a chunk's rows within 2 GiB)
    const int64_t tok_bytes = per_tok * (int64_t)io_bytes_of(d->io);
    const bool narrow = tok_bytes < (INT64_C(1) << 24) && d->chunk * tok_bytes < (INT64_C(1) << 31);
    if (nc > 0 && !(d->flags & M3_SCAN_SPLIT) && narrow) {
        scan_launch_fn f = nullptr;
        scan_launch_fn pc = find_fused_impl(d->io, d->dstate, d->headdim, d->rank, d->chunk);
        if (!(d->flags & M3_SCAN_PER_CHUNK)) f = find_seg_impl(d->io, d->dstate, d->headdim, d->rank, d->chunk);
        if (!f) f = pc;
        if (f) { impl->launch = f; impl->fused = true; impl->per_chunk = pc; }
    }
    *nchunks = nc;
    return M3_OK;
}

extern "C" size_t m3_scan_workspace_bytes(const m3_dims *d) {
    ScanImpl impl;
    int64_t nc = 0;
    if (check_scan_dims(d, &impl, &nc) != M3_OK) return 0;
    return scan_workspace_layout(d->batch * d->nheads, nc, d->dstate, d->headdim,
                                 io_bytes_of(d->io), impl.acc_bytes, impl.fused)
        .total;
}

// Both scan entry points; `gated` requires z (a token array like x).  With
// `dry_run` only the checks run (nothing is launched).
static m3_status scan_fwd(const m3_dims *d, const void *x, const void *B, const void *C,
                          const float *dt, const float *A, const float *lambda,
                          const float *theta, const float *D, bool gated, const void *z,
                          const float *init_state, const void *init_carryB,
                          const void *init_carryX, void *y, float *final_state, void *carryB,
                          void *carryX, void *workspace, size_t workspace_bytes, void *stream,
                          bool dry_run = false, const m3_prologue *pro = nullptr) {
    ScanImpl impl;
    int64_t nc = 0;
    m3_status s = check_scan_dims(d, &impl, &nc);
    if (s != M3_OK) return s;
    Prologue pr;
    s = check_prologue(pro, gated, d->headdim, &pr);
    if (s != M3_OK) return s;
    if (pr.on) {
        // the block prologue runs in the per-chunk kernel (same workspace
        // layout), or, where the segmented kernel's launcher would choose the
        // warp-specialised kernel (one segment per slice), in that kernel
        // built with the prologue: the launcher then hands everything else to
        // the per-chunk kernel with the prologue
        scan_launch_fn f = (d->flags & M3_SCAN_SPLIT) ? nullptr
                                                      : find_fused_pro_impl(d->io, d->dstate, d->headdim,
                                                                            d->rank, d->chunk);
        if (!f) return M3_ERR_UNSUPPORTED;
        if (nc > 0) {
            if (!impl.fused) return M3_ERR_UNSUPPORTED;
            const bool seg = impl.launch != impl.per_chunk &&
                             find_ws_pro_impl(d->io, d->dstate, d->headdim, d->rank, d->chunk) != nullptr;
            if (!seg) impl.launch = f;
            impl.per_chunk = f;
        }
    }
    // token arrays may be NULL only for an empty sequence (empty tensors)
    const bool tok_ok = d->seqlen == 0 || (x && B && C && dt && lambda && theta && y && (z || !gated));
    if (!tok_ok || !A || !D || !final_state || !carryB || !carryX) return M3_ERR_NULL;
    if ((init_carryB == nullptr) != (init_carryX == nullptr)) return M3_ERR_NULL;
    if (!gated || d->seqlen == 0) z = nullptr;
    const void *vec[] = {x, B, C, theta, z, init_state, init_carryB, init_carryX,
                         y, final_state, carryB, carryX, workspace};
    for (const void *p : vec)
        if (!aligned16(p)) return M3_ERR_ALIGN;
    const void *scal[] = {dt, A, lambda, D};
    for (const void *p : scal)
        if (!aligned4(p)) return M3_ERR_ALIGN;
    const ScanWorkspaceLayout wl = scan_workspace_layout(d->batch * d->nheads, nc, d->dstate,
                                                         d->headdim, io_bytes_of(d->io),
                                                         impl.acc_bytes, impl.fused);
    if (nc > 0 && (workspace == nullptr || workspace_bytes < wl.total)) return M3_ERR_WORKSPACE;
    if (dry_run) return M3_OK;

    ScanArgs a;
    a.x = x; a.B = B; a.C = C;
    a.dt = dt; a.A = A; a.lam = lambda; a.theta = theta; a.D = D;
    a.init_state = init_state; a.init_cB = init_carryB; a.init_cX = init_carryX;
    a.y = y; a.z = z; a.final_state = final_state; a.cB = carryB; a.cX = carryX;
    a.theta_ph = (d->flags & M3_THETA_PER_HEAD) ? 1 : 0;
    char *ws = static_cast<char *>(workspace);
    a.M = nullptr; a.Sin = nullptr; a.tot = nullptr;
    a.ctl = nullptr; a.flags = nullptr; a.agg = nullptr; a.inc = nullptr;
    if (nc > 0 && !impl.fused) {
        a.M = reinterpret_cast<float *>(ws + wl.off_M);
        a.Sin = ws + wl.off_Sin;
        a.tot = ws + wl.off_tot;
    } else if (nc > 0) {
        a.ctl = reinterpret_cast<uint32_t *>(ws + wl.off_ctl);
        a.flags = reinterpret_cast<uint32_t *>(ws + wl.off_flags);
        a.tot = ws + wl.off_tot;
        a.agg = reinterpret_cast<float *>(ws + wl.off_agg);
        a.inc = reinterpret_cast<float *>(ws + wl.off_inc);
    }
    a.batch = d->batch; a.L = d->seqlen; a.H = d->nheads; a.nchunks = nc;
    a.a_sb = d->a_stride_b; a.a_st = d->a_stride_t; a.a_sh = d->a_stride_h;
    a.G = d->seg_chunks; a.nseg = 0; a.per_chunk = impl.per_chunk;
    a.spin_max = g_spin_max.load(std::memory_order_relaxed);
    a.pro = pr;
    const hipError_t e = impl.launch(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) {
        g_last_hip_error = (int)e;
        return M3_ERR_HIP;
    }
    return M3_OK;
}

extern "C" m3_status m3_scan_fwd(const m3_dims *d, const void *x, const void *B, const void *C,
                                 const float *dt, const float *A, const float *lambda,
                                 const float *theta, const float *D, const float *init_state,
                                 const void *init_carryB, const void *init_carryX, void *y,
                                 float *final_state, void *carryB, void *carryX, void *workspace,
                                 size_t workspace_bytes, void *stream) {
    return scan_fwd(d, x, B, C, dt, A, lambda, theta, D, false, nullptr, init_state, init_carryB,
                    init_carryX, y, final_state, carryB, carryX, workspace, workspace_bytes, stream);
}

extern "C" m3_status m3_scan_fwd_pro(const m3_dims *d, const m3_prologue *pro, const void *x,
                                     const void *B, const void *C, const float *dt, const float *A,
                                     const float *lambda, const float *theta, const float *D,
                                     const void *z, const float *init_state,
                                     const void *init_carryB, const void *init_carryX, void *y,
                                     float *final_state, void *carryB, void *carryX,
                                     void *workspace, size_t workspace_bytes, void *stream) {
    if (!pro) return M3_ERR_NULL;
    return scan_fwd(d, x, B, C, dt, A, lambda, theta, D, z != nullptr, z, init_state, init_carryB,
                    init_carryX, y, final_state, carryB, carryX, workspace, workspace_bytes, stream,
                    false, pro);
}

extern "C" m3_status m3_scan_fwd_gated(const m3_dims *d, const void *x, const void *B,
                                       const void *C, const float *dt, const float *A,
                                       const float *lambda, const float *theta, const float *D,
                                       const void *z, const float *init_state,
                                       const void *init_carryB, const void *init_carryX, void *y,
                                       float *final_state, void *carryB, void *carryX,
                                       void *workspace, size_t workspace_bytes, void *stream) {
    return scan_fwd(d, x, B, C, dt, A, lambda, theta, D, true, z, init_state, init_carryB,
                    init_carryX, y, final_state, carryB, carryX, workspace, workspace_bytes, stream);
}

// Packed sequences of different lengths: sequence i is tokens cu_seqlens[i]
// .. cu_seqlens[i+1] - 1 of the token axis.  Runs of consecutive sequences of
// equal length go out as one m3_scan_fwd over a batch of them (as far as the
// workspace holds what that batch needs), every other sequence as an
// m3_scan_fwd of its own; the calls run in order on `stream` and share the
// workspace.  Every call's arguments are checked before the first launch.
// ---------------------------------------------------------------------------
// Varlen single launch: every (sequence, head, chunk) item of the packed
// batch in one launch of the per-chunk kernel, from tables the host builds
// out of the offsets and copies into the workspace.
// ---------------------------------------------------------------------------

namespace m3 {
namespace {

struct VarlenPlan {
    scan_launch_fn launch = nullptr;   // null: the single launch does not apply
    int64_t slots = 0, maxn = 0;
    size_t off_flags = 0, off_tot = 0, off_agg = 0, off_inc = 0, off_tab = 0, tab_bytes = 0, total = 0;
};

// Whether one launch serves the packed batch (the per-chunk kernel built for
// the shape, no M3_SCAN_SPLIT and no segment length asked for, every
// sequence non-empty, token rows within
// the kernel's 32-bit offsets, items within its ticket range), and its
// workspace layout.  d and cu_seqlens already validated.
VarlenPlan varlen_plan(const m3_dims *d, const int64_t *cu) {
    VarlenPlan p;
    if ((d->flags & M3_SCAN_SPLIT) || d->seg_chunks > 0 || d->batch < 1) return p;
    scan_launch_fn f = find_fused_var_impl(d->io, d->dstate, d->headdim, d->rank, d->chunk);
    const ScanImpl impl = find_scan_impl(d->io, d->dstate, d->headdim, d->rank, d->chunk);
    if (!f || !impl.launch) return p;
    const int64_t per_tok = d->nheads * d->rank * (d->dstate > d->headdim ? d->dstate : d->headdim);
    const int64_t tok_bytes = per_tok * (int64_t)io_bytes_of(d->io);
    if (!(tok_bytes < (INT64_C(1) << 24) && d->chunk * tok_bytes < (INT64_C(1) << 31))) return p;
    int64_t chunks = 0, maxn = 0;
    for (int64_t s = 0; s < d->batch; ++s) {
        const int64_t len = cu[s + 1] - cu[s];
        if (len <= 0) return p;
        const int64_t n = (len + d->chunk - 1) / d->chunk;
        chunks += n;
        maxn = n > maxn ? n : maxn;
    }
    const int64_t slots = chunks * d->nheads, nsl = d->batch * d->nheads;
    if (slots >= (int64_t)INT_MAX || maxn >= (int64_t)INT_MAX / kGroups) return p;
    const size_t N = d->dstate, P = d->headdim;
    p.launch = f;
    p.slots = slots;
    p.maxn = maxn;
    p.off_flags = kCtlBytes;
    p.off_tot = align_up(p.off_flags + (size_t)slots * 4, 256);
    p.off_agg = align_up(p.off_tot + (size_t)slots * (N / 2 + 1) * (size_t)impl.acc_bytes, 256);
    p.off_inc = align_up(p.off_agg + (size_t)slots * N * P * 4, 256);
    p.off_tab = align_up(p.off_inc + (size_t)slots * N * P * 4, 256);
    p.tab_bytes = (size_t)d->batch * 20 + 4 * ((size_t)(kGroups + 1) + (size_t)kGroups * (maxn + 1) + (size_t)nsl);
    p.total = align_up(p.off_tab + p.tab_bytes, 256);
    return p;
}

// The tables (layout of varlen_plan's table block): first packed token,
// first flag slot (int64) and length (int32) of each sequence; per slice
// group the start of its slice list, the item counts below each chunk level,
// and the slice lists (each group's slices by decreasing chunk count).
void varlen_tables(const m3_dims *d, const int64_t *cu, const VarlenPlan &p, std::vector<char> &buf) {
    const int64_t S = d->batch, H = d->nheads, Q = d->chunk, nsl = S * H, maxn = p.maxn;
    buf.assign(p.tab_bytes, 0);
    int64_t *tok = reinterpret_cast<int64_t *>(buf.data());
    int64_t *slot = tok + S;
    int32_t *len = reinterpret_cast<int32_t *>(slot + S);
    int32_t *gstart = len + S;
    int32_t *grp = gstart + kGroups + 1;
    int32_t *order = grp + kGroups * (maxn + 1);
    std::vector<int32_t> nch(S);
    int64_t base = 0;
    for (int64_t s = 0; s < S; ++s) {
        const int64_t l = cu[s + 1] - cu[s];
        tok[s] = cu[s];
        slot[s] = base;
        len[s] = (int32_t)l;
        nch[s] = (int32_t)((l + Q - 1) / Q);
        base += H * nch[s];
    }
    int32_t at = 0;
    for (int y = 0; y < kGroups; ++y) {
        gstart[y] = at;
        std::vector<int32_t> mine;
        for (int64_t sl = y; sl < nsl; sl += kGroups) mine.push_back((int32_t)sl);
        std::stable_sort(mine.begin(), mine.end(),
                         [&](int32_t a, int32_t b) { return nch[a / H] > nch[b / H]; });
        for (int32_t sl : mine) order[at++] = sl;
        // items below level c: the slices with more than c' chunks, c' < c
        // (a prefix of the list, shrinking as c grows)
        int32_t *gy = grp + y * (maxn + 1);
        gy[0] = 0;
        size_t pre = mine.size();
        for (int64_t c = 0; c < maxn; ++c) {
            while (pre > 0 && nch[mine[pre - 1] / H] <= c) --pre;
            gy[c + 1] = gy[c] + (int32_t)pre;
        }
    }
    gstart[kGroups] = at;
}

}  // namespace
}  // namespace m3

// The single launch of a checked varlen batch (every run's arguments passed
// m3_scan_fwd's checks): tables copied into the workspace, then the kernel.
static m3_status varlen_single(const m3_dims *d, const int64_t *cu, const VarlenPlan &plan,
                               const void *x, const void *B, const void *C, const float *dt,
                               const float *A, const float *lambda, const float *theta,
                               const float *D, const void *z, const float *init_state,
                               const void *init_carryB, const void *init_carryX, void *y,
                               float *final_state, void *carryB, void *carryX, void *workspace,
                               void *stream) {
    static thread_local std::vector<char> tab;
    varlen_tables(d, cu, plan, tab);
    char *ws = static_cast<char *>(workspace);
    const hipStream_t st = static_cast<hipStream_t>(stream);
    // (pageable source: the call returns once the bytes are staged)
    hipError_t e = hipMemcpyAsync(ws + plan.off_tab, tab.data(), plan.tab_bytes, hipMemcpyHostToDevice, st);
    if (e != hipSuccess) {
        g_last_hip_error = (int)e;
        return M3_ERR_HIP;
    }
    ScanArgs a = {};
    a.x = x; a.B = B; a.C = C;
    a.dt = dt; a.A = A; a.lam = lambda; a.theta = theta; a.D = D;
    a.init_state = init_state; a.init_cB = init_carryB; a.init_cX = init_carryX;
    a.y = y; a.z = z; a.final_state = final_state; a.cB = carryB; a.cX = carryX;
    a.theta_ph = (d->flags & M3_THETA_PER_HEAD) ? 1 : 0;
    a.ctl = reinterpret_cast<uint32_t *>(ws);
    a.flags = reinterpret_cast<uint32_t *>(ws + plan.off_flags);
    a.tot = ws + plan.off_tot;
    a.agg = reinterpret_cast<float *>(ws + plan.off_agg);
    a.inc = reinterpret_cast<float *>(ws + plan.off_inc);
    a.batch = d->batch; a.L = d->seqlen; a.H = d->nheads; a.nchunks = plan.maxn;
    a.a_sb = 0; a.a_st = d->a_stride_t; a.a_sh = d->a_stride_h;
    const int64_t S = d->batch;
    const char *tb = ws + plan.off_tab;
    a.vl_tok = reinterpret_cast<const int64_t *>(tb);
    a.vl_slot = a.vl_tok + S;
    a.vl_len = reinterpret_cast<const int32_t *>(a.vl_slot + S);
    a.vl_gstart = a.vl_len + S;
    a.vl_grp = a.vl_gstart + kGroups + 1;
    a.vl_order = a.vl_grp + kGroups * (plan.maxn + 1);
    a.vl_maxn = (int)plan.maxn;
    a.vl_slots = plan.slots;
    a.spin_max = g_spin_max.load(std::memory_order_relaxed);
    e = plan.launch(a, st);
    if (e != hipSuccess) {
        g_last_hip_error = (int)e;
        return M3_ERR_HIP;
    }
    return M3_OK;
}

extern "C" size_t m3_scan_varlen_workspace_bytes(const m3_dims *d, const int64_t *cu_seqlens) {
    if (check_dims_common(d) != M3_OK || !cu_seqlens || d->seqlen < 0 || d->a_stride_b != 0 ||
        cu_seqlens[0] != 0 || cu_seqlens[d->batch] != d->seqlen)
        return 0;
    for (int64_t i = 0; i < d->batch; ++i)
        if (cu_seqlens[i + 1] < cu_seqlens[i]) return 0;
    return varlen_plan(d, cu_seqlens).total;
}

extern "C" m3_status m3_scan_fwd_varlen(const m3_dims *d, const int64_t *cu_seqlens,
                                        const void *x, const void *B, const void *C,
                                        const float *dt, const float *A, const float *lambda,
                                        const float *theta, const float *D, const void *z,
                                        const float *init_state, const void *init_carryB,
                                        const void *init_carryX, void *y, float *final_state,
                                        void *carryB, void *carryX, void *workspace,
                                        size_t workspace_bytes, void *stream) {
    m3_status s = check_dims_common(d);
    if (s != M3_OK) return s;
    if (!cu_seqlens) return M3_ERR_NULL;
    if (d->seqlen < 0 || d->a_stride_b != 0 || cu_seqlens[0] != 0 || cu_seqlens[d->batch] != d->seqlen)
        return M3_ERR_SHAPE;
    for (int64_t i = 0; i < d->batch; ++i)
        if (cu_seqlens[i + 1] < cu_seqlens[i]) return M3_ERR_SHAPE;
    const int64_t H = d->nheads, N = d->dstate, P = d->headdim, R = d->rank;
    const int64_t io = io_bytes_of(d->io);
    const bool ph = (d->flags & M3_THETA_PER_HEAD) != 0;
    auto off = [](const void *p, int64_t bytes) -> const void * {
        return p ? static_cast<const char *>(p) + bytes : nullptr;
    };
    // Consecutive sequences of equal length lie in the packed arrays exactly
    // as a batch of them would: such runs go out as one launch, as long as
    // the workspace holds what that batch needs.
    auto run_end = [&](int64_t i) -> int64_t {
        const int64_t len = cu_seqlens[i + 1] - cu_seqlens[i];
        int64_t j = i + 1;
        for (; j < d->batch && cu_seqlens[j + 1] - cu_seqlens[j] == len; ++j) {
            m3_dims dj = *d;
            dj.batch = j - i + 1;
            dj.seqlen = len;
            dj.a_stride_b = len * d->a_stride_t;
            // (0: the batched dims are invalid, e.g. too many chunk items,
            // while the sequences alone may be fine: stop the run)
            const size_t need = m3_scan_workspace_bytes(&dj);
            if ((need == 0 && len > 0) || need > workspace_bytes) break;
        }
        return j;
    };
    for (int pass = 0; pass < 2; ++pass) {   // 0: every call checked, 1: launched
        if (pass == 1) {   // one launch for the whole batch, where it applies and fits
            const VarlenPlan plan = varlen_plan(d, cu_seqlens);
            if (plan.launch && workspace_bytes >= plan.total)
                return varlen_single(d, cu_seqlens, plan, x, B, C, dt, A, lambda, theta, D, z,
                                     init_state, init_carryB, init_carryX, y, final_state, carryB,
                                     carryX, workspace, stream);
        }
        for (int64_t i = 0, j = 0; i < d->batch; i = j) {
            j = run_end(i);
            const int64_t t0 = cu_seqlens[i], len = cu_seqlens[i + 1] - t0;
            m3_dims di = *d;
            di.batch = j - i;
            di.seqlen = len;
            di.a_stride_b = len * d->a_stride_t;
            const int64_t tx = t0 * H * R * P * io, tb = t0 * H * R * N * io, ts = t0 * H * 4;
            s = scan_fwd(&di, off(x, tx), off(B, tb), off(C, tb), static_cast<const float *>(off(dt, ts)),
                         A ? A + t0 * d->a_stride_t : nullptr, static_cast<const float *>(off(lambda, ts)),
                         ph ? theta : static_cast<const float *>(off(theta, t0 * H * (N / 2) * 4)), D,
                         z != nullptr, off(z, tx),
                         static_cast<const float *>(off(init_state, i * H * N * P * 4)),
                         off(init_carryB, i * H * R * N * io), off(init_carryX, i * H * R * P * io),
                         const_cast<void *>(off(y, tx)),
                         static_cast<float *>(const_cast<void *>(off(final_state, i * H * N * P * 4))),
                         const_cast<void *>(off(carryB, i * H * R * N * io)),
                         const_cast<void *>(off(carryX, i * H * R * P * io)), workspace, workspace_bytes,
                         stream, pass == 0);
            if (s != M3_OK) return s;
        }
    }
    return M3_OK;
}

static m3_status step(const m3_dims *d, float *state, void *carryB, void *carryX,
                      const void *x_t, const void *B_t, const void *C_t, const float *dt_t,
                      const float *A, const float *lambda_t, const float *theta_t, const float *D,
                      bool gated, const void *z_t, void *y_t, void *stream,
                      const m3_prologue *pro = nullptr) {
    m3_status s = check_dims_common(d);
    if (s != M3_OK) return s;
    Prologue pr;
    s = check_prologue(pro, gated, d->headdim, &pr);
    if (s != M3_OK) return s;
    step_launch_fn fn = pr.on ? find_step_pro_impl(d->io, d->dstate, d->headdim, d->rank)
                              : find_step_impl(d->io, d->dstate, d->headdim, d->rank);
    if (!fn) return M3_ERR_UNSUPPORTED;
    if (!state || !carryB || !carryX || !x_t || !B_t || !C_t || !dt_t || !A || !lambda_t ||
        !theta_t || !D || !y_t || (gated && !z_t))
        return M3_ERR_NULL;
    if (!gated) z_t = nullptr;
    const void *vec[] = {state, carryB, carryX, x_t, B_t, C_t, theta_t, z_t, y_t};
    for (const void *p : vec)
        if (!aligned16(p)) return M3_ERR_ALIGN;
    const void *scal[] = {dt_t, A, lambda_t, D};
    for (const void *p : scal)
        if (!aligned4(p)) return M3_ERR_ALIGN;
    StepArgs a;
    a.state = state; a.cB = carryB; a.cX = carryX;
    a.x = x_t; a.B = B_t; a.C = C_t;
    a.dt = dt_t; a.A = A; a.lam = lambda_t; a.theta = theta_t; a.D = D;
    a.y = y_t; a.z = z_t;
    a.theta_ph = (d->flags & M3_THETA_PER_HEAD) ? 1 : 0;
    a.batch = d->batch; a.H = d->nheads;
    a.a_sb = d->a_stride_b; a.a_sh = d->a_stride_h;
    a.pro = pr;
    const hipError_t e = fn(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) {
        g_last_hip_error = (int)e;
        return M3_ERR_HIP;
    }
    return M3_OK;
}

extern "C" m3_status m3_step(const m3_dims *d, float *state, void *carryB, void *carryX,
                             const void *x_t, const void *B_t, const void *C_t,
                             const float *dt_t, const float *A, const float *lambda_t,
                             const float *theta_t, const float *D, void *y_t, void *stream) {
    return step(d, state, carryB, carryX, x_t, B_t, C_t, dt_t, A, lambda_t, theta_t, D, false,
                nullptr, y_t, stream);
}

extern "C" m3_status m3_step_pro(const m3_dims *d, const m3_prologue *pro, float *state,
                                 void *carryB, void *carryX, const void *x_t, const void *B_t,
                                 const void *C_t, const float *dt_t, const float *A,
                                 const float *lambda_t, const float *theta_t, const float *D,
                                 const void *z_t, void *y_t, void *stream) {
    if (!pro) return M3_ERR_NULL;
    return step(d, state, carryB, carryX, x_t, B_t, C_t, dt_t, A, lambda_t, theta_t, D,
                z_t != nullptr, z_t, y_t, stream, pro);
}

extern "C" m3_status m3_step_gated(const m3_dims *d, float *state, void *carryB, void *carryX,
                                   const void *x_t, const void *B_t, const void *C_t,
                                   const float *dt_t, const float *A, const float *lambda_t,
                                   const float *theta_t, const float *D, const void *z_t,
                                   void *y_t, void *stream) {
    return step(d, state, carryB, carryX, x_t, B_t, C_t, dt_t, A, lambda_t, theta_t, D, true, z_t,
                y_t, stream);
}

// ---------------------------------------------------------------------------
// Backward scan
// ---------------------------------------------------------------------------

static m3_status check_bwd_dims(const m3_dims *d, bwd_launch_fn *fn, int64_t *nchunks) {
    m3_status s = check_dims_common(d);
    if (s != M3_OK) return s;
    if (d->seqlen < 0 || d->chunk < 1 || d->seg_chunks < 0) return M3_ERR_SHAPE;
    const int64_t per_tok = d->nheads * d->rank * (d->dstate > d->headdim ? d->dstate : d->headdim);
    if (d->seqlen > (INT64_MAX / 4) / (d->batch * per_tok)) return M3_ERR_SHAPE;
    const int64_t nc = (d->seqlen + d->chunk - 1) / d->chunk;
    if (d->batch * d->nheads * nc > (int64_t)INT_MAX) return M3_ERR_SHAPE;
    if (d->flags & M3_THETA_PER_HEAD) return M3_ERR_UNSUPPORTED;
    // A per head (summed gradient) or per token (gradient per token)
    if (!(d->a_stride_t != 0 || d->a_stride_b == 0)) return M3_ERR_UNSUPPORTED;
    *fn = find_bwd_impl(d->io, d->dstate, d->headdim, d->rank, d->chunk);
    if (!*fn) return M3_ERR_UNSUPPORTED;
    *nchunks = nc;
    return M3_OK;
}

extern "C" size_t m3_scan_bwd_workspace_bytes(const m3_dims *d) {
    bwd_launch_fn fn;
    int64_t nc = 0;
    if (check_bwd_dims(d, &fn, &nc) != M3_OK) return 0;
    return bwd_workspace_layout(d->batch * d->nheads, nc, d->dstate, d->headdim).total;
}

extern "C" m3_status m3_scan_bwd(const m3_dims *d, const void *x, const void *B, const void *C,
                                 const float *dt, const float *A, const float *lambda,
                                 const float *theta, const float *D, const float *init_state,
                                 const void *dy, const float *dfinal_state, void *dx, void *dB,
                                 void *dC, float *ddt, float *dA, float *dlambda, float *dtheta,
                                 float *dD, float *dinit_state, void *workspace,
                                 size_t workspace_bytes, void *stream) {
    bwd_launch_fn fn;
    int64_t nc = 0;
    m3_status s = check_bwd_dims(d, &fn, &nc);
    if (s != M3_OK) return s;
    const bool tok_ok = d->seqlen == 0 || (x && B && C && dt && lambda && theta && dy && dx && dB &&
                                           dC && ddt && dlambda && dtheta);
    if (!tok_ok || !A || !D || !dA || !dD) return M3_ERR_NULL;
    const void *vec[] = {x, B, C, dy, dx, dB, dC, init_state, dfinal_state, dinit_state, workspace};
    for (const void *p : vec)
        if (!aligned16(p)) return M3_ERR_ALIGN;
    const void *scal[] = {dt, A, lambda, theta, D, ddt, dA, dlambda, dtheta, dD};
    for (const void *p : scal)
        if (!aligned4(p)) return M3_ERR_ALIGN;
    const BwdWorkspaceLayout wl = bwd_workspace_layout(d->batch * d->nheads, nc, d->dstate, d->headdim);
    if (workspace == nullptr || workspace_bytes < wl.total) return M3_ERR_WORKSPACE;
    BwdArgs a;
    a.x = x; a.B = B; a.C = C; a.dy = dy;
    a.dt = dt; a.A = A; a.lam = lambda; a.theta = theta; a.D = D;
    a.init_state = init_state; a.dfinal = dfinal_state;
    a.dx = dx; a.dB = dB; a.dC = dC;
    a.ddt = ddt; a.dA = dA; a.dlam = dlambda; a.dtheta = dtheta; a.dD = dD; a.dinit = dinit_state;
    a.dA_per_token = d->a_stride_t != 0 ? 1 : 0;
    char *ws = static_cast<char *>(workspace);
    a.Af = reinterpret_cast<float *>(ws + wl.off_Af);
    a.Mb = reinterpret_cast<float *>(ws + wl.off_Mb);
    a.Sst = reinterpret_cast<float *>(ws + wl.off_Sst);
    a.Ust = reinterpret_cast<float *>(ws + wl.off_Ust);
    a.tot = reinterpret_cast<float *>(ws + wl.off_tot);
    a.pst = reinterpret_cast<float *>(ws + wl.off_pst);
    a.dsig = reinterpret_cast<float *>(ws + wl.off_dsig);
    a.dApart = reinterpret_cast<float *>(ws + wl.off_dA);
    a.dDpart = reinterpret_cast<float *>(ws + wl.off_dD);
    a.batch = d->batch; a.L = d->seqlen; a.H = d->nheads; a.nchunks = nc;
    a.a_sb = d->a_stride_b; a.a_st = d->a_stride_t; a.a_sh = d->a_stride_h;
    const hipError_t e = fn(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) {
        g_last_hip_error = (int)e;
        return M3_ERR_HIP;
    }
    return M3_OK;
}

extern "C" void m3_set_wait_limit(uint32_t polls) {
    g_spin_max.store(polls ? polls : kSpinMaxDefault, std::memory_order_relaxed);
}

// The last finished single-pass call's timeout count from the control block.
static m3_status read_timeouts(const void *workspace, uint32_t *timeouts, void *stream) {
    // the control words up to group 0's ticket counter: the last finished
    // call ran with epoch (group 0's epoch - 1) and counted its timeouts in
    // that epoch's word (a call without look-back zeroes both words)
    const char *ctl = static_cast<const char *>(workspace);
    uint32_t w[kGroupStride + 2] = {};
    const hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e = hipMemcpyAsync(w, ctl, sizeof(w), hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) {
        g_last_hip_error = (int)e;
        return M3_ERR_HIP;
    }
    const uint32_t last_epoch = w[kGroupStride + 1] - 1u;
    *timeouts = w[(last_epoch & 1u) ? kCtlTimeouts1 : kCtlTimeouts0];
    return M3_OK;
}

extern "C" m3_status m3_scan_check(const m3_dims *d, const void *workspace, size_t workspace_bytes,
                                   uint32_t *timeouts, void *stream) {
    ScanImpl impl;
    int64_t nc = 0;
    m3_status s = check_scan_dims(d, &impl, &nc);
    if (s != M3_OK) return s;
    if (!timeouts) return M3_ERR_NULL;
    if (nc == 0 || !impl.fused) {   // the three-kernel path and the empty scan never wait
        *timeouts = 0;
        return M3_OK;
    }
    const ScanWorkspaceLayout wl = scan_workspace_layout(d->batch * d->nheads, nc, d->dstate,
                                                         d->headdim, io_bytes_of(d->io),
                                                         impl.acc_bytes, impl.fused);
    if (!workspace || workspace_bytes < wl.total) return M3_ERR_WORKSPACE;
    if (!aligned16(workspace)) return M3_ERR_ALIGN;
    return read_timeouts(workspace, timeouts, stream);
}

extern "C" m3_status m3_scan_varlen_check(const m3_dims *d, const int64_t *cu_seqlens,
                                          const void *workspace, size_t workspace_bytes,
                                          uint32_t *timeouts, void *stream) {
    m3_status s = check_dims_common(d);
    if (s != M3_OK) return s;
    if (!cu_seqlens || !timeouts) return M3_ERR_NULL;
    if (d->seqlen < 0 || d->a_stride_b != 0 || cu_seqlens[0] != 0 || cu_seqlens[d->batch] != d->seqlen)
        return M3_ERR_SHAPE;
    for (int64_t i = 0; i < d->batch; ++i)
        if (cu_seqlens[i + 1] < cu_seqlens[i]) return M3_ERR_SHAPE;
    const VarlenPlan plan = varlen_plan(d, cu_seqlens);
    if (plan.launch && workspace_bytes >= plan.total) {   // the call was one launch
        if (!workspace) return M3_ERR_WORKSPACE;
        if (!aligned16(workspace)) return M3_ERR_ALIGN;
        return read_timeouts(workspace, timeouts, stream);
    }
    if (d->batch == 0) {
        *timeouts = 0;
        return M3_OK;
    }
    // else its last launch: the last sequence (batched with the equal-length
    // run it ends, as far as the workspace held it; that run's launch wrote
    // the control block either way)
    const int64_t S = d->batch, len = cu_seqlens[S] - cu_seqlens[S - 1];
    m3_dims dl = *d;
    dl.batch = 1;
    dl.seqlen = len;
    dl.a_stride_b = 0;
    return m3_scan_check(&dl, workspace, workspace_bytes, timeouts, stream);
}


// ---------------------------------------------------------------------------
// Allocation-free prefill: the workspace is a library-owned device array.
// ---------------------------------------------------------------------------

namespace m3 {
namespace {

// Each device the library runs on holds one copy of this array (in the code
// object's zero-initialised data) until the process ends.  Host code never
// uses the array's name as an address: it takes each device's copy from
// hipGetSymbolAddress once per device (scratch_ptr) and passes that pointer.
static __device__ __align__(256) unsigned char scratch[M3_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void *> g_scratch[kMaxDevices];

// Device address of this device's scratch array (looked up once per device,
// with the device current), or null on error (g_last_hip_error set).
void *scratch_ptr() {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess || dev < 0 || dev >= kMaxDevices) {
        g_last_hip_error = (int)(e != hipSuccess ? e : hipErrorInvalidDevice);
        return nullptr;
    }
    void *p = g_scratch[dev].load(std::memory_order_acquire);
    if (p) return p;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr) {
        g_last_hip_error = (int)(e != hipSuccess ? e : hipErrorInvalidSymbol);
        return nullptr;
    }
    g_scratch[dev].store(p, std::memory_order_release);   // (a racing first call stores the same address)
    return p;
}

}  // namespace
}  // namespace m3

extern "C" m3_status m3_scan_fwd_noalloc(const m3_dims *d, const void *x, const void *B,
                                         const void *C, const float *dt, const float *A,
                                         const float *lambda, const float *theta, const float *D,
                                         const float *init_state, const void *init_carryB,
                                         const void *init_carryX, void *y, float *final_state,
                                         void *carryB, void *carryX, void *stream) {
    // every argument check of m3_scan_fwd first (no device call), then the size
    m3_status s = scan_fwd(d, x, B, C, dt, A, lambda, theta, D, false, nullptr, init_state,
                           init_carryB, init_carryX, y, final_state, carryB, carryX,
                           reinterpret_cast<void *>(uintptr_t(256)), M3_SCRATCH_BYTES, stream,
                           /*dry_run=*/true);
    if (s != M3_OK) return s;
    const size_t need = m3_scan_workspace_bytes(d);
    if (need > M3_SCRATCH_BYTES) return M3_ERR_WORKSPACE;
    void *ws = nullptr;
    if (need > 0) {
        ws = scratch_ptr();
        if (!ws) return M3_ERR_HIP;
    }
    return scan_fwd(d, x, B, C, dt, A, lambda, theta, D, false, nullptr, init_state, init_carryB,
                    init_carryX, y, final_state, carryB, carryX, ws, M3_SCRATCH_BYTES, stream);
}
