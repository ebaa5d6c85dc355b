// Internal interface between the C-ABI front end (m3_api.hip) and the
// kernel translation units.  Not installed; include/m3.h is the public API.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace m3 {

// The block prologue fused into the input loads (active when `on`): B and
// C columns RMS-normalised over N when `bcnorm` (gain gB / gC [H][R][N] or
// null for ones), then the biases bB / bC [H][R][N] (null: zeros); x (and z)
// hold X' (Z') [.., H, P] and X = wx o X' (Z = wz o Z'), wx / wz [H][R][P],
// when those pointers are set.
struct Prologue {
    int on, bcnorm;
    float eps;
    const float *gB, *gC, *bB, *bC, *wx, *wz;
    int onorm, ogroup;     // output norm: 0 none, 1 before the gate, 2 after it; channels a group
    float oeps;
    const float *og;       // output norm gain [nheads][rank][headdim] (null: ones)
};

// Arguments of one prefill scan, already validated by the front end.
struct ScanArgs {
    const void *x, *B, *C;
    const float *dt, *A, *lam, *theta, *D;
    const float *init_state;
    const void *init_cB, *init_cX;      // both null or both set
    void *y;
    const void *z;                      // output gate [B,L,H,R,P] (io), or null
    int theta_ph;                       // theta holds per-head frequencies omega [H][N/2]:
                                        // the angle of token t is dt_t * omega
    float *final_state;
    void *cB, *cX;
    // workspace regions (see scan_workspace_layout)
    float *M;        // [BH][nchunks][N][P] fp32  per-chunk state contributions
    void *Sin;       // [BH][nchunks][P][N] io    state entering each chunk
    void *tot;       // [BH][nchunks][1+N/2] acc  chunk log-decay and angle totals
    // single-pass (look-back) scan only
    uint32_t *ctl;   // control block (ticket counters, epoch, timeout counts)
    uint32_t *flags; // [BH][nchunks] 0 / aggregate ready / inclusive state ready
    float *agg;      // [BH][nchunks][N*P] chunk aggregates (owner's lane layout)
    float *inc;      // [BH][nchunks][N*P] inclusive states (same layout)
    int64_t batch, L, H, nchunks;
    int64_t a_sb, a_st, a_sh;
    // varlen single launch (per-chunk kernel, sequences packed along the
    // token axis; batch = sequences, L = packed tokens): item and sequence
    // tables in the workspace (null: a uniform batch)
    const int32_t *vl_grp;     // [kGroups][vl_maxn + 1] items of group y with chunk index < c
    const int32_t *vl_gstart;  // [kGroups + 1] start of group y's slices in vl_order
    const int32_t *vl_order;   // [batch * H] each group's slices by decreasing chunk count
    const int64_t *vl_tok;     // [batch] first packed token of each sequence
    const int64_t *vl_slot;    // [batch] first flag slot of each sequence (H x its chunks)
    const int32_t *vl_len;     // [batch] tokens of each sequence (all > 0)
    int vl_maxn;               // chunks of the longest sequence
    int64_t vl_slots;          // flag slots in all
    // segmented kernel: chunks per segment (0 = chosen at launch), segments
    // per slice (set at launch), and the one-chunk-per-workgroup kernel it
    // hands over to when its own choice would give short chunks several
    // segments per slice (null: none).  With the block prologue (pro.on) the
    // segmented kernel itself never runs: one segment per slice goes to the
    // warp-specialised kernel with the prologue, anything else to per_chunk
    // (then the per-chunk kernel with the prologue).
    int64_t G, nseg;
    hipError_t (*per_chunk)(const ScanArgs &, hipStream_t);
    // polls of a look-back wait before it gives up (counts a timeout in the
    // control block and makes the entering state NaN)
    uint32_t spin_max;
    Prologue pro;
};

struct StepArgs {
    float *state;
    void *cB, *cX;
    const void *x, *B, *C;
    const float *dt, *A, *lam, *theta, *D;
    void *y;
    const void *z;                      // output gate [B,H,R,P] (io), or null
    int theta_ph;                       // theta holds omega [H][N/2] (angle dt * omega)
    int64_t batch, H;
    int64_t a_sb, a_sh;
    Prologue pro;
};

// Arguments of one backward scan (gradients of a loss through y and the
// final state), already validated by the front end.
struct BwdArgs {
    const void *x, *B, *C, *dy;
    const float *dt, *A, *lam, *theta, *D, *init_state, *dfinal;
    void *dx, *dB, *dC;
    float *ddt, *dA, *dlam, *dtheta, *dD, *dinit;
    int dA_per_token;                   // dA [B][L][H] (else [H], summed)
    // workspace regions (bwd_workspace_layout), per (slice, chunk)
    float *Af;      // [N][P] chunk aggregate R(psi_e) sum_j v_j B^_j x_j^T
    float *Mb;      // [N][P] sum_t e^{cum_t} C^_t dy_t^T
    float *tot;     // [1 + N/2] cum_e, psi_e
    float *Sst;     // [N][P] state entering the chunk, stored as bf16 (an MFMA operand; the decay term)
    float *Ust;     // [N][P] R(-psi_e) dJ/dS_out, stored as bf16 (an MFMA operand only)
    float *pst;     // [2][N/2] state terms of dpsi_e and dcum_e (per pair)
    float *dsig;    // [1] dJ/dsigma of the chunk's last token
    float *dApart;  // [1] sum over the chunk of dt dJ/d(dt A)
    float *dDpart;  // [1] sum over the chunk of <x, dy>
    int64_t batch, L, H, nchunks;
    int64_t a_sb, a_st, a_sh;
};
typedef hipError_t (*bwd_launch_fn)(const BwdArgs &, hipStream_t);
// backward kernels for the shape (null: none built)
bwd_launch_fn find_bwd_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q);
struct BwdWorkspaceLayout {
    size_t off_Af, off_Mb, off_tot, off_Sst, off_Ust, off_pst, off_dsig, off_dA, off_dD, total;
};
BwdWorkspaceLayout bwd_workspace_layout(int64_t BH, int64_t nchunks, int64_t N, int64_t P);

// default bound of a look-back wait (polls; ~seconds), then an error count
constexpr uint32_t kSpinMaxDefault = 1u << 22;

typedef hipError_t (*scan_launch_fn)(const ScanArgs &, hipStream_t);
typedef hipError_t (*step_launch_fn)(const StepArgs &, hipStream_t);

struct ScanImpl {
    scan_launch_fn launch;
    int acc_bytes;   // bytes of the prologue scalar type (4: fp32, 8: fp64)
    bool fused;      // a single-pass look-back kernel (else the three-kernel path)
    scan_launch_fn per_chunk;   // one-chunk-per-workgroup kernel for the shape, if built
};

// Kernel lookup by shape; null launch when no kernel is built for it.
ScanImpl find_scan_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q);
step_launch_fn find_step_impl(int io, int64_t N, int64_t P, int64_t R);
scan_launch_fn find_fused_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q);
// the per-chunk kernel over varlen tables (null: not built for the shape)
scan_launch_fn find_fused_var_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q);
scan_launch_fn find_seg_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q);
// warp-specialised kernel for one segment per slice (null: none for the shape)
scan_launch_fn find_ws_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q);
// kernels built with the block prologue (null: none for the shape)
scan_launch_fn find_fused_pro_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q);
scan_launch_fn find_ws_pro_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q);
step_launch_fn find_step_pro_impl(int io, int64_t N, int64_t P, int64_t R);

// Control block of the single-pass scans (the first kCtlBytes of every scan
// workspace; no other path writes there).  Zero before a workspace's first
// use, the scans keep it valid from one call to the next:
//   ctl[kCtlTimeouts0], ctl[kCtlTimeouts1]  look-back waits that gave up in
//                      the call of an even / odd epoch (the call's janitor
//                      zeroes the next epoch's word)
//   ctl[kCtlReady]     epoch + 1 once the running call's flags are cleared
// and per slice group y, 128 bytes apart (so that the groups' atomics do not
// share a cache line), at ctl[kGroupStride * (y + 1)] the group's 64-bit
// ticket counter: ticket, a flags-cleared bit, and the call epoch (the count
// of calls finished on the workspace).  The last call's timeout count is
// the word of epoch (group 0's epoch - 1).
constexpr int kCtlTimeouts0 = 1, kCtlTimeouts1 = 3, kCtlReady = 5;
constexpr int kGroups = 8;           // slice groups (one per XCD)
constexpr int kGroupStride = 32;     // words
constexpr int kCtlWords = kGroupStride * (kGroups + 1);
constexpr size_t kCtlBytes = (kCtlWords * sizeof(uint32_t) + 255) / 256 * 256;

// Byte offsets of the workspace regions for a scan.
struct ScanWorkspaceLayout {
    size_t off_M, off_Sin, off_tot;                 // three-kernel path
    size_t off_ctl, off_flags, off_agg, off_inc;    // single-pass path (off_tot shared)
    size_t total;
};
ScanWorkspaceLayout scan_workspace_layout(int64_t BH, int64_t nchunks, int64_t N,
                                          int64_t P, int io_bytes, int acc_bytes, bool fused);

}  // namespace m3
