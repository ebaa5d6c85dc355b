/*
 * libm3 - the Mamba-3 SSM layer's data-parallel hot path on AMD MI355X
 * (gfx950): the chunked prefill scan and the single-token decode step.
 *
 * The operation (Mamba-3, Sec. 3.1 Prop. "Exponential-Trapezoidal
 * Discretization"; Sec. 3.2 Props. "Complex-to-Real SSM Equivalence" and
 * "Rotary Embedding Equivalence with Exponential-Trapezoidal
 * Discretization"; Sec. 3.3 and App. "MIMO for Mamba-3"), for every batch
 * row b and head h independently, over tokens t = 0 .. L-1:
 *
 *     alpha_t = exp(dt_t A_t)
 *     beta_t  = (1 - lambda_t) dt_t alpha_t
 *     gamma_t = lambda_t dt_t
 *     h_t = alpha_t R_t h_{t-1} + beta_t R_t B_{t-1} X_{t-1}^T + gamma_t B_t X_t^T
 *     Y_t = h_t^T C_t + D X_t
 *
 * h is the N x P fp32 state (N even: N/2 complex entries stored as real
 * parts in rows 0 .. N/2-1 and imaginary parts in rows N/2 .. N-1).  B_t and
 * C_t are N x R, X_t and Y_t are P x R (R = 1 is the SISO layer).  R_t
 * rotates every row pair (i, i + N/2) by the angle theta_t[i]:
 *     [h_i; h_{i+N/2}] <- [[cos, -sin], [sin, cos]] [h_i; h_{i+N/2}].
 * theta is the per-step angle (the paper's Delta_t theta_t[i]); the library
 * does not multiply it by dt, except with the flag M3_THETA_PER_HEAD, where
 * theta holds per-head frequencies omega [nheads][dstate/2] and the angle of
 * token t is dt_t * omega (an fp32 product, formed in the kernels: the
 * per-token angle array is then never read).  D is a per-head skip (Mamba convention; the
 * paper has no skip term).  With no initial state, h_{-1} = 0 and
 * B_{-1} X_{-1}^T = 0 (the unrolled state starts at gamma_0 B_0 x_0).
 *
 * The persistent decode state is (h, B_{t-1}, X_{t-1}): h in the physical
 * (unrotated) frame plus the "carry", the previous token's B and X, which
 * the next step's beta term needs.
 *
 * Memory layouts (all row-major, contiguous, innermost last):
 *     x, y        [batch][seqlen][nheads][rank][headdim]     io dtype
 *     B, C        [batch][seqlen][nheads][rank][dstate]      io dtype
 *     dt, lambda  [batch][seqlen][nheads]                    fp32
 *     theta       [batch][seqlen][nheads][dstate/2]          fp32
 *                 ([nheads][dstate/2] with M3_THETA_PER_HEAD)
 *     A           A[b*a_stride_b + t*a_stride_t + h*a_stride_h]  fp32 (< 0)
 *     D           [nheads]                                   fp32
 *     state       [batch][nheads][dstate][headdim]           fp32
 *     carryB      [batch][nheads][rank][dstate]              io dtype
 *     carryX      [batch][nheads][rank][headdim]             io dtype
 * Decode-step tensors drop the seqlen axis.
 *
 * Ownership and errors: every data pointer is a DEVICE pointer owned by the
 * caller; the library allocates no device memory.  Calls are asynchronous
 * on `stream` (a hipStream_t; NULL is the default stream).  Every argument
 * error is detected on the host before any launch and leaves all outputs
 * untouched; a failed launch returns M3_ERR_HIP.  No call prints, throws or
 * aborts.  Results are deterministic: no floating-point atomics, and the
 * single-pass kernels' look-back forms each entering state by the same fold
 * from the sequence start whatever the timing (bit-equal across runs, given
 * the same device and kernel choice).  Calls on
 * disjoint buffers may run concurrently; the library's only mutable global
 * state is a once-initialised cache of device properties and the look-back
 * wait limit (m3_set_wait_limit).
 *
 * Look-back waits: the single-pass prefill kernels link the chunks (or
 * segments) of a slice by waiting on their predecessors' published states.
 * Every such wait is bounded; one that gives up counts a timeout in the
 * workspace and makes the entering state NaN, so y from that chunk on and the
 * final state of the slice come out NaN.  m3_scan_check reads the count; a
 * non-zero count means y and the final state of that call are invalid.  The
 * work-item order makes a timeout unreachable in normal operation (every
 * predecessor of a waiting workgroup is running or done).
 */
#ifndef M3_H
#define M3_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    M3_OK = 0,
    M3_ERR_NULL = 1,        /* a required pointer is NULL                      */
    M3_ERR_SHAPE = 2,       /* a size is out of range or inconsistent          */
    M3_ERR_DTYPE = 3,       /* unknown io dtype                                */
    M3_ERR_UNSUPPORTED = 4, /* valid, but no kernel is built for this shape    */
    M3_ERR_ALIGN = 5,       /* a pointer is misaligned (see each call)         */
    M3_ERR_WORKSPACE = 6,   /* workspace missing or smaller than required      */
    M3_ERR_HIP = 7          /* the HIP runtime reported an error               */
} m3_status;

typedef enum { M3_F32 = 0, M3_BF16 = 1 } m3_dtype;

/* m3_dims.flags select the prefill kernels (same results up to rounding).
 * Default (0), wherever built (dstate 128, headdim 64): the segmented
 * single-pass kernel: each workgroup scans a segment of consecutive chunks of
 * one (batch, head) slice and carries the state across them; segments of a
 * slice are linked by a decoupled look-back over their state maps.  When
 * seg_chunks is 0 and several segments per slice would be needed, the
 * one-chunk-per-workgroup kernel runs instead for chunks of fewer than 128
 * rows (chunk * rank), and for chunks of 64 or more tokens when the scan has
 * at least 16384 chunks in all (batch * nheads * chunks per slice): it is
 * faster there.  When a slice is one segment and io is bf16
 * with rank 4 and chunk 64, a warp-specialised variant runs (half of its
 * waves form the outputs, half stage the inputs and carry the state).
 * M3_SCAN_SPLIT: three kernels (chunk states, a state pass over chunks,
 * chunk outputs); the only path for other shapes, and for tokens wider than
 * the single-pass kernels' 32-bit row offsets allow (nheads * rank *
 * max(dstate, headdim) elements of at least 16 MiB, or a chunk of such
 * tokens of at least 2 GiB).
 * M3_SCAN_PER_CHUNK: the single-pass kernel with one chunk per workgroup
 * (a look-back across every chunk).  Ignored together with M3_SCAN_SPLIT.
 * M3_THETA_PER_HEAD (m3_scan_fwd and m3_step, gated or not): theta / theta_t
 * are the per-head frequencies omega [nheads][dstate/2] and every angle is
 * dt * omega (Sec. 3.2: the rotation angle is Delta_t times theta, here with
 * a data-independent theta per head, as in RoPE); saves reading
 * 2 * dstate bytes per token and head. */
#define M3_SCAN_SPLIT 1
#define M3_SCAN_PER_CHUNK 2
#define M3_THETA_PER_HEAD 4

typedef struct {
    int64_t batch;     /* >= 1                                              */
    int64_t seqlen;    /* L >= 0 (ignored by m3_step)                        */
    int64_t nheads;    /* >= 1                                              */
    int64_t headdim;   /* P                                                  */
    int64_t dstate;    /* N, even                                            */
    int64_t rank;      /* R >= 1 (MIMO rank)                                 */
    int64_t chunk;     /* Q: tokens per chunk of the prefill scan            */
    int32_t io;        /* m3_dtype of x, B, C, y and the carry               */
    int32_t flags;     /* M3_SCAN_* bits; other bits must be 0               */
    int64_t a_stride_b, a_stride_t, a_stride_h; /* strides of A, in floats   */
    int64_t seg_chunks; /* chunks per workgroup of the segmented kernel; 0 =
                           enough that all workgroups are resident at once
                           (results then depend on the device's CU count in
                           the last bits); ignored by m3_step              */
} m3_dims;

/*
 * Bytes of device workspace m3_scan_fwd needs for `dims` (0 on invalid
 * dims).  The workspace holds the per-chunk state contributions and the
 * states entering each chunk, after a control block of M3_CTL_BYTES at its
 * start (work-item counters, the look-back timeout count, a call counter).
 * The control block must be zero before the workspace's first use with any
 * m3_scan_* call (a zero-filled allocation, or a memset of its first
 * M3_CTL_BYTES); every call then leaves it ready for the next one (the call's last
 * workgroup resets it), so a single-pass scan is one kernel launch.  No m3
 * call writes anything else there (m3_scan_bwd's workspace layout skips it
 * too), so one workspace can serve every scan entry point and dims in turn;
 * a caller that reuses its memory for anything else zeroes the block again
 * before the next scan.  The rest of the workspace needs no initialisation.
 */
#define M3_CTL_BYTES ((size_t)1280)
size_t m3_scan_workspace_bytes(const m3_dims *dims);

/*
 * Chunked prefill scan (Sec. 3.3 "Chunked Algorithm for MIMO SSMs"; the
 * recurrence above).  Writes y for every token, final_state = h_{L-1}, and
 * the carry (B_{L-1}, X_{L-1}) ready for m3_step or a further m3_scan_fwd.
 *
 * init_state (may be NULL) is h_{-1}; init_carryB / init_carryX (both NULL
 * or both set) are B_{-1}, X_{-1}: passing the state and carry returned by
 * an earlier call continues that sequence exactly.  With seqlen == 0 the
 * outputs are the initial state and carry (zeros when not given), and the
 * token arrays (x, B, C, dt, lambda, theta, y) may be NULL.
 *
 * Supported shapes (else M3_ERR_UNSUPPORTED): io bf16 with dstate 128,
 * headdim 64, rank 1/2/4 and chunk*rank a multiple of 64 with chunk in
 * {32, 64, 128}; io bf16 with headdim 64 and the smaller states of the
 * paper's state-size sweep on the three-kernel path: dstate 64 with (rank,
 * chunk) in {(1, 64), (1, 128), (2, 32), (2, 64), (4, 16), (4, 32)}, dstate 32
 * with (1, 64), (2, 32), (4, 16); io fp32 with (dstate, headdim) = (16, 16) or
 * (128, 64), rank 1/2/4, chunk in {16, 32, 64} and chunk*rank a multiple of
 * 64.
 * x, B, C, theta, y, the states, the carries and the workspace must be
 * 16-byte aligned; dt, A, lambda and D 4-byte aligned (else M3_ERR_ALIGN).
 * Output buffers must not overlap the inputs.  A must be <= 0 (a positive
 * log-decay can overflow the chunk-local decay factors); dt and lambda are
 * expected in (0, inf) and [0, 1].
 */
m3_status m3_scan_fwd(const m3_dims *dims,
                      const void *x, const void *B, const void *C,
                      const float *dt, const float *A, const float *lambda,
                      const float *theta, const float *D,
                      const float *init_state, const void *init_carryB,
                      const void *init_carryX,
                      void *y, float *final_state, void *carryB, void *carryX,
                      void *workspace, size_t workspace_bytes, void *stream);

/*
 * m3_scan_fwd with the block's output gate fused into the y store (App.
 * "MIMO for Mamba-3", paragraph "Mamba with MIMO": Y' = Y o SiLU(Z), the
 * residual function phi, with Z computed like X).  z has the layout, dtype
 * and alignment of x ([batch][seqlen][nheads][rank][headdim], io dtype,
 * 16-byte aligned) and may be NULL only when seqlen == 0; it must not
 * overlap y.  y receives (SSM output + D x) o SiLU(z), SiLU(u) = u / (1 +
 * e^{-u}), evaluated in fp32; with io bf16 the single-pass kernels gate the
 * bf16-rounded y and round again (the three-kernel path and m3_step gate
 * before their one rounding).  The final state and the carry are those of
 * m3_scan_fwd (the gate acts on the output only).  Everything else,
 * including the errors, as m3_scan_fwd.
 */
m3_status m3_scan_fwd_gated(const m3_dims *dims,
                            const void *x, const void *B, const void *C,
                            const float *dt, const float *A, const float *lambda,
                            const float *theta, const float *D, const void *z,
                            const float *init_state, const void *init_carryB,
                            const void *init_carryX,
                            void *y, float *final_state, void *carryB, void *carryX,
                            void *workspace, size_t workspace_bytes, void *stream);

/*
 * Varlen prefill: a batch of sequences of different lengths packed along one
 * token axis.  dims->batch is the number of sequences S, dims->seqlen the
 * total number of tokens T; cu_seqlens is a HOST array of S + 1 offsets
 * (cu_seqlens[0] = 0, nondecreasing, cu_seqlens[S] = T): sequence i is tokens
 * cu_seqlens[i] .. cu_seqlens[i+1] - 1, scanned from its own initial state
 * and carry (entry i of init_state / init_carry, or zeros) into entry i of
 * final_state and of the carry outputs.  Token arrays are those of
 * m3_scan_fwd without the batch axis: x, y and z [T][nheads][rank][headdim],
 * B and C [T][nheads][rank][dstate], dt and lambda [T][nheads], theta
 * [T][nheads][dstate/2] (or [nheads][dstate/2] with M3_THETA_PER_HEAD);
 * A[t * a_stride_t + h * a_stride_h] over the packed tokens (a_stride_b must
 * be 0).  z may be NULL (no gate) or a gate input as in m3_scan_fwd_gated.
 * One launch: when m3_scan_varlen_workspace_bytes(dims, cu_seqlens) is
 * non-zero and workspace_bytes is at least that, every (sequence, head,
 * chunk) item of the batch runs in one launch of the one-chunk-per-workgroup
 * kernel (small tables built on the host from cu_seqlens are copied into the
 * workspace first, on `stream`); its results are bit-identical to the same
 * sequences scanned alone with M3_SCAN_PER_CHUNK.  Otherwise (a shape
 * without that kernel, an empty sequence, M3_SCAN_SPLIT, a seg_chunks
 * request, or a smaller workspace) the sequences run one after another on
 * `stream`, each as one m3_scan_fwd (so each picks its own kernel), sharing
 * the workspace: size it at least with m3_scan_workspace_bytes for one
 * sequence of the largest length.  A run of consecutive sequences of equal
 * length then goes out as one m3_scan_fwd over a batch of them (they lie in
 * the packed arrays as that batch would) as far as the workspace holds what
 * the batch needs (m3_scan_workspace_bytes with batch = the run's length,
 * a_stride_b = length * a_stride_t).  The kernel (and its segment count) is
 * chosen per launch, so the last bits of a sequence's results can depend on
 * how many equal-length neighbours it is batched with and hence on
 * workspace_bytes; every grouping is within the scan's tolerance of the
 * recurrence.  Every call's arguments are checked before the first launch
 * (errors as m3_scan_fwd; M3_ERR_NULL for a NULL cu_seqlens, M3_ERR_SHAPE
 * for bad offsets).  m3_scan_varlen_check reads the look-back timeouts of
 * the call (of its last launch when it made several).
 */
size_t m3_scan_varlen_workspace_bytes(const m3_dims *dims, const int64_t *cu_seqlens);
m3_status m3_scan_varlen_check(const m3_dims *dims, const int64_t *cu_seqlens,
                               const void *workspace, size_t workspace_bytes,
                               uint32_t *timeouts, void *stream);
m3_status m3_scan_fwd_varlen(const m3_dims *dims, const int64_t *cu_seqlens,
                             const void *x, const void *B, const void *C,
                             const float *dt, const float *A, const float *lambda,
                             const float *theta, const float *D, const void *z,
                             const float *init_state, const void *init_carryB,
                             const void *init_carryX,
                             void *y, float *final_state, void *carryB, void *carryX,
                             void *workspace, size_t workspace_bytes, void *stream);

/*
 * One decode step (one iteration of the recurrence) for every (b, h):
 * state <- h_t, carry <- (B_t, X_t) in place, y_t written.  dims->seqlen
 * and dims->chunk are ignored; A is read at t = 0 (a_stride_t unused).
 * Tensors: x_t [batch][nheads][rank][headdim], B_t and C_t
 * [batch][nheads][rank][dstate] (io dtype), dt_t and lambda_t
 * [batch][nheads], theta_t [batch][nheads][dstate/2] (fp32),
 * y_t [batch][nheads][rank][headdim] (io dtype).  Supported shapes: the
 * (io, dstate, headdim, rank) of m3_scan_fwd (chunk ignored).
 */
m3_status m3_step(const m3_dims *dims,
                  float *state, void *carryB, void *carryX,
                  const void *x_t, const void *B_t, const void *C_t,
                  const float *dt_t, const float *A, const float *lambda_t,
                  const float *theta_t, const float *D,
                  void *y_t, void *stream);

/*
 * m3_step with the output gate (as m3_scan_fwd_gated): y_t = (S'^T C_t +
 * D X_t) o SiLU(z_t), z_t [batch][nheads][rank][headdim] in the io dtype,
 * 16-byte aligned, not NULL (M3_ERR_NULL), gated in fp32 before the one
 * rounding.  State and carry updates as m3_step.
 */
m3_status m3_step_gated(const m3_dims *dims,
                        float *state, void *carryB, void *carryX,
                        const void *x_t, const void *B_t, const void *C_t,
                        const float *dt_t, const float *A, const float *lambda_t,
                        const float *theta_t, const float *D, const void *z_t,
                        void *y_t, void *stream);

/*
 * The block prologue: the cheap per-token operations of the Mamba-3 block
 * that turn the projections' outputs into the SSM's B, C, X (and the gate's
 * Z), fused into the kernels' input loads so that no separate pass over
 * them touches HBM.
 *   - BCNorm (Sec. 3.4, paragraph "BC / QK Normalization"): with bc_norm,
 *     every rank column of B and C (dstate values of one token, head and
 *     rank) is divided by sqrt(mean of its squares + eps) and multiplied
 *     elementwise by the gain norm_B / norm_C [nheads][rank][dstate] (NULL:
 *     ones).  eps must be > 0 with bc_norm; the gains need bc_norm.
 *   - B, C biases (Sec. 3.4, paragraph "B, C Biases"; App. "B, C Bias
 *     Parameterization"): head-specific, channel-wise bias_B / bias_C
 *     [nheads][rank][dstate] added after the norm (NULL: none; allowed
 *     without bc_norm).
 *   - Structured MIMO input (App. "MIMO for Mamba-3", paragraph "Mamba with
 *     MIMO"): with w_x [nheads][rank][headdim], x holds X'
 *     [..][nheads][headdim] (one headdim-vector per token and head) and the
 *     recurrence uses X[r][p] = w_x[h][r][p] X'[p] (rounded to the io dtype);
 *     w_z does the same for the gate input z (Z = w_z o Z'), and needs z.
 *   - Output norm (Sec. 4, hybrid models; App. table of the norm type and
 *     placement ablation), the block's epilogue, fused into the y store:
 *     with out_norm = M3_OUT_NORM_PRE_GATE, y becomes
 *     out_gain o rms(y) o SiLU(z) (z NULL: no SiLU factor); with
 *     M3_OUT_NORM_POST_GATE, out_gain o rms(y o SiLU(z)).  rms divides each
 *     run of out_group consecutive channels of a (token, head, rank) row of
 *     y by sqrt(mean of their squares + out_eps); out_group is a power of two
 *     with 8 <= out_group <= headdim (headdim: one RMS per row).  y here is
 *     the SSM output with the D skip, rounded to the io dtype, as the plain
 *     scan would store it; out_gain [nheads][rank][headdim] (NULL: ones);
 *     out_eps > 0.  The paper gives no group size: it is the caller's.
 * All tables are fp32 device arrays, 16-byte aligned.  The norm, gain and
 * bias are evaluated in fp32.  The carry written (and read back as
 * init_carry) holds the B and X that the recurrence used, after the
 * prologue.
 */
#define M3_OUT_NORM_NONE 0
#define M3_OUT_NORM_PRE_GATE 1
#define M3_OUT_NORM_POST_GATE 2
typedef struct {
    int32_t bc_norm;                  /* nonzero: RMS-normalise B and C columns  */
    float eps;                        /* > 0 when bc_norm                         */
    const float *norm_B, *norm_C;     /* gains [nheads][rank][dstate] or NULL     */
    const float *bias_B, *bias_C;     /* biases [nheads][rank][dstate] or NULL    */
    const float *w_x;                 /* [nheads][rank][headdim] or NULL          */
    const float *w_z;                 /* [nheads][rank][headdim] or NULL          */
    int32_t out_norm;                 /* M3_OUT_NORM_*                            */
    int32_t out_group;                /* channels per RMS group (with out_norm)   */
    float out_eps;                    /* > 0 with out_norm                        */
    const float *out_gain;            /* [nheads][rank][headdim] or NULL          */
} m3_prologue;

/*
 * m3_scan_fwd (m3_scan_fwd_gated when z is not NULL) with the block
 * prologue `pro` (not NULL) applied to B, C, x and z as they are read.  x
 * (and z with w_z) is [batch][seqlen][nheads][headdim] when w_x (w_z) is
 * given, else as in m3_scan_fwd.  Runs the one-chunk-per-workgroup
 * single-pass kernel, except where the default choice (flags without
 * M3_SCAN_PER_CHUNK, seg_chunks as for m3_scan_fwd) gives one segment per
 * slice at rank 4 and chunk 64: then the warp-specialised kernel runs with
 * the prologue (the workspace is sized by m3_scan_workspace_bytes(dims) as
 * usual).  Supported shapes: io bf16,
 * dstate 128, headdim 64, rank 1/2/4 and chunk 32/64/128 with chunk*rank a
 * multiple of 64 and at most 512 (else M3_ERR_UNSUPPORTED, also with
 * M3_SCAN_SPLIT).  Errors as m3_scan_fwd; M3_ERR_NULL for a NULL pro, or
 * w_z without z; M3_ERR_SHAPE for bc_norm with eps <= 0 (or NaN), for
 * gains without bc_norm, for an unknown out_norm, and with out_norm for
 * out_eps <= 0 (or NaN), an out_gain without it, or an out_group that is
 * not a power of two in [8, headdim]; M3_ERR_ALIGN for a misaligned table.
 */
m3_status m3_scan_fwd_pro(const m3_dims *dims, const m3_prologue *pro,
                          const void *x, const void *B, const void *C,
                          const float *dt, const float *A, const float *lambda,
                          const float *theta, const float *D, const void *z,
                          const float *init_state, const void *init_carryB,
                          const void *init_carryX,
                          void *y, float *final_state, void *carryB, void *carryX,
                          void *workspace, size_t workspace_bytes, void *stream);

/*
 * m3_step (m3_step_gated when z_t is not NULL) with the block prologue:
 * B_t and C_t normalised, biased; x_t (z_t) is [batch][nheads][headdim]
 * when w_x (w_z) is given.  The new carry holds the prologue's B_t and X_t.
 * Supported shapes: io bf16, dstate 128, headdim 64, rank 1/2/4.  Errors as
 * m3_step and m3_scan_fwd_pro.
 */
m3_status m3_step_pro(const m3_dims *dims, const m3_prologue *pro,
                      float *state, void *carryB, void *carryX,
                      const void *x_t, const void *B_t, const void *C_t,
                      const float *dt_t, const float *A, const float *lambda_t,
                      const float *theta_t, const float *D, const void *z_t,
                      void *y_t, void *stream);

/*
 * Backward pass of the scan (training): the gradients of a scalar loss J
 * with respect to every input of m3_scan_fwd, given dy = dJ/dy and
 * dfinal_state = dJ/d(final state) (NULL: zero), for the recurrence above
 * started from init_state (NULL: zero) with no initial carry.  It runs the
 * chunked algorithm (Sec. 3.3 "Chunked Algorithm for MIMO SSMs") in reverse:
 * the chunk states are recomputed, the state gradient is passed from the last
 * chunk to the first, and each chunk's gradients are formed from its own
 * rows with bf16 MFMA and fp32 accumulation.
 * Outputs: dx, dB, dC shaped and typed like x, B, C (io dtype); ddt,
 * dlambda [batch][seqlen][nheads], dtheta [batch][seqlen][nheads][dstate/2]
 * (fp32; the gradient of the per-step angle); dD [nheads]; dA [nheads] (the
 * sum over batch and tokens) when A is per head (a_stride_b = a_stride_t =
 * 0), else dA [batch][seqlen][nheads] (A per token, a_stride_t != 0);
 * dinit_state [batch][nheads][dstate][headdim] when not NULL.  Everything is
 * overwritten.  Supported (else M3_ERR_UNSUPPORTED): io bf16, dstate 128,
 * headdim 64, chunk * rank = 64 (rank 1 chunk 64, rank 2 chunk 32, rank 4
 * chunk 16), no M3_THETA_PER_HEAD; A strided per head or per token.
 * Workspace: m3_scan_bwd_workspace_bytes(dims) bytes (16-byte aligned; two
 * fp32 and two bf16 N x P maps per chunk, after the scans' control block of M3_CTL_BYTES, which
 * this call neither reads nor writes; no initialisation).  Token arrays may be NULL when seqlen == 0.
 * Alignment: x, B, C, dy, dx, dB, dC, the states and the workspace 16 bytes,
 * the rest 4 bytes (else M3_ERR_ALIGN).  Outputs must not overlap inputs.
 * Deterministic (no atomics).  Errors as m3_scan_fwd.
 */
size_t m3_scan_bwd_workspace_bytes(const m3_dims *dims);
m3_status m3_scan_bwd(const m3_dims *dims,
                      const void *x, const void *B, const void *C,
                      const float *dt, const float *A, const float *lambda,
                      const float *theta, const float *D, const float *init_state,
                      const void *dy, const float *dfinal_state,
                      void *dx, void *dB, void *dC,
                      float *ddt, float *dA, float *dlambda, float *dtheta, float *dD,
                      float *dinit_state,
                      void *workspace, size_t workspace_bytes, void *stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc): m3_scan_fwd
 * without a workspace argument.  The workspace is a library-owned device
 * array of M3_SCRATCH_BYTES (256 MiB), one per device the library runs on,
 * held until the process ends; its device address is looked up once per
 * device on the first call made with that device current (that call is not
 * capturable; later ones are).  Nothing is allocated: no hipMalloc, hipFree
 * or allocating library call.  Kernels, results and errors are those of
 * m3_scan_fwd with a workspace (the same bits), except that a scan whose
 * m3_scan_workspace_bytes(dims) exceeds M3_SCRATCH_BYTES returns
 * M3_ERR_WORKSPACE before any device call.  Every call on a device shares
 * that device's array: calls that overlap in time on one device (other
 * streams, other threads) race and give wrong results; calls ordered on
 * one stream are safe (the array starts zero-filled, and each call leaves
 * its control block ready for the next).  The
 * look-back timeout count of these calls is not readable (m3_scan_check
 * takes a workspace); a timeout still shows as NaN results.
 */
#define M3_SCRATCH_BYTES ((size_t)256 << 20)
m3_status m3_scan_fwd_noalloc(const m3_dims *dims,
                              const void *x, const void *B, const void *C,
                              const float *dt, const float *A, const float *lambda,
                              const float *theta, const float *D,
                              const float *init_state, const void *init_carryB,
                              const void *init_carryX,
                              void *y, float *final_state, void *carryB, void *carryX,
                              void *stream);

/*
 * Count of look-back waits that gave up in the last m3_scan_fwd (gated or
 * not) run with `dims` on `workspace` (Sec. 3.3: the inter-chunk state
 * passing whose waits these are).  Copies one word from the workspace to
 * *timeouts after all work queued on `stream` (synchronises the stream).
 * *timeouts = 0 without touching the device for dims that select the
 * three-kernel path or an empty sequence (no waits there).  A non-zero count
 * means that call's y and final state are invalid (they hold NaN from the
 * chunk that gave up on).  Errors: those of m3_scan_fwd for `dims`,
 * M3_ERR_NULL for a NULL `timeouts`, M3_ERR_WORKSPACE when the workspace is
 * smaller than m3_scan_workspace_bytes(dims), M3_ERR_ALIGN, M3_ERR_HIP.
 */
m3_status m3_scan_check(const m3_dims *dims, const void *workspace, size_t workspace_bytes,
                        uint32_t *timeouts, void *stream);

/*
 * Polls a look-back wait makes before it gives up (process-wide, all
 * devices, read at each scan call; 0 restores the default, 2^22 polls of a
 * few hundred nanoseconds each).  For tests of the timeout path: with a
 * limit of 1 a waiting workgroup gives up at once, so the scan finishes with
 * NaN results and a non-zero m3_scan_check count instead of waiting.  The
 * wait at the end of a scan for every work item to be past its look-back
 * (before the workspace's control block is reset for the next call) is
 * bounded by the larger of this limit and the default, so that a short limit
 * leaves the control block clean.
 */
void m3_set_wait_limit(uint32_t polls);

/* Static description of a status code. */
const char *m3_status_string(m3_status status);

/* The hipError_t of the last M3_ERR_HIP returned on this thread (0 if none). */
int m3_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* M3_H */
