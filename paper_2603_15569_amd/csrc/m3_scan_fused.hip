// Single-pass chunked prefill scan of the Mamba-3 SSM on gfx950 (N = 128,
// P = 64): one workgroup per chunk, chunks of a (batch, head) slice linked by
// a decoupled look-back over their N x P fp32 state maps.
//
// Math (Sec. 3.3 "Chunked Algorithm for MIMO SSMs", the two-band mask of
// Sec. 3.1.2 eq. mamba3-mask, the rotary form of Sec. 3.2 Prop. "Rotary
// Embedding Equivalence with Exponential-Trapezoidal Discretization"); for a
// chunk of Q tokens with chunk-local prefix sums cum_t (of dt A) and psi_t
// (of theta), C^_t = R(-psi_t) C_t, B^_j = R(-psi_j) B_j, gamma_t = lambda_t dt_t
// and sigma_j = gamma_j + (1 - lambda_{j+1}) dt_{j+1} (sigma_{L-1} = gamma_{L-1}):
//   y_t   = sum_{j<=t} w_tj (C^_t . B^_j) x_j + e^{cum_t} C^_t . S_in + D x_t,
//           w_tt = gamma_t, w_tj = e^{cum_t - cum_j} sigma_j
//   S_out = T_c S_in + A_c,  T_c = e^{cum_e} R(psi_e),
//           A_c = R(psi_e) sum_j e^{cum_e - cum_j} sigma_j B^_j x_j^T
// S is the physical-frame state with the next token's previous-input term
// folded in.  Rows of every chunk operand are (token, rank) pairs.
//
// Work of one workgroup (NW waves; each wave owns TPW tiles of 16 rows):
//   1. ticket -> (slice, chunk), chunk-major within a slice group, so every
//      predecessor of a chunk holds an earlier ticket of the same counter and
//      is already resident (forward progress);
//   2. prologue: cum (wavefront scans), gamma, sigma, w; angle prefix sums and
//      a cos/sin table in LDS;
//   3. aggregate first: per 64-row block, B^ and W x staged row-major in LDS
//      and M += B^T W x (MFMA, K = rows, operands read with transposing LDS
//      reads); A_c published (flag AGG) unless the predecessor is already
//      inclusive.  bf16 chunks of several blocks (two LDS buffers) form the
//      intra-chunk outputs of step 5 in this same pass (the merged pass),
//      taking the blocks last to first without the prologue;
//   4. decoupled look-back: predecessors' flags probed 16 at a time back to
//      the nearest inclusive state (flag INC) or the sequence start, then the
//      aggregates after it folded forward with the step the owners use for
//      their own S_out (the entering state does not depend on timing); S_out
//      published (flag INC) before any output work, so the chain across
//      chunks advances at the speed of the look-back alone; the last chunk
//      writes the final state and the carry;
//   5. outputs: C^ rows rotated straight into MFMA fragments; y starts as
//      e^{cum_t} C^ S_in (MFMA, K = N); per block at or below each owned tile
//      G^T = B^ C^T (MFMA, K = N) masked by w_tj, y += (w o G) x (MFMA,
//      K = rows); D x added; y staged per wave from the (transposed)
//      accumulator tiles and stored.  A chunk of a single 64-row block
//      stages B^ once for both uses; merged chunks only add the inter-chunk
//      term here; other longer chunks (fp32) restage their blocks.
// The workspace's control block carries the tickets from call to call: the
// call's first item clears the flags (every other item waits for that before
// its first flag access), every item counts itself done after its last flag
// access, and the item of group 0's last ticket resets the counters once all
// are done, so a scan is one launch.
#include <type_traits>

#include "m3_device.h"
#include "m3_internal.h"
#include "m3_scan_common.h"

namespace m3 {
namespace {

using namespace scan;

template <typename T, int Q, int R, bool kGate, bool kPro, bool kVar = false>
// Two waves per SIMD: two 4-wave workgroups or one 8-wave workgroup per CU
// (more waves spill the tile registers of the output phase).  kGate: the
// stored y is multiplied by SiLU(z) (the block's output gate).  kPro: the
// block prologue is applied as the rows arrive (B and C: RMS norm over N,
// gain, bias; x and z: X = W_X o X', Z = W_Z o Z'), from per-head tables in
// LDS.  kVar: sequences of different lengths packed along the token axis,
// items and sequences from the varlen tables.
__global__ __launch_bounds__((FShape<T, Q, R>::NTHR), 2)
void k_scan_fused(ScanArgs a) {
    typedef FShape<T, Q, R> S;
    typedef typename S::Acc Acc;
    typedef typename S::CS CS;
    typedef Mma<T> MM;
    typedef typename MM::frag Frag;
    typedef typename Vec16<T>::type V16;
    constexpr int N = S::N, P = S::P, NH = S::NH, NW = S::NW, TPW = S::TPW, PTW = S::PTW;
    constexpr int NK = N / MM::K;       // MFMA K-steps over the state axis
    constexpr int JK = S::JB / MM::K;   // MFMA K-steps over a 64-row block
    constexpr int PT = P / 16;
    // cos/sin table [token][pair]: a thread's consecutive pairs are 16-byte
    // LDS pieces; rows 32 bytes longer than the pairs (bank spread)
    constexpr int LDT = NH + 32 / (int)sizeof(typename S::CS);

    __shared__ Acc s_cum[Q];
    __shared__ float s_c2[Q];   // cum_t log2(e): the causal weights are 2^{c2_t - c2_j} sigma_j
    __shared__ Acc s_wtot[NW];
    __shared__ Acc s_psie[NH];
    __shared__ float s_gam[Q], s_sig[Q], s_w[Q];
    __shared__ __attribute__((aligned(16))) CS s_cs[Q * LDT];
    // Chunks of several row blocks double-buffer the staged blocks: block
    // jb + 1 is committed while the MFMAs read block jb (one barrier a block).
    constexpr int NBUF = (S::NJB > 1 && sizeof(T) == 2) ? 2 : 1;   // (fp32 blocks: LDS too small)
    // With two buffers the intra-chunk outputs are formed in the aggregate
    // pass itself, from the same staged blocks (B^, x and W x): one pass over
    // the chunk's rows; only e^{cum_t} C^ S_in waits for the look-back.
    constexpr bool kMerged = NBUF == 2;
    // Row blocks are staged row-major (16-byte writes): B^ [row][n], x and
    // W x [row][p]; MFMA operands whose K axis runs along the rows (B^T and
    // (W x)^T for M, x^T for y) are read with the LDS transposing reads.
    constexpr int LDP = P + S::PAD;
    constexpr int kSB = S::JB * S::LDN, kSXr = S::JB * LDP;
    __shared__ __attribute__((aligned(16))) T s_B[NBUF * kSB];        // B^ blocks [row][n]
    __shared__ __attribute__((aligned(16))) T s_XW[2 * NBUF * kSXr];  // x blocks, then W x blocks [row][p]
    __shared__ __attribute__((aligned(16))) T s_S[P * S::LDN];        // S_in^T [p][n] (io dtype)
    __shared__ int s_i[4];
    __shared__ uint32_t s_ctl[2];   // call epoch, whether this item is the janitor
    // block prologue tables of the head (fp32): B gain and bias as 16-byte
    // entries (gain, bias of element i, gain, bias of element i + N/2 of rank
    // row r: one read serves a rotation pair) at bgb(r, i), C gain, C bias
    // [R][N], then W_X, W_Z and the output norm's gain [R][P] (ones / zeros
    // where not given)
    constexpr int kPB = 0, kPC = 2 * R * N, kPCb = 3 * R * N, kPWX = 4 * R * N,
                  kPWZ = 4 * R * N + R * P, kPGY = 4 * R * N + 2 * R * P;
    __shared__ __attribute__((aligned(16))) float s_pro[kPro ? 4 * R * N + 3 * R * P : 4];
    // B table entry of (rank row r, element i = piece * CE + e): ordered by
    // (e, piece, r), so that the lanes staging one element of their pieces
    // (consecutive pieces, all ranks) read consecutive entries
    constexpr int BPR = NH / S::CE;   // 16-byte pieces per half row
    auto bgb = [](int r, int i) { return kPB + 4 * (((i % S::CE) * BPR + i / S::CE) * R + r); };
    Acc *s_segtot = reinterpret_cast<Acc *>(s_B);              // prologue only
    static_assert(sizeof(Acc) * S::NSEG * NH <= sizeof(T) * S::JB * S::LDN, "alias");
    static_assert(P <= S::JB && NW * 16 <= 2 * NBUF * S::JB, "y staging fits in the x / W x buffers");

    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);   // uniform: scalar branches
    const int g = lane >> 4, l16 = lane & 15;

    // ---- 1. ticket -> (slice, chunk) ----
    const int64_t nsl = a.batch * a.H;
    if (tid == 0) {
        int64_t ci, si;
        uint32_t ep;
        bool rd, jan;
        if constexpr (kVar) {
            take_item_var(a.ctl, a.vl_grp, a.vl_gstart, a.vl_order, a.vl_maxn, &ci, &si, &ep, &rd, &jan);
        } else {
            take_item(a.ctl, nsl, a.nchunks, &ci, &si, &ep, &rd);
            jan = is_janitor(ci, si, nsl, a.nchunks);
        }
        s_i[0] = (int)ci;
        s_i[1] = (int)si;
        s_i[2] = (int)ep;
        s_i[3] = rd ? 1 : 0;
        s_ctl[0] = ep;
        s_ctl[1] = jan ? 1u : 0u;
    }
    __syncthreads();
    const int64_t c = s_i[0], sl = s_i[1];
    const uint32_t epoch = (uint32_t)s_i[2];
    bool flags_ready = s_i[3] != 0;
    __syncthreads();
    if (c < 0) return;   // (cannot happen: one workgroup per item)
    if (c == 0 && sl == 0) {   // the call's first item clears the look-back flags
        clear_flags(a.ctl, a.flags, kVar ? a.vl_slots : nsl * a.nchunks, epoch, tid, S::NTHR);
        flags_ready = true;
    }
    const int64_t b = sl / a.H, h = sl % a.H;
    // the item's sequence: its first token in the token arrays, its length,
    // its chunks, the first flag slot of the slice, and A's offset for it
    int64_t seq_tok, seq_len, seq_n, seq_slot, a_off;
    if constexpr (kVar) {
        seq_tok = a.vl_tok[b];
        seq_len = a.vl_len[b];
        seq_n = (seq_len + Q - 1) / Q;
        seq_slot = a.vl_slot[b] + h * seq_n;
        a_off = seq_tok * a.a_st;   // (a_sb = 0: A runs over the packed tokens)
    } else {
        seq_tok = b * a.L;
        seq_len = a.L;
        seq_n = a.nchunks;
        seq_slot = sl * a.nchunks;
        a_off = b * a.a_sb;
    }
    const int64_t t0 = c * Q;
    const int nvalid = (int)min((int64_t)Q, seq_len - t0);
    const int64_t slot = seq_slot + c;
    const int64_t tok0 = (seq_tok + t0) * a.H + h;       // (token, head) flat index of the chunk's first row
    const int64_t tstr = a.H;                             // token stride in token-heads
    const bool last = (c == seq_n - 1);

    const T *Cg = static_cast<const T *>(a.C) + tok0 * (R * N);
    const T *Bg = static_cast<const T *>(a.B) + tok0 * (R * N);
    const int64_t bstr = tstr * R * N, xstr = tstr * R * P;   // token strides of B/C and x (y, z)
    // x as read: P x R per token-head, or (structured input) the P-vector X'
    // that every rank row reads (row offset 0)
    const bool sx = kPro && a.pro.wx != nullptr, sz = kPro && a.pro.wz != nullptr;
    const int64_t xin_tok = sx ? (int64_t)P : (int64_t)(R * P);
    const int xr_el = sx ? 0 : P;
    const T *Xg = static_cast<const T *>(a.x) + tok0 * xin_tok;
    const int64_t xin_str = tstr * xin_tok;

    // K consecutive prologue-table floats (16-byte LDS reads; p a multiple of 4)
    auto tab = [&](int p, float *v, int K) {
        for (int q = 0; q < K; q += 4) {
            const float4 f = *reinterpret_cast<const float4 *>(&s_pro[p + q]);
            v[q] = f.x; v[q + 1] = f.y; v[q + 2] = f.z; v[q + 3] = f.w;
        }
    };
    // Rows jb*64 .. of the chunk are staged in two steps so that the global
    // loads of the next block overlap the MFMA work on this one: fetch()
    // issues the loads into registers, commit() rotates B^ = R(-psi_t) B and
    // writes it to LDS row-major, together with W x (aggregate: operand of M)
    // and/or x (outputs: operand of y).  Consecutive lanes take consecutive
    // rows, so the cos/sin table reads are conflict-free.
    constexpr int TB = S::JB * (NH / S::CE) / S::NTHR;   // B tasks per thread
    constexpr int TX = S::JB * (P / S::CE) / S::NTHR;    // x tasks per thread
    static_assert(TB * S::NTHR == S::JB * (NH / S::CE) && TX * S::NTHR == S::JB * (P / S::CE), "tasks");
    struct Blk { V16 lo[TB], hi[TB], xv[TX]; };
    // The loads are unconditional and go through buffer resources that end
    // at the chunk's last valid token (rows past the end of the sequence read
    // as zeros), so the number of loads in flight is static and the
    // compiler's waits stop at exactly the loads a step needs, leaving later
    // prefetches in flight.
    const uint32_t bstr_b = (uint32_t)(bstr * sizeof(T)), xstr_b = (uint32_t)(xstr * sizeof(T));
    const uint32_t xin_b = (uint32_t)(xin_str * sizeof(T));
    const Rsrc rb = make_rsrc(Bg, (uint32_t)(((nvalid - 1) * bstr + R * N) * (int64_t)sizeof(T)));
    const Rsrc rc = make_rsrc(Cg, (uint32_t)(((nvalid - 1) * bstr + R * N) * (int64_t)sizeof(T)));
    const Rsrc rx = make_rsrc(Xg, (uint32_t)(((nvalid - 1) * xin_str + (R - 1) * xr_el + P) * (int64_t)sizeof(T)));
    // B row pieces: consecutive lanes take consecutive rows (conflict-free
    // cos/sin reads); with the prologue the NH / CE pieces of a row sit in
    // consecutive lanes of one wave instead, so that its norm is a lane sum.
    auto brow = [](int task) { return kPro ? task / BPR : task % S::JB; };
    auto bpiece = [](int task) { return kPro ? task % BPR : task / S::JB; };
    auto fetch = [&](int jb, Blk &f) {
#pragma unroll
        for (int k = 0; k < TB; ++k) {
            const int task = tid + k * S::NTHR, jr = brow(task), cp = bpiece(task);
            const int row = jb * S::JB + jr, t = row / R, r = row % R;
            const uint32_t off = tok_off(t, bstr_b) + (uint32_t)((r * N + cp * S::CE) * sizeof(T));
            f.lo[k] = buf_load<V16>(rb, off);
            f.hi[k] = buf_load<V16>(rb, off + NH * sizeof(T));
        }
#pragma unroll
        for (int k = 0; k < TX; ++k) {
            const int task = tid + k * S::NTHR, jr = task % S::JB, pc = task / S::JB;
            const int row = jb * S::JB + jr, t = row / R, r = row % R;
            f.xv[k] = buf_load<V16>(rx, tok_off(t, xin_b) + (uint32_t)((r * xr_el + pc * S::CE) * sizeof(T)));
        }
    };
    // A thread's B tasks have the same rank rows and pieces in every block
    // (JB is a multiple of R): chunks of up to 256 rows hold their table
    // entries in registers for the whole chunk; the 512-row chunks need those
    // registers for their tiles and read the entries per block.
    constexpr bool kHoldB = kPro && S::QR <= 256;
    static_assert(S::JB % R == 0, "rank row of a B task independent of the block");
    float4 bgr[kHoldB ? TB : 1][kHoldB ? S::CE : 1];
    // kAgg: stage W x too (operand of M); kOut: stage x too (operand of y)
    auto commit = [&](int jb, const Blk &f, auto kAgg, auto kOut) {
        T *sB = s_B + (jb % NBUF) * kSB, *sX = s_XW + (jb % NBUF) * kSXr, *sWX = s_XW + (NBUF + jb % NBUF) * kSXr;
#pragma unroll
        for (int k = 0; k < TB; ++k) {
            const int task = tid + k * S::NTHR, jr = brow(task), cp = bpiece(task);
            const int t = (jb * S::JB + jr) / R;
            V16 lo = f.lo[k], hi = f.hi[k];
            float csv[S::CE], snv[S::CE];
            cs_getn<S::CE>(&s_cs[t * LDT + cp * S::CE], csv, snv);
            float sc = 1.f, bsc = 1.f;
            int pb = 0;
            if constexpr (kPro) {   // B = g o B' / rms(B') + b (rows past the end stay zero)
                float ss = sumsq(lo) + sumsq(hi);
#pragma unroll
                for (int o = 1; o < BPR; o <<= 1) ss += __shfl_xor(ss, o, kWave);
                const bool ok = t < nvalid;
                sc = !ok ? 0.f : (a.pro.bcnorm ? rsqrtf(ss * (1.f / N) + a.pro.eps) : 1.f);
                bsc = ok ? 1.f : 0.f;
                pb = bgb(jr % R, cp * S::CE);
                // (opaque per block: the reads stay in the block loop)
                if constexpr (!kHoldB) asm volatile("" : "+v"(pb));
            }
#pragma unroll
            for (int e = 0; e < S::CE; ++e) {
                float u = fget(lo, e), w = fget(hi, e);
                if constexpr (kPro) {   // (one 16-byte table entry a pair)
                    const float4 gb = kHoldB ? bgr[k][e] : *reinterpret_cast<const float4 *>(&s_pro[pb + 4 * BPR * R * e]);
                    u = sc * gb.x * u + bsc * gb.y;
                    w = sc * gb.z * w + bsc * gb.w;
                }
                fset(lo, e, csv[e] * u + snv[e] * w);
                fset(hi, e, csv[e] * w - snv[e] * u);
            }
            *reinterpret_cast<V16 *>(&sB[jr * S::LDN + cp * S::CE]) = lo;
            *reinterpret_cast<V16 *>(&sB[jr * S::LDN + NH + cp * S::CE]) = hi;
        }
#pragma unroll
        for (int k = 0; k < TX; ++k) {
            const int task = tid + k * S::NTHR, jr = task % S::JB, pc = task / S::JB;
            V16 xv = f.xv[k];
            if constexpr (kPro) {   // X = W_X o X' (ones without structured input)
                int pw = kPWX + ((jb * S::JB + jr) % R) * P + pc * S::CE;
                asm volatile("" : "+v"(pw));
                float wv[S::CE];
                tab(pw, wv, S::CE);
#pragma unroll
                for (int e = 0; e < S::CE; ++e) fset(xv, e, fget(xv, e) * wv[e]);
            }
            if constexpr (decltype(kOut)::value) *reinterpret_cast<V16 *>(&sX[jr * LDP + pc * S::CE]) = xv;
            if constexpr (decltype(kAgg)::value) {
                const float wt = s_w[(jb * S::JB + jr) / R];
                V16 wx;
#pragma unroll
                for (int e = 0; e < S::CE; ++e) fset(wx, e, wt * fget(xv, e));
                *reinterpret_cast<V16 *>(&sWX[jr * LDP + pc * S::CE]) = wx;
            }
        }
    };
    // Prefetch depth (blocks in flight, register ring): the aggregate phase
    // has registers to spare; the output phase keeps C^ fragments and
    // accumulators live, so wide-tile shapes prefetch less.
    constexpr int DA = kMerged ? 1 : (S::NJB < 4 ? S::NJB : 4);
    constexpr int DC = S::NJB < 1 ? S::NJB : 1;
    constexpr int DR = DA > DC ? DA : DC;
    Blk ring[DR];
    // The merged pass takes the row blocks last to first: the first blocks
    // worked on need the C^ fragments of few owned tiles (the last rows'), so
    // each tile's C rows are waited for and rotated only when its first block
    // comes, inside the block loop, instead of all before it (the sums of the
    // aggregate and of the outputs are taken in that order too).  With the
    // prologue the rotation also normalises, and the blocks keep their order
    // (the per-tile normalisations measured slower there): all tiles are
    // rotated at once, after the first block's aggregate products, with
    // their C rows loaded once the first block is staged.
    constexpr bool kRev = kMerged && !kPro;
    auto blk = [](int sb) { return kRev ? S::NJB - 1 - sb : sb; };

    Frag cf[TPW][NK];   // C rows of the owned output tiles (rotated in the output phase)
    constexpr bool kEarlyC = S::NJB > 1;
    // In the reversed order, owned tile m is first used (and rotated) in
    // block pass c_rot(m); its C rows are loaded two passes before that,
    // after that pass's prefetch of the next block (so the block waits do
    // not wait for them), and only the tiles used in the first two passes
    // load with the prologue: its burst of loads stays small.
    auto c_rot = [](int m) { return S::NJB - 1 - ((m + 1) * S::NWO - 1) / 4; };
    auto c_issue = [&](int m) { return kRev && c_rot(m) >= 2 ? c_rot(m) - 2 : -1; };
    // the owned tiles' C rows issued at pass `at` (-1: the prologue)
    auto load_c = [&](int at) {
#pragma unroll
        for (int mi = 0; mi < TPW; ++mi) {
            const int m = kRev ? TPW - 1 - mi : mi;   // (in the order the tiles are first used)
            if (c_issue(m) != at) continue;
            const int row = owned_tile<S>(wave, m) * 16 + l16, t = row / R, r = row % R;
            const uint32_t off = tok_off(t, bstr_b) + (uint32_t)((r * N + MM::KPL * g) * sizeof(T));
#pragma unroll
            for (int kk = 0; kk < NK; ++kk) cf[m][kk] = buf_load<Frag>(rc, off + kk * MM::K * sizeof(T));
        }
    };
    // ---- 2. prologue ----
    // The head's prologue tables: every thread's entries are loaded at once,
    // ahead of the item's other loads (buffer loads: a table that is not
    // given reads as zeros through an empty range and takes its default
    // below), and written to LDS before the prologue's first barrier; they
    // are read after the prologue's barriers.
    constexpr int TEN = (R * N + S::NTHR - 1) / S::NTHR, TEP = (R * P + S::NTHR - 1) / S::NTHR;
    float pvn[kPro ? TEN : 1][4], pvp[kPro ? TEP : 1][3];
    if constexpr (kPro) {
        const int64_t hn = h * (R * N), hp = h * (R * P);
        auto trs = [&](const float *t, int64_t off, int n) {
            return make_rsrc(t ? t + off : a.D, t ? (uint32_t)(n * 4) : 0u);
        };
        const Rsrc rt[4] = {trs(a.pro.gB, hn, R * N), trs(a.pro.bB, hn, R * N), trs(a.pro.gC, hn, R * N),
                            trs(a.pro.bC, hn, R * N)};
        const Rsrc rp[3] = {trs(a.pro.wx, hp, R * P), trs(a.pro.wz, hp, R * P), trs(a.pro.og, hp, R * P)};
#pragma unroll
        for (int k = 0; k < TEN; ++k)
#pragma unroll
            for (int u = 0; u < 4; ++u) pvn[k][u] = buf_load<float>(rt[u], (uint32_t)((tid + k * S::NTHR) * 4));
#pragma unroll
        for (int k = 0; k < TEP; ++k)
#pragma unroll
            for (int u = 0; u < 3; ++u) pvp[k][u] = buf_load<float>(rp[u], (uint32_t)((tid + k * S::NTHR) * 4));
    }
    auto write_tables = [&]() {
        if constexpr (kPro) {
#pragma unroll
            for (int k = 0; k < TEN; ++k) {
                const int e = tid + k * S::NTHR;
                if (e < R * N) {
                    const int r = e / N, n = e % N;
                    const int q = bgb(r, n % NH) + (n < NH ? 0 : 2);
                    s_pro[q] = a.pro.gB ? pvn[k][0] : 1.f;
                    s_pro[q + 1] = a.pro.bB ? pvn[k][1] : 0.f;
                    s_pro[kPC + e] = a.pro.gC ? pvn[k][2] : 1.f;
                    s_pro[kPCb + e] = a.pro.bC ? pvn[k][3] : 0.f;
                }
            }
#pragma unroll
            for (int k = 0; k < TEP; ++k) {
                const int e = tid + k * S::NTHR;
                if (e < R * P) {
                    s_pro[kPWX + e] = a.pro.wx ? pvp[k][0] : 1.f;
                    s_pro[kPWZ + e] = a.pro.wz ? pvp[k][1] : 1.f;
                    s_pro[kPGY + e] = a.pro.og ? pvp[k][2] : 1.f;
                }
            }
        }
    };
    {
        // angles first (the largest prologue load): thread (pair i, segment seg)
        const int i = tid % NH, seg = tid / NH;
        // (tokens past the end of the sequence read as zeros; the dt and
        // lambda ranges extend to the next chunk's first token if there is one)
        // (per-head frequencies: every token reads the head's omega row, and
        // the angle is dt * omega: the segment's dt values are loaded too)
        const Rsrc rth = a.theta_ph ? make_rsrc(a.theta + h * NH, (uint32_t)(NH * 4))
                                    : make_rsrc(a.theta + tok0 * NH, (uint32_t)(((nvalid - 1) * tstr + 1) * NH * 4));
        const uint32_t thstr_b = a.theta_ph ? 0u : (uint32_t)(tstr * NH * 4), tstr_b = (uint32_t)(tstr * 4);
        float th[S::TPS];
#pragma unroll
        for (int k = 0; k < S::TPS; ++k) th[k] = buf_load<float>(rth, tok_off(seg * S::TPS + k, thstr_b) + i * 4);
        const int nvn = nvalid + (t0 + nvalid < seq_len ? 1 : 0);
        const Rsrc rdt = make_rsrc(a.dt + tok0, (uint32_t)(((nvn - 1) * tstr + 1) * 4));
        float dts[S::TPS];
        if (a.theta_ph) {
            const Rsrc rdv = make_rsrc(a.dt + tok0, (uint32_t)(((nvalid - 1) * tstr + 1) * 4));   // zero past the end
#pragma unroll
            for (int k = 0; k < S::TPS; ++k) dts[k] = buf_load<float>(rdv, tok_off(seg * S::TPS + k, tstr_b));
        }
        const Rsrc rlam = make_rsrc(a.lam + tok0, (uint32_t)(((nvn - 1) * tstr + 1) * 4));
        const uint32_t o = tok_off(tid, tstr_b);
        const float dtv = buf_load<float>(rdt, o), lamv = buf_load<float>(rlam, o);
        const float dtn = buf_load<float>(rdt, o + tstr_b), lamn = buf_load<float>(rlam, o + tstr_b);
        const int64_t tg = t0 + min(tid, nvalid - 1);
        const float Av = a.A[a_off + tg * a.a_st + h * a.a_sh];
        // the first blocks' loads go out after the prologue's own loads (memory
        // counters retire in order), so they overlap the prologue's arithmetic
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int d = 0; d < DA; ++d) fetch(blk(d), ring[d]);
        __builtin_amdgcn_sched_barrier(0);
        // chunks of several row blocks load the C rows of their output tiles
        // now too (in the reversed block order only those of the tiles used
        // first; in the forward order, with the prologue, after the first
        // block is staged): the round trip overlaps the aggregate and the
        // look-back (single-block chunks load them in the output phase: earlier
        // loads measured slower there, their waits delaying the publications)
        if constexpr (kEarlyC && !(kMerged && !kRev)) load_c(-1);
        __builtin_amdgcn_sched_barrier(0);
        // dt and lambda are zero past the end of the sequence, so
        // sigma_{L-1} = gamma_{L-1} and rows past the end carry zeros
        const bool ok = tid < Q;
        const Acc lg = ok ? (Acc)dtv * (Acc)Av : (Acc)0;
        const float gam = lamv * dtv;
        const float sig = gam + (1.f - lamn) * dtn;
        Acc ps[S::TPS];
#pragma unroll
        for (int k = 0; k < S::TPS; ++k) ps[k] = (Acc)(a.theta_ph ? th[k] * dts[k] : th[k]);
        if (tid < Q) {
            s_gam[tid] = gam;
            s_sig[tid] = sig;
        }
        Acc v = wave_incl_scan(lg, lane);
        if (lane == kWave - 1) s_wtot[wave] = v;
        // running sums of the segment's angles
        Acc run = 0;
#pragma unroll
        for (int k = 0; k < S::TPS; ++k) {
            run += ps[k];
            ps[k] = run;
        }
        s_segtot[seg * NH + i] = run;
        if constexpr (kPro) write_tables();
        __syncthreads();
        if (tid < Q) {
            Acc off = 0;
            for (int w2 = 0; w2 < wave; ++w2) off += s_wtot[w2];
            s_cum[tid] = v + off;
            s_c2[tid] = (float)((v + off) * (Acc)1.4426950408889634);
        }
        Acc off = 0;
        for (int s2 = 0; s2 < seg; ++s2) off += s_segtot[s2 * NH + i];
#pragma unroll
        for (int k = 0; k < S::TPS; ++k) {
            const int t = seg * S::TPS + k;
            if (t < Q) {
                const Acc psi = ps[k] + off;
                Acc sn, cs;
                sincos_fast(psi, &sn, &cs);
                cs_put(&s_cs[t * LDT + i], (float)cs, (float)sn);
                if (t == nvalid - 1) s_psie[i] = psi;
            }
        }
        __syncthreads();
        if (tid < Q) {
            const Acc cum_e = s_cum[nvalid - 1];
            s_w[tid] = (tid < nvalid) ? (float)(exp_fast(cum_e - s_cum[tid]) * (Acc)s_sig[tid]) : 0.f;
        }
        __syncthreads();
    }
    if constexpr (kHoldB) {   // the B table entries of this thread's tasks (tables written before the barriers above)
#pragma unroll
        for (int k = 0; k < TB; ++k) {
            const int task = tid + k * S::NTHR;
#pragma unroll
            for (int e = 0; e < S::CE; ++e)
                bgr[k][e] = *reinterpret_cast<const float4 *>(&s_pro[bgb(brow(task) % R, bpiece(task) * S::CE + e)]);
        }
    }


    using True = std::integral_constant<bool, true>;
    using False = std::integral_constant<bool, false>;

    // C^ fragments of the owned row tiles, rotated by -psi_t (rows past the
    // end of the sequence were loaded as zeros).  With the prologue the
    // rotation first normalises each element, c = sc g c + b in fp32 (sc the
    // row's RMS scale from a sum of squares over its fragments; a row sits in
    // lanes l16 + 16 g), so the fragments are rounded once.  A lane's rank
    // row r = l16 % R is the same in all its tiles, so the gain and bias of
    // its elements are read once per fragment pair (16-byte reads) and serve
    // every tile.  `only` >= 0 rotates that owned tile alone.
    auto rotate_cf = [&](int only) {
        float scm[TPW], bscm[TPW];
        if constexpr (kPro) {
#pragma unroll
            for (int m = 0; m < TPW; ++m) {
                if (only >= 0 && m != only) continue;
                const int t = (owned_tile<S>(wave, m) * 16 + l16) / R;
                float ss = 0.f;
#pragma unroll
                for (int kk = 0; kk < NK; ++kk) ss += sumsq(cf[m][kk]);
                ss += __shfl_xor(ss, 16, kWave);
                ss += __shfl_xor(ss, 32, kWave);
                const bool ok = t < nvalid;
                scm[m] = !ok ? 0.f : (a.pro.bcnorm ? rsqrtf(ss * (1.f / N) + a.pro.eps) : 1.f);
                bscm[m] = ok ? 1.f : 0.f;
            }
        }
#pragma unroll
        for (int kk = 0; kk < NK / 2; ++kk) {
            float gu[MM::KPL], gw[MM::KPL], bu[MM::KPL], bw[MM::KPL];
            if constexpr (kPro) {
                static_assert(MM::KPL % 4 == 0 && 16 % R == 0, "16-byte table reads; r = l16 % R");
                const int pu = (l16 % R) * N + kk * MM::K + MM::KPL * g, pw = pu + NH;
#pragma unroll
                for (int e4 = 0; e4 < MM::KPL; e4 += 4) {
                    const float4 a0 = *reinterpret_cast<const float4 *>(&s_pro[kPC + pu + e4]);
                    const float4 a1 = *reinterpret_cast<const float4 *>(&s_pro[kPC + pw + e4]);
                    const float4 c0 = *reinterpret_cast<const float4 *>(&s_pro[kPCb + pu + e4]);
                    const float4 c1 = *reinterpret_cast<const float4 *>(&s_pro[kPCb + pw + e4]);
                    gu[e4] = a0.x; gu[e4 + 1] = a0.y; gu[e4 + 2] = a0.z; gu[e4 + 3] = a0.w;
                    gw[e4] = a1.x; gw[e4 + 1] = a1.y; gw[e4 + 2] = a1.z; gw[e4 + 3] = a1.w;
                    bu[e4] = c0.x; bu[e4 + 1] = c0.y; bu[e4 + 2] = c0.z; bu[e4 + 3] = c0.w;
                    bw[e4] = c1.x; bw[e4 + 1] = c1.y; bw[e4 + 2] = c1.z; bw[e4 + 3] = c1.w;
                }
            }
#pragma unroll
            for (int m = 0; m < TPW; ++m) {
                if (only >= 0 && m != only) continue;
                const int t = (owned_tile<S>(wave, m) * 16 + l16) / R;
                float csv[MM::KPL], snv[MM::KPL];
                cs_getn<MM::KPL>(&s_cs[t * LDT + kk * MM::K + MM::KPL * g], csv, snv);
#pragma unroll
                for (int e = 0; e < MM::KPL; ++e) {
                    float u = fget(cf[m][kk], e), w = fget(cf[m][kk + NK / 2], e);
                    if constexpr (kPro) {
                        u = scm[m] * gu[e] * u + bscm[m] * bu[e];
                        w = scm[m] * gw[e] * w + bscm[m] * bw[e];
                    }
                    fset(cf[m][kk], e, csv[e] * u + snv[e] * w);
                    fset(cf[m][kk + NK / 2], e, csv[e] * w - snv[e] * u);
                }
            }
        }
    };
    // Output tiles are transposed (y^T = S^T C^T, y^T += x^T (w o G)^T):
    // lane l holds row l % 16 of a tile and four consecutive columns.
    f32x4 acc[TPW][PT];
    const float Dh = a.D[h];
    // Intra-chunk outputs of staged block jb: per pair of 16-row j-tiles, the
    // masked G^T tiles of every owned tile at or below it and y += (w o G) x.
    auto out_block = [&](int jb) {
        const T *sB = s_B + (jb % NBUF) * kSB, *sX = s_XW + (jb % NBUF) * kSXr;
        // Owned tile m of any wave lies in rows 16 m NWO .. 16 (m + 1) NWO - 1,
        // i.e. in blocks m NWO / 4 .. ((m + 1) NWO - 1) / 4: tiles whose blocks
        // all come before block jb have no work in it, tiles whose blocks all
        // come after it take every pair unmasked; only the others compare rows.
        auto tile_above = [&](int m) { return ((m + 1) * S::NWO - 1) / 4 < jb; };
        auto tile_below = [&](int m) { return (m * S::NWO) / 4 > jb; };
#pragma unroll
        for (int jp = 0; jp < S::JB / 32; ++jp) {
            const int J0 = jb * 4 + 2 * jp;        // first j-tile of the pair (chunk-global)
            if (J0 > owned_tile<S>(wave, TPW - 1) && J0 > owned_tile<S>(wave, 0)) continue;
            // x^T columns of the pair, shared by all owned tiles
            bf16x8 xf[PT];
            if constexpr (MM::KPL == 8) {
#pragma unroll
                for (int pt = 0; pt < PT; ++pt) {
                    // rows 32 jp + 4g .. +3 and 32 jp + 16 + 4g .. +3 of x, column l16
                    const T *xr = &sX[(32 * jp + 4 * g + l16 / 4) * LDP + pt * 16 + 4 * (l16 % 4)];
                    const bf16x4 lo = lds_tr4(xr), hi = lds_tr4(xr + 16 * LDP);
#pragma unroll
                    for (int v = 0; v < 4; ++v) { xf[pt][v] = lo[v]; xf[pt][4 + v] = hi[v]; }
                }
            }
            // G^T tiles (K = N) for every owned tile at or below the pair; each
            // B^ fragment is loaded once and used by all owned tiles
            f32x4 gt[TPW][2];
#pragma unroll
            for (int m = 0; m < TPW; ++m) gt[m][0] = gt[m][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < 2; ++q)
#pragma unroll
                for (int kk = 0; kk < NK; ++kk) {
                    const Frag bf = MM::load(&sB[((2 * jp + q) * 16 + l16) * S::LDN + kk * MM::K + MM::KPL * g]);
#pragma unroll
                    for (int m = 0; m < TPW; ++m)
                        if (!tile_above(m) && (tile_below(m) || J0 + q <= owned_tile<S>(wave, m)))
                            gt[m][q] = MM::mma(bf, cf[m][kk], gt[m][q]);
                }
            // mask weights (branch-free): w_tj = e^{cum_t - cum_j} sigma_j (j < t),
            // gamma_t (j = t), 0 (j > t); D x_t as D on the diagonal row = column
#pragma unroll
            for (int m = 0; m < TPW; ++m) {
                const int TT = owned_tile<S>(wave, m);
                if (tile_above(m) || (!tile_below(m) && J0 > TT)) continue;
                const int tt = (TT * 16 + l16) / R;
                const float c2_t = s_c2[tt], cum_t = (float)s_cum[tt], gam_t = s_gam[tt];
                // the lane's 4 rows 4g+v of a j-tile span NV tokens (one when R >= 4)
                constexpr int NV = R >= 4 ? 1 : 4 / R;
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    float wv[NV];
#pragma unroll
                    for (int u = 0; u < NV; ++u) {
                        const int tj = ((J0 + q) * 16 + 4 * g + u * R) / R;
                        // (above the diagonal the exponent may be large: the select drops
                        // it; rank 4 with the prologue keeps the base-e form, whose
                        // register allocation there spills less)
                        const float e = (R >= 4 && kPro) ? exp_fast(fminf(cum_t - (float)s_cum[tj], 0.f)) * s_sig[tj]
                                                         : exp2_fast(c2_t - s_c2[tj]) * s_sig[tj];
                        wv[u] = (tile_below(m) || tj < tt) ? e : (tj == tt ? gam_t : 0.f);
                    }
#pragma unroll
                    for (int v = 0; v < 4; ++v) gt[m][q][v] *= wv[(v * NV) / 4];
                    if (!tile_below(m) && J0 + q == TT) {   // diagonal tile (wave-uniform): the skip term
#pragma unroll
                        for (int v = 0; v < 4; ++v) gt[m][q][v] += (4 * g + v == l16) ? Dh : 0.f;
                    }
                }
                // y^T += x^T (w o G)^T  (K = the pair's 32 rows)
                if constexpr (MM::KPL == 8) {
                    bf16x8 af;
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        af[v] = (bf16)gt[m][0][v];
                        af[4 + v] = (bf16)gt[m][1][v];
                    }
#pragma unroll
                    for (int pt = 0; pt < PT; ++pt) acc[m][pt] = MM::mma(xf[pt], af, acc[m][pt]);
                } else {
#pragma unroll
                    for (int q = 0; q < 2; ++q)
#pragma unroll
                        for (int v = 0; v < 4; ++v)
#pragma unroll
                            for (int pt = 0; pt < PT; ++pt) {
                                const float xv = to_f32(sX[(32 * jp + 16 * q + 4 * g + v) * LDP + pt * 16 + l16]);
                                acc[m][pt] = MM::mma(xv, gt[m][q][v], acc[m][pt]);
                            }
                }
            }
        }
    };

    // ---- 3. aggregate: M = B^T W x over the chunk (state pair-tiles) ----
    f32x4 ms[PTW][2];
#pragma unroll
    for (int m2 = 0; m2 < PTW; ++m2) ms[m2][0] = ms[m2][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    if constexpr (kMerged) {
#pragma unroll
        for (int m = 0; m < TPW; ++m)
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) acc[m][pt] = f32x4{0.f, 0.f, 0.f, 0.f};
        commit(blk(0), ring[0], True{}, True{});
        __syncthreads();
        if (DA < S::NJB) fetch(blk(DA), ring[0]);
        if constexpr (!kRev) load_c(-1);
    }
#pragma unroll
    for (int sb = 0; sb < S::NJB; ++sb) {
        const int jb = blk(sb);
        if constexpr (NBUF == 2) {
            if (sb + 1 < S::NJB) {   // stage the next block while this one feeds the MFMAs
                commit(blk(sb + 1), ring[(sb + 1) % DA], True{}, True{});
                if (sb + 1 + DA < S::NJB) fetch(blk(sb + 1 + DA), ring[(sb + 1) % DA]);
                if constexpr (kRev) load_c(sb);
            }
        } else {
            if constexpr (S::NJB == 1) commit(jb, ring[0], True{}, True{});   // one block: keep B^ for the outputs
            else commit(jb, ring[jb % DA], True{}, False{});
            __syncthreads();
            if (jb + DA < S::NJB) fetch(jb + DA, ring[jb % DA]);
        }
        // M += B^T (W x) (a wave's state tiles share their row tiles,
        // wave % 4 and wave % 4 + 4: each B^T fragment is loaded once for all
        // of them, each (W x)^T fragment once for both halves)
        static_assert(NW % 4 == 0, "state row tiles shared across a wave's tiles");
        const T *sB = s_B + (jb % NBUF) * kSB, *sWX = s_XW + (NBUF + jb % NBUF) * kSXr;
        const int ntl = wave % 4;
#pragma unroll
        for (int ks = 0; ks < JK; ++ks) {
            Frag af[2];
#pragma unroll
            for (int half = 0; half < 2; ++half)
                af[half] = load_kt(sB, S::LDN, ks * MM::K, (ntl + 4 * half) * 16, g, l16);
#pragma unroll
            for (int m2 = 0; m2 < PTW; ++m2) {
                const int pt = (wave + NW * m2) / 4;
                const Frag bf = load_kt(sWX, LDP, ks * MM::K, pt * 16, g, l16);
#pragma unroll
                for (int half = 0; half < 2; ++half) ms[m2][half] = MM::mma(af[half], bf, ms[m2][half]);
            }
        }
        if constexpr (kMerged) {
            // an owned tile's C^ fragments are rotated just before the first
            // block (in the reversed order) that works on it: its own last
            // block, whose rows reach the tile's
            if constexpr (kRev) {
#pragma unroll
                for (int m = 0; m < TPW; ++m)
                    if (((m + 1) * S::NWO - 1) / 4 == jb) rotate_cf(m);
            } else if (sb == 0) {
                rotate_cf(-1);   // (after the first block's aggregate: the C rows arrive meanwhile)
            }
            out_block(jb);
        }
        __syncthreads();
    }


    // Owned state element (m2, half, v): row n = 16*(ntl + 4*half) + 4g + v,
    // column p = 16*pt + l16; rows (i, i + N/2) of a pair sit in one lane.
    const Acc cum_e = s_cum[nvalid - 1];
    float Ast[PTW][2][4];   // A_c = R(psi_e) M
#pragma unroll
    for (int m2 = 0; m2 < PTW; ++m2) {
        const int ntl = (wave + NW * m2) % 4;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            Acc sn, cs;
            sincos_fast(s_psie[ntl * 16 + 4 * g + v], &sn, &cs);
            const Acc re = ms[m2][0][v], im = ms[m2][1][v];
            Ast[m2][0][v] = (float)(cs * re - sn * im);
            Ast[m2][1][v] = (float)(sn * re + cs * im);
        }
    }
    // Published maps: 8-byte words (v, v+1) of each owned (m2, half), laid out
    // so that the lanes of a wave touch consecutive words (coalesced).
    auto word_index = [&](int m2, int half, int vp) -> int64_t {
        return (int64_t)((m2 * 2 + half) * 2 + vp) * S::NTHR + tid;
    };
    const int64_t SZ = (int64_t)N * P;
    Acc *totp = static_cast<Acc *>(a.tot);
    // publish the aggregate (only successors read it), unless (chunks of
    // several row blocks) the predecessor's inclusive state is already there:
    // this chunk's own then follows at once, and successors that find no flag
    // wait for it.  (Single-block chunks measured faster always publishing.)
    bool flags_lost = false;   // the wait for cleared flags gave up (error path)
    if (!flags_ready && (c > 0 || !last)) {
        if (tid == 0) s_i[0] = wait_flags_ready(a.ctl, s_ctl[0], a.spin_max) ? 0 : 1;
        __syncthreads();
        flags_lost = s_i[0] != 0;
        __syncthreads();
    }
    // (chunks of several blocks read the predecessor's flag first: if it is
    // inclusive, the look-back below takes that state without probing)
    bool publish_agg = c > 0 && !last && !flags_lost, pred_inc = false;
    if (S::NJB > 1 && c > 0 && !flags_lost) {
        if (tid == 0)
            s_i[0] = __hip_atomic_load(a.flags + slot - 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == kFlagInc;
        __syncthreads();
        pred_inc = s_i[0] != 0;
        publish_agg = publish_agg && !pred_inc;
    }
    if (publish_agg) {
        unsigned long long *dst = reinterpret_cast<unsigned long long *>(a.agg + slot * SZ);
#pragma unroll
        for (int m2 = 0; m2 < PTW; ++m2)
#pragma unroll
            for (int half = 0; half < 2; ++half)
#pragma unroll
                for (int vp = 0; vp < 2; ++vp)
                    st_coh2(dst + word_index(m2, half, vp), Ast[m2][half][2 * vp], Ast[m2][half][2 * vp + 1]);
        if (tid == 0) st_coh(totp + slot * (NH + 1), cum_e);
        if (tid < NH) st_coh(totp + slot * (NH + 1) + 1 + tid, s_psie[tid]);
        wait_stores_done();
        __syncthreads();
        if (tid == 0) __hip_atomic_store(a.flags + slot, kFlagAgg, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }

    // ---- 4. look-back: S_in of this chunk ----
    // S_init (owned): initial state plus the carried previous-input term of token 0
    auto load_init = [&](float (&Si)[PTW][2][4]) {
        const float *ist = a.init_state ? a.init_state + sl * SZ : nullptr;
        float wb = 0.f;
        if (a.init_cB) {
            const int64_t k0 = seq_tok * a.H + h;
            wb = (1.f - a.lam[k0]) * a.dt[k0];
        }
        const T *iB = a.init_cB ? static_cast<const T *>(a.init_cB) + sl * (R * N) : nullptr;
        const T *iX = a.init_cX ? static_cast<const T *>(a.init_cX) + sl * (R * P) : nullptr;
        // element (m2, half, v): row 16 (ntl + 4 half) + 4g + v, column 16 pt + l16
        init_elems<T, R, N, P, PTW * 8>(
            ist, iB, iX, wb,
            [&](int e) { return 16 * ((wave + NW * (e / 8)) % 4 + 4 * ((e / 4) % 2)) + 4 * g + e % 4; },
            [&](int e) { return (wave + NW * (e / 8)) / 4 * 16 + l16; }, &Si[0][0][0]);
    };

    // ---- entering state ----
    // The nearest predecessor whose inclusive state is published (or the
    // sequence start) is found first, waiting on any predecessor in between
    // that has published nothing yet; the aggregates after it are then folded
    // forward, S <- T_k S + A_k, with the arithmetic their owners use for
    // their own inclusive states (state_step).  So S_in is the same fold from
    // the sequence start whichever predecessors happened to be done: the
    // results do not depend on timing.
    const int ntl_w = wave % 4;   // all owned pair rows of a lane are 16 ntl_w + 4g + v
    float Sin[PTW][2][4];
    if (c == 0) {
        load_init(Sin);
    } else {
        const int64_t sbase = seq_slot;
        int64_t j = c - 1;        // next predecessor to probe
        int64_t jt = (flags_lost || pred_inc) ? c - 1 : -2;   // terminal: -1 sequence start, >= 0 inclusive state
        bool timed_out = flags_lost;
        while (jt == -2) {
            // probe predecessors j, j-1, ..., j-15 at once (lanes of wave 0)
            if (wave == 0) {
                uint32_t f = 0;
                if (lane < kProbe) {
                    const int64_t jj = j - lane;
                    f = (jj < 0) ? kFlagInit
                                 : __hip_atomic_load(a.flags + sbase + jj, __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_AGENT);
                }
                const uint64_t mterm = __ballot(lane < kProbe && (f == kFlagInc || f == kFlagInit));
                const uint64_t mzero = __ballot(lane < kProbe && f == 0u);
                const int ft = mterm ? __ffsll((unsigned long long)mterm) - 1 : kProbe;
                const int fz = mzero ? __ffsll((unsigned long long)mzero) - 1 : kProbe;
                if (lane == 0) {
                    s_i[1] = (fz < ft) ? fz : ft;                  // predecessors passed
                    s_i[2] = (ft < fz && ft < kProbe) ? 1 : 0;     // terminal found
                    s_i[3] = (fz < ft) ? 1 : 0;                    // must wait on one
                }
            }
            __syncthreads();
            const int adv = s_i[1], found = s_i[2], needwait = s_i[3];
            __syncthreads();
            if (found) {
                jt = (j - adv < 0) ? -1 : j - adv;
            } else if (needwait) {   // predecessor j - adv has published nothing: wait for it
                j -= adv;
                if (tid == 0) {
                    uint32_t f = 0u;
                    for (uint32_t spin = 0; spin < a.spin_max; ++spin) {
                        f = __hip_atomic_load(a.flags + sbase + j, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        if (f != 0u) break;
                        __builtin_amdgcn_s_sleep(2);
                    }
                    if (f == 0u) count_timeout(a.ctl, s_ctl[0]);   // timed out: report and stop waiting
                    s_i[1] = (f == 0u) ? 1 : 0;
                }
                __syncthreads();
                timed_out = s_i[1] != 0;
                __syncthreads();
                if (timed_out) jt = c - 1;   // (error path: the entering state is NaN)
            } else {
                j -= kProbe;                 // sixteen aggregates: probe further back
            }
        }
        if (timed_out) {   // y of this chunk and of every later one, and the final state, become NaN
#pragma unroll
            for (int m2 = 0; m2 < PTW; ++m2)
#pragma unroll
                for (int v = 0; v < 4; ++v) Sin[m2][0][v] = Sin[m2][1][v] = __builtin_nanf("");
        } else if (jt < 0) {
            load_init(Sin);
        } else {
            const unsigned long long *src = reinterpret_cast<const unsigned long long *>(a.inc + (sbase + jt) * SZ);
#pragma unroll
            for (int m2 = 0; m2 < PTW; ++m2)
#pragma unroll
                for (int half = 0; half < 2; ++half)
#pragma unroll
                    for (int vp = 0; vp < 2; ++vp)
                        ld_coh2(src + word_index(m2, half, vp), Sin[m2][half][2 * vp], Sin[m2][half][2 * vp + 1]);
        }
        // Fold forward from the terminal, one aggregate a round trip; each round
        // also probes the nearest predecessors, and an inclusive state published
        // meanwhile replaces the rest of the fold (it is that fold: same bits).
        for (int64_t k = jt; k < c - 1;) {
            if (wave == 0) {
                const int64_t jj = c - 1 - lane;
                uint32_t f = 0;
                if (lane < kProbe && jj > k + 1)
                    f = __hip_atomic_load(a.flags + sbase + jj, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                const uint64_t minc = __ballot(f == kFlagInc);
                if (lane == 0) s_i[1] = minc ? __ffsll((unsigned long long)minc) - 1 : -1;
            }
            const int64_t kn = k + 1;
            const unsigned long long *src = reinterpret_cast<const unsigned long long *>(a.agg + (sbase + kn) * SZ);
            const Acc *tp = totp + (sbase + kn) * (NH + 1);
            float d[PTW][2][4];
            Acc ps[4];
            const Acc cm = ld_coh(tp);
#pragma unroll
            for (int v = 0; v < 4; ++v) ps[v] = ld_coh(tp + 1 + ntl_w * 16 + 4 * g + v);
#pragma unroll
            for (int m2 = 0; m2 < PTW; ++m2)
#pragma unroll
                for (int half = 0; half < 2; ++half)
#pragma unroll
                    for (int vp = 0; vp < 2; ++vp)
                        ld_coh2(src + word_index(m2, half, vp), d[m2][half][2 * vp], d[m2][half][2 * vp + 1]);
            __syncthreads();
            const int near = s_i[1];
            __syncthreads();
            if (near >= 0) {   // inclusive state of predecessor c - 1 - near: continue from it
                k = c - 1 - near;
                const unsigned long long *isrc = reinterpret_cast<const unsigned long long *>(a.inc + (sbase + k) * SZ);
#pragma unroll
                for (int m2 = 0; m2 < PTW; ++m2)
#pragma unroll
                    for (int half = 0; half < 2; ++half)
#pragma unroll
                        for (int vp = 0; vp < 2; ++vp)
                            ld_coh2(isrc + word_index(m2, half, vp), Sin[m2][half][2 * vp], Sin[m2][half][2 * vp + 1]);
                continue;
            }
            k = kn;
            const Acc de = exp_fast(cm);
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                Acc sn, cs;
                sincos_fast(ps[v], &sn, &cs);
#pragma unroll
                for (int m2 = 0; m2 < PTW; ++m2) state_step(Sin[m2][0][v], Sin[m2][1][v], de, cs, sn, d[m2][0][v], d[m2][1][v]);
            }
        }
    }

    // S_out = e^{cum_e} R(psi_e) S_in + A_c (the same step a successor's fold takes)
    {
        float Sout[PTW][2][4];
        const Acc de = exp_fast(cum_e);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            Acc sn, cs;
            sincos_fast(s_psie[ntl_w * 16 + 4 * g + v], &sn, &cs);
#pragma unroll
            for (int m2 = 0; m2 < PTW; ++m2) {
                Sout[m2][0][v] = Sin[m2][0][v];
                Sout[m2][1][v] = Sin[m2][1][v];
                state_step(Sout[m2][0][v], Sout[m2][1][v], de, cs, sn, Ast[m2][0][v], Ast[m2][1][v]);
            }
        }
        if (!last && !flags_lost) {
            unsigned long long *dst = reinterpret_cast<unsigned long long *>(a.inc + slot * SZ);
#pragma unroll
            for (int m2 = 0; m2 < PTW; ++m2)
#pragma unroll
                for (int half = 0; half < 2; ++half)
#pragma unroll
                    for (int vp = 0; vp < 2; ++vp)
                        st_coh2(dst + word_index(m2, half, vp), Sout[m2][half][2 * vp], Sout[m2][half][2 * vp + 1]);
            wait_stores_done();
            __syncthreads();
            if (tid == 0) __hip_atomic_store(a.flags + slot, kFlagInc, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else if (last) {
            float *fs = a.final_state + sl * SZ;
#pragma unroll
            for (int m2 = 0; m2 < PTW; ++m2) {
                const int k = wave + NW * m2, ntl = k % 4, pt = k / 4;
#pragma unroll
                for (int half = 0; half < 2; ++half)
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        fs[(16 * (ntl + 4 * half) + 4 * g + v) * P + pt * 16 + l16] = Sout[m2][half][v];
            }
            T *cB = static_cast<T *>(a.cB) + sl * (R * N);
            T *cX = static_cast<T *>(a.cX) + sl * (R * P);
            const int64_t kl = (seq_tok + seq_len - 1) * a.H + h;
            const T *Bl = static_cast<const T *>(a.B) + kl * (R * N);
            const T *Xl = static_cast<const T *>(a.x) + kl * xin_tok;
            if constexpr (kPro) {   // the carry holds the B and X the recurrence used
                static_assert(N == 2 * kWave, "two elements of a B row per lane");
                for (int r = wave; r < R; r += NW) {
                    const float v0 = to_f32(Bl[r * N + lane]), v1 = to_f32(Bl[r * N + kWave + lane]);
                    float ss = v0 * v0 + v1 * v1;
#pragma unroll
                    for (int o = 1; o < kWave; o <<= 1) ss += __shfl_xor(ss, o, kWave);
                    const float sc = a.pro.bcnorm ? rsqrtf(ss * (1.f / N) + a.pro.eps) : 1.f;
                    const int e0 = r * N + lane, e1 = e0 + kWave;   // elements lane and lane + N/2
                    const float4 gb = *reinterpret_cast<const float4 *>(&s_pro[bgb(r, lane)]);
                    cB[e0] = from_f32<T>(sc * gb.x * v0 + gb.y);
                    cB[e1] = from_f32<T>(sc * gb.z * v1 + gb.w);
                }
                for (int e = tid; e < R * P; e += S::NTHR)
                    cX[e] = from_f32<T>(to_f32(Xl[sx ? e % P : e]) * s_pro[kPWX + e]);
            } else {
                for (int e = tid; e < R * N; e += S::NTHR) cB[e] = Bl[e];
                for (int e = tid; e < R * P; e += S::NTHR) cX[e] = Xl[e];
            }
        }
    }

    // ---- 5. outputs ----
    // Single-pass chunks (two buffers) only add e^{cum_t} C^ S_in to the
    // accumulators; the others restage their blocks (the first ones fetched
    // now, after the look-back and the publication, whose waits would drain
    // them) and form the intra-chunk term here.
    if constexpr (!kMerged && S::NJB > 1) {
#pragma unroll
        for (int d = 0; d < DC; ++d) fetch(d, ring[d]);
    }
#pragma unroll
    for (int m2 = 0; m2 < PTW; ++m2) {
        const int k = wave + NW * m2, ntl = k % 4, pt = k / 4;
#pragma unroll
        for (int half = 0; half < 2; ++half)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                s_S[(pt * 16 + l16) * S::LDN + 16 * (ntl + 4 * half) + 4 * g + v] = from_f32<T>(Sin[m2][half][v]);
    }
    // y leaves in 16-byte pieces of its rows (NPC per lane and owned tile);
    // with the gate, the matching pieces of z are loaded before the
    // inter-chunk products and arrive during them (the 512-row chunks load a
    // tile's pieces once its products are done, when its C^ fragments are
    // dead: their registers are full until then)
    constexpr int RP = P / S::CE;                   // 16-byte pieces of a row
    constexpr int NPC = 16 * RP / kWave;
    static_assert(NPC * kWave == 16 * RP, "store pieces");
    constexpr bool kLateZ = S::QR > 256;
    V16 zp[kGate ? TPW : 1][NPC];
    // z as read: like x, or (structured) the P-vector Z' of each token;
    // the pieces of owned tile m, or of all (m < 0)
    auto load_z = [&](int m) {
        const int64_t zin_tok = sz ? (int64_t)P : (int64_t)(R * P);
        const int zr_el = sz ? 0 : P;
        const uint32_t zin_b = (uint32_t)(tstr * zin_tok * sizeof(T));
        const Rsrc rz = make_rsrc(static_cast<const T *>(a.z) + tok0 * zin_tok,
                                  (uint32_t)(((nvalid - 1) * tstr * zin_tok + (R - 1) * zr_el + P) *
                                             (int64_t)sizeof(T)));
#pragma unroll
        for (int mm = 0; mm < TPW; ++mm)
#pragma unroll
            for (int i = 0; i < NPC; ++i) {
                if (m >= 0 && mm != m) continue;
                const int k = lane + i * kWave, rl = k / RP, col = (k % RP) * S::CE;
                const int row = owned_tile<S>(wave, mm) * 16 + rl, t = row / R, r = row % R;
                zp[mm][i] = buf_load<V16>(rz, tok_off(t, zin_b) + (uint32_t)((r * zr_el + col) * sizeof(T)));
            }
    };
    if constexpr (kGate && !kLateZ) load_z(-1);
    if constexpr (!kMerged) {
        if constexpr (!kEarlyC) load_c(-1);
        rotate_cf(-1);
    }
    __syncthreads();   // s_S complete
    // inter-chunk term e^{cum_t} C^_t . S_in
#pragma unroll
    for (int m = 0; m < TPW; ++m) {
        const int TT = owned_tile<S>(wave, m);
        const float ecum = (float)exp_fast(s_cum[(TT * 16 + l16) / R]);
#pragma unroll
        for (int pt = 0; pt < PT; ++pt) {
            f32x4 tmp = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < NK; ++kk)
                tmp = MM::mma(MM::load(&s_S[(pt * 16 + l16) * S::LDN + kk * MM::K + MM::KPL * g]), cf[m][kk], tmp);
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                if constexpr (kMerged) acc[m][pt][v] += ecum * tmp[v];
                else acc[m][pt][v] = ecum * tmp[v];
            }
        }
        if constexpr (kGate && kLateZ) load_z(m);
    }
    if constexpr (!kMerged) {
        // intra-chunk term over the row blocks at or below each owned tile
#pragma unroll
        for (int jb = 0; jb < S::NJB; ++jb) {
            if constexpr (S::NJB > 1) {
                commit(jb, ring[jb % DC], False{}, True{});
                __syncthreads();
                if (jb + DC < S::NJB) fetch(jb + DC, ring[jb % DC]);
            }
            out_block(jb);
            if constexpr (S::NJB > 1) __syncthreads();
        }
    }
    // store: once every wave is past its last LDS read, each wave stages its
    // tiles in its own part of the x / W x buffers (a wave's LDS accesses
    // execute in order: no further barrier) and writes whole 16-byte pieces
    // of the y rows
    __syncthreads();
    T *s_y = s_XW + wave * (16 * LDP);
    T *Yg = static_cast<T *>(a.y) + tok0 * (R * P);
#pragma unroll
    for (int m = 0; m < TPW; ++m) {
        const int TT = owned_tile<S>(wave, m);
#pragma unroll
        for (int pt = 0; pt < PT; ++pt) store4(&s_y[l16 * LDP + pt * 16 + 4 * g], acc[m][pt]);
        asm volatile("" ::: "memory");
#pragma unroll
        for (int i = 0; i < NPC; ++i) {
            const int k = lane + i * kWave, rl = k / RP, col = (k % RP) * S::CE;
            const int row = TT * 16 + rl, t = row / R, r = row % R;
            V16 yv = *reinterpret_cast<const V16 *>(&s_y[rl * LDP + col]);
            if constexpr (kPro) {
                // gate factor SiLU(W_Z o Z') in fp32, then (optionally) the
                // output norm: the group's pieces sit in consecutive lanes
                // (a row's RP pieces are RP consecutive lanes), so its sum of
                // squares is a lane sum (rows past the end of the sequence
                // hold finite values and are not stored)
                float yf[S::CE], gz[S::CE], wz[S::CE];
                if constexpr (kGate) tab(kPWZ + r * P + col, wz, S::CE);
#pragma unroll
                for (int e = 0; e < S::CE; ++e) {
                    yf[e] = fget(yv, e);
                    gz[e] = kGate ? silu(fget(zp[m][i], e) * wz[e]) : 1.f;
                }
                if (a.pro.onorm) {   // (uniform)
                    const bool post = a.pro.onorm == 2;
                    float ss = 0.f;
#pragma unroll
                    for (int e = 0; e < S::CE; ++e) {
                        if (post) yf[e] *= gz[e];
                        ss += yf[e] * yf[e];
                    }
                    // (a fixed count of lane steps, those past the group adding nothing:
                    // a loop of constant length stays unrolled)
#pragma unroll
                    for (int o = 1; o < RP; o <<= 1) {
                        const float so = __shfl_xor(ss, o, kWave);
                        ss += o < a.pro.ogroup / S::CE ? so : 0.f;
                    }
                    const float sc = rsqrtf(ss / (float)a.pro.ogroup + a.pro.oeps);
                    float gy[S::CE];
                    tab(kPGY + r * P + col, gy, S::CE);
#pragma unroll
                    for (int e = 0; e < S::CE; ++e) {
                        yf[e] *= sc * gy[e];
                        if (!post) yf[e] *= gz[e];
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < S::CE; ++e) yf[e] *= gz[e];
                }
#pragma unroll
                for (int e = 0; e < S::CE; ++e) fset(yv, e, yf[e]);
            } else if constexpr (kGate) {
                yv = gate_piece<T>(yv, zp[m][i]);
            }
            if (t < nvalid) *reinterpret_cast<V16 *>(Yg + t * xstr + r * P + col) = yv;
        }
        asm volatile("" ::: "memory");
    }
    if (tid == 0 && s_ctl[1])
        janitor_reset(a.ctl, nsl, a.nchunks, s_ctl[0], a.spin_max, kVar ? a.vl_grp : nullptr, a.vl_maxn);
}

template <typename T, int Q, int R, bool kPro = false>
hipError_t launch_fused(const ScanArgs &a, hipStream_t stream) {
    typedef FShape<T, Q, R> S;
    const int64_t nsl = a.batch * a.H;
    if (a.z)
        hipLaunchKernelGGL((k_scan_fused<T, Q, R, true, kPro>), dim3((unsigned)(nsl * a.nchunks)),
                           dim3(S::NTHR), 0, stream, a);
    else
        hipLaunchKernelGGL((k_scan_fused<T, Q, R, false, kPro>), dim3((unsigned)(nsl * a.nchunks)),
                           dim3(S::NTHR), 0, stream, a);
    return hipGetLastError();
}

// Varlen single launch: one workgroup per (sequence, head, chunk) item.
template <typename T, int Q, int R>
hipError_t launch_fused_var(const ScanArgs &a, hipStream_t stream) {
    typedef FShape<T, Q, R> S;
    if (a.z)
        hipLaunchKernelGGL((k_scan_fused<T, Q, R, true, false, true>), dim3((unsigned)a.vl_slots),
                           dim3(S::NTHR), 0, stream, a);
    else
        hipLaunchKernelGGL((k_scan_fused<T, Q, R, false, false, true>), dim3((unsigned)a.vl_slots),
                           dim3(S::NTHR), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

#define M3_FUSED_SHAPES(X)   \
    X(0, float, 2, 32)       \
    X(0, float, 4, 16)       \
    X(0, float, 4, 32)       \
    X(1, bf16, 1, 64)        \
    X(1, bf16, 1, 128)       \
    X(1, bf16, 2, 32)        \
    X(1, bf16, 2, 64)        \
    X(1, bf16, 2, 128)       \
    X(1, bf16, 4, 32)        \
    X(1, bf16, 4, 64)        \
    X(1, bf16, 4, 128)

scan_launch_fn find_fused_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q) {
    if (N != 128 || P != 64) return nullptr;
#define M3_CASE(IO, T, R_, Q_) \
    if (io == IO && R == R_ && Q == Q_) return &launch_fused<T, Q_, R_>;
    M3_FUSED_SHAPES(M3_CASE)
#undef M3_CASE
    return nullptr;
}

scan_launch_fn find_fused_var_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q) {
    if (N != 128 || P != 64) return nullptr;
#define M3_CASE(IO, T, R_, Q_) \
    if (io == IO && R == R_ && Q == Q_) return &launch_fused_var<T, Q_, R_>;
    M3_FUSED_SHAPES(M3_CASE)
#undef M3_CASE
    return nullptr;
}

// The block prologue is built into the bf16 per-chunk kernels.
scan_launch_fn find_fused_pro_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q) {
    if (N != 128 || P != 64 || io != 1) return nullptr;
#define M3_CASE(R_, Q_) \
    if (R == R_ && Q == Q_) return &launch_fused<bf16, Q_, R_, true>;
    M3_CASE(1, 64) M3_CASE(1, 128) M3_CASE(2, 32) M3_CASE(2, 64) M3_CASE(2, 128)
    M3_CASE(4, 32) M3_CASE(4, 64) M3_CASE(4, 128)
#undef M3_CASE
    return nullptr;
}

}  // namespace m3
