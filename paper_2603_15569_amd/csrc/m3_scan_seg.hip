// Segmented single-pass prefill scan of the Mamba-3 SSM on gfx950 (N = 128,
// P = 64): each workgroup owns a segment of G consecutive chunks of one
// (batch, head) slice and carries the state from chunk to chunk itself;
// segments of a slice are linked by a decoupled look-back over their N x P
// fp32 state maps.
//
// Chunk math as in the one-chunk-per-workgroup kernel (Sec. 3.3 chunked
// algorithm, the two-band mask of Sec. 3.1.2 eq. mamba3-mask, the rotary form
// of Sec. 3.2): with chunk-local prefix sums cum_t (of dt A) and psi_t (of
// theta), C^_t = R(-psi_t) C_t, B^_j = R(-psi_j) B_j, w_tt = gamma_t,
// w_tj = e^{cum_t - cum_j} sigma_j,
//   y_t = sum_{j<=t} w_tj (C^_t . B^_j) x_j + e^{cum_t} C^_t . S + D x_t,
//   S  <-  R(psi_e) (e^{cum_e} S + M),   M = sum_j e^{cum_e - cum_j} sigma_j B^_j x_j^T.
// A segment composes its chunks' maps into one map S -> T S + A with
// T = e^{sum cum_e} R(sum psi_e).
//
// Work of one workgroup:
//   1. ticket -> (segment, slice), segment-major within a slice group, so
//      every predecessor of a segment holds an earlier ticket of the same
//      counter and is resident (forward progress);
//      with one segment per slice there is no look-back and no ticket;
//   2. (several segments) aggregate pass: per chunk the prologue (decay and
//      angle prefix scans, cos/sin table, weights) and M from the row blocks
//      (MFMA, K = rows); A <- R(psi_e)(e^{cum_e} A + M); the aggregate is
//      published, the look-back yields the entering state, the segment's
//      outgoing state is published (or written as the final state);
//   3. output pass: per chunk the prologue again, C^ rotated into MFMA
//      fragments, y = e^{cum_t} C^ S (MFMA, K = N), then per row block the
//      masked G^T = B^ C^T (MFMA, K = N), y += (w o G) x (MFMA, K = rows) and,
//      when the segment continues, M for the next chunk's state; y stored.
// Loads run one chunk ahead: the next chunk's angles and scalars right after
// this chunk's prologue, its first row blocks while this chunk's last blocks
// are in use, its C rows after this chunk's last use of C^ (the last chunk of
// a segment reloads its own rows instead, so that every iteration issues the
// same loads).
#include <type_traits>

#include "m3_device.h"
#include "m3_internal.h"
#include "m3_scan_common.h"

namespace m3 {
namespace {

using namespace scan;

// Eight waves per workgroup: all of them stage row blocks and carry the
// state; output row tiles are owned by NWO waves each, or, when a chunk has
// fewer row tiles than waves, by NSP waves each (one share of the columns).
template <typename T, int Q, int R>
using SegShape = FShape<T, Q, R, 8>;

// kGate: the stored y is multiplied by SiLU(z) (the block's output gate).
template <typename T, int Q, int R, bool kGate>
__global__ __launch_bounds__((SegShape<T, Q, R>::NTHR), 2)
void k_scan_seg(ScanArgs a) {
    typedef SegShape<T, Q, R> S;
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
    constexpr int NJB = S::NJB;
    constexpr int NSP = S::NW / S::NWO;  // waves sharing a row tile (column split)
    constexpr int PTS = PT / NSP;       // 16-column tiles of y per wave
    static_assert(NSP * S::NWO == S::NW && PTS * NSP == PT, "column split");

    // chunk-parity double buffers: the tail of a chunk (state rotation by
    // psi_e, the aggregate's cum_e) may still read them while faster waves
    // run the next chunk's prologue
    __shared__ Acc s_cumb[2][Q];
    __shared__ Acc s_psieb[2][NH];
    Acc *s_cum = s_cumb[0], *s_psie = s_psieb[0];
    __shared__ Acc s_segps[NH];         // angle totals of the segment
    __shared__ float s_gam[Q], s_sig[Q], s_w[Q];
    // Chunks of up to 64 tokens tabulate the causal weights of the chunk:
    // s_W[t][j] = e^{cum_t - cum_j} sigma_j (j < t), gamma_t (j = t), 0 (j > t)
    constexpr bool kWTab = Q <= 64;
    constexpr int LDW = Q + 4;
    __shared__ float s_W[kWTab ? Q * LDW : 1];
    __shared__ __attribute__((aligned(16))) CS s_cs[Q * LDT];
    // Chunks of several row blocks double-buffer the staged blocks: in the
    // output pass block jb + 1 is committed while block jb feeds the MFMAs.
    constexpr int NBUF = (NJB > 1 && sizeof(T) == 2) ? 2 : 1;
    // Row blocks are staged row-major (16-byte writes): B^ [row][n], x and
    // W x [row][p].  MFMA operands whose K axis runs along the rows (x^T for
    // y, B^T and (W x)^T for M) are read with the LDS transposing reads.
    constexpr int LDP = P + S::PAD;
    constexpr int kSB = S::JB * S::LDN, kSXr = S::JB * LDP;
    __shared__ __attribute__((aligned(16))) T s_B[NBUF * kSB];        // B^ blocks [row][n]; S^T [p][n]
    __shared__ __attribute__((aligned(16))) T s_XW[2 * NBUF * kSXr];  // x blocks, then W x blocks [row][p]
    __shared__ int s_i[4];
    __shared__ uint32_t s_ctl[2];   // call epoch, whether this item is the janitor
    static_assert(P == S::JB, "S^T [p][n] fits in the B^ block");
    static_assert(NW * 16 <= 2 * NBUF * S::JB, "y staging fits in the x / W x buffers");

    // Lane indices are re-derived from an opaque copy of the thread index at
    // the top of every chunk iteration (relane), so that the compiler
    // recomputes addresses instead of keeping them live across the loops.
    int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);   // uniform: scalar branches
    int g = lane >> 4, l16 = lane & 15;
    const bool ow = true;                      // every wave owns output tiles
    const int wt = wave % S::NWO;              // row-tile owner index (uniform)
    const int pofs = (wave / S::NWO) * PTS;    // first owned column tile (uniform)
    auto relane = [&]() {
        asm volatile("" : "+v"(tid));
        lane = tid & (kWave - 1);
        g = lane >> 4;
        l16 = lane & 15;
    };

    // ---- 1. (segment, slice) ----
    const int64_t nsl = a.batch * a.H;
    // linked segments take (segment, slice) items from the slice groups'
    // counters (segment-major within a group: every predecessor segment holds
    // an earlier ticket); independent slices take their block index
    int64_t sg = 0, sl = blockIdx.x;
    uint32_t epoch = 0;
    bool flags_ready = true;
    if (a.nseg > 1) {
        if (tid == 0) {
            int64_t si, sli;
            uint32_t ep;
            bool rd;
            take_item(a.ctl, nsl, a.nseg, &si, &sli, &ep, &rd);
            s_i[0] = (int)si;
            s_i[1] = (int)sli;
            s_i[2] = (int)ep;
            s_i[3] = rd ? 1 : 0;
            s_ctl[0] = ep;
            s_ctl[1] = is_janitor(si, sli, nsl, a.nseg) ? 1u : 0u;
        }
        __syncthreads();
        sg = s_i[0];
        sl = s_i[1];
        epoch = (uint32_t)s_i[2];
        flags_ready = s_i[3] != 0;
        __syncthreads();
        if (sg < 0) return;   // (cannot happen: one workgroup per item)
        if (sg == 0 && sl == 0) {   // the call's first item clears the look-back flags
            clear_flags(a.ctl, a.flags, nsl * a.nseg, epoch, tid, S::NTHR);
            flags_ready = true;
        }
    } else if (sl == 0 && tid == 0) {
        a.ctl[kCtlTimeouts0] = a.ctl[kCtlTimeouts1] = 0u;   // no look-back: no timeouts
    }
    const int64_t b = sl / a.H, h = sl % a.H;
    const int64_t cbeg = sg * a.G, cend = min(cbeg + a.G, a.nchunks);
    const int64_t slot = sl * a.nseg + sg;
    const bool last_seg = (sg == a.nseg - 1);
    const bool run_agg = a.nseg > 1;     // segments are linked: aggregate pass + look-back
    const int64_t tstr = a.H;            // token stride in token-heads
    const int64_t bstr = tstr * R * N, xstr = tstr * R * P;
    const T *Bs = static_cast<const T *>(a.B);
    const T *Cs = static_cast<const T *>(a.C);
    const T *Xs = static_cast<const T *>(a.x);
    auto tok_of = [&](int64_t c) -> int64_t { return (b * a.L + c * Q) * a.H + h; };
    auto nvalid_of = [&](int64_t c) -> int { return (int)min((int64_t)Q, a.L - c * Q); };
    // The prefetch groups are issued in the same order before and inside the
    // chunk loops, so that the compiler's count of loads in flight agrees on
    // both paths into a loop and its waits stay exact.
    auto sched_fence = []() { __builtin_amdgcn_sched_barrier(0); };

    // Row blocks: fetch() issues the global loads of B and x rows into
    // registers, commit() rotates B^ = R(-psi_t) B and writes it to LDS
    // row-major (operand of G^T and, read transposed, of M), together with
    // W x (operand of M) and, in the output pass, x.  Consecutive lanes take
    // consecutive rows, so the cos/sin table reads are conflict-free.
    constexpr int TB = S::JB * (NH / S::CE) / S::NTHR;   // B tasks per thread
    constexpr int TX = S::JB * (P / S::CE) / S::NTHR;    // x tasks per thread
    static_assert(TB * S::NTHR == S::JB * (NH / S::CE) && TX * S::NTHR == S::JB * (P / S::CE), "tasks");
    struct Blk { V16 lo[TB], hi[TB], xv[TX]; };
    // Every load below is unconditional and goes through a buffer resource
    // that ends at the chunk's last valid token (rows past the end of the
    // sequence read as zeros), so the number of loads in flight is static and
    // the waits the compiler inserts stop at exactly the loads a step needs,
    // leaving later prefetches in flight.
    const uint32_t bstr_b = (uint32_t)(bstr * sizeof(T)), xstr_b = (uint32_t)(xstr * sizeof(T));
    auto rows_rsrc = [&](const T *base, int64_t c, int64_t str, int width) {
        const int nv = nvalid_of(c);
        return make_rsrc(base + tok_of(c) * width, (uint32_t)(((nv - 1) * str + width) * (int64_t)sizeof(T)));
    };
    auto fetch = [&](int64_t c, int jb, Blk &f) {
        const Rsrc rb = rows_rsrc(Bs, c, bstr, R * N), rx = rows_rsrc(Xs, c, xstr, R * P);
#pragma unroll
        for (int k = 0; k < TB; ++k) {
            const int task = tid + k * S::NTHR, jr = task % S::JB, cp = task / S::JB;
            const int row = jb * S::JB + jr, t = row / R, r = row % R;
            const uint32_t off = tok_off(t, bstr_b) + (uint32_t)((r * N + cp * S::CE) * sizeof(T));
            f.lo[k] = buf_load<V16>(rb, off);
            f.hi[k] = buf_load<V16>(rb, off + NH * sizeof(T));
        }
#pragma unroll
        for (int k = 0; k < TX; ++k) {
            const int task = tid + k * S::NTHR, jr = task % S::JB, pc = task / S::JB;
            const int row = jb * S::JB + jr, t = row / R, r = row % R;
            f.xv[k] = buf_load<V16>(rx, tok_off(t, xstr_b) + (uint32_t)((r * P + pc * S::CE) * sizeof(T)));
        }
    };
    // kX: also stage x itself (the output pass's operand of y)
    auto commit = [&](int jb, const Blk &f, auto kX) {
        T *sB = s_B + (jb % NBUF) * kSB, *sX = s_XW + (jb % NBUF) * kSXr, *sWX = s_XW + (NBUF + jb % NBUF) * kSXr;
#pragma unroll
        for (int k = 0; k < TB; ++k) {
            const int task = tid + k * S::NTHR, jr = task % S::JB, cp = task / S::JB;
            const int t = (jb * S::JB + jr) / R;
            V16 lo = f.lo[k], hi = f.hi[k];
            float csv[S::CE], snv[S::CE];
            cs_getn<S::CE>(&s_cs[t * LDT + cp * S::CE], csv, snv);
#pragma unroll
            for (int e = 0; e < S::CE; ++e) {
                const float u = fget(lo, e), w = fget(hi, e);
                fset(lo, e, csv[e] * u + snv[e] * w);
                fset(hi, e, csv[e] * w - snv[e] * u);
            }
            *reinterpret_cast<V16 *>(&sB[jr * S::LDN + cp * S::CE]) = lo;
            *reinterpret_cast<V16 *>(&sB[jr * S::LDN + NH + cp * S::CE]) = hi;
        }
#pragma unroll
        for (int k = 0; k < TX; ++k) {
            const int task = tid + k * S::NTHR, jr = task % S::JB, pc = task / S::JB;
            const float wt = s_w[(jb * S::JB + jr) / R];
            if constexpr (decltype(kX)::value) *reinterpret_cast<V16 *>(&sX[jr * LDP + pc * S::CE]) = f.xv[k];
            V16 wx;
#pragma unroll
            for (int e = 0; e < S::CE; ++e) fset(wx, e, wt * fget(f.xv[k], e));
            *reinterpret_cast<V16 *>(&sWX[jr * LDP + pc * S::CE]) = wx;
        }
    };
    auto load_kt = [&](const T *M, int ld, int r0, int c0) -> Frag { return scan::load_kt(M, ld, r0, c0, g, l16); };
    // M += B^T (W x) over one staged block (owned state pair-tiles)
    // (a wave's state tiles share their row tiles, wave % 4 and wave % 4 + 4:
    // each B^T fragment is loaded once for all of them, each (W x)^T
    // fragment once for both halves)
    static_assert(NW % 4 == 0, "state row tiles shared across a wave's tiles");
    auto m_block = [&](f32x4 (&ms)[PTW][2], int jb) {
        const T *sB = s_B + (jb % NBUF) * kSB, *sWX = s_XW + (NBUF + jb % NBUF) * kSXr;
        const int ntl = wave % 4;
#pragma unroll
        for (int ks = 0; ks < JK; ++ks) {
            Frag af[2];   // B^T
#pragma unroll
            for (int half = 0; half < 2; ++half) af[half] = load_kt(sB, S::LDN, ks * MM::K, (ntl + 4 * half) * 16);
#pragma unroll
            for (int m2 = 0; m2 < PTW; ++m2) {
                const int pt = (wave + NW * m2) / 4;
                const Frag bf = load_kt(sWX, LDP, ks * MM::K, pt * 16);   // (W x)^T
#pragma unroll
                for (int half = 0; half < 2; ++half) ms[m2][half] = MM::mma(af[half], bf, ms[m2][half]);
            }
        }
    };

    // Prologue inputs of a chunk, loaded one chunk ahead (raw values only, so
    // that nothing waits for them before the prologue itself).  Lanes are
    // tokens (TPL consecutive tokens per lane); wave w owns angle pairs
    // w*PPW .. w*PPW + PPW-1.
    constexpr int TPL = Q > kWave ? Q / kWave : 1;   // tokens per lane
    constexpr int PPW = NH / NW;                     // angle pairs per wave
    static_assert(TPL * kWave >= Q && PPW % 4 == 0, "prologue layout");
    struct Pro { f32x4 th[TPL][PPW / 4]; float dtv[TPL], lamv[TPL], Av[TPL], dtn[TPL], lamn[TPL]; };
    // Tokens past the end of the sequence read as zeros; the dt and lambda
    // ranges extend to the next chunk's first token when there is one.
    auto load_pro = [&](int64_t c, Pro &p) {
        const int64_t tk = tok_of(c);
        const int nv = nvalid_of(c);
        const int nvn = nv + (c * Q + nv < a.L ? 1 : 0);
        // per-head frequencies: every token reads the head's omega row
        const Rsrc rth = a.theta_ph ? make_rsrc(a.theta + h * NH, (uint32_t)(NH * 4))
                                    : make_rsrc(a.theta + tk * NH, (uint32_t)(((nv - 1) * tstr + 1) * NH * 4));
        const Rsrc rdt = make_rsrc(a.dt + tk, (uint32_t)(((nvn - 1) * tstr + 1) * 4));
        const Rsrc rlam = make_rsrc(a.lam + tk, (uint32_t)(((nvn - 1) * tstr + 1) * 4));
        const uint32_t thstr_b = a.theta_ph ? 0u : (uint32_t)(tstr * NH * 4), tstr_b = (uint32_t)(tstr * 4);
#pragma unroll
        for (int u = 0; u < TPL; ++u) {
            const int t = lane * TPL + u;
            const uint32_t oth = tok_off(t, thstr_b) + wave * PPW * 4;
#pragma unroll
            for (int q = 0; q < PPW / 4; ++q) p.th[u][q] = buf_load<f32x4>(rth, oth + 16 * q);
            const uint32_t o = tok_off(t, tstr_b);
            p.dtv[u] = buf_load<float>(rdt, o);
            p.lamv[u] = buf_load<float>(rlam, o);
            p.dtn[u] = buf_load<float>(rdt, o + tstr_b);
            p.lamn[u] = buf_load<float>(rlam, o + tstr_b);
            p.Av[u] = a.A[b * a.a_sb + (c * Q + min(t, nv - 1)) * a.a_st + h * a.a_sh];
        }
    };
    // cum, gamma, sigma, w (wave 0 publishes them) and the angle prefix sums,
    // the cos/sin table and psi_e of each wave's pairs: lane prefix sums over
    // tokens (wavefront scans), no LDS round trip.  Ends with the one barrier.
    auto prologue = [&](int64_t c, const Pro &p) {
        const int nv = nvalid_of(c);
        s_cum = s_cumb[c & 1];
        s_psie = s_psieb[c & 1];
        // dt and lambda read as zero past the end of the sequence, so
        // sigma_{L-1} = gamma_{L-1} and rows past the end carry zeros
        Acc cumv[TPL];
        float gamv[TPL], sigv[TPL];
        {
            Acc lg[TPL], loc = 0;
#pragma unroll
            for (int u = 0; u < TPL; ++u) {
                lg[u] = (Acc)p.dtv[u] * (Acc)p.Av[u];
                loc += lg[u];
                gamv[u] = p.lamv[u] * p.dtv[u];
                sigv[u] = gamv[u] + (1.f - p.lamn[u]) * p.dtn[u];
            }
            Acc cum = lane_scan(loc) - loc;   // exclusive over lanes
#pragma unroll
            for (int u = 0; u < TPL; ++u) {
                cum += lg[u];
                cumv[u] = cum;
            }
        }
        if (wave == 0) {
            // cum_e = cum of token nv - 1
            Acc cum_e = cumv[0];
#pragma unroll
            for (int u = 1; u < TPL; ++u) cum_e = ((nv - 1) % TPL == u) ? cumv[u] : cum_e;
            cum_e = lane_bcast(cum_e, (nv - 1) / TPL);
#pragma unroll
            for (int u = 0; u < TPL; ++u) {
                const int t = lane * TPL + u;
                if (t < Q) {
                    s_cum[t] = cumv[u];
                    s_gam[t] = gamv[u];
                    s_sig[t] = sigv[u];
                    s_w[t] = (t < nv) ? (float)(exp_fast(cum_e - cumv[u]) * (Acc)sigv[u]) : 0.f;
                }
            }
        }
        if constexpr (kWTab) {   // wave w fills rows w*Q/NW ..; lane j is column j
            static_assert(TPL == 1 && Q % NW == 0, "weight table layout");
            const float cum_j = (float)cumv[0], sig_j = sigv[0];
#pragma unroll
            for (int k = 0; k < Q / NW; ++k) {
                const int t = wave * (Q / NW) + k;
                const float cum_t = (float)lane_bcast(cumv[0], t), gam_t = lane_bcast(gamv[0], t);
                const float e = exp_fast(fminf(cum_t - cum_j, 0.f)) * sig_j;
                if (lane < Q) s_W[t * LDW + lane] = lane < t ? e : (lane == t ? gam_t : 0.f);
            }
        }
        float csv[TPL][PPW], snv[TPL][PPW];
        // angle of each lane token: theta, or dt * omega (zero past the end)
        float tsc[TPL];
#pragma unroll
        for (int u = 0; u < TPL; ++u) tsc[u] = a.theta_ph ? (lane * TPL + u < nv ? p.dtv[u] : 0.f) : 1.f;
#pragma unroll
        for (int k = 0; k < PPW; ++k) {
            const int i = wave * PPW + k;
            Acc th[TPL], loc = 0;
#pragma unroll
            for (int u = 0; u < TPL; ++u) {
                th[u] = (Acc)(p.th[u][k / 4][k % 4] * tsc[u]);   // zero past the end of the sequence
                loc += th[u];
            }
            Acc psi = lane_scan(loc) - loc;
#pragma unroll
            for (int u = 0; u < TPL; ++u) {
                const int t = lane * TPL + u;
                psi += th[u];
                Acc sn, cs;
                sincos_fast(psi, &sn, &cs);
                csv[u][k] = (float)cs;
                snv[u][k] = (float)sn;
                if (t == nv - 1) s_psie[i] = psi;
            }
        }
#pragma unroll
        for (int u = 0; u < TPL; ++u) {
            const int t = lane * TPL + u;
            if (t < Q) cs_putn<PPW>(&s_cs[t * LDT + wave * PPW], csv[u], snv[u]);
        }
        __syncthreads();
    };
    // Owned state element (m2, half, v): row n = 16*(ntl + 4*half) + 4g + v,
    // column p = 16*pt + l16; rows (i, i + N/2) of a pair sit in one lane.
    // X <- R(psi_e)(de X + M) with this chunk's psi_e.
    auto chunk_update = [&](float (&X)[PTW][2][4], const f32x4 (&ms)[PTW][2], Acc de) {
#pragma unroll
        for (int m2 = 0; m2 < PTW; ++m2) {
            const int ntl = (wave + NW * m2) % 4;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                Acc sn, cs;
                sincos_fast(s_psie[ntl * 16 + 4 * g + v], &sn, &cs);
                const Acc re = de * (Acc)X[m2][0][v] + (Acc)ms[m2][0][v];
                const Acc im = de * (Acc)X[m2][1][v] + (Acc)ms[m2][1][v];
                X[m2][0][v] = (float)(cs * re - sn * im);
                X[m2][1][v] = (float)(sn * re + cs * im);
            }
        }
    };
    // X <- R(psi_e) M (the output pass's accumulator already holds e^{cum_e} S + M)
    auto rotate_psie = [&](const f32x4 (&ms)[PTW][2], float (&X)[PTW][2][4]) {
#pragma unroll
        for (int m2 = 0; m2 < PTW; ++m2) {
            const int ntl = (wave + NW * m2) % 4;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                Acc sn, cs;
                sincos_fast(s_psie[ntl * 16 + 4 * g + v], &sn, &cs);
                const Acc re = ms[m2][0][v], im = ms[m2][1][v];
                X[m2][0][v] = (float)(cs * re - sn * im);
                X[m2][1][v] = (float)(sn * re + cs * im);
            }
        }
    };
    const int64_t SZ = (int64_t)N * P;
    auto write_final = [&](const float (&X)[PTW][2][4]) {
        float *fs = a.final_state + sl * SZ;
#pragma unroll
        for (int m2 = 0; m2 < PTW; ++m2) {
            const int k = wave + NW * m2, ntl = k % 4, pt = k / 4;
#pragma unroll
            for (int half = 0; half < 2; ++half)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    fs[(16 * (ntl + 4 * half) + 4 * g + v) * P + pt * 16 + l16] = X[m2][half][v];
        }
        T *cB = static_cast<T *>(a.cB) + sl * (R * N);
        T *cX = static_cast<T *>(a.cX) + sl * (R * P);
        const int64_t kl = (b * a.L + a.L - 1) * a.H + h;
        const T *Bl = Bs + kl * (R * N);
        const T *Xl = Xs + kl * (R * P);
        for (int e = tid; e < R * N; e += S::NTHR) cB[e] = Bl[e];
        for (int e = tid; e < R * P; e += S::NTHR) cX[e] = Xl[e];
    };
    // Initial state plus the carried previous-input term of token 0 (owned)
    auto load_init = [&](float (&Si)[PTW][2][4]) {
        const float *ist = a.init_state ? a.init_state + sl * SZ : nullptr;
        float wb = 0.f;
        if (a.init_cB) {
            const int64_t k0 = (b * a.L) * a.H + h;
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

    using True = std::integral_constant<bool, true>;
    using False = std::integral_constant<bool, false>;
    constexpr int DA = NJB < 4 ? NJB : 4;   // blocks in flight, aggregate pass
    constexpr int DC = 1;                   // blocks in flight, output pass
    Blk ring[DA];
    Pro pro;
    float Sst[PTW][2][4];                   // state entering the current chunk

    // ---- 2. aggregate pass, look-back, segment state ----
    if (run_agg) {
        float Aseg[PTW][2][4];
#pragma unroll
        for (int m2 = 0; m2 < PTW; ++m2)
#pragma unroll
            for (int v = 0; v < 4; ++v) Aseg[m2][0][v] = Aseg[m2][1][v] = 0.f;
        Acc seg_lg = 0, segps = 0;
        load_pro(cbeg, pro);
        sched_fence();
#pragma unroll
        for (int d = 0; d < DA; ++d) fetch(cbeg, d, ring[d]);
        sched_fence();
        for (int64_t c = cbeg; c < cend; ++c) {
            relane();
            prologue(c, pro);
            sched_fence();
            load_pro(min(c + 1, cend - 1), pro);
            sched_fence();
            f32x4 ms[PTW][2];
#pragma unroll
            for (int m2 = 0; m2 < PTW; ++m2) ms[m2][0] = ms[m2][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int jb = 0; jb < NJB; ++jb) {
                commit(jb, ring[jb % DA], False{});
                __syncthreads();
                {
                    const int jn = jb + DA;
                    sched_fence();
                    fetch(min(c + jn / NJB, cend - 1), jn % NJB, ring[jb % DA]);
                    sched_fence();
                }
                m_block(ms, jb);
                __syncthreads();
            }
            const Acc cum_e = s_cum[nvalid_of(c) - 1];
            chunk_update(Aseg, ms, exp_fast(cum_e));
            seg_lg += cum_e;
            if (tid < NH) {
                segps += s_psie[tid];
                if constexpr (sizeof(Acc) == 4) segps = reduce_angle(segps);
            }
        }
        if (tid < NH) s_segps[tid] = segps;
        __syncthreads();

        auto word_index = [&](int m2, int half, int vp) -> int64_t {
            return (int64_t)((m2 * 2 + half) * 2 + vp) * S::NTHR + tid;
        };
        Acc *totp = static_cast<Acc *>(a.tot);
        bool flags_lost = false;   // the wait for cleared flags gave up (error path)
        if (!flags_ready) {
            if (tid == 0) s_i[0] = wait_flags_ready(a.ctl, s_ctl[0], a.spin_max) ? 0 : 1;
            __syncthreads();
            flags_lost = s_i[0] != 0;
            __syncthreads();
        }
        if (sg > 0 && !last_seg && !flags_lost) {   // publish the aggregate (only successors read it)
            unsigned long long *dst = reinterpret_cast<unsigned long long *>(a.agg + slot * SZ);
#pragma unroll
            for (int m2 = 0; m2 < PTW; ++m2)
#pragma unroll
                for (int half = 0; half < 2; ++half)
#pragma unroll
                    for (int vp = 0; vp < 2; ++vp)
                        st_coh2(dst + word_index(m2, half, vp), Aseg[m2][half][2 * vp], Aseg[m2][half][2 * vp + 1]);
            if (tid == 0) st_coh(totp + slot * (NH + 1), seg_lg);
            if (tid < NH) st_coh(totp + slot * (NH + 1) + 1 + tid, s_segps[tid]);
            wait_stores_done();
            __syncthreads();
            if (tid == 0) __hip_atomic_store(a.flags + slot, kFlagAgg, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }

        // Entering state of the segment: the nearest preceding segment whose
        // inclusive state is published (or the sequence start) is found first,
        // waiting on any segment in between that has published nothing yet;
        // the aggregates after it are then folded forward, S <- T_k S + A_k,
        // with the arithmetic their owners use for their own inclusive states
        // (state_step): the result does not depend on timing.
        const int ntl_w = wave % 4;   // all owned pair rows of a lane are 16 ntl_w + 4g + v
        if (sg == 0) {
            load_init(Sst);
        } else {
            const int64_t sbase = sl * a.nseg;
            int64_t j = sg - 1;       // next predecessor to probe
            int64_t jt = flags_lost ? sg - 1 : -2;   // terminal: -1 sequence start, >= 0 inclusive state
            bool timed_out = flags_lost;
            while (jt == -2) {
                if (wave == 0) {   // probe predecessors j, j-1, ..., j-15 at once
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
                } else if (needwait) {   // segment j - adv has published nothing: wait for it
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
                    if (timed_out) jt = sg - 1;   // (error path: the entering state is NaN)
                } else {
                    j -= kProbe;                 // sixteen aggregates: probe further back
                }
            }
            if (timed_out) {   // y of this segment and of every later one, and the final state, become NaN
#pragma unroll
                for (int m2 = 0; m2 < PTW; ++m2)
#pragma unroll
                    for (int v = 0; v < 4; ++v) Sst[m2][0][v] = Sst[m2][1][v] = __builtin_nanf("");
            } else if (jt < 0) {
                load_init(Sst);
            } else {
                const unsigned long long *src = reinterpret_cast<const unsigned long long *>(a.inc + (sbase + jt) * SZ);
#pragma unroll
                for (int m2 = 0; m2 < PTW; ++m2)
#pragma unroll
                    for (int half = 0; half < 2; ++half)
#pragma unroll
                        for (int vp = 0; vp < 2; ++vp)
                            ld_coh2(src + word_index(m2, half, vp), Sst[m2][half][2 * vp], Sst[m2][half][2 * vp + 1]);
            }
            // Fold forward from the terminal, one aggregate a round trip; each round
            // also probes the nearest predecessors, and an inclusive state published
            // meanwhile replaces the rest of the fold (it is that fold: same bits).
            for (int64_t k = jt; k < sg - 1;) {
                if (wave == 0) {
                    const int64_t jj = sg - 1 - lane;
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
                if (near >= 0) {   // inclusive state of predecessor sg - 1 - near: continue from it
                    k = sg - 1 - near;
                    const unsigned long long *isrc = reinterpret_cast<const unsigned long long *>(a.inc + (sbase + k) * SZ);
#pragma unroll
                    for (int m2 = 0; m2 < PTW; ++m2)
#pragma unroll
                        for (int half = 0; half < 2; ++half)
#pragma unroll
                            for (int vp = 0; vp < 2; ++vp)
                                ld_coh2(isrc + word_index(m2, half, vp), Sst[m2][half][2 * vp], Sst[m2][half][2 * vp + 1]);
                    continue;
                }
                k = kn;
                const Acc de = exp_fast(cm);
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    Acc sn, cs;
                    sincos_fast(ps[v], &sn, &cs);
#pragma unroll
                    for (int m2 = 0; m2 < PTW; ++m2)
                        state_step(Sst[m2][0][v], Sst[m2][1][v], de, cs, sn, d[m2][0][v], d[m2][1][v]);
                }
            }
        }

        // outgoing state of the segment: e^{seg_lg} R(segps) S + A (the same
        // step a successor's fold takes)
        {
            float Sout[PTW][2][4];
            const Acc de = exp_fast(seg_lg);
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                Acc sn, cs;
                sincos_fast(s_segps[ntl_w * 16 + 4 * g + v], &sn, &cs);
#pragma unroll
                for (int m2 = 0; m2 < PTW; ++m2) {
                    Sout[m2][0][v] = Sst[m2][0][v];
                    Sout[m2][1][v] = Sst[m2][1][v];
                    state_step(Sout[m2][0][v], Sout[m2][1][v], de, cs, sn, Aseg[m2][0][v], Aseg[m2][1][v]);
                }
            }
            if (!last_seg && !flags_lost) {
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
            } else if (last_seg) {
                write_final(Sout);
            }
        }
    } else {
        load_init(Sst);
    }

    // ---- 3. output pass over the segment's chunks ----
    Frag cf[TPW][NK];
    auto load_cf = [&](int64_t c) {
        if (!ow) return;
        const Rsrc rc = rows_rsrc(Cs, c, bstr, R * N);
#pragma unroll
        for (int m = 0; m < TPW; ++m) {
            const int row = owned_tile<S>(wt, m) * 16 + l16, t = row / R, r = row % R;
            const uint32_t off = tok_off(t, bstr_b) + (uint32_t)((r * N + MM::KPL * g) * sizeof(T));
#pragma unroll
            for (int kk = 0; kk < NK; ++kk) cf[m][kk] = buf_load<Frag>(rc, off + kk * MM::K * sizeof(T));
        }
    };
    load_pro(cbeg, pro);
    sched_fence();
#pragma unroll
    for (int d = 0; d < DC; ++d) fetch(cbeg, d, ring[d]);
    sched_fence();
    load_cf(cbeg);
    sched_fence();
    const float Dh = a.D[h];
    for (int64_t c = cbeg; c < cend; ++c) {
        relane();
        const int nv = nvalid_of(c);
        const int64_t tk = tok_of(c);
        // the state leaving this chunk is needed inside the segment, or as the
        // final state when no aggregate pass produced it
        const bool chain = (c + 1 < cend) || (!run_agg && c == a.nchunks - 1);
        prologue(c, pro);
        sched_fence();
        load_pro(min(c + 1, cend - 1), pro);
        sched_fence();
        // C^ fragments of the owned row tiles, rotated by -psi_t (rows past the
        // end of the sequence were loaded as zeros)
#pragma unroll
        for (int m = 0; m < TPW; ++m) {
            if (!ow) break;
            const int row = owned_tile<S>(wt, m) * 16 + l16, t = row / R;
#pragma unroll
            for (int kk = 0; kk < NK / 2; ++kk) {
                float csv[MM::KPL], snv[MM::KPL];
                cs_getn<MM::KPL>(&s_cs[t * LDT + kk * MM::K + MM::KPL * g], csv, snv);
#pragma unroll
                for (int e = 0; e < MM::KPL; ++e) {
                    const float u = fget(cf[m][kk], e), w = fget(cf[m][kk + NK / 2], e);
                    fset(cf[m][kk], e, csv[e] * u + snv[e] * w);
                    fset(cf[m][kk + NK / 2], e, csv[e] * w - snv[e] * u);
                }
            }
        }
        // S^T in the io dtype (the last B^ buffer) for the inter-chunk term
        T *s_S = s_B + (NBUF - 1) * kSB;
#pragma unroll
        for (int m2 = 0; m2 < PTW; ++m2) {
            const int k = wave + NW * m2, ntl = k % 4, pt = k / 4;
#pragma unroll
            for (int half = 0; half < 2; ++half)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    s_S[(pt * 16 + l16) * S::LDN + 16 * (ntl + 4 * half) + 4 * g + v] = from_f32<T>(Sst[m2][half][v]);
        }
        if constexpr (NBUF == 2) {   // the first block stages beside S^T
            commit(0, ring[0], True{});
            sched_fence();
            fetch(min(c + 1 / NJB, cend - 1), 1 % NJB, ring[0]);
            sched_fence();
        }
        __syncthreads();
        // inter-chunk term e^{cum_t} C^_t . S starts the accumulators.  The
        // output tiles are transposed (y^T = S^T C^T, y^T += x^T (w o G)^T):
        // lane l holds row l % 16 of a tile and four consecutive columns.
        f32x4 acc[TPW][PTS];
#pragma unroll
        for (int m = 0; m < TPW; ++m) {
            if (!ow) break;
            const int TT = owned_tile<S>(wt, m);
            const float ecum = (float)exp_fast(s_cum[(TT * 16 + l16) / R]);
#pragma unroll
            for (int pt = 0; pt < PTS; ++pt) {
                f32x4 tmp = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kk = 0; kk < NK; ++kk)
                    tmp = MM::mma(MM::load(&s_S[((pofs + pt) * 16 + l16) * S::LDN + kk * MM::K + MM::KPL * g]), cf[m][kk], tmp);
#pragma unroll
                for (int v = 0; v < 4; ++v) tmp[v] *= ecum;
                acc[m][pt] = tmp;
            }
        }
        __syncthreads();   // S^T read: the B^ block is rewritten below
        // y leaves in 16-byte pieces of the wave's columns of its rows (NPC
        // per lane and owned tile); with the gate, the matching pieces of z
        // are loaded now and arrive during the intra-chunk products
        constexpr int RP = PTS * 16 / S::CE;        // 16-byte pieces of a row per wave
        constexpr int NPC = (16 * RP + kWave - 1) / kWave;
        V16 zp[kGate ? TPW : 1][NPC];
        if constexpr (kGate) {
            const Rsrc rz = rows_rsrc(static_cast<const T *>(a.z), c, xstr, R * P);
#pragma unroll
            for (int m = 0; m < TPW; ++m)
#pragma unroll
                for (int i = 0; i < NPC; ++i) {
                    const int k = min(lane + i * kWave, 16 * RP - 1), rl = k / RP, col = (k % RP) * S::CE;
                    const int row = owned_tile<S>(wt, m) * 16 + rl, t = row / R, r = row % R;
                    zp[m][i] = buf_load<V16>(rz, tok_off(t, xstr_b) + (uint32_t)((r * P + pofs * 16 + col) * sizeof(T)));
                }
        }
        // the state accumulator starts as e^{cum_e} S and collects M
        f32x4 ms[PTW][2];
        if (chain) {
            const float de = (float)exp_fast(s_cum[nv - 1]);
#pragma unroll
            for (int m2 = 0; m2 < PTW; ++m2)
#pragma unroll
                for (int half = 0; half < 2; ++half)
#pragma unroll
                    for (int v = 0; v < 4; ++v) ms[m2][half][v] = de * Sst[m2][half][v];
        }
#pragma unroll
        for (int jb = 0; jb < NJB; ++jb) {
            if constexpr (NBUF == 2) {   // stage the next block while this one feeds the MFMAs
                if (jb + 1 < NJB) {
                    commit(jb + 1, ring[0], True{});
                    const int jn = jb + 2;
                    sched_fence();
                    fetch(min(c + jn / NJB, cend - 1), jn % NJB, ring[0]);
                    sched_fence();
                }
            } else {
                commit(jb, ring[jb % DC], True{});
                __syncthreads();
                const int jn = jb + DC;
                sched_fence();
                fetch(min(c + jn / NJB, cend - 1), jn % NJB, ring[jb % DC]);
                sched_fence();
            }
            const T *sBc = s_B + (jb % NBUF) * kSB, *sXc = s_XW + (jb % NBUF) * kSXr;
            // Owned tile m lies in rows 16 m NWO .. 16 (m + 1) NWO - 1: tiles
            // whose blocks all come before block jb have no work in it, tiles
            // whose blocks all come after it take every pair unmasked; only
            // the others compare rows.
            auto tile_above = [&](int m) { return ((m + 1) * S::NWO - 1) / 4 < jb; };
            auto tile_below = [&](int m) { return (m * S::NWO) / 4 > jb; };
#pragma unroll
            for (int jp = 0; jp < S::JB / 32; ++jp) {
                const int J0 = jb * 4 + 2 * jp;        // first j-tile of the pair (chunk-global)
                if (!ow) break;
                if (J0 > owned_tile<S>(wt, TPW - 1) && J0 > owned_tile<S>(wt, 0)) continue;
                // x^T columns of the pair, shared by all owned tiles
                bf16x8 xf[PTS];
                if constexpr (MM::KPL == 8) {
#pragma unroll
                    for (int pt = 0; pt < PTS; ++pt) {
                        // rows 32 jp + 4g .. +3 and 32 jp + 16 + 4g .. +3 of x, column l16
                        const T *xr = &sXc[(32 * jp + 4 * g + l16 / 4) * LDP + (pofs + pt) * 16 + 4 * (l16 % 4)];
                        const bf16x4 lo = lds_tr4(xr), hi = lds_tr4(xr + 16 * LDP);
#pragma unroll
                        for (int v = 0; v < 4; ++v) { xf[pt][v] = lo[v]; xf[pt][4 + v] = hi[v]; }
                    }
                }
                // G^T tiles (K = N) for every owned tile at or below the pair
                f32x4 gt[TPW][2];
#pragma unroll
                for (int m = 0; m < TPW; ++m) gt[m][0] = gt[m][1] = f32x4{0.f, 0.f, 0.f, 0.f};
                // (the pair's B^ fragments are loaded before the MFMAs, whose
                // per-tile conditions split the code into small blocks)
                Frag bfr[2][NK];
#pragma unroll
                for (int q = 0; q < 2; ++q)
#pragma unroll
                    for (int kk = 0; kk < NK; ++kk)
                        bfr[q][kk] = MM::load(&sBc[((2 * jp + q) * 16 + l16) * S::LDN + kk * MM::K + MM::KPL * g]);
#pragma unroll
                for (int q = 0; q < 2; ++q)
#pragma unroll
                    for (int kk = 0; kk < NK; ++kk) {
#pragma unroll
                        for (int m = 0; m < TPW; ++m)
                            if (!tile_above(m) && (tile_below(m) || J0 + q <= owned_tile<S>(wt, m)))
                                gt[m][q] = MM::mma(bfr[q][kk], cf[m][kk], gt[m][q]);
                    }
                // mask weights (branch-free): w_tj = e^{cum_t - cum_j} sigma_j (j < t),
                // gamma_t (j = t), 0 (j > t); D x_t as D on the diagonal row = column
#pragma unroll
                for (int m = 0; m < TPW; ++m) {
                    const int TT = owned_tile<S>(wt, m);
                    if (tile_above(m) || (!tile_below(m) && J0 > TT)) continue;
                    const int tt = (TT * 16 + l16) / R;
                    constexpr int NV = R >= 4 ? 1 : 4 / R;
#pragma unroll
                    for (int q = 0; q < 2; ++q) {
                        float wv[NV];
#pragma unroll
                        for (int u = 0; u < NV; ++u) {
                            const int tj = ((J0 + q) * 16 + 4 * g + u * R) / R;
                            if constexpr (kWTab) {
                                wv[u] = s_W[tt * LDW + tj];
                            } else {
                                const float cum_t = (float)s_cum[tt], gam_t = s_gam[tt];
                                const float e = exp_fast(fminf(cum_t - (float)s_cum[tj], 0.f)) * s_sig[tj];
                                wv[u] = (tile_below(m) || tj < tt) ? e : (tj == tt ? gam_t : 0.f);
                            }
                        }
#pragma unroll
                        for (int v = 0; v < 4; ++v) gt[m][q][v] *= wv[(v * NV) / 4];
                        if (!tile_below(m) && J0 + q == TT) {
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
                        for (int pt = 0; pt < PTS; ++pt) acc[m][pt] = MM::mma(xf[pt], af, acc[m][pt]);
                    } else {
#pragma unroll
                        for (int q = 0; q < 2; ++q)
#pragma unroll
                            for (int v = 0; v < 4; ++v)
#pragma unroll
                                for (int pt = 0; pt < PTS; ++pt) {
                                    const float xv = to_f32(sXc[(32 * jp + 16 * q + 4 * g + v) * LDP + (pofs + pt) * 16 + l16]);
                                    acc[m][pt] = MM::mma(xv, gt[m][q][v], acc[m][pt]);
                                }
                    }
                }
            }
            // M of this block for the state, once the G^T operands are dead
            __builtin_amdgcn_sched_barrier(0);
            if (chain) m_block(ms, jb);
            __syncthreads();   // staged block read: the next commit may overwrite it
        }
        sched_fence();
        load_cf(min(c + 1, cend - 1));
        sched_fence();
        if (chain) {
            rotate_psie(ms, Sst);
            if (c == a.nchunks - 1) write_final(Sst);
        }
        // store: each wave stages its tiles in its own part of the x / W x
        // buffers, free after the last block's barrier (a wave's LDS accesses
        // execute in order: no barrier), and writes whole 16-byte pieces of
        // its columns of the y rows
        T *s_y = s_XW + wave * (16 * LDP);
        T *Yg = static_cast<T *>(a.y) + tk * (R * P);
#pragma unroll
        for (int m = 0; m < TPW; ++m) {
            if (!ow) break;
            const int TT = owned_tile<S>(wt, m);
#pragma unroll
            for (int pt = 0; pt < PTS; ++pt) store4(&s_y[l16 * LDP + pt * 16 + 4 * g], acc[m][pt]);
            asm volatile("" ::: "memory");
#pragma unroll
            for (int i = 0; i < NPC; ++i) {
                const int k = lane + i * kWave, rl = k / RP, col = (k % RP) * S::CE;
                const int row = TT * 16 + rl, t = row / R, r = row % R;
                if (k < 16 * RP && t < nv) {
                    V16 yv = *reinterpret_cast<const V16 *>(&s_y[rl * LDP + col]);
                    if constexpr (kGate) yv = gate_piece<T>(yv, zp[m][i]);
                    *reinterpret_cast<V16 *>(Yg + t * xstr + r * P + pofs * 16 + col) = yv;
                }
            }
            asm volatile("" ::: "memory");
        }
    }
    if (run_agg && tid == 0 && s_ctl[1]) janitor_reset(a.ctl, nsl, a.nseg, s_ctl[0], a.spin_max);
}

template <typename T, int Q, int R>
hipError_t launch_seg(const ScanArgs &a0, hipStream_t stream) {
    typedef SegShape<T, Q, R> S;
    static int cap_cache[2][64];
    ScanArgs a = a0;
    const bool gate = a.z != nullptr;
    const void *kfn = gate ? reinterpret_cast<const void *>(&k_scan_seg<T, Q, R, true>)
                           : reinterpret_cast<const void *>(&k_scan_seg<T, Q, R, false>);
    const int64_t nsl = a.batch * a.H;
    int64_t G = a.G;
    if (G <= 0) {   // one resident wave of workgroups covers the whole scan
        const int cap = resident_capacity(kfn, S::NTHR, cap_cache[gate ? 1 : 0]);
        if (cap <= 0) return hipErrorInvalidDevice;
        G = (nsl * a.nchunks + cap - 1) / cap;
        // Short chunks (fewer than 128 rows) split over several segments run
        // faster one chunk per workgroup: the aggregate pass and the per-chunk
        // fixed costs of a segment then outweigh what it saves.  So do chunks
        // of 64 or more tokens in scans of at least 16384 chunk items, where
        // the per-chunk kernel's single pass over each chunk pays off.
        if (G < a.nchunks && a.per_chunk &&
            (S::QR < 128 || (Q >= 64 && nsl * a.nchunks >= 16384)))
            return a.per_chunk(a0, stream);
    }
    G = G < 1 ? 1 : (G > a.nchunks ? a.nchunks : G);
    a.G = G;
    a.nseg = (a.nchunks + G - 1) / G;
    // one segment per slice: the warp-specialised kernel, where built
    if (a.nseg == 1 && std::is_same<T, bf16>::value) {
        if (scan_launch_fn f = a.pro.on ? find_ws_pro_impl(1, S::N, S::P, R, Q) : find_ws_impl(1, S::N, S::P, R, Q))
            return f(a, stream);
    }
    if (a.pro.on) return a.per_chunk ? a.per_chunk(a0, stream) : hipErrorInvalidValue;   // (no prologue here)
    if (gate)
        hipLaunchKernelGGL((k_scan_seg<T, Q, R, true>), dim3((unsigned)(nsl * a.nseg)), dim3(S::NTHR), 0, stream, a);
    else
        hipLaunchKernelGGL((k_scan_seg<T, Q, R, false>), dim3((unsigned)(nsl * a.nseg)), dim3(S::NTHR), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

#define M3_SEG_SHAPES(X)     \
    X(0, float, 2, 32)       \
    X(0, float, 4, 16)       \
    X(0, float, 4, 32)       \
    X(1, bf16, 1, 64)        \
    X(1, bf16, 1, 128)       \
    X(1, bf16, 2, 32)        \
    X(1, bf16, 2, 64)        \
    X(1, bf16, 2, 128)       \
    X(1, bf16, 4, 32)        \
    X(1, bf16, 4, 64)

scan_launch_fn find_seg_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q) {
    if (N != 128 || P != 64) return nullptr;
#define M3_CASE(IO, T, R_, Q_) \
    if (io == IO && R == R_ && Q == Q_) return &launch_seg<T, Q_, R_>;
    M3_SEG_SHAPES(M3_CASE)
#undef M3_CASE
    return nullptr;
}

}  // namespace m3
