// Warp-specialised prefill scan of the Mamba-3 SSM on gfx950 (N = 128,
// P = 64, bf16 operands), one workgroup per (batch, head) slice carrying the
// state through all of the slice's chunks.
//
// Chunk math (Sec. 3.3 chunked algorithm, the two-band mask of Sec. 3.1.2
// eq. mamba3-mask, the rotary form of Sec. 3.2): with chunk-local prefix sums
// cum_t (of dt A) and psi_t (of theta), C^_t = R(-psi_t) C_t,
// B^_j = R(-psi_j) B_j, w_tt = gamma_t, w_tj = e^{cum_t - cum_j} sigma_j,
//   y_t = sum_{j<=t} w_tj (C^_t . B^_j) x_j + e^{cum_t} C^_t . S + D x_t,
//   S  <-  R(psi_e) (e^{cum_e} S + M),   M = sum_j e^{cum_e - cum_j} sigma_j B^_j x_j^T.
//
// The eight waves take two roles, one wave of each on every SIMD (waves w and
// w + 4 share a SIMD), so that the two roles' work can overlap there (the
// outputs are MFMA-heavy, the staging and prologue VALU-heavy):
//   output waves (0-3) own 16-row output tiles: they rotate their C rows,
//     form y = e^{cum_t} C^ S and, per staged row block, the masked
//     G^T = B^ C^T, y += (w o G) x, and store y;
//   state waves (4-7) own the N x P state: they compute each chunk's
//     prologue (decay and angle prefix scans, cos/sin table) one chunk ahead,
//     stage the row blocks (B^ rotated, x, W x) one block ahead, accumulate
//     M = B^T (W x) per block and update the state at the end of the chunk.
// A chunk is four steps (one per 64-row block) separated by workgroup
// barriers; both roles pass the same barriers.
//
// With the block prologue (Sec. 3.4 "BCNorm" and "B, C Biases"; App. "MIMO for
// Mamba-3", structured MIMO input and gate) the rows are transformed as they
// arrive, from per-head tables in LDS: the state waves normalise and bias B
// while staging it and scale x' by W_X; the output waves normalise and bias C
// inside its rotation, scale z' by W_Z and apply the optional output norm at
// the store.
#include <type_traits>

#include "m3_device.h"
#include "m3_internal.h"
#include "m3_scan_common.h"

namespace m3 {
namespace {

using namespace scan;

template <int Q_, int R_>
struct WsShape {
    static constexpr int N = 128, P = 64, NH = 64, Q = Q_, R = R_;
    static constexpr int QR = Q * R, RT = QR / 16;     // 16-row tiles of a chunk
    static constexpr int NW = 8, NTHR = NW * kWave;
    static constexpr int NWO = 4;                      // output waves
    static constexpr int NSW = NW - NWO;               // state waves
    static constexpr int NST = NSW * kWave;            // state threads
    static constexpr int TPW = RT / NWO;               // row tiles per output wave
    static constexpr int JB = 64, NJB = QR / JB;       // staged row blocks
    static constexpr int PAD = 8;                      // bf16 elements (16 bytes)
    static constexpr int LDN = N + PAD, LDP = P + PAD;
    static constexpr int CE = 8;                       // bf16 per 16-byte vector
    static constexpr int PPW = NH / NSW;               // angle pairs per state wave
    static_assert(Q == kWave, "prologue: one token per lane");
    static_assert(TPW == NJB, "output tile m lies in row block m");
    static_assert(16 % R == 0, "row tiles hold whole tokens");
    static_assert(PPW == 16, "prologue parts");
};

// kGate: the stored y is multiplied by SiLU(z) (the block's output gate).
// kPro: the block prologue (B and C: RMS norm over N, gain, bias; x and z:
// X = W_X o X', Z = W_Z o Z'; the output norm).
template <int Q, int R, bool kGate, bool kPro>
__global__ __launch_bounds__(512, 1)
void k_scan_ws(ScanArgs a) {
    typedef bf16 T;
    typedef WsShape<Q, R> S;
    typedef Mma<T> MM;
    typedef MM::frag Frag;
    typedef bf16x8 V16;
    typedef h2 CS;
    constexpr int N = S::N, P = S::P, NH = S::NH, TPW = S::TPW, NJB = S::NJB;
    constexpr int LDN = S::LDN, LDP = S::LDP, CE = S::CE, PPW = S::PPW;
    constexpr int NK = N / MM::K;        // MFMA K-steps over the state axis
    constexpr int JK = S::JB / MM::K;    // MFMA K-steps over a 64-row block
    constexpr int PT = P / 16;           // 16-column tiles of y and of the state
    constexpr int LDT = NH + 32 / (int)sizeof(CS);   // cos/sin table row [token][pair]

    // Per-chunk scalars and tables, by chunk parity: the state waves write
    // chunk c + 1's while chunk c's are in use.
    // s_c2: the log-decay prefix sums in base 2 (cum_t log2(e)): e^{cum} = 2^{c2}
    __shared__ float s_c2[2][Q], s_gam[2][Q], s_sig[2][Q], s_w[2][Q], s_psie[2][NH];
    __shared__ __attribute__((aligned(16))) CS s_cs[2][Q * LDT];
    // Row blocks, double-buffered: B^ [row][n], x and W x [row][p].
    __shared__ __attribute__((aligned(16))) T s_B[2][S::JB * LDN];
    __shared__ __attribute__((aligned(16))) T s_X[2][S::JB * LDP];
    __shared__ __attribute__((aligned(16))) T s_WX[2][S::JB * LDP];
    // State entering the chunk, transposed [p][n], in bf16 (operand of y).
    __shared__ __attribute__((aligned(16))) T s_S[P * LDN];
    // y staging, one 16-row tile per output wave.
    __shared__ __attribute__((aligned(16))) T s_Y[S::NWO][16 * LDP];
    // Block prologue tables of the head (fp32): B gain and bias as 16-byte
    // entries at bgb(r, i) (gain and bias of element i, then of element
    // i + N/2, of rank row r: one read serves a rotation pair; ordered so that
    // the lanes staging one element of consecutive pieces of all rank rows
    // read consecutive entries), C gain and bias [R][N], then W_X, W_Z and
    // the output norm's gain [R][P] (ones / zeros where not given).
    constexpr int kPB = 0, kPC = 2 * R * N, kPCb = 3 * R * N, kPWX = 4 * R * N, kPWZ = kPWX + R * P,
                  kPGY = kPWZ + R * P;
    __shared__ __attribute__((aligned(16))) float s_pro[kPro ? 4 * R * N + 3 * R * P : 4];
    constexpr int BPR = NH / CE;   // 16-byte pieces of a half row
    auto bgb = [](int r, int i) { return kPB + 4 * (((i % CE) * BPR + i / CE) * R + r); };
    // K consecutive table floats (16-byte reads; p a multiple of 4)
    auto tab = [&](int p, float *v, int K) {
        for (int q = 0; q < K; q += 4) {
            const float4 f = *reinterpret_cast<const float4 *>(&s_pro[p + q]);
            v[q] = f.x; v[q + 1] = f.y; v[q + 2] = f.z; v[q + 3] = f.w;
        }
    };

    // Lane indices are re-derived from an opaque copy of the thread index at
    // the top of every chunk (relane), so that the compiler recomputes
    // addresses instead of keeping them live across the chunk loop.
    int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
    int g = lane >> 4, l16 = lane & 15;
    auto relane = [&]() {
        asm volatile("" : "+v"(tid));
        lane = tid & (kWave - 1);
        g = lane >> 4;
        l16 = lane & 15;
    };

    const int64_t sl = blockIdx.x;
    // no look-back here: the timeout count of the workspace reads zero
    if (sl == 0 && tid == 0) a.ctl[kCtlTimeouts0] = a.ctl[kCtlTimeouts1] = 0u;
    const int64_t b = sl / a.H, h = sl % a.H;
    const int64_t nch = a.nchunks;
    const int64_t tstr = a.H;
    const int64_t bstr = tstr * R * N, xstr = tstr * R * P;
    const uint32_t bstr_b = (uint32_t)(bstr * sizeof(T));
    const T *Bs = static_cast<const T *>(a.B);
    const T *Cs = static_cast<const T *>(a.C);
    const T *Xs = static_cast<const T *>(a.x);
    auto tok_of = [&](int64_t c) -> int64_t { return (b * a.L + c * Q) * a.H + h; };
    auto nvalid_of = [&](int64_t c) -> int { return (int)min((int64_t)Q, a.L - c * Q); };
    // Every row load goes through a buffer resource that ends at the chunk's
    // last valid token (rows past the end of the sequence read as zeros).
    auto rows_rsrc = [&](const T *base, int64_t c, int64_t str, int width) {
        const int nv = nvalid_of(c);
        return make_rsrc(base + tok_of(c) * width, (uint32_t)(((nv - 1) * str + width) * (int64_t)sizeof(T)));
    };
    auto sched_fence = []() { __builtin_amdgcn_sched_barrier(0); };
    const int64_t SZ = (int64_t)N * P;
    // x and z as read: P x R per token-head, or (structured input) the
    // P-vector X' (Z') that every rank row reads (row offset 0)
    const bool sx = kPro && a.pro.wx != nullptr, sz = kPro && a.pro.wz != nullptr;
    const int64_t xin_tok = sx ? (int64_t)P : (int64_t)(R * P), zin_tok = sz ? (int64_t)P : (int64_t)(R * P);
    const int xr_el = sx ? 0 : P, zr_el = sz ? 0 : P;
    const int64_t xin_str = tstr * xin_tok, zin_str = tstr * zin_tok;
    const uint32_t xin_b = (uint32_t)(xin_str * sizeof(T)), zin_b = (uint32_t)(zin_str * sizeof(T));
    if constexpr (kPro) {   // the head's tables (read after the first barrier of both roles)
        const int64_t hn = h * (R * N), hp = h * (R * P);
        for (int e = tid; e < R * N; e += S::NTHR) {
            const int r = e / N, n = e % N;
            const int q = bgb(r, n % NH) + (n < NH ? 0 : 2);
            s_pro[q] = a.pro.gB ? a.pro.gB[hn + e] : 1.f;
            s_pro[q + 1] = a.pro.bB ? a.pro.bB[hn + e] : 0.f;
            s_pro[kPC + e] = a.pro.gC ? a.pro.gC[hn + e] : 1.f;
            s_pro[kPCb + e] = a.pro.bC ? a.pro.bC[hn + e] : 0.f;
        }
        for (int e = tid; e < R * P; e += S::NTHR) {
            s_pro[kPWX + e] = a.pro.wx ? a.pro.wx[hp + e] : 1.f;
            s_pro[kPWZ + e] = a.pro.wz ? a.pro.wz[hp + e] : 1.f;
            s_pro[kPGY + e] = a.pro.og ? a.pro.og[hp + e] : 1.f;
        }
    }

    if (wave < S::NWO) {
        // ================= output waves =================
        const int ow = wave;
        int TT[TPW];
#pragma unroll
        for (int m = 0; m < TPW; ++m) TT[m] = owned_tile<S>(ow, m);
        Frag cf[TPW][NK];
        auto load_c = [&](int64_t c, int m) {
            const Rsrc rc = rows_rsrc(Cs, c, bstr, R * N);
            const int row = TT[m] * 16 + l16, t = row / R, r = row % R;
            const uint32_t off = tok_off(t, bstr_b) + (uint32_t)((r * N + MM::KPL * g) * sizeof(T));
#pragma unroll
            for (int kk = 0; kk < NK; ++kk) cf[m][kk] = buf_load<Frag>(rc, off + kk * MM::K * sizeof(T));
        };
#pragma unroll
        for (int m = 0; m < TPW; ++m) load_c(0, m);
        __syncthreads();   // prologue of chunk 0 written
        __syncthreads();   // block 0 and the entering state staged
        const float Dh = a.D[h];
        for (int64_t c = 0; c < nch; ++c) {
            relane();
            const int par = (int)(c & 1);
            const int nv = nvalid_of(c);
            const int64_t cn = min(c + 1, nch - 1);
            // C^ = R(-psi_t) C of the owned rows
            if constexpr (kPro) {
                // each element first normalised, c = sc g c + b in fp32 (sc the
                // row's RMS scale from a sum of squares over its fragments: a
                // row sits in lanes l16 + 16 g; zero past the end of the
                // sequence); a lane's rank row l16 % R is the same in all its
                // tiles, so its gains and biases are read once per fragment pair
                float scm[TPW], bscm[TPW];
#pragma unroll
                for (int m = 0; m < TPW; ++m) {
                    const int t = (TT[m] * 16 + l16) / R;
                    float ss = 0.f;
#pragma unroll
                    for (int kk = 0; kk < NK; ++kk) ss += sumsq(cf[m][kk]);
                    ss += __shfl_xor(ss, 16, kWave);
                    ss += __shfl_xor(ss, 32, kWave);
                    const bool ok = t < nv;
                    scm[m] = !ok ? 0.f : (a.pro.bcnorm ? rsqrtf(ss * (1.f / N) + a.pro.eps) : 1.f);
                    bscm[m] = ok ? 1.f : 0.f;
                }
#pragma unroll
                for (int kk = 0; kk < NK / 2; ++kk) {
                    static_assert(MM::KPL % 4 == 0, "16-byte table reads");
                    const int pu = (l16 % R) * N + kk * MM::K + MM::KPL * g, pw = pu + NH;
                    float gu[MM::KPL], gw[MM::KPL], bu[MM::KPL], bw[MM::KPL];
                    tab(kPC + pu, gu, MM::KPL);
                    tab(kPC + pw, gw, MM::KPL);
                    tab(kPCb + pu, bu, MM::KPL);
                    tab(kPCb + pw, bw, MM::KPL);
#pragma unroll
                    for (int m = 0; m < TPW; ++m) {
                        const int t = (TT[m] * 16 + l16) / R;
                        float csv[MM::KPL], snv[MM::KPL];
                        cs_getn<MM::KPL>(&s_cs[par][t * LDT + kk * MM::K + MM::KPL * g], csv, snv);
#pragma unroll
                        for (int e = 0; e < MM::KPL; ++e) {
                            const float u = scm[m] * gu[e] * fget(cf[m][kk], e) + bscm[m] * bu[e];
                            const float w = scm[m] * gw[e] * fget(cf[m][kk + NK / 2], e) + bscm[m] * bw[e];
                            fset(cf[m][kk], e, csv[e] * u + snv[e] * w);
                            fset(cf[m][kk + NK / 2], e, csv[e] * w - snv[e] * u);
                        }
                    }
                }
            } else {
#pragma unroll
                for (int m = 0; m < TPW; ++m) {
                    const int t = (TT[m] * 16 + l16) / R;
#pragma unroll
                    for (int kk = 0; kk < NK / 2; ++kk) {
                        float csv[MM::KPL], snv[MM::KPL];
                        cs_getn<MM::KPL>(&s_cs[par][t * LDT + kk * MM::K + MM::KPL * g], csv, snv);
#pragma unroll
                        for (int e = 0; e < MM::KPL; ++e) {
                            const float u = fget(cf[m][kk], e), w = fget(cf[m][kk + NK / 2], e);
                            fset(cf[m][kk], e, csv[e] * u + snv[e] * w);
                            fset(cf[m][kk + NK / 2], e, csv[e] * w - snv[e] * u);
                        }
                    }
                }
            }
            // inter-chunk term: y^T = e^{cum_t} S^T C^T (lane l: row l % 16 of
            // the tile, four consecutive y columns)
            f32x4 acc[TPW][PT];
#pragma unroll
            for (int m = 0; m < TPW; ++m)
#pragma unroll
                for (int pt = 0; pt < PT; ++pt) acc[m][pt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int pt = 0; pt < PT; ++pt)
#pragma unroll
                for (int kk = 0; kk < NK; ++kk) {
                    const Frag sf = MM::load(&s_S[(pt * 16 + l16) * LDN + kk * MM::K + MM::KPL * g]);
#pragma unroll
                    for (int m = 0; m < TPW; ++m) acc[m][pt] = MM::mma(sf, cf[m][kk], acc[m][pt]);
                }
            float c2_t[TPW], gam_t[TPW];
#pragma unroll
            for (int m = 0; m < TPW; ++m) {
                const int t = (TT[m] * 16 + l16) / R;
                c2_t[m] = s_c2[par][t];
                gam_t[m] = s_gam[par][t];
                const float ec = exp2_fast(c2_t[m]);
#pragma unroll
                for (int pt = 0; pt < PT; ++pt)
#pragma unroll
                    for (int v = 0; v < 4; ++v) acc[m][pt][v] *= ec;
            }
            // y leaves in 16-byte pieces of its rows (NPC per lane and owned
            // tile); with the gate, the matching pieces of z are loaded at the
            // start of the last step and arrive during its products
            constexpr int RP = P / CE;   // 16-byte pieces of a row
            constexpr int NPC = 16 * RP / kWave;
            static_assert(NPC * kWave == 16 * RP, "store pieces");
            V16 zp[kGate ? TPW : 1][NPC];
#pragma unroll
            for (int jb = 0; jb < NJB; ++jb) {
                const T *sBc = s_B[jb & 1], *sXc = s_X[jb & 1];
                if constexpr (kGate) {
                    if (jb == NJB - 1) {
                        const Rsrc rz = rows_rsrc(static_cast<const T *>(a.z), c, zin_str, (int)zin_tok);
#pragma unroll
                        for (int m = 0; m < TPW; ++m)
#pragma unroll
                            for (int i = 0; i < NPC; ++i) {
                                const int k = lane + i * kWave, rl = k / RP, col = (k % RP) * CE;
                                const int row = TT[m] * 16 + rl, t = row / R, r = row % R;
                                zp[m][i] = buf_load<V16>(rz, tok_off(t, zin_b) + (uint32_t)((r * zr_el + col) * sizeof(T)));
                            }
                    }
                }
#pragma unroll
                for (int jp = 0; jp < S::JB / 32; ++jp) {
                    // Owned tile m lies in block m (rows 64 m .. 64 m + 63): tiles
                    // m < jb are above this block (no work), tiles m > jb below
                    // it (every pair unmasked); only tile jb needs the row test.
                    const int J0 = jb * 4 + 2 * jp;   // first j-tile of the pair (chunk-global)
                    if (jb == NJB - 1 && J0 > TT[TPW - 1]) continue;
                    // x^T columns of the pair: rows 32 jp + 4g .. +3 and +16, column l16
                    bf16x8 xf[PT];
#pragma unroll
                    for (int pt = 0; pt < PT; ++pt) {
                        const T *xr = &sXc[(32 * jp + 4 * g + l16 / 4) * LDP + pt * 16 + 4 * (l16 % 4)];
                        const bf16x4 lo = lds_tr4(xr), hi = lds_tr4(xr + 16 * LDP);
#pragma unroll
                        for (int v = 0; v < 4; ++v) { xf[pt][v] = lo[v]; xf[pt][4 + v] = hi[v]; }
                    }
                    f32x4 gt[TPW][2];
#pragma unroll
                    for (int m = 0; m < TPW; ++m) gt[m][0] = gt[m][1] = f32x4{0.f, 0.f, 0.f, 0.f};
                    constexpr int NV = R >= 4 ? 1 : 4 / R;   // tokens among a lane's 4 rows
                    float cj[2][NV], sj[2][NV];
#pragma unroll
                    for (int q = 0; q < 2; ++q) {
#pragma unroll
                        for (int u = 0; u < NV; ++u) {
                            const int tj = ((J0 + q) * 16 + 4 * g + u * R) / R;
                            cj[q][u] = s_c2[par][tj];
                            sj[q][u] = s_sig[par][tj];
                        }
                        Frag bfr[NK];
#pragma unroll
                        for (int kk = 0; kk < NK; ++kk)
                            bfr[kk] = MM::load(&sBc[((2 * jp + q) * 16 + l16) * LDN + kk * MM::K + MM::KPL * g]);
#pragma unroll
                        for (int kk = 0; kk < NK; ++kk)
#pragma unroll
                            for (int m = 0; m < TPW; ++m)
                                if (m > jb || (m == jb && J0 + q <= TT[m]))
                                    gt[m][q] = MM::mma(bfr[kk], cf[m][kk], gt[m][q]);
                    }
                    // mask weights: w_tj = e^{cum_t - cum_j} sigma_j (j < t),
                    // gamma_t (j = t), 0 (j > t); D x_t on the diagonal
#pragma unroll
                    for (int m = 0; m < TPW; ++m) {
                        if (m < jb || (m == jb && J0 > TT[m])) continue;
                        const int tt = (TT[m] * 16 + l16) / R;
#pragma unroll
                        for (int q = 0; q < 2; ++q) {
                            float wv[NV];
#pragma unroll
                            for (int u = 0; u < NV; ++u) {
                                // (above the diagonal the exponent may be large: the select drops it)
                                const float e = exp2_fast(c2_t[m] - cj[q][u]) * sj[q][u];
                                if (m > jb || J0 + q < TT[m]) {
                                    wv[u] = e;
                                } else {
                                    const int tj = ((J0 + q) * 16 + 4 * g + u * R) / R;
                                    wv[u] = tj < tt ? e : (tj == tt ? gam_t[m] : 0.f);
                                }
                            }
#pragma unroll
                            for (int v = 0; v < 4; ++v) gt[m][q][v] *= wv[(v * NV) / 4];
                            if (m == jb && J0 + q == TT[m]) {
#pragma unroll
                                for (int v = 0; v < 4; ++v) gt[m][q][v] += (4 * g + v == l16) ? Dh : 0.f;
                            }
                        }
                        // y^T += x^T (w o G)^T  (K = the pair's 32 rows)
                        bf16x8 af;
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            af[v] = (bf16)gt[m][0][v];
                            af[4 + v] = (bf16)gt[m][1][v];
                        }
#pragma unroll
                        for (int pt = 0; pt < PT; ++pt) acc[m][pt] = MM::mma(xf[pt], af, acc[m][pt]);
                    }
                }
                // owned tile jb lies in this block: its C rows are dead, load
                // the next chunk's
                sched_fence();
                load_c(cn, jb);
                sched_fence();
                if (jb == NJB - 1) {
                    // store y: stage each tile in the wave's own LDS rows (a
                    // wave's LDS accesses execute in order) and write whole
                    // 16-byte pieces of the rows
                    T *sy = s_Y[ow];
                    T *Yg = static_cast<T *>(a.y) + tok_of(c) * (R * P);
#pragma unroll
                    for (int m = 0; m < TPW; ++m) {
#pragma unroll
                        for (int pt = 0; pt < PT; ++pt) store4(&sy[l16 * LDP + pt * 16 + 4 * g], acc[m][pt]);
                        asm volatile("" ::: "memory");
#pragma unroll
                        for (int i = 0; i < NPC; ++i) {
                            const int k = lane + i * kWave, rl = k / RP, col = (k % RP) * CE;
                            const int row = TT[m] * 16 + rl, t = row / R, r = row % R;
                            if constexpr (kPro) {
                                // gate factor SiLU(W_Z o Z') in fp32, then
                                // (optionally) the output norm: a row's RP
                                // pieces are RP consecutive lanes, so a group's
                                // sum of squares is a lane sum (all lanes take
                                // part; rows past the end are not stored)
                                V16 yv = *reinterpret_cast<const V16 *>(&sy[rl * LDP + col]);
                                float yf[CE], gz[CE], wz[CE];
                                if constexpr (kGate) tab(kPWZ + r * P + col, wz, CE);
#pragma unroll
                                for (int e = 0; e < CE; ++e) {
                                    yf[e] = fget(yv, e);
                                    gz[e] = kGate ? silu(fget(zp[m][i], e) * wz[e]) : 1.f;
                                }
                                if (a.pro.onorm) {   // (uniform)
                                    const bool post = a.pro.onorm == 2;
                                    float ss = 0.f;
#pragma unroll
                                    for (int e = 0; e < CE; ++e) {
                                        if (post) yf[e] *= gz[e];
                                        ss += yf[e] * yf[e];
                                    }
                                    // (a fixed count of lane steps, those past the group adding nothing:
                                    // a loop of constant length stays unrolled)
#pragma unroll
                                    for (int o = 1; o < RP; o <<= 1) {
                                        const float so = __shfl_xor(ss, o, kWave);
                                        ss += o < a.pro.ogroup / CE ? so : 0.f;
                                    }
                                    const float sc = rsqrtf(ss / (float)a.pro.ogroup + a.pro.oeps);
                                    float gy[CE];
                                    tab(kPGY + r * P + col, gy, CE);
#pragma unroll
                                    for (int e = 0; e < CE; ++e) {
                                        yf[e] *= sc * gy[e];
                                        if (!post) yf[e] *= gz[e];
                                    }
                                } else {
#pragma unroll
                                    for (int e = 0; e < CE; ++e) yf[e] *= gz[e];
                                }
#pragma unroll
                                for (int e = 0; e < CE; ++e) fset(yv, e, yf[e]);
                                if (t < nv) *reinterpret_cast<V16 *>(Yg + t * xstr + r * P + col) = yv;
                            } else if (t < nv) {
                                V16 yv = *reinterpret_cast<const V16 *>(&sy[rl * LDP + col]);
                                if constexpr (kGate) yv = gate_piece<T>(yv, zp[m][i]);
                                *reinterpret_cast<V16 *>(Yg + t * xstr + r * P + col) = yv;
                            }
                        }
                        asm volatile("" ::: "memory");
                    }
                }
                __syncthreads();   // step jb of the chunk
            }
        }
    } else {
        // ================= state waves =================
        const int sw = wave - S::NWO;        // state wave index: state rows 16 sw .. and + N/2
        constexpr int TB = S::JB * (NH / CE) / S::NST;   // B tasks per thread
        constexpr int TX = S::JB * (P / CE) / S::NST;    // x tasks per thread
        static_assert(TB * S::NST == S::JB * (NH / CE) && TX * S::NST == S::JB * (P / CE), "tasks");
        struct Blk { V16 lo[TB], hi[TB], xv[TX]; };
        // B row pieces: consecutive lanes take consecutive rows (conflict-free
        // cos/sin reads); with the prologue the BPR pieces of a half row sit in
        // consecutive lanes instead, so that the row's norm is a lane sum.
        auto brow = [](int task) { return kPro ? task / BPR : task % S::JB; };
        auto bpiece = [](int task) { return kPro ? task % BPR : task / S::JB; };
        auto fetch = [&](int64_t c, int jb, Blk &f) {
            const Rsrc rb = rows_rsrc(Bs, c, bstr, R * N), rx = rows_rsrc(Xs, c, xin_str, (int)xin_tok);
#pragma unroll
            for (int k = 0; k < TB; ++k) {
                const int task = (tid - S::NWO * kWave) + k * S::NST, jr = brow(task), cp = bpiece(task);
                const int row = jb * S::JB + jr, t = row / R, r = row % R;
                const uint32_t off = tok_off(t, bstr_b) + (uint32_t)((r * N + cp * CE) * sizeof(T));
                f.lo[k] = buf_load<V16>(rb, off);
                f.hi[k] = buf_load<V16>(rb, off + NH * sizeof(T));
            }
#pragma unroll
            for (int k = 0; k < TX; ++k) {
                const int task = (tid - S::NWO * kWave) + k * S::NST, jr = task % S::JB, pc = task / S::JB;
                const int row = jb * S::JB + jr, t = row / R, r = row % R;
                f.xv[k] = buf_load<V16>(rx, tok_off(t, xin_b) + (uint32_t)((r * xr_el + pc * CE) * sizeof(T)));
            }
        };
        // stage block jb of a chunk with nvs valid tokens (tables of parity
        // par) into buffer jb & 1
        auto commit = [&](int jb, int par, int nvs, const Blk &f) {
            T *sB = s_B[jb & 1], *sX = s_X[jb & 1], *sWX = s_WX[jb & 1];
#pragma unroll
            for (int k = 0; k < TB; ++k) {
                const int task = (tid - S::NWO * kWave) + k * S::NST, jr = brow(task), cp = bpiece(task);
                const int t = (jb * S::JB + jr) / R;
                V16 lo = f.lo[k], hi = f.hi[k];
                float csv[CE], snv[CE];
                cs_getn<CE>(&s_cs[par][t * LDT + cp * CE], csv, snv);
                float sc = 1.f, bsc = 1.f;
                int pb = 0;
                if constexpr (kPro) {   // B = g o B' / rms(B') + b (rows past the end stay zero)
                    float ss = sumsq(lo) + sumsq(hi);
#pragma unroll
                    for (int o = 1; o < BPR; o <<= 1) ss += __shfl_xor(ss, o, kWave);
                    const bool ok = t < nvs;
                    sc = !ok ? 0.f : (a.pro.bcnorm ? rsqrtf(ss * (1.f / N) + a.pro.eps) : 1.f);
                    bsc = ok ? 1.f : 0.f;
                    static_assert(S::JB % R == 0, "rank row of a task independent of the block");
                    pb = bgb(jr % R, cp * CE);
                }
#pragma unroll
                for (int e = 0; e < CE; ++e) {
                    float u = fget(lo, e), w = fget(hi, e);
                    if constexpr (kPro) {   // (one 16-byte table entry a pair)
                        const float4 gb = *reinterpret_cast<const float4 *>(&s_pro[pb + 4 * BPR * R * e]);
                        u = sc * gb.x * u + bsc * gb.y;
                        w = sc * gb.z * w + bsc * gb.w;
                    }
                    fset(lo, e, csv[e] * u + snv[e] * w);
                    fset(hi, e, csv[e] * w - snv[e] * u);
                }
                *reinterpret_cast<V16 *>(&sB[jr * LDN + cp * CE]) = lo;
                *reinterpret_cast<V16 *>(&sB[jr * LDN + NH + cp * CE]) = hi;
            }
#pragma unroll
            for (int k = 0; k < TX; ++k) {
                const int task = (tid - S::NWO * kWave) + k * S::NST, jr = task % S::JB, pc = task / S::JB;
                const float wt = s_w[par][(jb * S::JB + jr) / R];
                V16 xv = f.xv[k];
                if constexpr (kPro) {   // X = W_X o X' (ones without structured input)
                    float wv[CE];
                    tab(kPWX + (jr % R) * P + pc * CE, wv, CE);
#pragma unroll
                    for (int e = 0; e < CE; ++e) fset(xv, e, fget(xv, e) * wv[e]);
                }
                *reinterpret_cast<V16 *>(&sX[jr * LDP + pc * CE]) = xv;
                V16 wx;
#pragma unroll
                for (int e = 0; e < CE; ++e) fset(wx, e, wt * fget(xv, e));
                *reinterpret_cast<V16 *>(&sWX[jr * LDP + pc * CE]) = wx;
            }
        };
        // M += B^T (W x) over a staged block: state rows 16 (sw + 4 half) + 4g + v,
        // columns 16 pt + l16
        auto m_block = [&](f32x4 (&ms)[PT][2], int jb) {
            const T *sB = s_B[jb & 1], *sWX = s_WX[jb & 1];
#pragma unroll
            for (int ks = 0; ks < JK; ++ks) {
                Frag af[2];
#pragma unroll
                for (int half = 0; half < 2; ++half)
                    af[half] = load_kt(sB, LDN, ks * MM::K, (sw + 4 * half) * 16, g, l16);
#pragma unroll
                for (int pt = 0; pt < PT; ++pt) {
                    const Frag bf = load_kt(sWX, LDP, ks * MM::K, pt * 16, g, l16);
#pragma unroll
                    for (int half = 0; half < 2; ++half) ms[pt][half] = MM::mma(af[half], bf, ms[pt][half]);
                }
            }
        };
        // prologue inputs of a chunk (lane = token; this wave's 16 angle pairs)
        struct Pro { f32x4 th[PPW / 4]; float dtv, lamv, Av, dtn, lamn; };
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
            const int t = lane;
            const uint32_t oth = tok_off(t, thstr_b) + sw * PPW * 4;
#pragma unroll
            for (int q = 0; q < PPW / 4; ++q) p.th[q] = buf_load<f32x4>(rth, oth + 16 * q);
            const uint32_t o = tok_off(t, tstr_b);
            p.dtv = buf_load<float>(rdt, o);
            p.lamv = buf_load<float>(rlam, o);
            p.dtn = buf_load<float>(rdt, o + tstr_b);
            p.lamn = buf_load<float>(rlam, o + tstr_b);
            p.Av = a.A[b * a.a_sb + (c * Q + min(t, nv - 1)) * a.a_st + h * a.a_sh];
        };
        // cum, gamma, sigma and the W x weights of a chunk (one wave)
        auto pro_scalars = [&](int64_t c, const Pro &p) {
            const int nv = nvalid_of(c), par = (int)(c & 1);
            const float lg = p.dtv * p.Av;
            const float gam = p.lamv * p.dtv;
            const float sig = gam + (1.f - p.lamn) * p.dtn;
            const float cum = lane_scan(lg);
            const float cum_e = lane_bcast(cum, nv - 1);
            s_c2[par][lane] = cum * 1.44269504f;
            s_gam[par][lane] = gam;
            s_sig[par][lane] = sig;
            s_w[par][lane] = (lane < nv) ? exp_fast(cum_e - cum) * sig : 0.f;
        };
        // angle prefix sums of pairs K0 .. K0 + K - 1 of this wave: cos/sin
        // table and psi_e
        auto pro_pairs = [&](int64_t c, const Pro &p, auto K0c, auto Kc) {
            constexpr int K0 = decltype(K0c)::value, K = decltype(Kc)::value;
            const int nv = nvalid_of(c), par = (int)(c & 1);
            // angle of this lane's token: theta, or dt * omega (zero past the end)
            const float tsc = a.theta_ph ? (lane < nv ? p.dtv : 0.f) : 1.f;
            float csv[K], snv[K];
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const int i = sw * PPW + K0 + k;
                const float psi = lane_scan(p.th[(K0 + k) / 4][(K0 + k) % 4] * tsc);   // zero past the end
                float sn, cs;
                sincos_fast(psi, &sn, &cs);
                csv[k] = cs;
                snv[k] = sn;
                if (lane == nv - 1) s_psie[par][i] = psi;
            }
            cs_putn<K>(&s_cs[par][lane * LDT + sw * PPW + K0], csv, snv);
        };
        using I0 = std::integral_constant<int, 0>;
        using I4 = std::integral_constant<int, 4>;
        using I8 = std::integral_constant<int, 8>;
        using I12 = std::integral_constant<int, 12>;
        using I16 = std::integral_constant<int, 16>;

        // state element (pt, half, v): row n = 16 (sw + 4 half) + 4g + v, column p = 16 pt + l16
        float Sst[PT][2][4];
        {
            const float *ist = a.init_state ? a.init_state + sl * SZ : nullptr;
            float wb = 0.f;
            if (a.init_cB) {
                const int64_t k0 = (b * a.L) * a.H + h;
                wb = (1.f - a.lam[k0]) * a.dt[k0];
            }
            const T *iB = a.init_cB ? static_cast<const T *>(a.init_cB) + sl * (R * N) : nullptr;
            const T *iX = a.init_cX ? static_cast<const T *>(a.init_cX) + sl * (R * P) : nullptr;
            // element (pt, half, v): row 16 (sw + 4 half) + 4g + v, column 16 pt + l16
            init_elems<T, R, N, P, PT * 8>(
                ist, iB, iX, wb, [&](int e) { return 16 * (sw + 4 * ((e / 4) % 2)) + 4 * g + e % 4; },
                [&](int e) { return 16 * (e / 8) + l16; }, &Sst[0][0][0]);
        }
        auto write_st = [&]() {   // S^T [p][n] in bf16, 8-byte pieces
#pragma unroll
            for (int pt = 0; pt < PT; ++pt)
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    bf16x4 o;
#pragma unroll
                    for (int v = 0; v < 4; ++v) o[v] = (bf16)Sst[pt][half][v];
                    *reinterpret_cast<bf16x4 *>(&s_S[(16 * pt + l16) * LDN + 16 * (sw + 4 * half) + 4 * g]) = o;
                }
        };
        auto write_final = [&]() {
            float *fs = a.final_state + sl * SZ;
#pragma unroll
            for (int pt = 0; pt < PT; ++pt)
#pragma unroll
                for (int half = 0; half < 2; ++half)
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        fs[(16 * (sw + 4 * half) + 4 * g + v) * P + 16 * pt + l16] = Sst[pt][half][v];
            T *cB = static_cast<T *>(a.cB) + sl * (R * N);
            T *cX = static_cast<T *>(a.cX) + sl * (R * P);
            const int64_t kl = (b * a.L + a.L - 1) * a.H + h;
            const T *Bl = Bs + kl * (R * N);
            const T *Xl = Xs + kl * xin_tok;
            if constexpr (kPro) {   // the carry holds the B and X the recurrence used
                static_assert(N == 2 * kWave, "two elements of a B row per lane");
                for (int r = sw; r < R; r += S::NSW) {
                    const float v0 = to_f32(Bl[r * N + lane]), v1 = to_f32(Bl[r * N + kWave + lane]);
                    float ss = v0 * v0 + v1 * v1;
#pragma unroll
                    for (int o = 1; o < kWave; o <<= 1) ss += __shfl_xor(ss, o, kWave);
                    const float sc = a.pro.bcnorm ? rsqrtf(ss * (1.f / N) + a.pro.eps) : 1.f;
                    const float4 gb = *reinterpret_cast<const float4 *>(&s_pro[bgb(r, lane)]);
                    cB[r * N + lane] = from_f32<T>(sc * gb.x * v0 + gb.y);
                    cB[r * N + kWave + lane] = from_f32<T>(sc * gb.z * v1 + gb.w);
                }
                for (int e = (tid - S::NWO * kWave); e < R * P; e += S::NST)
                    cX[e] = from_f32<T>(to_f32(Xl[sx ? e % P : e]) * s_pro[kPWX + e]);
            } else {
                for (int e = (tid - S::NWO * kWave); e < R * N; e += S::NST) cB[e] = Bl[e];
                for (int e = (tid - S::NWO * kWave); e < R * P; e += S::NST) cX[e] = Xl[e];
            }
        };

        // Blocks are numbered k = c * NJB + jb; the ring holds the loads of
        // blocks k + 1 and k + 2 during step k.
        Blk ring[2];
        auto fetch_k = [&](int64_t k, Blk &f) {
            const int64_t c = min(k / NJB, nch - 1);
            fetch(c, (int)(k % NJB), f);
        };
        Pro pro;
        load_pro(0, pro);
        sched_fence();
        fetch_k(0, ring[0]);
        fetch_k(1, ring[1]);
        sched_fence();
        if (sw == 0) pro_scalars(0, pro);
        pro_pairs(0, pro, I0{}, I16{});
        write_st();
        sched_fence();
        load_pro(min((int64_t)1, nch - 1), pro);
        sched_fence();
        __syncthreads();   // prologue of chunk 0 written
        commit(0, 0, nvalid_of(0), ring[0]);
        sched_fence();
        fetch_k(2, ring[0]);
        sched_fence();
        __syncthreads();   // block 0 and the entering state staged
        for (int64_t c = 0; c < nch; ++c) {
            relane();
            const int par = (int)(c & 1);
            const int nv = nvalid_of(c);
            const int64_t cn = min(c + 1, nch - 1);
            f32x4 ms[PT][2];
            {
                const float de = exp2_fast(s_c2[par][nv - 1]);
#pragma unroll
                for (int pt = 0; pt < PT; ++pt)
#pragma unroll
                    for (int half = 0; half < 2; ++half)
#pragma unroll
                        for (int v = 0; v < 4; ++v) ms[pt][half][v] = de * Sst[pt][half][v];
            }
#pragma unroll
            for (int jb = 0; jb < NJB; ++jb) {
                m_block(ms, jb);
                // stage block k + 1 (chunk c's next block, or chunk c + 1's first)
                // and load block k + 3
                const int64_t k = c * NJB + jb;
                sched_fence();
                if (jb + 1 < NJB) commit(jb + 1, par, nv, ring[(jb + 1) & 1]);
                else commit(0, (int)(cn & 1), nvalid_of(cn), ring[(jb + 1) & 1]);
                sched_fence();
                fetch_k(k + 3, ring[(jb + 1) & 1]);
                sched_fence();
                // prologue of chunk c + 1, in three parts
                if (jb == 0) {
                    if (sw == 0) pro_scalars(cn, pro);
                    pro_pairs(cn, pro, I0{}, I4{});
                } else if (jb == 1) {
                    pro_pairs(cn, pro, I4{}, I8{});
                } else if (jb == 2) {
                    pro_pairs(cn, pro, I12{}, I4{});
                    sched_fence();
                    load_pro(min(c + 2, nch - 1), pro);
                    sched_fence();
                } else {
                    // S <- R(psi_e) (e^{cum_e} S + M): rows i and i + N/2 of a
                    // pair sit in one lane
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        float sn, cs;
                        sincos_fast(s_psie[par][16 * sw + 4 * g + v], &sn, &cs);
#pragma unroll
                        for (int pt = 0; pt < PT; ++pt) {
                            const float re = ms[pt][0][v], im = ms[pt][1][v];
                            Sst[pt][0][v] = cs * re - sn * im;
                            Sst[pt][1][v] = sn * re + cs * im;
                        }
                    }
                    write_st();
                    if (c == nch - 1) write_final();
                }
                __syncthreads();   // step jb of the chunk
            }
        }
    }
}

template <int Q, int R, bool kPro = false>
hipError_t launch_ws(const ScanArgs &a, hipStream_t stream) {
    typedef WsShape<Q, R> S;
    const int64_t nsl = a.batch * a.H;
    if (a.z)
        hipLaunchKernelGGL((k_scan_ws<Q, R, true, kPro>), dim3((unsigned)nsl), dim3(S::NTHR), 0, stream, a);
    else
        hipLaunchKernelGGL((k_scan_ws<Q, R, false, kPro>), dim3((unsigned)nsl), dim3(S::NTHR), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

// Shapes with a warp-specialised kernel (bf16 operands, N = 128, P = 64).
scan_launch_fn find_ws_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q) {
    if (io != 1 || N != 128 || P != 64) return nullptr;
    if (Q == 64 && R == 4) return &launch_ws<64, 4>;
    return nullptr;
}

// The same kernels built with the block prologue.
scan_launch_fn find_ws_pro_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q) {
    if (io != 1 || N != 128 || P != 64) return nullptr;
    if (Q == 64 && R == 4) return &launch_ws<64, 4, true>;
    return nullptr;
}

}  // namespace m3
