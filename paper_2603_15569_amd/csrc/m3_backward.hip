// Backward pass of the chunked prefill scan (training; Sec. 3.3 "Chunked
// Algorithm for MIMO SSMs": the same chunk decomposition run in reverse) on
// gfx950, bf16 inputs, N = 128, P = 64, chunks of 64 rows (chunk * rank =
// 64: SISO chunk 64, rank 2 chunk 32, rank 4 chunk 16).
//
// Forward, per chunk c with chunk-local prefix sums cum_t (of dt A) and
// psi_t (of theta), C^_t = R(-psi_t) C_t, B^_j = R(-psi_j) B_j, gamma_t =
// lambda_t dt_t, sigma_j = gamma_j + (1 - lambda_{j+1}) dt_{j+1},
// w_tt = gamma_t, w_tj = e^{cum_t - cum_j} sigma_j (j < t), v_j = e^{cum_e -
// cum_j} sigma_j (e the chunk's last token):
//   y_t = sum_{j<=t} w_tj (C^_t . B^_j) x_j + e^{cum_t} C^_t^T S_{c-1} + D x_t
//   S_c = R(psi_e) (e^{cum_e} S_{c-1} + M_c),  M_c = sum_j v_j B^_j x_j^T
// Reverse, for a loss J with dy = dJ/dy and G_c = dJ/dS_c (G_last = dJ/d
// final state):
//   U_c = R(-psi_e) G_c                                  (dJ/dM_c)
//   G_{c-1} = e^{cum_e} U_c + sum_t e^{cum_t} C^_t dy_t^T
//   dG[t][j] = dy_t . x_j (chunk rows), G[t][j] = C^_t . B^_j
//   dx_j  = sum_t w_tj G[t][j] dy_t + D dy_j + v_j U^T B^_j
//   dB^_j = sum_t w_tj dG[t][j] C^_t + v_j U x_j
//   dC^_t = sum_j w_tj dG[t][j] B^_j + e^{cum_t} S_{c-1} dy_t
//   dJ/dw_tj = dG[t][j] G[t][j] -> cum_t, cum_j, sigma_j (j < t), gamma_t (j = t)
//   dJ/dv_j = <B^_j, U x_j>      -> cum_e, cum_j, sigma_j
//   y's state term               -> cum_t (e^{cum_t} <C^_t, S_{c-1} dy_t>)
//   S_c's rotation and decay     -> psi_e, cum_e
//   dpsi_t[i] = (dC^ x C^ + dB^ x B^)_t[i] (the 2-D cross product of the
//   pair (i, i + N/2)), dB = R(psi_t) dB^, dC = R(psi_t) dC^;
//   then the prefix sums are transposed (suffix sums over the chunk:
//   d(dt_u A_u) = sum_{t>=u} dcum_t, dtheta_u = sum_{t>=u} dpsi_t) and the
//   chain runs through gamma, sigma, dt, lambda and A.
//
// Kernels (one stream, in order):
//   k_bwd_aggr   per chunk: M_c rotated by psi_e (A_c), sum_t e^{cum_t} C^_t dy_t^T,
//                and the chunk totals (cum_e, psi_e)                    (MFMA)
//   k_bwd_pass   per (slice, pair i, column p): the forward states S_{c-1},
//                then the reverse sweep G -> U, the state terms of dpsi_e
//                and dcum_e, and dJ/d(initial state)
//   k_bwd_chunk  per chunk: every gradient of the chunk's tokens         (MFMA)
//   k_bwd_finish the sigma term that crosses into the next chunk's first
//                token; per-head sums of dA and dD (fixed order)
// Operands are bf16 with fp32 accumulation (as the forward); the prefix
// sums, weights and every scalar gradient are fp32.  Results are
// deterministic: no atomics.
#include "m3_device.h"
#include "m3_internal.h"
#include "m3_scan_common.h"

namespace m3 {
namespace {

using namespace scan;

constexpr int kN = 128, kP = 64, kNH = 64, kRows = 64, kThr = 256;
constexpr int LDN = kN + 8;   // bf16 row strides (16-byte padding)
constexpr int LDP = kP + 8;
typedef Mma<bf16> MM;

// Per-chunk scalars shared by the chunk kernels (NT threads a workgroup).
template <int Q, int NT>
struct alignas(16) Pro {
    static constexpr int kSeg = NT / kNH;     // token segments of the angle scans
    float cum[Q], gam[Q], sig[Q], v[Q], ec[Q];
    h2 cs[Q * kNH];      // cos / sin of psi_t[i]
    float psie[kNH];
    float seg[kSeg][kNH];
};

// Chunk-local prefix sums, trapezoid weights, v_j and e^{cum_t}: the
// log-decay by one wavefront scan over the tokens; the angles by thread
// (pair i, token segment), all of a thread's angle loads issued together,
// segment totals combined through LDS.  Tokens past the end of the sequence
// get zero weights and zero angles.
template <int Q, int NT>
__device__ void bwd_prologue(const BwdArgs &a, int64_t b, int64_t h, int64_t t0, int nvalid,
                             Pro<Q, NT> &sp) {
    constexpr int TPS = (Q + Pro<Q, NT>::kSeg - 1) / Pro<Q, NT>::kSeg;
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int i = tid % kNH, seg = tid / kNH;
    const float *th = a.theta + ((b * a.L + t0) * a.H + h) * kNH + i;
    float ps[TPS];
#pragma unroll
    for (int k = 0; k < TPS; ++k) {
        const int t = seg * TPS + k;
        ps[k] = t < nvalid ? th[(int64_t)t * a.H * kNH] : 0.f;
    }
    float lg = 0.f, gam = 0.f, sig = 0.f;
    if (tid < kWave && tid < nvalid) {
        const int64_t t = t0 + tid, k = (b * a.L + t) * a.H + h;
        const float dtv = a.dt[k], lamv = a.lam[k];
        lg = dtv * a.A[b * a.a_sb + t * a.a_st + h * a.a_sh];
        gam = lamv * dtv;
        sig = gam;
        if (t + 1 < a.L) sig += (1.f - a.lam[k + a.H]) * a.dt[k + a.H];
    }
    float run = 0.f;
#pragma unroll
    for (int k = 0; k < TPS; ++k) {
        run += ps[k];
        ps[k] = run;
    }
    sp.seg[seg][i] = run;
    if (tid < kWave) {
        const float cum = wave_incl_scan(lg, lane);
        if (tid < Q) {
            sp.cum[tid] = cum;
            sp.gam[tid] = gam;
            sp.sig[tid] = sig;
        }
    }
    __syncthreads();
    float off = 0.f;
    for (int s2 = 0; s2 < seg; ++s2) off += sp.seg[s2][i];
#pragma unroll
    for (int k = 0; k < TPS; ++k) {
        const int t = seg * TPS + k;
        if (t < Q) {
            const float psi = ps[k] + off;
            float sn, cs;
            sincos_fast(psi, &sn, &cs);
            cs_put(&sp.cs[t * kNH + i], cs, sn);
            if (t == nvalid - 1) sp.psie[i] = psi;
        }
    }
    if (tid < Q) {
        const float cume = sp.cum[nvalid - 1];
        sp.v[tid] = tid < nvalid ? __expf(cume - sp.cum[tid]) * sp.sig[tid] : 0.f;
        sp.ec[tid] = tid < nvalid ? __expf(sp.cum[tid]) : 0.f;
    }
    __syncthreads();
}

// B or C rows of the chunk rotated by -psi_t into LDS [row][LDN] (bf16);
// rows past the end are zero.  Row = (token, rank).
template <int R, int NT>
__device__ void stage_rot(bf16 *dst, const bf16 *src, int64_t tokstr, int nvalid, const h2 *cs) {
    for (int task = threadIdx.x; task < kRows * 8; task += NT) {
        const int row = task / 8, cp = task % 8, t = row / R, r = row % R;
        bf16x8 lo, hi;
        if (t < nvalid) {
            const bf16 *p = src + t * tokstr + r * kN + cp * 8;
            lo = *reinterpret_cast<const bf16x8 *>(p);
            hi = *reinterpret_cast<const bf16x8 *>(p + kNH);
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) lo[e] = hi[e] = (bf16)0.f;
        }
        float c[8], s[8];
        cs_getn<8>(&cs[t * kNH + cp * 8], c, s);   // (t < chunk: rows are within it)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float u = (float)lo[e], w = (float)hi[e];
            lo[e] = (bf16)(c[e] * u + s[e] * w);
            hi[e] = (bf16)(c[e] * w - s[e] * u);
        }
        *reinterpret_cast<bf16x8 *>(&dst[row * LDN + cp * 8]) = lo;
        *reinterpret_cast<bf16x8 *>(&dst[row * LDN + kNH + cp * 8]) = hi;
    }
}

// x-like rows (P wide) into LDS [row][LDP], optionally scaled per token.
template <int R, int NT>
__device__ void stage_rows(bf16 *dst, const bf16 *src, int64_t tokstr, int nvalid, const float *scale) {
    for (int task = threadIdx.x; task < kRows * 8; task += NT) {
        const int row = task / 8, cp = task % 8, t = row / R, r = row % R;
        bf16x8 v;
        if (t < nvalid) {
            v = *reinterpret_cast<const bf16x8 *>(src + t * tokstr + r * kP + cp * 8);
            if (scale) {
                const float sc = scale[t];
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = (bf16)(sc * (float)v[e]);
            }
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = (bf16)0.f;
        }
        *reinterpret_cast<bf16x8 *>(&dst[row * LDP + cp * 8]) = v;
    }
}

// ---------------------------------------------------------------------------
// k_bwd_aggr: A_c = R(psi_e) sum_j v_j B^_j x_j^T and Mb_c = sum_t e^{cum_t}
// C^_t dy_t^T (N x P, fp32), chunk totals.  Wave w owns the N-row tiles w
// and w + 4 (the two rows of a rotation pair) for all four P tiles.
// ---------------------------------------------------------------------------
template <int R>
__global__ __launch_bounds__(kThr) void k_bwd_aggr(BwdArgs a) {
    constexpr int Q = kRows / R;
    __shared__ Pro<Q, kThr> sp;
    __shared__ __attribute__((aligned(16))) bf16 s_B[kRows * LDN];
    __shared__ __attribute__((aligned(16))) bf16 s_C[kRows * LDN];
    __shared__ __attribute__((aligned(16))) bf16 s_vX[kRows * LDP];
    __shared__ __attribute__((aligned(16))) bf16 s_eY[kRows * LDP];

    const int64_t slot = blockIdx.x, bh = slot / a.nchunks, c = slot % a.nchunks;
    const int64_t b = bh / a.H, h = bh % a.H, t0 = c * Q;
    const int nvalid = (int)min((int64_t)Q, a.L - t0);
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int g = lane >> 4, l16 = lane & 15;
    bwd_prologue<Q, kThr>(a, b, h, t0, nvalid, sp);

    const int64_t tok0 = (b * a.L + t0) * a.H + h;
    stage_rot<R, kThr>(s_B, static_cast<const bf16 *>(a.B) + tok0 * (R * kN), a.H * R * kN, nvalid, sp.cs);
    stage_rot<R, kThr>(s_C, static_cast<const bf16 *>(a.C) + tok0 * (R * kN), a.H * R * kN, nvalid, sp.cs);
    stage_rows<R, kThr>(s_vX, static_cast<const bf16 *>(a.x) + tok0 * (R * kP), a.H * R * kP, nvalid, sp.v);
    stage_rows<R, kThr>(s_eY, static_cast<const bf16 *>(a.dy) + tok0 * (R * kP), a.H * R * kP, nvalid, sp.ec);
    __syncthreads();

    f32x4 am[2][4], bm[2][4];
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int pt = 0; pt < 4; ++pt) am[q][pt] = bm[q][pt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        bf16x8 ab[2], ac[2];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            ab[q] = load_kt(s_B, LDN, ks * 32, (wave + 4 * q) * 16, g, l16);
            ac[q] = load_kt(s_C, LDN, ks * 32, (wave + 4 * q) * 16, g, l16);
        }
#pragma unroll
        for (int pt = 0; pt < 4; ++pt) {
            const bf16x8 bx = load_kt(s_vX, LDP, ks * 32, pt * 16, g, l16);
            const bf16x8 by = load_kt(s_eY, LDP, ks * 32, pt * 16, g, l16);
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                am[q][pt] = MM::mma(ab[q], bx, am[q][pt]);
                bm[q][pt] = MM::mma(ac[q], by, bm[q][pt]);
            }
        }
    }
    const int64_t NP = kN * kP;
    float *Af = a.Af + slot * NP, *Mb = a.Mb + slot * NP;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const int i = wave * 16 + 4 * g + v;          // pair (i, i + N/2)
        float sn, cs;
        sincos_fast(sp.psie[i], &sn, &cs);
#pragma unroll
        for (int pt = 0; pt < 4; ++pt) {
            const int p = pt * 16 + l16;
            const float re = am[0][pt][v], im = am[1][pt][v];
            Af[i * kP + p] = cs * re - sn * im;
            Af[(i + kNH) * kP + p] = sn * re + cs * im;
            Mb[i * kP + p] = bm[0][pt][v];
            Mb[(i + kNH) * kP + p] = bm[1][pt][v];
        }
    }
    float *tot = a.tot + slot * (1 + kNH);
    if (tid == 0) tot[0] = sp.cum[nvalid - 1];
    if (tid < kNH) tot[1 + tid] = sp.psie[tid];
}

// ---------------------------------------------------------------------------
// k_bwd_pass: per (slice, pair i, column p) the forward chunk states, then the
// reverse sweep.  A wavefront holds the 64 columns of one pair, so the state
// terms of dpsi_e[i] and dcum_e (sums over columns) are wavefront sums.
// Grid: slices x (N/2 * P / 256).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThr) void k_bwd_pass(BwdArgs a, int per) {
    const int64_t bh = blockIdx.x / per;
    const int idx = (blockIdx.x % per) * kThr + threadIdx.x;
    const int i = idx / kP, p = idx % kP;   // (a wavefront: one i, all p)
    const int64_t NP = kN * kP, base = bh * a.nchunks;
    const int o_re = i * kP + p, o_im = (i + kNH) * kP + p;
    constexpr int DEPTH = 8;   // chunks whose loads are issued together
    bf16 *Sb = reinterpret_cast<bf16 *>(a.Sst);   // (bf16: an MFMA operand, and the decay term below)
    float sre = 0.f, sim = 0.f;
    if (a.init_state) {
        sre = a.init_state[bh * NP + o_re];
        sim = a.init_state[bh * NP + o_im];
    }
    for (int64_t c0 = 0; c0 < a.nchunks; c0 += DEPTH) {
        float ce[DEPTH], ps[DEPTH], are[DEPTH], aim[DEPTH];
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            const int64_t s = base + min(c0 + d, a.nchunks - 1);
            ce[d] = a.tot[s * (1 + kNH)];
            ps[d] = a.tot[s * (1 + kNH) + 1 + i];
            are[d] = a.Af[s * NP + o_re];
            aim[d] = a.Af[s * NP + o_im];
        }
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            if (c0 + d >= a.nchunks) break;
            const int64_t s = base + c0 + d;
            Sb[s * NP + o_re] = (bf16)sre;
            Sb[s * NP + o_im] = (bf16)sim;
            const float e = __expf(ce[d]);
            float sn, cs;
            sincos_fast(ps[d], &sn, &cs);
            const float nre = e * (cs * sre - sn * sim) + are[d];
            const float nim = e * (sn * sre + cs * sim) + aim[d];
            sre = nre;
            sim = nim;
        }
    }
    float gre = 0.f, gim = 0.f;
    if (a.dfinal) {
        gre = a.dfinal[bh * NP + o_re];
        gim = a.dfinal[bh * NP + o_im];
    }
    float xre = sre, xim = sim;   // S_c, from the last chunk down
    for (int64_t c1 = a.nchunks - 1; c1 >= 0; c1 -= DEPTH) {
        float ce[DEPTH], ps[DEPTH], pre[DEPTH], pim[DEPTH], mre[DEPTH], mim[DEPTH];
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            const int64_t s = base + max(c1 - d, (int64_t)0);
            ce[d] = a.tot[s * (1 + kNH)];
            ps[d] = a.tot[s * (1 + kNH) + 1 + i];
            pre[d] = (float)Sb[s * NP + o_re];
            pim[d] = (float)Sb[s * NP + o_im];
            mre[d] = a.Mb[s * NP + o_re];
            mim[d] = a.Mb[s * NP + o_im];
        }
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            if (c1 - d < 0) break;
            const int64_t s = base + c1 - d;
            float sn, cs;
            sincos_fast(ps[d], &sn, &cs);
            const float e = __expf(ce[d]);
            float dps = gim * xre - gre * xim;                  // rotation of S_c by psi_e
            const float ure = cs * gre + sn * gim, uim = -sn * gre + cs * gim;
            float dcm = e * (ure * pre[d] + uim * pim[d]);      // decay e^{cum_e} of S_{c-1}
#pragma unroll
            for (int o = 1; o < kWave; o <<= 1) {
                dps += __shfl_xor(dps, o, kWave);
                dcm += __shfl_xor(dcm, o, kWave);
            }
            if (p == 0) {
                a.pst[s * (2 * kNH) + i] = dps;
                a.pst[s * (2 * kNH) + kNH + i] = dcm;
            }
            bf16 *Ub = reinterpret_cast<bf16 *>(a.Ust);   // (bf16: read only as an MFMA operand)
            Ub[s * NP + o_re] = (bf16)ure;
            Ub[s * NP + o_im] = (bf16)uim;
            gre = e * ure + mre[d];
            gim = e * uim + mim[d];
            xre = pre[d];
            xim = pim[d];
        }
    }
    if (a.dinit) {
        a.dinit[bh * NP + o_re] = gre;
        a.dinit[bh * NP + o_im] = gim;
    }
}

// Sum over the 16 lanes of a row group (lanes l16 = 0..15 with the same g).
__device__ __forceinline__ float sum16(float v) {
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

// ---------------------------------------------------------------------------
// k_bwd_chunk: every gradient of one chunk, eight waves.  Waves 0-3 own row
// tile w as a column block (j rows: dx, dB^, the masked-score columns),
// waves 4-7 row tile w - 4 as a row block (t rows: dC^, the y state term);
// the two halves only read the staged operands, so they run side by side
// (two waves a SIMD).
// ---------------------------------------------------------------------------
constexpr int kThrC = 512;
template <int R>
__global__ __launch_bounds__(kThrC) void k_bwd_chunk(BwdArgs a) {
    constexpr int Q = kRows / R;
    __shared__ Pro<Q, kThrC> sp;
    __shared__ __attribute__((aligned(16))) bf16 s_B[kRows * LDN];
    __shared__ __attribute__((aligned(16))) bf16 s_C[kRows * LDN];
    __shared__ __attribute__((aligned(16))) bf16 s_X[kRows * LDP];
    __shared__ __attribute__((aligned(16))) bf16 s_dY[kRows * LDP];
    __shared__ __attribute__((aligned(16))) bf16 s_S[kN * LDP];   // S_{c-1} [n][p]
    __shared__ __attribute__((aligned(16))) bf16 s_U[kN * LDP];   // U_c [n][p]
    __shared__ float s_dpsi[2][kRows * kNH];                      // per row, per pair: B^ and C^ parts
    __shared__ float s_rc[4][kRows], s_rg[4][kRows];              // per-wave row sums of the mask terms
    __shared__ float s_cc[kRows], s_cs[kRows];                    // column sums (cum, sigma)
    __shared__ float s_dv[kRows], s_dcy[kRows];                   // dJ/dv_j, y state term of cum_t
    __shared__ float s_tok[3][kWave];                             // per token: dcum, dsigma, dgamma
    __shared__ float s_red[2][4];
    __shared__ float s_segd[kThrC / kWave - 1][kNH];                // dtheta: segment totals

    const int64_t slot = blockIdx.x, bh = slot / a.nchunks, c = slot % a.nchunks;
    const int64_t b = bh / a.H, h = bh % a.H, t0 = c * Q;
    const int nvalid = (int)min((int64_t)Q, a.L - t0);
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int g = lane >> 4, l16 = lane & 15;
    bwd_prologue<Q, kThrC>(a, b, h, t0, nvalid, sp);

    const int64_t tok0 = (b * a.L + t0) * a.H + h;
    const int64_t bstr = a.H * R * kN, xstr = a.H * R * kP;
    stage_rot<R, kThrC>(s_B, static_cast<const bf16 *>(a.B) + tok0 * (R * kN), bstr, nvalid, sp.cs);
    stage_rot<R, kThrC>(s_C, static_cast<const bf16 *>(a.C) + tok0 * (R * kN), bstr, nvalid, sp.cs);
    stage_rows<R, kThrC>(s_X, static_cast<const bf16 *>(a.x) + tok0 * (R * kP), xstr, nvalid, nullptr);
    stage_rows<R, kThrC>(s_dY, static_cast<const bf16 *>(a.dy) + tok0 * (R * kP), xstr, nvalid, nullptr);
    {
        const int64_t NP = kN * kP;
        const bf16x4 *Sg = reinterpret_cast<const bf16x4 *>(reinterpret_cast<const bf16 *>(a.Sst) + slot * NP);
        const bf16x4 *Ug = reinterpret_cast<const bf16x4 *>(reinterpret_cast<const bf16 *>(a.Ust) + slot * NP);
        for (int q = tid; q < kN * kP / 4; q += kThrC) {
            const int n = (4 * q) / kP, p = (4 * q) % kP;
            *reinterpret_cast<bf16x4 *>(&s_S[n * LDP + p]) = Sg[q];
            *reinterpret_cast<bf16x4 *>(&s_U[n * LDP + p]) = Ug[q];
        }
    }
    __syncthreads();
    const float Dh = a.D[h];

    float xdy = 0.f;
    if (wave < 4) {
    // ============ column block J = wave: dx and dB^ of rows j ============
    const int J = wave;
    f32x4 gt[4], dg[4];   // G and dG tiles (T, J): lane element (t = 16T + 4g + v, j = 16J + l16)
#pragma unroll
    for (int T = 0; T < 4; ++T) {
        gt[T] = dg[T] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (T >= J) {
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
                gt[T] = MM::mma(MM::load(&s_C[(T * 16 + l16) * LDN + kk * 32 + 8 * g]),
                                MM::load(&s_B[(J * 16 + l16) * LDN + kk * 32 + 8 * g]), gt[T]);
#pragma unroll
            for (int kk = 0; kk < 2; ++kk)
                dg[T] = MM::mma(MM::load(&s_dY[(T * 16 + l16) * LDP + kk * 32 + 8 * g]),
                                MM::load(&s_X[(J * 16 + l16) * LDP + kk * 32 + 8 * g]), dg[T]);
        }
    }
    {
        const int jrow = J * 16 + l16, tj = jrow / R;
        const float cum_j = sp.cum[tj], sig_j = sp.sig[tj];
        float colc = 0.f, cols = 0.f;
#pragma unroll
        for (int T = 0; T < 4; ++T) {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int trow = T * 16 + 4 * g + v, tt = trow / R;
                float w = 0.f, e = 0.f;
                if (T >= J) {
                    if (tj < tt) {
                        e = __expf(sp.cum[tt] - cum_j);
                        w = e * sig_j;
                    } else if (tj == tt) {
                        w = sp.gam[tt];
                    }
                }
                const float dW = dg[T][v] * gt[T][v];      // dJ/dw_tj
                const float val = (tj < tt) ? dW * w : 0.f;
                const float rg = (tj == tt) ? dW : 0.f;
                colc += val;
                cols += (tj < tt) ? dW * e : 0.f;
                gt[T][v] *= w;
                dg[T][v] *= w;
                const float rcs = sum16(val), rgs = sum16(rg);
                if (l16 == 0) {
                    s_rc[J][trow] = rcs;
                    s_rg[J][trow] = rgs;
                }
            }
        }
        colc += __shfl_xor(colc, 16, kWave);
        colc += __shfl_xor(colc, 32, kWave);
        cols += __shfl_xor(cols, 16, kWave);
        cols += __shfl_xor(cols, 32, kWave);
        if (g == 0) {
            s_cc[jrow] = colc;
            s_cs[jrow] = cols;
        }
    }
    // dx_j = sum_t Gw[t][j] dy_t (K = t in pairs of row tiles; the lane's
    // K elements are rows 4g..4g+3 of both tiles, matched by transposing reads)
    f32x4 dxa[4], bu[4];
#pragma unroll
    for (int pt = 0; pt < 4; ++pt) dxa[pt] = bu[pt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kp = 0; kp < 2; ++kp) {
        if (2 * kp + 1 < J) continue;
        bf16x8 af;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            af[v] = (bf16)gt[2 * kp][v];
            af[4 + v] = (bf16)gt[2 * kp + 1][v];
        }
#pragma unroll
        for (int pt = 0; pt < 4; ++pt) {
            const bf16 *yr = &s_dY[(32 * kp + 4 * g + l16 / 4) * LDP + pt * 16 + 4 * (l16 % 4)];
            const bf16x4 lo = lds_tr4(yr), hi = lds_tr4(yr + 16 * LDP);
            bf16x8 bfr;
#pragma unroll
            for (int v = 0; v < 4; ++v) { bfr[v] = lo[v]; bfr[4 + v] = hi[v]; }
            dxa[pt] = MM::mma(af, bfr, dxa[pt]);
        }
    }
    // (B^ U)_j, K = N
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        const bf16x8 ab = MM::load(&s_B[(J * 16 + l16) * LDN + kk * 32 + 8 * g]);
#pragma unroll
        for (int pt = 0; pt < 4; ++pt)
            bu[pt] = MM::mma(ab, load_kt(s_U, LDP, kk * 32, pt * 16, g, l16), bu[pt]);
    }
    {
        bf16 *dxg = static_cast<bf16 *>(a.dx) + tok0 * (R * kP);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int j = J * 16 + 4 * g + v, t = j / R, r = j % R;
            const float vj = sp.v[t];
            float dvp = 0.f;
#pragma unroll
            for (int pt = 0; pt < 4; ++pt) {
                const int p = pt * 16 + l16;
                const float xv = (float)s_X[j * LDP + p], yv = (float)s_dY[j * LDP + p];
                dvp += xv * bu[pt][v];
                xdy += xv * yv;
                const float d = dxa[pt][v] + vj * bu[pt][v] + Dh * yv;
                if (t < nvalid) dxg[t * xstr + r * kP + p] = (bf16)d;
            }
            dvp = sum16(dvp);
            if (l16 == 0) s_dv[j] = dvp;
        }
    }
    // dB^_j = sum_t Wd[t][j] C^_t + v_j U x_j
    f32x4 db[8], xu[8];
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) db[nt] = xu[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kp = 0; kp < 2; ++kp) {
        if (2 * kp + 1 < J) continue;
        bf16x8 af;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            af[v] = (bf16)dg[2 * kp][v];
            af[4 + v] = (bf16)dg[2 * kp + 1][v];
        }
#pragma unroll
        for (int nt = 0; nt < 8; ++nt) {
            const bf16 *cr = &s_C[(32 * kp + 4 * g + l16 / 4) * LDN + nt * 16 + 4 * (l16 % 4)];
            const bf16x4 lo = lds_tr4(cr), hi = lds_tr4(cr + 16 * LDN);
            bf16x8 bfr;
#pragma unroll
            for (int v = 0; v < 4; ++v) { bfr[v] = lo[v]; bfr[4 + v] = hi[v]; }
            db[nt] = MM::mma(af, bfr, db[nt]);
        }
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
        const bf16x8 ax = MM::load(&s_X[(J * 16 + l16) * LDP + kk * 32 + 8 * g]);
#pragma unroll
        for (int nt = 0; nt < 8; ++nt)
            xu[nt] = MM::mma(ax, MM::load(&s_U[(nt * 16 + l16) * LDP + kk * 32 + 8 * g]), xu[nt]);
    }
    {
        bf16 *dbg = static_cast<bf16 *>(a.dB) + tok0 * (R * kN);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int j = J * 16 + 4 * g + v, t = j / R, r = j % R;
            const float vj = sp.v[t];
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) {
                const int i = nt * 16 + l16;
                const float re = db[nt][v] + vj * xu[nt][v], im = db[nt + 4][v] + vj * xu[nt + 4][v];
                const float bre = (float)s_B[j * LDN + i], bim = (float)s_B[j * LDN + i + kNH];
                s_dpsi[0][j * kNH + i] = re * bim - im * bre;
                float cs, sn;
                cs_get(sp.cs[t * kNH + i], cs, sn);
                if (t < nvalid) {
                    dbg[t * bstr + r * kN + i] = (bf16)(cs * re - sn * im);
                    dbg[t * bstr + r * kN + i + kNH] = (bf16)(sn * re + cs * im);
                }
            }
        }
    }

    } else {
    // ============ row block T = wave - 4: dC^ of rows t ============
    const int T = wave - 4;
    f32x4 gT[4];   // dG^T tiles (J, T): lane element (j = 16J + 4g + v, t = 16T + l16)
#pragma unroll
    for (int Jt = 0; Jt < 4; ++Jt) {
        gT[Jt] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (Jt <= T) {
#pragma unroll
            for (int kk = 0; kk < 2; ++kk)
                gT[Jt] = MM::mma(MM::load(&s_X[(Jt * 16 + l16) * LDP + kk * 32 + 8 * g]),
                                 MM::load(&s_dY[(T * 16 + l16) * LDP + kk * 32 + 8 * g]), gT[Jt]);
            const int tt = (T * 16 + l16) / R;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int tj = (Jt * 16 + 4 * g + v) / R;
                float w = 0.f;
                if (tj < tt) w = __expf(sp.cum[tt] - sp.cum[tj]) * sp.sig[tj];
                else if (tj == tt) w = sp.gam[tt];
                gT[Jt][v] *= w;
            }
        }
    }
    f32x4 dc[8], t2[8];
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) dc[nt] = t2[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int jp = 0; jp < 2; ++jp) {
        if (2 * jp > T) continue;
        bf16x8 af;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            af[v] = (bf16)gT[2 * jp][v];
            af[4 + v] = (bf16)gT[2 * jp + 1][v];
        }
#pragma unroll
        for (int nt = 0; nt < 8; ++nt) {
            const bf16 *br = &s_B[(32 * jp + 4 * g + l16 / 4) * LDN + nt * 16 + 4 * (l16 % 4)];
            const bf16x4 lo = lds_tr4(br), hi = lds_tr4(br + 16 * LDN);
            bf16x8 bfr;
#pragma unroll
            for (int v = 0; v < 4; ++v) { bfr[v] = lo[v]; bfr[4 + v] = hi[v]; }
            dc[nt] = MM::mma(af, bfr, dc[nt]);
        }
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
        const bf16x8 ay = MM::load(&s_dY[(T * 16 + l16) * LDP + kk * 32 + 8 * g]);
#pragma unroll
        for (int nt = 0; nt < 8; ++nt)
            t2[nt] = MM::mma(ay, MM::load(&s_S[(nt * 16 + l16) * LDP + kk * 32 + 8 * g]), t2[nt]);
    }
    {
        bf16 *dcg = static_cast<bf16 *>(a.dC) + tok0 * (R * kN);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int trow = T * 16 + 4 * g + v, t = trow / R, r = trow % R;
            const float ec = sp.ec[t];
            float dcy = 0.f;
#pragma unroll
            for (int nt = 0; nt < 8; ++nt) dcy += (float)s_C[trow * LDN + nt * 16 + l16] * t2[nt][v];
            dcy = sum16(dcy);
            if (l16 == 0) s_dcy[trow] = ec * dcy;
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) {
                const int i = nt * 16 + l16;
                const float re = dc[nt][v] + ec * t2[nt][v], im = dc[nt + 4][v] + ec * t2[nt + 4][v];
                const float cre = (float)s_C[trow * LDN + i], cim = (float)s_C[trow * LDN + i + kNH];
                s_dpsi[1][trow * kNH + i] = re * cim - im * cre;
                float cs, sn;
                cs_get(sp.cs[t * kNH + i], cs, sn);
                if (t < nvalid) {
                    dcg[t * bstr + r * kN + i] = (bf16)(cs * re - sn * im);
                    dcg[t * bstr + r * kN + i + kNH] = (bf16)(sn * re + cs * im);
                }
            }
        }
    }
    }
    // <x, dy> over the chunk (the skip term's gradient), one value per
    // column-block wave
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) xdy += __shfl_xor(xdy, o, kWave);
    if (lane == 0 && wave < 4) s_red[0][wave] = xdy;
    __syncthreads();

    // ============ per-token scalars ============
    const float *pst = a.pst + slot * (2 * kNH);
    if (tid < kRows) {   // rows -> tokens
        const int row = tid;
        const float rc = s_rc[0][row] + s_rc[1][row] + s_rc[2][row] + s_rc[3][row];
        const float rg = s_rg[0][row] + s_rg[1][row] + s_rg[2][row] + s_rg[3][row];
        const int t = row / R;
        const float vt = sp.v[t];
        const float et = t < nvalid ? __expf(sp.cum[nvalid - 1] - sp.cum[t]) : 0.f;   // v_t / sigma_t
        const float dcum = rc - s_cc[row] - s_dv[row] * vt + s_dcy[row];
        const float dsig = s_cs[row] + s_dv[row] * et;
        // rank rows of a token are R consecutive lanes: sum them
        float sc = dcum, ss = dsig, sg = rg;
#pragma unroll
        for (int o = 1; o < R; o <<= 1) {
            sc += __shfl_xor(sc, o, kWave);
            ss += __shfl_xor(ss, o, kWave);
            sg += __shfl_xor(sg, o, kWave);
        }
        if (row % R == 0) {
            s_tok[0][t] = sc;
            s_tok[1][t] = ss;
            s_tok[2][t] = sg;
        }
        // dcum_e: the v_j terms and the state decay (per pair, from the pass)
        float ce = s_dv[row] * vt + pst[kNH + row];
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) ce += __shfl_xor(ce, o, kWave);
        if (row == 0) s_red[1][0] = ce;
    }
    __syncthreads();
    if (tid < kWave) {   // one lane per token (Q <= 64)
        const int t = tid;
        float dcum = t < Q ? s_tok[0][t] : 0.f;
        if (t == nvalid - 1) dcum += s_red[1][0];
        // d(dt_u A_u) = sum_{t >= u} dcum_t: an inclusive scan in reverse token
        // order (lane m holds token Q - 1 - m; lanes past the chunk hold zero)
        const int rev = max(Q - 1 - t, 0);
        const float rv = __shfl(dcum, rev, kWave);
        const float rsc = wave_incl_scan(t < Q ? rv : 0.f, t);
        const float da = __shfl(rsc, rev, kWave);
        const float dsig = t < Q ? s_tok[1][t] : 0.f;
        const float dsig_prev = __shfl(dsig, t > 0 ? t - 1 : 0, kWave);
        const float dgam = (t < Q ? s_tok[2][t] : 0.f) + dsig;   // sigma_t = gamma_t + ...
        float dAt = 0.f;
        if (t < nvalid) {
            const int64_t tg = t0 + t, k = (b * a.L + tg) * a.H + h;
            const float dtv = a.dt[k], lamv = a.lam[k];
            const float Av = a.A[b * a.a_sb + tg * a.a_st + h * a.a_sh];
            float ddt = Av * da + lamv * dgam;
            float dl = dtv * dgam;
            if (t > 0) {   // the previous token's sigma reads this token's lambda and dt
                ddt += (1.f - lamv) * dsig_prev;
                dl -= dtv * dsig_prev;
            }
            a.ddt[k] = ddt;
            a.dlam[k] = dl;
            dAt = dtv * da;
            if (a.dA_per_token) a.dA[k] = dAt;
            if (t == nvalid - 1) a.dsig[slot] = dsig;
        }
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) dAt += __shfl_xor(dAt, o, kWave);
        if (t == 0) {
            a.dApart[slot] = dAt;
            a.dDpart[slot] = s_red[0][0] + s_red[0][1] + s_red[0][2] + s_red[0][3];
        }
    }
    // dtheta: suffix sums over the chunk's tokens of dpsi per pair (lane i),
    // by waves 1 .. 7, one segment of TSD consecutive tokens each: the
    // segment's own suffix sums, then the totals of the later segments
    // through LDS
    constexpr int NSD = kThrC / kWave - 1, TSD = (Q + NSD - 1) / NSD;
    const int sd = wave - 1, i = lane;
    float dl[TSD];
    if (wave >= 1) {
        float acc = 0.f;
#pragma unroll
        for (int k = TSD - 1; k >= 0; --k) {
            const int t = sd * TSD + k;
            float d = 0.f;
            if (t < nvalid) {
#pragma unroll
                for (int r = 0; r < R; ++r)
                    d += s_dpsi[0][(t * R + r) * kNH + i] + s_dpsi[1][(t * R + r) * kNH + i];
                if (t == nvalid - 1) d += pst[i];
            }
            acc += d;
            dl[k] = acc;
        }
        s_segd[sd][i] = acc;
    }
    __syncthreads();
    if (wave >= 1) {
        float off = 0.f;
        for (int s2 = sd + 1; s2 < NSD; ++s2) off += s_segd[s2][i];
        float *dth = a.dtheta + tok0 * kNH + i;
#pragma unroll
        for (int k = 0; k < TSD; ++k) {
            const int t = sd * TSD + k;
            if (t < nvalid) dth[(int64_t)t * a.H * kNH] = dl[k] + off;
        }
    }
}

// The sigma term of each chunk's last token reaching the next chunk's first
// token: sigma_e = gamma_e + (1 - lambda_{e+1}) dt_{e+1}.
__global__ __launch_bounds__(kThr) void k_bwd_finish(BwdArgs a, int Q) {
    const int64_t s = (int64_t)blockIdx.x * kThr + threadIdx.x;
    if (s >= a.batch * a.H * a.nchunks) return;
    const int64_t bh = s / a.nchunks, c = s % a.nchunks;
    if (c == 0) return;
    const int64_t b = bh / a.H, h = bh % a.H;
    const int64_t k = (b * a.L + c * Q) * a.H + h;
    const float d = a.dsig[s - 1];
    a.ddt[k] += (1.f - a.lam[k]) * d;
    a.dlam[k] -= a.dt[k] * d;
}

// Per-head sums of the chunk partials (dD; dA when A is per head), in a fixed
// order: one workgroup per head.
__global__ __launch_bounds__(kThr) void k_bwd_reduce(BwdArgs a) {
    __shared__ float s_a[kThr], s_d[kThr];
    const int64_t h = blockIdx.x;
    const int64_t n = a.batch * a.nchunks;
    float sa = 0.f, sd = 0.f;
    for (int64_t q = threadIdx.x; q < n; q += kThr) {
        const int64_t b = q / a.nchunks, c = q % a.nchunks;
        const int64_t s = (b * a.H + h) * a.nchunks + c;
        sa += a.dApart[s];
        sd += a.dDpart[s];
    }
    s_a[threadIdx.x] = sa;
    s_d[threadIdx.x] = sd;
    __syncthreads();
    for (int w = kThr / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) {
            s_a[threadIdx.x] += s_a[threadIdx.x + w];
            s_d[threadIdx.x] += s_d[threadIdx.x + w];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        a.dD[h] = s_d[0];
        if (!a.dA_per_token) a.dA[h] = s_a[0];
    }
}

template <int R>
hipError_t launch_bwd(const BwdArgs &a, hipStream_t stream) {
    constexpr int Q = kRows / R;
    const int64_t BH = a.batch * a.H, nslot = BH * a.nchunks;
    if (a.nchunks > 0)
        hipLaunchKernelGGL((k_bwd_aggr<R>), dim3((unsigned)nslot), dim3(kThr), 0, stream, a);
    constexpr int per = kNH * kP / kThr;
    hipLaunchKernelGGL(k_bwd_pass, dim3((unsigned)(BH * per)), dim3(kThr), 0, stream, a, per);
    if (a.nchunks > 0) {
        hipLaunchKernelGGL((k_bwd_chunk<R>), dim3((unsigned)nslot), dim3(kThrC), 0, stream, a);
        hipLaunchKernelGGL(k_bwd_finish, dim3((unsigned)((nslot + kThr - 1) / kThr)), dim3(kThr), 0,
                           stream, a, Q);
    }
    hipLaunchKernelGGL(k_bwd_reduce, dim3((unsigned)a.H), dim3(kThr), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

BwdWorkspaceLayout bwd_workspace_layout(int64_t BH, int64_t nchunks, int64_t N, int64_t P) {
    auto up = [](size_t v) { return (v + 255) / 256 * 256; };
    const size_t per = (size_t)BH * (size_t)nchunks;
    const size_t st = per * (size_t)(N * P) * sizeof(float);
    BwdWorkspaceLayout w = {};
    w.off_Af = kCtlBytes;   // (the scans' control block, left untouched in a shared workspace)
    w.off_Mb = up(w.off_Af + st);
    w.off_Sst = up(w.off_Mb + st);
    w.off_Ust = up(w.off_Sst + st / 2);   // (bf16 maps)
    w.off_tot = up(w.off_Ust + st / 2);
    w.off_pst = up(w.off_tot + per * (size_t)(1 + N / 2) * sizeof(float));
    w.off_dsig = up(w.off_pst + per * (size_t)N * sizeof(float));
    w.off_dA = up(w.off_dsig + per * sizeof(float));
    w.off_dD = up(w.off_dA + per * sizeof(float));
    w.total = up(w.off_dD + per * sizeof(float));
    return w;
}

bwd_launch_fn find_bwd_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q) {
    if (io != 1 || N != kN || P != kP || R * Q != kRows) return nullptr;
    if (R == 1) return &launch_bwd<1>;
    if (R == 2) return &launch_bwd<2>;
    if (R == 4) return &launch_bwd<4>;
    return nullptr;
}

}  // namespace m3
