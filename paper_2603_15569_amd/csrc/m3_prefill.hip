// Chunked prefill scan of the Mamba-3 SSM on gfx950.
//
// Decomposition (Sec. 3.3 "Chunked Algorithm for MIMO SSMs", with the
// two-band mask of Sec. 3.1.2 eq. mamba3-mask and the rotary form of the
// complex state, Sec. 3.2 Prop. "Rotary Embedding Equivalence with
// Exponential-Trapezoidal Discretization").  For a chunk of Q tokens
// starting at t0, with chunk-local inclusive prefix sums
//     cum_t = sum_{u=t0..t} dt_u A_u,   psi_t[i] = sum_{u=t0..t} theta_u[i],
// rotated operands  C^_t = R(-psi_t) C_t,  B^_j = R(-psi_j) B_j  and the
// trapezoid weights  gamma_t = lambda_t dt_t,
//     sigma_j = gamma_j + (1 - lambda_{j+1}) dt_{j+1}   (sigma_{L-1} = gamma_{L-1}):
//   y_t = sum_{j<=t in chunk} w_tj (C^_t . B^_j) x_j + e^{cum_t} C^_t S_in + D x_t
//         w_tt = gamma_t,  w_tj = e^{cum_t - cum_j} sigma_j
//   S_out = R(psi_e) (e^{cum_e} S_in + M),  M = sum_j e^{cum_e - cum_j} sigma_j B^_j x_j^T
// where e is the chunk's last token and S is kept in the physical frame with
// the next token's previous-input term already folded in.  (Rows index
// (token, rank column) pairs, so every product above is a rank-R sum.)
//
// Three kernels:
//   k_chunk_state : M and (cum_e, psi_e) for every chunk      (MFMA, K = chunk rows)
//   k_state_pass  : S_in of every chunk, final state, carry   (sequential over chunks)
//   k_chunk_out   : y for every chunk                          (MFMA, K = N and chunk rows)
#include "m3_device.h"
#include "m3_internal.h"

namespace m3 {
namespace {

template <typename T, int N_, int P_, int R_, int Q_>
struct Shape {
    static constexpr int N = N_, P = P_, R = R_, Q = Q_;
    static constexpr int NH = N / 2;
    static constexpr int QR = Q * R;
    static constexpr int BLK = 64;                 // chunk rows staged per block
    static constexpr int NBLK = QR / BLK;
    static constexpr int PAD = 16 / (int)sizeof(T); // 16-byte row padding
    static constexpr int LDN = N + PAD;            // stride of [rows][N] tiles
    static constexpr int LDB = BLK + PAD;          // stride of [N or P][BLK] tiles
    static constexpr int LDPSI = NH + 1;
    typedef typename AccOf<T>::type Acc;
    static_assert(QR % BLK == 0, "chunk*rank must be a multiple of 64");
    static_assert(N % Mma<T>::K == 0 && BLK % Mma<T>::K == 0, "K tiling");
    static_assert(N % 16 == 0 && P % 16 == 0, "16x16 tiles");
    static_assert(16 % R == 0, "16-row tiles must hold whole tokens");
    static_assert(Q <= kBlock, "one thread per token in the prologue");
};

// Per-chunk scalars: cum (inclusive prefix of dt*A), gamma, sigma and the
// angle prefix psi[t][i], all chunk-local.  Tokens past the end of the
// sequence get dt = lambda = 0 (no decay, no weight) and zero angles.
template <class S>
__device__ void chunk_prologue(const ScanArgs &a, int64_t b, int64_t h, int64_t t0, int nvalid,
                               typename S::Acc *s_cum, float *s_gam, float *s_sig,
                               typename S::Acc *s_psi) {
    typedef typename S::Acc Acc;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    if (tid < S::Q) {
        Acc lg = 0;
        float gam = 0.f, sig = 0.f;
        if (tid < nvalid) {
            const int64_t t = t0 + tid;
            const int64_t k = (b * a.L + t) * a.H + h;
            const float dtv = a.dt[k], lamv = a.lam[k];
            const float Av = a.A[b * a.a_sb + t * a.a_st + h * a.a_sh];
            lg = (Acc)dtv * (Acc)Av;
            gam = lamv * dtv;
            sig = gam;
            if (t + 1 < a.L) {
                const int64_t kn = k + a.H;
                sig += (1.f - a.lam[kn]) * a.dt[kn];
            }
        }
        s_cum[tid] = lg;
        s_gam[tid] = gam;
        s_sig[tid] = sig;
    }
    // per-token angles, or dt * omega with the head's frequencies omega
    const float *th = a.theta_ph ? a.theta + h * S::NH : a.theta + ((b * a.L + t0) * a.H + h) * S::NH;
    const int64_t tstride = a.theta_ph ? 0 : a.H * S::NH;
    const float *dtc = a.dt + (b * a.L + t0) * a.H + h;
    for (int e = tid; e < S::Q * S::NH; e += kBlock) {
        const int t = e / S::NH, i = e % S::NH;
        const float v = (t < nvalid) ? th[t * tstride + i] * (a.theta_ph ? dtc[t * a.H] : 1.f) : 0.f;
        s_psi[t * S::LDPSI + i] = (Acc)v;
    }
    __syncthreads();
    // Columns 0..NH-1 are the angle scans, column NH the log-decay scan.
    for (int col = wave; col <= S::NH; col += kBlock / kWave) {
        Acc carry = 0;
        for (int seg = 0; seg < S::Q; seg += kWave) {
            const int t = seg + lane;
            Acc v = 0;
            if (t < S::Q) v = (col < S::NH) ? s_psi[t * S::LDPSI + col] : s_cum[t];
            v = wave_incl_scan(v, lane) + carry;
            if (t < S::Q) {
                if (col < S::NH) s_psi[t * S::LDPSI + col] = v;
                else s_cum[t] = v;
            }
            carry = __shfl(v, kWave - 1, kWave);
        }
    }
    __syncthreads();
}

// Rotate rows row0 .. row0+63 of a chunk operand (B or C, rows = (token,
// rank) pairs) by -psi_t and store them row-major in dst[64][LDN].
template <class S, typename T>
__device__ void stage_rot_rows(T *dst, const T *src, int64_t tok_stride, int row0, int nvalid,
                               const typename S::Acc *s_psi) {
    typedef typename S::Acc Acc;
    for (int e = threadIdx.x; e < S::BLK * S::NH; e += kBlock) {
        const int rl = e / S::NH, i = e % S::NH;
        const int row = row0 + rl, t = row / S::R, r = row % S::R;
        Acc re = 0, im = 0;
        if (t < nvalid) {
            const T *p = src + t * tok_stride + r * S::N;
            const Acc u = (Acc)to_f32(p[i]), v = (Acc)to_f32(p[i + S::NH]);
            Acc sn, cs;
            sincos_acc(s_psi[t * S::LDPSI + i], &sn, &cs);
            re = cs * u + sn * v;
            im = cs * v - sn * u;
        }
        dst[rl * S::LDN + i] = from_f32<T>((float)re);
        dst[rl * S::LDN + i + S::NH] = from_f32<T>((float)im);
    }
}

// Same rotation, scaled by w[t], stored transposed: dst[n][row - row0].
template <class S, typename T>
__device__ void stage_rot_rows_t(T *dst, const T *src, int64_t tok_stride, int row0, int nvalid,
                                 const typename S::Acc *s_psi, const typename S::Acc *s_w) {
    typedef typename S::Acc Acc;
    for (int e = threadIdx.x; e < S::BLK * S::NH; e += kBlock) {
        const int rl = e / S::NH, i = e % S::NH;
        const int row = row0 + rl, t = row / S::R, r = row % S::R;
        Acc re = 0, im = 0;
        if (t < nvalid) {
            const T *p = src + t * tok_stride + r * S::N;
            const Acc u = (Acc)to_f32(p[i]), v = (Acc)to_f32(p[i + S::NH]);
            Acc sn, cs;
            sincos_acc(s_psi[t * S::LDPSI + i], &sn, &cs);
            const Acc w = s_w[t];
            re = w * (cs * u + sn * v);
            im = w * (cs * v - sn * u);
        }
        dst[i * S::LDB + rl] = from_f32<T>((float)re);
        dst[(i + S::NH) * S::LDB + rl] = from_f32<T>((float)im);
    }
}

// x rows row0 .. row0+63 of the chunk, transposed: dst[p][row - row0].
template <class S, typename T>
__device__ void stage_x_t(T *dst, const T *src, int64_t tok_stride, int row0, int nvalid) {
    for (int e = threadIdx.x; e < S::BLK * S::P; e += kBlock) {
        const int rl = e / S::P, p = e % S::P;
        const int row = row0 + rl, t = row / S::R, r = row % S::R;
        T v = from_f32<T>(0.f);
        if (t < nvalid) v = src[t * tok_stride + r * S::P + p];
        dst[p * S::LDB + rl] = v;
    }
}

// ---------------------------------------------------------------------------
// k_chunk_state: M = sum_j w_j B^_j x_j^T (N x P) per chunk, plus totals.
// Grid: one workgroup per (slice, chunk), slice-major.
// ---------------------------------------------------------------------------
template <typename T, int N, int P, int R, int Q>
__global__ __launch_bounds__(kBlock) void k_chunk_state(ScanArgs a) {
    typedef Shape<T, N, P, R, Q> S;
    typedef typename S::Acc Acc;
    typedef Mma<T> MM;
    __shared__ Acc s_cum[Q], s_w[Q];
    __shared__ float s_gam[Q], s_sig[Q];
    __shared__ Acc s_psi[Q * S::LDPSI];
    __shared__ __attribute__((aligned(16))) T s_Bt[N * S::LDB];
    __shared__ __attribute__((aligned(16))) T s_Xt[P * S::LDB];

    const int64_t blk = blockIdx.x;
    const int64_t bh = blk / a.nchunks, c = blk % a.nchunks;
    const int64_t b = bh / a.H, h = bh % a.H;
    const int64_t t0 = c * Q;
    const int nvalid = (int)min((int64_t)Q, a.L - t0);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4, l16 = lane & 15;

    chunk_prologue<S>(a, b, h, t0, nvalid, s_cum, s_gam, s_sig, s_psi);
    const Acc cum_e = s_cum[nvalid - 1];
    if (tid < Q) s_w[tid] = (tid < nvalid) ? exp_acc(cum_e - s_cum[tid]) * (Acc)s_sig[tid] : (Acc)0;
    __syncthreads();

    const T *Bsrc = static_cast<const T *>(a.B) + ((b * a.L + t0) * a.H + h) * (R * N);
    const T *Xsrc = static_cast<const T *>(a.x) + ((b * a.L + t0) * a.H + h) * (R * P);
    const int64_t bstride = a.H * R * N, xstride = a.H * R * P;

    constexpr int NT = (N / 16) * (P / 16);
    constexpr int TPW = (NT + 3) / 4;
    f32x4 acc[TPW];
#pragma unroll
    for (int k = 0; k < TPW; ++k) acc[k] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int jb = 0; jb < S::NBLK; ++jb) {
        stage_rot_rows_t<S, T>(s_Bt, Bsrc, bstride, jb * S::BLK, nvalid, s_psi, s_w);
        stage_x_t<S, T>(s_Xt, Xsrc, xstride, jb * S::BLK, nvalid);
        __syncthreads();
#pragma unroll
        for (int k = 0; k < TPW; ++k) {
            const int tile = wave + 4 * k;
            if (tile < NT) {
                const int nt = tile / (P / 16), pt = tile % (P / 16);
#pragma unroll
                for (int kk = 0; kk < S::BLK; kk += MM::K) {
                    auto af = MM::load(&s_Bt[(nt * 16 + l16) * S::LDB + kk + MM::KPL * g]);
                    auto bf = MM::load(&s_Xt[(pt * 16 + l16) * S::LDB + kk + MM::KPL * g]);
                    acc[k] = MM::mma(af, bf, acc[k]);
                }
            }
        }
        __syncthreads();
    }

    float *M = a.M + (bh * a.nchunks + c) * (int64_t)(N * P);
#pragma unroll
    for (int k = 0; k < TPW; ++k) {
        const int tile = wave + 4 * k;
        if (tile < NT) {
            const int nt = tile / (P / 16), pt = tile % (P / 16);
#pragma unroll
            for (int v = 0; v < 4; ++v) M[(nt * 16 + 4 * g + v) * P + pt * 16 + l16] = acc[k][v];
        }
    }
    Acc *tot = static_cast<Acc *>(a.tot) + (bh * a.nchunks + c) * (S::NH + 1);
    if (tid == 0) tot[0] = cum_e;
    for (int i = tid; i < S::NH; i += kBlock) tot[1 + i] = s_psi[(nvalid - 1) * S::LDPSI + i];
}

// ---------------------------------------------------------------------------
// k_state_pass: for each slice and each row pair (i, i+N/2) x column p,
// walk the chunks: store S_in (transposed, io dtype) and advance
// S <- R(psi_e) (e^{cum_e} S + M).  Also writes final_state and the carry.
// Grid: (slices) x ceil(NH*P / 256).
// ---------------------------------------------------------------------------
template <typename T, int N, int P, int R, int Q>
__global__ __launch_bounds__(kBlock) void k_state_pass(ScanArgs a, int per_slice_blocks) {
    typedef Shape<T, N, P, R, Q> S;
    typedef typename S::Acc Acc;
    const int64_t bh = blockIdx.x / per_slice_blocks;
    const int sub = blockIdx.x % per_slice_blocks;
    const int64_t b = bh / a.H, h = bh % a.H;
    const int idx = sub * kBlock + threadIdx.x;

    // carry outputs: the last token's B and x (or the initial carry if L == 0)
    if (sub == 0) {
        T *cB = static_cast<T *>(a.cB) + bh * (R * N);
        T *cX = static_cast<T *>(a.cX) + bh * (R * P);
        if (a.L > 0) {
            const int64_t k = (b * a.L + a.L - 1) * a.H + h;
            const T *Bl = static_cast<const T *>(a.B) + k * (R * N);
            const T *Xl = static_cast<const T *>(a.x) + k * (R * P);
            for (int e = threadIdx.x; e < R * N; e += kBlock) cB[e] = Bl[e];
            for (int e = threadIdx.x; e < R * P; e += kBlock) cX[e] = Xl[e];
        } else {
            const T *iB = static_cast<const T *>(a.init_cB);
            const T *iX = static_cast<const T *>(a.init_cX);
            for (int e = threadIdx.x; e < R * N; e += kBlock)
                cB[e] = iB ? iB[bh * (R * N) + e] : from_f32<T>(0.f);
            for (int e = threadIdx.x; e < R * P; e += kBlock)
                cX[e] = iX ? iX[bh * (R * P) + e] : from_f32<T>(0.f);
        }
    }
    if (idx >= S::NH * P) return;
    const int i = idx / P, p = idx % P;

    float sre = 0.f, sim = 0.f;
    if (a.init_state) {
        const float *st = a.init_state + bh * (int64_t)(N * P);
        sre = st[i * P + p];
        sim = st[(i + S::NH) * P + p];
    }
    if (a.L > 0 && a.init_cB) {
        // previous-input term of token 0: (1 - lambda_0) dt_0 B_{-1} X_{-1}^T
        const int64_t k0 = (b * a.L) * a.H + h;
        const float wb = (1.f - a.lam[k0]) * a.dt[k0];
        const T *iB = static_cast<const T *>(a.init_cB) + bh * (R * N);
        const T *iX = static_cast<const T *>(a.init_cX) + bh * (R * P);
        float ure = 0.f, uim = 0.f;
        for (int r = 0; r < R; ++r) {
            const float xv = to_f32(iX[r * P + p]);
            ure += to_f32(iB[r * N + i]) * xv;
            uim += to_f32(iB[r * N + i + S::NH]) * xv;
        }
        sre += wb * ure;
        sim += wb * uim;
    }
    const float *M = a.M + bh * a.nchunks * (int64_t)(N * P);
    T *Sin = static_cast<T *>(a.Sin) + bh * a.nchunks * (int64_t)(N * P);
    const Acc *tot = static_cast<const Acc *>(a.tot) + bh * a.nchunks * (S::NH + 1);

    constexpr int DEPTH = 8;   // chunks whose inputs are loaded ahead
    for (int64_t c0 = 0; c0 < a.nchunks; c0 += DEPTH) {
        float mre[DEPTH], mim[DEPTH];
        Acc ce[DEPTH], ps[DEPTH];
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            const int64_t c = c0 + d;
            if (c < a.nchunks) {
                mre[d] = M[c * (N * P) + i * P + p];
                mim[d] = M[c * (N * P) + (i + S::NH) * P + p];
                ce[d] = tot[c * (S::NH + 1)];
                ps[d] = tot[c * (S::NH + 1) + 1 + i];
            }
        }
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            const int64_t c = c0 + d;
            if (c < a.nchunks) {
                Sin[c * (N * P) + p * N + i] = from_f32<T>(sre);
                Sin[c * (N * P) + p * N + i + S::NH] = from_f32<T>(sim);
                const Acc e = exp_acc(ce[d]);
                const Acc ure = e * (Acc)sre + (Acc)mre[d], uim = e * (Acc)sim + (Acc)mim[d];
                Acc sn, cs;
                sincos_acc(ps[d], &sn, &cs);
                sre = (float)(cs * ure - sn * uim);
                sim = (float)(sn * ure + cs * uim);
            }
        }
    }
    float *fs = a.final_state + bh * (int64_t)(N * P);
    fs[i * P + p] = sre;
    fs[(i + S::NH) * P + p] = sim;
}

// ---------------------------------------------------------------------------
// k_chunk_out: y for every token of a chunk.  Rows of the chunk are handled in
// groups of 64 (16 per wave); for each group the diagonal and earlier blocks
// of B^ and x are staged in LDS and contracted with MFMA:
//   acc  = e^{cum_t} C^_rows S_in                        (K = N)
//   G^T  = B^_blk C^_rows^T, masked by w_tj               (K = N)
//   acc += (w o G) x_blk                                   (K = 64 rows)
// Grid: one workgroup per (slice, chunk), slice-major.
// ---------------------------------------------------------------------------
template <typename T, int N, int P, int R, int Q>
__global__ __launch_bounds__(kBlock) void k_chunk_out(ScanArgs a) {
    typedef Shape<T, N, P, R, Q> S;
    typedef typename S::Acc Acc;
    typedef Mma<T> MM;
    __shared__ Acc s_cum[Q];
    __shared__ float s_gam[Q], s_sig[Q];
    __shared__ Acc s_psi[Q * S::LDPSI];
    __shared__ __attribute__((aligned(16))) T s_C[S::BLK * S::LDN];
    __shared__ __attribute__((aligned(16))) T s_B[S::BLK * S::LDN];
    __shared__ __attribute__((aligned(16))) T s_Xt[P * S::LDB];
    __shared__ __attribute__((aligned(16))) T s_S[P * S::LDN];

    const int64_t blk = blockIdx.x;
    const int64_t bh = blk / a.nchunks, c = blk % a.nchunks;
    const int64_t b = bh / a.H, h = bh % a.H;
    const int64_t t0 = c * Q;
    const int nvalid = (int)min((int64_t)Q, a.L - t0);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4, l16 = lane & 15;

    chunk_prologue<S>(a, b, h, t0, nvalid, s_cum, s_gam, s_sig, s_psi);

    // state entering the chunk, [P][N] in the io dtype
    const T *Sin = static_cast<const T *>(a.Sin) + (bh * a.nchunks + c) * (int64_t)(N * P);
    for (int e = tid; e < N * P; e += kBlock) {
        const int p = e / N, n = e % N;
        s_S[p * S::LDN + n] = Sin[e];
    }
    const float Dh = a.D[h];
    const int64_t tok_bc = ((b * a.L + t0) * a.H + h);
    const T *Csrc = static_cast<const T *>(a.C) + tok_bc * (R * N);
    const T *Bsrc = static_cast<const T *>(a.B) + tok_bc * (R * N);
    const T *Xsrc = static_cast<const T *>(a.x) + tok_bc * (R * P);
    T *Ydst = static_cast<T *>(a.y) + tok_bc * (R * P);
    const T *Zsrc = a.z ? static_cast<const T *>(a.z) + tok_bc * (R * P) : nullptr;   // output gate
    const int64_t bstride = a.H * R * N, xstride = a.H * R * P;
    constexpr int PT = P / 16;

    for (int rg = 0; rg < S::NBLK; ++rg) {
        stage_rot_rows<S, T>(s_C, Csrc, bstride, rg * S::BLK, nvalid, s_psi);
        __syncthreads();
        // inter-chunk term: e^{cum_t} C^_t . S_in
        f32x4 acc[PT];
#pragma unroll
        for (int pt = 0; pt < PT; ++pt) {
            acc[pt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kk = 0; kk < N; kk += MM::K) {
                auto af = MM::load(&s_C[(wave * 16 + l16) * S::LDN + kk + MM::KPL * g]);
                auto bf = MM::load(&s_S[(pt * 16 + l16) * S::LDN + kk + MM::KPL * g]);
                acc[pt] = MM::mma(af, bf, acc[pt]);
            }
        }
        const int trow_acc = rg * S::BLK + wave * 16 + 4 * g;   // + v
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const float e = (float)exp_acc(s_cum[(trow_acc + v) / R]);
#pragma unroll
            for (int pt = 0; pt < PT; ++pt) acc[pt][v] *= e;
        }
        // intra-chunk term over the blocks up to the diagonal
        const int tt = (rg * S::BLK + wave * 16 + l16) / R;      // this lane's G^T column token
        for (int jb = 0; jb <= rg; ++jb) {
            stage_rot_rows<S, T>(s_B, Bsrc, bstride, jb * S::BLK, nvalid, s_psi);
            stage_x_t<S, T>(s_Xt, Xsrc, xstride, jb * S::BLK, nvalid);
            __syncthreads();
            const int ntile = (jb < rg) ? 4 : wave + 1;          // j-tiles at or below the diagonal
            f32x4 gt[4];
#pragma unroll
            for (int jt = 0; jt < 4; ++jt) {
                gt[jt] = f32x4{0.f, 0.f, 0.f, 0.f};
                if (jt < ntile) {
#pragma unroll
                    for (int kk = 0; kk < N; kk += MM::K) {
                        auto af = MM::load(&s_B[(jt * 16 + l16) * S::LDN + kk + MM::KPL * g]);
                        auto bf = MM::load(&s_C[(wave * 16 + l16) * S::LDN + kk + MM::KPL * g]);
                        gt[jt] = MM::mma(af, bf, gt[jt]);
                    }
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const int tj = (jb * S::BLK + jt * 16 + 4 * g + v) / R;
                        float w = 0.f;
                        if (tj < tt) w = (float)exp_acc(s_cum[tt] - s_cum[tj]) * s_sig[tj];
                        else if (tj == tt) w = s_gam[tt];
                        gt[jt][v] *= w;
                    }
                }
            }
            if constexpr (MM::KPL == 8) {
                // K-step of 32 rows = j-tiles (2kk, 2kk+1); this lane holds rows
                // 4g..4g+3 of each, matched by the same rows of x.
#pragma unroll
                for (int kk = 0; kk < 2; ++kk) {
                    if (2 * kk < ntile) {
                        bf16x8 af;
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            af[v] = from_f32<bf16>(gt[2 * kk][v]);
                            af[4 + v] = from_f32<bf16>(gt[2 * kk + 1][v]);
                        }
#pragma unroll
                        for (int pt = 0; pt < PT; ++pt) {
                            const T *xr = &s_Xt[(pt * 16 + l16) * S::LDB + 32 * kk + 4 * g];
                            const bf16x4 lo = *reinterpret_cast<const bf16x4 *>(xr);
                            const bf16x4 hi = *reinterpret_cast<const bf16x4 *>(xr + 16);
                            bf16x8 bfr;
#pragma unroll
                            for (int v = 0; v < 4; ++v) { bfr[v] = lo[v]; bfr[4 + v] = hi[v]; }
                            acc[pt] = MM::mma(af, bfr, acc[pt]);
                        }
                    }
                }
            } else {
                // fp32: one K-step of 4 per accumulator value of a j-tile
#pragma unroll
                for (int jt = 0; jt < 4; ++jt) {
                    if (jt < ntile) {
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
#pragma unroll
                            for (int pt = 0; pt < PT; ++pt) {
                                const float xv = to_f32(s_Xt[(pt * 16 + l16) * S::LDB + jt * 16 + 4 * g + v]);
                                acc[pt] = MM::mma(gt[jt][v], xv, acc[pt]);
                            }
                        }
                    }
                }
            }
            __syncthreads();
        }
        // skip term and store (s_Xt still holds the diagonal block jb == rg)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int rl = wave * 16 + 4 * g + v;
            const int row = rg * S::BLK + rl, t = row / R, r = row % R;
            if (t < nvalid) {
#pragma unroll
                for (int pt = 0; pt < PT; ++pt) {
                    const int p = pt * 16 + l16;
                    float yv = acc[pt][v] + Dh * to_f32(s_Xt[p * S::LDB + rl]);
                    if (Zsrc) yv *= silu(to_f32(Zsrc[t * xstride + r * P + p]));
                    Ydst[t * xstride + r * P + p] = from_f32<T>(yv);
                }
            }
        }
        __syncthreads();
    }
}

template <typename T, int N, int P, int R, int Q>
hipError_t launch_scan(const ScanArgs &a, hipStream_t stream) {
    const int64_t BH = a.batch * a.H;
    constexpr int per = (N / 2 * P + kBlock - 1) / kBlock;
    if (a.nchunks > 0) {
        hipLaunchKernelGGL((k_chunk_state<T, N, P, R, Q>), dim3((unsigned)(BH * a.nchunks)),
                           dim3(kBlock), 0, stream, a);
    }
    hipLaunchKernelGGL((k_state_pass<T, N, P, R, Q>), dim3((unsigned)(BH * per)), dim3(kBlock), 0,
                       stream, a, per);
    if (a.nchunks > 0) {
        hipLaunchKernelGGL((k_chunk_out<T, N, P, R, Q>), dim3((unsigned)(BH * a.nchunks)),
                           dim3(kBlock), 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace

// Instantiated shapes: (io, N, P, R, Q).  io 0 = fp32, 1 = bf16.
#define M3_SCAN_SHAPES(X)          \
    X(0, float, 16, 16, 1, 64)     \
    X(0, float, 16, 16, 2, 32)     \
    X(0, float, 16, 16, 2, 64)     \
    X(0, float, 16, 16, 4, 16)     \
    X(0, float, 16, 16, 4, 32)     \
    X(0, float, 16, 16, 4, 64)     \
    X(0, float, 128, 64, 2, 32)    \
    X(0, float, 128, 64, 4, 16)    \
    X(0, float, 128, 64, 4, 32)    \
    X(1, bf16, 32, 64, 1, 64)      \
    X(1, bf16, 32, 64, 2, 32)      \
    X(1, bf16, 32, 64, 4, 16)      \
    X(1, bf16, 64, 64, 1, 64)      \
    X(1, bf16, 64, 64, 1, 128)     \
    X(1, bf16, 64, 64, 2, 32)      \
    X(1, bf16, 64, 64, 2, 64)      \
    X(1, bf16, 64, 64, 4, 16)      \
    X(1, bf16, 64, 64, 4, 32)      \
    X(1, bf16, 128, 64, 1, 64)     \
    X(1, bf16, 128, 64, 1, 128)    \
    X(1, bf16, 128, 64, 2, 32)     \
    X(1, bf16, 128, 64, 2, 64)     \
    X(1, bf16, 128, 64, 2, 128)    \
    X(1, bf16, 128, 64, 4, 32)     \
    X(1, bf16, 128, 64, 4, 64)     \
    X(1, bf16, 128, 64, 4, 128)

ScanImpl find_scan_impl(int io, int64_t N, int64_t P, int64_t R, int64_t Q) {
#define M3_CASE(IO, T, N_, P_, R_, Q_)                                      \
    if (io == IO && N == N_ && P == P_ && R == R_ && Q == Q_)               \
        return ScanImpl{&launch_scan<T, N_, P_, R_, Q_>, (int)sizeof(typename AccOf<T>::type), false, nullptr};
    M3_SCAN_SHAPES(M3_CASE)
#undef M3_CASE
    return ScanImpl{nullptr, 0, false, nullptr};
}

}  // namespace m3
