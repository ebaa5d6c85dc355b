// Single-token decode step of the Mamba-3 SSM on gfx950 (one iteration of
// the exponential-trapezoidal recurrence with the rotating complex state and
// MIMO rank R; Sec. 3.1 Prop. "Exponential-Trapezoidal Discretization",
// Sec. 3.2 eq. trap-real-rot, Sec. 3.3):
//     G  = h + beta'_t B_{t-1} X_{t-1}^T,    beta'_t = (1 - lambda_t) dt_t
//     h' = alpha_t R_t G + gamma_t B_t X_t^T
//     Y  = h'^T C_t + D X_t
// The step reads and writes the N x P fp32 state once; everything else is a
// few KB per (batch, head), so the kernel streams the state: each thread owns
// float4 column groups of the row pairs (i, i+N/2) that R_t couples, keeps
// them in registers across the update and the output reduction, and writes
// them back in place.  The rank-R outer products (MIMO raises their cost R
// times, Sec. 3.3 "Decoding Arithmetic Intensity") run on the VALU from
// LDS-broadcast vectors.
#include "m3_device.h"
#include "m3_internal.h"

namespace m3 {
namespace {

// 16-byte piece of the io dtype
template <typename T> struct Vec8;
template <> struct Vec8<bf16> { typedef bf16x8 type; static constexpr int n = 8; };
template <> struct Vec8<float> { typedef f32x4 type; static constexpr int n = 4; };

// kPro: the block prologue on the step's inputs (B_t and C_t: RMS norm over
// N, gain, bias; x_t and z_t: X = W_X o X', Z = W_Z o Z'); the new carry
// holds the B_t and X_t that the recurrence used.
template <typename T, int N, int P, int R, int NT, bool kGate, bool kPro>
__global__ __launch_bounds__(NT) void k_step(StepArgs a) {
    constexpr int NH = N / 2;
    constexpr int TX = P / 4;                   // threads across columns (float4 each)
    constexpr int TY = NT / TX;                 // thread rows
    constexpr int NPT = (NH + TY - 1) / TY;     // row pairs per thread
    constexpr int NW = NT / kWave;
    static_assert(P % 4 == 0 && NT % TX == 0 && kWave % TX == 0 && NT % kWave == 0, "column split");
    static_assert(NH <= NT, "one thread per rotation angle");

    // Per-slice vectors in LDS (fp32), rank innermost so that one 16-byte read
    // fetches all ranks of a state row; the step's scalars are folded in:
    // s_Bp = beta' B_{t-1}, s_B = gamma B_t, s_cs = alpha (cos, sin).
    constexpr int RV = R == 1 ? 1 : (R == 2 ? 2 : 4);   // ranks per vector read
    static_assert(R % RV == 0, "rank vectors");
    __shared__ __attribute__((aligned(16))) float s_B[N * R], s_Bp[N * R], s_C[N * R];
    __shared__ float s_X[R * P], s_Xp[R * P];
    __shared__ float s_cs[NH], s_sn[NH];
    __shared__ float s_red[NW * R * P];

    const int64_t bh = blockIdx.x;
    const int64_t b = bh / a.H, h = bh % a.H;
    const int tid = threadIdx.x, tx = tid % TX, ty = tid / TX;
    const int lane = tid & (kWave - 1), wave = tid / kWave;

    // per-slice vectors into LDS
    const T *Bt = static_cast<const T *>(a.B) + bh * (R * N);
    const T *Ct = static_cast<const T *>(a.C) + bh * (R * N);
    const bool sx = kPro && a.pro.wx != nullptr, sz = kPro && a.pro.wz != nullptr;
    const T *Xt = static_cast<const T *>(a.x) + bh * (sx ? P : R * P);
    T *cB = static_cast<T *>(a.cB) + bh * (R * N);
    T *cX = static_cast<T *>(a.cX) + bh * (R * P);
    const float dtv = a.dt[bh], lamv = a.lam[bh], Av = a.A[b * a.a_sb + h * a.a_sh];
    const float Dh = a.D[h];   // (loaded with the step's scalars: used only by the last stage)
    // B_t, C_t, the carry and X in 16-byte pieces; the loaded B_t and X_t
    // pieces are also the new carry (written after the barrier below)
    typedef typename Vec8<T>::type V8;
    constexpr int VE = Vec8<T>::n;                      // elements per piece
    constexpr int PB = R * N / VE, PX = R * P / VE;     // pieces per vector
    constexpr int TPB = (PB + NT - 1) / NT, TPX = (PX + NT - 1) / NT;
    // The small per-slice loads go out before the state loads (memory
    // counters retire in order), so their LDS staging overlaps the state's
    // flight time.
    V8 vb[TPB], vc[TPB], vbp[TPB], vx[TPX], vxp[TPX];
#pragma unroll
    for (int k = 0; k < TPB; ++k) {
        const int pc = min(tid + k * NT, PB - 1);
        vb[k] = *reinterpret_cast<const V8 *>(Bt + pc * VE);
        vc[k] = *reinterpret_cast<const V8 *>(Ct + pc * VE);
        vbp[k] = *reinterpret_cast<const V8 *>(cB + pc * VE);
    }
#pragma unroll
    for (int k = 0; k < TPX; ++k) {
        const int pc = min(tid + k * NT, PX - 1);
        // (structured input: piece pc of rank row r reads X' at its column)
        vx[k] = *reinterpret_cast<const V8 *>(Xt + (sx ? (pc * VE) % P : pc * VE));
        vxp[k] = *reinterpret_cast<const V8 *>(cX + pc * VE);
    }
    // per-step angles, or dt * omega with the head's frequencies omega
    const float *th = a.theta_ph ? a.theta + h * NH : a.theta + bh * NH;
    const float thv = th[min(tid, NH - 1)] * (a.theta_ph ? dtv : 1.f);
    // gate inputs of this thread's outputs (y_t o SiLU(z_t))
    constexpr int TZ = (R * P + NT - 1) / NT;
    float zv[TZ];
    if constexpr (kGate) {
        if (sz) {   // structured gate input: Z = W_Z o Z' (Z' [batch][nheads][headdim])
            const T *Zp = static_cast<const T *>(a.z) + bh * P;
#pragma unroll
            for (int k = 0; k < TZ; ++k) {
                const int e = min(tid + k * NT, R * P - 1);
                zv[k] = to_f32(Zp[e % P]) * a.pro.wz[h * (R * P) + e];
            }
        } else {
            const T *Zt = static_cast<const T *>(a.z) + bh * (R * P);
#pragma unroll
            for (int k = 0; k < TZ; ++k) zv[k] = to_f32(Zt[min(tid + k * NT, R * P - 1)]);
        }
    }
    // 1. the state: the bytes that matter
    float *st = a.state + bh * (int64_t)(N * P);
    float4 re[NPT], im[NPT];
#pragma unroll
    for (int k = 0; k < NPT; ++k) {
        const int i = ty + TY * k;
        if (i < NH) {
            re[k] = *reinterpret_cast<const float4 *>(&st[i * P + 4 * tx]);
            im[k] = *reinterpret_cast<const float4 *>(&st[(i + NH) * P + 4 * tx]);
        }
    }
    const float alpha = (float)exp_fast((typename AccOf<T>::type)dtv * Av);
    const float bprev = (1.f - lamv) * dtv, gam = lamv * dtv;
    if constexpr (kPro) {
        // B_t, C_t: a rank row's N / VE pieces are consecutive threads of one
        // wave, so its sum of squares is a lane sum; then gain and bias
        static_assert(kWave % (N / VE) == 0 && PB <= NT, "a row's pieces in one wave");
        const int pc = min(tid, PB - 1), r = (pc * VE) / N, n0 = (pc * VE) % N;
        float sb = 0.f, sc = 0.f;
#pragma unroll
        for (int e = 0; e < VE; ++e) {
            sb += to_f32(vb[0][e]) * to_f32(vb[0][e]);
            sc += to_f32(vc[0][e]) * to_f32(vc[0][e]);
        }
#pragma unroll
        for (int o = 1; o < N / VE; o <<= 1) {
            sb += __shfl_xor(sb, o, kWave);
            sc += __shfl_xor(sc, o, kWave);
        }
        const float kb = a.pro.bcnorm ? rsqrtf(sb * (1.f / N) + a.pro.eps) : 1.f;
        const float kc = a.pro.bcnorm ? rsqrtf(sc * (1.f / N) + a.pro.eps) : 1.f;
        const int64_t hb = h * (R * N) + r * N + n0;
#pragma unroll
        for (int e = 0; e < VE; ++e) {
            const float gb = a.pro.gB ? a.pro.gB[hb + e] : 1.f, bb = a.pro.bB ? a.pro.bB[hb + e] : 0.f;
            const float gc = a.pro.gC ? a.pro.gC[hb + e] : 1.f, bc = a.pro.bC ? a.pro.bC[hb + e] : 0.f;
            vb[0][e] = from_f32<T>(kb * gb * to_f32(vb[0][e]) + bb);
            vc[0][e] = from_f32<T>(kc * gc * to_f32(vc[0][e]) + bc);
        }
        if (sx) {   // X = W_X o X' (rounded to the io dtype, as a stored x would be)
#pragma unroll
            for (int k = 0; k < TPX; ++k) {
                const int px = min(tid + k * NT, PX - 1);
#pragma unroll
                for (int e = 0; e < VE; ++e)
                    vx[k][e] = from_f32<T>(to_f32(vx[k][e]) * a.pro.wx[h * (R * P) + px * VE + e]);
            }
        }
    }
#pragma unroll
    for (int k = 0; k < TPB; ++k) {
        const int pc = tid + k * NT;
        if (pc < PB) {
#pragma unroll
            for (int e = 0; e < VE; ++e) {   // element pc*VE + e = r*N + n  ->  [n][r]
                const int r = (pc * VE + e) / N, n = (pc * VE + e) % N;
                s_B[n * R + r] = gam * to_f32(vb[k][e]);
                s_C[n * R + r] = to_f32(vc[k][e]);
                s_Bp[n * R + r] = bprev * to_f32(vbp[k][e]);
            }
        }
    }
#pragma unroll
    for (int k = 0; k < TPX; ++k) {
        const int pc = tid + k * NT;
        if (pc < PX) {
#pragma unroll
            for (int e = 0; e < VE; ++e) {
                s_X[pc * VE + e] = to_f32(vx[k][e]);
                s_Xp[pc * VE + e] = to_f32(vxp[k][e]);
            }
        }
    }
    if (tid < NH) {
        typename AccOf<T>::type sn, cs;   // hardware sin/cos for the bf16 build, accurate for fp32
        sincos_fast((typename AccOf<T>::type)thv, &sn, &cs);
        s_cs[tid] = alpha * (float)cs;
        s_sn[tid] = alpha * (float)sn;
    }
    __syncthreads();
    // 3. the carry becomes (B_t, X_t)
#pragma unroll
    for (int k = 0; k < TPB; ++k)
        if (tid + k * NT < PB) *reinterpret_cast<V8 *>(cB + (tid + k * NT) * VE) = vb[k];
#pragma unroll
    for (int k = 0; k < TPX; ++k)
        if (tid + k * NT < PX) *reinterpret_cast<V8 *>(cX + (tid + k * NT) * VE) = vx[k];

    // 4. update the owned state elements and accumulate Y partials:
    //    u = h + beta' B_{t-1} X_{t-1}^T,  h' = alpha R(theta) u + gamma B_t X_t^T
    float yp[R][4];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int q = 0; q < 4; ++q) yp[r][q] = 0.f;
    float xp[R][4], xc[R][4];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            xp[r][q] = s_Xp[r * P + 4 * tx + q];
            xc[r][q] = s_X[r * P + 4 * tx + q];
        }
    auto rank_vec = [&](const float *base, float (&v)[R]) {
#pragma unroll
        for (int r0 = 0; r0 < R; r0 += RV) {
            if constexpr (RV == 4) {
                const float4 t = *reinterpret_cast<const float4 *>(base + r0);
                v[r0] = t.x; v[r0 + 1] = t.y; v[r0 + 2] = t.z; v[r0 + 3] = t.w;
            } else if constexpr (RV == 2) {
                const float2 t = *reinterpret_cast<const float2 *>(base + r0);
                v[r0] = t.x; v[r0 + 1] = t.y;
            } else {
                v[r0] = base[r0];
            }
        }
    };
#pragma unroll
    for (int k = 0; k < NPT; ++k) {
        const int i = ty + TY * k;
        if (i < NH) {
            const float cs = s_cs[i], sn = s_sn[i];
            float bp0[R], bp1[R], bc0[R], bc1[R], c0[R], c1[R];
            rank_vec(&s_Bp[i * R], bp0);
            rank_vec(&s_Bp[(i + NH) * R], bp1);
            rank_vec(&s_B[i * R], bc0);
            rank_vec(&s_B[(i + NH) * R], bc1);
            rank_vec(&s_C[i * R], c0);
            rank_vec(&s_C[(i + NH) * R], c1);
            float hr[4] = {re[k].x, re[k].y, re[k].z, re[k].w};
            float hi[4] = {im[k].x, im[k].y, im[k].z, im[k].w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                float ur = hr[q], ui = hi[q], vr = 0.f, vi = 0.f;
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    ur = fmaf(bp0[r], xp[r][q], ur);
                    ui = fmaf(bp1[r], xp[r][q], ui);
                    vr = fmaf(bc0[r], xc[r][q], vr);
                    vi = fmaf(bc1[r], xc[r][q], vi);
                }
                hr[q] = fmaf(cs, ur, fmaf(-sn, ui, vr));
                hi[q] = fmaf(sn, ur, fmaf(cs, ui, vi));
#pragma unroll
                for (int r = 0; r < R; ++r) yp[r][q] = fmaf(hr[q], c0[r], fmaf(hi[q], c1[r], yp[r][q]));
            }
            *reinterpret_cast<float4 *>(&st[i * P + 4 * tx]) = make_float4(hr[0], hr[1], hr[2], hr[3]);
            *reinterpret_cast<float4 *>(&st[(i + NH) * P + 4 * tx]) = make_float4(hi[0], hi[1], hi[2], hi[3]);
        }
    }
    // 5. reduce the partials over the thread rows: inside the wave, then across waves
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            float v = yp[r][q];
#pragma unroll
            for (int o = TX; o < kWave; o <<= 1) v += __shfl_xor(v, o, kWave);
            yp[r][q] = v;
        }
    if (lane < TX) {
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int q = 0; q < 4; ++q) s_red[(wave * R + r) * P + 4 * tx + q] = yp[r][q];
    }
    __syncthreads();
    T *yt = static_cast<T *>(a.y) + bh * (R * P);
#pragma unroll
    for (int k = 0; k < TZ; ++k) {
        const int e = tid + k * NT, ec = min(e, R * P - 1);
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w) v += s_red[w * R * P + ec];
        v += Dh * s_X[ec];
        if constexpr (kPro) {
            // output norm (optional) on y as stored (io dtype): a group's
            // channels are consecutive lanes of one wave (R P is a multiple
            // of the wave, so lanes past the outputs fill whole waves)
            static_assert((R * P) % kWave == 0, "whole waves of outputs");
            const float gz = kGate ? silu(zv[k]) : 1.f;
            if (a.pro.onorm) {
                const bool post = a.pro.onorm == 2;
                v = to_f32(from_f32<T>(v));
                if (post) v *= gz;
                float ss = v * v;
                for (int o = 1; o < a.pro.ogroup; o <<= 1) ss += __shfl_xor(ss, o, kWave);
                v *= rsqrtf(ss / (float)a.pro.ogroup + a.pro.oeps) * (a.pro.og ? a.pro.og[h * (R * P) + ec] : 1.f);
                if (!post) v *= gz;
            } else {
                v *= gz;
            }
        } else if constexpr (kGate) {
            v *= silu(zv[k]);
        }
        if (e < R * P) yt[e] = from_f32<T>(v);
    }
}

// Threads per (batch, head): four row pairs per thread (four waves for the
// 128 x 64 state; fewer threads per slice measured slower there: longer
// per-thread update chains), at least one wave.
template <int N, int P> struct StepThreads {
    static constexpr int v = (N / 8) * (P / 4);
    static constexpr int value = v < 64 ? 64 : v;
};

template <typename T, int N, int P, int R, bool kPro = false>
hipError_t launch_step(const StepArgs &a, hipStream_t stream) {
    constexpr int NT = StepThreads<N, P>::value;
    if (a.z)
        hipLaunchKernelGGL((k_step<T, N, P, R, NT, true, kPro>), dim3((unsigned)(a.batch * a.H)), dim3(NT), 0,
                           stream, a);
    else
        hipLaunchKernelGGL((k_step<T, N, P, R, NT, false, kPro>), dim3((unsigned)(a.batch * a.H)), dim3(NT), 0,
                           stream, a);
    return hipGetLastError();
}

}  // namespace

#define M3_STEP_SHAPES(X)      \
    X(0, float, 16, 16, 1)     \
    X(0, float, 16, 16, 2)     \
    X(0, float, 16, 16, 4)     \
    X(0, float, 128, 64, 1)    \
    X(0, float, 128, 64, 2)    \
    X(0, float, 128, 64, 4)    \
    X(1, bf16, 32, 64, 1)      \
    X(1, bf16, 32, 64, 2)      \
    X(1, bf16, 32, 64, 4)      \
    X(1, bf16, 64, 64, 1)      \
    X(1, bf16, 64, 64, 2)      \
    X(1, bf16, 64, 64, 4)      \
    X(1, bf16, 128, 64, 1)     \
    X(1, bf16, 128, 64, 2)     \
    X(1, bf16, 128, 64, 4)

step_launch_fn find_step_impl(int io, int64_t N, int64_t P, int64_t R) {
#define M3_CASE(IO, T, N_, P_, R_) \
    if (io == IO && N == N_ && P == P_ && R == R_) return &launch_step<T, N_, P_, R_>;
    M3_STEP_SHAPES(M3_CASE)
#undef M3_CASE
    return nullptr;
}

// The block prologue is built into the bf16 step kernels.
step_launch_fn find_step_pro_impl(int io, int64_t N, int64_t P, int64_t R) {
    if (io != 1 || N != 128 || P != 64) return nullptr;
    if (R == 1) return &launch_step<bf16, 128, 64, 1, true>;
    if (R == 2) return &launch_step<bf16, 128, 64, 2, true>;
    if (R == 4) return &launch_step<bf16, 128, 64, 4, true>;
    return nullptr;
}

}  // namespace m3
