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

template <typename T, int N, int P, int R>
__global__ __launch_bounds__(kBlock) void k_step(StepArgs a) {
    constexpr int NH = N / 2;
    constexpr int TX = P / 4;                   // threads across columns (float4 each)
    constexpr int TY = kBlock / TX;             // thread rows
    constexpr int NPT = (NH + TY - 1) / TY;     // row pairs per thread
    constexpr int NW = kBlock / kWave;
    static_assert(P % 4 == 0 && kBlock % TX == 0 && kWave % TX == 0, "column split");

    __shared__ float s_B[R * N], s_Bp[R * N], s_C[R * N];
    __shared__ float s_X[R * P], s_Xp[R * P];
    __shared__ float s_cs[NH], s_sn[NH];
    __shared__ float s_red[NW * R * P];

    const int64_t bh = blockIdx.x;
    const int64_t b = bh / a.H, h = bh % a.H;
    const int tid = threadIdx.x, tx = tid % TX, ty = tid / TX;
    const int lane = tid & (kWave - 1), wave = tid / kWave;

    // 1. issue the state loads first: they are the bytes that matter
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
    // 2. per-slice vectors into LDS (fp32)
    const T *Bt = static_cast<const T *>(a.B) + bh * (R * N);
    const T *Ct = static_cast<const T *>(a.C) + bh * (R * N);
    const T *Xt = static_cast<const T *>(a.x) + bh * (R * P);
    T *cB = static_cast<T *>(a.cB) + bh * (R * N);
    T *cX = static_cast<T *>(a.cX) + bh * (R * P);
    for (int e = tid; e < R * N; e += kBlock) {
        s_B[e] = to_f32(Bt[e]);
        s_C[e] = to_f32(Ct[e]);
        s_Bp[e] = to_f32(cB[e]);
    }
    for (int e = tid; e < R * P; e += kBlock) {
        s_X[e] = to_f32(Xt[e]);
        s_Xp[e] = to_f32(cX[e]);
    }
    const float *th = a.theta + bh * NH;
    for (int i = tid; i < NH; i += kBlock) {
        float sn, cs;
        sincosf(th[i], &sn, &cs);
        s_cs[i] = cs;
        s_sn[i] = sn;
    }
    const float dtv = a.dt[bh], lamv = a.lam[bh];
    const float alpha = expf(dtv * a.A[b * a.a_sb + h * a.a_sh]);
    const float bprev = (1.f - lamv) * dtv, gam = lamv * dtv;
    __syncthreads();
    // 3. the carry becomes (B_t, X_t)
    for (int e = tid; e < R * N; e += kBlock) cB[e] = Bt[e];
    for (int e = tid; e < R * P; e += kBlock) cX[e] = Xt[e];

    // 4. update the owned state elements and accumulate Y partials
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
#pragma unroll
    for (int k = 0; k < NPT; ++k) {
        const int i = ty + TY * k;
        if (i < NH) {
            const float cs = s_cs[i], sn = s_sn[i];
            float hr[4] = {re[k].x, re[k].y, re[k].z, re[k].w};
            float hi[4] = {im[k].x, im[k].y, im[k].z, im[k].w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                float ur = hr[q], ui = hi[q], vr = 0.f, vi = 0.f;
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    ur += bprev * s_Bp[r * N + i] * xp[r][q];
                    ui += bprev * s_Bp[r * N + i + NH] * xp[r][q];
                    vr += s_B[r * N + i] * xc[r][q];
                    vi += s_B[r * N + i + NH] * xc[r][q];
                }
                hr[q] = alpha * (cs * ur - sn * ui) + gam * vr;
                hi[q] = alpha * (sn * ur + cs * ui) + gam * vi;
#pragma unroll
                for (int r = 0; r < R; ++r)
                    yp[r][q] += hr[q] * s_C[r * N + i] + hi[q] * s_C[r * N + i + NH];
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
    const float Dh = a.D[h];
    for (int e = tid; e < R * P; e += kBlock) {
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < NW; ++w) v += s_red[w * R * P + e];
        yt[e] = from_f32<T>(v + Dh * s_X[e]);
    }
}

template <typename T, int N, int P, int R>
hipError_t launch_step(const StepArgs &a, hipStream_t stream) {
    hipLaunchKernelGGL((k_step<T, N, P, R>), dim3((unsigned)(a.batch * a.H)), dim3(kBlock), 0,
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

}  // namespace m3
