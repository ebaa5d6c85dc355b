// Pieces shared by the single-pass prefill kernels (one chunk per workgroup,
// and G chunks per workgroup): shape traits of the N = 128, P = 64 tiling,
// element helpers, coherent accesses of the look-back, the control block.
#pragma once
#include <type_traits>

#include "m3_device.h"
#include "m3_internal.h"

namespace m3 {
namespace scan {

constexpr uint32_t kFlagAgg = 1, kFlagInc = 2;

struct alignas(4) h2 { _Float16 c, s; };
template <typename T> struct CsOf { typedef h2 type; };          // bf16 path: fp16 cos/sin
template <> struct CsOf<float> { typedef float2 type; };         // fp32 path: fp32 cos/sin
__device__ __forceinline__ void cs_put(h2 *p, float c, float s) { *p = h2{(_Float16)c, (_Float16)s}; }
__device__ __forceinline__ void cs_put(float2 *p, float c, float s) { *p = make_float2(c, s); }
__device__ __forceinline__ void cs_get(const h2 &v, float &c, float &s) { c = (float)v.c; s = (float)v.s; }
__device__ __forceinline__ void cs_get(const float2 &v, float &c, float &s) { c = v.x; s = v.y; }
// K consecutive (cos, sin) entries of a row of the table (16-byte LDS reads
// when K fills them; p is then 16-byte aligned)
struct alignas(16) h2x4 { h2 v[4]; };
struct alignas(16) f2x2 { float2 v[2]; };
template <int K>
__device__ __forceinline__ void cs_getn(const h2 *p, float (&c)[K], float (&s)[K]) {
    if constexpr (K % 4 == 0) {
#pragma unroll
        for (int q = 0; q < K / 4; ++q) {
            const h2x4 w = *reinterpret_cast<const h2x4 *>(p + 4 * q);
#pragma unroll
            for (int j = 0; j < 4; ++j) cs_get(w.v[j], c[4 * q + j], s[4 * q + j]);
        }
    } else {
#pragma unroll
        for (int j = 0; j < K; ++j) cs_get(p[j], c[j], s[j]);
    }
}
template <int K>
__device__ __forceinline__ void cs_getn(const float2 *p, float (&c)[K], float (&s)[K]) {
    if constexpr (K % 2 == 0) {
#pragma unroll
        for (int q = 0; q < K / 2; ++q) {
            const f2x2 w = *reinterpret_cast<const f2x2 *>(p + 2 * q);
#pragma unroll
            for (int j = 0; j < 2; ++j) cs_get(w.v[j], c[2 * q + j], s[2 * q + j]);
        }
    } else {
#pragma unroll
        for (int j = 0; j < K; ++j) cs_get(p[j], c[j], s[j]);
    }
}
// K consecutive entries written from registers (16-byte LDS writes)
template <int K>
__device__ __forceinline__ void cs_putn(h2 *p, const float (&c)[K], const float (&s)[K]) {
    static_assert(K % 4 == 0, "16-byte pieces");
#pragma unroll
    for (int q = 0; q < K / 4; ++q) {
        h2x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j) w.v[j] = h2{(_Float16)c[4 * q + j], (_Float16)s[4 * q + j]};
        *reinterpret_cast<h2x4 *>(p + 4 * q) = w;
    }
}
template <int K>
__device__ __forceinline__ void cs_putn(float2 *p, const float (&c)[K], const float (&s)[K]) {
    static_assert(K % 2 == 0, "16-byte pieces");
#pragma unroll
    for (int q = 0; q < K / 2; ++q) {
        f2x2 w;
#pragma unroll
        for (int j = 0; j < 2; ++j) w.v[j] = make_float2(c[2 * q + j], s[2 * q + j]);
        *reinterpret_cast<f2x2 *>(p + 2 * q) = w;
    }
}

template <typename T> struct Vec16;            // 16-byte vector of T
template <> struct Vec16<bf16> { typedef bf16x8 type; static constexpr int n = 8; };
template <> struct Vec16<float> { typedef f32x4 type; static constexpr int n = 4; };

__device__ __forceinline__ float fget(const bf16x8 &v, int e) { return (float)v[e]; }
__device__ __forceinline__ void fset(bf16x8 &v, int e, float x) { v[e] = (bf16)x; }
__device__ __forceinline__ float fget(const float &v, int) { return v; }
__device__ __forceinline__ void fset(float &v, int, float x) { v = x; }
__device__ __forceinline__ float fget(const f32x4 &v, int e) { return v[e]; }
__device__ __forceinline__ void fset(f32x4 &v, int e, float x) { v[e] = x; }

// Sum of squares of a 16-byte vector, accumulated in fp32 straight from the
// packed elements (v_dot2_f32_bf16 for bf16: no unpacked copy of the
// vector is formed, so nothing extra stays live until the values are used).
__device__ __forceinline__ float sumsq(const bf16x8 &v) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const bf16x2 p = {v[2 * q], v[2 * q + 1]};
        s = __builtin_amdgcn_fdot2_f32_bf16(p, p, s, false);
    }
    return s;
}
__device__ __forceinline__ float sumsq(const f32x4 &v) {
    return v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
}
__device__ __forceinline__ float sumsq(float v) { return v * v; }   // (fp32 MFMA fragments)

// Look-back traffic uses device-scope atomic accesses only (the sc1 scope
// bit): they are coherent across the XCDs' L2 caches by themselves, so no
// cache-wide write-back or invalidate is needed.  A publisher waits until its
// stores are acknowledged (vmcnt(0)) before the flag store; a reader issues
// its data loads only after it has seen the flag.
// Raw buffer resource (stride 0) over `bytes` bytes from `base`: a load at
// an offset at or past `bytes` returns zeros, so rows past the end of a
// sequence read as zero without address clamping or masks, and addresses are
// a scalar base plus a 32-bit per-lane offset.
typedef __amdgpu_buffer_rsrc_t Rsrc;
__device__ __forceinline__ Rsrc make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}
template <typename V> __device__ __forceinline__ V buf_load(Rsrc r, uint32_t off) {
    if constexpr (sizeof(V) == 16) {
        typedef int i32x4 __attribute__((ext_vector_type(4)));
        return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
    } else {
        static_assert(sizeof(V) == 4, "16- or 4-byte loads");
        return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0));
    }
}
// Offset of token t at a per-token stride below 2^24 bytes (full-rate 24-bit
// multiply; the library routes larger strides to the three-kernel path).
__device__ __forceinline__ uint32_t tok_off(int t, uint32_t stride_bytes) {
    return __umul24((uint32_t)t, stride_bytes);
}

// Inclusive prefix sum over the 64 lanes of a wavefront.  fp32: six DPP
// adds on the VALU (row shifts by 1, 2, 4, 8 within each 16-lane row, then
// the last lane of a row broadcast into the next rows); fp64 (the fp32
// build's prologue): lane shuffles.
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_src(float v) {
    // lanes with no source in the pattern, or outside ROWS, read 0
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROWS, 0xf, false));
}
__device__ __forceinline__ float lane_scan(float v) {
    v += dpp_src<0x111, 0xf>(v);   // row_shr:1
    v += dpp_src<0x112, 0xf>(v);   // row_shr:2
    v += dpp_src<0x114, 0xf>(v);   // row_shr:4
    v += dpp_src<0x118, 0xf>(v);   // row_shr:8
    v += dpp_src<0x142, 0xa>(v);   // row_bcast:15 into rows 1 and 3
    v += dpp_src<0x143, 0xc>(v);   // row_bcast:31 into rows 2 and 3
    return v;
}
__device__ __forceinline__ double lane_scan(double v) { return wave_incl_scan(v, (int)(threadIdx.x % kWave)); }
// Value of lane l (uniform l) in every lane.
__device__ __forceinline__ float lane_bcast(float v, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ __forceinline__ double lane_bcast(double v, int l) {
    const long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_readlane((int)(b & 0xffffffff), l), hi = __builtin_amdgcn_readlane((int)(b >> 32), l);
    return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

// LDS transposing read (gfx950 ds_read_b64_tr_b16) of a 4 x 16 bf16 block of
// a row-major LDS array: lane s of each 16-lane group addresses row s / 4,
// columns 4 (s % 4) .. +3 of the block (here `p`), and lane i of the group
// receives the block's column i, rows 0 .. 3.
__device__ __forceinline__ bf16x4 lds_tr4(const bf16 *p) {
    typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
    return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(p));
}

// MFMA operand whose K axis runs down the rows of a row-major LDS block M
// (leading dimension ld): lane (g, l16) receives M[r0 + k][c0 + l16] for its
// K elements k — 8g .. 8g+7 (bf16: two transposing reads) or g (fp32).
__device__ __forceinline__ bf16x8 load_kt(const bf16 *M, int ld, int r0, int c0, int g, int l16) {
    const bf16 *p0 = M + (r0 + 8 * g + l16 / 4) * ld + c0 + 4 * (l16 % 4);
    const bf16x4 lo = lds_tr4(p0), hi = lds_tr4(p0 + 4 * ld);
    bf16x8 fr;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        fr[v] = lo[v];
        fr[4 + v] = hi[v];
    }
    return fr;
}
__device__ __forceinline__ float load_kt(const float *M, int ld, int r0, int c0, int g, int l16) {
    return M[(r0 + g) * ld + c0 + l16];
}

// Four consecutive output columns of one row, held by one lane of a
// transposed MFMA tile (the lane's four accumulator rows are y columns).
__device__ __forceinline__ void store4(bf16 *dst, const f32x4 &v) {
    bf16x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = (bf16)v[e];
    *reinterpret_cast<bf16x4 *>(dst) = o;
}
__device__ __forceinline__ void store4(float *dst, const f32x4 &v) { *reinterpret_cast<f32x4 *>(dst) = v; }

// Output gate on one 16-byte piece of y: y o SiLU(z), elementwise in fp32.
template <typename T>
__device__ __forceinline__ typename Vec16<T>::type gate_piece(typename Vec16<T>::type y,
                                                            const typename Vec16<T>::type &z) {
#pragma unroll
    for (int e = 0; e < Vec16<T>::n; ++e) fset(y, e, fget(y, e) * silu(fget(z, e)));
    return y;
}

// One step of the state recurrence on a lane's owned pair (re, im) of state
// rows: S <- e^{cum} R(psi) S + A (de = e^{cum}, (cs, sn) of psi), every
// rounding explicit (no contraction), so that a look-back folding a
// predecessor's published map and the map's owner compute the same bits.
__device__ __forceinline__ void state_step(float &re, float &im, float de, float cs, float sn,
                                           float are, float aim) {
    const float r = __fmul_rn(de, __fsub_rn(__fmul_rn(cs, re), __fmul_rn(sn, im)));
    const float i = __fmul_rn(de, __fadd_rn(__fmul_rn(sn, re), __fmul_rn(cs, im)));
    re = __fadd_rn(r, are);
    im = __fadd_rn(i, aim);
}
__device__ __forceinline__ void state_step(float &re, float &im, double de, double cs, double sn,
                                           float are, float aim) {
    const double r = __dmul_rn(de, __dsub_rn(__dmul_rn(cs, (double)re), __dmul_rn(sn, (double)im)));
    const double i = __dmul_rn(de, __dadd_rn(__dmul_rn(sn, (double)re), __dmul_rn(cs, (double)im)));
    re = __fadd_rn((float)r, are);
    im = __fadd_rn((float)i, aim);
}

__device__ __forceinline__ void wait_stores_done() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

__device__ __forceinline__ void st_coh2(unsigned long long *p, float x, float y) {
    const unsigned long long w = (unsigned long long)__float_as_uint(x) |
                                 ((unsigned long long)__float_as_uint(y) << 32);
    __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void ld_coh2(const unsigned long long *p, float &x, float &y) {
    const unsigned long long w = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    x = __uint_as_float((unsigned)(w & 0xffffffffull));
    y = __uint_as_float((unsigned)(w >> 32));
}
__device__ __forceinline__ void st_coh(float *p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coh(double *p, double v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_coh(const float *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ double ld_coh(const double *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <typename T, int Q_, int R_, int NW_ = 0>
struct FShape {
    static constexpr int N = 128, P = 64, NH = 64, Q = Q_, R = R_;
    static constexpr int QR = Q * R;
    static constexpr int RT = QR / 16;                    // 16-row tiles in a chunk
    static constexpr int NW = NW_ ? NW_ : (RT >= 16 ? 8 : 4);   // waves per workgroup
    static constexpr int NWO = NW < RT ? NW : RT;         // waves owning output row tiles
    static constexpr int NTHR = NW * kWave;
    static constexpr int TPW = RT / NWO;                  // row tiles per output wave
    static constexpr int PTW = 16 / NW;                   // state pair-tiles per wave
    static constexpr int JB = 64, NJB = QR / JB;          // staged row blocks
    static constexpr int PAD = 16 / (int)sizeof(T);
    static constexpr int LDN = N + PAD;                   // [rows][N] and [P][N] tiles
    static constexpr int LDJ = JB + PAD;                  // [N or P][rows] tiles
    static constexpr int NSEG = NTHR / NH;                // angle-scan segments
    static constexpr int TPS = (Q + NSEG - 1) / NSEG;     // tokens per segment
    static constexpr int CE = Vec16<T>::n;                // elements per 16-byte vector
    static constexpr int ST_ELEMS = PTW * 2 * 4;          // state floats owned per lane
    typedef typename AccOf<T>::type Acc;
    typedef typename CsOf<T>::type CS;
    static_assert(QR % 64 == 0 && RT <= 32, "chunk*rank in {64, ..., 512}");
    static_assert(16 % R == 0, "row tiles hold whole tokens");
    static_assert(Q <= 256 && NTHR % NH == 0, "prologue mapping");
    static_assert(TPW >= 1 && TPW <= 4 && (TPW == 1 || TPW % 2 == 0), "tile assignment");
};

// Row tile owned as the m-th tile of output wave w: pairs of tiles from both
// ends of the chunk so that every wave gets the same causal work.
template <class S>
__device__ __forceinline__ int owned_tile(int w, int m) {
    const int base = (m / 2) * 2 * S::NWO;
    return (m % 2 == 0) ? base + w : base + 2 * S::NWO - 1 - w;
}

// Control block words of slice group y: the 64-bit ticket counter (ticket in
// bits 0-30, bit 31 set once the call's flags are cleared, the call epoch in
// bits 32-63).
__device__ __forceinline__ unsigned long long *group_counter(uint32_t *ctl, int y) {
    return reinterpret_cast<unsigned long long *>(ctl + kGroupStride * (y + 1));
}
constexpr uint32_t kTicketReady = 0x80000000u;

// Work item of a one-item-per-workgroup launch (grid = nsl * nchunks) whose
// chunks chain within a slice: slices are split into kGroups groups (slice %
// kGroups) and each group hands out its (chunk, slice) items chunk-major from
// its own counter, so every predecessor of an item holds an earlier ticket of
// the same counter and is resident or done (forward progress).  A workgroup
// asks the group of the XCD it runs on first (workgroups are spread over the
// XCDs, so the eight counters share the traffic), then the others; since the
// grid has exactly one workgroup per item, every workgroup finds one.  The
// ticket's word also brings the call epoch and whether the flags were
// already cleared.  Called by one thread.
__device__ __forceinline__ void take_item(uint32_t *ctl, int64_t nsl, int64_t nchunks, int64_t *c,
                                          int64_t *sl, uint32_t *epoch, bool *ready) {
    const int x = (int)(__builtin_amdgcn_s_getreg((3 << 11) | 20) & (kGroups - 1));   // XCC id
    for (int tries = 0; tries < kGroups; ++tries) {
        const int y = (x + tries) & (kGroups - 1);
        const int64_t ny = (nsl - y + kGroups - 1) / kGroups;   // slices of group y
        if (ny <= 0) continue;
        const unsigned long long w =
            __hip_atomic_fetch_add(group_counter(ctl, y), 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const int64_t k = (int64_t)((uint32_t)w & ~kTicketReady);
        if (k < ny * nchunks) {
            *c = k / ny;
            *sl = y + kGroups * (k % ny);
            *epoch = (uint32_t)(w >> 32);
            *ready = ((uint32_t)w & kTicketReady) != 0;
            return;
        }
    }
    *c = -1;   // unreachable with one workgroup per item
    *sl = -1;
    *epoch = 0;
    *ready = false;
}

// The same for sequences of different lengths (varlen tables): group y hands
// out its items chunk-major too, chunk level c holding the group's slices
// with more than c chunks; listed by decreasing chunk count, those are the
// first grp[y][c+1] - grp[y][c] slices of the group's list, so ticket k is
// chunk level c (the last with grp[y][c] <= k) and list entry k - grp[y][c].
// Every predecessor of an item again holds an earlier ticket of its counter.
// janitor: the item of group 0's last ticket.
__device__ __forceinline__ void take_item_var(uint32_t *ctl, const int32_t *grp, const int32_t *gstart,
                                              const int32_t *order, int maxn, int64_t *c, int64_t *sl,
                                              uint32_t *epoch, bool *ready, bool *janitor) {
    const int x = (int)(__builtin_amdgcn_s_getreg((3 << 11) | 20) & (kGroups - 1));   // XCC id
    for (int tries = 0; tries < kGroups; ++tries) {
        const int y = (x + tries) & (kGroups - 1);
        const int32_t *gy = grp + y * (maxn + 1);
        const int32_t items = gy[maxn];
        if (items <= 0) continue;
        const unsigned long long w =
            __hip_atomic_fetch_add(group_counter(ctl, y), 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const int32_t k = (int32_t)((uint32_t)w & ~kTicketReady);
        if (k < items) {
            int lo = 0, hi = maxn - 1;   // last level c with gy[c] <= k (gy[0] = 0)
            while (lo < hi) {
                const int mid = (lo + hi + 1) / 2;
                if (gy[mid] <= k) lo = mid; else hi = mid - 1;
            }
            *c = lo;
            *sl = order[gstart[y] + (k - gy[lo])];
            *epoch = (uint32_t)(w >> 32);
            *ready = ((uint32_t)w & kTicketReady) != 0;
            *janitor = y == 0 && k == items - 1;
            return;
        }
    }
    *c = -1;   // unreachable with one workgroup per item
    *sl = -1;
    *epoch = 0;
    *ready = false;
    *janitor = false;
}

// The call's first item clears the look-back flags [0, n) (all threads of the
// workgroup), then marks them cleared: the ready bit of every group's counter
// (seen by the items that take their tickets after), and, once those have
// landed, the ready word (polled by items that took theirs before, and by the
// janitor before it resets the counters).
__device__ __forceinline__ void clear_flags(uint32_t *ctl, uint32_t *flags, int64_t n, uint32_t epoch,
                                            int tid, int nthr) {
    unsigned long long *f2 = reinterpret_cast<unsigned long long *>(flags);   // 256-byte aligned
    for (int64_t i = tid; i < n / 2; i += nthr)
        __hip_atomic_store(f2 + i, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if ((n & 1) && tid == 0) __hip_atomic_store(flags + n - 1, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    wait_stores_done();
    __syncthreads();
    if (tid == 0) {
        for (int y = 0; y < kGroups; ++y)   // (the low word of each counter)
            __hip_atomic_fetch_or(reinterpret_cast<uint32_t *>(group_counter(ctl, y)), kTicketReady,
                                  __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        wait_stores_done();
        __hip_atomic_store(ctl + kCtlReady, epoch + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// A look-back wait of the call of this epoch gave up (counted in the epoch's
// own timeout word: the janitor never resets it while the call runs).
__device__ __forceinline__ void count_timeout(uint32_t *ctl, uint32_t epoch) {
    atomicAdd(ctl + ((epoch & 1u) ? kCtlTimeouts1 : kCtlTimeouts0), 1u);
}

// Bounded wait (one thread) until the flags of this epoch are cleared; false
// (and a timeout counted) if the wait gave up.
__device__ __forceinline__ bool wait_flags_ready(uint32_t *ctl, uint32_t epoch, uint32_t spin_max) {
    for (uint32_t spin = 0; spin < spin_max; ++spin) {
        if (__hip_atomic_load(ctl + kCtlReady, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == epoch + 1u)
            return true;
        __builtin_amdgcn_s_sleep(2);
    }
    count_timeout(ctl, epoch);
    return false;
}

// The call's janitor (the item of group 0's last ticket, one of the last to
// start), at its very end, one thread: waits (bounded) until every group has
// handed out all its tickets (so every workgroup holds its own and will touch
// no counter again) and the flags-cleared marks have landed, then resets the
// counters for the next epoch (ticket 0, flags not cleared) and zeroes the
// next epoch's timeout word, so the next call on the workspace starts from a
// clean block without a reset launch.  The wait is bounded by at least the
// default limit; one that gives up counts a timeout and resets all the same.
// Items of group y: (nsl - y + kGroups - 1) / kGroups slices of nunits each
// (0 past the last slice), or the varlen table's count.
__device__ __forceinline__ int64_t group_items(int y, int64_t nsl, int64_t nunits, const int32_t *grp, int maxn) {
    if (grp) return grp[y * (maxn + 1) + maxn];
    const int64_t items = (nsl - y + kGroups - 1) / kGroups * nunits;
    return items > 0 ? items : 0;
}

__device__ __forceinline__ void janitor_reset(uint32_t *ctl, int64_t nsl, int64_t nunits, uint32_t epoch,
                                              uint32_t spin_max, const int32_t *grp = nullptr, int maxn = 0) {
    const uint32_t lim = spin_max > kSpinMaxDefault ? spin_max : kSpinMaxDefault;
    bool all = false;
    for (uint32_t spin = 0; spin < lim && !all; ++spin) {
        all = __hip_atomic_load(ctl + kCtlReady, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == epoch + 1u;
#pragma unroll
        for (int y = 0; y < kGroups; ++y) {
            const int64_t items = group_items(y, nsl, nunits, grp, maxn);
            const uint32_t w = __hip_atomic_load(reinterpret_cast<uint32_t *>(group_counter(ctl, y)),
                                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            all = all && (int64_t)(w & ~kTicketReady) >= items;
        }
        if (!all) __builtin_amdgcn_s_sleep(2);
    }
    if (!all) count_timeout(ctl, epoch);
    __hip_atomic_store(ctl + ((epoch & 1u) ? kCtlTimeouts0 : kCtlTimeouts1), 0u, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
    const unsigned long long next = (unsigned long long)(epoch + 1u) << 32;
    for (int y = 0; y < kGroups; ++y)
        __hip_atomic_store(group_counter(ctl, y), next, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Whether item (unit u, slice sl) holds group 0's last ticket: the last unit
// of group 0's last slice.
__device__ __forceinline__ bool is_janitor(int64_t u, int64_t sl, int64_t nsl, int64_t nunits) {
    const int64_t ny0 = (nsl + kGroups - 1) / kGroups;
    return u == nunits - 1 && sl == (int64_t)kGroups * (ny0 - 1);
}

constexpr uint32_t kFlagInit = 3;   // probe result for "before the first chunk"
constexpr int kProbe = 16;          // predecessors probed per look-back round

// Workgroups of one kernel resident on the whole device at once (cached per
// device in `cache`; 0 on error).
inline int resident_capacity(const void *fn, int nthr, int *cache) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    int v = __atomic_load_n(&cache[dev], __ATOMIC_RELAXED);
    if (v > 0) return v;
    int ncu = 0, per = 0;
    if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, fn, nthr, 0) != hipSuccess) return 0;
    v = ncu * (per > 0 ? per : 1);
    __atomic_store_n(&cache[dev], v, __ATOMIC_RELAXED);
    return v;
}

// Initial state plus the carried previous-input term of token 0 for the K
// state elements a lane owns (element k at row n_of(k), column p_of(k) of the
// N x P state): h_{-1}[n][p] + wb sum_r B_{-1}[r][n] X_{-1}[r][p], with either
// part absent when its pointer is null (the carry's B and X come together).
// The null tests are taken once, outside the element loop, so that each
// case's element loads are issued together instead of one round trip each.
template <typename T, int R, int N, int P, int K, class FN, class FP>
__device__ __forceinline__ void init_elems(const float *ist, const T *iB, const T *iX, float wb, FN n_of,
                                           FP p_of, float *out) {
    auto fill = [&](auto kI, auto kB) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const int n = n_of(k), p = p_of(k);
            float sv = 0.f;
            if constexpr (decltype(kI)::value) sv = ist[n * P + p];
            if constexpr (decltype(kB)::value) {
                float u = 0.f;
#pragma unroll
                for (int r = 0; r < R; ++r) u += to_f32(iB[r * N + n]) * to_f32(iX[r * P + p]);
                sv += wb * u;
            }
            out[k] = sv;
        }
    };
    using Yes = std::integral_constant<bool, true>;
    using No = std::integral_constant<bool, false>;
    if (ist) {
        if (iB) fill(Yes{}, Yes{});
        else fill(Yes{}, No{});
    } else {
        if (iB) fill(No{}, Yes{});
        else fill(No{}, No{});
    }
}

}  // namespace scan
}  // namespace m3
