// On-device weight transform, tap calibration and tap-wise quantization: the
// offline step of the method (Sec. III-B: U = G f G^T, one power-of-two scale
// 2^e_G per Winograd tap from the tap's largest magnitude, Uq = clamp(R(U /
// 2^e_G))), run on the GPU.  The paper transforms weights inside the
// accelerator because Winograd-domain weights are four times the spatial ones
// (Sec. IV, weight buffer and on-the-fly weight transform); here the transform
// is a plan-time pass that writes Uq straight into the tap-GEMM layout.
//
// Two inputs:
//  * fp32 weights.  d^2 U for one tap is the sum of nine exact doubles
//    Gint[a][i] Gint[b][j] f[i][j]; each sum is grown into a non-overlapping
//    expansion with TwoSum (Shewchuk 1997, GROW-EXPANSION), so every rounding
//    and range decision is exact and the tables equal the host plan's bit for
//    bit.  Three passes: (1) the per-tap maximum of the sums' double
//    approximations; (2) exact tests of the sums near the two candidate
//    power-of-two bounds, which fix e_G; (3) the exact quantization.
//  * int8 spatial weights f_hat = w * 2^e_f (the quantized weights that the
//    tap-wise formula of Sec. III starts from).  d^2 U = Gint w Gint^T is an
//    integer (|.| <= 128 * 24^2 for F4), so both passes are integer-exact.
//
// Thread mapping (both inputs): grid (plane / 256, ntap); block y = tap t;
// thread j of the tap plane is Uq's element [kb][co][c] of the k-blocked
// layout [ntap][cin_pad / 64][cout_pad][64], ci = 64 kb + c, so pass 3 writes
// each tap plane contiguously and one wave holds one (kb, co) row.
#include <hip/hip_runtime.h>
#include <cmath>
#include "winof4_internal.h"

// TwoSum is exact only without contraction or reassociation.
#pragma clang fp contract(off)

using namespace winof4;

namespace {

constexpr int kBlock = 256;

// Per-tap slot of the device state, one 128-byte line per tap so that the
// workgroups' atomics on different taps do not queue on one line.
struct alignas(128) TapSlot {
    unsigned long long amax;          // bit pattern of max |approx d^2 U| (non-negative doubles order as integers)
    int hi;                           // some |d^2 U| > 128 d^2 2^e_c
    int lo;                           // some |d^2 U| > 128 d^2 2^(e_c - 1)
    int imax;                         // int8 input: max |d^2 U|
    int e_g;                          // result
};

// Per-call device state, cleared before pass 1.
struct CalState {
    TapSlot tap[kTaps];
    int bad;                          // a non-finite weight was seen
};

struct TapExps {
    int given;                        // 1: e_G supplied by the caller
    int e[kTaps];
};

struct Geo {
    int cin, cout, cout_pad, nkb;
    long long plane;                  // nkb * cout_pad * 64
};

__host__ __device__ inline void two_sum(double a, double b, double& s, double& e) {
    s = a + b;
    double bv = s - a;
    double av = s - bv;
    e = (a - av) + (b - bv);
}

// Locates thread j of a tap plane; returns false for padding.
__device__ inline bool locate(const Geo& g, long long j, int& co, int& ci) {
    const long long row = j >> 6;
    co = (int)(row % g.cout_pad);
    ci = (int)(row / g.cout_pad) * 64 + (int)(j & 63);
    return co < g.cout && ci < g.cin;
}

// The nine exact terms of d^2 U[a][b] grown into an expansion c[0..8]
// (increasing magnitude, zero components allowed); returns its double
// approximation (components summed small to large).  Sets `finite`.
__host__ __device__ inline double tap_expansion(const Xform& X, const float* f9, int a, int b, double c[9],
                                       bool& finite) {
    finite = true;
#pragma unroll
    for (int k = 0; k < 9; ++k) {
        const float fv = f9[k];
        finite = finite && __builtin_isfinite(fv);
        double q = (double)(X.gint[a][k / 3] * X.gint[b][k % 3]) * (double)fv;
#pragma unroll
        for (int i = 0; i < k; ++i) {
            double s, e;
            two_sum(q, c[i], s, e);
            c[i] = e;
            q = s;
        }
        c[k] = q;
    }
    double s = 0.0;
#pragma unroll
    for (int i = 0; i < 9; ++i) s += c[i];
    return s;
}

// Sign of (sum of the expansion) - thr, exactly: the largest non-zero
// component of a non-overlapping expansion carries the sign of the sum.
__host__ __device__ inline int sign_minus(const double c[9], double thr) {
    double q = -thr;
    int sg = 0;
#pragma unroll
    for (int i = 0; i < 9; ++i) {
        double s, e;
        two_sum(q, c[i], s, e);
        if (e != 0.0) sg = e > 0.0 ? 1 : -1;
        q = s;
    }
    if (q != 0.0) sg = q > 0.0 ? 1 : -1;
    return sg;
}

// Smallest e with amax <= unit 2^e for a double amax > 0.
__host__ __device__ inline int cexp_of(double amax, double unit) {
    int e;
    frexp(amax / unit, &e);
    e -= 1;
    while (ldexp(unit, e) < amax) ++e;
    while (ldexp(unit, e - 1) >= amax) --e;
    return e;
}

// e_G of tap t from the pass-1 maximum and the pass-2 flags.  The double
// approximations are within a few ulps of the exact sums, so with e_c the
// exponent of the approximate maximum the exact one is e_c - 1, e_c or
// e_c + 1, and the two flags tell which.
__device__ inline int tap_exponent(const CalState* st, const TapExps& te, int t, double unit) {
    if (te.given) return te.e[t];
    const double amax = __longlong_as_double((long long)st->tap[t].amax);
    if (amax == 0.0) return 0;        // an expansion sums to 0.0 only when it is exactly 0
    const int ec = cexp_of(amax, unit);
    return st->tap[t].hi ? ec + 1 : (st->tap[t].lo ? ec : ec - 1);
}

__device__ inline double wave_max(double v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o));
    return v;
}

__device__ inline int wave_sum(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

__device__ inline int wave_max_i(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o));
    return v;
}

// Maximum over the workgroup (kBlock / 64 waves), valid in thread 0.
template <class T>
__device__ inline T block_max(T v, T* red) {
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    if (threadIdx.x == 0)
        for (int i = 1; i < kBlock / 64; ++i) v = red[i] > v ? red[i] : v;
    return v;
}

// Pass 1 (fp32): per-tap maximum of |approx d^2 U|; non-finite weights.
__global__ void __launch_bounds__(kBlock) wt_f32_max(Xform X, Geo g, const float* __restrict__ w,
                                                     CalState* st) {
    const int t = blockIdx.y, a = t / X.n, b = t % X.n;
    const long long j = (long long)blockIdx.x * kBlock + threadIdx.x;
    int co, ci;
    double v = 0.0;
    bool bad = false;
    if (j < g.plane && locate(g, j, co, ci)) {
        double c[9];
        bool finite;
        v = fabs(tap_expansion(X, w + ((long long)co * g.cin + ci) * 9, a, b, c, finite));
        bad = !finite;
        if (bad) v = 0.0;
    }
    __shared__ double red[kBlock / 64];
    const bool any_bad = __any(bad);
    v = block_max(wave_max(v), red);
    if (threadIdx.x == 0 && v > 0.0) atomicMax(&st->tap[t].amax, (unsigned long long)__double_as_longlong(v));
    if (any_bad && (threadIdx.x & 63) == 0) atomicOr(&st->bad, 1);
}

// Pass 2 (fp32): exact tests against 128 d^2 2^e_c and 128 d^2 2^(e_c - 1).
__global__ void __launch_bounds__(kBlock) wt_f32_flags(Xform X, Geo g, const float* __restrict__ w,
                                                       CalState* st) {
    const int t = blockIdx.y, a = t / X.n, b = t % X.n;
    const double unit = 128.0 * X.den2;
    const double amax = __longlong_as_double((long long)st->tap[t].amax);
    if (amax == 0.0) return;                        // uniform per block
    const int ec = cexp_of(amax, unit);
    const double hi = ldexp(unit, ec), lo = ldexp(unit, ec - 1);
    const double rel = 1e-9;
    const long long j = (long long)blockIdx.x * kBlock + threadIdx.x;
    int co, ci;
    bool over_hi = false, over_lo = false;
    if (j < g.plane && locate(g, j, co, ci)) {
        double c[9];
        bool finite;
        const double v = fabs(tap_expansion(X, w + ((long long)co * g.cin + ci) * 9, a, b, c, finite));
        if (finite) {
            if (v >= hi * (1 - rel)) over_hi = sign_minus(c, hi) > 0 || sign_minus(c, -hi) < 0;
            if (v > lo * (1 + rel)) over_lo = true;
            else if (v >= lo * (1 - rel)) over_lo = sign_minus(c, lo) > 0 || sign_minus(c, -lo) < 0;
        }
    }
    // one atomic per workgroup and flag, skipped once the flag is seen set
    const int any_hi = __syncthreads_or(over_hi), any_lo = __syncthreads_or(over_lo);
    if (threadIdx.x == 0) {
        if (any_hi && !__hip_atomic_load(&st->tap[t].hi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
            atomicOr(&st->tap[t].hi, 1);
        if (any_lo && !__hip_atomic_load(&st->tap[t].lo, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
            atomicOr(&st->tap[t].lo, 1);
    }
}

// clamp(R(S / (d^2 2^e)), -128, 127) for the exact sum S held in c.
__host__ __device__ inline int quantize_exact(const double c[9], double approx, int den2, int e) {
    const double scale = ldexp((double)den2, e);
    const double u = approx / scale;
    if (!(u < 200.0)) return 127;
    if (!(u > -200.0)) return -128;
    double q = floor(u + 0.5);
    // need (q - 1/2) scale <= S < (q + 1/2) scale; the approximation is off by
    // far less than one step, so at most one correction is needed
    for (int guard = 0; guard < 4; ++guard) {
        if (sign_minus(c, (q - 0.5) * scale) < 0) { q -= 1.0; continue; }
        if (sign_minus(c, (q + 0.5) * scale) >= 0) { q += 1.0; continue; }
        break;
    }
    return (int)fmin(127.0, fmax(-128.0, q));
}

// Pass 3 (fp32): quantize, write Uq (zeros in the padding), column sums.
__global__ void __launch_bounds__(kBlock) wt_f32_quant(Xform X, Geo g, TapExps te, const float* __restrict__ w,
                                                       CalState* st, int8_t* __restrict__ uq,
                                                       int* __restrict__ colsum) {
    const int t = blockIdx.y, a = t / X.n, b = t % X.n;
    const int e = tap_exponent(st, te, t, 128.0 * X.den2);
    if (blockIdx.x == 0 && threadIdx.x == 0) st->tap[t].e_g = e;
    const bool ok = e >= -126 && e <= 126;
    const long long j = (long long)blockIdx.x * kBlock + threadIdx.x;
    if (j >= g.plane) return;                        // whole waves: plane is a multiple of 64
    int co, ci;
    int q = 0;
    const bool valid = locate(g, j, co, ci);
    if (valid && ok) {
        double c[9];
        bool finite;
        const double approx = tap_expansion(X, w + ((long long)co * g.cin + ci) * 9, a, b, c, finite);
        if (finite) q = quantize_exact(c, approx, X.den2, e);
    }
    uq[(long long)t * g.plane + j] = (int8_t)q;
    const int s = wave_sum(q < 0 ? -q : q);
    if ((threadIdx.x & 63) == 0 && co < g.cout && s != 0) atomicAdd(&colsum[(long long)t * g.cout + co], s);
}

// d^2 U[a][b] of int8 weights, exactly.
__host__ __device__ inline int tap_int(const Xform& X, const int8_t* f9, int a, int b) {
    int s = 0;
#pragma unroll
    for (int k = 0; k < 9; ++k) s += X.gint[a][k / 3] * X.gint[b][k % 3] * (int)f9[k];
    return s;
}

// Pass 1 (int8): per-tap maximum of |d^2 U|.
__global__ void __launch_bounds__(kBlock) wt_i8_max(Xform X, Geo g, const int8_t* __restrict__ w, CalState* st) {
    const int t = blockIdx.y, a = t / X.n, b = t % X.n;
    const long long j = (long long)blockIdx.x * kBlock + threadIdx.x;
    int co, ci, v = 0;
    if (j < g.plane && locate(g, j, co, ci)) v = abs(tap_int(X, w + ((long long)co * g.cin + ci) * 9, a, b));
    __shared__ int red[kBlock / 64];
    v = block_max(wave_max_i(v), red);
    if (threadIdx.x == 0 && v > 0) atomicMax(&st->tap[t].imax, v);
}

// m <= unit 2^d for 1 <= m < 2^20, unit < 2^20, -40 <= d <= 40.
__host__ __device__ inline bool fits_pow2(long long m, long long unit, int d) {
    return d >= 0 ? m <= (unit << d) : (m << -d) <= unit;
}

__host__ __device__ inline long long floor_div(long long a, long long b) {   // b > 0
    return a >= 0 ? a / b : -((-a + b - 1) / b);
}

// e_G of an int8 tap with max|S| = m > 0, S = d^2 U 2^-e_f an integer:
// e_f + k with k the smallest integer such that m <= 128 d^2 2^k
// (m <= 128 (sum_i |Gint[a][i]|)^2, so k ends in [-17, 2]).
__host__ __device__ inline int int8_tap_exponent(long long m, int den2, int e_f) {
    const long long unit = 128LL * den2;
    int k = 0;
    while (!fits_pow2(m, unit, k)) ++k;
    while (fits_pow2(m, unit, k - 1)) --k;
    return e_f + k;
}

// clamp(R(s / (d^2 2^k)), -128, 127) for an integer s, |s| < 2^17.
__host__ __device__ inline int int8_quantize(long long s, int den2, int k) {
    long long r;
    if (k > 40) {
        r = 0;                                        // |s| / (d^2 2^k) < 1/2
    } else if (k >= 0) {
        const long long den = (long long)den2 << k;
        r = floor_div(2 * s + den, 2 * den);
    } else if (k < -40) {
        r = s > 0 ? 127 : (s < 0 ? -128 : 0);
    } else {
        r = floor_div(2 * s * (1LL << -k) + den2, 2LL * den2);
    }
    return (int)(r > 127 ? 127 : (r < -128 ? -128 : r));
}

// Pass 2 (int8): U / 2^e_G = S 2^(e_f - e_G) / d^2; e_G = 0 for an all-zero tap.
__global__ void __launch_bounds__(kBlock) wt_i8_quant(Xform X, Geo g, TapExps te, int e_f,
                                                      const int8_t* __restrict__ w, CalState* st,
                                                      int8_t* __restrict__ uq, int* __restrict__ colsum) {
    const int t = blockIdx.y, a = t / X.n, b = t % X.n;
    const int e = te.given ? te.e[t] : (st->tap[t].imax == 0 ? 0 : int8_tap_exponent(st->tap[t].imax, X.den2, e_f));
    if (blockIdx.x == 0 && threadIdx.x == 0) st->tap[t].e_g = e;
    const long long j = (long long)blockIdx.x * kBlock + threadIdx.x;
    if (j >= g.plane) return;
    int co, ci, q = 0;
    if (locate(g, j, co, ci) && e >= -126 && e <= 126)
        q = int8_quantize(tap_int(X, w + ((long long)co * g.cin + ci) * 9, a, b), X.den2, e - e_f);
    uq[(long long)t * g.plane + j] = (int8_t)q;
    const int sum = wave_sum(q < 0 ? -q : q);
    if ((threadIdx.x & 63) == 0 && co < g.cout && sum != 0) atomicAdd(&colsum[(long long)t * g.cout + co], sum);
}

// Shared set-up, launch and read-back of both inputs.
template <class Launch>
wino_status run_device_tables(const Xform& X, wino_f4_plan_s* p, const int8_t* w_exp, hipStream_t stream,
                              std::vector<int32_t>& colsum, Launch launch) {
    Geo g;
    g.cin = p->cin;
    g.cout = p->cout;
    g.cout_pad = p->cout_pad;
    g.nkb = p->cin_pad / kKStep;
    g.plane = (long long)g.nkb * g.cout_pad * 64;
    TapExps te{};
    te.given = w_exp ? 1 : 0;
    for (int t = 0; t < X.ntap; ++t) te.e[t] = w_exp ? w_exp[t] : 0;
    const long long nblocks = g.plane / kBlock + (g.plane % kBlock ? 1 : 0);
    if (nblocks > 0x7fffffffLL) return WINO_EUNSUPPORTED;
    const dim3 grid((unsigned)nblocks, X.ntap);

    const size_t uq_bytes = (size_t)X.ntap * g.plane;
    const size_t cs_bytes = (size_t)X.ntap * g.cout * sizeof(int32_t);
    char* scratch = nullptr;
    if (hipMalloc(&p->uq_dev, uq_bytes) != hipSuccess) {
        p->uq_dev = nullptr;
        return WINO_ENOMEM;
    }
    if (hipMalloc(&scratch, sizeof(CalState) + cs_bytes) != hipSuccess) return WINO_ENOMEM;
    CalState* st = reinterpret_cast<CalState*>(scratch);
    int* cs = reinterpret_cast<int*>(scratch + sizeof(CalState));
    CalState host{};
    try {
        colsum.assign((size_t)X.ntap * g.cout, 0);
    } catch (...) {
        (void)hipFree(scratch);
        return WINO_ENOMEM;
    }
    bool ok = hipMemsetAsync(scratch, 0, sizeof(CalState) + cs_bytes, stream) == hipSuccess;
    if (ok) ok = launch(grid, g, te, st, cs);
    ok = ok && hipMemcpyAsync(&host, st, sizeof(CalState), hipMemcpyDeviceToHost, stream) == hipSuccess &&
         hipMemcpyAsync(colsum.data(), cs, cs_bytes, hipMemcpyDeviceToHost, stream) == hipSuccess &&
         hipStreamSynchronize(stream) == hipSuccess;
    (void)hipFree(scratch);
    if (!ok) return WINO_EHIP;
    if (host.bad) return WINO_EINVAL;
    for (int t = 0; t < X.ntap; ++t) {
        if (host.tap[t].e_g < -126 || host.tap[t].e_g > 126) return WINO_ERANGE;
        p->e_g[t] = (int8_t)host.tap[t].e_g;
    }
    return WINO_OK;
}

}  // namespace

namespace winof4 {

wino_status device_weight_tables(const Xform& X, wino_f4_plan_s* p, const float* w_dev, const int8_t* w_exp,
                                 hipStream_t stream, std::vector<int32_t>& colsum) {
    return run_device_tables(X, p, w_exp, stream, colsum,
                             [&](dim3 grid, const Geo& g, const TapExps& te, CalState* st, int* cs) {
        // pass 1 also finds non-finite weights, so it runs with given exponents too
        hipLaunchKernelGGL(wt_f32_max, grid, dim3(kBlock), 0, stream, X, g, w_dev, st);
        if (!te.given) hipLaunchKernelGGL(wt_f32_flags, grid, dim3(kBlock), 0, stream, X, g, w_dev, st);
        hipLaunchKernelGGL(wt_f32_quant, grid, dim3(kBlock), 0, stream, X, g, te, w_dev, st, p->uq_dev, cs);
        return hipGetLastError() == hipSuccess;
    });
}

wino_status device_weight_tables_int8(const Xform& X, wino_f4_plan_s* p, const int8_t* w_dev, int32_t w_scale_exp,
                                      const int8_t* w_exp, hipStream_t stream, std::vector<int32_t>& colsum) {
    return run_device_tables(X, p, w_exp, stream, colsum,
                             [&](dim3 grid, const Geo& g, const TapExps& te, CalState* st, int* cs) {
        if (!te.given) hipLaunchKernelGGL(wt_i8_max, grid, dim3(kBlock), 0, stream, X, g, w_dev, st);
        hipLaunchKernelGGL(wt_i8_quant, grid, dim3(kBlock), 0, stream, X, g, te, w_scale_exp, w_dev, st,
                           p->uq_dev, cs);
        return hipGetLastError() == hipSuccess;
    });
}

}  // namespace winof4
