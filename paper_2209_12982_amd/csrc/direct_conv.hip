// Direct int8 3x3 convolution (stride 1, pad 1) as an implicit GEMM on int8
// MFMA: the "standard algorithm" baseline the paper measures Winograd
// against (im2col lowering on the GEMM engine, Sec. IV-A and Sec. V).
//
// GEMM view: rows = output channels (A = weights [cout][9 * cin]), columns =
// output pixels (B = implicit im2col [9 * cin][pixels]), k = (kernel position,
// input channel).  z = sum x * w is exact in int32 for cin <= 8192
// (|x w| <= 2^14, 9 * 8192 * 2^14 < 2^31); then z + bias is requantized with
// R(v) = floor(v + 1/2) and clamped like the Winograd path.
#include "winof4_internal.h"

using namespace winof4;

typedef int v4i __attribute__((ext_vector_type(4)));

namespace {

constexpr int DC_WCO = 64;        // output channels per wave (4 MFMA rows)
constexpr int DC_WPX = 32;        // pixels per wave (2 MFMA columns)
constexpr int DC_CO = 2 * DC_WCO; // per workgroup
constexpr int DC_PX = 2 * DC_WPX;
constexpr int DC_THREADS = 256;

struct DCArgs {
    int n, cin, cout, h, w;
    long long npix;
    int nbco, nblocks;
    int out_shift, relu;
    int vec;                      // 16-byte loads allowed (Cin % 16 == 0, x and w aligned)
};

__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
    const int nx = 8;
    const int full = nblocks / nx * nx;
    if (bid >= full) return bid;
    return (bid % nx) * (full / nx) + bid / nx;
}

// 16 consecutive int8 values starting at channel c of one row of `cin`
// contiguous channels, zero beyond cin.
__device__ __forceinline__ v4i load16_channels(const int8_t* row, int c, int cin, int vec) {
    if (c >= cin) return (v4i){0, 0, 0, 0};
    if (vec) return *(const v4i*)(row + c);
    uint32_t wv[4] = {0, 0, 0, 0};
    for (int k = 0; k < 16; ++k)
        if (c + k < cin) wv[k >> 2] |= (uint32_t)(uint8_t)row[c + k] << (8 * (k & 3));
    return (v4i){(int)wv[0], (int)wv[1], (int)wv[2], (int)wv[3]};
}

template <int LAYOUT>
__global__ __launch_bounds__(DC_THREADS) void direct_conv_kernel(const int8_t* __restrict__ x,
                                                                 const int8_t* __restrict__ wt,
                                                                 const int32_t* __restrict__ bias,
                                                                 int8_t* __restrict__ y, DCArgs g) {
    const int lbid = xcd_remap(blockIdx.x, g.nblocks);
    const int bco = lbid % g.nbco, bpx = lbid / g.nbco;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int lr = lane & 15, lk = lane >> 4;
    const int co_base = bco * DC_CO + DC_WCO * (wave & 1);
    const long long px_base = (long long)bpx * DC_PX + DC_WPX * (wave >> 1);
    const long long hw = (long long)g.h * g.w;

    // the two pixel columns this lane feeds
    int pimg[2], ph[2], pw[2];
    bool pok[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        long long p = px_base + 16 * b + lr;
        pok[b] = p < g.npix;
        long long pp = pok[b] ? p : 0;
        pimg[b] = (int)(pp / hw);
        long long rem = pp - (long long)pimg[b] * hw;
        ph[b] = (int)(rem / g.w);
        pw[b] = (int)(rem - (long long)ph[b] * g.w);
    }
    v4i acc[4][2];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = (v4i){0, 0, 0, 0};

    const long long wrow = 9ll * g.cin;   // weights per output channel
    for (int rs = 0; rs < 9; ++rs) {
        const int dr = rs / 3 - 1, ds = rs % 3 - 1;
        for (int c0 = 0; c0 < g.cin; c0 += kKStep) {
            const int c = c0 + 16 * lk;
            v4i av[4], bv[2];
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                const int co = co_base + 16 * a + lr;
                av[a] = co < g.cout ? load16_channels(wt + co * wrow + rs * g.cin, c, g.cin, g.vec)
                                    : (v4i){0, 0, 0, 0};
            }
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const int hh = ph[b] + dr, ww = pw[b] + ds;
                bv[b] = (v4i){0, 0, 0, 0};
                if (pok[b] && hh >= 0 && hh < g.h && ww >= 0 && ww < g.w) {
                    if (LAYOUT == WINO_NHWC) {
                        bv[b] = load16_channels(x + (((long long)pimg[b] * g.h + hh) * g.w + ww) * g.cin, c, g.cin, g.vec);
                    } else {
                        uint32_t wv[4] = {0, 0, 0, 0};
                        const int8_t* src = x + ((long long)pimg[b] * g.cin * g.h + hh) * g.w + ww;
                        for (int k = 0; k < 16; ++k)
                            if (c + k < g.cin) wv[k >> 2] |= (uint32_t)(uint8_t)src[(long long)(c + k) * hw] << (8 * (k & 3));
                        bv[b] = (v4i){(int)wv[0], (int)wv[1], (int)wv[2], (int)wv[3]};
                    }
                }
            }
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b)
                    acc[a][b] = __builtin_amdgcn_mfma_i32_16x16x64_i8(av[a], bv[b], acc[a][b], 0, 0, 0);
        }
    }

    const int s = g.out_shift;
    const int rnd = s > 0 ? 1 << (s - 1) : 0;
    const int lo = g.relu ? 0 : -128;
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        if (!pok[b]) continue;
        const long long p = px_base + 16 * b + lr;
#pragma unroll
        for (int a = 0; a < 4; ++a) {
            const int co0 = co_base + 16 * a + 4 * lk;
            int qv[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int co = co0 + r;
                long long z = (long long)acc[a][b][r] + (bias && co < g.cout ? bias[co] : 0) + rnd;
                long long v = z >> s;
                v = v < lo ? lo : (v > 127 ? 127 : v);
                qv[r] = (int)v;
            }
            if (LAYOUT == WINO_NHWC) {
                int8_t* dst = y + p * g.cout + co0;
                if (co0 + 3 < g.cout && (g.cout & 3) == 0) {
                    *(uint32_t*)dst = (uint32_t)(qv[0] & 255) | ((uint32_t)(qv[1] & 255) << 8) |
                                      ((uint32_t)(qv[2] & 255) << 16) | ((uint32_t)(qv[3] & 255) << 24);
                } else {
                    for (int r = 0; r < 4; ++r)
                        if (co0 + r < g.cout) dst[r] = (int8_t)qv[r];
                }
            } else {
                const long long pimg_ = p / hw, rem = p - pimg_ * hw;
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (co0 + r < g.cout) y[(pimg_ * g.cout + co0 + r) * hw + rem] = (int8_t)qv[r];
            }
        }
    }
}

}  // namespace

extern "C" wino_status direct_conv_int8(const int8_t* x, const int8_t* w_ohwi, const int32_t* bias, int8_t* y,
                                        int32_t n, int32_t cin, int32_t cout, int32_t h, int32_t w,
                                        wino_layout layout, int32_t out_shift, int32_t relu, hipStream_t stream) {
    if (!x || !w_ohwi || !y) return WINO_EINVAL;
    if (n < 0 || h < 0 || w < 0 || cin < 1 || cout < 1) return WINO_EINVAL;
    if (layout != WINO_NCHW && layout != WINO_NHWC) return WINO_EINVAL;
    if (out_shift < 0 || out_shift > 31 || (relu != 0 && relu != 1)) return WINO_EINVAL;
    if (cin > 8192 || cout > 65536 || h > 65536 || w > 65536) return WINO_EUNSUPPORTED;
    DCArgs a;
    a.n = n;
    a.cin = cin;
    a.cout = cout;
    a.h = h;
    a.w = w;
    a.npix = (long long)n * h * w;
    if (a.npix == 0) return WINO_OK;
    a.nbco = (cout + DC_CO - 1) / DC_CO;
    long long blocks = (a.npix + DC_PX - 1) / DC_PX * a.nbco;
    if (blocks > 0x7fffffffll) return WINO_EUNSUPPORTED;
    a.nblocks = (int)blocks;
    a.out_shift = out_shift;
    a.relu = relu;
    a.vec = (cin % 16 == 0) && (((uintptr_t)x & 15) == 0) && (((uintptr_t)w_ohwi & 15) == 0);
    if (layout == WINO_NHWC)
        hipLaunchKernelGGL(direct_conv_kernel<WINO_NHWC>, dim3((unsigned)blocks), dim3(DC_THREADS), 0, stream, x,
                           w_ohwi, bias, y, a);
    else
        hipLaunchKernelGGL(direct_conv_kernel<WINO_NCHW>, dim3((unsigned)blocks), dim3(DC_THREADS), 0, stream, x,
                           w_ohwi, bias, y, a);
    return hipGetLastError() == hipSuccess ? WINO_OK : WINO_EHIP;
}
