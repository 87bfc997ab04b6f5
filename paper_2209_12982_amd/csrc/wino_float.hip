// Unquantized Winograd F(4x4, 3x3) in fp32: the floating-point algorithm of
// Eq. (winograd), Sec. II, with the F(4x4,3x3) matrices printed there and no
// tap-wise quantization.  It is the real-valued convolution that the integer
// pipeline of Sec. III approximates, kept as a reference stage: every
// intermediate (V, U, M, Y) is an fp32 value, which lets a test hold the
// floating-point stages to a relative tolerance.  One thread per (tile,
// output channel); not on the hot path and not tuned.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "winof4.h"

namespace {

// B^T (6x6), G (6x3) and A^T (4x6) of F(4x4, 3x3), Sec. II.  G is printed as
// (1/3) [[3/4,0,0], [-1/2,-1/2,-1/2], [-1/2,1/2,-1/2], [1/8,1/4,1/2],
// [1/8,-1/4,1/2], [0,0,3]]; the entries below are those products.
__constant__ float kBT[6][6] = {
    {4.f, 0.f, -5.f, 0.f, 1.f, 0.f},   {0.f, -4.f, -4.f, 1.f, 1.f, 0.f}, {0.f, 4.f, -4.f, -1.f, 1.f, 0.f},
    {0.f, -2.f, -1.f, 2.f, 1.f, 0.f}, {0.f, 2.f, -1.f, -2.f, 1.f, 0.f}, {0.f, 4.f, 0.f, -5.f, 0.f, 1.f},
};
__constant__ float kG[6][3] = {
    {1.f / 4.f, 0.f, 0.f},
    {-1.f / 6.f, -1.f / 6.f, -1.f / 6.f},
    {-1.f / 6.f, 1.f / 6.f, -1.f / 6.f},
    {1.f / 24.f, 1.f / 12.f, 1.f / 6.f},
    {1.f / 24.f, -1.f / 12.f, 1.f / 6.f},
    {0.f, 0.f, 1.f},
};
__constant__ float kAT[4][6] = {
    {1.f, 1.f, 1.f, 1.f, 1.f, 0.f},
    {0.f, 1.f, -1.f, 2.f, -2.f, 0.f},
    {0.f, 1.f, 1.f, 4.f, 4.f, 0.f},
    {0.f, 1.f, -1.f, 8.f, -8.f, 1.f},
};

struct FloatArgs {
    int n, cin, cout, h, w, th, tw;
    long long ntiles;
    int layout;
};

__global__ __launch_bounds__(256) void wino_f4_float(const int8_t* __restrict__ x, const float* __restrict__ wt,
                                                     float* __restrict__ y, FloatArgs g) {
    const long long gid = (long long)blockIdx.x * 256 + threadIdx.x;
    if (gid >= g.ntiles * g.cout) return;
    const int co = (int)(gid % g.cout);
    const long long tile = gid / g.cout;
    const long long per_img = (long long)g.th * g.tw;
    const int img = (int)(tile / per_img);
    const int rem = (int)(tile - img * per_img);
    const int ty = rem / g.tw, tx = rem - (rem / g.tw) * g.tw;

    // M is summed over blocks of 16 input channels and the block sums are
    // added up, which keeps the fp32 rounding growth at ~16 + cin/16 terms
    // instead of cin
    float m[6][6], mb[6][6];
    for (int i = 0; i < 6; ++i)
        for (int j = 0; j < 6; ++j) m[i][j] = mb[i][j] = 0.f;
    for (int ci = 0; ci < g.cin; ++ci) {
        // the 6x6 input window at rows 4ty-1 .. 4ty+4, cols 4tx-1 .. 4tx+4,
        // zero outside the image
        float d[6][6];
        for (int r = 0; r < 6; ++r) {
            const int yy = 4 * ty - 1 + r;
            for (int c = 0; c < 6; ++c) {
                const int xx = 4 * tx - 1 + c;
                float v = 0.f;
                if (yy >= 0 && yy < g.h && xx >= 0 && xx < g.w) {
                    const long long idx = g.layout == WINO_NCHW
                                              ? (((long long)img * g.cin + ci) * g.h + yy) * g.w + xx
                                              : (((long long)img * g.h + yy) * g.w + xx) * g.cin + ci;
                    v = (float)x[idx];
                }
                d[r][c] = v;
            }
        }
        // V = B^T d B: columns first (t = B^T d), then rows (V = t B)
        float t[6][6], v[6][6];
        for (int i = 0; i < 6; ++i)
            for (int c = 0; c < 6; ++c) {
                float s = 0.f;
                for (int k = 0; k < 6; ++k) s += kBT[i][k] * d[k][c];
                t[i][c] = s;
            }
        for (int i = 0; i < 6; ++i)
            for (int j = 0; j < 6; ++j) {
                float s = 0.f;
                for (int k = 0; k < 6; ++k) s += t[i][k] * kBT[j][k];
                v[i][j] = s;
            }
        // U = G f G^T for the kernel f of (co, ci)
        const float* f = wt + ((long long)co * g.cin + ci) * 9;
        float gf[6][3], u[6][6];
        for (int i = 0; i < 6; ++i)
            for (int c = 0; c < 3; ++c) {
                float s = 0.f;
                for (int k = 0; k < 3; ++k) s += kG[i][k] * f[3 * k + c];
                gf[i][c] = s;
            }
        for (int i = 0; i < 6; ++i)
            for (int j = 0; j < 6; ++j) {
                float s = 0.f;
                for (int k = 0; k < 3; ++k) s += gf[i][k] * kG[j][k];
                u[i][j] = s;
            }
        for (int i = 0; i < 6; ++i)
            for (int j = 0; j < 6; ++j) mb[i][j] += v[i][j] * u[i][j];
        if ((ci & 15) == 15 || ci == g.cin - 1)
            for (int i = 0; i < 6; ++i)
                for (int j = 0; j < 6; ++j) {
                    m[i][j] += mb[i][j];
                    mb[i][j] = 0.f;
                }
    }
    // Y = A^T M A, stored where the 4x4 tile lies inside the image
    float am[4][6];
    for (int i = 0; i < 4; ++i)
        for (int c = 0; c < 6; ++c) {
            float s = 0.f;
            for (int k = 0; k < 6; ++k) s += kAT[i][k] * m[k][c];
            am[i][c] = s;
        }
    for (int i = 0; i < 4; ++i) {
        const int yy = 4 * ty + i;
        if (yy >= g.h) break;
        for (int j = 0; j < 4; ++j) {
            const int xx = 4 * tx + j;
            if (xx >= g.w) break;
            float s = 0.f;
            for (int k = 0; k < 6; ++k) s += am[i][k] * kAT[j][k];
            const long long idx = g.layout == WINO_NCHW ? (((long long)img * g.cout + co) * g.h + yy) * g.w + xx
                                                        : (((long long)img * g.h + yy) * g.w + xx) * g.cout + co;
            y[idx] = s;
        }
    }
}

}  // namespace

extern "C" wino_status wino_f4_conv_float(const int8_t* x, const float* w_oihw, float* y, int32_t n, int32_t cin,
                                          int32_t cout, int32_t h, int32_t w, wino_layout layout,
                                          hipStream_t stream) {
    if (!x || !w_oihw || !y) return WINO_EINVAL;
    if (n < 0 || h < 0 || w < 0 || cin < 1 || cout < 1) return WINO_EINVAL;
    if (layout != WINO_NCHW && layout != WINO_NHWC) return WINO_EINVAL;
    if (cin > 65536 || cout > 65536 || h > 65536 || w > 65536) return WINO_EUNSUPPORTED;
    FloatArgs a;
    a.n = n;
    a.cin = cin;
    a.cout = cout;
    a.h = h;
    a.w = w;
    a.th = (h + 3) / 4;
    a.tw = (w + 3) / 4;
    a.ntiles = (long long)n * a.th * a.tw;
    a.layout = layout;
    const long long threads = a.ntiles * cout;
    if (threads == 0) return WINO_OK;
    const long long blocks = (threads + 255) / 256;
    if (blocks > 0x7fffffffll) return WINO_EUNSUPPORTED;
    hipLaunchKernelGGL(wino_f4_float, dim3((unsigned)blocks), dim3(256), 0, stream, x, w_oihw, y, a);
    return hipGetLastError() == hipSuccess ? WINO_OK : WINO_EHIP;
}
