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

// ---------------------------------------------------------------------------
// Fast path (NHWC, Cin % 64 == 0): 32x32x32 int8 MFMA implicit GEMM.
// Rows = output channels (A = weights [cout][9][cin]), columns = pixels (B =
// the implicit im2col), k = (kernel position, 64-channel block).  A
// workgroup (8 waves) computes 128 channels x 256 pixels; wave w owns
// channels 64*(w%2).. and pixels 64*(w/2).. as 2x2 blocks of 32x32.  Each k
// step's A (128 rows x 64 B) and B (256 rows x 64 B) slices are copied
// global -> LDS with buffer loads straight into LDS, four stages in flight.
// A pixel outside the image (the 3x3 halo's zero padding) or beyond the
// batch gets an offset past the buffer's end, which the buffer load turns
// into zeros; the same holds for channels beyond Cout in the weights.
// LDS rows hold their 16-byte parts at slot p ^ ((row >> 1) & 3).
// ---------------------------------------------------------------------------
constexpr int DF_CO = 128, DF_PX = 256, DF_THREADS = 512, DF_NBUF = 4, DF_LPW = 3;
constexpr int DF_A = DF_CO * 64;
constexpr int DF_B = DF_PX * 64;
constexpr int DF_STAGE = DF_A + DF_B;

typedef int v16i __attribute__((ext_vector_type(16)));

struct DFArgs {
    int n, cin, cout, h, w;
    int npix, nbco, nblocks, nkb;
    int out_shift, relu;
    int x_bytes, w_bytes;
};

__device__ __forceinline__ int df_slot(int row, int part) { return part ^ ((row >> 1) & 3); }

__device__ __forceinline__ void df_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}
#define DF_WAIT_VM(n) __builtin_amdgcn_s_waitcnt(0x0f70 | (n))

__global__ __launch_bounds__(DF_THREADS) void direct_conv_nhwc_mfma(const int8_t* __restrict__ x,
                                                                   const int8_t* __restrict__ wt,
                                                                   const int32_t* __restrict__ bias,
                                                                   int8_t* __restrict__ y, DFArgs g) {
    __shared__ __attribute__((aligned(1024))) uint8_t lds[DF_NBUF * DF_STAGE];
    const int lbid = xcd_remap(blockIdx.x, g.nblocks);
    const int bco = lbid % g.nbco, bpx = lbid / g.nbco;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int co_blk = bco * DF_CO, px_blk = bpx * DF_PX;
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc((void*)x, 0, g.x_bytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc((void*)wt, 0, g.w_bytes, 0x00020000);
    const int wrow = 9 * g.cin;

    // this wave's three 1-KB load instructions per stage
    int rowi[DF_LPW], parti[DF_LPW], dsti[DF_LPW];
    bool isa[DF_LPW];
    int pimg[DF_LPW], ph[DF_LPW], pw_[DF_LPW];
#pragma unroll
    for (int i = 0; i < DF_LPW; ++i) {
        const int j = wave + 8 * i;                   // 0..23
        const int rr = lane >> 2, slot = lane & 3;
        isa[i] = j < DF_A / 1024;
        const int row = isa[i] ? 16 * j + rr : 16 * (j - DF_A / 1024) + rr;
        rowi[i] = row;
        parti[i] = df_slot(row, slot);
        dsti[i] = j * 1024;
        const int p = px_blk + row;
        const int pp = p < g.npix ? p : 0;
        pimg[i] = pp / (g.h * g.w);
        const int rem = pp - pimg[i] * g.h * g.w;
        ph[i] = p < g.npix ? rem / g.w : -100000;      // marks a pixel beyond the batch
        pw_[i] = rem - (rem / g.w) * g.w;
    }
    const int nst = 9 * g.nkb;
    auto issue = [&](int st) {
        const int rs = st / g.nkb, cb = st - rs * g.nkb;
        const int dr = rs / 3 - 1, ds = rs % 3 - 1;
        const int ci0 = cb * 64;
        uint8_t* base = lds + (st & (DF_NBUF - 1)) * DF_STAGE;
#pragma unroll
        for (int i = 0; i < DF_LPW; ++i) {
            int off;
            if (isa[i]) {
                const int co = co_blk + rowi[i];
                off = co < g.cout ? co * wrow + rs * g.cin + ci0 + 16 * parti[i] : 0x7fffffff;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (__attribute__((address_space(3))) void*)(base + dsti[i]),
                                                         16, off, 0, 0, 0);
            } else {
                const int hh = ph[i] + dr, ww = pw_[i] + ds;
                const bool ok = hh >= 0 && hh < g.h && ww >= 0 && ww < g.w;
                off = ok ? ((pimg[i] * g.h + hh) * g.w + ww) * g.cin + ci0 + 16 * parti[i] : 0x7fffffff;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (__attribute__((address_space(3))) void*)(base + dsti[i]),
                                                         16, off, 0, 0, 0);
            }
        }
    };

    const int cw = wave & 1, pwv = wave >> 1;
    const int l32 = lane & 31, lh = lane >> 5;
    v16i acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = (v16i){};
    int fa[2][2], fb[2][2];                   // [block][k half] LDS offsets
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int kh = 0; kh < 2; ++kh) {
            const int ra = 64 * cw + 32 * q + l32, rb = 64 * pwv + 32 * q + l32;
            fa[q][kh] = ra * 64 + 16 * df_slot(ra, 2 * kh + lh);
            fb[q][kh] = DF_A + rb * 64 + 16 * df_slot(rb, 2 * kh + lh);
        }

    for (int st = 0; st < DF_NBUF - 1 && st < nst; ++st) issue(st);
    for (int st = 0; st < nst; ++st) {
        const int ahead = nst - 1 - st;
        if (ahead >= 2) DF_WAIT_VM(2 * DF_LPW);
        else if (ahead == 1) DF_WAIT_VM(DF_LPW);
        else DF_WAIT_VM(0);
        df_barrier();
        if (st + DF_NBUF - 1 < nst) issue(st + DF_NBUF - 1);
        const uint8_t* base = lds + (st & (DF_NBUF - 1)) * DF_STAGE;
#pragma unroll
        for (int kh = 0; kh < 2; ++kh) {
            v4i av[2], bv[2];
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                av[q] = *(const v4i*)(base + fa[q][kh]);
                bv[q] = *(const v4i*)(base + fb[q][kh]);
            }
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b)
                    acc[a][b] = __builtin_amdgcn_mfma_i32_32x32x32_i8(av[a], bv[b], acc[a][b], 0, 0, 0);
        }
    }

    // accumulator layout (32x32 block): lane holds column l32 (a pixel) and
    // rows 8*(r/4) + 4*lh + r%4 (output channels) for r = 0..15
    const int s = g.out_shift;
    const int rnd = s > 0 ? 1 << (s - 1) : 0;
    const int lo = g.relu ? 0 : -128;
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        const int p = px_blk + 64 * pwv + 32 * b + l32;
        if (p >= g.npix) continue;
        int8_t* yp = y + (long long)p * g.cout;
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                const int co0 = co_blk + 64 * cw + 32 * a + 8 * r4 + 4 * lh;
                int qv[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int co = co0 + e;
                    const int z = acc[a][b][4 * r4 + e] + (bias && co < g.cout ? bias[co] : 0) + rnd;
                    int v = z >> s;
                    v = v < lo ? lo : (v > 127 ? 127 : v);
                    qv[e] = v;
                }
                if (co0 + 3 < g.cout && (g.cout & 3) == 0) {
                    *(uint32_t*)(yp + co0) = __builtin_amdgcn_perm((uint32_t)qv[1], (uint32_t)qv[0], 0x0c0c0400u) |
                                             (__builtin_amdgcn_perm((uint32_t)qv[3], (uint32_t)qv[2], 0x0c0c0400u) << 16);
                } else {
                    for (int e = 0; e < 4; ++e)
                        if (co0 + e < g.cout) yp[co0 + e] = (int8_t)qv[e];
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
    const long long xb = (long long)n * h * w * cin, wb = 9ll * cin * cout;
    // z = sum x w + bias + rounding must fit int32: |x w| <= 2^14, 9 cin <= 73728
    if (layout == WINO_NHWC && cin % 64 == 0 && xb < 0x7fffffffll && wb < 0x7fffffffll &&
        a.npix < 0x7fffffffll && (((uintptr_t)x & 15) == 0) && (((uintptr_t)w_ohwi & 15) == 0)) {
        DFArgs f;
        f.n = n;
        f.cin = cin;
        f.cout = cout;
        f.h = h;
        f.w = w;
        f.npix = (int)a.npix;
        f.nbco = (cout + DF_CO - 1) / DF_CO;
        f.nkb = cin / 64;
        long long nb = (a.npix + DF_PX - 1) / DF_PX * f.nbco;
        if (nb > 0x7fffffffll) return WINO_EUNSUPPORTED;
        f.nblocks = (int)nb;
        f.out_shift = out_shift;
        f.relu = relu;
        f.x_bytes = (int)xb;
        f.w_bytes = (int)wb;
        hipLaunchKernelGGL(direct_conv_nhwc_mfma, dim3((unsigned)nb), dim3(DF_THREADS), 0, stream, x, w_ohwi, bias,
                           y, f);
        return hipGetLastError() == hipSuccess ? WINO_OK : WINO_EHIP;
    }
    if (layout == WINO_NHWC)
        hipLaunchKernelGGL(direct_conv_kernel<WINO_NHWC>, dim3((unsigned)blocks), dim3(DC_THREADS), 0, stream, x,
                           w_ohwi, bias, y, a);
    else
        hipLaunchKernelGGL(direct_conv_kernel<WINO_NCHW>, dim3((unsigned)blocks), dim3(DC_THREADS), 0, stream, x,
                           w_ohwi, bias, y, a);
    return hipGetLastError() == hipSuccess ? WINO_OK : WINO_EHIP;
}
