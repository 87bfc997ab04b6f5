// FUSED variant of the online path: one launch per convolution, for F4 and
// F2 plans.  Each workgroup (8 waves, 64 output channels x 32 tiles) computes
// its tiles' Winograd-domain input in the GEMM prologue, so the tap-major Vq
// never goes to memory (the input transform of Sec. IV-B2's operator dataflow
// feeding the Cube from on-chip memory).  Per 64-channel k step:
//   1. each thread takes two (tile, channel pair) items: it loads the N x N
//      window of two channels, computes B^T d B in two 16-bit lanes and the
//      tap-wise requantization, and writes the NTAP resulting byte pairs into
//      the LDS Vq block [NTAP taps][32 tiles][64 B] (two channels at a time
//      keeps the transform next to the accumulators: 144 registers for F4's
//      36 taps, 64 for F2's 16);
//   2. the tap MFMAs read Vq from LDS and Uq from a three-stage ring that the
//      direct-to-LDS load keeps filled (the ring also loads while step 1
//      runs);
// then the same fused output-transform epilogue as the SPLIT tap GEMM.
// The input transform is recomputed once per 64-output-channel block
// (Cout/64 times in all), so this variant pays off when Cout is small.  F2's
// workgroup needs 80 KB of LDS and at most 128 registers a lane, so two run
// on a CU.
#include "wino_device.h"

using namespace winof4;

namespace {

constexpr int K4_CO = 64;
constexpr int K4_TL = 32;
constexpr int K4_THREADS = 512;
constexpr int K4_WAVES = K4_THREADS / 64;
constexpr int K4_NBUF = 3;
static_assert(K4_TL * 32 == 2 * K4_THREADS, "two (tile, channel pair) items per thread per k step");

template <int M>
struct K4Cfg {
    static constexpr int N = Wino<M>::N, NT = Wino<M>::NTAP;
    static constexpr int G = M == 4 ? 6 : 4;                 // taps per Uq ring stage
    static constexpr int A_STAGE = G * K4_CO * 64;           // 24 KB (F4), 16 KB (F2)
    static constexpr int B_BYTES = NT * K4_TL * 64;          // Vq block: 72 KB, 32 KB
    static constexpr int LPW = A_STAGE / 1024 / K4_WAVES;    // 1-KB loads per wave per stage
    static constexpr int LDS = B_BYTES + K4_NBUF * A_STAGE;
    static constexpr int WAVES_PER_EU = M == 4 ? 1 : 4;     // F2: two workgroups per CU
    static_assert(NT % G == 0 && A_STAGE / 1024 % K4_WAVES == 0, "stages tile the taps; loads split evenly");
    static_assert(K4_WAVES * LPW == 4 * G, "wave -> (tap, 16-row group) map of the ring loads");
    static_assert(LDS <= 160 * 1024 && (M == 4 || 2 * LDS <= 160 * 1024), "LDS");
};

struct K4Args {
    int cin, cin_pad, cout, cout_pad;
    int n, h, w, th, tw;
    long long ntiles;
    int nbco, nblocks;
    int out_shift, relu;
    int x_vec;                      // NHWC 2-byte channel-pair loads allowed
    FastDiv dimg, dtw;              // division by th * tw and by tw (tile coordinates)
    TapTables tab;
};

// Channels c0, c0+1 of pixel (img, hh, ww) as two sign-extended 16-bit
// lanes, zero outside the image and beyond Cin.
template <int LAYOUT>
__device__ __forceinline__ v2s load_pair(const int8_t* __restrict__ x, const K4Args& g, int img, int hh, int ww,
                                         int c0) {
    uint32_t u = 0;
    if (hh >= 0 && hh < g.h && ww >= 0 && ww < g.w && c0 < g.cin) {
        if (LAYOUT == WINO_NHWC) {
            const int8_t* p = x + (((long long)img * g.h + hh) * g.w + ww) * g.cin + c0;
            if (g.x_vec) u = *(const uint16_t*)p;
            else u = (uint32_t)(uint8_t)p[0] | (c0 + 1 < g.cin ? (uint32_t)(uint8_t)p[1] << 8 : 0u);
        } else {
            const long long hw = (long long)g.h * g.w;
            const int8_t* p = x + ((long long)img * g.cin + c0) * hw + (long long)hh * g.w + ww;
            u = (uint32_t)(uint8_t)p[0] | (c0 + 1 < g.cin ? (uint32_t)(uint8_t)p[hw] << 8 : 0u);
        }
    }
    // byte 0 -> high byte of lane 0, byte 1 -> high byte of lane 1, then an
    // arithmetic shift sign-extends both
    return __builtin_bit_cast(v2s, __builtin_amdgcn_perm(0u, u, 0x010c000cu)) >> splat(8);
}

template <int M, int LAYOUT, int EPI>
__global__ __launch_bounds__(K4_THREADS, K4Cfg<M>::WAVES_PER_EU) void wino_fused(const int8_t* __restrict__ x,
                                                                               const int8_t* __restrict__ uq,
                                                                               const int32_t* __restrict__ bias,
                                                                               int8_t* __restrict__ y, K4Args g) {
    using C = K4Cfg<M>;
    constexpr int N = C::N, NT = C::NT, G = C::G, NGRP = NT / G;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[C::LDS];
    uint8_t* const ldsB = lds;
    uint8_t* const ldsA = lds + C::B_BYTES;
    const int lbid = xcd_remap(blockIdx.x, g.nblocks);
    const int bco = lbid % g.nbco, btl = lbid / g.nbco;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int cw = wave & 3, tw = wave >> 2;
    const int lr = lane & 15, lk = lane >> 4;
    const int co_blk = bco * K4_CO;
    const long long tl_blk = (long long)btl * K4_TL;

    // this thread's transform items: (tile, channel pair) for it = tid and
    // tid + 512; item it covers tile it / 32 and channels 2 * (it % 32) + {0, 1}
    int it_img[2], it_ty[2], it_tx[2], it_off[2], it_c[2];
    bool it_ok[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int it = tid + K4_THREADS * k;
        const int tl = it >> 5, pr = it & 31;
        const long long tile = tl_blk + tl;
        it_ok[k] = tile < g.ntiles;
        const long long mt = it_ok[k] ? tile : 0;
        it_img[k] = (int)(mt / ((long long)g.th * g.tw));
        const int trem = (int)(mt - (long long)it_img[k] * g.th * g.tw);
        it_ty[k] = trem / g.tw;
        it_tx[k] = trem - it_ty[k] * g.tw;
        it_c[k] = 2 * pr;
        it_off[k] = tl * 64 + 16 * lds_slot(tl, (2 * pr) >> 4) + ((2 * pr) & 15);
    }

    // Uq ring: this wave's 1-KB load instructions per stage; load j copies
    // 16 rows (group j % 4) of the stage's tap j / 4
    const long long sa = (long long)g.cout_pad * g.cin_pad;   // tap stride
    const long long ka = (long long)g.cout_pad * kKStep;      // k-block stride
    const int8_t* src[C::LPW];
    int dst[C::LPW];
#pragma unroll
    for (int i = 0; i < C::LPW; ++i) {
        const int j = wave + K4_WAVES * i;
        const int u = j >> 2, row = 16 * (j & 3) + (lane >> 2);
        src[i] = uq + u * sa + (long long)(co_blk + row) * kKStep + 16 * lds_slot(row, lane & 3);
        dst[i] = j * 1024;
    }
    const int nkc = g.cin_pad / kKStep;
    const int nst = nkc * NGRP;
    auto issue = [&](int st) {
        const int kc = st / NGRP, grp = st - kc * NGRP;
        const long long off = (long long)(G * grp) * sa + kc * ka;
        uint8_t* base = ldsA + (st % K4_NBUF) * C::A_STAGE;
#pragma unroll
        for (int i = 0; i < C::LPW; ++i)
            __builtin_amdgcn_global_load_lds((const void*)(src[i] + off),
                                             (__attribute__((address_space(3))) void*)(base + dst[i]), 16, 0, 0);
    };

    const int row_a = 16 * cw + lr, row_b = 16 * tw + lr;
    const int frag_a = row_a * 64 + 16 * lds_slot(row_a, lk);
    const int frag_b = row_b * 64 + 16 * lds_slot(row_b, lk);

    v4i acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = (v4i){0, 0, 0, 0};

    issue(0);
    if (nst > 1) issue(1);
    for (int kc = 0; kc < nkc; ++kc) {
        // 1. input transform of this k step's 64 channels into the LDS Vq block
        // (one item at a time: only one window's registers live next to acc)
#pragma unroll 1
        for (int k = 0; k < 2; ++k) {
            v2s v[N][N];
#pragma unroll
            for (int r = 0; r < N; ++r)
#pragma unroll
                for (int c = 0; c < N; ++c)
                    v[r][c] = it_ok[k] ? load_pair<LAYOUT>(x, g, it_img[k], M * it_ty[k] - 1 + r, M * it_tx[k] - 1 + c,
                                                           kc * kKStep + it_c[k])
                                       : splat(0);
            const v2s two = splat(2), four = splat(4);
#pragma unroll
            for (int c = 0; c < N; ++c) {      // columns: B^T d
                v2s col[N], res[N];
#pragma unroll
                for (int r = 0; r < N; ++r) col[r] = v[r][c];
                Wino<M>::bt(col, res, two, four);
#pragma unroll
                for (int r = 0; r < N; ++r) v[r][c] = res[r];
            }
#pragma unroll
            for (int r = 0; r < N; ++r) {      // rows: (B^T d) B
                v2s res[N];
                Wino<M>::bt(v[r], res, two, four);
#pragma unroll
                for (int c = 0; c < N; ++c) v[r][c] = res[c];
            }
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int e = g.tab.eb[t];
                v2s q = (v[t / N][t % N] + splat(e ? (1 << (e - 1)) : 0)) >> splat(e);
                q = __builtin_elementwise_min(__builtin_elementwise_max(q, splat(-128)), splat(127));
                *(uint16_t*)(ldsB + t * K4_TL * 64 + it_off[k]) =
                    (uint16_t)__builtin_amdgcn_perm(0u, __builtin_bit_cast(uint32_t, q), 0x0c0c0200u);
            }
        }
        __syncthreads();
        // 2. the tap MFMAs of this k step
#pragma unroll
        for (int grp = 0; grp < NGRP; ++grp) {
            const int st = kc * NGRP + grp;
            if (st + 1 < nst) WINO_WAIT_VM(C::LPW);   // stage st done, st + 1 may be in flight
            else WINO_WAIT_VM(0);
            ring_barrier();
            if (st + 2 < nst) issue(st + 2);
            const uint8_t* abase = ldsA + (st % K4_NBUF) * C::A_STAGE;
#pragma unroll
            for (int u = 0; u < G; ++u) {
                const int t = G * grp + u;
                v4i av = *(const v4i*)(abase + frag_a + u * K4_CO * 64);
                v4i bv = *(const v4i*)(ldsB + frag_b + t * K4_TL * 64);
                acc[t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(av, bv, acc[t], 0, 0, 0);
            }
        }
        __syncthreads();   // every wave is done with this Vq block
    }
    tap_epilogue<M, LAYOUT, EPI, 0>(acc, g, bias, y, nullptr, co_blk + 16 * cw, tl_blk + 16 * tw, lane);
}

template <int M>
void launch_fused(wino_layout layout, int epi_bits, dim3 grid, dim3 block, hipStream_t stream, const int8_t* x,
                  const wino_f4_plan_s* p, int8_t* y, const K4Args& a) {
    if (layout == WINO_NHWC) {
        if (epi_bits == 32)
            hipLaunchKernelGGL((wino_fused<M, WINO_NHWC, 32>), grid, block, 0, stream, x, p->uq_dev, p->bias_dev, y, a);
        else
            hipLaunchKernelGGL((wino_fused<M, WINO_NHWC, 64>), grid, block, 0, stream, x, p->uq_dev, p->bias_dev, y, a);
    } else {
        if (epi_bits == 32)
            hipLaunchKernelGGL((wino_fused<M, WINO_NCHW, 32>), grid, block, 0, stream, x, p->uq_dev, p->bias_dev, y, a);
        else
            hipLaunchKernelGGL((wino_fused<M, WINO_NCHW, 64>), grid, block, 0, stream, x, p->uq_dev, p->bias_dev, y, a);
    }
}

}  // namespace

wino_status wino_f4_conv_fused(const wino_f4_plan_s* p, const int8_t* x, int8_t* y, int n, int h, int w,
                               wino_layout layout, hipStream_t stream) {
    K4Args a;
    a.cin = p->cin;
    a.cin_pad = p->cin_pad;
    a.cout = p->cout;
    a.cout_pad = p->cout_pad;
    a.n = n;
    a.h = h;
    a.w = w;
    const int m = p->m;
    a.th = (h + m - 1) / m;
    a.tw = (w + m - 1) / m;
    a.ntiles = (long long)n * a.th * a.tw;
    if (a.ntiles == 0) return WINO_OK;
    a.dimg = make_fastdiv((uint32_t)(a.th * a.tw));
    a.dtw = make_fastdiv((uint32_t)a.tw);
    a.nbco = p->cout_pad / K4_CO;
    const long long blocks = (a.ntiles + K4_TL - 1) / K4_TL * a.nbco;
    if (blocks > 0x7fffffffll) return WINO_EUNSUPPORTED;
    a.nblocks = (int)blocks;
    a.out_shift = p->out_shift;
    a.relu = p->relu;
    a.x_vec = layout == WINO_NHWC && p->cin % 2 == 0 && ((uintptr_t)x & 1) == 0;
    for (int i = 0; i < kTaps; ++i) {
        a.tab.eb[i] = p->e_b[i];
        a.tab.sh[i] = p->sh[i];
    }
    dim3 grid((unsigned)blocks), block(K4_THREADS);
    if (m == 4) launch_fused<4>(layout, p->epi_bits, grid, block, stream, x, p, y, a);
    else launch_fused<2>(layout, p->epi_bits, grid, block, stream, x, p, y, a);
    return hipGetLastError() == hipSuccess ? WINO_OK : WINO_EHIP;
}
