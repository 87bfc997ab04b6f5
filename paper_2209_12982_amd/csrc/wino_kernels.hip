// Online path of integer Winograd F(4x4,3x3) with tap-wise power-of-two
// quantization (Sec. III), for gfx950.
//
//   K1 wino_input_xform   6x6 input tiles (stride 4, halo band staged in LDS),
//                         V = B^T d B in packed 16-bit integer lanes (the
//                         separable row-by-row form of Eq. general_wino_xform
//                         with shared subexpressions, Sec. IV-B1), tap-wise
//                         requantization R(V / 2^e_B) clamped to int8, and a
//                         tap-major scatter into Vq[36][Cin/64][tiles][64]
//                         (k-blocked: 64 input channels contiguous per tile,
//                         the "fractal" C1/C0 split of Sec. IV-A).
//   K2 wino_tap_gemm      36 int8 GEMMs M_t = Uq_t * Vq_t on MFMA with int32
//                         accumulation; the epilogue aligns taps by 2^sh,
//                         applies Y = A^T M A, adds bias, requantizes and
//                         stores int8 (Sec. III rearranged scheme; the
//                         out_xform / dconv / write steps of the operator
//                         dataflow, Sec. IV-B2).
//
// Bit exactness: all arithmetic is integer.  B^T d B of int8 data is at most
// 12768 in magnitude and every intermediate of its row pass at most 1278, so
// 16-bit lanes hold it (with a rounding constant of at most 2^14 added).  The
// GEMM sums |Vq Uq| <= 2^14 per input channel in int32.  The output transform
// runs in 32-bit integers when the plan's bound proves every partial sum fits,
// otherwise in 64-bit.
#include <algorithm>
#include <atomic>
#include <mutex>
#include "wino_device.h"

using namespace winof4;

namespace {

// ---------------------------------------------------------------------------
// K1: input transform
// ---------------------------------------------------------------------------
// tiles per block along x (TX below): 16, one thread per (tile, 4 channels).
// Blocks of 20 tiles would leave no idle tiles in a row of 40 (C5: three
// blocks of 16, the third half empty), but measured slower there (24.3 against
// 23.3 us).
constexpr int K1_TX = 16;
constexpr int K1_CG = 64;               // channels per block
constexpr int K1_CS = 20;               // LDS words per pixel (16 used, 4 pad)
// halo band of a block: M + 2 rows x (M * TX + 2) pixels
template <int M, int TX>
struct K1Band {
    static constexpr int ROWS = M + 2, COLS = M * TX + 2, THREADS = 16 * TX;
};


struct K1Args {
    int n, cin, h, w, th, tw, cin_pad;
    int ntxb, ncg;
    int x_vec;                          // 16-byte loads allowed (Cin % 16 == 0, x aligned)
    int x_dw;                           // NCHW word loads allowed (W % 4 == 0, x aligned, image < 2 GiB)
    int vq_buf;                         // tap planes below 4 GiB: buffer stores with a scalar base
    long long t_pad;                    // tile stride of a tap plane in Vq
    long long plane_bytes;              // bytes of one tap plane of Vq
    TapTables tab;
    uint32_t rnd2[kTaps];               // 2^(e_B - 1) (0 for e_B = 0) in both 16-bit halves
    int q_sat;                          // every e_B <= 16 - Q: one-instruction requantization
    int* sk_cnt;                        // stream-K counters of the tap GEMM that follows, zeroed
    int sk_ncnt;                        //   by workgroup 0 (MODE 0; none when sk_ncnt is 0)
};

// zero the stream-K counters of the tap GEMM that reads this Vq (workgroup 0)
__device__ __forceinline__ void k1_zero_counters(const K1Args& g) {
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i < g.sk_ncnt; i += blockDim.x) g.sk_cnt[i] = 0;
}

// Requantize the tile's taps and store them to the tap planes of Vq at byte
// offset off (see the kernel); SAT: the one-instruction saturating form.
// The saturating form takes 2^(16-Q-e) (a scalar per tap) and 2^(15-Q) as
// the addend for every tap: for e = 0 that adds half a unit below the kept
// bits, which leaves the floor of an integer unchanged.
template <int N, int Q, bool SAT>
__device__ __forceinline__ void k1_store(const v2s (&ev)[N][N], const v2s (&od)[N][N], const K1Args& g,
                                         int8_t* __restrict__ vq, long long off) {
    constexpr int NT = N * N;
    constexpr uint32_t kAdd2 = (1u << (15 - Q)) * 0x10001u;
    auto scale2 = [&](int t) { return (1u << (16 - Q - g.tab.eb[t])) * 0x10001u; };
    if (g.vq_buf) {
        // per tap a buffer resource on the tap plane (scalar base and size)
        // and one 32-bit lane offset for all taps
        const int voff = (int)off;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const __amdgpu_buffer_rsrc_t rs =
                __builtin_amdgcn_make_buffer_rsrc(vq + t * g.plane_bytes, 0, (int)g.plane_bytes, 0x00020000);
            if constexpr (Q == 10) {
                const uint2 v = SAT ? requant10_pack_sat(ev[t / N][t % N], od[t / N][t % N], scale2(t), kAdd2)
                                    : requant10_pack(ev[t / N][t % N], od[t / N][t % N], g.tab.eb[t], g.rnd2[t]);
                __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(v2u, v), rs, voff, 0, 0);
            } else {
                const uint32_t v = SAT ? requant_pack_sat(ev[t / N][t % N], od[t / N][t % N], scale2(t), kAdd2)
                                       : requant_pack(ev[t / N][t % N], od[t / N][t % N], g.tab.eb[t], g.rnd2[t]);
                __builtin_amdgcn_raw_buffer_store_b32(v, rs, voff, 0, 0);
            }
        }
    } else {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            int8_t* dst = vq + t * g.plane_bytes + off;
            if constexpr (Q == 10)
                *(uint2*)dst = SAT ? requant10_pack_sat(ev[t / N][t % N], od[t / N][t % N], scale2(t), kAdd2)
                                   : requant10_pack(ev[t / N][t % N], od[t / N][t % N], g.tab.eb[t], g.rnd2[t]);
            else
                *(uint32_t*)dst = SAT ? requant_pack_sat(ev[t / N][t % N], od[t / N][t % N], scale2(t), kAdd2)
                                      : requant_pack(ev[t / N][t % N], od[t / N][t % N], g.tab.eb[t], g.rnd2[t]);
        }
    }
}

// Stage the halo band of one block into LDS as [row][col][channel] bytes
// (channel fastest, K1_CS words per pixel).  Rows M ty - 1 .. M ty + M,
// columns M tx0 - 1 .. M (tx0 + TX), channels ci0 .. ci0+63; zero outside
// the image and beyond Cin.
template <int M, int LAYOUT, int TX>
__device__ __forceinline__ void k1_stage_band(uint32_t* lds, const int8_t* __restrict__ x,
                                              const K1Args& g, int img, int ty, int tx0, int ci0) {
    constexpr int ROWS = K1Band<M, TX>::ROWS, COLS = K1Band<M, TX>::COLS, THREADS = K1Band<M, TX>::THREADS;
    const int h0 = M * ty - 1, w0 = M * tx0 - 1;
    if (LAYOUT == WINO_NHWC) {
        for (int id = threadIdx.x; id < ROWS * COLS * 4; id += THREADS) {
            int pix = id >> 2, part = id & 3;
            int r = pix / COLS, c = pix - r * COLS;
            int hh = h0 + r, ww = w0 + c, cb = ci0 + 16 * part;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (hh >= 0 && hh < g.h && ww >= 0 && ww < g.w && cb < g.cin) {
                const int8_t* src = x + (((long long)img * g.h + hh) * g.w + ww) * g.cin + cb;
                if (g.x_vec) {
                    v = *(const uint4*)src;
                } else {
                    uint32_t wv[4] = {0, 0, 0, 0};
                    for (int k = 0; k < 16; ++k)
                        if (cb + k < g.cin) wv[k >> 2] |= (uint32_t)(uint8_t)src[k] << (8 * (k & 3));
                    v = make_uint4(wv[0], wv[1], wv[2], wv[3]);
                }
            }
            *(uint4*)(lds + pix * K1_CS + 4 * part) = v;
        }
    } else if (g.x_dw) {
        // NCHW with W % 4 == 0: an item moves 4 channels x 8 band columns of
        // one band row.  The band starts at column M tx0 - 1, so a group of
        // eight columns straddles three aligned words of each channel's image
        // row: three word loads and two byte alignments per channel, then two
        // 4x4 byte transposes (the four channels of a column into one word)
        // and eight LDS word stores.  A word left or right of the image row,
        // in a row outside the image or of a channel >= Cin gets an offset
        // past the image's bytes and reads as zero (with W % 4 == 0 a word is
        // either wholly inside a row or wholly outside it).
        constexpr int NG = (COLS + 7) / 8;
        constexpr int kOut = 0x7ffffff0;  // >= the image's bytes (checked on the host)
        const int img_bytes = g.cin * g.h * g.w;
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void*)(x + (long long)img * img_bytes), 0, img_bytes, 0x00020000);
        for (int id = threadIdx.x; id < 16 * ROWS * NG; id += THREADS) {
            const int gc = id % NG;
            const int rest = id / NG;
            const int r = rest % ROWS, cq = rest / ROWS;
            const int hh = h0 + r;
            const int cc = w0 + 8 * gc;           // first column of the group
            const int a = cc >> 2;                // its word (floor), then the next two
            const int sh = cc & 3;                // byte offset of the group in word a
            const bool rok = hh >= 0 && hh < g.h;
            const bool ok0 = rok && a >= 0 && 4 * a < g.w;
            const bool ok1 = rok && a + 1 >= 0 && 4 * (a + 1) < g.w;
            const bool ok2 = rok && a + 2 >= 0 && 4 * (a + 2) < g.w;
            const int hr = rok ? hh : 0;
            uint32_t v[2][4];
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const int ci = ci0 + 4 * cq + kk;
                const bool cok = ci < g.cin;
                const int base = ((cok ? ci : 0) * g.h + hr) * g.w + 4 * a;
                const uint32_t w0_ = __builtin_amdgcn_raw_buffer_load_b32(rs, cok && ok0 ? base : kOut, 0, 0);
                const uint32_t w1_ = __builtin_amdgcn_raw_buffer_load_b32(rs, cok && ok1 ? base + 4 : kOut, 0, 0);
                const uint32_t w2_ = __builtin_amdgcn_raw_buffer_load_b32(rs, cok && ok2 ? base + 8 : kOut, 0, 0);
                v[0][kk] = __builtin_amdgcn_alignbyte(w1_, w0_, (uint32_t)sh);
                v[1][kk] = __builtin_amdgcn_alignbyte(w2_, w1_, (uint32_t)sh);
            }
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                // v[hf][k] byte j = channel k, column 4 hf + j  ->  col[j] byte k
                const uint32_t ab_lo = __builtin_amdgcn_perm(v[hf][1], v[hf][0], 0x05010400u);
                const uint32_t ab_hi = __builtin_amdgcn_perm(v[hf][1], v[hf][0], 0x07030602u);
                const uint32_t cd_lo = __builtin_amdgcn_perm(v[hf][3], v[hf][2], 0x05010400u);
                const uint32_t cd_hi = __builtin_amdgcn_perm(v[hf][3], v[hf][2], 0x07030602u);
                const uint32_t col[4] = {__builtin_amdgcn_perm(cd_lo, ab_lo, 0x05040100u),
                                         __builtin_amdgcn_perm(cd_lo, ab_lo, 0x07060302u),
                                         __builtin_amdgcn_perm(cd_hi, ab_hi, 0x05040100u),
                                         __builtin_amdgcn_perm(cd_hi, ab_hi, 0x07060302u)};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int c = 8 * gc + 4 * hf + j;
                    if (c < COLS) lds[(r * COLS + c) * K1_CS + cq] = col[j];
                }
            }
        }
    } else {
        uint8_t* lb = (uint8_t*)lds;
        for (int id = threadIdx.x; id < K1_CG * ROWS * COLS; id += THREADS) {
            int c = id % COLS;
            int rest = id / COLS;
            int r = rest % ROWS, ch = rest / ROWS;
            int hh = h0 + r, ww = w0 + c, ci = ci0 + ch;
            int8_t v = 0;
            if (hh >= 0 && hh < g.h && ww >= 0 && ww < g.w && ci < g.cin)
                v = x[(((long long)img * g.cin + ci) * g.h + hh) * g.w + ww];
            lb[(r * COLS + c) * K1_CS * 4 + ch] = (uint8_t)v;
        }
    }
}

// MODE 0: write Vq.  MODE 1: per-tap max |V| into tapmax[NTAP] (calibration).
// Q: Winograd-domain width, 8 (int8 Vq) or 10 (int8/10: fp16 Vq holding
// 10-bit integers, [ntap][cin_pad/32][t_pad][32]).
// SAT: requantize with the one-instruction saturating form (every e_B <=
// 16 - Q), a kernel of its own so the other form's per-tap constants are not
// held in scalar registers too.
template <int M, int LAYOUT, int MODE, int Q = 8, int TX = K1_TX, bool SAT = false>
__global__ __launch_bounds__(16 * TX, 5) void wino_input_xform(const int8_t* __restrict__ x,
                                                               int8_t* __restrict__ vq,
                                                               int* __restrict__ tapmax, K1Args g) {
    constexpr int N = Wino<M>::N, NT = Wino<M>::NTAP;
    constexpr int COLS = K1Band<M, TX>::COLS;
    __shared__ uint32_t band[K1Band<M, TX>::ROWS * COLS * K1_CS];
    __shared__ int red[NT];
    // Logical block order: channel group fastest, then tile-column block,
    // then tile row; consecutive logical ids are kept on one XCD (its L2),
    // so the channel groups sharing each 128-byte line of an NHWC pixel and
    // the tile rows sharing halo rows are read by concurrent workgroups.
    if constexpr (MODE == 0) k1_zero_counters(g);
    int bid = xcd_remap((int)blockIdx.x, (int)gridDim.x);
    const int cgi = bid % g.ncg;
    bid /= g.ncg;
    const int txb = bid % g.ntxb;
    const int row = bid / g.ntxb;         // img * th + ty
    const int img = row / g.th, ty = row - img * g.th;
    const int tx0 = txb * TX, ci0 = cgi * K1_CG;
    if (MODE == 1 && threadIdx.x < NT) red[threadIdx.x] = 0;

    k1_stage_band<M, LAYOUT, TX>(band, x, g, img, ty, tx0, ci0);
    __syncthreads();

    // thread -> (tile j, channel quad q): 16 quads x 16 tiles
    const int q = threadIdx.x & 15;
    const int j = threadIdx.x >> 4;
    const int tx = tx0 + j;
    const bool valid = tx < g.tw;

    uint32_t wv[N][N];
#pragma unroll
    for (int r = 0; r < N; ++r)
#pragma unroll
        for (int c = 0; c < N; ++c) wv[r][c] = band[(r * COLS + M * j + c) * K1_CS + q];
    v2s ev[N][N], od[N][N];
    input_tile_transform<M>(wv, ev, od);

    if (MODE == 0) {
        if (!valid) return;
        const long long tile = (long long)row * g.tw + tx;
        // byte offset of this thread's values within a tap plane:
        //   Q = 8:  Vq[t][cgi][tile][64], 4 bytes (channels 4q .. 4q + 3)
        //   Q = 10: Vq[t][2 cgi + q / 8][tile][32] fp16 (this block's 64
        //           channels are the 32-channel k rows 2 cgi and 2 cgi + 1),
        //           8 bytes (4 halves)
        const long long off = Q == 10 ? (((long long)(2 * cgi + (q >> 3)) * g.t_pad + tile) * 32 + 4 * (q & 7)) * 2
                                      : ((long long)cgi * g.t_pad + tile) * K1_CG + 4 * q;
        k1_store<N, Q, SAT>(ev, od, g, vq, off);
    } else {
        if (valid) {
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                v2s a = ev[t / N][t % N], b = od[t / N][t % N];
                a = __builtin_elementwise_max(a, -a);
                b = __builtin_elementwise_max(b, -b);
                int m = max(max((int)a.x, (int)a.y), max((int)b.x, (int)b.y));
                atomicMax(&red[t], m);
            }
        }
        __syncthreads();
        if (threadIdx.x < NT) atomicMax(&tapmax[threadIdx.x], red[threadIdx.x]);
    }
}

// K1 for NHWC input without the LDS band: each thread reads its tile's
// (M+2) x (M+2) pixels x 4 channels straight from global memory (L1 and L2
// serve the halo that neighbouring tiles share).  Row r of the patch goes
// through a buffer resource on that image row (num_records: the row's bytes,
// 0 above or below the image) and column c through a per-lane offset (past
// the row's end left or right of the image, for idle tiles and for channels
// >= Cin), so pixels outside the image read as zero with no arithmetic per
// load.  No LDS and no barrier: one wave's loads overlap other waves'
// arithmetic.  Needs Cin % 4 == 0 (whole 4-channel words), a 4-byte aligned
// x and image rows below 2 GiB.
// TX = 16 or 8 tiles per block (256 or 128 threads), 20 waves per CU either
// way; the launch takes the width that leaves fewer idle tiles at the end of
// a tile row (C5's rows of 40 tiles: 8, measured 16.6 -> 15.0 us).
template <int M, int Q, int TX, bool SAT>
__global__ __launch_bounds__(16 * TX, 80 / TX) void wino_input_xform_nhwc(const int8_t* __restrict__ x,
                                                                    int8_t* __restrict__ vq, K1Args g) {
    constexpr int N = Wino<M>::N;
    k1_zero_counters(g);
    // the block order of wino_input_xform
    int bid = xcd_remap((int)blockIdx.x, (int)gridDim.x);
    const int cgi = bid % g.ncg;
    bid /= g.ncg;
    const int txb = bid % g.ntxb;
    const int row = bid / g.ntxb;         // img * th + ty
    const int img = row / g.th, ty = row - img * g.th;
    const int q = threadIdx.x & 15, j = threadIdx.x >> 4;
    const int tx = txb * TX + j;
    const int ci = cgi * K1_CG + 4 * q;
    const bool lane_ok = tx < g.tw && ci < g.cin;
    const int row_bytes = g.w * g.cin;
    constexpr int kOut = 0x7ffffff0;      // >= any row's num_records
    int coff[N];
#pragma unroll
    for (int c = 0; c < N; ++c) {
        const int xx = M * tx - 1 + c;
        coff[c] = (lane_ok && xx >= 0 && xx < g.w) ? xx * g.cin + ci : kOut;
    }
    uint32_t wv[N][N];
#pragma unroll
    for (int r = 0; r < N; ++r) {
        const int yy = M * ty - 1 + r;
        const bool rok = yy >= 0 && yy < g.h;
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void*)(x + (rok ? ((long long)img * g.h + yy) * row_bytes : 0)), 0, rok ? row_bytes : 0, 0x00020000);
#pragma unroll
        for (int c = 0; c < N; ++c) wv[r][c] = __builtin_amdgcn_raw_buffer_load_b32(rs, coff[c], 0, 0);
    }
    v2s ev[N][N], od[N][N];
    input_tile_transform<M>(wv, ev, od);
    if (tx >= g.tw) return;
    const long long tile = (long long)row * g.tw + tx;
    const long long off = Q == 10 ? (((long long)(2 * cgi + (q >> 3)) * g.t_pad + tile) * 32 + 4 * (q & 7)) * 2
                                  : ((long long)cgi * g.t_pad + tile) * K1_CG + 4 * q;
    k1_store<N, Q, SAT>(ev, od, g, vq, off);
}

// ---------------------------------------------------------------------------
// K2: tap GEMM with fused output transform
// ---------------------------------------------------------------------------
// Workgroup = CW x TW waves computing 16*CW output channels x 16*TW tiles for
// all 36 taps; wave w owns channels 16*(w%CW).. and tiles 16*(w/CW).. (one
// 16x16 int8 MFMA block per tap, 36 x 4 int32 accumulators per lane).  The k
// loop runs over input channels in steps of 64; each step is split into
// three tap groups ("stages").  A stage's Uq slice (12 taps x 16*CW rows x
// 64 B) and Vq slice (12 taps x 16*TW rows x 64 B) are copied global -> LDS
// by the direct-to-LDS load (no VGPR staging) into a ring of NBUF stages, so
// NBUF - 1 stages load while one feeds the MFMAs.  Every such load writes
// 1 KB of LDS contiguously (16 bytes per lane); the 16-byte slot of a row
// holding input bytes [16p, 16p+16) is p ^ ((row >> 1) & 3).  Measured on
// gfx950, this swizzle lets the fragment reads (16 rows x one 16-byte part
// per 16 lanes) run at the full 256 B/clk per CU; unswizzled or padded rows
// run 1.5x slower.
//
// Three block shapes: 64x32 (8 waves, double buffer), the default; 32x32
// (4 waves) and 16x16 (one wave) with 6-tap stages and rings small enough for
// two and four workgroups per CU, selectable for small layers.
template <int CW_, int TW_, int G_, int NBUF_, int PF_ = G_ / 2>
struct K2Cfg {
    static constexpr int CW = CW_, TW = TW_, G = G_, NBUF = NBUF_;   // G: taps per stage
    static constexpr int CO = 16 * CW, TL = 16 * TW;
    static constexpr int WAVES = CW * TW, THREADS = 64 * WAVES;
    static constexpr int A_BYTES = G * CO * 64, B_BYTES = G * TL * 64;
    static constexpr int STAGE = A_BYTES + B_BYTES;
    static constexpr int KB = STAGE / 1024;              // 1-KB load instructions per stage
    static constexpr int LPW = (KB + WAVES - 1) / WAVES; // load instructions per wave per stage
    static constexpr int PF = PF_;                       // taps whose LDS fragments are in flight ahead
    static_assert(NBUF * STAGE <= 160 * 1024, "LDS");
    static_assert((NBUF - 2) * LPW <= 63, "vmcnt range");
    static_assert(G > PF, "stage shape");
};
// 64 x 32, one workgroup per CU; 32 x 32 and 16 x 16 with rings small
// enough for two and four workgroups per CU
using K2Big = K2Cfg<4, 2, 12, 2>;
using K2Mid = K2Cfg<2, 2, 6, 3>;
using K2Small = K2Cfg<1, 1, 6, 3>;
// F(2x2,3x3): 16 taps in two 8-tap stages per k step, 64 x 32 blocks
using K2F2 = K2Cfg<4, 2, 8, 3>;
// int8/10 (fp16 operands): shallower fragment prefetch, as each fp16 MFMA
// result also needs registers until it is
// folded into the int32 accumulator (64x32 keeps a one-tap prefetch; with
// the 64-bit epilogue only the 32x32 shape stays clear of spills)
using K2Big10 = K2Cfg<4, 2, 12, 2, 1>;
using K2Mid10 = K2Cfg<2, 2, 12, 2, 2>;
using K2Small10 = K2Cfg<2, 2, 6, 2, 2>;   // 48 KB of LDS: two workgroups per CU
using K2F2_10 = K2Cfg<4, 2, 8, 3, 2>;

struct K2Args {
    int cin_pad, cout, cout_pad;
    int n, h, w, th, tw;
    long long ntiles, t_pad;
    int nbco, nblocks;
    int out_shift, relu;
    int y_staged;              // row-streamed kernel: stage NHWC output through LDS
    int n_dp;                  // row-streamed kernel: blocks run whole; the rest are split
    int sk_groups;             // stream-K workgroups sharing the split blocks (0: none)
    int sk_units;              // stages of the split blocks: their count x 6 cin_pad / 64
    int* sk_cnt;               // per split block: pieces counted (zero between launches)
    int* sk_part;              // partial Y, two slots of KR_SLOT int32 per stream-K workgroup
    FastDiv dimg, dtw;         // division by th * tw and by tw (tile coordinates)
    TapTables tab;
    uint32_t shrow[6];         // sh of row a's six taps, 5 bits each (wave-specialized kernel)
};

// MODE 0: store y.  MODE 1: max |Y + bias| into *zmax (calibration).
// MODE 2: store raw M (debug export).
// Q = 8: int8 operands, 16x16x64 int8 MFMA.  Q = 10 (int8/10): fp16 operands
// holding 10-bit integers, 32 channels per 64-byte k row (g.cin_pad counts
// k-row bytes, i.e. twice the channels), 16x16x32 fp16 MFMA.  Each fp16 MFMA
// starts from zero: its 32 products and their partial sums are integers of
// magnitude <= 32 * 2^18 = 2^23, so the fp32 result is exact, and it is
// converted and added to the int32 accumulator right away.
template <class C, int M, int LAYOUT, int EPI, int MODE, int Q = 8>
__global__ __launch_bounds__(C::THREADS) void wino_tap_gemm(const int8_t* __restrict__ uq,
                                                            const int8_t* __restrict__ vq,
                                                            const int32_t* __restrict__ bias,
                                                            int8_t* __restrict__ y,
                                                            void* __restrict__ aux, K2Args g) {
    __shared__ __attribute__((aligned(1024))) uint8_t lds[C::NBUF * C::STAGE];
    const int lbid = xcd_remap(blockIdx.x, g.nblocks);
    const int bco = lbid % g.nbco, btl = lbid / g.nbco;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int cw = wave % C::CW, tw = wave / C::CW;
    const int co_blk = bco * C::CO;
    const long long tl_blk = (long long)btl * C::TL;
    const int co_base = co_blk + 16 * cw;
    const long long tl_base = tl_blk + 16 * tw;
    const int lr = lane & 15, lk = lane >> 4;
    // k-blocked operands: Uq[36][cin_pad/64][cout_pad][64], Vq[36][cin_pad/64][t_pad][64]
    const long long sa = (long long)g.cout_pad * g.cin_pad;   // tap stride of Uq
    const long long sb = g.t_pad * g.cin_pad;                  // tap stride of Vq
    const long long ka = (long long)g.cout_pad * kKStep;      // k-block stride of Uq
    const long long kb = g.t_pad * kKStep;                     // k-block stride of Vq

    // This wave's 1-KB load instructions of a stage: global source of this
    // lane (stage 0) and LDS destination offset within a stage buffer.
    // Each load instruction covers 16 rows x 64 B; a lane's byte offset within
    // those 1 KB is the same for every instruction of the wave (the swizzle
    // depends on the row only through bits that are equal across the 16-row
    // groups), so the addresses are a wave-uniform base (scalar registers)
    // plus one 32-bit lane offset.
    const int wv_id = __builtin_amdgcn_readfirstlane(wave);
    const int rr = lane >> 2;
    const int lane_off = rr * 64 + 16 * lds_slot(rr, lane & 3);
    long long ubase[C::LPW];
    int dst[C::LPW];
    bool isa[C::LPW];
#pragma unroll
    for (int i = 0; i < C::LPW; ++i) {
        // when the stage's loads do not split evenly, the last round repeats
        // an earlier load (same bytes to the same place)
        int j = wv_id + C::WAVES * i;
        if (j >= C::KB) j -= C::WAVES;
        isa[i] = j < C::A_BYTES / 1024;
        if (isa[i]) {
            const int u = j / C::CW, q = j % C::CW;
            ubase[i] = u * sa + (long long)(co_blk + 16 * q) * kKStep;
        } else {
            const int jj = j - C::A_BYTES / 1024;
            const int u = jj / C::TW, q = jj % C::TW;
            ubase[i] = u * sb + (tl_blk + 16 * q) * kKStep;
        }
        dst[i] = j * 1024;
    }
    constexpr int NT = Wino<M>::NTAP;
    static_assert(NT % C::G == 0, "stages split the taps evenly");
    constexpr int GPS = NT / C::G;                     // stages per k-chunk
    const int nkc = g.cin_pad / kKStep;
    const int nstage = nkc * GPS;
    auto issue = [&](int st) {
        const int kc = st / GPS, grp = st - kc * GPS;
        uint8_t* base = lds + (st % C::NBUF) * C::STAGE;
#pragma unroll
        for (int i = 0; i < C::LPW; ++i) {
            const long long off = ubase[i] + (long long)(C::G * grp) * (isa[i] ? sa : sb) + kc * (isa[i] ? ka : kb);
            // Vq is streamed once per output-channel block: non-temporal, so it
            // does not push the small, hot Uq out of L2
            if (isa[i])
                __builtin_amdgcn_global_load_lds((const void*)(uq + off + lane_off),
                                                 (__attribute__((address_space(3))) void*)(base + dst[i]), 16, 0, 0);
            else
                __builtin_amdgcn_global_load_lds((const void*)(vq + off + lane_off),
                                                 (__attribute__((address_space(3))) void*)(base + dst[i]), 16, 0, 2);
        }
    };

    v4i acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = (v4i){0, 0, 0, 0};

    // fragment offsets within a stage buffer (tap u adds u * rows * 64)
    const int row_a = 16 * cw + lr, row_b = 16 * tw + lr;
    const int frag_a = row_a * 64 + 16 * lds_slot(row_a, lk);
    const int frag_b = C::A_BYTES + row_b * 64 + 16 * lds_slot(row_b, lk);

    for (int st = 0; st < C::NBUF - 1 && st < nstage; ++st) issue(st);
    for (int kc = 0; kc < nkc; ++kc) {
#pragma unroll
        for (int grp = 0; grp < GPS; ++grp) {
            const int st = kc * GPS + grp;
            // stage st has landed once only the stages issued after it are
            // pending: min(NBUF - 2, nstage - 1 - st) of them, LPW loads each
            const int ahead = min(C::NBUF - 2, nstage - 1 - st);
            if (C::NBUF >= 4 && ahead >= 2)
                WINO_WAIT_VM_LDS(2 * C::LPW);
            else if (C::NBUF >= 3 && ahead >= 1)
                WINO_WAIT_VM_LDS(C::LPW);
            else
                WINO_WAIT_VM_LDS(0);
            ring_barrier();                              // stage st visible; stage st-1 consumed
            if (st + C::NBUF - 1 < nstage) issue(st + C::NBUF - 1);
            const uint8_t* base = lds + (st % C::NBUF) * C::STAGE;
            // software pipeline over the stage's taps: fragments of PF taps
            // are in flight ahead of the MFMA that consumes the oldest, so the
            // LDS read latency hides behind MFMAs
            v4i fa[C::PF], fb[C::PF];
#pragma unroll
            for (int u = 0; u < C::PF; ++u) {
                fa[u] = *(const v4i*)(base + frag_a + u * C::CO * 64);
                fb[u] = *(const v4i*)(base + frag_b + u * C::TL * 64);
            }
#pragma unroll
            for (int u = 0; u < C::G; ++u) {
                const int slot = u % C::PF;
                if constexpr (Q == 10) {
                    const v4f r = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                        __builtin_bit_cast(v8h, fa[slot]), __builtin_bit_cast(v8h, fb[slot]), (v4f){0.f, 0.f, 0.f, 0.f},
                        0, 0, 0);
                    // unsigned (wrapping) add: with a signed add the compiler
                    // may carry the accumulators in 64 bits for the int64
                    // epilogue (overflow being undefined), doubling them
                    acc[C::G * grp + u] = __builtin_bit_cast(
                        v4i, __builtin_bit_cast(v4u, acc[C::G * grp + u]) +
                                 __builtin_bit_cast(v4u, __builtin_convertvector(r, v4i)));
                } else {
                    acc[C::G * grp + u] =
                        __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[slot], fb[slot], acc[C::G * grp + u], 0, 0, 0);
                }
                if (u + C::PF < C::G) {
                    fa[slot] = *(const v4i*)(base + frag_a + (u + C::PF) * C::CO * 64);
                    fb[slot] = *(const v4i*)(base + frag_b + (u + C::PF) * C::TL * 64);
                }
            }
            // keep that order: the scheduler would otherwise pull the reads
            // next to their MFMAs to save registers (masks: 0x100 LDS read,
            // 0x008 MFMA, 0x002 VALU).  With fp16 operands each MFMA is
            // followed by the eight VALU ops that fold an earlier result into
            // the int32 accumulators, so at most a few results are live.
            __builtin_amdgcn_sched_group_barrier(0x100, 2 * C::PF, 0);
#pragma unroll
            for (int u = 0; u < C::G - C::PF; ++u) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
                if constexpr (Q == 10) __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
            }
#pragma unroll
            for (int u = 0; u < C::PF; ++u) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                if constexpr (Q == 10) __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
            }
        }
    }

    tap_epilogue<M, LAYOUT, EPI, MODE>(acc, g, bias, y, aux, co_base, tl_base, lane);
}

// ---------------------------------------------------------------------------
// K2R wino_tap_gemm_rows: the same contraction with the output transform
// folded in row by row.
//
// Y = A^T M' A is linear in the taps, and its row pass only mixes the six
// taps of one row a of the 6x6 tile: Y = sum_a A^T[:, a] (M'[a, :] A).  So the
// GEMM can stream the taps row by row: accumulate the six M_t of row a over
// all input channels, fold them into Y (row pass on the six values, then the
// rank-one update with column a of A^T), and reuse the six accumulators for
// the next row.  Per (tile, channel) pair that keeps 16 + 6 values live
// instead of 36, which buys a 64 x 64 block per workgroup (half the L2 ->
// LDS operand traffic per MAC of the 64 x 32 block above) and spreads the
// output transform over the main loop instead of a serial epilogue.
//
// Ring stage = one row a and one 64-channel k-chunk: six (tap, chunk) slices
// of 64 Uq rows + 64 Vq rows, 8 KB each; three stages rotate through 144 KB
// of LDS, two in flight.  The 16 waves form 4 (channels) x 4 (tiles), one
// 16x16x64 MFMA block each: 16 + 6 values per pair is 88 registers a lane,
// which fits the 128 a wave has at four waves per SIMD.  (Two blocks per
// wave at eight waves would need 176 of 256 and the compiler spills.)
// A slice is 8 groups of 16 rows; wave w copies group w % 8 of the slices
// b = w / 8, w / 8 + 2, w / 8 + 4 (groups 0-3: Uq, 4-7: Vq), so its loads
// never branch.
//
// Integer arithmetic is exact: the int32 epilogue is only selected when the
// plan bound, which also bounds every partial sum of the folds, is < 2^31.
// ---------------------------------------------------------------------------
constexpr int KR_CO = 64;
constexpr int KR_TL = 64;
constexpr int KR_CHUNK = (KR_CO + KR_TL) * kKStep;      // one tap, one k-chunk
constexpr int KR_STAGE = 6 * KR_CHUNK;                  // one row of taps
constexpr int KR_NBUF = 3;
constexpr int KR_TB = 1;                                // 16x16 tile blocks per wave
constexpr int KR_WAVES = 16 / KR_TB;
constexpr int KR_THREADS = 64 * KR_WAVES;
constexpr int KR_LPW = KR_STAGE / 1024 / KR_WAVES;      // 1-KB loads per wave per stage
static_assert((KR_CO + KR_TL) / 16 == 8 && KR_WAVES % 8 == 0, "wave -> (row group, slices) map");
static_assert((KR_CO / 16) * (KR_TL / 16) == KR_WAVES * KR_TB, "the waves' blocks tile the workgroup block");
static_assert(KR_NBUF * KR_STAGE <= 160 * 1024, "LDS");
static_assert(KR_CO % kCoutPad == 0 || kCoutPad % KR_CO == 0, "channel blocks tile the padded channels");
static_assert(kTilePad % KR_TL == 0, "tile blocks tile the padded tiles");

// Requantize and store the 4 channels x 16 pixels of one tile held by a lane:
// q[r][4i+j] is Y + bias + rounding constant of channel co0 + r at pixel
// (i, j) of the tile.
// Y (int32 or int64 T) -> clamp(Y >> out_shift, lo, 127) as int
template <class T>
__device__ __forceinline__ int requant_out(T yv, int s, int lo) {
    if constexpr (sizeof(T) == 4) {
        return med3_i32(yv >> s, lo, 127);
    } else {
        const T v = yv >> s;
        return (int)(v < (T)lo ? (T)lo : (v > (T)127 ? (T)127 : v));
    }
}

template <int LAYOUT, class G, class T>
__device__ __forceinline__ void store_tile(const T (&q)[4][16], const G& g, int8_t* __restrict__ y, int co0,
                                           long long tile) {
    if (tile >= g.ntiles) return;
    int img, ty, tx;
    tile_coords(tile, g, img, ty, tx);
    const int s = g.out_shift;
    const int lo = g.relu ? 0 : -128;
    int v[4][16];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int p = 0; p < 16; ++p) v[r][p] = requant_out(q[r][p], s, lo);
    if (LAYOUT == WINO_NCHW) {
        const bool full_cols = (4 * tx + 3 < g.w) && ((g.w & 3) == 0);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int co = co0 + r;
            if (co >= g.cout) continue;
            int8_t* base = y + (((long long)img * g.cout + co) * g.h + 4 * ty) * g.w + 4 * tx;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (4 * ty + i >= g.h) continue;
                if (full_cols) {
                    const uint32_t wv = __builtin_amdgcn_perm((uint32_t)v[r][4 * i + 1], (uint32_t)v[r][4 * i], 0x0c0c0400u) |
                                        (__builtin_amdgcn_perm((uint32_t)v[r][4 * i + 3], (uint32_t)v[r][4 * i + 2],
                                                               0x0c0c0400u) << 16);
                    *(uint32_t*)(base + (long long)i * g.w) = wv;
                } else {
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        if (4 * tx + j < g.w) base[(long long)i * g.w + j] = (int8_t)v[r][4 * i + j];
                }
            }
        }
    } else {
        const long long rs = (long long)g.w * g.cout;
        int8_t* ob = y + (((long long)img * g.h + 4 * ty) * g.w + 4 * tx) * g.cout + co0;
        const bool full = (co0 + 3 < g.cout) && ((g.cout & 3) == 0) && (4 * ty + 3 < g.h) && (4 * tx + 3 < g.w);
        if (full) {
#pragma unroll
            for (int p = 0; p < 16; ++p) {
                uint32_t pk = put_byte<0>(0u, (uint32_t)v[0][p]);
                pk = put_byte<1>(pk, (uint32_t)v[1][p]);
                pk = put_byte<2>(pk, (uint32_t)v[2][p]);
                pk = put_byte<3>(pk, (uint32_t)v[3][p]);
                *(uint32_t*)(ob + (p >> 2) * rs + (p & 3) * g.cout) = pk;
            }
        } else {
#pragma unroll
            for (int p = 0; p < 16; ++p) {
                if (4 * ty + (p >> 2) >= g.h || 4 * tx + (p & 3) >= g.w) continue;
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (co0 + r < g.cout) ob[(p >> 2) * rs + (p & 3) * g.cout + r] = (int8_t)v[r][p];
            }
        }
    }
}

// Stream-K over the last, partial round of row-streamed blocks.  A launch runs
// n_dp blocks whole (logical blocks [0, n_dp)) and sk_groups workgroups that
// share the stages of the remaining blocks: with U = those blocks x 6 nkc
// stages in sequence (blocks in logical order, each block's stages in ring
// order), workgroup g runs stages [g U / G, (g + 1) U / G), so one workgroup
// may hold the end of one block and the start of the next.  Y is linear in
// the stages (each stage's M folds into Y through the same row pass and
// column update), so a block's Y is the sum of its pieces' partial Y; the
// plan's bound on the sum of the terms' magnitudes also bounds every partial
// sum, so int32 stays exact.  Each piece checks the block's counter: the piece
// that finds every other piece counted adds their partial Y to its own and
// runs the epilogue; any other piece stores its partial Y to its slot in the
// workspace (2 per workgroup: for the first and the last piece of its range),
// then counts itself, and the piece whose count completes the block finishes
// it instead.  No workgroup ever waits for another.  The finisher resets the
// counter, so counters stay zero between launches (the input transform zeroes
// them before the first).
constexpr int KR_SLOT = KR_THREADS * 64;   // int32 of one partial Y (64 per lane)
static_assert(KR_TB == 1, "a partial Y slot holds one 16x16 block per wave");

// first stage (counted from the first split block) of stream-K workgroup sk;
// the host keeps sk_units * sk_groups below 2^31
__device__ __forceinline__ int sk_start(int sk, const K2Args& g) { return sk * g.sk_units / g.sk_groups; }

// the stream-K workgroup whose range holds stage u
__device__ __forceinline__ int sk_owner(int u, const K2Args& g) {
    int c = u * g.sk_groups / g.sk_units;
    while (c + 1 < g.sk_groups && sk_start(c + 1, g) <= u) ++c;
    while (c > 0 && sk_start(c, g) > u) --c;
    return c;
}

// The row-streamed kernel's body; SK: with the stream-K split (the kernel
// wino_tap_gemm_rows_sk), else every workgroup runs one whole block.
template <int LAYOUT, bool SK>
__device__ __forceinline__ void tap_gemm_rows_body(const int8_t* __restrict__ uq, const int8_t* __restrict__ vq,
                                                   const int32_t* __restrict__ bias, int8_t* __restrict__ y,
                                                   const K2Args& g) {
    __shared__ __attribute__((aligned(1024))) uint8_t lds[KR_NBUF * KR_STAGE];
    __shared__ __attribute__((aligned(16))) int bias_blk[KR_CO];
    __shared__ int sk_last;
    // the alignment shifts of the split kernel, read per row fold (from the
    // kernel arguments the compiler would keep all 36 in scalar registers
    // across its pieces)
    __shared__ int sh_tab[SK ? kTaps : 1];
    if constexpr (SK)
        if (threadIdx.x < kTaps) sh_tab[threadIdx.x] = g.tab.sh[threadIdx.x];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int cw = wave & 3, tw = wave >> 2;
    const int lr = lane & 15, lk = lane >> 4;
    const int nkc = g.cin_pad / kKStep;
    const int nstage = 6 * nkc;

    // stream-K workgroup index (-1: a whole block)
    const int sk = !SK || (int)blockIdx.x < g.n_dp ? -1 : xcd_remap((int)blockIdx.x - g.n_dp, g.sk_groups);

    // copy side, fixed parts: this wave's 16 rows, this lane's 16 bytes of
    // slices b0, b0 + step, ... of a stage (k-blocked operands
    // Uq[36][cin_pad/64][cout_pad][64] and Vq[36][cin_pad/64][t_pad][64])
    constexpr int step = KR_WAVES / 8;
    const int grp = wave & 7, b0 = wave >> 3;
    const bool copies_u = grp < 4;
    const int rr = lane >> 2;
    const uint32_t lane_off = (uint32_t)(rr * 64 + 16 * lds_slot(rr, lane & 3));
    const long long tap_stride = copies_u ? (long long)g.cout_pad * g.cin_pad : g.t_pad * g.cin_pad;
    const long long kc_stride = copies_u ? (long long)g.cout_pad * kKStep : g.t_pad * kKStep;
    uint8_t* const dst = lds + 1024 * grp + b0 * KR_CHUNK;
    // The copy source advances by one k-chunk per stage and by a row of taps
    // (minus the chunks walked) at the end of a row: one 64-bit add per stage
    // instead of rebuilding the address from (row, chunk) products, which
    // cost ~50 scalar instructions per stage and wave.
    const long long row_adv = 6 * tap_stride - (long long)(nkc - 1) * kc_stride;
    const long long slice_step = step * tap_stride;

    // compute side: fragment offsets within a slice
    const int row_a = 16 * cw + lr, row_b = KR_CO + 16 * KR_TB * tw + lr;
    const int frag_a = row_a * 64 + 16 * lds_slot(row_a, lk);
    const int frag_b = row_b * 64 + 16 * lds_slot(row_b, lk);   // block tb: + 16 tb rows
    // the rounding constant of the final shift
    const int rnd = g.out_shift > 0 ? 1 << (g.out_shift - 1) : 0;

    // one piece: stages [sb, se) of logical block lbid; at_start: the piece
    // opens this workgroup's range
    auto piece = [&](const int lbid, const int sb, const int se, const bool at_start) {
        const int nst = se - sb;
        const int bco = lbid % g.nbco, btl = lbid / g.nbco;
        const int co_blk = bco * KR_CO;
        const long long tl_blk = (long long)btl * KR_TL;
        // the block's bias (padded to the plan's channel count) into LDS before
        // the ring starts: read from global memory where row 1 uses it, its
        // load would be waited for with every ring copy issued before it
        // (vmcnt counts in order)
        if (threadIdx.x < KR_CO) bias_blk[threadIdx.x] = bias[co_blk + threadIdx.x];
        const int co0 = co_blk + 16 * cw + 4 * lk;   // the lane's four channels

        const int8_t* next_src = (copies_u ? uq + (long long)(co_blk + 16 * grp) * kKStep
                                           : vq + (tl_blk + 16 * (grp - 4)) * kKStep) +
                                 b0 * tap_stride + (long long)(sb / nkc) * 6 * tap_stride +
                                 (long long)(sb % nkc) * kc_stride;
        int next_kc = sb % nkc, next_buf = 0;
        auto issue_next = [&]() {
            uint8_t* d = dst + next_buf * KR_STAGE;
            // plain (temporal) loads for Vq too: the four channel blocks of one
            // tile block run side by side on one XCD (consecutive logical ids)
            // and share that L2's copy; measured, a non-temporal hint on Vq made
            // the later readers go back to memory and cost 8%
#pragma unroll
            for (int i = 0; i < KR_LPW; ++i)
                lds_copy16(next_src + i * slice_step + lane_off,
                           (__attribute__((address_space(3))) void*)(d + step * i * KR_CHUNK));
            if (++next_kc == nkc) {
                next_kc = 0;
                next_src += row_adv;
            } else {
                next_src += kc_stride;
            }
            next_buf = next_buf == KR_NBUF - 1 ? 0 : next_buf + 1;
        };

        // Y of the lane's KR_TB tiles x 4 channels, 4x4 each
        int yv[KR_TB][4][16];
#pragma unroll
        for (int tb = 0; tb < KR_TB; ++tb)
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int p = 0; p < 16; ++p) yv[tb][r][p] = 0;

        issue_next();
        if (nst > 1) issue_next();
        int s = 0, buf = 0;
#pragma unroll
        for (int a = 0; a < 6; ++a) {
            // the piece's k-chunks of row a
            const int klo = sb > a * nkc ? sb - a * nkc : 0;
            const int khi = se < (a + 1) * nkc ? se - a * nkc : nkc;
            if (klo >= khi) continue;
            v4i m[6][KR_TB];
            // one stage: the six taps of row a, 64 input channels; the first
            // k-chunk of the row starts the accumulators from zero
            auto stage = [&](bool first) {
                // stage s has landed once only the next stage's loads are pending
                if (s + 1 < nst)
                    WINO_WAIT_VM_LDS(KR_LPW);
                else
                    WINO_WAIT_VM_LDS(0);
                ring_barrier();   // stage s visible; stage s-1 (same buffer as s+2) consumed
                if (s + 2 < nst) issue_next();
                const uint8_t* base = lds + buf * KR_STAGE;
                buf = buf == KR_NBUF - 1 ? 0 : buf + 1;
                ++s;
                // fragments of two taps in flight ahead of the MFMAs
                v4i fa[2], fb[2][KR_TB];
                auto frag = [&](int b) {
                    fa[b & 1] = *(const v4i*)(base + b * KR_CHUNK + frag_a);
#pragma unroll
                    for (int tb = 0; tb < KR_TB; ++tb)
                        fb[b & 1][tb] = *(const v4i*)(base + b * KR_CHUNK + frag_b + 16 * 64 * tb);
                };
                frag(0);
                frag(1);
                const v4i zero = (v4i){0, 0, 0, 0};
#pragma unroll
                for (int b = 0; b < 6; ++b) {
#pragma unroll
                    for (int tb = 0; tb < KR_TB; ++tb)
                        m[b][tb] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[b & 1], fb[b & 1][tb],
                                                                         first ? zero : m[b][tb], 0, 0, 0);
                    if (b + 2 < 6) frag(b + 2);
                }
                // keep that order (masks: 0x100 LDS read, 0x008 MFMA)
                __builtin_amdgcn_sched_group_barrier(0x100, 2 * (1 + KR_TB), 0);
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    __builtin_amdgcn_sched_group_barrier(0x008, KR_TB, 0);
                    __builtin_amdgcn_sched_group_barrier(0x100, 1 + KR_TB, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x008, 2 * KR_TB, 0);
            };
            stage(true);
            for (int kc = klo + 1; kc < khi; ++kc) stage(false);

            // bias plus rounding constant, injected through tap (1,1): its row
            // and column of A^T are all ones, so it reaches every output of
            // the tile once.  Taken by the piece holding row 1's first chunk,
            // and read only here, after the stages' barriers: wave 0 wrote
            // bias_blk at the start of the piece, and a piece that starts at
            // row 1 has no barrier before its first stage.
            v4i bias_rnd = (v4i){0, 0, 0, 0};
            if (a == 1 && klo == 0) bias_rnd = *(const v4i*)(bias_blk + (co0 - co_blk)) + rnd;

            // fold row a: z = (M'[a, :]) A, then Y += A^T[:, a] z
#pragma unroll
            for (int tb = 0; tb < KR_TB; ++tb)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    int mv[6], z[4];
#pragma unroll
                    for (int b = 0; b < 6; ++b) mv[b] = m[b][tb][r] << (SK ? sh_tab[6 * a + b] : g.tab.sh[6 * a + b]);
                    if (a == 1) mv[1] += bias_rnd[r];
                    at_1d(mv, z);
                    int* yr = yv[tb][r];
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        // column a of A^T: 1 1 1 1 1 0 / 0 1 -1 2 -2 0 / 0 1 1 4 4 0 / 0 1 -1 8 -8 1
                        if (a < 5) yr[j] += z[j];
                        if (a == 1) { yr[4 + j] += z[j]; yr[8 + j] += z[j]; yr[12 + j] += z[j]; }
                        if (a == 2) { yr[4 + j] -= z[j]; yr[8 + j] += z[j]; yr[12 + j] -= z[j]; }
                        if (a == 3) { yr[4 + j] += z[j] << 1; yr[8 + j] += z[j] << 2; yr[12 + j] += z[j] << 3; }
                        if (a == 4) { yr[4 + j] -= z[j] << 1; yr[8 + j] += z[j] << 2; yr[12 + j] -= z[j] << 3; }
                        if (a == 5) yr[12 + j] += z[j];
                    }
                }
            // materialize Y here: Y is only read at the very end, and the
            // compiler would otherwise sink the folds past the later rows and
            // keep every row's accumulators live at once
#pragma unroll
            for (int tb = 0; tb < KR_TB; ++tb)
#pragma unroll
                for (int r = 0; r < 4; ++r)
#pragma unroll
                    for (int p = 0; p < 16; ++p) asm volatile("" : "+v"(yv[tb][r][p]));
        }

        if (SK && (sb != 0 || se != nstage)) {
            // a piece of a split block: finish the block or leave a partial Y
            const int jb = (lbid - g.n_dp) * nstage;   // its first stage in the split sequence
            const int glo = sk_owner(jb, g), ghi = sk_owner(jb + nstage - 1, g);
            const int others = ghi - glo;
            int* const cnt = g.sk_cnt + (lbid - g.n_dp);
            if (threadIdx.x == 0) {
                const int c = __hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (c == others) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                sk_last = c == others;
            }
            __syncthreads();
            bool last = sk_last;
            if (!last) {
                int* const slot = g.sk_part + (size_t)(2 * sk + (at_start ? 0 : 1)) * KR_SLOT;
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    *(v4i*)(slot + 4 * (i * KR_THREADS + (int)threadIdx.x)) =
                        (v4i){yv[0][i >> 2][4 * (i & 3)], yv[0][i >> 2][4 * (i & 3) + 1],
                              yv[0][i >> 2][4 * (i & 3) + 2], yv[0][i >> 2][4 * (i & 3) + 3]};
                WINO_WAIT_VM(0);   // this wave's stores have reached L2
                __syncthreads();
                if (threadIdx.x == 0) {
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
                    const int c = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (c == others) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                    sk_last = c == others;
                }
                __syncthreads();
                last = sk_last;
            }
            if (!last) return;
            // the other pieces' partial Y: slot 0 of a workgroup whose range
            // starts inside this block, slot 1 of the one that enters it
            for (int c = glo; c <= ghi; ++c) {
                if (c == sk) continue;
                const int* const slot = g.sk_part + (size_t)(2 * c + (sk_start(c, g) >= jb ? 0 : 1)) * KR_SLOT;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const v4i v = *(const v4i*)(slot + 4 * (i * KR_THREADS + (int)threadIdx.x));
#pragma unroll
                    for (int e = 0; e < 4; ++e) yv[0][i >> 2][4 * (i & 3) + e] += v[e];
                }
            }
            if (threadIdx.x == 0) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }

        if (LAYOUT == WINO_NHWC && g.y_staged) {
            // NHWC with whole 64-channel blocks: gather the block's output in
            // LDS (the ring is idle now) so every pixel's 64 channel bytes leave
            // as four 16-byte stores of adjacent lanes -- 64-byte write requests
            // instead of 16-byte pieces scattered over 16 lines per instruction
            constexpr int PITCH = 16 * 64 + 16;   // bytes per tile; the pad spreads lanes over banks
            static_assert(KR_TL * PITCH <= KR_NBUF * KR_STAGE, "output staging fits the ring");
            const int sft = g.out_shift, lo = g.relu ? 0 : -128;
            __syncthreads();                      // every wave is done reading the ring
#pragma unroll
            for (int tb = 0; tb < KR_TB; ++tb) {
                uint8_t* ot = lds + (16 * (KR_TB * tw + tb) + lr) * PITCH + 16 * cw + 4 * lk;
#pragma unroll
                for (int p = 0; p < 16; ++p) {
                    uint32_t pk = put_byte<0>(0u, (uint32_t)med3_i32(yv[tb][0][p] >> sft, lo, 127));
                    pk = put_byte<1>(pk, (uint32_t)med3_i32(yv[tb][1][p] >> sft, lo, 127));
                    pk = put_byte<2>(pk, (uint32_t)med3_i32(yv[tb][2][p] >> sft, lo, 127));
                    pk = put_byte<3>(pk, (uint32_t)med3_i32(yv[tb][3][p] >> sft, lo, 127));
                    *(uint32_t*)(ot + 64 * p) = pk;
                }
            }
            __syncthreads();
            // wave w copies tiles w, w + 16, ...: lane = 16-byte quarter q of pixel p
            const int p = lane >> 2, q = lane & 3;
            for (int tl = wave; tl < KR_TL; tl += KR_WAVES) {
                const long long tile = tl_blk + tl;   // wave-uniform
                if (tile >= g.ntiles) break;
                int img, ty, tx;
                tile_coords(tile, g, img, ty, tx);
                const int yy = 4 * ty + (p >> 2), xx = 4 * tx + (p & 3);
                if (yy < g.h && xx < g.w) {
                    // non-temporal: the output is not read again here, and in
                    // L2 it would evict the operands the next round of blocks
                    // reads (measured 2-3% of the kernel at C5 and C4)
                    __builtin_nontemporal_store(*(const v4i*)(lds + tl * PITCH + 64 * p + 16 * q),
                                                (v4i*)(y + (((long long)img * g.h + yy) * g.w + xx) * g.cout +
                                                       co_blk + 16 * q));
                }
            }
        } else {
#pragma unroll
            for (int tb = 0; tb < KR_TB; ++tb)
                store_tile<LAYOUT>(yv[tb], g, y, co0, tl_blk + 16 * (KR_TB * tw + tb) + lr);
        }
    };

    // Whole blocks and the (at most two) pieces of a stream-K range each take
    // a copy of the piece code: as a loop over pieces, the compiler kept the
    // loop-invariant scalars of the whole body live across it and spilled.
    if (!SK || sk < 0) {
        piece(xcd_remap(blockIdx.x, g.n_dp), 0, nstage, true);
        return;
    }
    // this workgroup's stages [u0, u1) of the split sequence (stage s of split
    // block j is j * nstage + s); the host keeps u1 - u0 <= nstage, so the
    // range ends in the block it starts in or in the next one
    const int u0 = sk_start(sk, g), u1 = sk_start(sk + 1, g);
    const int j = u0 / nstage;
    const int sb = u0 - j * nstage;
    const int se = u1 - u0 < nstage - sb ? sb + (u1 - u0) : nstage;
    piece(g.n_dp + j, sb, se, true);
    if (u0 + (se - sb) < u1) {
        // The ring's vmcnt waits count its own copies and assume they complete
        // in issue order; stores still in flight from the first piece's
        // epilogue may complete after later loads, so they are waited for
        // first.  Then every wave is done with the first piece's LDS.
        WINO_WAIT_VM(0);
        __syncthreads();
        piece(g.n_dp + j + 1, 0, u1 - u0 - (se - sb), false);
    }
}

template <int LAYOUT>
__global__ __launch_bounds__(KR_THREADS) void wino_tap_gemm_rows(const int8_t* __restrict__ uq,
                                                                 const int8_t* __restrict__ vq,
                                                                 const int32_t* __restrict__ bias,
                                                                 int8_t* __restrict__ y, K2Args g) {
    tap_gemm_rows_body<LAYOUT, false>(uq, vq, bias, y, g);
}

template <int LAYOUT>
__global__ __launch_bounds__(KR_THREADS) void wino_tap_gemm_rows_sk(const int8_t* __restrict__ uq,
                                                                    const int8_t* __restrict__ vq,
                                                                    const int32_t* __restrict__ bias,
                                                                    int8_t* __restrict__ y, K2Args g) {
    tap_gemm_rows_body<LAYOUT, true>(uq, vq, bias, y, g);
}

#include "wino_tap_ws.h"

// ---------------------------------------------------------------------------
// K2W wino_tap_gemm_rows_wide: the row-streamed scheme of wino_tap_gemm_rows
// for the int8/10 operands (Q = 10: fp16 holding 10-bit integers, 32
// channels per 64-byte k row) and a 32- or 64-bit output accumulator YT.
// With the 64-bit epilogue the tap-resident kernel needs 144 accumulators
// plus the int64 fold per lane and only fits 32x32 blocks of four waves;
// here a lane keeps the six accumulators of the current row of taps and
// 4 x 16 YT values, so a 64 (channels) x 32 (tiles) block of eight waves fits
// (two waves per SIMD, one workgroup per CU: the ring takes 144 KB of LDS).
//
// Ring stage = one row a of taps and one 64-byte k row: six slices of 64 Uq +
// 32 Vq rows (6 KB each, 36 KB); four stages rotate through 144 KB of LDS,
// three in flight.  A stage is 36 loads of 16 rows x 64 B; wave w issues
// loads w, w + 8, ..., w + 32 (the last wraps onto an earlier load: the same
// bytes to the same place).  Load j covers slice j / 6 and row group j % 6
// (groups 0-3: Uq, 4-5: Vq).
// ---------------------------------------------------------------------------
constexpr int KW_CO = 64;
constexpr int KW_TL = 32;
constexpr int KW_WAVES = (KW_CO / 16) * (KW_TL / 16);
constexpr int KW_THREADS = 64 * KW_WAVES;
constexpr int KW_GROUPS = (KW_CO + KW_TL) / 16;            // 16-row groups per slice
constexpr int KW_CHUNK = (KW_CO + KW_TL) * kKStep;         // one slice
constexpr int KW_STAGE = 6 * KW_CHUNK;
constexpr int KW_NBUF = 4;
constexpr int KW_LOADS = 6 * KW_GROUPS;                     // 1-KB loads per stage
constexpr int KW_LPW = (KW_LOADS + KW_WAVES - 1) / KW_WAVES;
static_assert(KW_NBUF * KW_STAGE <= 160 * 1024, "LDS");
static_assert((KW_NBUF - 2) * KW_LPW <= 63, "vmcnt range");
static_assert(kTilePad % KW_TL == 0 && kCoutPad % KW_CO == 0, "blocks tile the padded sizes");

template <int LAYOUT, int Q, class YT>
__global__ __launch_bounds__(KW_THREADS) void wino_tap_gemm_rows_wide(const int8_t* __restrict__ uq,
                                                                        const int8_t* __restrict__ vq,
                                                                        const int32_t* __restrict__ bias,
                                                                        int8_t* __restrict__ y, K2Args g) {
    __shared__ __attribute__((aligned(1024))) uint8_t lds[KW_NBUF * KW_STAGE];
    const int lbid = xcd_remap(blockIdx.x, g.nblocks);
    const int bco = lbid % g.nbco, btl = lbid / g.nbco;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int cw = wave & 3, tw = wave >> 2;
    const int co_blk = bco * KW_CO;
    const long long tl_blk = (long long)btl * KW_TL;
    const int lr = lane & 15, lk = lane >> 4;
    const int nkc = g.cin_pad / kKStep;          // 64-byte k rows
    const int nstage = 6 * nkc;

    // copy side: every load advances by one k row per stage and by a row of
    // taps (minus the k rows walked) at the end of a row of taps
    const long long su = (long long)g.cout_pad * g.cin_pad, sv = g.t_pad * g.cin_pad;   // tap strides
    const long long ku = (long long)g.cout_pad * kKStep, kv = g.t_pad * kKStep;           // k-row strides
    const int rr = lane >> 2;
    const uint32_t lane_off = (uint32_t)(rr * 64 + 16 * lds_slot(rr, lane & 3));
    const int8_t* src[KW_LPW];
    long long kadv[KW_LPW], radv[KW_LPW];
    int dsto[KW_LPW];
#pragma unroll
    for (int i = 0; i < KW_LPW; ++i) {
        int j = wave + KW_WAVES * i;
        if (j >= KW_LOADS) j -= KW_WAVES;
        const int b = j / KW_GROUPS, q = j % KW_GROUPS;
        const bool isu = q < KW_CO / 16;
        src[i] = isu ? uq + b * su + (long long)(co_blk + 16 * q) * kKStep
                     : vq + b * sv + (tl_blk + 16 * (q - KW_CO / 16)) * kKStep;
        kadv[i] = isu ? ku : kv;
        radv[i] = (isu ? 6 * su : 6 * sv) - (long long)(nkc - 1) * kadv[i];
        dsto[i] = b * KW_CHUNK + q * 1024;
    }
    int next_kc = 0, next_buf = 0;
    auto issue_next = [&]() {
        uint8_t* d = lds + next_buf * KW_STAGE;
        const bool row_end = ++next_kc == nkc;
        if (row_end) next_kc = 0;
#pragma unroll
        for (int i = 0; i < KW_LPW; ++i) {
            lds_copy16(src[i] + lane_off, (__attribute__((address_space(3))) void*)(d + dsto[i]));
            src[i] += row_end ? radv[i] : kadv[i];
        }
        next_buf = next_buf == KW_NBUF - 1 ? 0 : next_buf + 1;
    };

    // compute side
    const int row_a = 16 * cw + lr, row_b = KW_CO + 16 * tw + lr;
    const int frag_a = row_a * 64 + 16 * lds_slot(row_a, lk);
    const int frag_b = row_b * 64 + 16 * lds_slot(row_b, lk);
    const int co0 = co_blk + 16 * cw + 4 * lk;
    const YT rnd = g.out_shift > 0 ? (YT)1 << (g.out_shift - 1) : (YT)0;
    // loaded ahead of the ring: a load issued behind the prefetched stages
    // would make its first use wait for all of them
    const v4i bias4 = *(const v4i*)(bias + co0);

    YT yv[4][16];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int p = 0; p < 16; ++p) yv[r][p] = 0;

#pragma unroll
    for (int st = 0; st < KW_NBUF - 1; ++st)
        if (st < nstage) issue_next();
    int s = 0, buf = 0;
#pragma unroll
    for (int a = 0; a < 6; ++a) {
        v4i m[6];
        auto stage = [&](bool first) {
            // stage s has landed once only the stages issued after it are
            // pending: min(NBUF - 2, nstage - 1 - s) of them
            const int ahead = min(KW_NBUF - 2, nstage - 1 - s);
            if (ahead >= 2)
                WINO_WAIT_VM_LDS(2 * KW_LPW);
            else if (ahead == 1)
                WINO_WAIT_VM_LDS(KW_LPW);
            else
                WINO_WAIT_VM_LDS(0);
            ring_barrier();   // stage s visible; stage s-1 (the buffer refilled next) consumed
            if (s + KW_NBUF - 1 < nstage) issue_next();
            const uint8_t* base = lds + buf * KW_STAGE;
            buf = buf == KW_NBUF - 1 ? 0 : buf + 1;
            ++s;
            v4i fa[2], fb[2];
            auto frag = [&](int b) {
                fa[b & 1] = *(const v4i*)(base + b * KW_CHUNK + frag_a);
                fb[b & 1] = *(const v4i*)(base + b * KW_CHUNK + frag_b);
            };
            frag(0);
            frag(1);
            const v4i zero = (v4i){0, 0, 0, 0};
#pragma unroll
            for (int b = 0; b < 6; ++b) {
                if constexpr (Q == 10) {
                    // fp16 10-bit integers: 32 products and their sums are
                    // integers below 2^24, exact in fp32
                    const v4f r = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                        __builtin_bit_cast(v8h, fa[b & 1]), __builtin_bit_cast(v8h, fb[b & 1]),
                        (v4f){0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                    const v4i ri = __builtin_convertvector(r, v4i);
                    m[b] = first ? ri
                                 : __builtin_bit_cast(v4i, __builtin_bit_cast(v4u, m[b]) + __builtin_bit_cast(v4u, ri));
                } else {
                    m[b] = __builtin_amdgcn_mfma_i32_16x16x64_i8(fa[b & 1], fb[b & 1], first ? zero : m[b], 0, 0, 0);
                }
                if (b + 2 < 6) frag(b + 2);
            }
        };
        stage(true);
        for (int kc = 1; kc < nkc; ++kc) stage(false);

        // fold row a: z = (M'[a, :]) A, then Y += A^T[:, a] z, in YT
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            YT mv[6], z[4];
#pragma unroll
            for (int b = 0; b < 6; ++b) mv[b] = (YT)m[b][r] << g.tab.sh[6 * a + b];
            if (a == 1) mv[1] += (YT)bias4[r] + rnd;      // tap (1, 1): bias and rounding constant
            at_1d(mv, z);
            YT* yr = yv[r];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                // column a of A^T: 1 1 1 1 1 0 / 0 1 -1 2 -2 0 / 0 1 1 4 4 0 / 0 1 -1 8 -8 1
                if (a < 5) yr[j] += z[j];
                if (a == 1) { yr[4 + j] += z[j]; yr[8 + j] += z[j]; yr[12 + j] += z[j]; }
                if (a == 2) { yr[4 + j] -= z[j]; yr[8 + j] += z[j]; yr[12 + j] -= z[j]; }
                if (a == 3) { yr[4 + j] += z[j] << 1; yr[8 + j] += z[j] << 2; yr[12 + j] += z[j] << 3; }
                if (a == 4) { yr[4 + j] -= z[j] << 1; yr[8 + j] += z[j] << 2; yr[12 + j] -= z[j] << 3; }
                if (a == 5) yr[12 + j] += z[j];
            }
        }
        // keep the folds here (the compiler would sink them past later rows)
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int p = 0; p < 16; ++p) asm volatile("" : "+v"(yv[r][p]));
    }
    store_tile<LAYOUT>(yv, g, y, co0, tl_blk + 16 * tw + lr);
}

// ---------------------------------------------------------------------------
// host-side helpers
// ---------------------------------------------------------------------------
// compute units of the current device (the launch heuristics use it),
// queried once per device
int num_cus() {
    static std::atomic<int> cached[64] = {};
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (dev >= 0 && dev < 64 && (n = cached[dev].load(std::memory_order_relaxed)) > 0) return n;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 256;
    if (dev >= 0 && dev < 64) cached[dev].store(n, std::memory_order_relaxed);
    return n;
}

struct Geometry {
    int n, h, w, th, tw;
    long long ntiles, t_pad;
};

// Tile grid of F(m x m, 3 x 3) over an n x h x w input.
wino_status geometry(int32_t n, int32_t h, int32_t w, int m, Geometry& g) {
    if (n < 0 || h < 0 || w < 0) return WINO_EINVAL;
    if (h > 65536 || w > 65536) return WINO_EUNSUPPORTED;
    g.n = n;
    g.h = h;
    g.w = w;
    g.th = (h + m - 1) / m;
    g.tw = (w + m - 1) / m;
    g.ntiles = (long long)n * g.th * g.tw;
    if (g.ntiles >= (1ll << 26)) return WINO_EUNSUPPORTED;
    g.t_pad = round_up(g.ntiles, kTilePad);
    return WINO_OK;
}

size_t vq_bytes(const wino_f4_plan_s* p, const Geometry& g) {
    return (size_t)p->ntap * (size_t)g.t_pad * (size_t)p->cin_pad * kbytes_per_channel(p->bits);
}

TapTables tables_of(const wino_f4_plan_s* p) {
    TapTables t = {};
    for (int i = 0; i < p->ntap; ++i) {
        t.eb[i] = p->e_b[i];
        t.sh[i] = p->sh[i];
    }
    return t;
}

K1Args k1_args(const Geometry& g, int cin, int cin_pad, const TapTables& tab, int bits = 8) {
    K1Args a;
    a.n = g.n;
    a.cin = cin;
    a.h = g.h;
    a.w = g.w;
    a.th = g.th;
    a.tw = g.tw;
    a.cin_pad = cin_pad;
    a.ntxb = 0;                          // set at launch with the block width
    a.ncg = cin_pad / K1_CG;
    a.t_pad = g.t_pad;
    a.tab = tab;
    for (int t = 0; t < kTaps; ++t) {
        const int e = tab.eb[t];
        const uint32_t r = e > 0 ? (1u << (e - 1)) : 0u;
        a.rnd2[t] = r | (r << 16);
    }
    // the saturating requantization needs 0 <= e_B <= 16 - bits for every tap
    a.q_sat = 1;
    for (int t = 0; t < kTaps; ++t)
        if (tab.eb[t] < 0 || tab.eb[t] > 16 - bits) a.q_sat = 0;
    a.plane_bytes = g.t_pad * cin_pad * kbytes_per_channel(bits);
    a.vq_buf = a.plane_bytes < 0x7fffffffLL;
    a.x_vec = 0;
    a.x_dw = 0;
    a.sk_cnt = nullptr;
    a.sk_ncnt = 0;
    return a;
}

// tiles per block of the direct NHWC transform: 8 unless 16 leaves fewer
// idle tiles at the end of a row of tw tiles (measured: 8-tile blocks are as
// fast or faster on every layer here; C4's rows of 128 tiles 10.7 -> 10.3 us)
int k1_direct_tx(int tw) {
    const int idle16 = (tw + 15) / 16 * 16 - tw, idle8 = (tw + 7) / 8 * 8 - tw;
    return idle8 <= idle16 ? 8 : 16;
}

template <int M, int MODE, int Q, int TX>
wino_status launch_k1_tx(const K1Args& a, wino_layout layout, const int8_t* x, int8_t* vq, int* tapmax,
                         hipStream_t stream) {
    K1Args args = a;
    args.ntxb = (a.tw + TX - 1) / TX;
    long long blocks = (long long)args.ntxb * a.ncg * a.n * a.th;
    if (blocks == 0) return WINO_OK;
    if (blocks > 0x7fffffffll) return WINO_EUNSUPPORTED;
    args.x_vec = (a.cin % 16 == 0) && (((uintptr_t)x & 15) == 0);
    args.x_dw = layout == WINO_NCHW && a.w % 4 == 0 && (((uintptr_t)x & 3) == 0) &&
                (long long)a.cin * a.h * a.w < 0x7ffffff0ll;
#define K1_LAUNCH(L, S)                                                                                      \
    hipLaunchKernelGGL((wino_input_xform<M, L, MODE, Q, TX, S>), dim3((unsigned)blocks), dim3(16 * TX), 0, stream, \
                       x, vq, tapmax, args)
    const bool sat = MODE == 0 && a.q_sat;
    if constexpr (MODE == 0) {
        if (layout == WINO_NHWC && a.cin % 4 == 0 && ((uintptr_t)x & 3) == 0 && (long long)a.w * a.cin < 0x7ffffff0ll) {
            const int tx = k1_direct_tx(a.tw);
            args.ntxb = (a.tw + tx - 1) / tx;
            const long long nb = (long long)args.ntxb * a.ncg * a.n * a.th;
            if (nb > 0x7fffffffll) return WINO_EUNSUPPORTED;
#define K1D_LAUNCH(T, S)                                                                                            \
    hipLaunchKernelGGL((wino_input_xform_nhwc<M, Q, T, S>), dim3((unsigned)nb), dim3(16 * T), 0, stream, x, vq, args)
            if (tx == 8) {
                if (sat) K1D_LAUNCH(8, true); else K1D_LAUNCH(8, false);
            } else {
                if (sat) K1D_LAUNCH(16, true); else K1D_LAUNCH(16, false);
            }
#undef K1D_LAUNCH
            return hipGetLastError() == hipSuccess ? WINO_OK : WINO_EHIP;
        }
    }
    if (layout == WINO_NHWC) {
        if (sat) K1_LAUNCH(WINO_NHWC, MODE == 0); else K1_LAUNCH(WINO_NHWC, false);
    } else {
        if (sat) K1_LAUNCH(WINO_NCHW, MODE == 0); else K1_LAUNCH(WINO_NCHW, false);
    }
#undef K1_LAUNCH
    return hipGetLastError() == hipSuccess ? WINO_OK : WINO_EHIP;
}

template <int M, int MODE, int Q = 8>
wino_status launch_k1(const K1Args& a, wino_layout layout, const int8_t* x, int8_t* vq, int* tapmax,
                      hipStream_t stream) {
    return launch_k1_tx<M, MODE, Q, K1_TX>(a, layout, x, vq, tapmax, stream);
}

template <class C>
long long resident_blocks(const wino_f4_plan_s* p, const Geometry& g) {
    return (long long)(p->cout_pad / C::CO) * ((g.ntiles + C::TL - 1) / C::TL);
}

// The tap-GEMM kernel of a convolution (a wino_tap_kernel value other than
// AUTO and RESIDENT).  The row-streamed kernel needs the 32-bit epilogue and
// an output convolution; AUTO takes it when its 64x64 blocks fill the device.
// Otherwise the 64x32 tap-resident shape: on the small layers where too few
// blocks exist the smaller shapes were measured no faster (C1-C3: 14-16 us
// against 11-14 us), as the time there is the serial chain of ring-stage
// latencies and the epilogue inside each block, not the block count.
// Calibration and debug exports (MODE 1, 2) always use the 64x32 shape.
int tap_kernel_for(const wino_f4_plan_s* p, const Geometry& g, int mode) {
    const int k = p->tap_kernel;
    // int8/10 (fp16 operands): the row-streamed 64x32 kernel by default; a
    // forced resident shape (16X16 stands for the 32x32 shape with 6-tap
    // stages), or RESIDENT: 64x32, 32x32 with the 64-bit epilogue (its only
    // resident shape without spills), as for calibration and exports
    if (p->bits == 10 && p->m == 4) {
        if (mode == 0 && (k == WINO_TAP_RESIDENT_64X32 || k == WINO_TAP_RESIDENT_32X32 ||
                          k == WINO_TAP_RESIDENT_16X16))
            return k;
        if (mode == 0 && k != WINO_TAP_RESIDENT) return WINO_TAP_ROWS;
        return p->epi_bits == 64 ? WINO_TAP_RESIDENT_32X32 : WINO_TAP_RESIDENT_64X32;
    }
    // F2: its own 64x32 configuration
    if (mode != 0 || p->m != 4 || p->bits != 8) return WINO_TAP_RESIDENT_64X32;
    if (k == WINO_TAP_RESIDENT_64X32 || k == WINO_TAP_RESIDENT_32X32 || k == WINO_TAP_RESIDENT_16X16) return k;
    // the wave-specialized kernel (forced only: measured slower than ROWS on
    // every layer here) packs the alignment shifts in 5 bits, which the
    // 32-bit epilogue bound keeps far below 32
    if (p->epi_bits == 32 && k == WINO_TAP_WAVES) {
        bool sh5 = true;
        for (int t = 0; t < p->ntap; ++t) sh5 = sh5 && p->sh[t] >= 0 && p->sh[t] < 32;
        return sh5 ? WINO_TAP_WAVES : WINO_TAP_ROWS;
    }
    if (p->epi_bits == 32 && k != WINO_TAP_RESIDENT &&
        (k == WINO_TAP_ROWS || k == WINO_TAP_ROWS_STREAMK ||
         (long long)(p->cout_pad / KR_CO) * (g.t_pad / KR_TL) >= num_cus()))
        return WINO_TAP_ROWS;
    return WINO_TAP_RESIDENT_64X32;
}

// 64-channel chunks per ring stage of the wave-specialized kernel: the
// largest of 4, 3, 2, 1 that divides the padded input channels' chunks
int ws_chunks_per_stage(int cin_pad) {
    const int nkc = cin_pad / kKStep;
    for (int nk = 4; nk > 1; --nk)
        if (nkc % nk == 0) return nk;
    return 1;
}

// Stream-K split of the row-streamed tap GEMM's last round (the workspace
// past Vq holds its counters and partial sums), forced only
// (WINO_TAP_ROWS_STREAMK): it splits whenever a partial round exists (also
// below one round), spreading the stages as thinly as one per workgroup.
// Measured at C5 (400 blocks: one whole round, 144 blocks split over 256
// workgroups), K2 takes 80 us against 52 us unsplit: the split round alone
// takes 57 us, 30 us of it without the partial-sum exchange (each workgroup
// runs two pieces and pays a block's fixed costs -- ring start, row folds,
// epilogue -- for each) and the rest in the exchange (61 MB of partial sums
// written and read back, and the agent-scope fences).
struct SkPlan {
    int n_dp = 0, groups = 0, nsplit = 0, units = 0;
    size_t cnt_off = 0, part_off = 0, end = 0;   // byte offsets in the workspace
};

bool sk_plan_for(const wino_f4_plan_s* p, const Geometry& g, SkPlan& sk) {
    if (p->bits != 8 || p->m != 4 || g.ntiles == 0 || tap_kernel_for(p, g, 0) != WINO_TAP_ROWS) return false;
    const long long nblocks = (long long)(p->cout_pad / KR_CO) * (g.t_pad / KR_TL);
    const long long ncu = num_cus();
    const long long rem = nblocks % ncu;
    if (rem == 0 || p->tap_kernel != WINO_TAP_ROWS_STREAMK) return false;
    const long long nstage = 6 * (p->cin_pad / kKStep);
    const long long units = rem * nstage, groups = std::min<long long>(ncu, units);
    // 32-bit stage arithmetic in the kernel; every range within two blocks
    if (units * groups >= (1ll << 31) || (units + groups - 1) / groups > nstage) return false;
    sk.n_dp = (int)(nblocks - rem);
    sk.nsplit = (int)rem;
    sk.units = (int)units;
    sk.groups = (int)groups;
    sk.cnt_off = (size_t)round_up((long long)vq_bytes(p, g), 256);
    sk.part_off = sk.cnt_off + (size_t)round_up(rem * 4, 256);
    sk.end = sk.part_off + (size_t)2 * sk.groups * KR_SLOT * sizeof(int32_t);
    return true;
}

// The split applies when the plan and shape call for it and the caller's
// workspace holds it.
bool sk_in_workspace(const wino_f4_plan_s* p, const Geometry& g, size_t ws_bytes, SkPlan& sk) {
    return sk_plan_for(p, g, sk) && ws_bytes >= sk.end;
}

template <class C, int M, int MODE, int Q = 8>
wino_status launch_resident(const wino_f4_plan_s* p, const Geometry& g, wino_layout layout, const int8_t* vq,
                            int8_t* y, void* aux, K2Args a, hipStream_t stream) {
    const long long blocks = resident_blocks<C>(p, g);
    if (blocks == 0) return WINO_OK;
    if (blocks > 0x7fffffffll) return WINO_EUNSUPPORTED;
    a.nbco = p->cout_pad / C::CO;
    a.nblocks = (int)blocks;
    a.cin_pad = p->cin_pad * kbytes_per_channel(Q);      // bytes of one operand row
    dim3 grid((unsigned)blocks), block(C::THREADS);
#define K2_LAUNCH(L, E)                                                                              \
    hipLaunchKernelGGL((wino_tap_gemm<C, M, L, E, MODE, Q>), grid, block, 0, stream, p->uq_dev, vq, p->bias_dev, \
                       y, aux, a)
    if (layout == WINO_NHWC) {
        if (p->epi_bits == 32) K2_LAUNCH(WINO_NHWC, 32); else K2_LAUNCH(WINO_NHWC, 64);
    } else {
        if (p->epi_bits == 32) K2_LAUNCH(WINO_NCHW, 32); else K2_LAUNCH(WINO_NCHW, 64);
    }
#undef K2_LAUNCH
    return hipGetLastError() == hipSuccess ? WINO_OK : WINO_EHIP;
}

// the row-streamed kernel for int8/10 operands, with the plan's epilogue width
wino_status launch_rows_wide(const wino_f4_plan_s* p, const Geometry& g, wino_layout layout, const int8_t* vq,
                             int8_t* y, K2Args a, hipStream_t stream) {
    const long long blocks = (long long)(p->cout_pad / KW_CO) * (g.t_pad / KW_TL);
    if (blocks > 0x7fffffffll) return WINO_EUNSUPPORTED;
    a.nbco = p->cout_pad / KW_CO;
    a.nblocks = (int)blocks;
    a.cin_pad = p->cin_pad * kbytes_per_channel(10);
    dim3 grid((unsigned)blocks), block(KW_THREADS);
#define KW_LAUNCH(L, T) \
    hipLaunchKernelGGL((wino_tap_gemm_rows_wide<L, 10, T>), grid, block, 0, stream, p->uq_dev, vq, p->bias_dev, y, a)
    if (layout == WINO_NHWC) {
        if (p->epi_bits == 32) KW_LAUNCH(WINO_NHWC, int); else KW_LAUNCH(WINO_NHWC, long long);
    } else {
        if (p->epi_bits == 32) KW_LAUNCH(WINO_NCHW, int); else KW_LAUNCH(WINO_NCHW, long long);
    }
#undef KW_LAUNCH
    return hipGetLastError() == hipSuccess ? WINO_OK : WINO_EHIP;
}

// ws_bytes: the workspace at vq (the stream-K split uses the part past Vq)
template <int MODE>
wino_status launch_k2(const wino_f4_plan_s* p, const Geometry& g, wino_layout layout, const int8_t* vq,
                      int8_t* y, void* aux, hipStream_t stream, size_t ws_bytes = 0) {
    if (g.ntiles == 0) return WINO_OK;
    K2Args a;
    a.cin_pad = p->cin_pad;
    a.cout = p->cout;
    a.cout_pad = p->cout_pad;
    a.n = g.n;
    a.h = g.h;
    a.w = g.w;
    a.th = g.th;
    a.tw = g.tw;
    a.ntiles = g.ntiles;
    a.t_pad = g.t_pad;
    a.out_shift = p->out_shift;
    a.relu = p->relu;
    a.y_staged = layout == WINO_NHWC && p->cout % KR_CO == 0 && ((uintptr_t)y & 15) == 0;
    a.n_dp = 0;
    a.sk_groups = 0;
    a.sk_units = 0;
    a.sk_cnt = nullptr;
    a.sk_part = nullptr;
    a.dimg = make_fastdiv((uint32_t)(g.th * g.tw));
    a.dtw = make_fastdiv((uint32_t)g.tw);
    a.tab = tables_of(p);
    for (int r = 0; r < 6; ++r) {
        a.shrow[r] = 0;
        for (int b = 0; b < 6 && 6 * r + b < p->ntap; ++b) a.shrow[r] |= (uint32_t)(p->sh[6 * r + b] & 31) << (5 * b);
    }
    if (p->bits == 10) {
        if (p->m == 2) return launch_resident<K2F2_10, 2, MODE, 10>(p, g, layout, vq, y, aux, a, stream);
        switch (tap_kernel_for(p, g, MODE)) {
            case WINO_TAP_ROWS:
                if constexpr (MODE == 0) return launch_rows_wide(p, g, layout, vq, y, a, stream);
                break;
            case WINO_TAP_RESIDENT_64X32:
                return launch_resident<K2Big10, 4, MODE, 10>(p, g, layout, vq, y, aux, a, stream);
            case WINO_TAP_RESIDENT_16X16:
                if constexpr (MODE == 0)
                    return launch_resident<K2Small10, 4, MODE, 10>(p, g, layout, vq, y, aux, a, stream);
                break;
            default:
                break;
        }
        return launch_resident<K2Mid10, 4, MODE, 10>(p, g, layout, vq, y, aux, a, stream);
    }
    if (p->m == 2) return launch_resident<K2F2, 2, MODE>(p, g, layout, vq, y, aux, a, stream);
    switch (tap_kernel_for(p, g, MODE)) {
        case WINO_TAP_ROWS: {
            const long long rblocks = (long long)(p->cout_pad / KR_CO) * (g.t_pad / KR_TL);
            if (rblocks > 0x7fffffffll) return WINO_EUNSUPPORTED;
            a.nbco = p->cout_pad / KR_CO;
            a.nblocks = (int)rblocks;
            a.n_dp = (int)rblocks;
            SkPlan sk;
            if (MODE == 0 && sk_in_workspace(p, g, ws_bytes, sk)) {
                uint8_t* const ws = (uint8_t*)const_cast<int8_t*>(vq);
                a.n_dp = sk.n_dp;
                a.sk_groups = sk.groups;
                a.sk_units = sk.units;
                a.sk_cnt = (int*)(ws + sk.cnt_off);
                a.sk_part = (int*)(ws + sk.part_off);
            }
            const unsigned grid = (unsigned)(a.n_dp + a.sk_groups);
            if (a.sk_groups > 0) {
                if (layout == WINO_NHWC)
                    hipLaunchKernelGGL(wino_tap_gemm_rows_sk<WINO_NHWC>, dim3(grid), dim3(KR_THREADS), 0, stream,
                                       p->uq_dev, vq, p->bias_dev, y, a);
                else
                    hipLaunchKernelGGL(wino_tap_gemm_rows_sk<WINO_NCHW>, dim3(grid), dim3(KR_THREADS), 0, stream,
                                       p->uq_dev, vq, p->bias_dev, y, a);
            } else if (layout == WINO_NHWC) {
                hipLaunchKernelGGL(wino_tap_gemm_rows<WINO_NHWC>, dim3(grid), dim3(KR_THREADS), 0, stream, p->uq_dev,
                                   vq, p->bias_dev, y, a);
            } else {
                hipLaunchKernelGGL(wino_tap_gemm_rows<WINO_NCHW>, dim3(grid), dim3(KR_THREADS), 0, stream, p->uq_dev,
                                   vq, p->bias_dev, y, a);
            }
            return hipGetLastError() == hipSuccess ? WINO_OK : WINO_EHIP;
        }
        case WINO_TAP_WAVES: {
            const long long wblocks = (long long)(p->cout_pad / WS_CO) * (g.t_pad / WS_TL);
            if (wblocks > 0x7fffffffll) return WINO_EUNSUPPORTED;
            a.nbco = p->cout_pad / WS_CO;
            a.nblocks = (int)wblocks;
            // persistent: at most one workgroup per CU, each walking its blocks
            const dim3 grid((unsigned)std::min<long long>(wblocks, num_cus())), block(WS_THREADS);
#define WS_LAUNCH(L, NK) \
    hipLaunchKernelGGL((wino_tap_gemm_ws<L, NK>), grid, block, 0, stream, p->uq_dev, vq, p->bias_dev, y, a)
#define WS_LAUNCH_NK(L)                            \
    switch (ws_chunks_per_stage(p->cin_pad)) {     \
        case 4: WS_LAUNCH(L, 4); break;            \
        case 3: WS_LAUNCH(L, 3); break;            \
        case 2: WS_LAUNCH(L, 2); break;            \
        default: WS_LAUNCH(L, 1); break;           \
    }
            if constexpr (MODE == 0) {
                if (layout == WINO_NHWC) {
                    WS_LAUNCH_NK(WINO_NHWC);
                } else {
                    WS_LAUNCH_NK(WINO_NCHW);
                }
#undef WS_LAUNCH_NK
#undef WS_LAUNCH
                return hipGetLastError() == hipSuccess ? WINO_OK : WINO_EHIP;
            }
            break;
        }
        case WINO_TAP_RESIDENT_32X32:
            if constexpr (MODE == 0) return launch_resident<K2Mid, 4, MODE>(p, g, layout, vq, y, aux, a, stream);
            break;
        case WINO_TAP_RESIDENT_16X16:
            if constexpr (MODE == 0) return launch_resident<K2Small, 4, MODE>(p, g, layout, vq, y, aux, a, stream);
            break;
        default:
            break;
    }
    return launch_resident<K2Big, 4, MODE>(p, g, layout, vq, y, aux, a, stream);
}

wino_status check_common(const wino_f4_plan_s* p, const void* x, int32_t n, int32_t h, int32_t w,
                         wino_layout layout, Geometry& g) {
    if (!p || !x) return WINO_EINVAL;
    if (layout != WINO_NCHW && layout != WINO_NHWC) return WINO_EINVAL;
    // the plan's tables live on the device that was current when it was
    // made; a launch on another device would read them from the wrong one
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return WINO_EHIP;
    if (dev != p->device) return WINO_EINVAL;
    return geometry(n, h, w, p->m, g);
}

// K1 for the plan's transform and Winograd-domain width
template <int MODE>
wino_status run_k1(int m, int bits, const K1Args& a, wino_layout layout, const int8_t* x, int8_t* vq,
                   int* tapmax, hipStream_t stream) {
    if constexpr (MODE == 0) {
        if (bits == 10)
            return m == 2 ? launch_k1<2, MODE, 10>(a, layout, x, vq, tapmax, stream)
                          : launch_k1<4, MODE, 10>(a, layout, x, vq, tapmax, stream);
    }
    return m == 2 ? launch_k1<2, MODE>(a, layout, x, vq, tapmax, stream)
                  : launch_k1<4, MODE>(a, layout, x, vq, tapmax, stream);
}

int cexp_int(unsigned long long a, int bits = 8) {
    // smallest e >= 0 with a <= 2^(bits-1) * 2^e (callers clamp at 0 anyway)
    int e = 0;
    while (((unsigned __int128)1 << (bits - 1 + e)) < a) ++e;
    return e;
}

}  // namespace

extern "C" size_t wino_f4_workspace_bytes(wino_f4_plan_t p, int32_t n, int32_t h, int32_t w,
                                          wino_variant variant) {
    Geometry g;
    if (!p || geometry(n, h, w, p->m, g) != WINO_OK) return 0;
    if (variant == WINO_FUSED) return 0;
    SkPlan sk;
    return sk_plan_for(p, g, sk) ? sk.end : vq_bytes(p, g);
}

namespace {
// K1 arguments of a SPLIT launch; with a stream-K tap GEMM to follow, K1
// also zeroes its counters
K1Args split_k1_args(const wino_f4_plan_s* p, const Geometry& g, void* ws, size_t ws_bytes) {
    K1Args a = k1_args(g, p->cin, p->cin_pad, tables_of(p), p->bits);
    SkPlan sk;
    if (sk_in_workspace(p, g, ws_bytes, sk)) {
        a.sk_cnt = (int*)((uint8_t*)ws + sk.cnt_off);
        a.sk_ncnt = sk.nsplit;
    }
    return a;
}
}  // namespace

// FUSED is served by the kernel in wino_fused.hip.
wino_status wino_f4_conv_fused(const wino_f4_plan_s* p, const int8_t* x, int8_t* y, int n, int h, int w,
                               wino_layout layout, hipStream_t stream);

extern "C" wino_status wino_select_algorithm(int32_t n, int32_t cin, int32_t cout, int32_t h, int32_t w,
                                             wino_layout layout, int32_t* algo) {
    if (!algo || n < 0 || h < 0 || w < 0 || cin < 1 || cout < 1) return WINO_EINVAL;
    if (layout != WINO_NCHW && layout != WINO_NHWC) return WINO_EINVAL;
    const double ops = 2.0 * 9 * (double)n * h * w * (double)cin * cout;
    // direct only in NHWC: small NCHW layers (Cin not a multiple of 64, or
    // W not a multiple of 4) run the simple MFMA kernel, which F2 beats
    // (C1: 12.3 against 31 us), and the NCHW tile kernel's byte transposes
    // leave it behind the Winograd paths on the large layers
    if (ops < (double)(1 << 27) && layout == WINO_NHWC) {
        *algo = WINO_ALGO_DIRECT;
        return WINO_OK;
    }
    const long long tiles4 = (long long)n * ((h + 3) / 4) * ((w + 3) / 4);
    const long long blocks = (long long)((cout + KR_CO - 1) / KR_CO) * ((tiles4 + KR_TL - 1) / KR_TL);
    *algo = blocks >= num_cus() ? WINO_ALGO_F4 : WINO_ALGO_F2;
    return WINO_OK;
}

extern "C" wino_status wino_f4_tap_kernel_choice(wino_f4_plan_t p, int32_t n, int32_t h, int32_t w,
                                                 int32_t* kind) {
    if (!p || !kind) return WINO_EINVAL;
    Geometry g;
    const wino_status st = geometry(n, h, w, p->m, g);
    if (st != WINO_OK) return st;
    *kind = tap_kernel_for(p, g, 0);
    SkPlan sk;
    if (*kind == WINO_TAP_ROWS && sk_plan_for(p, g, sk)) *kind = WINO_TAP_ROWS_STREAMK;
    return WINO_OK;
}

extern "C" wino_status wino_f4_conv_int8(wino_f4_plan_t p, const int8_t* x, int8_t* y, int32_t n,
                                         int32_t h, int32_t w, wino_layout layout, wino_variant variant,
                                         void* ws, size_t ws_bytes, hipStream_t stream) {
    Geometry g;
    wino_status st = check_common(p, x, n, h, w, layout, g);
    if (st != WINO_OK) return st;
    if (!y) return WINO_EINVAL;
    if (variant != WINO_SPLIT && variant != WINO_FUSED) return WINO_EINVAL;
    if (g.ntiles == 0) return WINO_OK;
    if (variant == WINO_FUSED) {
        if (p->bits != 8) return WINO_EUNSUPPORTED;
        return wino_f4_conv_fused(p, x, y, n, h, w, layout, stream);
    }
    if (!ws || ws_bytes < vq_bytes(p, g)) return WINO_EWORKSPACE;
    int8_t* vq = (int8_t*)ws;
    st = run_k1<0>(p->m, p->bits, split_k1_args(p, g, ws, ws_bytes), layout, x, vq, nullptr, stream);
    if (st != WINO_OK) return st;
    return launch_k2<0>(p, g, layout, vq, y, nullptr, stream, ws_bytes);
}

// ---------------------------------------------------------------------------
// The SPLIT convolution without allocation: the input-transform workspace
// (Vq) lives in a file-scope device array instead of caller memory.  Each
// device holds its own copy of the array for the life of the process; its
// address is looked up once per device (first call on that device, with the
// device current) and kept.
// ---------------------------------------------------------------------------
static __device__ __align__(256) uint8_t scratch[WINO_NOALLOC_SCRATCH_BYTES];

namespace {
std::mutex g_scratch_mu;
std::atomic<void*> g_scratch_ptr[64];   // per device id

wino_status scratch_for_device(int dev, void** out) {
    if (dev < 0 || dev >= 64) return WINO_EUNSUPPORTED;
    void* q = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (!q) {
        std::lock_guard<std::mutex> lk(g_scratch_mu);
        q = g_scratch_ptr[dev].load(std::memory_order_relaxed);
        if (!q) {
            // the device current now is `dev` (the caller checked it)
            if (hipGetSymbolAddress(&q, HIP_SYMBOL(scratch)) != hipSuccess || !q) return WINO_EHIP;
            g_scratch_ptr[dev].store(q, std::memory_order_release);
        }
    }
    *out = q;
    return WINO_OK;
}
}  // namespace

extern "C" wino_status wino_f4_conv_int8_noalloc(wino_f4_plan_t p, const int8_t* x, int8_t* y, int32_t n,
                                                 int32_t h, int32_t w, wino_layout layout, hipStream_t stream) {
    Geometry g;
    wino_status st = check_common(p, x, n, h, w, layout, g);
    if (st != WINO_OK) return st;
    if (!y) return WINO_EINVAL;
    if (g.ntiles == 0) return WINO_OK;
    if (vq_bytes(p, g) > (size_t)WINO_NOALLOC_SCRATCH_BYTES) return WINO_EWORKSPACE;
    void* ws = nullptr;
    st = scratch_for_device(p->device, &ws);
    if (st != WINO_OK) return st;
    // K1 writes every Vq byte that K2 reads into a nonzero product (padded
    // channels meet zero Uq rows, padded tiles are never stored), so the
    // scratch needs no clearing between calls
    int8_t* vq = (int8_t*)ws;
    st = run_k1<0>(p->m, p->bits, k1_args(g, p->cin, p->cin_pad, tables_of(p), p->bits), layout, x, vq, nullptr, stream);
    if (st != WINO_OK) return st;
    return launch_k2<0>(p, g, layout, vq, y, nullptr, stream);
}

extern "C" wino_status wino_f4_input_transform(wino_f4_plan_t p, const int8_t* x, int32_t n, int32_t h,
                                               int32_t w, wino_layout layout, void* ws, size_t ws_bytes,
                                               hipStream_t stream) {
    Geometry g;
    wino_status st = check_common(p, x, n, h, w, layout, g);
    if (st != WINO_OK) return st;
    if (g.ntiles == 0) return WINO_OK;
    if (!ws || ws_bytes < vq_bytes(p, g)) return WINO_EWORKSPACE;
    return run_k1<0>(p->m, p->bits, split_k1_args(p, g, ws, ws_bytes), layout, x, (int8_t*)ws, nullptr, stream);
}

extern "C" wino_status wino_f4_tap_gemm(wino_f4_plan_t p, void* ws, size_t ws_bytes, int8_t* y, int32_t n,
                                        int32_t h, int32_t w, wino_layout layout, hipStream_t stream) {
    Geometry g;
    wino_status st = check_common(p, ws, n, h, w, layout, g);
    if (st != WINO_OK) return st;
    if (!y) return WINO_EINVAL;
    if (g.ntiles == 0) return WINO_OK;
    if (ws_bytes < vq_bytes(p, g)) return WINO_EWORKSPACE;
    return launch_k2<0>(p, g, layout, (const int8_t*)ws, y, nullptr, stream, ws_bytes);
}

// per-tap max |V| over the input and the exponents e_B = max(0, cexp(.)) for
// bits-wide input taps
static wino_status calibrate_input(int m, int bits, const int8_t* x, int32_t n, int32_t cin, int32_t h,
                                   int32_t w, wino_layout layout, int32_t* absmax, int8_t* e_b,
                                   hipStream_t stream) {
    if (!x || cin < 1) return WINO_EINVAL;
    if (cin > 65536) return WINO_EUNSUPPORTED;
    if (layout != WINO_NCHW && layout != WINO_NHWC) return WINO_EINVAL;
    Geometry g;
    wino_status st = geometry(n, h, w, m, g);
    if (st != WINO_OK) return st;
    const int ntap = (m + 2) * (m + 2);
    int host[kTaps] = {0};
    if (g.ntiles > 0) {
        int* dmax = nullptr;
        if (hipMalloc(&dmax, sizeof(int) * kTaps) != hipSuccess) return WINO_ENOMEM;
        TapTables tab = {};
        bool ok = hipMemsetAsync(dmax, 0, sizeof(int) * kTaps, stream) == hipSuccess;
        if (ok) ok = run_k1<1>(m, 8, k1_args(g, cin, (int)round_up(cin, kKStep), tab), layout, x, nullptr, dmax,
                               stream) == WINO_OK;
        if (ok) ok = hipMemcpyAsync(host, dmax, sizeof(int) * kTaps, hipMemcpyDeviceToHost, stream) == hipSuccess;
        if (ok) ok = hipStreamSynchronize(stream) == hipSuccess;
        (void)hipFree(dmax);
        if (!ok) return WINO_EHIP;
    }
    for (int t = 0; t < ntap; ++t) {
        if (absmax) absmax[t] = host[t];
        if (e_b) {
            int e = cexp_int((unsigned long long)host[t], bits);
            e_b[t] = (int8_t)(e > 15 ? 15 : e);
        }
    }
    return WINO_OK;
}

extern "C" wino_status wino_f4_calibrate_input(const int8_t* x, int32_t n, int32_t cin, int32_t h, int32_t w,
                                               wino_layout layout, int32_t* absmax, int8_t* e_b,
                                               hipStream_t stream) {
    return calibrate_input(4, 8, x, n, cin, h, w, layout, absmax, e_b, stream);
}

extern "C" wino_status wino_f4_calibrate_input_i10(const int8_t* x, int32_t n, int32_t cin, int32_t h, int32_t w,
                                                   wino_layout layout, int32_t* absmax, int8_t* e_b,
                                                   hipStream_t stream) {
    return calibrate_input(4, 10, x, n, cin, h, w, layout, absmax, e_b, stream);
}

extern "C" wino_status wino_f2_calibrate_input_i10(const int8_t* x, int32_t n, int32_t cin, int32_t h, int32_t w,
                                                   wino_layout layout, int32_t* absmax, int8_t* e_b,
                                                   hipStream_t stream) {
    return calibrate_input(2, 10, x, n, cin, h, w, layout, absmax, e_b, stream);
}

extern "C" wino_status wino_f2_calibrate_input(const int8_t* x, int32_t n, int32_t cin, int32_t h, int32_t w,
                                               wino_layout layout, int32_t* absmax, int8_t* e_b,
                                               hipStream_t stream) {
    return calibrate_input(2, 8, x, n, cin, h, w, layout, absmax, e_b, stream);
}

extern "C" wino_status wino_f4_calibrate_output(wino_f4_plan_t p, const int8_t* x, int32_t n, int32_t h,
                                                int32_t w, wino_layout layout, void* ws, size_t ws_bytes,
                                                int64_t* zmax, int32_t* out_shift, hipStream_t stream) {
    Geometry g;
    wino_status st = check_common(p, x, n, h, w, layout, g);
    if (st != WINO_OK) return st;
    unsigned long long host = 0;
    if (g.ntiles > 0) {
        if (!ws || ws_bytes < vq_bytes(p, g)) return WINO_EWORKSPACE;
        unsigned long long* dmax = nullptr;
        if (hipMalloc(&dmax, sizeof(unsigned long long)) != hipSuccess) return WINO_ENOMEM;
        bool ok = hipMemsetAsync(dmax, 0, sizeof(unsigned long long), stream) == hipSuccess;
        if (ok) ok = run_k1<0>(p->m, p->bits, k1_args(g, p->cin, p->cin_pad, tables_of(p), p->bits), layout, x, (int8_t*)ws,
                               nullptr, stream) == WINO_OK;
        if (ok) ok = launch_k2<1>(p, g, layout, (const int8_t*)ws, nullptr, dmax, stream) == WINO_OK;
        if (ok) ok = hipMemcpyAsync(&host, dmax, sizeof(host), hipMemcpyDeviceToHost, stream) == hipSuccess;
        if (ok) ok = hipStreamSynchronize(stream) == hipSuccess;
        (void)hipFree(dmax);
        if (!ok) return WINO_EHIP;
    }
    if (zmax) *zmax = (int64_t)host;
    if (out_shift) *out_shift = cexp_int(host);
    return WINO_OK;
}

extern "C" wino_status wino_f4_debug_input_transform(wino_f4_plan_t p, const int8_t* x, int32_t n, int32_t h,
                                                     int32_t w, wino_layout layout, int8_t* vq_out, void* ws,
                                                     size_t ws_bytes, hipStream_t stream) {
    Geometry g;
    wino_status st = check_common(p, x, n, h, w, layout, g);
    if (st != WINO_OK) return st;
    if (!vq_out) return WINO_EINVAL;
    if (g.ntiles == 0) return WINO_OK;
    if (!ws || ws_bytes < vq_bytes(p, g)) return WINO_EWORKSPACE;
    st = run_k1<0>(p->m, p->bits, k1_args(g, p->cin, p->cin_pad, tables_of(p), p->bits), layout, x, (int8_t*)ws, nullptr, stream);
    if (st != WINO_OK) return st;
    // compact [ntap][cin_pad/kpr][t_pad][kpr] -> [ntap][ntiles][cin] (elements
    // of es bytes: int8, or fp16 for 10-bit plans), one 2-D copy per (tap, k row)
    const size_t es = kbytes_per_channel(p->bits);
    const int kpr = kKStep / (int)es;                      // channels per 64-byte k row
    const int nkb = p->cin_pad / kpr;
    for (int t = 0; t < p->ntap; ++t)
        for (int b = 0; b < nkb; ++b) {
            const int width = std::min(kpr, p->cin - b * kpr);
            if (width <= 0) break;
            if (hipMemcpy2DAsync(vq_out + es * ((size_t)t * g.ntiles * p->cin + (size_t)b * kpr), es * p->cin,
                                 (const int8_t*)ws + ((size_t)t * nkb + b) * g.t_pad * kKStep, (size_t)kKStep,
                                 es * width, (size_t)g.ntiles, hipMemcpyDeviceToDevice, stream) != hipSuccess)
                return WINO_EHIP;
        }
    return WINO_OK;
}

extern "C" wino_status wino_f4_debug_tap_gemm(wino_f4_plan_t p, const int8_t* x, int32_t n, int32_t h,
                                              int32_t w, wino_layout layout, int32_t* m_out, void* ws,
                                              size_t ws_bytes, hipStream_t stream) {
    Geometry g;
    wino_status st = check_common(p, x, n, h, w, layout, g);
    if (st != WINO_OK) return st;
    if (!m_out) return WINO_EINVAL;
    if (g.ntiles == 0) return WINO_OK;
    if (!ws || ws_bytes < vq_bytes(p, g)) return WINO_EWORKSPACE;
    st = run_k1<0>(p->m, p->bits, k1_args(g, p->cin, p->cin_pad, tables_of(p), p->bits), layout, x, (int8_t*)ws, nullptr, stream);
    if (st != WINO_OK) return st;
    return launch_k2<2>(p, g, layout, (const int8_t*)ws, nullptr, m_out, stream);
}
