// Device code shared by the input-transform, tap-GEMM and fused kernels:
// the F(4x4,3x3) transforms of Sec. II in integer form, the tap-wise
// requantization of Sec. III, the fused output-transform epilogue, and the
// LDS / barrier / wait helpers of the operand rings.
#pragma once
#include <type_traits>
#include "winof4_internal.h"

namespace winof4 {

typedef short v2s __attribute__((ext_vector_type(2)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));
typedef unsigned v2u __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef _Float16 v2h __attribute__((ext_vector_type(2)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));

__device__ __forceinline__ v2s splat(int v) { return (v2s){(short)v, (short)v}; }

// sign-extended bytes 0 and 2 of w as two 16-bit lanes
__device__ __forceinline__ v2s lanes_even(uint32_t w) {
    return __builtin_bit_cast(v2s, __builtin_amdgcn_perm(0u, w, 0x020c000cu)) >> splat(8);
}
// sign-extended bytes 1 and 3 of w
__device__ __forceinline__ v2s lanes_odd(uint32_t w) { return __builtin_bit_cast(v2s, w) >> splat(8); }

// One-dimensional B^T transform of a 6-vector, twelve additions with shared
// subexpressions; the rows of B^T (Sec. II) are
//   4 0 -5 0 1 0 / 0 -4 -4 1 1 0 / 0 4 -4 -1 1 0 / 0 -2 -1 2 1 0 /
//   0 2 -1 -2 1 0 / 0 4 0 -5 0 1.
template <class T>
__device__ __forceinline__ void bt_1d(const T* v, T* r, T two, T four);

// d = a * b + c in each 16-bit lane (v_pk_mad_i16; the compiler would emit a
// shift and an add for each multiply-add by 2 or 4).
__device__ __forceinline__ v2s pk_mad(v2s a, v2s b, v2s c) {
    v2s d;
    asm("v_pk_mad_i16 %0, %1, %2, %3" : "=v"(d) : "v"(a), "s"(b), "v"(c));
    return d;
}

// The B^T row pass on packed 16-bit lanes with one multiply-add per product:
// the same values as the generic form below, 12 instructions instead of 18.
template <>
__device__ __forceinline__ void bt_1d<v2s>(const v2s* v, v2s* r, v2s two, v2s four) {
    const v2s m4 = -four, m2 = -two;
    const v2s a = pk_mad(v[2], m4, v[4]);   // v4 - 4 v2
    const v2s nb = pk_mad(v[1], m4, v[3]);  // v3 - 4 v1 = -b
    const v2s c = v[4] - v[2];
    const v2s d = v[1] - v[3];
    const v2s e = v[0] - v[2];
    const v2s f = v[5] - v[3];
    r[0] = pk_mad(e, four, c);
    r[1] = a + nb;
    r[2] = a - nb;
    r[3] = pk_mad(d, m2, c);
    r[4] = pk_mad(d, two, c);
    r[5] = pk_mad(d, four, f);
}

template <class T>
__device__ __forceinline__ void bt_1d(const T* v, T* r, T two, T four) {
    T a = v[4] - four * v[2];
    T b = four * v[1] - v[3];
    T c = v[4] - v[2];
    T d = v[1] - v[3];
    T e = v[0] - v[2];
    T f = v[5] - v[3];
    r[0] = four * e + c;
    r[1] = a - b;
    r[2] = a + b;
    r[3] = c - two * d;
    r[4] = c + two * d;
    r[5] = four * d + f;
}

// Tap-wise requantization of tap t (Sec. III, power-of-two scale 2^e_B):
// clamp(R(V / 2^e), -128, 127) with R(v) = floor(v + 1/2), for the four
// channels, packed back into one word (channel k in byte k).
// rnd2 = the rounding constant 2^(e-1) (0 for e = 0) in both 16-bit halves,
// precomputed per tap on the host.
__device__ __forceinline__ uint32_t requant_pack(v2s ev, v2s od, int e, uint32_t rnd2) {
    const v2s rnd = __builtin_bit_cast(v2s, rnd2);
    const v2s sh = splat(e);
    v2s a = (ev + rnd) >> sh;
    v2s b = (od + rnd) >> sh;
    a = __builtin_elementwise_min(__builtin_elementwise_max(a, splat(-128)), splat(127));
    b = __builtin_elementwise_min(__builtin_elementwise_max(b, splat(-128)), splat(127));
    // bytes: ch0 = a.lo, ch1 = b.lo, ch2 = a.hi, ch3 = b.hi
    return __builtin_amdgcn_perm(__builtin_bit_cast(uint32_t, b), __builtin_bit_cast(uint32_t, a), 0x06020400u);
}

// The int8/10 variant: requantize four channels to 10 bits ([-512, 511])
// and store them as fp16, which holds every such integer exactly.
// Halves: ch0 = a.x, ch1 = b.x, ch2 = a.y, ch3 = b.y (the channel order of
// requant_pack).
__device__ __forceinline__ uint2 requant10_pack(v2s ev, v2s od, int e, uint32_t rnd2) {
    const v2s rnd = __builtin_bit_cast(v2s, rnd2);
    const v2s sh = splat(e);
    v2s a = (ev + rnd) >> sh;
    v2s b = (od + rnd) >> sh;
    a = __builtin_elementwise_min(__builtin_elementwise_max(a, splat(-512)), splat(511));
    b = __builtin_elementwise_min(__builtin_elementwise_max(b, splat(-512)), splat(511));
    const v2h lo = {(_Float16)a.x, (_Float16)b.x};
    const v2h hi = {(_Float16)a.y, (_Float16)b.y};
    return make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
}

// R(v / 2^e) clamped to Q bits with one instruction per pair of lanes, for
// e <= 16 - Q: x = v * 2^(16-Q-e) + 2^(15-Q) (the rounding constant 2^(e-1)
// scaled alike; 0 for e = 0) is formed at full width and saturated to int16
// by v_pk_mad_i16's clamp, and x >> (16 - Q) = floor((v + 2^(e-1)) / 2^e)
// clamped to [-2^(Q-1), 2^(Q-1) - 1] (for Q = 8: the high byte of each lane).
// scale2 / add2: 2^(16-Q-e) and the scaled rounding constant in both halves.
// (s: a wave-uniform multiplier, read from a scalar register)
__device__ __forceinline__ uint32_t pk_mad_sat(uint32_t a, uint32_t s, uint32_t c) {
    uint32_t r;
    asm("v_pk_mad_i16 %0, %1, %2, %3 clamp" : "=v"(r) : "v"(a), "s"(s), "v"(c));
    return r;
}
__device__ __forceinline__ uint32_t requant_pack_sat(v2s ev, v2s od, uint32_t scale2, uint32_t add2) {
    const uint32_t a = pk_mad_sat(__builtin_bit_cast(uint32_t, ev), scale2, add2);
    const uint32_t b = pk_mad_sat(__builtin_bit_cast(uint32_t, od), scale2, add2);
    // high bytes: ch0 = a.lo, ch1 = b.lo, ch2 = a.hi, ch3 = b.hi
    return __builtin_amdgcn_perm(b, a, 0x07030501u);
}
__device__ __forceinline__ uint2 requant10_pack_sat(v2s ev, v2s od, uint32_t scale2, uint32_t add2) {
    const v2s a = __builtin_bit_cast(v2s, pk_mad_sat(__builtin_bit_cast(uint32_t, ev), scale2, add2)) >> splat(6);
    const v2s b = __builtin_bit_cast(v2s, pk_mad_sat(__builtin_bit_cast(uint32_t, od), scale2, add2)) >> splat(6);
    const v2h lo = {(_Float16)a.x, (_Float16)b.x};
    const v2h hi = {(_Float16)a.y, (_Float16)b.y};
    return make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
}

// median of three (clamp a to [lo, hi]) in one instruction
__device__ __forceinline__ int med3_i32(int a, int lo, int hi) {
    int r;
    asm("v_med3_i32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(lo), "v"(hi));
    return r;
}

// word w with byte k replaced by the low byte of b
template <int K>
__device__ __forceinline__ uint32_t put_byte(uint32_t w, uint32_t b) {
    constexpr uint32_t sel = K == 0 ? 0x07060500u : K == 1 ? 0x07060004u : K == 2 ? 0x07000504u : 0x00060504u;
    return __builtin_amdgcn_perm(w, b, sel);
}

// One-dimensional A^T transform of a 6-vector (rows of A^T, Sec. II:
// 1 1 1 1 1 0 / 0 1 -1 2 -2 0 / 0 1 1 4 4 0 / 0 1 -1 8 -8 1).
template <class T>
__device__ __forceinline__ void at_1d(const T* v, T* y) {
    T p = v[1] + v[2], m = v[1] - v[2], q = v[3] + v[4], r = v[3] - v[4];
    y[0] = v[0] + p + q;
    y[1] = m + (r << 1);
    y[2] = p + (q << 2);
    y[3] = m + (r << 3) + v[5];
}

// One-dimensional B^T and A^T transforms of F(2x2,3x3) (Sec. II: rows of
// B^T 1 0 -1 0 / 0 1 1 0 / 0 -1 1 0 / 0 1 0 -1, rows of A^T 1 1 1 0 /
// 0 1 -1 -1).
template <class T>
__device__ __forceinline__ void bt2_1d(const T* v, T* r) {
    r[0] = v[0] - v[2];
    r[1] = v[1] + v[2];
    r[2] = v[2] - v[1];
    r[3] = v[1] - v[3];
}
template <class T>
__device__ __forceinline__ void at2_1d(const T* v, T* y) {
    y[0] = v[0] + v[1] + v[2];
    y[1] = v[1] - v[2] - v[3];
}

// F(M x M, 3 x 3): N = M + 2 input rows per tile, NTAP = N^2 taps; bt / at
// are the one-dimensional transforms above.  Tap (1,1), t = N + 1, has an
// all-ones row and column of A^T for both, so a constant added to it reaches
// every output of the tile once (used for bias and the rounding constant).
template <int M>
struct Wino;
template <>
struct Wino<4> {
    static constexpr int N = 6, NTAP = 36;
    template <class T>
    __device__ static __forceinline__ void bt(const T* v, T* r, T two, T four) { bt_1d(v, r, two, four); }
    template <class T>
    __device__ static __forceinline__ void at(const T* v, T* y) { at_1d(v, y); }
};
template <>
struct Wino<2> {
    static constexpr int N = 4, NTAP = 16;
    template <class T>
    __device__ static __forceinline__ void bt(const T* v, T* r, T, T) { bt2_1d(v, r); }
    template <class T>
    __device__ static __forceinline__ void at(const T* v, T* y) { at2_1d(v, y); }
};

// V = B^T d B for four channels of one N x N tile.  wv[r][c] holds the int8
// values of the four channels at tile pixel (r, c), channel k in byte k.
// On return ev[r][c] holds V[r][c] of channels (0, 2) and od[r][c] of
// channels (1, 3), as 16-bit lanes: |V| <= 12768 for int8 inputs (F4; 512
// for F2) and the row-pass intermediates are at most 1278, so 16 bits hold
// everything.
template <int M, int N = Wino<M>::N>
__device__ __forceinline__ void input_tile_transform(const uint32_t (&wv)[N][N], v2s (&ev)[N][N], v2s (&od)[N][N]) {
#pragma unroll
    for (int r = 0; r < N; ++r)
#pragma unroll
        for (int c = 0; c < N; ++c) {
            ev[r][c] = lanes_even(wv[r][c]);
            od[r][c] = lanes_odd(wv[r][c]);
        }
    const v2s two = splat(2), four = splat(4);
    // columns: T1 = B^T d
#pragma unroll
    for (int c = 0; c < N; ++c) {
        v2s ve[N], vo[N], re[N], ro[N];
#pragma unroll
        for (int r = 0; r < N; ++r) {
            ve[r] = ev[r][c];
            vo[r] = od[r][c];
        }
        Wino<M>::bt(ve, re, two, four);
        Wino<M>::bt(vo, ro, two, four);
#pragma unroll
        for (int r = 0; r < N; ++r) {
            ev[r][c] = re[r];
            od[r][c] = ro[r];
        }
    }
    // rows: V = T1 B
#pragma unroll
    for (int r = 0; r < N; ++r) {
        v2s re[N], ro[N];
        Wino<M>::bt(ev[r], re, two, four);
        Wino<M>::bt(od[r], ro, two, four);
#pragma unroll
        for (int c = 0; c < N; ++c) {
            ev[r][c] = re[c];
            od[r][c] = ro[c];
        }
    }
}

// Consecutive workgroup ids are dispatched round robin over the 8 XCDs
// (workgroup i runs on XCD i % 8).  Remap so that each XCD works through one
// contiguous range of logical block ids, i.e. blocks with neighbouring ids
// share that XCD's L2.
// floor(n / f.d) for 0 <= n < 2^31 (FastDiv).
__device__ __forceinline__ uint32_t fast_div(uint32_t n, const winof4::FastDiv& f) {
    return f.d == 1 ? n : __umulhi(n, f.mul) >> f.shr;
}

// Image, tile row and tile column of a tile index (tiles < 2^26); G provides
// th, tw and the FastDivs dimg (th * tw) and dtw (tw).
template <class G>
__device__ __forceinline__ void tile_coords(long long tile, const G& g, int& img, int& ty, int& tx) {
    const uint32_t t = (uint32_t)tile;
    img = (int)fast_div(t, g.dimg);
    const uint32_t trem = t - (uint32_t)img * (uint32_t)(g.th * g.tw);
    ty = (int)fast_div(trem, g.dtw);
    tx = (int)(trem - (uint32_t)ty * (uint32_t)g.tw);
}

__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
    const int nx = 8;
    const int full = nblocks / nx * nx;
    if (bid >= full) return bid;
    return (bid % nx) * (full / nx) + bid / nx;
}

// 16-byte slot holding bytes [16p, 16p+16) of a 64-byte LDS row.  Measured
// on gfx950, this swizzle lets the MFMA fragment reads (16 rows x one 16-byte
// part per 16 lanes) run at the full 256 B/clk per CU; unswizzled or padded
// rows run 1.5x slower.
__device__ __forceinline__ int lds_slot(int row, int part) { return part ^ ((row >> 1) & 3); }

// Global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4) for a
// ring whose stages the caller waits for explicitly (s_waitcnt vmcnt(n), then
// a barrier).  Issued as inline assembly: with the builtin, the compiler has
// to assume that any later LDS read may overlap a copy still in flight, and
// it waits for every copy (vmcnt(0)) before each fragment read -- the copies
// of the ring's next stages included.  M0, the LDS destination, is an input
// operand the compiler sets; the s_nop is the one wait state an M0 write
// needs before an LDS-DMA load.
__device__ __forceinline__ void lds_copy16(const void* src, __attribute__((address_space(3))) void* dst) {
    const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)dst);
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(m0) : "memory");
}

// Workgroup barrier without the implicit wait for outstanding global loads
// that __syncthreads() carries: callers wait for exactly the loads they need
// with s_waitcnt.  The empty asm statements keep the compiler from moving
// LDS accesses across the barrier.
__device__ __forceinline__ void ring_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// s_waitcnt vmcnt(n), 0 <= n <= 63, leaving the other counters untouched
// (gfx9 encoding: vmcnt[3:0] and vmcnt[5:4] at bits 15:14, expcnt[6:4],
// lgkmcnt[11:8]).
#define WINO_VMCNT_BITS(n) ((((n) & 15)) | ((((n) >> 4) & 3) << 14))
#define WINO_WAIT_VM(n) __builtin_amdgcn_s_waitcnt(0x0f70 | WINO_VMCNT_BITS(n))
// the same, and also every LDS read of this wave returned (lgkmcnt 0): a
// ring stage's buffer is refilled right after the next barrier, so each wave
// must be done reading it before it arrives there
#define WINO_WAIT_VM_LDS(n) __builtin_amdgcn_s_waitcnt(0x0070 | WINO_VMCNT_BITS(n))

// Epilogue of a 16-channel x 16-tile MFMA block holding all NTAP taps of
// F(M x M, 3 x 3): the accumulator of tap t, register r, lane l is
// M_t[co_base + 4*(l/16) + r][tile tl_base + l%16].  Per output channel: align
// taps by 2^sh (exact), add bias and the rounding constant once through tap
// (1,1) (its row and column of A^T are all ones, so they reach every output
// of the tile once), apply Y = A^T M A in two separable passes, then shift,
// clamp, ReLU, crop, store.
// MODE 0: store y.  MODE 1: max |Y + bias| into *aux (calibration).
// MODE 2: store raw M to aux [NTAP][ntiles][cout] (debug export).
// G provides cout, h, w, th, tw, ntiles, out_shift, relu, tab.
template <int M, int LAYOUT, int EPI, int MODE, class G>
__device__ __forceinline__ void tap_epilogue(const v4i (&acc)[Wino<M>::NTAP], const G& g,
                                             const int32_t* __restrict__ bias, int8_t* __restrict__ y,
                                             void* __restrict__ aux, int co_base, long long tl_base, int lane) {
    typedef typename std::conditional<EPI == 64, long long, int>::type acc_t;
    constexpr int N = Wino<M>::N, NT = Wino<M>::NTAP;
    const int lr = lane & 15, lk = lane >> 4;
    const long long tile = tl_base + lr;
    const bool tile_ok = tile < g.ntiles;

    if (MODE == 2) {
        int32_t* m_out = (int32_t*)aux;
        if (!tile_ok) return;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int co = co_base + 4 * lk + r;
            if (co >= g.cout) continue;
#pragma unroll
            for (int t = 0; t < NT; ++t) m_out[((long long)t * g.ntiles + tile) * g.cout + co] = acc[t][r];
        }
        return;
    }

    const long long tt = tile_ok ? tile : 0;
    int img, ty, tx;
    tile_coords(tt, g, img, ty, tx);
    const int s = g.out_shift;
    const acc_t rnd = (MODE == 0 && s > 0) ? ((acc_t)1 << (s - 1)) : 0;
    const int lo = g.relu ? 0 : -128;
    unsigned long long zmax = 0;
    uint32_t packed[M * M];  // NHWC: 4 output channels per pixel
#pragma unroll
    for (int p = 0; p < M * M; ++p) packed[p] = 0;

#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int co = co_base + 4 * lk + r;
        // row pass one row of taps at a time, so only N widened values are
        // live besides the row results
        acc_t rp[N][M];
#pragma unroll
        for (int a = 0; a < N; ++a) {
            acc_t mv[N];
#pragma unroll
            for (int bb = 0; bb < N; ++bb) mv[bb] = (acc_t)acc[N * a + bb][r] << g.tab.sh[N * a + bb];
            if (a == 1) mv[1] += (acc_t)bias[co] + rnd;   // tap (1, 1)
            Wino<M>::at(mv, rp[a]);
        }
        acc_t yv[M][M];
#pragma unroll
        for (int jj = 0; jj < M; ++jj) {
            acc_t col[N], o[M];
#pragma unroll
            for (int a = 0; a < N; ++a) col[a] = rp[a][jj];
            Wino<M>::at(col, o);
#pragma unroll
            for (int i = 0; i < M; ++i) yv[i][jj] = o[i];
        }
        if (MODE == 1) {
            if (tile_ok && co < g.cout) {
#pragma unroll
                for (int i = 0; i < M; ++i)
#pragma unroll
                    for (int jj = 0; jj < M; ++jj)
                        if (M * ty + i < g.h && M * tx + jj < g.w) {
                            acc_t v = yv[i][jj];
                            unsigned long long av = (unsigned long long)(v < 0 ? -(long long)v : (long long)v);
                            zmax = av > zmax ? av : zmax;
                        }
            }
            continue;
        }
        int qv[M][M];
#pragma unroll
        for (int i = 0; i < M; ++i)
#pragma unroll
            for (int jj = 0; jj < M; ++jj) {
                if (EPI == 32) {
                    qv[i][jj] = med3_i32((int)(yv[i][jj] >> s), lo, 127);
                } else {
                    acc_t v = yv[i][jj] >> s;
                    v = v < (acc_t)lo ? (acc_t)lo : v;
                    v = v > (acc_t)127 ? (acc_t)127 : v;
                    qv[i][jj] = (int)v;
                }
            }
        if (LAYOUT == WINO_NCHW) {
            if (!tile_ok || co >= g.cout) continue;
            int8_t* base = y + (((long long)img * g.cout + co) * g.h + M * ty) * g.w + M * tx;
            const bool full_cols = (M * tx + M - 1 < g.w) && (g.w % M == 0);
#pragma unroll
            for (int i = 0; i < M; ++i) {
                if (M * ty + i >= g.h) continue;
                if (full_cols) {
                    if (M == 4) {
                        uint32_t wv = __builtin_amdgcn_perm((uint32_t)qv[i][1], (uint32_t)qv[i][0], 0x0c0c0400u) |
                                      (__builtin_amdgcn_perm((uint32_t)qv[i][M - 1], (uint32_t)qv[i][M - 2],
                                                             0x0c0c0400u) << 16);
                        *(uint32_t*)(base + (long long)i * g.w) = wv;
                    } else {
                        *(uint16_t*)(base + (long long)i * g.w) =
                            (uint16_t)__builtin_amdgcn_perm((uint32_t)qv[i][1], (uint32_t)qv[i][0], 0x0c0c0400u);
                    }
                } else {
#pragma unroll
                    for (int jj = 0; jj < M; ++jj)
                        if (M * tx + jj < g.w) base[(long long)i * g.w + jj] = (int8_t)qv[i][jj];
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < M; ++i)
#pragma unroll
                for (int jj = 0; jj < M; ++jj) {
                    uint32_t& pk = packed[M * i + jj];
                    const uint32_t q = (uint32_t)qv[i][jj];
                    pk = r == 0 ? put_byte<0>(pk, q) : r == 1 ? put_byte<1>(pk, q) : r == 2 ? put_byte<2>(pk, q)
                                                                                        : put_byte<3>(pk, q);
                }
        }
    }

    if (MODE == 1) {
        // wave reduction, then one atomic per wave
        for (int off = 32; off > 0; off >>= 1) {
            unsigned long long o = __shfl_xor(zmax, off, 64);
            zmax = o > zmax ? o : zmax;
        }
        if (lane == 0) atomicMax((unsigned long long*)aux, zmax);
        return;
    }
    if (LAYOUT == WINO_NHWC && tile_ok) {
        const int co0 = co_base + 4 * lk;
        const long long rs = (long long)g.w * g.cout;
        int8_t* ob = y + (((long long)img * g.h + M * ty) * g.w + M * tx) * g.cout + co0;
        const bool full = (co0 + 3 < g.cout) && ((g.cout & 3) == 0) && (M * ty + M - 1 < g.h) &&
                          (M * tx + M - 1 < g.w);
        if (full) {
#pragma unroll
            for (int i = 0; i < M; ++i)
#pragma unroll
                for (int jj = 0; jj < M; ++jj) *(uint32_t*)(ob + i * rs + jj * g.cout) = packed[M * i + jj];
        } else {
#pragma unroll
            for (int i = 0; i < M; ++i)
#pragma unroll
                for (int jj = 0; jj < M; ++jj) {
                    if (M * ty + i >= g.h || M * tx + jj >= g.w) continue;
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (co0 + r < g.cout) ob[i * rs + jj * g.cout + r] = (int8_t)(packed[M * i + jj] >> (8 * r));
                }
        }
    }
}

}  // namespace winof4
