// Tap GEMM + output transform for F(4x4,3x3), int8 operands, 32-bit
// epilogue: the wave-specialized kernel wino_tap_gemm_ws.  Included by
// wino_kernels.hip inside its anonymous namespace (it uses K2Args,
// tile_coords, put_byte, med3_i32 and the ring helpers defined there).
//
// The work of a 64-channel x 64-tile block is split over two kinds of wave
// so that the matrix cores, the integer ALUs and the operand copies run at
// the same time instead of one after another:
//
//  * four MFMA waves, one per SIMD, each owning a 32 (channels) x 32 (tiles)
//    block: per tap t the 32x32x32 int8 MFMA accumulates M_t over the input
//    channels (Sec. III: M = sum_ci Vq Uq, exact in int32), and the wave then
//    folds the finished tap into the row-pass result of its row a of the 6x6
//    tile, z_a = (M' [a, :]) A with M' = M 2^sh (the alignment of S_BG by
//    exact left shifts), while the MFMAs of the next tap run.
//  * eight fold waves, two per SIMD: they issue the global -> LDS operand
//    copies of the ring, and each keeps two rows of the output tile of its
//    partner MFMA wave's pairs, adding A^T[i, a] z_a when the partner hands
//    over z_a through LDS at the end of each row of taps.
//
// Y = A^T M' A = sum_a A^T[:, a] z_a is linear in the taps, so streaming the
// taps in row order and folding each one as it completes gives the same
// exact integers as the output transform applied to all 36 taps at once
// (the bias and the rounding constant of the final shift start every output,
// as they would reach each output once through tap (1, 1)).
//
// Ring stage = one tap x NK 64-channel chunks: per chunk 64 Uq rows (output
// channels) and 64 Vq rows (tiles) of 64 bytes, 8 KB; four 32 KB buffers,
// copies issued three stages ahead (96 KB in flight).  One barrier per stage.  z_a is handed over in two halves (j = 0, 1 in the
// first stage of the next row, j = 2, 3 two stages later: the next row's
// first fold only touches j = 0, its second rewrites j = 1..3), so the
// hand-over buffer is 8 KB per MFMA wave: 128 + 32 = 160 KB of LDS.
//
// Persistent: workgroup p runs the blocks p, p + G, p + 2G, ... (G = grid
// size, at most one workgroup per CU) with one continuous copy ring, so the
// next block's operands stream in while the current one finishes; z_5 of a
// block is handed over in the first stages of the next block, and the fold
// waves requantize and store a block's outputs straight from registers while
// the next block's first taps run.  (A block-per-workgroup launch paid the
// ring's start-up latency and the output store burst once per round of
// blocks: ~8-10 us of C5's tap GEMM.)
//
// MFMA orientation: A = Uq (rows = output channels), B = Vq (columns =
// tiles), so lane l holds tile l % 32 and, in accumulator register r, output
// channel 8 (r / 4) + 4 (l / 32) + r % 4 of the wave's 32.
//
// Measured, it is slower than the row-streamed kernel (C5: 58 against 47 us;
// C4: 28 against 20 us): its copies run at the same ~25 B/clk per CU as the
// row-streamed ring's, and an MFMA wave and a fold wave on one SIMD mostly
// take turns rather than overlap.  The automatic choice never picks it; it is
// run only when forced (WINO_TAP_WAVES).
// ---------------------------------------------------------------------------
constexpr int WS_CO = 64;
constexpr int WS_TL = 64;
constexpr int WS_WAVES = 12;
constexpr int WS_THREADS = 64 * WS_WAVES;
constexpr int WS_NBUF = 4;
constexpr int WS_BUF = 32 * 1024;
constexpr int WS_ZHALF = 8 * 1024;
constexpr int WS_LDS = WS_NBUF * WS_BUF + 4 * WS_ZHALF;
static_assert(WS_LDS <= 160 * 1024, "LDS");
static_assert((WS_NBUF & (WS_NBUF - 1)) == 0, "ring index by mask");
static_assert(kTilePad % WS_TL == 0 && kCoutPad % WS_CO == 0, "blocks tile the padded sizes");

typedef int v16i __attribute__((ext_vector_type(16)));

// LDS slot of 16-byte part p of row R (0..15) of a 1-KB block of 16 rows x
// 64 bytes: the 32x32x32 fragment read (lanes 0-15 rows 0-15 of one part)
// then touches every 16-byte bank group once (measured 1.7x the unswizzled
// rate on gfx950).
__device__ __forceinline__ int ws_slot(int r, int p) { return p ^ ((r >> 2) & 3); }

// z + v * 2^s in wrapping 32-bit arithmetic (v_lshl_add_u32)
__device__ __forceinline__ int shl_add(int v, int s, int z) { return (int)(((uint32_t)v << s) + (uint32_t)z); }

// y + c v for a constant c in {0, +-1, +-2, +-4, +-8} (the entries of A^T)
template <int C>
__device__ __forceinline__ int add_coef(int y, int v) {
    if constexpr (C == 0) return y;
    else if constexpr (C == 1) return y + v;
    else if constexpr (C == -1) return y - v;
    else if constexpr (C > 0) return shl_add(v, C == 2 ? 1 : C == 4 ? 2 : 3, y);
    else return shl_add(-v, C == -2 ? 1 : C == -4 ? 2 : 3, y);
}

// Materialize accumulators here: they are only read much later, and the
// compiler would otherwise sink the folds past later taps and keep several
// taps' accumulators live at once (spilling).
template <int N>
__device__ __forceinline__ void ws_pin(int (&v)[N][16]) {
#pragma unroll
    for (int j = 0; j < N; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) asm volatile("" : "+v"(v[j][r]));
}

// A^T of F(4x4,3x3) (Sec. II), entry (i, a), as a compile-time constant
template <int I, int A>
struct AtCoef {
    static constexpr int value = I == 0 ? (A < 5 ? 1 : 0)
                               : A == 0 ? 0
                               : A == 5 ? (I == 3 ? 1 : 0)
                               : A == 1 ? 1
                               : A == 2 ? (I == 2 ? 1 : -1)
                               : A == 3 ? (1 << I)
                               : (I == 2 ? 4 : -(1 << I));
};

template <int LAYOUT, int NK>
__global__ __launch_bounds__(WS_THREADS) void wino_tap_gemm_ws(const int8_t* __restrict__ uq,
                                                               const int8_t* __restrict__ vq,
                                                               const int32_t* __restrict__ bias,
                                                               int8_t* __restrict__ y, K2Args g) {
    __shared__ __attribute__((aligned(1024))) uint8_t lds[WS_LDS];
    constexpr int KS = 2 * NK;                      // 32-channel MFMA k-steps per stage
    // the arguments as scalars (no indexing into the argument block, which
    // would make the compiler copy it to scratch memory)
    const int nblocks = g.nblocks, nbco = g.nbco, cin_pad = g.cin_pad, cout_pad = g.cout_pad, cout = g.cout;
    const int hh = g.h, ww = g.w, s_out = g.out_shift, relu = g.relu;
    const long long ntiles = g.ntiles, t_pad = g.t_pad;
    const int G = gridDim.x;
    const int nblk = (nblocks - (int)blockIdx.x + G - 1) / G;   // blocks of this workgroup (>= 1)
    // output channel block and tile block of this workgroup's k-th block
    auto block_of = [&](int k, int& co_blk, long long& tl_blk) __attribute__((always_inline)) {
        const int lbid = xcd_remap((int)blockIdx.x + k * G, nblocks);
        co_blk = (lbid % nbco) * WS_CO;
        tl_blk = (long long)(lbid / nbco) * WS_TL;
    };
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wq = wave & 3;                        // MFMA wave, or the fold wave's partner
    const int wc = wq & 1, wt = wq >> 1;            // 32-channel half, 32-tile half
    const int hl = lane >> 5;
    const int nsl = cin_pad / (64 * NK);            // stages per tap
    const int nstage = 36 * nsl;                    // stages per block
    uint8_t* const zbuf = lds + WS_NBUF * WS_BUF + wq * WS_ZHALF;
    // z hand-over layout: [j of the half][q][lane] x 16 bytes (registers 4q .. 4q+3)
    auto zaddr = [&](int jj, int q) __attribute__((always_inline)) { return zbuf + ((jj * 4 + q) * 64 + lane) * 16; };

    if (wave < 4) {
        // ------------------------------ MFMA wave ------------------------------
        const int r16 = lane & 15, g16 = (lane & 31) >> 4;
        const int offA = (2 * wc + g16) * 1024 + r16 * 64;
        const int offB = (4 + 2 * wt + g16) * 1024 + r16 * 64;
        const int po0 = 16 * ws_slot(r16, hl), po1 = 16 * ws_slot(r16, 2 + hl);
        v16i acc0 = (v16i){}, acc1 = (v16i){};
        const uint32_t shr0 = g.shrow[0], shr1 = g.shrow[1], shr2 = g.shrow[2], shr3 = g.shrow[3],
                       shr4 = g.shrow[4], shr5 = g.shrow[5];
        auto shrow_of = [&](int a) __attribute__((always_inline)) {
            return a == 0 ? shr0 : a == 1 ? shr1 : a == 2 ? shr2 : a == 3 ? shr3 : a == 4 ? shr4 : shr5;
        };
        int z[4][16];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) z[j][r] = 0;
        // fold finished tap (a, b) of accumulator m into z, pairs r0 .. r1-1
        // (the row pass of Y = A^T M' A; column b of A^T: 0: (1,0,0,0),
        // 1: (1,1,1,1), 2: (1,-1,1,-1), 3: (1,2,4,8), 4: (1,-2,4,-8),
        // 5: (0,0,0,1))
        auto fold = [&](const v16i& m, auto bc, int sh, int r0, int r1) __attribute__((always_inline)) {
            constexpr int b = decltype(bc)::value;
#pragma unroll
            for (int r = r0; r < r1; ++r) {
                const int v = m[r];
                if constexpr (b == 0) {
                    z[0][r] = (int)((uint32_t)v << sh);
                } else if constexpr (b == 1) {
                    const int u = (int)((uint32_t)v << sh);
                    z[0][r] += u;
                    z[1][r] = u;
                    z[2][r] = u;
                    z[3][r] = u;
                } else if constexpr (b == 2) {
                    const int u = (int)((uint32_t)v << sh);
                    z[0][r] += u;
                    z[1][r] -= u;
                    z[2][r] += u;
                    z[3][r] -= u;
                } else if constexpr (b == 3) {
                    z[0][r] = shl_add(v, sh, z[0][r]);
                    z[1][r] = shl_add(v, sh + 1, z[1][r]);
                    z[2][r] = shl_add(v, sh + 2, z[2][r]);
                    z[3][r] = shl_add(v, sh + 3, z[3][r]);
                } else if constexpr (b == 4) {
                    const int nv = -v;
                    z[0][r] = shl_add(v, sh, z[0][r]);
                    z[1][r] = shl_add(nv, sh + 1, z[1][r]);
                    z[2][r] = shl_add(v, sh + 2, z[2][r]);
                    z[3][r] = shl_add(nv, sh + 3, z[3][r]);
                } else {
                    z[3][r] = shl_add(v, sh, z[3][r]);
                }
            }
        };
        // hand half h of z (j = 2h, 2h + 1) to the fold waves
        auto z_out = [&](int h) __attribute__((always_inline)) {
#pragma unroll
            for (int jj = 0; jj < 2; ++jj)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    *(v4i*)zaddr(jj, q) = (v4i){z[2 * h + jj][4 * q], z[2 * h + jj][4 * q + 1],
                                                z[2 * h + jj][4 * q + 2], z[2 * h + jj][4 * q + 3]};
        };
        int buf = 0;
        // One ring stage of tap (a, b): wait for the stage, then per 32-channel
        // k-step one MFMA, a share of the fold of the previous tap and the
        // fragment reads P k-steps ahead, each group fenced so the compiler
        // keeps that interleaving.  FIRST: the first stage of the tap (its
        // accumulator starts from zero; the fold and the hand-over of z
        // happen there).  NOPREV: the workgroup's very first row (nothing
        // finished before tap (0, 0) of its first block).  The tap before
        // (a, 0) is (a - 1, 5), for a = 0 tap (5, 5) of the previous block,
        // whose z_5 is handed over like z_{a-1}.
        auto stage = [&](auto bc, auto first_c, auto noprev_c, int a) __attribute__((always_inline)) {
            constexpr int b = decltype(bc)::value;
            constexpr bool FIRST = decltype(first_c)::value, NOPREV = decltype(noprev_c)::value;
            constexpr bool FOLD = FIRST && !(NOPREV && b == 0);
            constexpr int PB = b == 0 ? 5 : b - 1;
            // alignment shift of the folded tap: row a (b > 0) or the row before (b = 0)
            const int sh = FOLD ? (int)((shrow_of(b == 0 ? (a == 0 ? 5 : a - 1) : a) >> (5 * PB)) & 31u) : 0;
            v16i& acc = (b & 1) ? acc1 : acc0;
            const v16i& prev = (b & 1) ? acc0 : acc1;
            __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): this wave's LDS traffic done
            ring_barrier();
            const uint8_t* base = lds + buf * WS_BUF;
            buf = (buf + 1) & (WS_NBUF - 1);
            constexpr int P = KS < 4 ? KS : 4;
            v4i fa[P], fb[P];
            auto ld = [&](int ks) __attribute__((always_inline)) {
                const int c = ks >> 1, po = (ks & 1) ? po1 : po0;
                fa[ks % P] = *(const v4i*)(base + c * 8192 + offA + po);
                fb[ks % P] = *(const v4i*)(base + c * 8192 + offB + po);
            };
#pragma unroll
            for (int ks = 0; ks < P; ++ks) ld(ks);
            if constexpr (FIRST && !NOPREV && b == 0) {
                // j = 0, 1 of the finished row (the fold of its tap 5 only adds to j = 3)
                z_out(0);
            }
            if constexpr (FIRST && !NOPREV && b == 2) {
                // j = 2, 3 of the finished row, before the fold of tap (a, 1) rewrites them
                z_out(1);
            }
            __builtin_amdgcn_sched_barrier(0);
            const v16i zero = (v16i){};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[ks % P], fb[ks % P], (ks == 0 && FIRST) ? zero : acc,
                                                            0, 0, 0);
                if constexpr (FOLD) fold(prev, std::integral_constant<int, PB>{}, sh, 16 * ks / KS, 16 * (ks + 1) / KS);
                if (ks + P < KS) ld(ks + P);
                __builtin_amdgcn_sched_barrier(0);
            }
            // the fold completes within its stage
            if constexpr (FOLD) ws_pin(z);
        };
        using TT = std::true_type;
        using FF = std::false_type;
        auto tap = [&](auto bc, auto noprev_c, int a) __attribute__((always_inline)) {
            stage(bc, TT{}, noprev_c, a);
            for (int sl = 1; sl < nsl; ++sl) stage(bc, FF{}, noprev_c, a);
        };
        auto row = [&](auto noprev_c, int a) __attribute__((always_inline)) {
            tap(std::integral_constant<int, 0>{}, noprev_c, a);
            tap(std::integral_constant<int, 1>{}, noprev_c, a);
            tap(std::integral_constant<int, 2>{}, noprev_c, a);
            tap(std::integral_constant<int, 3>{}, noprev_c, a);
            tap(std::integral_constant<int, 4>{}, noprev_c, a);
            tap(std::integral_constant<int, 5>{}, noprev_c, a);
        };
        row(TT{}, 0);
        for (int a = 1; a < 6; ++a) row(FF{}, a);
        for (int k = 1; k < nblk; ++k)
            for (int a = 0; a < 6; ++a) row(FF{}, a);
        // the last block's tap (5, 5), then both halves of its z_5
        fold(acc1, std::integral_constant<int, 5>{}, (int)((shr5 >> 25) & 31u), 0, 16);
        z_out(0);
        __builtin_amdgcn_s_waitcnt(0xc07f);
        ring_barrier();
        ring_barrier();   // the fold waves have read j = 0, 1
        z_out(1);
        __builtin_amdgcn_s_waitcnt(0xc07f);
        ring_barrier();
    } else {
        // ------------------------------ fold wave ------------------------------
        const int fw = wave - 4;          // 0..7
        const int hf = fw >> 2;           // rows 2 hf, 2 hf + 1 of the output tile
        // copies: for every chunk of a stage, fold wave fw fetches 16-row
        // group fw of the stage's 8 KB chunk (groups 0-3: Uq rows co_blk +
        // 16 fw ..; 4-7: Vq rows tl_blk + 16 (fw - 4) ..), one 1-KB load;
        // lane l fetches the 16-byte part that the swizzle places at LDS
        // offset 16 l of the group (row l / 4, slot l % 4)
        const int rr = lane >> 2;
        const int lane_off = rr * 64 + 16 * ws_slot(rr, lane & 3);
        const bool cu = fw < 4;
        const long long kstride = cu ? (long long)cout_pad * 64 : t_pad * 64;
        // (wave-uniform base; the lane's offset is added at the load)
        auto src_of = [&](int k) __attribute__((always_inline)) {
            int co_blk;
            long long tl_blk;
            block_of(k, co_blk, tl_blk);
            const int8_t* p = cu ? uq + (long long)(co_blk + 16 * fw) * 64 : vq + (tl_blk + 16 * (fw - 4)) * 64;
            const uint64_t u = (uint64_t)p;
            return (const int8_t*)(((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(u >> 32)) << 32) |
                                   (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)u));
        };
        // the ring's source: the block of the stage being issued
        int ib = 0, is = 0;               // block and stage within it of the next issue
        const int8_t* isrc = src_of(0);
        auto issue = [&](int sglob) __attribute__((always_inline)) {
            uint8_t* d = lds + (sglob & (WS_NBUF - 1)) * WS_BUF + fw * 1024;
#pragma unroll
            for (int c = 0; c < NK; ++c)
                lds_copy16(isrc + ((long long)is * NK + c) * kstride + lane_off,
                           (__attribute__((address_space(3))) void*)(d + c * 8192));
            if (++is == nstage) {
                is = 0;
                if (++ib < nblk) isrc = src_of(ib);
            }
        };
        const int ntot = nblk * nstage;   // stages of the whole workgroup
        const int rnd = s_out > 0 ? 1 << (s_out - 1) : 0;
        const int lo = relu ? 0 : -128;
        int yv[2][4][16];                 // rows 2 hf, 2 hf + 1 of the output tile
        // bias plus the rounding constant of the final shift start every
        // output (Y + bias, then R(. / 2^out_shift)); output channels of
        // registers r = 4q + k: co_blk + 32 wc + 4 hl + 8q + k.  Loaded in
        // the stage before the block's first z arrives (row 0's), so it is
        // live for three stages only.
        v4i bv[4];
        auto load_bias = [&](int k) __attribute__((always_inline)) {
            int co_blk;
            long long tl_blk;
            block_of(k, co_blk, tl_blk);
#pragma unroll
            for (int q = 0; q < 4; ++q) bv[q] = *(const v4i*)(bias + co_blk + 32 * wc + 4 * hl + 8 * q);
        };
        // Y[i, j] += A^T[i, a] z_a[j] for the wave's rows i and half h of j;
        // for a = 0, Y[i, j] = bias + rounding constant + A^T[i, 0] z_0[j]
        auto take_z = [&](auto ac, auto hc) __attribute__((always_inline)) {
            constexpr int a = decltype(ac)::value, h = decltype(hc)::value;
#pragma unroll
            for (int jj = 0; jj < 2; ++jj)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const v4i zz = *(const v4i*)zaddr(jj, q);
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const int r = 4 * q + k, j = 2 * h + jj;
                        if constexpr (a == 0) {
                            yv[0][j][r] = bv[q][k] + rnd;
                            yv[1][j][r] = bv[q][k] + rnd;
                        }
                        if (hf == 0) {
                            yv[0][j][r] = add_coef<AtCoef<0, a>::value>(yv[0][j][r], zz[k]);
                            yv[1][j][r] = add_coef<AtCoef<1, a>::value>(yv[1][j][r], zz[k]);
                        } else {
                            yv[0][j][r] = add_coef<AtCoef<2, a>::value>(yv[0][j][r], zz[k]);
                            yv[1][j][r] = add_coef<AtCoef<3, a>::value>(yv[1][j][r], zz[k]);
                        }
                    }
                }
#pragma unroll
            for (int i = 0; i < 2; ++i) ws_pin(yv[i]);
        };
        // requantize and store rows 2 hf, 2 hf + 1 of block k's tiles:
        // out = clamp(Y >> out_shift, lo, 127), straight from registers
        // (NCHW: a word of four pixels per lane, adjacent lanes adjacent
        // tiles; NHWC: a word of four channels)
        auto store = [&](int k) __attribute__((always_inline)) {
            int co_blk;
            long long tl_blk;
            block_of(k, co_blk, tl_blk);
            const long long tile = tl_blk + 32 * wt + (lane & 31);
            if (tile >= ntiles) return;
            int img, ty, tx;
            tile_coords(tile, g, img, ty, tx);
            const int co_lane = co_blk + 32 * wc + 4 * hl;
            if (LAYOUT == WINO_NCHW) {
                const bool full_cols = (4 * tx + 3 < ww) && ((ww & 3) == 0);
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int co = co_lane + 8 * (r >> 2) + (r & 3);
                    if (co >= cout) continue;
                    int8_t* base = y + (((long long)img * cout + co) * hh + 4 * ty) * ww + 4 * tx;
#pragma unroll
                    for (int i = 0; i < 2; ++i) {
                        const int oy = 2 * hf + i;
                        if (4 * ty + oy >= hh) continue;
                        int v[4];
#pragma unroll
                        for (int j = 0; j < 4; ++j) v[j] = med3_i32(yv[i][j][r] >> s_out, lo, 127);
                        if (full_cols) {
                            const uint32_t wv = __builtin_amdgcn_perm((uint32_t)v[1], (uint32_t)v[0], 0x0c0c0400u) |
                                                (__builtin_amdgcn_perm((uint32_t)v[3], (uint32_t)v[2], 0x0c0c0400u)
                                                 << 16);
                            *(uint32_t*)(base + (long long)oy * ww) = wv;
                        } else {
#pragma unroll
                            for (int j = 0; j < 4; ++j)
                                if (4 * tx + j < ww) base[(long long)oy * ww + j] = (int8_t)v[j];
                        }
                    }
                }
            } else {
                // NHWC: lane l (< 32) holds channels {0-3, 8-11, 16-19, 24-27} of
                // its 32, lane l + 32 (the same tile) {4-7, 12-15, ...}: two
                // permlane32 swaps give lane l channels 0-15 and lane l + 32
                // channels 16-31, one 16-byte store each
                const long long rs = (long long)ww * cout;
                const bool vec = (cout & 15) == 0 && ((uintptr_t)y & 15) == 0;
                const int cv = co_blk + 32 * wc + 16 * hl;      // the lane's first channel after the swaps
                int8_t* ob = y + (((long long)img * hh + 4 * ty) * ww + 4 * tx) * cout;
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    const int oy = 2 * hf + i;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        uint32_t d[4];
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            uint32_t pk = put_byte<0>(0u, (uint32_t)med3_i32(yv[i][j][4 * q] >> s_out, lo, 127));
                            pk = put_byte<1>(pk, (uint32_t)med3_i32(yv[i][j][4 * q + 1] >> s_out, lo, 127));
                            pk = put_byte<2>(pk, (uint32_t)med3_i32(yv[i][j][4 * q + 2] >> s_out, lo, 127));
                            d[q] = put_byte<3>(pk, (uint32_t)med3_i32(yv[i][j][4 * q + 3] >> s_out, lo, 127));
                        }
                        const bool inside = 4 * ty + oy < hh && 4 * tx + j < ww;
                        int8_t* o = ob + oy * rs + (long long)j * cout;
                        if (vec) {
                            const v2u s02 = __builtin_amdgcn_permlane32_swap(d[0], d[2], false, false);
                            const v2u s13 = __builtin_amdgcn_permlane32_swap(d[1], d[3], false, false);
                            if (inside && cv < cout)
                                *(uint4*)(o + cv) = make_uint4(s02[0], s02[1], s13[0], s13[1]);
                        } else if (inside) {
#pragma unroll
                            for (int q = 0; q < 4; ++q) {
                                const int co0 = co_lane + 8 * q;
                                if (co0 + 3 < cout && (cout & 3) == 0) {
                                    *(uint32_t*)(o + co0) = d[q];
                                } else {
#pragma unroll
                                    for (int kk = 0; kk < 4; ++kk)
                                        if (co0 + kk < cout) o[co0 + kk] = (int8_t)(d[q] >> (8 * kk));
                                }
                            }
                        }
                    }
                }
            }
        };
        int s = 0;                        // next stage to wait for (workgroup-wide count)
        auto fstage = [&]() __attribute__((always_inline)) {
            // stage s landed once only the later stages' loads are pending
            if (s + 2 < ntot)
                WINO_WAIT_VM(2 * NK);
            else if (s + 1 < ntot)
                WINO_WAIT_VM(NK);
            else
                WINO_WAIT_VM(0);
            ring_barrier();
            if (s + WS_NBUF - 1 < ntot) issue(s + WS_NBUF - 1);
            ++s;
        };
        // prologue: stages 0 .. NBUF-2 in flight
        for (int k = 0; k < WS_NBUF - 1 && k < ntot; ++k) issue(k);
        // z of the finished row: j = 0, 1 written in the first stage of the
        // next row's tap 0, read in the first stage of its tap 1; j = 2, 3
        // written in the first stage of tap 2, read in the first stage of tap
        // 3.  Row "a - 1" of row 0 is row 5 of the previous block: after its
        // j = 2, 3 that block's Y is complete and is stored while the next
        // taps run, then Y restarts from the new block's bias.
        auto row = [&](auto ac, int k) __attribute__((always_inline)) {
            constexpr int a = decltype(ac)::value;
            constexpr int pa = a == 0 ? 5 : a - 1;            // the finished row
            fstage();                                         // tap (a, 0)
            if (a == 1) load_bias(k);
            for (int kk = 1; kk < nsl; ++kk) fstage();
            fstage();                                         // tap (a, 1)
            if (a > 0 || k > 0) take_z(std::integral_constant<int, pa>{}, std::integral_constant<int, 0>{});
            for (int kk = 1; kk < nsl; ++kk) fstage();
            for (int kk = 0; kk < nsl; ++kk) fstage();        // tap (a, 2)
            fstage();                                         // tap (a, 3)
            if (a > 0 || k > 0) take_z(std::integral_constant<int, pa>{}, std::integral_constant<int, 1>{});
            if (a == 0 && k > 0) store(k - 1);
            for (int kk = 1; kk < nsl; ++kk) fstage();
            for (int kk = 0; kk < 2 * nsl; ++kk) fstage();    // taps (a, 4), (a, 5)
        };
        for (int k = 0; k < nblk; ++k) {
            row(std::integral_constant<int, 0>{}, k);
            row(std::integral_constant<int, 1>{}, k);
            row(std::integral_constant<int, 2>{}, k);
            row(std::integral_constant<int, 3>{}, k);
            row(std::integral_constant<int, 4>{}, k);
            row(std::integral_constant<int, 5>{}, k);
        }
        ring_barrier();   // the last block's z_5, j = 0, 1 written
        take_z(std::integral_constant<int, 5>{}, std::integral_constant<int, 0>{});
        __builtin_amdgcn_s_waitcnt(0xc07f);
        ring_barrier();
        ring_barrier();   // j = 2, 3 written
        take_z(std::integral_constant<int, 5>{}, std::integral_constant<int, 1>{});
        store(nblk - 1);
    }
}
