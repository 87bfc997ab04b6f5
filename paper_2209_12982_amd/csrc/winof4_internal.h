// Internal definitions shared by the host plan and the kernel launchers.
#pragma once
#include <stdint.h>
#include <vector>
#include <hip/hip_runtime.h>
#include "winof4.h"

namespace winof4 {

constexpr int kTaps = 36;
// Channel padding granule: one int8 MFMA k-step.
constexpr int kKStep = 64;
// Output-channel padding granule of the tap-GEMM workgroup.
constexpr int kCoutPad = 64;
// Tile padding granule of the tap-GEMM workgroup.
constexpr int kTilePad = 64;

inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

// Per-tap tables passed by value to the kernels.  They land in the kernarg
// segment; 32-bit entries keep every element 4-byte aligned, so the kernels
// read them with scalar loads into scalar registers (byte entries are read
// with vector loads and then occupy vector registers).
struct TapTables {
    int32_t eb[kTaps];   // input tap exponents e_B
    int32_t sh[kTaps];   // alignment shifts e_B + e_G - e_o
};

// Division by a fixed divisor 1 <= d < 2^26 of dividends n < 2^31 without a
// divide instruction (Granlund and Montgomery, "Division by Invariant
// Integers using Multiplication", 1994): with l = ceil(log2 d) and
// p = 31 + l, m = ceil(2^p / d) < 2^32 gives floor(n / d) =
// floor(n m / 2^p), because n m / 2^p - n / d < n / 2^p <= n / (2^31 d) < 1/d.
struct FastDiv {
    uint32_t mul;     // m (unused for d = 1)
    uint32_t shr;     // p - 32
    uint32_t d;
};
inline FastDiv make_fastdiv(uint32_t d) {
    FastDiv f = {0u, 0u, d};
    if (d <= 1) return f;
    int l = 0;
    while ((1ull << l) < d) ++l;
    const int p = 31 + l;
    f.mul = (uint32_t)(((1ull << p) + d - 1) / d);
    f.shr = (uint32_t)(p - 32);
    return f;
}

// One transform F(m x m, 3 x 3): n = m + 2 input rows, n^2 taps, Gint = d G
// with integer entries (Sec. II matrices: d = 24 for F4, 2 for F2),
// den2 = d^2, A^T (m x n).
struct Xform {
    int m, n, ntap, den2;
    int gint[6][3];
    int at[4][6];
};
inline constexpr Xform kF4 = {4, 6, 36, 576,
                              {{6, 0, 0}, {-4, -4, -4}, {-4, 4, -4}, {1, 2, 4}, {1, -2, 4}, {0, 0, 24}},
                              {{1, 1, 1, 1, 1, 0}, {0, 1, -1, 2, -2, 0}, {0, 1, 1, 4, 4, 0}, {0, 1, -1, 8, -8, 1}}};
inline constexpr Xform kF2 = {2, 4, 16, 4,
                              {{2, 0, 0}, {1, 1, 1}, {1, -1, 1}, {0, 0, 2}},
                              {{1, 1, 1, 0}, {0, 1, -1, -1}}};

}  // namespace winof4

struct wino_f4_plan_s;

namespace winof4 {
// Plan assembly shared by the host plan (plan.cpp) and the on-device weight
// transform (plan_device.hip).
wino_status plan_check_args(const Xform& X, int32_t cin, int32_t cout, const int8_t* in_exp,
                            const int8_t* w_exp, int32_t out_shift, int32_t relu);
// Bytes of one k-row of 64 channels in the GEMM operands: 64 int8 or 64 fp16.
inline int kbytes_per_channel(int bits) { return bits == 10 ? 2 : 1; }
void plan_set_shape(const Xform& X, wino_f4_plan_s* p, int32_t cin, int32_t cout, int32_t out_shift,
                    int32_t relu);
// Fills e_b, e_o, sh, bias_host and epi_bits from p->e_g and the column sums
// colsum[t * cout + co] = sum_ci |Uq[t][ci][co]|.
wino_status plan_finish(const Xform& X, wino_f4_plan_s* p, const int8_t* in_exp, const int32_t* bias,
                        const int32_t* colsum);
// Uploads the zero-padded bias; synchronizes `stream`.
wino_status plan_upload_bias(wino_f4_plan_s* p, hipStream_t stream);
// Device parts of the plan (plan_device.hip): fill p->e_g, write p->uq_dev
// (allocated here) and return the column sums.
wino_status device_weight_tables(const Xform& X, wino_f4_plan_s* p, const float* w_dev, const int8_t* w_exp,
                                 hipStream_t stream, std::vector<int32_t>& colsum);
wino_status device_weight_tables_int8(const Xform& X, wino_f4_plan_s* p, const int8_t* w_dev, int32_t w_scale_exp,
                                      const int8_t* w_exp, hipStream_t stream, std::vector<int32_t>& colsum);
}  // namespace winof4

struct wino_f4_plan_s {
    int32_t m = 4;                    // output tile: F(m x m, 3 x 3), m = 4 or 2
    int32_t ntap = 36;                // (m + 2)^2 taps
    int32_t bits = 8;                 // Winograd-domain integer width: 8, or 10 (int8/10)
    int32_t cin, cout, cin_pad, cout_pad;
    int8_t e_b[winof4::kTaps], e_g[winof4::kTaps], sh[winof4::kTaps];
    int32_t e_o;
    int32_t out_shift, relu;
    int32_t epi_bits;                 // 32 or 64
    int32_t tap_kernel = WINO_TAP_AUTO;
    int32_t device;
    int8_t* uq_dev;                   // bits 8: int8 [ntap][cin_pad/64][cout_pad][64];
                                      // bits 10: fp16 [ntap][cin_pad/32][cout_pad][32]; zero padded
    int32_t* bias_dev;                // [cout_pad], zero padded
    std::vector<int16_t> uq_host;     // [ntap][cin][cout]; empty for device-built plans
    std::vector<int32_t> bias_host;   // [cout]
};
