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

}  // namespace winof4

struct wino_f4_plan_s {
    int32_t m = 4;                    // output tile: F(m x m, 3 x 3), m = 4 or 2
    int32_t ntap = 36;                // (m + 2)^2 taps
    int32_t cin, cout, cin_pad, cout_pad;
    int8_t e_b[winof4::kTaps], e_g[winof4::kTaps], sh[winof4::kTaps];
    int32_t e_o;
    int32_t out_shift, relu;
    int32_t epi_bits;                 // 32 or 64
    int32_t tap_kernel = WINO_TAP_AUTO;
    int32_t device;
    int8_t* uq_dev;                   // [ntap][cin_pad/64][cout_pad][64], zero padded
    int32_t* bias_dev;                // [cout_pad], zero padded
    std::vector<int8_t> uq_host;      // [ntap][cin][cout]
    std::vector<int32_t> bias_host;   // [cout]
};
