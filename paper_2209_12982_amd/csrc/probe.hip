// Matrix-core rate probe: independent int8 MFMAs, nothing else, so a bench
// can state the int8 peak it measures at the run's clock next to the
// datasheet figure.  Not part of the convolution.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "winof4_probe.h"

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

// Every wave keeps eight (16x16) or four (32x32) accumulator chains in
// flight, enough to issue back to back.  The sink is written only if the
// results hit a value they cannot take, which keeps the work from being
// optimized away.
template <int SHAPE>
__global__ __launch_bounds__(256) void mfma_probe(int iters, int* __restrict__ sink) {
    const v4i a = {(int)threadIdx.x, 0x01020304, 0x05060708, 0x7f7f7f7f};
    const v4i b = {0x01010101, (int)blockIdx.x, 0x02020202, 0x03030303};
    int res = 0;
    if constexpr (SHAPE == 16) {
        v4i c[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) c[i] = (v4i){i, 0, 0, 0};
        for (int it = 0; it < iters; ++it) {
#pragma unroll
            for (int i = 0; i < 8; ++i) c[i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c[i], 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) res ^= c[i][0] ^ c[i][3];
    } else {
        v16i c[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            c[i] = (v16i){};
            c[i][0] = i;
        }
        for (int it = 0; it < iters; ++it) {
#pragma unroll
            for (int i = 0; i < 4; ++i) c[i] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c[i], 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) res ^= c[i][0] ^ c[i][15];
    }
    if (res == 0x7ee1babe) sink[0] = res;
}

}  // namespace

extern "C" wino_status wino_probe_mfma_int8(int32_t shape, int32_t iters, int32_t blocks, int32_t* sink,
                                            int64_t* ops, hipStream_t stream) {
    if ((shape != 16 && shape != 32) || iters < 1 || blocks < 1 || !sink || !ops) return WINO_EINVAL;
    // 4 waves per block; per wave and iteration 8 x 16x16x64 or 4 x 32x32x32
    // MACs, 2 operations each
    const long long per_iter = shape == 16 ? 8ll * 16 * 16 * 64 : 4ll * 32 * 32 * 32;
    *ops = 2ll * per_iter * 4 * blocks * iters;
    if (shape == 16)
        hipLaunchKernelGGL(mfma_probe<16>, dim3((unsigned)blocks), dim3(256), 0, stream, iters, sink);
    else
        hipLaunchKernelGGL(mfma_probe<32>, dim3((unsigned)blocks), dim3(256), 0, stream, iters, sink);
    return hipGetLastError() == hipSuccess ? WINO_OK : WINO_EHIP;
}
