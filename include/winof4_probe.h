/*
 * libwinof4 measurement probe -- not part of the convolution and not part of
 * the method's interface.  It is exported by the same library so that a
 * benchmark can state the int8 matrix-core rate it measures at the run's
 * clock next to the datasheet figure, the denominator a tap-GEMM utilisation
 * is read against.
 */
#ifndef WINOF4_PROBE_H
#define WINOF4_PROBE_H

#include "winof4.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * wino_probe_mfma_int8 -- measurement probe, not part of the convolution:
 * `blocks` workgroups of four waves issue independent int8 MFMAs only
 * (shape 16: v_mfma_i32_16x16x64_i8, eight chains per wave; shape 32:
 * v_mfma_i32_32x32x32_i8, four chains), `iters` rounds each, so that a
 * caller timing the launch measures the int8 matrix-core rate at the run's
 * clock.  *ops (host) receives the launch's operation count (2 per
 * multiply-add).  sink: device int32, never written in practice (it keeps
 * the results live).  Asynchronous on `stream`; WINO_EINVAL for a bad shape
 * or count or a NULL pointer.
 */
wino_status wino_probe_mfma_int8(int32_t shape, int32_t iters, int32_t blocks, int32_t* sink,
                                 int64_t* ops, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* WINOF4_PROBE_H */
