// FUSED variant of the online path: one launch per convolution.
#include "winof4_internal.h"

wino_status wino_f4_conv_fused(const wino_f4_plan_s* p, const int8_t* x, int8_t* y, int n, int h, int w,
                               wino_layout layout, hipStream_t stream) {
    (void)p; (void)x; (void)y; (void)n; (void)h; (void)w; (void)layout; (void)stream;
    return WINO_EUNSUPPORTED;
}
