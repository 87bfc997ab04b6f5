"""Integer Winograd F(4x4,3x3) convolution with tap-wise power-of-two
quantization on MI355X (gfx950): Python binding of libwinof4.

The compute path is the C-ABI library ``libwinof4.so`` built from ``csrc/``
(see ``include/winof4.h``); this package only marshals arguments.  PyTorch
provides device memory and streams.  Importing works without a GPU; calling
an entry point without the built library raises ``LibraryNotBuilt``.
"""
from .binding import (  # noqa: F401
    NCHW, NHWC, SPLIT, FUSED, TAPS, TAP_AUTO, TAP_RESIDENT, TAP_ROWS,
    TAP_RESIDENT_64X32, TAP_RESIDENT_32X32, TAP_RESIDENT_16X16, TAP_WAVES, TAP_ROWS_STREAMK, ALGO_DIRECT, ALGO_F2, ALGO_F4,
    LibraryNotBuilt, WinoError, WinoF4Plan,
    library_path, load_library, exported_symbols,
    wino_f4_plan, wino_f4_plan_tables, wino_f4_plan_info,
    wino_f2_plan, wino_f2_plan_tables, wino_f2_calibrate_input,
    wino_f4_plan_device, wino_f2_plan_device, wino_f4_plan_int8, wino_f2_plan_int8,
    wino_f4_plan_i10, wino_f2_plan_i10, wino_f4_plan_tables_i10, wino_f2_plan_tables_i10,
    wino_f4_calibrate_input_i10, wino_f2_calibrate_input_i10,
    wino_f4_plan_set_tap_kernel, wino_f4_tap_kernel_choice, wino_select_algorithm,
    wino_f4_workspace_bytes, wino_f4_conv_int8, wino_f4_conv_int8_noalloc, NOALLOC_SCRATCH_BYTES,
    wino_f4_input_transform, wino_f4_tap_gemm,
    wino_f4_calibrate_input, wino_f4_calibrate_output,
    wino_f4_debug_input_transform, wino_f4_debug_tap_gemm,
    direct_conv_quantize_weights, direct_conv_int8, wino_f4_conv_float, wino_probe_mfma_int8, wino_strerror,
)
