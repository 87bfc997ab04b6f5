"""CPU oracle for integer Winograd F(4x4, 3x3) convolution with tap-wise
power-of-two quantization (arxiv 2209.12982).

This package is test infrastructure.  Only the test suite, the smoke check in
``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may import it; the
library in ``paper_2209_12982_amd`` never does, and the two share no code.

Everything here is plain, slow and exact: exact rationals or Python/NumPy
integers for the method, float64 only where the paper's float algorithm is the
subject (float Winograd vs direct convolution).

Modules
  f4        transform matrices of F(4x4,3x3) and F(2x2,3x3) (Sec. II)
  quant     round / clamp / power-of-two exponent rules (Sec. III, Eq. quant)
  direct    direct 3x3 convolution: float64, integer, and brute force
  tapwise   the tap-wise quantized integer Winograd F4 pipeline (Sec. III),
            its offline plan, input/output calibration, and analytic bounds
"""
