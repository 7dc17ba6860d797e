"""CPU oracle for the SSDi8 INT8 SSD chunk scan — TEST INFRASTRUCTURE ONLY.

This package is the slow, plain, obviously-checkable definition that the HIP path is compared
against.  It is written from the paper ("SSDi8: Accurate and Efficient 8-bit Quantization for
State Space Duality") alone, in NumPy with fp64 for floating point and exact integer
arithmetic for the integer stages, and it shares no code with the HIP kernels or their
binding.  Only the test-suite, the package smoke check and the benchmark's CPU-baseline leg may
import it; the product path never does.

Modules
  exact      fp64 unquantized SSD: token recurrence, quadratic (attention) form and the chunked
             five-module form of Alg. 2 (Sec. 4.1).
  int8       the quantized SSDi8 path, stage by stage (Eq. 1, Sec. 4.2 with Eq. 7-9, Eq. 10).
  calibrate  static symmetric scale calibration and the single-layer mean correction
             (Sec. 5 setup, Eq. 10, Alg. 1 restricted to one layer).
  fp16       the unquantized FP16 SSD (Alg. 2 with fp16 operands, fp32 states), the reference
             of the on-box FP16 baseline the paper's speedups are measured against.

Parity status: every function is pinned by the CPU tests in tests/test_oracle_*.py (brute-force
equality of the three fp64 forms, exact special cases of the quantized path, integer closed
forms, stage error bounds).  The only unpinned quantity is the numerical value of the
floating-point output at the full workload sizes, for which the paper prints no values.
"""
