"""MI355X-native AQLM inference path: dequantize, GEMV and small-batch GEMM
on additive-quantized weights, backed by hand-written HIP kernels for gfx950."""
