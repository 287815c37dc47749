// projection GEMM kernels
