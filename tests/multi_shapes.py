"""Launch shapes of the several-vector, fused and quantised kernels
(include/tvl.h, tvl_tuning), shared by the GPU parity tests and the CPU check
that the header, the library and the tests list the same shapes.

VALU form: (R, waves per block, U, B) with B x vectors per launch; matrix-core
forms: (rows per wavefront, waves per block, U), any nrhs <= 16.
"""

MULTI = [(2, 4, 2, 2), (2, 4, 4, 2), (4, 4, 2, 2), (2, 4, 1, 4), (2, 4, 2, 4), (4, 4, 1, 4),
         (4, 4, 2, 4), (2, 4, 1, 8), (2, 4, 2, 8), (4, 4, 1, 8), (8, 4, 1, 4), (8, 2, 1, 4),
         (8, 2, 1, 2)]
# matrix-core forms, any nrhs <= 16: 4x4x1 (rows per wavefront 8 or 16, waves
# per block, unroll 1) and 16x16x4 (16 x row groups, waves per block, loads
# per row group in flight >= 4)
MFMA = [(8, 4, 1), (16, 1, 1), (16, 2, 1)]
MFMA16 = [(16, 4, 8), (32, 1, 4), (32, 2, 4), (64, 1, 4)]
# 16x16x4 with LDS-staged rows (U = 2)
MFMA_LDS = [(16, 1, 2), (16, 4, 2), (32, 1, 2), (32, 2, 2), (32, 4, 2), (64, 1, 2)]
# 16x16x4 with weights streamed into LDS (U = 10 stages + log2(columns per
# chunk / 16); fp32 and fp16 weights)
MFMA_DMA = [(16, 1, 33), (16, 2, 33), (32, 1, 33), (16, 1, 32), (16, 4, 32), (32, 1, 32),
            (32, 2, 32), (16, 4, 42), (32, 1, 42), (32, 1, 52)]
# the same with fp16 weights on the fp16 matrix cores, x split in two fp16
# parts (U + 100; launches holding fp32 weights take the LDS-staged form)
MFMA_HX = [(16, 1, 133), (16, 2, 133), (32, 1, 133), (32, 2, 133), (64, 1, 133), (32, 1, 132),
           (64, 1, 132)]
# streamed, x shared by the block's wavefronts through LDS (U = 200 +
# log2(columns per chunk / 16), + 100 for fp16 weights with split x; mixed
# launches, and fp32 ones for the split-x shapes, take the LDS-staged form)
MFMA_XS = [(16, 4, 202), (32, 2, 202), (32, 4, 202), (16, 2, 203), (16, 4, 203), (16, 8, 202),
           (16, 4, 303), (32, 2, 303), (32, 4, 303), (16, 8, 303), (16, 4, 302), (32, 4, 302)]
# launches holding RMSNorm or SwiGLU items: (R, waves per block, U), even R
FUSED_SHAPES = [(2, 4, 2), (2, 4, 3), (2, 4, 4), (2, 1, 4), (4, 1, 2), (4, 1, 4), (4, 4, 2),
                (2, 1, 8), (8, 4, 1), (8, 2, 1), (4, 4, 3)]
# launches holding block-quantised items: (R, waves per block, U), direct x
# and x staged in LDS (TVL_FLAG_X_LDS)
QUANT_SHAPES = [(2, 4, 2), (4, 4, 1), (4, 4, 2), (4, 1, 2), (8, 4, 1), (8, 2, 1)]
QUANT_LDS_SHAPES = [(4, 4, 1), (8, 4, 1), (8, 2, 1), (4, 4, 2)]
