// The 3x3 convolution tile's kernels are instantiations of the GEMM template in gemm.hip
// (implicit GEMM over the padded grid); see run_conv_* there. This file is kept for the
// conv-specific host declarations only.
#include "common.h"
