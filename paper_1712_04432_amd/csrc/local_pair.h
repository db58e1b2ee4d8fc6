// The local backward pass's Delta_X and Delta_W products in one launch (csrc/skinny.hip).
#pragma once

#include "common.h"

namespace imbd {

// dx: the Delta_X partial (skinny-batch kernel, K whole, fp32 store with the optional
// ReLU mask); dw: the Delta_W partial (large-tile kernel, fp32 store of alpha * Delta_W,
// the bias partial in its first column tile). Returns IMBD_OK when both were launched as
// one grid, 1 when this route does not take them (the caller launches them one after the
// other), or an error code from the launch. dy_dw4: Delta_Y (dx.B and dw.B) has rows that are
// only 4-byte aligned (base and pitch; K of dx even): both kernels then load it in 4-byte
// pieces, which this route takes for up to 128 samples and 128-row Delta_W tiles.
int run_local_dx_dw_pair(const GemmProblem &dx, const GemmProblem &dw, void *ws, hipStream_t s, bool dy_dw4);

}  // namespace imbd
