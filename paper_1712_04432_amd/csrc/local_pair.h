// The local backward pass's Delta_X and Delta_W products in one launch (csrc/skinny.hip).
#pragma once

#include "common.h"

namespace imbd {

// dx: the Delta_X partial (skinny-batch kernel, K whole, fp32 store with the optional
// ReLU mask); dw: the Delta_W partial (large-tile kernel, fp32 store of alpha * Delta_W,
// the bias partial in its first column tile). Returns IMBD_OK when both were launched as
// one grid, 1 when this route does not take them (the caller launches them one after the
// other), or an error code from the launch. With b_dw4 set on both (Delta_Y rows only 4-byte
// aligned) the two bodies read Delta_Y in 4-byte pieces.
int run_local_dx_dw_pair(const GemmProblem &dx, const GemmProblem &dw, void *ws, hipStream_t s);

}  // namespace imbd
