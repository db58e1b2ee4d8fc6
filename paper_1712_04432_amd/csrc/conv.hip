// 3x3 convolution tile of a domain-parallel layer (Sec. 2.2). Not built yet: every entry
// reports IMBD_EUNSUPPORTED so callers fail loudly instead of receiving garbage.
#include "common.h"

namespace imbd {

int run_conv_fwd(int, int, int, int, int, const void *, const void *, void *, int, hipStream_t) {
  set_error("conv3x3 tile forward is not implemented yet");
  return IMBD_EUNSUPPORTED;
}
int run_conv_dgrad(int, int, int, int, int, const void *, const void *, void *, int, hipStream_t) {
  set_error("conv3x3 tile dgrad is not implemented yet");
  return IMBD_EUNSUPPORTED;
}
int run_conv_wgrad(int, int, int, int, int, const void *, const void *, float *, void *, size_t, hipStream_t) {
  set_error("conv3x3 tile wgrad is not implemented yet");
  return IMBD_EUNSUPPORTED;
}
size_t conv_wgrad_ws_bytes(int, int, int, int, int) { return 0; }

}  // namespace imbd
