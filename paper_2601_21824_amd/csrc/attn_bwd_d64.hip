// attn_bwd_d64.hip -- the 128-row KV-tile main kernel (bwd_main.h) at head
// dim 64: the d = 64 calls with too few KV tiles for the 256-row kernel of
// attn_bwd64w.hip.  A translation unit of its own so that it is compiled with
// its MFMA results in VGPRs (S and dP reach the softmax without reads out of
// the AGPRs), which the d = 128 instantiation, with less room in its VGPRs,
// does not take.
#include "bwd_main.h"

namespace dash {

hipError_t launch_main64(const BwdArgs& a, int grid_main, hipStream_t stream) {
  return launch_main<64>(a, grid_main, stream);
}

int main64_occupancy() { return main_occupancy<64>(); }

}  // namespace dash
