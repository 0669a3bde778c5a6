// launch_stubs.cpp -- stand-ins for the device-code entry points of the attention library
// (csrc/attn_kernels.hip, csrc/state_copy.hip) in the host-only sanitizer build of the C ABI.
// Kernel configuration reports failure, so device set-up never succeeds and no call proceeds to
// a launch; the launch functions are never reached and say so if they are.
#include <cstdio>
#include <cstdlib>

#include "attn_launch.h"

namespace tsattn {

hipError_t configure_kernels() { return hipErrorNotSupported; }

hipError_t scratch_address(void**) {
  std::fprintf(stderr, "scratch_address reached in the host-only build\n");
  std::abort();
}

hipError_t launch_dense(const DenseArgs&, hipStream_t) {
  std::fprintf(stderr, "launch_dense reached in the host-only build\n");
  std::abort();
}

hipError_t launch_packed(const PackedArgs&, hipStream_t) {
  std::fprintf(stderr, "launch_packed reached in the host-only build\n");
  std::abort();
}

hipError_t launch_state_copy(const void*, void*, const CopyList&, bool, bool, hipStream_t) {
  std::fprintf(stderr, "launch_state_copy reached in the host-only build\n");
  std::abort();
}

}  // namespace tsattn
