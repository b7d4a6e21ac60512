// BF16 kernels of the OptCC executor (see optcc_launch.hpp).
#include "optcc_launch.hpp"

namespace optcc {

hipError_t launch_bf16(const kern::KArgs &a, bool servers, bool vec16, bool two, hipStream_t st) {
  return kern::launch_plan<kern::BF16>(a, servers, vec16, two, st);
}

}  // namespace optcc
