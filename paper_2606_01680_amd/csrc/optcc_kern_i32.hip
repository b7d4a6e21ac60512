// I32 kernels of the OptCC executor (see optcc_launch.hpp).
#include "optcc_launch.hpp"

namespace optcc {

hipError_t launch_i32(const kern::KArgs &a, bool servers, bool vec16, bool two, hipStream_t st) {
  return kern::launch_plan<kern::I32>(a, servers, vec16, two, st);
}

}  // namespace optcc
