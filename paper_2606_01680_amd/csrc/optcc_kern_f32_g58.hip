// F32 kernels of the OptCC executor for servers of 5-8 GPUs, 16-byte path
// (see optcc_launch.hpp); a file of its own so that it compiles in parallel.
#include "optcc_launch.hpp"

namespace optcc {

hipError_t launch_f32_g58(const kern::KArgs &a, bool two, hipStream_t st, int *occ) {
  return kern::launch_fixed_g<kern::F32, 5, 6, 7, 8>(a, two, st, occ);
}

}  // namespace optcc
