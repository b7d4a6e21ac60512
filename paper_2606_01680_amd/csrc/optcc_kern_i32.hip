// I32 kernels of the OptCC executor (see optcc_launch.hpp): one GPU per
// server; servers of 2-4 GPUs; element-aligned buffers and servers of more
// than 8 GPUs (general lane).  Servers of 5-8 GPUs: optcc_kern_i32_g58.hip.
#include "optcc_launch.hpp"

namespace optcc {

hipError_t launch_i32(const kern::KArgs &a, bool servers, bool vec16, bool two, hipStream_t st,
                     int *occ) {
  if (!servers) return kern::launch<kern::I32, false, 0>(a, vec16, two, st, occ);
  if (vec16 && a.g >= 2 && a.g <= 4) return kern::launch_fixed_g<kern::I32, 2, 3, 4>(a, two, st, occ);
  if (vec16 && a.g >= 5 && a.g <= 8) return launch_i32_g58(a, two, st, occ);
  return kern::launch<kern::I32, true, 0>(a, vec16, two, st, occ);
}

}  // namespace optcc
