// Kernel launches of the OptCC executor: the kernel variants of one element
// type and the choice among them.  Each optcc_kern_*.hip instantiates one
// element type; optcc_exec.hip calls them through launch_f32/bf16/i32.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>

#include "optcc_kernels.hpp"

namespace optcc {
namespace kern {

template <class D, bool S, int G>
hipError_t launch(const KArgs &a, bool vec16, bool two, hipStream_t st) {
  constexpr int W16 = 16 / (int)sizeof(typename D::S);
  const int64_t grid64 = std::min<int64_t>(a.ntiles, (int64_t)1 << 30);
  const dim3 grid((unsigned)std::max<int64_t>(grid64, 1)), block(kThreads);
  if (!vec16) {  // element-aligned buffers: the general lane, one element per access
    hipLaunchKernelGGL((optcc_exec_kernel<D, 1, 1, S, 0>), grid, block, 0, st, a);
    return hipGetLastError();
  }
  if constexpr (sizeof(typename D::S) == 4) {  // two vectors per lane: 32-bit types only
    if (two) {
      hipLaunchKernelGGL((optcc_exec_kernel<D, W16, 2, S, G>), grid, block, 0, st, a);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((optcc_exec_kernel<D, W16, 1, S, G>), grid, block, 0, st, a);
  return hipGetLastError();
}

// Several GPUs per server: the usual server sizes g = 2, 4, 8 get a kernel
// with the local ring fixed at compile time.
template <class D>
hipError_t launch_plan(const KArgs &a, bool servers, bool vec16, bool two, hipStream_t st) {
  if (!servers) return launch<D, false, 0>(a, vec16, two, st);
  switch (a.g) {
    case 2: return launch<D, true, 2>(a, vec16, two, st);
    case 4: return launch<D, true, 4>(a, vec16, two, st);
    case 8: return launch<D, true, 8>(a, vec16, two, st);
    default: return launch<D, true, 0>(a, vec16, two, st);
  }
}

}  // namespace kern

// One element type each (optcc_kern_f32.hip, optcc_kern_bf16.hip,
// optcc_kern_i32.hip): servers selects the several-GPUs-per-server lane,
// vec16 the 16-byte path, two the two-vectors-per-lane variant.
hipError_t launch_f32(const kern::KArgs &a, bool servers, bool vec16, bool two, hipStream_t st);
hipError_t launch_bf16(const kern::KArgs &a, bool servers, bool vec16, bool two, hipStream_t st);
hipError_t launch_i32(const kern::KArgs &a, bool servers, bool vec16, bool two, hipStream_t st);

}  // namespace optcc
