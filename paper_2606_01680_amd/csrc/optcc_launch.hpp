// Kernel launches of the OptCC executor: the kernel variants of one element
// type and the choice among them.  Each optcc_kern_*.hip instantiates one
// element type; optcc_exec.hip calls them through launch_f32/bf16/i32/f16.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>

#include "optcc_kernels.hpp"

namespace optcc {
namespace kern {

// Launch the kernel variant K, or, when occ is not NULL, only report how many
// of its workgroups one CU holds at this launch's dynamic LDS (no launch).
#define OPTCC_LAUNCH_OR_QUERY(K)                                                         \
  do {                                                                                  \
    if (occ)                                                                            \
      return hipOccupancyMaxActiveBlocksPerMultiprocessor(occ, K, kThreads,            \
                                                          (size_t)a.occ_lds);           \
    hipLaunchKernelGGL(K, grid, block, (unsigned)a.occ_lds, st, a);                     \
    return hipGetLastError();                                                           \
  } while (0)

// G = 0 covers element-aligned buffers (one element per access) too;
// G > 0 expects 16-byte-aligned buffers (vec16).
template <class D, bool S, int G>
hipError_t launch(const KArgs &a, bool vec16, bool two, hipStream_t st, int *occ) {
  constexpr int W16 = 16 / (int)sizeof(typename D::S);
  const int64_t grid64 = std::min<int64_t>(a.ntiles, a.grid > 0 ? (int64_t)a.grid : (int64_t)1 << 30);
  const dim3 grid((unsigned)std::max<int64_t>(grid64, 1)), block(kThreads);
  if constexpr (G == 0) {
    if (!vec16)  // element-aligned buffers: one element per access
      OPTCC_LAUNCH_OR_QUERY((optcc_exec_kernel<D, 1, 1, S, 0>));
  } else if (!vec16) {
    return hipErrorInvalidValue;
  }
  if constexpr (sizeof(typename D::S) == 4) {  // two vectors per lane: 32-bit types only
    if (two) OPTCC_LAUNCH_OR_QUERY((optcc_exec_kernel<D, W16, 2, S, G>));
    if constexpr (!S && G == 0) {  // long chains with large messages: the wider hop window
      if (a.wide_window) OPTCC_LAUNCH_OR_QUERY((optcc_exec_kernel<D, W16, 1, S, G, kHopWindowWide>));
    }
  }
  OPTCC_LAUNCH_OR_QUERY((optcc_exec_kernel<D, W16, 1, S, G>));
}

// Several GPUs per server, 16-byte path: the kernel with the local ring
// fixed at compile time when g is one of Gs (else hipErrorInvalidValue).
template <class D, int... Gs>
hipError_t launch_fixed_g(const KArgs &a, bool two, hipStream_t st, int *occ) {
  hipError_t err = hipErrorInvalidValue;
  (void)((a.g == Gs ? (err = launch<D, true, Gs>(a, true, two, st, occ), true) : false) || ...);
  return err;
}

}  // namespace kern

// One element type each (optcc_kern_<type>.hip: one GPU per server, and
// servers of 2-4 GPUs or any other size; optcc_kern_<type>_g58.hip: servers
// of 5-8 GPUs, split off so that the files compile in parallel): servers
// selects the several-GPUs-per-server lane, vec16 the 16-byte path, two the
// two-vectors-per-lane variant.  With occ not NULL nothing is launched: *occ
// receives the number of workgroups of the chosen variant one CU holds.
hipError_t launch_f32(const kern::KArgs &a, bool servers, bool vec16, bool two, hipStream_t st,
                      int *occ = nullptr);
hipError_t launch_bf16(const kern::KArgs &a, bool servers, bool vec16, bool two, hipStream_t st,
                       int *occ = nullptr);
hipError_t launch_i32(const kern::KArgs &a, bool servers, bool vec16, bool two, hipStream_t st,
                      int *occ = nullptr);
hipError_t launch_f16(const kern::KArgs &a, bool servers, bool vec16, bool two, hipStream_t st,
                      int *occ = nullptr);
hipError_t launch_f32_g58(const kern::KArgs &a, bool two, hipStream_t st, int *occ);
hipError_t launch_bf16_g58(const kern::KArgs &a, bool two, hipStream_t st, int *occ);
hipError_t launch_i32_g58(const kern::KArgs &a, bool two, hipStream_t st, int *occ);
hipError_t launch_f16_g58(const kern::KArgs &a, bool two, hipStream_t st, int *occ);

}  // namespace optcc
