// optcc_narrow_f32: the executor's per-step rounding rule applied to a plain
// array, so that it can be compared with an independent implementation over
// every fp32 bit pattern.  The element types (and with them the rounding
// code) are the ones the fused kernel instantiates.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <string>

#include "optcc_internal.hpp"
#include "optcc_kernels.hpp"

namespace optcc {
namespace {

// Types that narrow vectors two values at a time (D::kPairs) take pairs
// through the same instruction as the executor, and an odd last element
// through the single-value form.
template <class D>
__global__ __launch_bounds__(256) void narrow_kernel(const float *__restrict__ src,
                                                     typename D::S *__restrict__ dst, int64_t n) {
  using S = typename D::S;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t first = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if constexpr (D::kPairs) {
    for (int64_t i = first; i < n / 2; i += stride) {
      const uint32_t h = D::narrow_pair(src[2 * i], src[2 * i + 1]);
      dst[2 * i] = (S)h;
      dst[2 * i + 1] = (S)(h >> 16);
    }
    if ((n & 1) && first == 0) dst[n - 1] = D::narrow(src[n - 1]);
  } else {
    for (int64_t i = first; i < n; i += stride) dst[i] = D::narrow(src[i]);
  }
}

template <class D>
hipError_t launch_narrow(const float *src, void *dst, int64_t n, hipStream_t st) {
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 8192);
  hipLaunchKernelGGL((narrow_kernel<D>), dim3((unsigned)blocks), dim3(256), 0, st, src,
                     static_cast<typename D::S *>(dst), n);
  return hipGetLastError();
}

}  // namespace
}  // namespace optcc

extern "C" int optcc_narrow_f32(const float *src, void *dst, int64_t n, optcc_dtype_t dtype,
                                void *stream) {
  using namespace optcc;
  set_error("");
  if (n < 0) return fail(OPTCC_EINVAL, "n must be >= 0");
  if (dtype != OPTCC_BF16 && dtype != OPTCC_F16)
    return fail(OPTCC_EINVAL, "dtype must be OPTCC_BF16 or OPTCC_F16");
  if (n == 0) return OPTCC_OK;
  if (!src || !dst) return fail(OPTCC_EINVAL, "src and dst must be non-NULL");
  const uintptr_t s = reinterpret_cast<uintptr_t>(src), d = reinterpret_cast<uintptr_t>(dst);
  if (s % 4 || d % 2) return fail(OPTCC_EINVAL, "src and dst must be aligned to their element sizes");
  if ((uint64_t)n > (UINTPTR_MAX - s) / 4 || (uint64_t)n > (UINTPTR_MAX - d) / 2)
    return fail(OPTCC_EINVAL, "n elements would run past the end of the address space");
  if (s < d + (uintptr_t)n * 2 && d < s + (uintptr_t)n * 4)
    return fail(OPTCC_EINVAL, "src and dst overlap");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const hipError_t err = dtype == OPTCC_BF16 ? launch_narrow<kern::BF16>(src, dst, n, st)
                                             : launch_narrow<kern::F16>(src, dst, n, st);
  if (err != hipSuccess) return fail(OPTCC_EDEVICE, std::string("kernel launch: ") + hipGetErrorString(err));
  return OPTCC_OK;
}
