// Device code of the OptCC executor: element types, per-lane step
// sequences and the kernel.  Included by optcc_exec.hip only.
//
// The p logical ranks are p buffers in HBM.  One workgroup takes one tile of
// 2048 consecutive elements of one segment's ring sections (or of its
// point-to-point chunk) and runs, lane by lane, every step of the schedule
// that touches those elements, in the section's own stage order: the
// partial sum a hop forwards stays in registers, and every step still writes
// its destination rank's buffer.  All arithmetic is elementwise, so the work
// is a streaming reduction bound by HBM bandwidth; no matrix cores are used.
//
// Stage slots per section (paper: "Don't Let a Few Network Failures Slow the
// Entire AllReduce", Sec. 4.1 Stages 1-4 and the two stage orderings,
// Sec. 4.2 patterns and bubble filling, App. C, App. D):
//   0 straggler raw values folded into the chain start R[j]
//   1 Stage 1 reduce-scatter chain R[j] -> R[j+1] -> ... -> R[j-1] (holder)
//   2 Stage 2: the finalising straggler adds the holder's partial;
//     P2P up: the straggler sums its own chunk and every healthy rank's
//   3 Stage 3: the global sum returns to the holder; P2P down
//   4 Stage 4 allgather holder -> R[j] -> ... -> R[j+P'-2]
//   5 the global sum reaches the stragglers that did not finalise
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "optcc_internal.hpp"

namespace optcc {
namespace kern {

#ifndef OPTCC_NT_LOADS
#define OPTCC_NT_LOADS 1
#endif
#ifndef OPTCC_NT_FINAL
#define OPTCC_NT_FINAL 1
#endif
#ifndef OPTCC_NT_MID
#define OPTCC_NT_MID 0
#endif

constexpr int kThreads = 256;
constexpr int kMaxRanks = OPTCC_MAX_EMULATE_RANKS;
constexpr int kHopWindow = 16;  // hop loads in flight per vector along a chain
// Input values are read once: streaming (nontemporal) loads keep them from
// displacing lines in L2.  Stores of values that no later step overwrites
// are streamed too; Stage-1 partials that Stage 4 overwrites are ordinary
// stores, so that L2 can absorb the first write.
constexpr bool kNtLoads = OPTCC_NT_LOADS;
constexpr bool kNtFinal = OPTCC_NT_FINAL;
constexpr bool kNtMid = OPTCC_NT_MID;
// fp32/int32 plans with at most this many healthy ranks run two 16-byte
// vectors per lane in lockstep (measured faster for short chains)
constexpr int kTwoVectorMaxHealthy = 32;

struct KArgs {
  const TileDesc *tiles;
  const SegDesc *segs;
  int64_t ntiles;
  int64_t n;
  int32_t pp, m;
  int32_t sb, se;  // slot range [sb, se)
  int32_t xcd_runs;  // 1: each XCD takes a contiguous run of tiles
  // rank pointers: [0, pp) healthy ranks in ring order, [pp, pp+m) stragglers
  // sorted by slowdown (worst first)
  void *ptr[kMaxRanks];
};

// ----------------------------------------------------------- element types
// widen / narrow / add of one element; a step is narrow(widen(a) + widen(b)).
struct F32 {
  using S = float;
  using A = float;
  __device__ static A widen(S x) { return x; }
  __device__ static S narrow(A x) { return x; }
};
struct I32 {
  using S = uint32_t;  // two's complement adds wrap modulo 2^32
  using A = uint32_t;
  __device__ static A widen(S x) { return x; }
  __device__ static S narrow(A x) { return x; }
};
struct BF16 {
  using S = uint16_t;
  using A = float;
  __device__ static A widen(S x) { return __uint_as_float((uint32_t)x << 16); }
  // round to nearest, ties to even; NaN stays NaN
  __device__ static S narrow(A f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (S)((u >> 16) | 0x0040u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (S)(u >> 16);
  }
};

template <class D, int W>
struct alignas(sizeof(typename D::S) * W) Vec {
  typename D::S v[W];
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Loads and stores of W elements; NT selects the streaming hint.
template <class D, int W, bool NT = false>
__device__ __forceinline__ Vec<D, W> vload(const void *base, int64_t e) {
  const typename D::S *p = static_cast<const typename D::S *>(base) + e;
  if constexpr (sizeof(Vec<D, W>) == 16) {
    const u32x4 *q = reinterpret_cast<const u32x4 *>(p);
    const u32x4 r = NT ? __builtin_nontemporal_load(q) : *q;
    return __builtin_bit_cast(Vec<D, W>, r);
  } else {
    static_assert(W == 1, "vectors are 16 bytes or one element");
    Vec<D, W> r;
    r.v[0] = NT ? __builtin_nontemporal_load(p) : *p;
    return r;
  }
}
template <class D, int W, bool NT = false>
__device__ __forceinline__ void vstore(void *base, int64_t e, const Vec<D, W> &x) {
  typename D::S *p = static_cast<typename D::S *>(base) + e;
  if constexpr (sizeof(Vec<D, W>) == 16) {
    u32x4 *q = reinterpret_cast<u32x4 *>(p);
    const u32x4 v = __builtin_bit_cast(u32x4, x);
    if (NT) __builtin_nontemporal_store(v, q);
    else *q = v;
  } else {
    static_assert(W == 1, "vectors are 16 bytes or one element");
    if (NT) __builtin_nontemporal_store(x.v[0], p);
    else *p = x.v[0];
  }
}
// input loads and final stores with the configured hints
template <class D, int W>
__device__ __forceinline__ Vec<D, W> ld_in(const void *base, int64_t e) {
  return vload<D, W, kNtLoads>(base, e);
}
template <class D, int W>
__device__ __forceinline__ void st_fin(void *base, int64_t e, const Vec<D, W> &x) {
  vstore<D, W, kNtFinal>(base, e, x);
}
// stores of values a later step of the same section overwrites
template <class D, int W>
__device__ __forceinline__ void st_mid(void *base, int64_t e, const Vec<D, W> &x) {
  vstore<D, W, kNtMid>(base, e, x);
}
// One reduce step with a single source: narrow(widen(a) + widen(b)).
template <class D, int W>
__device__ __forceinline__ Vec<D, W> add2(const Vec<D, W> &a, const Vec<D, W> &b) {
  Vec<D, W> r;
#pragma unroll
  for (int i = 0; i < W; ++i) r.v[i] = D::narrow(D::widen(a.v[i]) + D::widen(b.v[i]));
  return r;
}
template <class D, int W>
struct AccV {
  typename D::A v[W];
};
template <class D, int W>
__device__ __forceinline__ AccV<D, W> widen(const Vec<D, W> &a) {
  AccV<D, W> r;
#pragma unroll
  for (int i = 0; i < W; ++i) r.v[i] = D::widen(a.v[i]);
  return r;
}
template <class D, int W>
__device__ __forceinline__ void accum(AccV<D, W> &acc, const Vec<D, W> &b) {
#pragma unroll
  for (int i = 0; i < W; ++i) acc.v[i] = acc.v[i] + D::widen(b.v[i]);
}
template <class D, int W>
__device__ __forceinline__ Vec<D, W> narrow(const AccV<D, W> &a) {
  Vec<D, W> r;
#pragma unroll
  for (int i = 0; i < W; ++i) r.v[i] = D::narrow(a.v[i]);
  return r;
}

__device__ __forceinline__ bool in_range(const KArgs &a, int q) { return a.sb <= q && q < a.se; }

// ------------------------------------------------------- one ring section
// Every step of the ring sections for L vectors of W elements per lane, in
// lockstep: vector l starts at element e[l] and lies in section j[l].
// rp[i] is the i-th healthy rank's buffer in ring order (LDS copy).
template <class D, int W, int L, int B>
__device__ void ring_lane(const KArgs &a, void *const *rp, const SegDesc &sd, const int (&j)[L],
                          const int64_t (&e)[L]) {
  using V = Vec<D, W>;
  const int pp = a.pp, m = a.m;
  const int ord = sd.ordering;
  const int nside = m == 0 ? 0 : (ord == 2 ? m : m - 1);
  const int sfirst = ord == 2 ? 0 : 1;
  const bool fin = m >= 1 && ord == 1;  // a straggler finalises in Stages 2/3
  auto rank = [&](int l, int t) {       // buffer of R[j[l] + t], 0 <= t < 2 pp
    int i = j[l] + t;
    return rp[i >= pp ? i - pp : i];
  };
  void *holder[L];
#pragma unroll
  for (int l = 0; l < L; ++l) holder[l] = rank(l, pp - 1);
  V v[L];
  bool have = false;

  // Stage 2's straggler operand does not depend on the chain: load it early.
  V xs[L];
  const bool do2 = fin && in_range(a, 2);
  if (do2) {
#pragma unroll
    for (int l = 0; l < L; ++l) xs[l] = ld_in<D, W>(a.ptr[pp], e[l]);
  }

  if (in_range(a, 0) && nside > 0) {  // slot 0
#pragma unroll
    for (int l = 0; l < L; ++l) {
      AccV<D, W> acc = widen(ld_in<D, W>(rp[j[l]], e[l]));
      for (int i = 0; i < nside; ++i) accum(acc, ld_in<D, W>(a.ptr[pp + sfirst + i], e[l]));
      v[l] = narrow(acc);
      st_mid<D, W>(rp[j[l]], e[l], v[l]);
    }
    have = true;
  }
  if (in_range(a, 1)) {  // slot 1: Stage 1 chain
    if (!have) {
#pragma unroll
      for (int l = 0; l < L; ++l) v[l] = ld_in<D, W>(rp[j[l]], e[l]);
    }
    // The hop loads are independent of the partial: keep B of them
    // in flight in a rolling window, refilling a slot as soon as it is used.
    const int nh = pp - 1;
    V buf[B][L];
#pragma unroll
    for (int u = 0; u < B; ++u)
      if (u < nh) {
#pragma unroll
        for (int l = 0; l < L; ++l) buf[u][l] = ld_in<D, W>(rank(l, 1 + u), e[l]);
      }
    for (int t = 0; t < nh; t += B) {
#pragma unroll
      for (int u = 0; u < B; ++u)
        if (t + u < nh) {
#pragma unroll
          for (int l = 0; l < L; ++l) {
            v[l] = add2<D, W>(buf[u][l], v[l]);
            st_mid<D, W>(rank(l, 1 + t + u), e[l], v[l]);
          }
          if (t + u + B < nh) {
#pragma unroll
            for (int l = 0; l < L; ++l)
              buf[u][l] = ld_in<D, W>(rank(l, 1 + t + u + B), e[l]);
          }
        }
    }
    have = true;
  }
  if (fin) {
    if (do2) {  // slot 2: straggler <- straggler + holder's partial
#pragma unroll
      for (int l = 0; l < L; ++l) {
        if (!have) v[l] = ld_in<D, W>(holder[l], e[l]);
        v[l] = add2<D, W>(xs[l], v[l]);
        st_fin<D, W>(a.ptr[pp], e[l], v[l]);
      }
      have = true;
    }
    if (in_range(a, 3)) {  // slot 3: holder <- global sum
#pragma unroll
      for (int l = 0; l < L; ++l) {
        if (!have) v[l] = ld_in<D, W>(a.ptr[pp], e[l]);
        st_fin<D, W>(holder[l], e[l], v[l]);
      }
      have = true;
    }
  }
  if (in_range(a, 4)) {  // slot 4: allgather
    if (!have) {
#pragma unroll
      for (int l = 0; l < L; ++l) v[l] = ld_in<D, W>(holder[l], e[l]);
    }
    for (int t = 0; t + 1 < pp; ++t) {
#pragma unroll
      for (int l = 0; l < L; ++l) st_fin<D, W>(rank(l, t), e[l], v[l]);
    }
    have = true;
  }
  if (in_range(a, 5) && nside > 0) {  // slot 5
    if (!have) {
#pragma unroll
      for (int l = 0; l < L; ++l) v[l] = ld_in<D, W>(holder[l], e[l]);
    }
    for (int i = 0; i < nside; ++i) {
#pragma unroll
      for (int l = 0; l < L; ++l) st_fin<D, W>(a.ptr[pp + sfirst + i], e[l], v[l]);
    }
  }
}

// ------------------------------------------------- one point-to-point chunk
// Bubble filling (Sec. 4.2, App. C): the straggler sums its own value and
// R[0..P'-1] in that order, rounding once, and broadcasts the result.
template <class D, int W, int L, int B>
__device__ void p2p_lane(const KArgs &a, void *const *rp, const int64_t (&e)[L]) {
  using V = Vec<D, W>;
  const int pp = a.pp;
  V g[L];
  bool have = false;
  if (in_range(a, 2)) {
    AccV<D, W> acc[L];
#pragma unroll
    for (int l = 0; l < L; ++l) acc[l] = widen(ld_in<D, W>(a.ptr[pp], e[l]));
    for (int t = 0; t < pp; t += B) {
      V x[B][L];
#pragma unroll
      for (int u = 0; u < B; ++u)
        if (t + u < pp) {
#pragma unroll
          for (int l = 0; l < L; ++l) x[u][l] = ld_in<D, W>(rp[t + u], e[l]);
        }
#pragma unroll
      for (int u = 0; u < B; ++u)
        if (t + u < pp) {
#pragma unroll
          for (int l = 0; l < L; ++l) accum(acc[l], x[u][l]);
        }
    }
#pragma unroll
    for (int l = 0; l < L; ++l) {
      g[l] = narrow(acc[l]);
      st_fin<D, W>(a.ptr[pp], e[l], g[l]);
    }
    have = true;
  }
  if (in_range(a, 3)) {
    if (!have) {
#pragma unroll
      for (int l = 0; l < L; ++l) g[l] = ld_in<D, W>(a.ptr[pp], e[l]);
    }
    for (int i = 0; i < pp; ++i) {
#pragma unroll
      for (int l = 0; l < L; ++l) st_fin<D, W>(rp[i], e[l], g[l]);
    }
  }
}

// Section index of the quantum u of a segment's ring part.
__device__ __forceinline__ int section_of(const SegDesc &sd, int64_t u64) {
  const uint32_t u = (uint32_t)u64;  // quanta within one segment fit in 32 bits
  const uint32_t big = (uint32_t)sd.nbig * (uint32_t)(sd.qbase + 1);
  if (u < big) return (int)(u / (uint32_t)(sd.qbase + 1));
  return sd.nbig + (int)((u - big) / (uint32_t)sd.qbase);
}

template <class D, int W, int L, int B>
__device__ __forceinline__ void run_elems(const KArgs &a, void *const *rp, const SegDesc &sd,
                                          bool p2p, const int64_t (&e)[L]) {
  if (p2p) {
    p2p_lane<D, W, L, B>(a, rp, e);
  } else {
    int j[L];
#pragma unroll
    for (int l = 0; l < L; ++l) j[l] = section_of(sd, (e[l] - sd.ring_begin) / kQuantum);
    ring_lane<D, W, L, B>(a, rp, sd, j, e);
  }
}

// W elements per lane access: 16 bytes when every rank buffer is 16-byte
// aligned, else 1 element.  A lane takes L such vectors of a tile
// at a stride of one workgroup-width, in lockstep; vectors past the tile's
// last whole group go one at a time, and elements past the last whole vector
// (only at the end of the rank vectors) one by one.
template <class D, int W, int L>
__global__ __launch_bounds__(kThreads) void optcc_exec_kernel(KArgs a) {
  constexpr int B = kHopWindow;
  constexpr int64_t kStride = (int64_t)kThreads * W;
  __shared__ void *rp[kMaxRanks];
  for (int i = threadIdx.x; i < a.pp; i += kThreads) rp[i] = a.ptr[i];
  __syncthreads();
  // Workgroups are dealt to the XCDs round robin by workgroup index.  With
  // xcd_runs, workgroup t0 takes tile (t0 mod X) * per + t0 / X, so each XCD
  // sweeps its own contiguous run of tiles.  Any XCD count keeps every tile
  // covered exactly once; X = 8 matches MI355X.
  constexpr int64_t kXcds = 8;
  const int64_t per = (a.ntiles + kXcds - 1) / kXcds;
  const int64_t cover = a.xcd_runs ? per * kXcds : a.ntiles;
  for (int64_t t0 = blockIdx.x; t0 < cover; t0 += gridDim.x) {
    const int64_t t = a.xcd_runs ? (t0 % kXcds) * per + t0 / kXcds : t0;
    if (t >= a.ntiles) continue;
    const TileDesc td = a.tiles[t];
    const bool p2p = td.meta & 1;
    const SegDesc sd = a.segs[td.meta >> 1];
    const int64_t end = td.begin + td.len;
    int64_t e0 = td.begin + (int64_t)threadIdx.x * W;
    for (; e0 + (L - 1) * kStride + W <= end; e0 += L * kStride) {
      int64_t e[L];
#pragma unroll
      for (int l = 0; l < L; ++l) e[l] = e0 + l * kStride;
      run_elems<D, W, L, B>(a, rp, sd, p2p, e);
    }
    for (; e0 < end; e0 += kStride) {
      if (e0 + W <= end) {
        const int64_t e[1] = {e0};
        run_elems<D, W, 1, B>(a, rp, sd, p2p, e);
      } else {
        for (int64_t x = e0; x < end; ++x) {
          const int64_t e[1] = {x};
          run_elems<D, 1, 1, B>(a, rp, sd, p2p, e);
        }
      }
    }
  }
}

}  // namespace kern
}  // namespace optcc
