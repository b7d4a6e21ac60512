// Device code of the OptCC executor: element types, per-lane step
// sequences and the kernel.  Included through optcc_launch.hpp.
//
// The p logical ranks are p buffers in HBM.  One workgroup takes one tile of
// consecutive elements (1024 to 8192, 2048 for most plans; the launch picks
// the length) of one segment's ring sections (or of its point-to-point
// chunk) and runs, lane by lane, every step of the schedule
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
// Plans with several GPUs per server (App. E) run twelve slots, the NVLink
// phases N1-N4 around the four NIC stages; see server_lane below.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

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
// the same for long chains of 32-bit elements at one workgroup per CU with
// large messages (142 VGPRs for one vector per lane: no spills)
constexpr int kHopWindowWide = 24;
constexpr int64_t kHopWindowWideMinElems = (int64_t)1 << 23;  // elements per rank
// Input values are read once: streaming (nontemporal) loads keep them from
// displacing lines in L2.  Stores of values that no later step overwrites
// are streamed too; Stage-1 partials that Stage 4 overwrites are ordinary
// stores, so that L2 can absorb the first write.
constexpr bool kNtLoads = OPTCC_NT_LOADS;
constexpr bool kNtFinal = OPTCC_NT_FINAL;
constexpr bool kNtMid = OPTCC_NT_MID;
// fp32/int32 plans whose lanes read at most this many inputs (the healthy
// ranks with one GPU per server, all p ranks with several) run two 16-byte
// vectors per lane in lockstep (measured faster for short chains)
constexpr int kTwoVectorMaxHealthy = 32;
// longer one-GPU-per-server chains take per-XCD tile runs up to this many
// tiles (measured faster at 2048 tiles and below, slower from 8192), and
// up to kXcdRunsMaxTilesMid when they have fewer than kXcdRunsWideHealthy
// healthy ranks (faster with runs at 4096 tiles too)
constexpr int64_t kXcdRunsMaxTiles = 2048;
constexpr int64_t kXcdRunsMaxTilesMid = 4096;
constexpr int kXcdRunsWideHealthy = 90;
// server plans of at least kXcdRunsWideHealthy ranks take work stealing
// above this many tiles
constexpr int64_t kServerStealMinTiles = 4096;
// ... and above kXcdRunsMaxTiles tiles from this many ranks
constexpr int kServerStealWideRanks = 120;
// mid-size messages on one-GPU-per-server chains of 32-bit elements with at
// most this many healthy ranks, whose rank buffers total at least
// kOneVectorMinBytes and less than kOneVectorMaxBytes, run one vector per
// lane in the identity tile order (measured faster than two vectors)
constexpr int kOneVectorMaxHealthy = 7;
constexpr int64_t kOneVectorMinBytes = (int64_t)16 << 20;
constexpr int64_t kOneVectorMaxBytes = (int64_t)2 << 30;
// of those, chains of at least this many healthy ranks with at least this
// many bytes of 16-byte-aligned rank buffers run three workgroups per CU
constexpr int kThreePerCuMinHealthy = 6;
constexpr int64_t kThreePerCuMinBytes = (int64_t)512 << 20;
// 32-bit chains of at least this many (and at most kTwoVectorMaxHealthy)
// healthy ranks with at least this many bytes of 16-byte-aligned rank
// buffers run one workgroup per CU (two vectors per lane)
constexpr int kTwoVecOnePerCuMinHealthy = 11;
constexpr int64_t kTwoVecOnePerCuMinBytes = (int64_t)1 << 30;
// bf16 chains of at least this many (and at most kTwoVectorMaxHealthy)
// healthy ranks, 16-byte-aligned, run three workgroups per CU at any size
constexpr int kBf16ThreePerCuMinHealthy = 13;

struct KArgs {
  const TileDesc *tiles;
  const SegDesc *segs;
  int64_t ntiles;
  int64_t n;
  int32_t pp, m;
  int32_t sb, se;  // slot range [sb, se)
  int32_t xcd_runs;  // 1: each XCD takes a contiguous run of tiles
  int32_t g;         // GPUs per server (1: one rank per server)
  // launch setting, not read by the kernel: dynamic LDS bytes reserved per
  // workgroup.  Reserving more than half of a CU's LDS holds the launch to
  // one workgroup per CU.
  int32_t occ_lds;
  // 1: the ring lanes of a whole AllReduce (slots [0, 6)) with one vector
  // per lane defer each vector's Stage 4 stores into the next vector's
  // Stage 1 chain (pipelined_ring_tile)
  int32_t pipe;
  // launch setting, not read by the kernel: workgroups to launch (0: one
  // per tile)
  int32_t grid;
  // launch setting, not read by the kernel: 1 selects the variant with the
  // hop window kHopWindowWide (32-bit, one vector per lane, one GPU per
  // server)
  int32_t wide_window;
  // work stealing when not NULL: [0] the next tile, [1] workgroups that have
  // finished; both zero at launch and reset to zero by the last workgroup
  uint32_t *steal;
  // rank pointers.  g = 1: [0, pp) healthy ranks in ring order, [pp, pp+m)
  // stragglers sorted by slowdown (worst first).  g > 1: [h*g, h*g+g) the g
  // GPUs (by local index) of the h-th healthy server in ring order, then the
  // straggler server's g GPUs at [pp*g, pp*g+g).
  void *ptr[kMaxRanks];
};

// ----------------------------------------------------------- element types
// widen / narrow / add of one element; a step is narrow(widen(a) + widen(b)).
struct F32 {
  using S = float;
  using A = float;
  static constexpr bool kPairs = false;
  __device__ static A widen(S x) { return x; }
  __device__ static S narrow(A x) { return x; }
};
struct I32 {
  using S = uint32_t;  // two's complement adds wrap modulo 2^32
  using A = uint32_t;
  static constexpr bool kPairs = false;
  __device__ static A widen(S x) { return x; }
  __device__ static S narrow(A x) { return x; }
};
// Narrowing rounds to nearest, ties to even, with gfx950's
// v_cvt_pk_bf16_f32, which also gives a NaN the required result (sign and
// top payload bits kept, made quiet): checked on all 2^32 fp32 patterns.
// Vectors narrow two values per instruction (narrow_pair, low half first).
struct BF16 {
  using S = uint16_t;
  using A = float;
  static constexpr bool kPairs = true;
  __device__ static A widen(S x) { return __uint_as_float((uint32_t)x << 16); }
  __device__ static S narrow(A f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
  __device__ static uint32_t narrow_pair(A lo, A hi) {
    typedef float f2 __attribute__((ext_vector_type(2)));
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f2){lo, hi}, b2));
  }
};

// IEEE binary16: widening is exact (v_cvt_f32_f16); narrowing rounds to
// nearest even in the default rounding mode, keeps subnormals (fp16
// denormals are not flushed) and overflows to infinity (v_cvt_f16_f32).
struct F16 {
  using S = uint16_t;
  using A = float;
  static constexpr bool kPairs = false;
  __device__ static A widen(S x) { return (float)__builtin_bit_cast(_Float16, x); }
  __device__ static S narrow(A f) { return __builtin_bit_cast(uint16_t, (_Float16)f); }
};

template <class D, int W>
struct alignas(sizeof(typename D::S) * W) Vec {
  typename D::S v[W];
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
// Address space of the rank-buffer accesses.  Pointers read from LDS are
// generic, which makes an access a FLAT instruction; FLAT accesses count
// against the LDS wait counter too, so every wait for an LDS pointer read
// also waits for the loads in flight.  Global (GA) accesses keep the two
// counters apart.  Measured: the server lane is 2 % faster with global
// accesses (q32g4_f32).  The one-GPU-per-server lanes gain at most 2 % from
// them at any message size (p = 4 to 128, 2^18 to 2^26 elements per rank;
// full-size workloads within 0.3 %): the waves of a CU keep enough loads in
// flight either way, so those lanes keep generic pointers.
template <class T, bool GA>
using MemPtr = typename std::conditional<GA, __attribute__((address_space(1))) T *, T *>::type;

// Loads and stores of W elements; NT selects the streaming hint.
template <class D, int W, bool NT, bool GA>
__device__ __forceinline__ Vec<D, W> vload(const void *base, int64_t e) {
  using S = typename D::S;
  const MemPtr<const S, GA> p = (MemPtr<const S, GA>)base + e;
  if constexpr (sizeof(Vec<D, W>) == 16) {
    const MemPtr<const u32x4, GA> q = (MemPtr<const u32x4, GA>)p;
    const u32x4 r = NT ? __builtin_nontemporal_load(q) : *q;
    return __builtin_bit_cast(Vec<D, W>, r);
  } else {
    static_assert(W == 1, "vectors are 16 bytes or one element");
    Vec<D, W> r;
    r.v[0] = NT ? __builtin_nontemporal_load(p) : *p;
    return r;
  }
}
template <class D, int W, bool NT, bool GA>
__device__ __forceinline__ void vstore(void *base, int64_t e, const Vec<D, W> &x) {
  using S = typename D::S;
  const MemPtr<S, GA> p = (MemPtr<S, GA>)base + e;
  if constexpr (sizeof(Vec<D, W>) == 16) {
    const MemPtr<u32x4, GA> q = (MemPtr<u32x4, GA>)p;
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
template <class D, int W, bool GA = false>
__device__ __forceinline__ Vec<D, W> ld_in(const void *base, int64_t e) {
  return vload<D, W, kNtLoads, GA>(base, e);
}
template <class D, int W, bool GA = false>
__device__ __forceinline__ void st_fin(void *base, int64_t e, const Vec<D, W> &x) {
  vstore<D, W, kNtFinal, GA>(base, e, x);
}
// stores of values a later step of the same section overwrites
template <class D, int W, bool GA = false>
__device__ __forceinline__ void st_mid(void *base, int64_t e, const Vec<D, W> &x) {
  vstore<D, W, kNtMid, GA>(base, e, x);
}
// One reduce step with a single source: narrow(widen(a) + widen(b)).
template <class D, int W>
__device__ __forceinline__ Vec<D, W> add2(const Vec<D, W> &a, const Vec<D, W> &b) {
  Vec<D, W> r;
  if constexpr (D::kPairs && W % 2 == 0) {
#pragma unroll
    for (int i = 0; i < W; i += 2) {
      const uint32_t h = D::narrow_pair(D::widen(a.v[i]) + D::widen(b.v[i]),
                                        D::widen(a.v[i + 1]) + D::widen(b.v[i + 1]));
      r.v[i] = (typename D::S)h;
      r.v[i + 1] = (typename D::S)(h >> 16);
    }
  } else {
#pragma unroll
    for (int i = 0; i < W; ++i) r.v[i] = D::narrow(D::widen(a.v[i]) + D::widen(b.v[i]));
  }
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
  if constexpr (D::kPairs && W % 2 == 0) {
#pragma unroll
    for (int i = 0; i < W; i += 2) {
      const uint32_t h = D::narrow_pair(a.v[i], a.v[i + 1]);
      r.v[i] = (typename D::S)h;
      r.v[i + 1] = (typename D::S)(h >> 16);
    }
  } else {
#pragma unroll
    for (int i = 0; i < W; ++i) r.v[i] = D::narrow(a.v[i]);
  }
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
    // Every destination receives the same value, so the stores may go in
    // any order: last hop first, so that the Stage-1 partials written most
    // recently are overwritten while L2 still holds them.
    for (int t = pp - 2; t >= 0; --t) {
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

// ------------------------------------------ several GPUs per server (App. E)
// Every step of one section of a part for L vectors per lane.  Each server's
// g GPUs form a local ring; position d of the part's ring is local GPU
// (part + d) mod g, position 0 the part's leader.  Collect phases (N1, N3 of
// type 2) run the ring backwards onto the leader, each GPU adding its own
// value; distribute phases (N2 of type 2, N4) copy forwards.  The NIC stages
// S1-S4 run among the leaders as in the one-GPU case.
//   type 1 (S1-S2-S3-S4): N1, S1, S2 (the straggler leader adds the holder's
//     partial), N2 fold (forward along the straggler's ring, each GPU adding
//     its own value: the last one holds the global sum), N3 (the sum copied
//     back to the leader), S3 (to the holder), S4, N4
//   type 2 (S3-S1-S4-S2): N3 collect on the straggler, N1, S3 (the
//     straggler's sum added into the chain start), S1, S4, N4, S2 (global sum
//     to the straggler leader), N2 distribute
// Every input value is read once, in the order the steps consume it: that
// flat sequence (straggler collect, then each chain server's collect, then
// the straggler's fold operands) is prefetched through a rolling window of B
// loads.  Partial sums stay in registers; every step writes its destination.
__device__ __forceinline__ int local_gpu(int part, int d, int g) {
  const int i = part + d;
  return i >= g ? i - g : i;
}

//
// G > 0: the plan has exactly G GPUs per server (a compile-time local ring).
// For slot ranges that start at slot 0 or 1 and reach slot 6 (the whole
// AllReduce among them) the lane then runs on units of one server's G
// values: the straggler server's G raw values are loaded first, the chain
// servers' units stream through a window of about B loads, and the steady
// state is straight-line code.  Other ranges, and G = 0, take the general
// path below (any g, any slot range).
template <class D, int W, int L, int B, int G>
__device__ __forceinline__ void server_lane(const KArgs &a, void *const *rp, const SegDesc &sd,
                                            const int (&j)[L], const int64_t (&e)[L]) {
  using V = Vec<D, W>;
  const int pp = a.pp, g = G > 0 ? G : a.g, part = sd.part;
  const bool t1 = sd.ordering == 1;
  // buffer of chain position t (server R[j+t], 0 <= t < pp) at local position d
  auto hr = [&](int l, int t, int d) __attribute__((always_inline)) {
    int h = j[l] + t;
    h = h >= pp ? h - pp : h;
    return rp[h * g + local_gpu(part, d, g)];
  };
  auto sr = [&](int d) __attribute__((always_inline)) { return rp[pp * g + local_gpu(part, d, g)]; };
  const bool i0 = !t1 && in_range(a, 0), i1 = in_range(a, 1), i2 = !t1 && in_range(a, 2);
  const bool i3 = in_range(a, 3), i4 = t1 && in_range(a, 4), i5 = t1 && in_range(a, 5);
  V v[L], acc[L], ss[L];
  bool have = false;  // v holds the value the next step reads
  bool head_done = false;

  if constexpr (G > 0) {
    if (a.sb <= 1 && a.se >= 6) {
      constexpr int BU = B / G > 2 ? B / G : 2;  // chain units in flight
      const bool s0 = !t1 && a.sb == 0;         // slot 0 runs
      V xs[G][L];                               // the straggler server's raw values
      if (s0 || t1) {
#pragma unroll
        for (int d = G - 1; d >= 0; --d)
#pragma unroll
          for (int l = 0; l < L; ++l) xs[d][l] = ld_in<D, W, true>(sr(d), e[l]);
      }
      V buf[BU][G][L];
      auto load_unit = [&](int t, V (&x)[G][L]) __attribute__((always_inline)) {
#pragma unroll
        for (int d = G - 1; d >= 0; --d)
#pragma unroll
          for (int l = 0; l < L; ++l) x[d][l] = ld_in<D, W, true>(hr(l, t, d), e[l]);
      };
      // slot 1: N1 collect of chain server t; acc ends as the leader's sum
      auto collect = [&](int t, const V (&x)[G][L]) __attribute__((always_inline)) {
#pragma unroll
        for (int l = 0; l < L; ++l) acc[l] = x[G - 1][l];
#pragma unroll
        for (int d = G - 2; d >= 0; --d)
#pragma unroll
          for (int l = 0; l < L; ++l) {
            acc[l] = add2<D, W>(x[d][l], acc[l]);
            st_mid<D, W, true>(hr(l, t, d), e[l], acc[l]);
          }
      };
      // slots 1 and 3 at chain server t >= 1
      auto hop = [&](int t, const V (&x)[G][L]) __attribute__((always_inline)) {
        collect(t, x);
#pragma unroll
        for (int l = 0; l < L; ++l) {
          v[l] = add2<D, W>(acc[l], v[l]);
          st_mid<D, W, true>(hr(l, t, 0), e[l], v[l]);
        }
      };
#pragma unroll
      for (int u = 0; u < BU; ++u)
        if (u < pp) load_unit(u, buf[u]);
      if (s0) {  // slot 0: N3 collect on the straggler server (type 2)
#pragma unroll
        for (int l = 0; l < L; ++l) ss[l] = xs[G - 1][l];
#pragma unroll
        for (int d = G - 2; d >= 0; --d)
#pragma unroll
          for (int l = 0; l < L; ++l) {
            ss[l] = add2<D, W>(xs[d][l], ss[l]);
            st_mid<D, W, true>(sr(d), e[l], ss[l]);
          }
      }
      collect(0, buf[0]);  // the chain start
      if (!t1) {           // slot 2: S3 into the chain start (type 2)
#pragma unroll
        for (int l = 0; l < L; ++l) {
          const V s2 = s0 ? ss[l] : ld_in<D, W, true>(sr(0), e[l]);
          v[l] = add2<D, W>(s2, acc[l]);
          st_mid<D, W, true>(hr(l, 0, 0), e[l], v[l]);
        }
      } else {
#pragma unroll
        for (int l = 0; l < L; ++l) v[l] = acc[l];
      }
      if (BU < pp) load_unit(BU, buf[0]);
      // chain servers t = 1 .. pp-1; unit t sits in buf[t mod BU]
      int t0 = 1;
      for (; t0 + 2 * BU <= pp; t0 += BU) {  // steady state: every refill exists
#pragma unroll
        for (int u = 0; u < BU; ++u) {
          hop(t0 + u, buf[(1 + u) % BU]);
          load_unit(t0 + u + BU, buf[(1 + u) % BU]);
        }
      }
      for (; t0 < pp; t0 += BU) {
#pragma unroll
        for (int u = 0; u < BU; ++u)
          if (t0 + u < pp) {
            hop(t0 + u, buf[(1 + u) % BU]);
            if (t0 + u + BU < pp) load_unit(t0 + u + BU, buf[(1 + u) % BU]);
          }
      }
      if (t1) {  // slot 4: S2; slot 5: N2 fold along the straggler's ring
#pragma unroll
        for (int l = 0; l < L; ++l) {
          v[l] = add2<D, W>(xs[0][l], v[l]);
          st_mid<D, W, true>(sr(0), e[l], v[l]);
        }
#pragma unroll
        for (int d = 1; d < G; ++d)
#pragma unroll
          for (int l = 0; l < L; ++l) {
            v[l] = add2<D, W>(xs[d][l], v[l]);
            if (d == G - 1) st_fin<D, W, true>(sr(d), e[l], v[l]);
            else st_mid<D, W, true>(sr(d), e[l], v[l]);
          }
      }
      have = true;
      head_done = true;
    }
  }
  if (!head_done) {  // general path: any g, any slot range
    // Slots 2/3 without slot 1 (partial slot ranges only): the leaders already
    // hold their collected values.
    if (!i1 && (i2 || i3)) {
#pragma unroll
      for (int l = 0; l < L; ++l) v[l] = ld_in<D, W, true>(hr(l, 0, 0), e[l]);
      if (i2) {
#pragma unroll
        for (int l = 0; l < L; ++l) {
          v[l] = add2<D, W>(ld_in<D, W, true>(sr(0), e[l]), v[l]);
          st_mid<D, W, true>(hr(l, 0, 0), e[l], v[l]);
        }
      }
      if (i3)
        for (int t = 1; t < pp; ++t) {
#pragma unroll
          for (int l = 0; l < L; ++l) {
            v[l] = add2<D, W>(ld_in<D, W, true>(hr(l, t, 0), e[l]), v[l]);
            st_mid<D, W, true>(hr(l, t, 0), e[l], v[l]);
          }
        }
      have = i3;
    }

    // The flat input sequence: [0, nA) straggler collect (slot 0), [nA, nA+nB)
    // chain servers' collects (slot 1, with slots 2/3 folded in at each
    // leader), then the straggler's operands of slots 4/5.
    const int nA = i0 ? g : 0, nB = i1 ? pp * g : 0;
    const int n = nA + nB + (i4 ? 1 : 0) + (i5 ? g - 1 : 0);
    const int c0 = i4 ? 0 : 1;  // straggler position of the first slot-4/5 operand
    struct Cur {
      int i, t, d;  // flat index; chain position and local position inside [nA, nA+nB)
    };
    auto cur_ptr = [&](int l, const Cur &c) __attribute__((always_inline)) {
      if (c.i < nA) return sr(g - 1 - c.i);
      if (c.i < nA + nB) return hr(l, c.t, c.d);
      return sr(c.i - nA - nB + c0);
    };
    auto cur_next = [&](Cur &c) __attribute__((always_inline)) {
      if (c.i >= nA && c.i < nA + nB && --c.d < 0) {
        c.d = g - 1;
        ++c.t;
      }
      ++c.i;
    };
    // Every input value feeds one running sum `acc`: the collects (slots 0, 1)
    // start from the raw value at the far end of a local ring and add one GPU
    // per step; the straggler's S2 and N2 fold (slots 4, 5) continue from the
    // holder's partial.  The chain steps (slots 2, 3) run when a leader's
    // collect completes.
    auto consume = [&](const Cur &c, const V (&x)[L]) __attribute__((always_inline)) {
      const bool inA = c.i < nA, inB = !inA && c.i < nA + nB, inC = !inA && !inB;
      const int d = inA ? g - 1 - c.i : (inB ? c.d : c.i - nA - nB + c0);
      const bool raw = !inC && d == g - 1;  // the far end of a collect: no step
      if (inC && c.i == nA + nB) {           // first of slots 4/5: the state it continues
#pragma unroll
        for (int l = 0; l < L; ++l)
          acc[l] = have ? v[l] : ld_in<D, W, true>(d == 0 ? hr(l, pp - 1, 0) : sr(0), e[l]);
      }
#pragma unroll
      for (int l = 0; l < L; ++l) {
        acc[l] = raw ? x[l] : add2<D, W>(x[l], acc[l]);
        if (!raw) {
          void *dst = inB ? hr(l, c.t, d) : sr(d);
          if (inC && d == g - 1) st_fin<D, W, true>(dst, e[l], acc[l]);  // the global sum
          else st_mid<D, W, true>(dst, e[l], acc[l]);
        }
      }
      if (inA && d == 0) {  // the straggler leader holds its server's sum
#pragma unroll
        for (int l = 0; l < L; ++l) ss[l] = acc[l];
      }
      if (inB && d == 0) {  // leader t holds its server's sum
        if (c.t == 0) {
          if (i2) {  // slot 2: S3 into the chain start (type 2)
#pragma unroll
            for (int l = 0; l < L; ++l) {
              const V s2 = i0 ? ss[l] : ld_in<D, W, true>(sr(0), e[l]);
              v[l] = add2<D, W>(s2, acc[l]);
              st_mid<D, W, true>(hr(l, 0, 0), e[l], v[l]);
            }
          } else {
#pragma unroll
            for (int l = 0; l < L; ++l) v[l] = acc[l];
          }
        } else if (i3) {  // slot 3: S1 hop into leader t
#pragma unroll
          for (int l = 0; l < L; ++l) {
            v[l] = add2<D, W>(acc[l], v[l]);
            st_mid<D, W, true>(hr(l, c.t, 0), e[l], v[l]);
          }
        }
        if (c.t == pp - 1) have = i3;
      }
    };
    {
      V buf[B][L];
      Cur pc{0, 0, g - 1}, cc{0, 0, g - 1};
#pragma unroll
      for (int u = 0; u < B; ++u)
        if (u < n) {
#pragma unroll
          for (int l = 0; l < L; ++l) buf[u][l] = ld_in<D, W, true>(cur_ptr(l, pc), e[l]);
          cur_next(pc);
        }
      for (int t0 = 0; t0 < n; t0 += B) {
#pragma unroll
        for (int u = 0; u < B; ++u)
          if (t0 + u < n) {
            consume(cc, buf[u]);
            cur_next(cc);
            if (t0 + u + B < n) {
#pragma unroll
              for (int l = 0; l < L; ++l) buf[u][l] = ld_in<D, W, true>(cur_ptr(l, pc), e[l]);
              cur_next(pc);
            }
          }
      }
    }
    if (i4 || i5) {  // slots 4/5 ran: the straggler's running sum is the state
#pragma unroll
      for (int l = 0; l < L; ++l) v[l] = acc[l];
      have = true;
    }
  }

  if (t1 && in_range(a, 6)) {  // slot 6: N3, the global sum back to the leader
#pragma unroll
    for (int l = 0; l < L; ++l)
      if (!have) v[l] = ld_in<D, W, true>(sr(g - 1), e[l]);
    for (int d = g - 2; d >= 0; --d) {
#pragma unroll
      for (int l = 0; l < L; ++l) st_fin<D, W, true>(sr(d), e[l], v[l]);
    }
    have = true;
  }
  if (t1 && in_range(a, 7)) {  // slot 7: S3, straggler leader -> holder
#pragma unroll
    for (int l = 0; l < L; ++l) {
      if (!have) v[l] = ld_in<D, W, true>(sr(0), e[l]);
      st_fin<D, W, true>(hr(l, pp - 1, 0), e[l], v[l]);
    }
    have = true;
  }
  // Slots 8 and 9 store one value everywhere, in any order: the servers
  // last in the chain first (as in ring_lane), so that the partials their
  // leaders and local GPUs wrote most recently are overwritten while L2
  // still holds them.
  if (in_range(a, 8)) {  // slot 8: S4 allgather from the holder
#pragma unroll
    for (int l = 0; l < L; ++l)
      if (!have) v[l] = ld_in<D, W, true>(hr(l, pp - 1, 0), e[l]);
    for (int t = pp - 2; t >= 0; --t) {
#pragma unroll
      for (int l = 0; l < L; ++l) st_fin<D, W, true>(hr(l, t, 0), e[l], v[l]);
    }
    have = true;
  }
  if (in_range(a, 9)) {  // slot 9: N4 distribute on every healthy server
    for (int t = pp - 1; t >= 0; --t) {
      V gt[L];
#pragma unroll
      for (int l = 0; l < L; ++l) gt[l] = have ? v[l] : ld_in<D, W, true>(hr(l, t, 0), e[l]);
      for (int d = 1; d < g; ++d) {
#pragma unroll
        for (int l = 0; l < L; ++l) st_fin<D, W, true>(hr(l, t, d), e[l], gt[l]);
      }
    }
  }
  if (!t1 && in_range(a, 10)) {  // slot 10: S2, holder -> straggler leader
#pragma unroll
    for (int l = 0; l < L; ++l) {
      if (!have) v[l] = ld_in<D, W, true>(hr(l, pp - 1, 0), e[l]);
      st_fin<D, W, true>(sr(0), e[l], v[l]);
    }
    have = true;
  }
  if (!t1 && in_range(a, 11)) {  // slot 11: N2 distribute on the straggler server
#pragma unroll
    for (int l = 0; l < L; ++l)
      if (!have) v[l] = ld_in<D, W, true>(sr(0), e[l]);
    for (int d = 1; d < g; ++d) {
#pragma unroll
      for (int l = 0; l < L; ++l) st_fin<D, W, true>(sr(d), e[l], v[l]);
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

// Every ring-section vector of one tile's lane, for a whole AllReduce
// (slots [0, 6)), one GPU per server, one vector at a time: vector v's
// Stage 1 chain carries, one per hop, the Stage 4 stores of vector v - 1
// (last hop first, as in ring_lane),
// and the stragglers' copies of vector v - 1 follow the chain, so that a
// wave keeps loads in flight while it writes the previous vector's
// allgather.  Each vector gets exactly the steps ring_lane gives it (other
// coordinates only move in time), so the result is the same bit for bit.
// Elements past the last whole vector of the tile are left to the caller.
template <class D, int W, int B>
__device__ void pipelined_ring_tile(const KArgs &a, void *const *rp, const SegDesc &sd,
                                    int64_t e0, int64_t end, int64_t stride) {
  using V = Vec<D, W>;
  const int pp = a.pp, m = a.m;
  const int ord = sd.ordering;
  const int nside = m == 0 ? 0 : (ord == 2 ? m : m - 1);
  const int sfirst = ord == 2 ? 0 : 1;
  const bool fin = m >= 1 && ord == 1;
  const int nh = pp - 1;
  bool pend = false;  // vector v - 1 still owes its Stage 4 and slot-5 stores
  V vp;
  int jp = 0;
  int64_t ep = 0;
  auto rank_at = [&](int j, int t) {  // buffer of R[j + t], 0 <= t < 2 pp
    int i = j + t;
    return rp[i >= pp ? i - pp : i];
  };
  for (; e0 + W <= end; e0 += stride) {
    const int j = section_of(sd, (e0 - sd.ring_begin) / kQuantum);
    V xs;
    if (fin) xs = ld_in<D, W>(a.ptr[pp], e0);
    V v;
    if (nside > 0) {  // slot 0: stragglers' raw values into the chain start
      AccV<D, W> acc = widen(ld_in<D, W>(rp[j], e0));
      for (int i = 0; i < nside; ++i) accum(acc, ld_in<D, W>(a.ptr[pp + sfirst + i], e0));
      v = narrow(acc);
      st_mid<D, W>(rp[j], e0, v);
    } else {
      v = ld_in<D, W>(rp[j], e0);
    }
    // slot 1: the chain, with a rolling window of B hop loads; hop t also
    // stores the t-th Stage 4 value of the previous vector
    V buf[B];
#pragma unroll
    for (int u = 0; u < B; ++u)
      if (u < nh) buf[u] = ld_in<D, W>(rank_at(j, 1 + u), e0);
    for (int t = 0; t < nh; t += B) {
#pragma unroll
      for (int u = 0; u < B; ++u)
        if (t + u < nh) {
          v = add2<D, W>(buf[u], v);
          st_mid<D, W>(rank_at(j, 1 + t + u), e0, v);
          if (t + u + B < nh) buf[u] = ld_in<D, W>(rank_at(j, 1 + t + u + B), e0);
          if (pend) st_fin<D, W>(rank_at(jp, nh - 1 - (t + u)), ep, vp);
        }
    }
    if (pend) {  // slot 5 of the previous vector
      for (int i = 0; i < nside; ++i) st_fin<D, W>(a.ptr[pp + sfirst + i], ep, vp);
    }
    if (fin) {  // slots 2 and 3: the finalising straggler and back to the holder
      v = add2<D, W>(xs, v);
      st_fin<D, W>(a.ptr[pp], e0, v);
      st_fin<D, W>(rank_at(j, pp - 1), e0, v);
    }
    pend = true;
    vp = v;
    jp = j;
    ep = e0;
  }
  if (pend) {
    for (int t = pp - 2; t >= 0; --t) st_fin<D, W>(rank_at(jp, t), ep, vp);
    for (int i = 0; i < nside; ++i) st_fin<D, W>(a.ptr[pp + sfirst + i], ep, vp);
  }
}

template <class D, int W, int L, int B, bool S, int G>
__device__ __forceinline__ void run_elems(const KArgs &a, void *const *rp, const SegDesc &sd,
                                          bool p2p, const int64_t (&e)[L]) {
  if (!S && p2p) {
    p2p_lane<D, W, L, B>(a, rp, e);
  } else {
    int j[L];
#pragma unroll
    for (int l = 0; l < L; ++l) j[l] = section_of(sd, (e[l] - sd.ring_begin) / kQuantum);
    if constexpr (S) server_lane<D, W, L, B, G>(a, rp, sd, j, e);
    else ring_lane<D, W, L, B>(a, rp, sd, j, e);
  }
}

// One tile: every step of the schedule on its elements.  W elements per
// lane access: 16 bytes when every rank buffer is 16-byte aligned, else 1
// element.  A lane takes L such vectors of the tile at a stride of one
// workgroup-width, in lockstep; vectors past the tile's last whole group go
// one at a time, and elements past the last whole vector (only at the end
// of the rank vectors) one by one.
template <class D, int W, int L, bool S, int G, int B>
__device__ __forceinline__ void run_tile(const KArgs &a, void *const *rp, int64_t t) {
  constexpr int64_t kStride = (int64_t)kThreads * W;
  const TileDesc td = a.tiles[t];
  const bool p2p = td.meta & 1;
  const SegDesc sd = a.segs[td.meta >> 1];
  const int64_t end = td.begin + td.len;
  int64_t e0 = td.begin + (int64_t)threadIdx.x * W;
  if constexpr (!S && L == 1) {
    if (a.pipe && !p2p && a.sb == 0 && a.se == OPTCC_NUM_SLOTS) {
      pipelined_ring_tile<D, W, B>(a, rp, sd, e0, end, kStride);
      int64_t x = e0 + (end - W - e0 >= 0 ? ((end - W - e0) / kStride + 1) * kStride : 0);
      for (; x < end; x += kStride)
        for (int64_t y = x; y < end && y < x + W; ++y) {
          const int64_t e[1] = {y};
          run_elems<D, 1, 1, B, S, G>(a, rp, sd, p2p, e);
        }
      return;
    }
  }
  for (; e0 + (L - 1) * kStride + W <= end; e0 += L * kStride) {
    int64_t e[L];
#pragma unroll
    for (int l = 0; l < L; ++l) e[l] = e0 + l * kStride;
    run_elems<D, W, L, B, S, G>(a, rp, sd, p2p, e);
  }
  for (; e0 < end; e0 += kStride) {
    if (e0 + W <= end) {
      const int64_t e[1] = {e0};
      run_elems<D, W, 1, B, S, G>(a, rp, sd, p2p, e);
    } else {
      for (int64_t x = e0; x < end; ++x) {
        const int64_t e[1] = {x};
        run_elems<D, 1, 1, B, S, G>(a, rp, sd, p2p, e);
      }
    }
  }
}

// S selects the several-GPUs-per-server lane (App. E); its plans have no
// point-to-point chunks.  G: GPUs per server when fixed at compile time
// (0: read from the arguments).  B: hop loads in flight per vector.
template <class D, int W, int L, bool S, int G, int B = kHopWindow>
__global__ __launch_bounds__(kThreads) void optcc_exec_kernel(KArgs a) {
  __shared__ void *rp[kMaxRanks];
  const int nrp = S ? (a.pp + 1) * a.g : a.pp;  // pointers the lanes index from LDS
  for (int i = threadIdx.x; i < nrp; i += kThreads) rp[i] = a.ptr[i];
  __syncthreads();
  if (a.steal) {
    // Work stealing: a grid of at most the resident workgroups takes tiles
    // in order from one device counter, so the CUs and XCDs that run ahead
    // take more of them.  Every workgroup leaves once the counter has passed
    // the last tile; the last one to leave resets the counters for the next
    // launch that uses them.
    __shared__ int64_t next;
    for (;;) {
      if (threadIdx.x == 0) {
        const uint32_t i = atomicAdd(&a.steal[0], 1u);
        next = (int64_t)i < a.ntiles ? (int64_t)i : -1;
      }
      __syncthreads();
      const int64_t t = next;
      __syncthreads();
      if (t < 0) break;
      run_tile<D, W, L, S, G, B>(a, rp, t);
    }
    if (threadIdx.x == 0) {
      __threadfence();
      if (atomicAdd(&a.steal[1], 1u) == gridDim.x - 1) {
        __threadfence();
        atomicExch(&a.steal[0], 0u);
        atomicExch(&a.steal[1], 0u);
      }
    }
    return;
  }
  // Static order.  Workgroups are dealt to the XCDs round robin by workgroup
  // index.  With xcd_runs, workgroup t0 takes tile (t0 mod X) * per + t0 / X,
  // so each XCD sweeps its own contiguous run of tiles.  Any XCD count keeps
  // every tile covered exactly once; X = 8 matches MI355X.
  constexpr int64_t kXcds = 8;
  const int64_t per = (a.ntiles + kXcds - 1) / kXcds;
  const int64_t cover = a.xcd_runs ? per * kXcds : a.ntiles;
  for (int64_t t0 = blockIdx.x; t0 < cover; t0 += gridDim.x) {
    const int64_t t = a.xcd_runs ? (t0 % kXcds) * per + t0 / kXcds : t0;
    if (t < a.ntiles) run_tile<D, W, L, S, G, B>(a, rp, t);
  }
}

}  // namespace kern
}  // namespace optcc
