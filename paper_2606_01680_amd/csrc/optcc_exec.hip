// Host side of the OptCC executor on one MI355X (gfx950, CDNA4): argument
// checks, the per-device plan tables and kernel launches.  The kernels are
// in optcc_kernels.hpp, instantiated per element type in optcc_kern_*.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <tuple>
#include <utility>
#include <vector>

#include "optcc_internal.hpp"
#include "optcc_launch.hpp"

namespace optcc {
namespace {

using namespace kern;

// The plan's host tile table for tiles of tile_elems elements: tile_elems-
// element pieces of every segment's ring part and P2P chunk, built once per
// tile length.  The caller holds pl.mu; the vector lives as long as the plan.
const std::vector<TileDesc> &host_tiles(const optcc_plan_t &pl, int tile_elems) {
  auto it = pl.host_tiles.find(tile_elems);
  if (it != pl.host_tiles.end()) return it->second;
  std::vector<TileDesc> &tiles = pl.host_tiles[tile_elems];
  for (int g = 0; g < pl.nseg; ++g) {
    const Segment &s = pl.seg[(size_t)g];
    auto cut = [&](int64_t b, int64_t e, int is_p2p) {
      for (int64_t x = b; x < e; x += tile_elems) {
        TileDesc t;
        t.begin = x;
        t.len = (int32_t)std::min<int64_t>(tile_elems, e - x);
        t.meta = (g << 1) | is_p2p;
        tiles.push_back(t);
      }
    };
    cut(std::min(s.ring_begin, pl.n), s.ring_end, 0);
    cut(s.p2p_begin, s.p2p_end, 1);
  }
  return tiles;
}

// Number of tiles host_tiles cuts for tiles of tile_elems elements.
int64_t tile_count(const optcc_plan_t &pl, int tile_elems) {
  int64_t t = 0;
  for (int g = 0; g < pl.nseg; ++g) {
    const Segment &s = pl.seg[(size_t)g];
    const int64_t rb = std::min(s.ring_begin, pl.n);
    if (s.ring_end > rb) t += (s.ring_end - rb + tile_elems - 1) / tile_elems;
    if (s.p2p_end > s.p2p_begin) t += (s.p2p_end - s.p2p_begin + tile_elems - 1) / tile_elems;
  }
  return t;
}

// The plan's tables for tiles of tile_elems elements on the current device,
// uploaded on first use and cached.  The upload (hipMalloc, hipMemcpy) may
// not run while `stream` is being captured into a graph: such a first call
// fails before touching the device, and the capture stays valid.
int device_tables(const optcc_plan_t &pl, int tile_elems, hipStream_t stream, DeviceTables *out) {
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return fail(OPTCC_EDEVICE, std::string("hipGetDevice: ") + hipGetErrorString(err));
  std::lock_guard<std::mutex> lk(pl.mu);
  auto it = pl.dev.find({dev, tile_elems});
  if (it != pl.dev.end()) {
    *out = it->second;
    return OPTCC_OK;
  }
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(stream, &cap) == hipSuccess && cap != hipStreamCaptureStatusNone)
    return fail(OPTCC_EINVAL,
                "the stream is being captured and this plan's tables for this device and "
                "element size are not uploaded yet: run the plan once outside the capture first");
  const std::vector<TileDesc> &tiles = host_tiles(pl, tile_elems);
  DeviceTables d;
  const size_t sb = pl.segdesc.size() * sizeof(SegDesc);
  const size_t tb = std::max<size_t>(tiles.size(), 1) * sizeof(TileDesc);
  err = hipMalloc(&d.segs, sb);
  if (err == hipSuccess) err = hipMalloc(&d.tiles, tb);
  if (err == hipSuccess) err = hipMemcpy(d.segs, pl.segdesc.data(), sb, hipMemcpyHostToDevice);
  if (err == hipSuccess && !tiles.empty())
    err = hipMemcpy(d.tiles, tiles.data(), tiles.size() * sizeof(TileDesc), hipMemcpyHostToDevice);
  if (err != hipSuccess) {
    if (d.segs) (void)hipFree(d.segs);
    if (d.tiles) (void)hipFree(d.tiles);
    return fail(err == hipErrorOutOfMemory ? OPTCC_ENOMEM : OPTCC_EDEVICE,
                std::string("uploading plan tables: ") + hipGetErrorString(err));
  }
  d.ntiles = (int64_t)tiles.size();
  pl.dev[{dev, tile_elems}] = d;
  *out = d;
  return OPTCC_OK;
}

// The work-stealing counter blocks of the plan's tables for tiles of
// tile_elems elements on the current device: kStealSlots blocks, allocated
// and zeroed on the first launch that steals (never under capture: such
// launches keep the static order).  NULL if they cannot be allocated; the
// caller then keeps the static order, which gives the same result.
uint32_t *steal_counters(const optcc_plan_t &pl, int tile_elems) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  std::lock_guard<std::mutex> lk(pl.mu);
  auto it = pl.dev.find({dev, tile_elems});
  if (it == pl.dev.end()) return nullptr;
  DeviceTables &d = it->second;
  if (!d.steal) {
    const size_t wb = (size_t)kStealSlots * kStealWords * sizeof(uint32_t);
    uint32_t *c = nullptr;
    if (hipMalloc(&c, wb) != hipSuccess) return nullptr;
    // zeroed in place before this call returns, like the tables
    const std::vector<uint32_t> zero((size_t)kStealSlots * kStealWords, 0u);
    if (hipMemcpy(c, zero.data(), wb, hipMemcpyHostToDevice) != hipSuccess) {
      (void)hipFree(c);
      return nullptr;
    }
    d.steal = c;
  }
  return d.steal;
}

// Device memory of optcc_allreduce_emulate_noalloc: the plan's tables are
// staged here on every call instead of in memory of their own.  One copy per
// GPU, held until the process ends; calls on one GPU share it.
static __device__ __align__(256) unsigned char scratch[OPTCC_NOALLOC_SCRATCH_BYTES];

// Device address of this GPU's `scratch` (the array's name is a host-side
// stand-in in host code): looked up once per device, with it current.
int scratch_address(void **out) {
  static std::mutex mu;
  static std::map<int, void *> addr;
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return fail(OPTCC_EDEVICE, std::string("hipGetDevice: ") + hipGetErrorString(err));
  std::lock_guard<std::mutex> lk(mu);
  auto it = addr.find(dev);
  if (it == addr.end()) {
    void *ptr = nullptr;
    err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (err != hipSuccess || !ptr)
      return fail(OPTCC_EDEVICE, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(err));
    it = addr.emplace(dev, ptr).first;
  }
  *out = it->second;
  return OPTCC_OK;
}

// Bytes of the plan's tables for `ntiles` tiles staged in the no-allocation
// array: segment descriptors (rounded up to 256 bytes), then the tiles.
size_t scratch_bytes(const optcc_plan_t &pl, int64_t ntiles) {
  const size_t seg_bytes = pl.segdesc.size() * sizeof(SegDesc);
  return (seg_bytes + 255) / 256 * 256 + (size_t)ntiles * sizeof(TileDesc);
}

// The plan's tables staged in `scratch` by two copies on `stream` (no device
// allocation).  The host tables are the plan's and live as long as it does.
int scratch_tables(const optcc_plan_t &pl, int tile_elems, hipStream_t stream, DeviceTables *out) {
  const std::vector<TileDesc> *tiles;
  {
    std::lock_guard<std::mutex> lk(pl.mu);
    tiles = &host_tiles(pl, tile_elems);
  }
  const size_t seg_bytes = pl.segdesc.size() * sizeof(SegDesc);
  const size_t tile_off = (seg_bytes + 255) / 256 * 256;
  const size_t tile_bytes = tiles->size() * sizeof(TileDesc);
  if (scratch_bytes(pl, (int64_t)tiles->size()) > (size_t)OPTCC_NOALLOC_SCRATCH_BYTES)
    return fail(OPTCC_EUNSUPPORTED,
                "the plan's tables need " + std::to_string(tile_off + tile_bytes) +
                    " bytes, more than the " + std::to_string(OPTCC_NOALLOC_SCRATCH_BYTES) +
                    " of the no-allocation scratch array: use optcc_allreduce_emulate");
  void *base = nullptr;
  int rc = scratch_address(&base);
  if (rc != OPTCC_OK) return rc;
  char *b = static_cast<char *>(base);
  hipError_t err = hipMemcpyAsync(b, pl.segdesc.data(), seg_bytes, hipMemcpyHostToDevice, stream);
  if (err == hipSuccess && tile_bytes)
    err = hipMemcpyAsync(b + tile_off, tiles->data(), tile_bytes, hipMemcpyHostToDevice, stream);
  if (err != hipSuccess)
    return fail(OPTCC_EDEVICE, std::string("staging plan tables: ") + hipGetErrorString(err));
  out->segs = reinterpret_cast<SegDesc *>(b);
  out->tiles = reinterpret_cast<TileDesc *>(b + tile_off);
  out->ntiles = (int64_t)tiles->size();
  return OPTCC_OK;
}

// Dynamic LDS (not used by the kernel) that holds a launch to at most n
// workgroups per CU on the current device (0 if the device cannot reserve
// that much), cached per device and n.  Measured on MI355X at one
// workgroup per CU: chains of more than 32 healthy ranks run 2.6-8 %
// faster at one workgroup (4 waves) per CU than at the 4 workgroups their
// registers allow (P' = 39, 47, 62, 95, 124); shorter chains gain nothing
// and p = 8 loses 10 %.  Server plans of more than 32 ranks (with per-XCD
// tile runs): q16g4 -1.5 %, q32g4 -6 %, 8x8 and 16x8 GPUs -2 to -4 %,
// 32x2 and 64x2 +1 to +4 %.
int workgroups_per_cu_lds(int n) {
  static std::mutex mu;
  static std::map<std::pair<int, int>, int> cache;
  int dev = 0;
  if (n < 1 || hipGetDevice(&dev) != hipSuccess) return 0;
  std::lock_guard<std::mutex> lk(mu);
  auto it = cache.find({dev, n});
  if (it != cache.end()) return it->second;
  int per_cu = 0, per_block = 0;
  int v = 0;
  if (hipDeviceGetAttribute(&per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) ==
          hipSuccess &&
      hipDeviceGetAttribute(&per_block, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) ==
          hipSuccess) {
    // fixed + want is just over 1/(n+1) of the CU's LDS, so n + 1
    // workgroups never fit, and n still do (n * 256 bytes of margin is far
    // below per_cu / (n + 1) for the n used here)
    const int fixed = (int)(sizeof(void *) * kMaxRanks);  // the kernel's rank-pointer table
    const int want = per_cu / (n + 1) + 256 - fixed;
    if (want > 0 && fixed + want <= per_block && (int64_t)n * (fixed + want) <= per_cu) v = want;
  }
  cache[{dev, n}] = v;
  return v;
}

// Workgroups of the launch's kernel variant the whole device holds at once
// (CUs x workgroups per CU at its registers and dynamic LDS), cached per
// device and variant; 0 if the runtime cannot tell.
int resident_workgroups(const KArgs &a, optcc_dtype_t dtype, bool servers, bool vec16, bool two) {
  static std::mutex mu;
  static std::map<std::tuple<int, int, int, int, int, int, int>, int> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  const auto key = std::make_tuple(dev, (int)dtype, (int)servers, (int)vec16, (int)two,
                                   servers ? a.g : 0, a.occ_lds);
  std::lock_guard<std::mutex> lk(mu);
  auto it = cache.find(key);
  if (it != cache.end()) return it->second;
  int per_cu = 0, cus = 0;
  hipError_t err = hipSuccess;
  switch (dtype) {
    case OPTCC_F32: err = launch_f32(a, servers, vec16, two, nullptr, &per_cu); break;
    case OPTCC_BF16: err = launch_bf16(a, servers, vec16, two, nullptr, &per_cu); break;
    case OPTCC_F16: err = launch_f16(a, servers, vec16, two, nullptr, &per_cu); break;
    default: err = launch_i32(a, servers, vec16, two, nullptr, &per_cu); break;
  }
  if (err != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    per_cu = cus = 0;
  const int v = per_cu > 0 && cus > 0 ? per_cu * cus : 0;
  cache[key] = v;
  return v;
}

int emulate(void *const *bufs, int p, int64_t N, optcc_dtype_t dtype, const optcc_plan_t *pl,
            int sb, int se, int launches, void *stream, bool noalloc = false) {
  set_error("");
  if (!pl) return fail(OPTCC_EINVAL, "plan is NULL");
  if (!bufs) return fail(OPTCC_EINVAL, "bufs is NULL");
  if (p != pl->p || N != pl->n) return fail(OPTCC_EINVAL, "p or N differ from the plan's");
  if (dtype != OPTCC_F32 && dtype != OPTCC_BF16 && dtype != OPTCC_I32 && dtype != OPTCC_F16)
    return fail(OPTCC_EINVAL, "unknown dtype");
  if (sb < 0 || se > pl->nslots || sb > se)
    return fail(OPTCC_EINVAL, "slot range must satisfy 0 <= begin <= end <= " + std::to_string(pl->nslots));
  if (launches != 0 && launches != 1)
    return fail(OPTCC_EINVAL, "launches must be 0 (one per slot) or 1 (fused)");
  if (p > kMaxRanks) return fail(OPTCC_EUNSUPPORTED, "p exceeds OPTCC_MAX_EMULATE_RANKS");
  if (N == 0 || sb == se) return OPTCC_OK;  // nothing to move; pointers are not touched
  const size_t es = dtype == OPTCC_BF16 || dtype == OPTCC_F16 ? 2 : 4;
  // pointers: non-NULL, element-aligned, pairwise disjoint
  std::vector<std::pair<uintptr_t, int>> ranges;
  bool vec16 = true;
  for (int r = 0; r < p; ++r) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(bufs[r]);
    if (!a) return fail(OPTCC_EINVAL, "bufs[" + std::to_string(r) + "] is NULL");
    if (a > UINTPTR_MAX - (uintptr_t)N * es)
      return fail(OPTCC_EINVAL, "bufs[" + std::to_string(r) + "] + N elements would run past the end of the address space");
    if (a % es)
      return fail(OPTCC_EINVAL, "bufs[" + std::to_string(r) + "] is not aligned to the element size");
    if (a % 16) vec16 = false;
    ranges.push_back({a, r});
  }
  std::sort(ranges.begin(), ranges.end());
  for (size_t i = 1; i < ranges.size(); ++i)
    if (ranges[i - 1].first + (uintptr_t)N * es > ranges[i].first)
      return fail(OPTCC_EINVAL, "rank buffers overlap");
  // The device tables index a segment's ring quanta in 32 bits (SegDesc,
  // section_of): refuse a plan whose segments would not fit.
  for (const Segment &s : pl->seg)
    if (s.qbase * (int64_t)pl->pp + s.nbig > (int64_t)INT32_MAX)
      return fail(OPTCC_EUNSUPPORTED, "a segment's ring sections hold 2^31 or more quanta; use "
                                      "more segments (n_chunks) or a smaller N");

  // Tile length: 2048 elements, doubled (up to 8192) while a tile would move
  // less than kTileMinBytes4/2 of algorithmic traffic (about 3p - 2
  // accesses per element).  Measured with one straggler, 2 GiB of buffers,
  // against 2048: fp32 p = 3 -7 % and p = 4 -3 % at 4096 (p = 5 +0.3 %);
  // int32 p = 4 -4 %; bf16 p = 3 -18 % at 8192, p = 4 -11 % and p = 6
  // -2 % at 4096, p = 7 +7 % and p = 8 +7 % at 4096; fp16 p = 4 -6 %,
  // p = 8 +7 % at 4096.
  int tile_elems = kTileElems;
  const int64_t per_elem = (3 * (int64_t)p - 2) * (int64_t)es;
  const int64_t min_bytes = es == 2 ? kTileMinBytes2 : kTileMinBytes4;
  while (tile_elems < kTileElemsMax && (int64_t)tile_elems * per_elem < min_bytes) tile_elems *= 2;
  // Small messages: halve the tile, down to one 16-byte vector per lane,
  // while there would be fewer than kTileMinCount tiles, so that more CUs
  // take part.  Measured with 200 back-to-back calls: p = 4 fp32 at 2^16
  // elements per rank 6.9 -> 4.1 us, p = 8 fp32 at 2^18 8.8 -> 6.1 us, no
  // change from 2^20 up or at p = 128; a bound of 4096 tiles was 4-7 %
  // slower at 2^22 (p = 8 and 128).
  const int vec_tile = kern::kThreads * (int)(16 / es);
  while (tile_elems > vec_tile && N / tile_elems < kTileMinCount) tile_elems /= 2;

  // Launch shape.  Short chains (inputs per lane: P' for one GPU per
  // server, p for several): two vectors per lane (measured faster up to 32
  // and neutral or slower beyond).  Longer chains run one workgroup per CU.
  // Per-XCD tile runs: for short chains, for server plans (beyond 32
  // ranks, together with one workgroup per CU, 2.4-27 % faster than with
  // neither; the largest take work stealing instead, below) and for longer one-GPU-per-server chains whose tiles are more
  // than one round of resident workgroups and at most kXcdRunsMaxTiles
  // (measured with 2048-element tiles, p = 64 and 128 at 2^19-2^22 elements
  // per rank: 2.4-14 % faster; at 4096 tiles -8 % at p = 64, +4 % at
  // p = 128; from 8192 tiles 0.8-0.9 % slower; with one round of tiles,
  // 2^17-2^18 elements per rank, 3-5 % slower).
  // bf16 long chains run one workgroup per CU as well (and take work
  // stealing like the others).  Measured against full occupancy (back-to-
  // back calls, results bit for bit equal): 34-256 ranks, 2^21-2^25
  // elements per rank, 2.9-16 % faster (p = 128 at 2^23 985 -> 891 us,
  // 256 ranks at 2^21 584 -> 504 us); p = 128 at 2^20 1 % and 64 ranks
  // with bubble filling at 2^23 0.5 % slower.  bf16 server plans of more
  // than 32 ranks gain from it too (16 x 4 -3 %, 8 x 8 -1.3 %).
  // A single-hop chain (two healthy ranks, p = 3 with one straggler) runs
  // one vector per lane in the identity order: 8 % faster than two vectors
  // with XCD runs (p = 4 is fastest with both).
  // Mid-size messages on short chains of 32-bit elements (3 to 7 healthy
  // ranks, rank buffers of 16 MiB to 2 GiB in total) run one vector per lane
  // in the identity order, in 1024-element tiles from 5 healthy ranks up.
  // Measured (back-to-back calls, against two vectors with XCD runs): p = 8
  // one straggler at 2^20-2^25 elements per rank 3-14 % faster (2^21:
  // 29.9 -> 27.1 us, 2^22: 52.8 -> 48.0 us), int32 likewise; p = 6 at 2^22
  // and 2^24 4-9 %; p = 4 (4096-element tiles) at 2^22 and 2^24 8-21 %; at
  // 2 GiB (p = 8, 2^26) two vectors stay 4 % faster.
  const bool servers = pl->kind == OPTCC_KIND_SERVERS;
  const int chain = servers ? pl->p : pl->pp;
  const bool long_chain = chain > kTwoVectorMaxHealthy;
  const bool single_hop = !servers && pl->pp == 2;
  const int64_t buf_bytes = (int64_t)p * N * (int64_t)es;
  const bool mid_short = !servers && es == 4 && pl->pp >= 3 && pl->pp <= kOneVectorMaxHealthy &&
                         buf_bytes >= kOneVectorMinBytes && buf_bytes < kOneVectorMaxBytes;
  if (mid_short && pl->pp >= 5) tile_elems = std::min(tile_elems, vec_tile);
  // Longer one-GPU-per-server chains take one vector per lane per tile too
  // (1024 elements for 32-bit types; 2-byte types have it already), so a
  // workgroup moves on to a new tile after every chain.  Measured against
  // 2048-element tiles (back-to-back calls, results bit for bit equal; the
  // tile count also decides per-XCD runs against work stealing below):
  // p64_f32 at 2^24 elements per rank 3.0 % faster, at 2^23 2.7 %, 2^22
  // equal; p128_f32 at 2^21 / 2^22 1.8 / 5.3 %, 2^23-2^25 0-0.6 %; one or
  // two stragglers with 33-256 ranks, fp32 and int32, 2^21-2^25: 0.5-14 %
  // faster in 27 of 30 plans, equal in one, 0.3 and 2.3 % slower in two
  // (48 ranks at 2^22; both faster again with the 4,096-tile runs limit
  // below).  Server plans were mixed (q32g4_f32 1.2 % slower, q16g4_f32
  // 0.4-3 % faster) and keep their tiles.
  if (long_chain && !servers) tile_elems = std::min(tile_elems, vec_tile);
  const int64_t ntiles = tile_count(*pl, tile_elems);
  if (noalloc && scratch_bytes(*pl, ntiles) > (size_t)OPTCC_NOALLOC_SCRATCH_BYTES)
    return fail(OPTCC_EUNSUPPORTED,
                "the plan's tables need " + std::to_string(scratch_bytes(*pl, ntiles)) +
                    " bytes, more than the " + std::to_string(OPTCC_NOALLOC_SCRATCH_BYTES) +
                    " of the no-allocation scratch array: use optcc_allreduce_emulate");
  const bool two = !long_chain && !single_hop && !mid_short;
  const bool two_vec = two && es == 4;  // two vectors per lane: 32-bit types only
  hipStream_t st = static_cast<hipStream_t>(stream);
  KArgs a;
  std::memset(&a, 0, sizeof(a));
  a.n = N;
  a.pp = pl->pp;
  a.m = pl->m;
  a.g = pl->g;
  if (servers) {  // per server (healthy in ring order, then the straggler): its g GPUs
    const int g = pl->g;
    for (int h = 0; h < pl->pp; ++h)
      for (int l = 0; l < g; ++l) a.ptr[h * g + l] = bufs[pl->ring[(size_t)h] * g + l];
    for (int l = 0; l < g; ++l) a.ptr[pl->pp * g + l] = bufs[pl->strag[0] * g + l];
  } else {
    for (int i = 0; i < pl->pp; ++i) a.ptr[i] = bufs[pl->ring[(size_t)i]];
    for (int i = 0; i < pl->m; ++i) a.ptr[pl->pp + i] = bufs[pl->strag[(size_t)i]];
  }
  a.occ_lds = long_chain ? workgroups_per_cu_lds(1) : 0;
  // 32-bit chains of 11-32 healthy ranks (one GPU per server, two vectors
  // per lane, 178 VGPRs: two workgroups per CU) with at most one straggler
  // and at least kTwoVecOnePerCuMinBytes of 16-byte-aligned rank buffers
  // run one workgroup per CU too.  Measured (back-to-back calls, results
  // bit for bit equal), from 1 GiB of buffers: one straggler, 12-16 ranks
  // 1.3-4.9 % faster, 20-33 ranks 2.0-3.2 %, with bubble filling 1.8 %,
  // int32 like fp32; rings of 12-32 ranks 2.3-6.5 %; 10 and 11 ranks 1-2 %
  // slower, p = 8 9 %.  Several stragglers split with the chain length
  // (13-14 healthy ranks 0.5-4.6 % slower, 18-29 from 1 % slower to 2.3 %
  // faster) and keep two per CU.  Below 1 GiB the effect swings both ways
  // (256 MiB at 32 ranks +7 %, 384 MiB at 12 ranks int32 -15 %, 64 MiB at
  // 16 ranks -14.5 %).  Server plans of at most 32 ranks (two vectors
  // per lane as well) take it with 4 or more GPUs per server: 4 x 4,
  // 5 x 4 (int32), 6 x 4 and 8 x 4 servers 2.7-4.0 % faster, 3 x 8 and
  // 4 x 8 0.3-0.4 %; with 2 GPUs per server it splits (16 x 2 +1.4 %,
  // 12 x 2 -0.7 %, 8 x 2 -3.4 %).
  const bool two_vec_one_per_cu =
      servers ? pl->g >= 4 : (pl->m <= 1 && pl->pp >= kTwoVecOnePerCuMinHealthy);
  if (two_vec && vec16 && two_vec_one_per_cu && buf_bytes >= kTwoVecOnePerCuMinBytes)
    a.occ_lds = workgroups_per_cu_lds(1);
  // The mid-size short chains of 6 or 7 healthy ranks with at least
  // kThreePerCuMinBytes of 16-byte-aligned rank buffers run at three
  // workgroups per CU instead of the four their registers allow: with fewer
  // lanes in flight more Stage-1 partial sums are still in L2 when Stage 4
  // overwrites them.  Measured (back-to-back calls, results bit for bit
  // equal): p = 8 with one straggler at 0.875, fp32, from 480 MiB to
  // 1.75 GiB of rank buffers 1.5-5 % faster (768 MiB equal), int32 1.7-2.9 %,
  // the straggler at 0.5 or 0.25 2.2-4.8 %, p = 9 with two stragglers
  // 1.4-2.2 %, p = 7 0-2.7 %; p = 8 at 384 and 448 MiB 2 and 1.3 % slower;
  // chains of 3-5 healthy ranks gain or lose up to 3 % with the size, and
  // element-aligned buffers lose 30-50 %, so neither takes it.
  if (mid_short && vec16 && pl->pp >= kThreePerCuMinHealthy && buf_bytes >= kThreePerCuMinBytes)
    a.occ_lds = workgroups_per_cu_lds(3);
  // bf16 chains of kBf16ThreePerCuMinHealthy to kTwoVectorMaxHealthy
  // healthy ranks (one GPU per server, 16-byte path) run at three
  // workgroups per CU as well.  Measured (same method): p16_bf16 at 2^20 /
  // 2^22 / 2^24 / 2^26 elements per rank 1.6 / 1.7 / 0.7 / 1.1 % faster,
  // p = 24 at 2^22 and 2^24 3.7 and 1.4 %, p = 33 1.4 %, p = 18 with two
  // stragglers 1.0 %; p = 20 at 2^20 1.4 % slower; shorter chains equal or
  // slower (p = 12 0 %, p = 10 up to 4 %, p = 9 0.7 %).
  if (!servers && dtype == OPTCC_BF16 && vec16 && pl->pp >= kBf16ThreePerCuMinHealthy &&
      pl->pp <= kTwoVectorMaxHealthy)
    a.occ_lds = workgroups_per_cu_lds(3);
  // The same mid-size short chains take each vector's Stage 4 stores into
  // the next vector's Stage 1 chain (the kernel's pipelined ring tiles).
  // Measured against one vector at a time (back-to-back calls, every result
  // bit for bit equal): p = 8 fp32 at 2^20 / 2^21 / 2^22 elements per rank
  // 3 / 1.2 / 1.5 % faster, int32 at 2^22 1.7 %, 2^24 equal; long chains
  // lose 1-8 % (p = 64, 128), so they keep one vector at a time.
  a.pipe = mid_short ? 1 : 0;
  // Long 32-bit chains (one GPU per server) with at least
  // kHopWindowWideMinElems elements per rank keep kHopWindowWide hop loads
  // in flight per vector instead of kHopWindow.  Measured against the
  // narrower window (back-to-back calls, results bit for bit equal):
  // p64_f32 at 2^23 and 2^24 elements per rank 1.4 % faster, 36-48 ranks
  // 1.4-1.6 %, 96 ranks with one straggler at 2^23 1.5 %, int32 0.6-0.7 %,
  // p128_f32 at 2^24 and 2^25 0.5-0.6 %; below 2^23 it was slower (p64 at
  // 2^22 0.9 %, p128 at 2^21 1.5 %), and bf16 long chains 8 % slower.
  a.wide_window = long_chain && !servers && es == 4 && vec16 && N >= kHopWindowWideMinElems ? 1 : 0;
  bool runs = servers || two;
  // With one-vector tiles, chains of fewer than kXcdRunsWideHealthy healthy
  // ranks keep the per-XCD runs up to kXcdRunsMaxTilesMid tiles.  Measured
  // at 4096 tiles against work stealing (back-to-back calls, results bit
  // for bit equal): p64_f32 at 2^22 elements per rank 2.7 % faster, 48
  // ranks 1.5 %, 48 ranks int32 with two stragglers 3.8 %, 80 ranks int32
  // 0.5 %, 64 ranks bf16 (no stealing: against the identity order) 0.3 %;
  // 96 and 128 ranks 2.4 and 3.5 % slower (bf16: 5 %); at 8192 tiles runs
  // were slower for every chain (36 ranks 1.5 %, p64 2.3 %, 48 ranks
  // 3.6 %, p128 11 %, bf16 2.4-4 %).
  const int64_t runs_max = pl->pp < kXcdRunsWideHealthy ? kXcdRunsMaxTilesMid : kXcdRunsMaxTiles;
  if (long_chain && !servers && ntiles <= runs_max) {
    const int resident = resident_workgroups(a, dtype, servers, vec16, two_vec);
    runs = resident <= 0 || ntiles > resident;
  }
  // Server plans of at least kXcdRunsWideHealthy ranks (one workgroup per
  // CU) with more than kServerStealMinTiles tiles (kXcdRunsMaxTiles from
  // kServerStealWideRanks ranks) take work stealing (below) instead of the
  // per-XCD runs, when it is available; otherwise the runs.  Measured
  // (back-to-back calls, results bit for bit equal) at 2^24 elements per
  // rank (8192 tiles): 32 x 4 fp32 0.8 %, int32 1.1 %, bf16 7.6 % faster,
  // 64 x 2 3.2 %, 16 x 8 4.2 %, 24 x 4 4.9 % (0.6 % slower on another
  // GPU); 32 x 4 fp32 at 2^25 0.4 % slower.  At 4096 tiles: 128 ranks and
  // more faster (32 x 4 fp32 3.7-4.3 %, bf16 2.6 %, 64 x 2 0.2 %, 30 x 4 3.2 %, 48 x 4
  // 4.6 %), 24 x 4 6.5 % slower; at 2048 tiles and below 5-10 % slower
  // (48 x 4 0.9 % faster); 64-rank server plans at 8192 tiles 2.7 % slower
  // (fp32, int32; bf16 2.5 % faster).
  const int64_t server_steal_min =
      pl->p >= kServerStealWideRanks ? kXcdRunsMaxTiles : kServerStealMinTiles;
  const bool server_steal = servers && long_chain && vec16 && pl->p >= kXcdRunsWideHealthy &&
                            ntiles > server_steal_min && !noalloc;
  if (server_steal) runs = false;
  a.xcd_runs = runs ? 1 : 0;
  // Work stealing for the same long chains at one workgroup per CU when
  // their tiles take the identity order (more than runs_max): a
  // grid of the resident workgroups takes tiles from a device counter.  The
  // eight XCDs do not run equally fast (per-wave timestamps of p128_f32:
  // XCDs 1, 3, 5, 7 spend about 5 % longer per tile than 0, 2, 4, 6), and
  // with one eighth of the tiles each the fast ones wait at the end.
  // Measured (back-to-back calls, results bit for bit equal): p = 128 fp32
  // at 2^23 / 2^24 / 2^25 elements per rank 2.1 / 4.2 / 3.6 % faster, p = 64
  // 3.4 / 2.2 / 2.5 %, int32 p = 128 at 2^24 2.6 %, one straggler at 0.875
  // with p = 96 (P2P chunks) 2.9 %, p = 40 and 48 1.5-3.2 %; bf16 long
  // chains at one workgroup per CU likewise (with the gain of that
  // occupancy, above).  Not under graph capture: a captured
  // launch keeps its counter block, and replays of the graph on two streams
  // at once would share it; the no-allocation entry point keeps the static
  // order too.
  bool steal = long_chain && (!servers || server_steal) && a.occ_lds > 0 && !runs && !noalloc;
  int steal_grid = 0;
  if (steal) {
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    steal = hipStreamIsCapturing(st, &cap) == hipSuccess && cap == hipStreamCaptureStatusNone;
  }
  if (steal) {
    steal_grid = resident_workgroups(a, dtype, servers, vec16, two_vec);
    steal = steal_grid > 0 && steal_grid < ntiles;
  }
  if (server_steal && !steal) a.xcd_runs = 1;  // captured: the server plans' runs
  DeviceTables dt;
  int rc = noalloc ? scratch_tables(*pl, tile_elems, st, &dt)
                   : device_tables(*pl, tile_elems, st, &dt);
  if (rc != OPTCC_OK) return rc;
  a.tiles = dt.tiles;
  a.segs = dt.segs;
  a.ntiles = dt.ntiles;
  uint32_t *counters = steal ? steal_counters(*pl, tile_elems) : nullptr;
  if (counters) {
    // one counter block per launch, round robin over kStealSlots: launches
    // in flight at once (any streams) use different blocks
    const uint32_t slot = pl->steal_next.fetch_add(1u, std::memory_order_relaxed) % kStealSlots;
    a.steal = counters + (size_t)slot * kStealWords;
    a.grid = steal_grid;
  }
  const int nl = launches == 1 ? 1 : se - sb;
  for (int l = 0; l < nl; ++l) {
    a.sb = launches == 1 ? sb : sb + l;
    a.se = launches == 1 ? se : sb + l + 1;
    hipError_t err = hipSuccess;
    switch (dtype) {
      case OPTCC_F32: err = launch_f32(a, servers, vec16, two_vec, st); break;
      case OPTCC_BF16: err = launch_bf16(a, servers, vec16, two_vec, st); break;
      case OPTCC_F16: err = launch_f16(a, servers, vec16, two_vec, st); break;
      default: err = launch_i32(a, servers, vec16, two_vec, st); break;
    }
    if (err != hipSuccess)
      return fail(OPTCC_EDEVICE, std::string("kernel launch: ") + hipGetErrorString(err));
  }
  return OPTCC_OK;
}

}  // namespace
}  // namespace optcc

using namespace optcc;

extern "C" int optcc_allreduce_emulate(void *const *bufs, int p, int64_t N, optcc_dtype_t dtype,
                                       const optcc_plan_t *plan, void *stream) {
  return emulate(bufs, p, N, dtype, plan, 0, plan ? plan->nslots : OPTCC_NUM_SLOTS, 1, stream);
}

extern "C" int optcc_allreduce_emulate_slots(void *const *bufs, int p, int64_t N,
                                             optcc_dtype_t dtype, const optcc_plan_t *plan,
                                             int slot_begin, int slot_end, int launches,
                                             void *stream) {
  return emulate(bufs, p, N, dtype, plan, slot_begin, slot_end, launches, stream);
}

extern "C" int optcc_allreduce_emulate_noalloc(void *const *bufs, int p, int64_t N,
                                               optcc_dtype_t dtype, const optcc_plan_t *plan,
                                               void *stream) {
  return emulate(bufs, p, N, dtype, plan, 0, plan ? plan->nslots : OPTCC_NUM_SLOTS, 1, stream,
                 true);
}

extern "C" void optcc_plan_free(optcc_plan_t *pl) {
  if (!pl) return;
  if (!pl->dev.empty()) {
    std::lock_guard<std::mutex> lk(pl->mu);
    int cur = -1;
    const bool have_dev = hipGetDevice(&cur) == hipSuccess;
    for (auto &kv : pl->dev) {
      if (have_dev) (void)hipSetDevice(kv.first.first);
      (void)hipFree(kv.second.segs);
      (void)hipFree(kv.second.tiles);
      (void)hipFree(kv.second.steal);
    }
    if (have_dev && !pl->dev.empty()) (void)hipSetDevice(cur);
    pl->dev.clear();
  }
  delete pl;
}
