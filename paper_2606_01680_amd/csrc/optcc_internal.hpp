// Internal definitions shared by the host planner and the GPU executor.
#pragma once

#include <atomic>
#include <cstdint>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "optcc.h"

namespace optcc {

// One segment as the executor sees it (device table, 32 bytes).
// Ring sections of the segment occupy [ring_begin, ring_begin + ring_len);
// section j has qbase + (j < nbig) quanta.  The point-to-point chunk, when
// present, follows the ring part up to the end of the segment.
struct SegDesc {
  int64_t ring_begin;
  int64_t p2p_begin;
  int32_t qbase;
  int32_t nbig;
  int32_t ordering;  // 1: S1-S2-S3-S4, 2: S3-S1-S4-S2 (Sec. 4.1; App. E types 1, 2)
  int32_t part;      // several GPUs per server: the part (leading local GPU), else 0
};
static_assert(sizeof(SegDesc) == 32, "SegDesc layout");

// One unit of work for a workgroup: `len` elements from `begin`, all in one
// segment's ring part (meta & 1 == 0) or its P2P chunk (meta & 1 == 1);
// meta >> 1 is the segment index.
struct TileDesc {
  int64_t begin;
  int32_t len;
  int32_t meta;
};
static_assert(sizeof(TileDesc) == 16, "TileDesc layout");

#ifndef OPTCC_TILE_QUANTA
#define OPTCC_TILE_QUANTA 32
#endif
constexpr int kQuantum = OPTCC_QUANTUM;
constexpr int kTileQuanta = OPTCC_TILE_QUANTA;  // 2048 elements per tile by default
constexpr int kTileElems = kQuantum * kTileQuanta;
// Plans that move little per element take longer tiles, up to this many
// elements, so that each workgroup moves at least kTileMinBytes4 (4-byte
// elements) or kTileMinBytes2 (2-byte elements) of algorithmic traffic.
constexpr int kTileElemsMax = 4 * kTileElems;
constexpr int64_t kTileMinBytes4 = 96 << 10;
constexpr int64_t kTileMinBytes2 = 72 << 10;
// Small messages take shorter tiles, down to one 16-byte vector per lane,
// while the launch would have fewer than this many tiles.
constexpr int64_t kTileMinCount = 1024;

// Counter blocks of work-stealing launches (kStealWords words each, one
// block per launch, taken round robin from kStealSlots per table).
constexpr int kStealSlots = 4096;
constexpr int kStealWords = 16;  // 64 bytes: blocks of concurrent launches share no cache line

struct DeviceTables {
  SegDesc *segs = nullptr;
  TileDesc *tiles = nullptr;
  uint32_t *steal = nullptr;  // kStealSlots blocks, zero between launches (on first use)
  int64_t ntiles = 0;
};

struct Segment {
  int64_t begin = 0, end = 0;          // element range of the segment
  int64_t ring_begin = 0, ring_end = 0; // ring sections
  int64_t p2p_begin = 0, p2p_end = 0;   // point-to-point chunk (may be empty)
  int64_t qbase = 0, nbig = 0;
  int ordering = 1;
  int part = 0;  // several GPUs per server: part index (App. E)
};

}  // namespace optcc

struct optcc_plan {
  int p = 0, k = 0, m = 0, kind = 0, pp = 0;
  int g = 1, q = 0;           // GPUs per server and servers (g = 1, q = p for optcc_plan)
  int nseg = 0, nslots = 0;   // segments in total (k or g*k) and stage slots
  int64_t n = 0;
  std::vector<double> ell;    // slowdown per rank
  std::vector<int> ring;      // healthy ranks (servers when g > 1), ascending
  std::vector<int> strag;     // stragglers (servers when g > 1), l descending, ties lower
  std::vector<optcc::Segment> seg;
  std::vector<optcc::SegDesc> segdesc;
  int64_t num_steps = 0, num_flows = 0;
  // device copies of segdesc/tiles, per (device ordinal, tile length)
  mutable std::mutex mu;
  mutable std::map<std::pair<int, int>, optcc::DeviceTables> dev;  // (device, tile elements)
  // host tile tables per tile length (the source of the device copies)
  mutable std::map<int, std::vector<optcc::TileDesc>> host_tiles;
  // next counter block for a work-stealing launch (round robin)
  mutable std::atomic<uint32_t> steal_next{0};
};

namespace optcc {
void set_error(const std::string &msg);
int fail(int status, const std::string &msg);
// Section j's element range inside segment s.
void section_range(const optcc_plan_t &pl, const Segment &s, int j, int64_t *b, int64_t *e);
}  // namespace optcc
