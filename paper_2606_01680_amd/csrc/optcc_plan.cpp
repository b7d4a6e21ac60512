// Host side of the OptCC library: schedule planning, the closed-form model
// and lower bounds, plan introspection and traffic accounting.  No device
// calls are made here.
//
// Paper: "Don't Let a Few Network Failures Slow the Entire AllReduce".
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <exception>
#include <future>
#include <new>
#include <queue>
#include <set>
#include <string>
#include <unordered_map>

#include "optcc_internal.hpp"

namespace optcc {

static thread_local std::string g_last_error;

void set_error(const std::string &msg) { g_last_error = msg; }

int fail(int status, const std::string &msg) {
  set_error(msg);
  return status;
}

void section_range(const optcc_plan_t &pl, const Segment &s, int j, int64_t *b, int64_t *e) {
  int64_t qoff = (int64_t)j * s.qbase + std::min<int64_t>(j, s.nbig);
  int64_t qlen = s.qbase + (j < s.nbig ? 1 : 0);
  int64_t lo = s.ring_begin + qoff * kQuantum, hi = lo + qlen * kQuantum;
  *b = std::min(lo, pl.n);
  *e = std::min(hi, pl.n);
}

namespace {

// Sources folded into the chain start before Stage 1 (slot 0) and stragglers
// that receive the global sum after Stage 4 (slot 5), per section ordering.
// Ordering 2 (Sec. 4.1): every straggler.  Ordering 1 with m >= 2 (App. D,
// patterns A'/C'): all but the worst straggler, which finalises in Stages 2/3.
int n_side(const optcc_plan_t &pl, int ordering) {
  if (pl.m == 0) return 0;
  return ordering == 2 ? pl.m : pl.m - 1;
}
int side_first(int ordering) { return ordering == 2 ? 0 : 1; }

int ring_at(const optcc_plan_t &pl, int j, int t) {
  int pp = pl.pp;
  return pl.ring[(size_t)(((j + t) % pp + pp) % pp)];
}

// Several GPUs per server (App. E): rank of local ring position d (0 = the
// part's leader) on server sv.
int srank(const optcc_plan_t &pl, int sv, int part, int d) { return sv * pl.g + (part + d) % pl.g; }

// Steps of a several-GPUs-per-server plan in execution order: slot, segment,
// section, hop (App. E, NVLink phases N1-N4 around Stages S1-S4).  Type 1 =
// S1-S2-S3-S4 with the straggler folding along its local ring; type 2 =
// S3-S1-S4-S2 with plain collect and distribute on the straggler.
template <class Fn>
void for_each_server_step(const optcc_plan_t &pl, Fn &&fn) {
  const int pp = pl.pp, g = pl.g, sv = pl.strag[0];
  int src[1];
  for (int slot = 0; slot < OPTCC_NUM_SERVER_SLOTS; ++slot) {
    for (int gs = 0; gs < pl.nseg; ++gs) {
      const Segment &s = pl.seg[(size_t)gs];
      const int part = s.part;
      const bool t1 = s.ordering == 1;
      auto loc = [&](int server, int d) { return srank(pl, server, part, d); };
      for (int j = 0; j < pp; ++j) {
        int64_t b, e;
        section_range(pl, s, j, &b, &e);
        if (e <= b) continue;
        auto lead = [&](int t) { return loc(ring_at(pl, j, t), 0); };
        const int holder = lead(pp - 1);
        auto step = [&](int op, int dst, int from) {
          src[0] = from;
          fn(slot, gs, j, op, dst, src, 1, b, e - b);
        };
        switch (slot) {
          case 0:  // N3 collect onto the straggler's leader (type 2)
            if (!t1) for (int d = g - 2; d >= 0; --d) step(1, loc(sv, d), loc(sv, d + 1));
            break;
          case 1:  // N1 collect onto every healthy leader
            for (int h = 0; h < pp; ++h)
              for (int d = g - 2; d >= 0; --d)
                step(1, loc(pl.ring[(size_t)h], d), loc(pl.ring[(size_t)h], d + 1));
            break;
          case 2:  // S3 (type 2): straggler's sum into the chain start
            if (!t1) step(1, lead(0), loc(sv, 0));
            break;
          case 3:  // S1 chain over the healthy leaders
            for (int t = 1; t < pp; ++t) step(1, lead(t), lead(t - 1));
            break;
          case 4:  // S2 (type 1): straggler leader adds the holder's partial
            if (t1) step(1, loc(sv, 0), holder);
            break;
          case 5:  // N2 (type 1): fold forward along the straggler's ring
            if (t1) for (int d = 1; d < g; ++d) step(1, loc(sv, d), loc(sv, d - 1));
            break;
          case 6:  // N3 (type 1): global sum back to the leader
            if (t1) for (int d = g - 2; d >= 0; --d) step(0, loc(sv, d), loc(sv, d + 1));
            break;
          case 7:  // S3 (type 1): straggler leader -> holder
            if (t1) step(0, holder, loc(sv, 0));
            break;
          case 8:  // S4 allgather from the holder
            for (int t = 0; t + 1 < pp; ++t) step(0, lead(t), lead(t - 1));
            break;
          case 9:  // N4 distribute on every healthy server
            for (int h = 0; h < pp; ++h)
              for (int d = 1; d < g; ++d) step(0, loc(pl.ring[(size_t)h], d), loc(pl.ring[(size_t)h], d - 1));
            break;
          case 10:  // S2 (type 2): holder -> straggler leader
            if (!t1) step(0, loc(sv, 0), holder);
            break;
          case 11:  // N2 (type 2): distribute on the straggler server
            if (!t1) for (int d = 1; d < g; ++d) step(0, loc(sv, d), loc(sv, d - 1));
            break;
        }
      }
    }
  }
}

// Visit every step in execution order: slot, segment, section (then the
// point-to-point chunk), hop.  fn(slot, seg, sec, op, dst, srcs, nsrc, off, len).
template <class Fn>
void for_each_step(const optcc_plan_t &pl, Fn &&fn) {
  if (pl.kind == OPTCC_KIND_SERVERS) {
    for_each_server_step(pl, fn);
    return;
  }
  const int pp = pl.pp;
  std::vector<int> srcs((size_t)std::max(pl.p, 1));
  for (int slot = 0; slot < OPTCC_NUM_SLOTS; ++slot) {
    for (int g = 0; g < pl.k; ++g) {
      const Segment &s = pl.seg[(size_t)g];
      const int ord = s.ordering;
      for (int j = 0; j < pp; ++j) {
        int64_t b, e;
        section_range(pl, s, j, &b, &e);
        if (e <= b) continue;
        const int holder = ring_at(pl, j, pp - 1);
        switch (slot) {
          case 0: {
            int ns = n_side(pl, ord);
            if (ns == 0) break;
            for (int i = 0; i < ns; ++i) srcs[(size_t)i] = pl.strag[(size_t)(side_first(ord) + i)];
            fn(0, g, j, 1, ring_at(pl, j, 0), srcs.data(), ns, b, e - b);
            break;
          }
          case 1:
            for (int t = 1; t < pp; ++t) {
              srcs[0] = ring_at(pl, j, t - 1);
              fn(1, g, j, 1, ring_at(pl, j, t), srcs.data(), 1, b, e - b);
            }
            break;
          case 2:
            if (pl.m >= 1 && ord == 1) {
              srcs[0] = holder;
              fn(2, g, j, 1, pl.strag[0], srcs.data(), 1, b, e - b);
            }
            break;
          case 3:
            if (pl.m >= 1 && ord == 1) {
              srcs[0] = pl.strag[0];
              fn(3, g, j, 0, holder, srcs.data(), 1, b, e - b);
            }
            break;
          case 4:
            for (int t = 0; t + 1 < pp; ++t) {
              srcs[0] = ring_at(pl, j, t - 1);
              fn(4, g, j, 0, ring_at(pl, j, t), srcs.data(), 1, b, e - b);
            }
            break;
          case 5: {
            int ns = n_side(pl, ord);
            for (int i = 0; i < ns; ++i) {
              srcs[0] = holder;
              fn(5, g, j, 0, pl.strag[(size_t)(side_first(ord) + i)], srcs.data(), 1, b, e - b);
            }
            break;
          }
        }
      }
      // Bubble filling (Sec. 4.2, App. C): star allreduce through the straggler.
      if (s.p2p_end > s.p2p_begin) {
        const int64_t b = s.p2p_begin, len = s.p2p_end - s.p2p_begin;
        if (slot == 2) {
          for (int i = 0; i < pp; ++i) srcs[(size_t)i] = pl.ring[(size_t)i];
          fn(2, g, -1, 1, pl.strag[0], srcs.data(), pp, b, len);
        } else if (slot == 3) {
          for (int i = 0; i < pp; ++i) {
            srcs[0] = pl.strag[0];
            fn(3, g, -1, 0, pl.ring[(size_t)i], srcs.data(), 1, b, len);
          }
        }
      }
    }
  }
}

// Loads and stores per coordinate that the executor issues for one lane of
// a section of the given ordering (or of a P2P chunk) over [sb, se) in one
// launch.  Mirrors the executor's per-lane control flow.
void lane_traffic(const optcc_plan_t &pl, int ordering, bool p2p, int sb, int se,
                  int64_t *loads, int64_t *stores) {
  auto in = [&](int q) { return sb <= q && q < se; };
  int64_t ld = 0, st = 0;
  bool have = false;
  const int64_t pp = pl.pp;
  if (p2p) {
    if (in(2)) { ld += 1 + pp; st += 1; have = true; }
    if (in(3)) { if (!have) ld += 1; st += pp; }
  } else {
    const int ns = n_side(pl, ordering);
    if (in(0) && ns > 0) { ld += 1 + ns; st += 1; have = true; }
    if (in(1)) { if (!have) ld += 1; ld += pp - 1; st += pp - 1; have = true; }
    if (pl.m >= 1 && ordering == 1) {
      if (in(2)) { if (!have) ld += 1; ld += 1; st += 1; have = true; }
      if (in(3)) { if (!have) ld += 1; st += 1; have = true; }
    }
    if (in(4)) { if (!have) ld += 1; st += pp - 1; have = true; }
    if (in(5) && ns > 0) { if (!have) ld += 1; st += ns; }
  }
  *loads = ld;
  *stores = st;
}

// The same for one lane of a section of a several-GPUs-per-server plan
// (schedule type 1 or 2).  Mirrors the executor's server lane.
void server_lane_traffic(const optcc_plan_t &pl, int type, int sb, int se, int64_t *loads,
                         int64_t *stores) {
  auto in = [&](int q) { return sb <= q && q < se; };
  const bool t1 = type == 1;
  const int64_t pp = pl.pp, g = pl.g;
  const bool i0 = !t1 && in(0), i1 = in(1), i2 = !t1 && in(2), i3 = in(3);
  int64_t ld = 0, st = 0;
  if (i0) { ld += g; st += g - 1; }
  if (i1) {
    ld += pp * g;
    st += pp * (g - 1);
    if (i2) { if (!i0) ld += 1; st += 1; }
    if (i3) st += pp - 1;
  } else if (i2 || i3) {
    ld += 1;
    if (i2) { ld += 1; st += 1; }
    if (i3) { ld += pp - 1; st += pp - 1; }
  }
  bool have = i3;
  if (t1) {
    if (in(4)) { ld += have ? 1 : 2; st += 1; have = true; }
    if (in(5)) { if (!have) ld += 1; ld += g - 1; st += g - 1; have = true; }
    if (in(6)) { if (!have) ld += 1; st += g - 1; have = true; }
    if (in(7)) { if (!have) ld += 1; st += 1; have = true; }
  }
  if (in(8)) { if (!have) ld += 1; st += pp - 1; have = true; }
  if (in(9)) { if (!have) ld += pp; st += pp * (g - 1); }
  if (!t1) {
    if (in(10)) { if (!have) ld += 1; st += 1; have = true; }
    if (in(11)) { if (!have) ld += 1; st += g - 1; }
  }
  *loads = ld;
  *stores = st;
}

bool valid_bw(int p, const double *bw, std::string *why) {
  if (!bw) { *why = "link_bandwidths is NULL"; return false; }
  for (int i = 0; i < p; ++i)
    if (!(bw[i] > 0.0) || !std::isfinite(bw[i])) {
      *why = "link_bandwidths[" + std::to_string(i) + "] must be finite and > 0";
      return false;
    }
  return true;
}

// Slowdowns l_i = max(b)/b_i and the stragglers sorted by l descending.
void slowdowns(int p, const double *bw, std::vector<double> *ell, std::vector<int> *strag,
               std::vector<int> *ring) {
  double bmax = 0.0;
  for (int i = 0; i < p; ++i) bmax = std::max(bmax, bw[i]);
  ell->assign((size_t)p, 1.0);
  strag->clear();
  ring->clear();
  for (int i = 0; i < p; ++i) {
    (*ell)[(size_t)i] = bmax / bw[i];
    if (bw[i] < bmax) strag->push_back(i);
    else ring->push_back(i);
  }
  std::stable_sort(strag->begin(), strag->end(),
                   [&](int a, int b) { return (*ell)[(size_t)a] > (*ell)[(size_t)b]; });
}

}  // namespace
}  // namespace optcc

using namespace optcc;

extern "C" const char *optcc_last_error(void) { return g_last_error.c_str(); }

extern "C" int optcc_plan(int p, const double *bw, int64_t N, int k, optcc_plan_t **out) {
  set_error("");
  if (!out) return fail(OPTCC_EINVAL, "out is NULL");
  if (p < 3)
    return fail(OPTCC_EUNSUPPORTED, "p must be >= 3 (the method needs a straggler and two healthy ranks)");
  if (p > OPTCC_MAX_RANKS) return fail(OPTCC_EUNSUPPORTED, "p exceeds OPTCC_MAX_RANKS");
  if (N < 0 || N > ((int64_t)1 << 46)) return fail(OPTCC_EINVAL, "N must be in [0, 2^46]");
  if (k < 4 || k % 4 != 0 || k > (1 << 24))
    return fail(OPTCC_EINVAL, "n_chunks must be a positive multiple of 4 (at most 2^24)");
  std::string why;
  if (!valid_bw(p, bw, &why)) return fail(OPTCC_EINVAL, why);

  optcc_plan_t *pl = new (std::nothrow) optcc_plan_t();
  if (!pl) return fail(OPTCC_ENOMEM, "out of host memory");
  try {
    pl->p = p;
    pl->k = k;
    pl->n = N;
    pl->g = 1;
    pl->q = p;
    pl->nseg = k;
    pl->nslots = OPTCC_NUM_SLOTS;
    slowdowns(p, bw, &pl->ell, &pl->strag, &pl->ring);
    pl->m = (int)pl->strag.size();
    pl->pp = (int)pl->ring.size();
    if (pl->pp < 2) {
      delete pl;
      return fail(OPTCC_EUNSUPPORTED, "fewer than 2 healthy ranks: no ring to reduce-scatter on");
    }
    if (pl->m == 0) pl->kind = OPTCC_KIND_RING;
    else if (pl->m == 1)
      pl->kind = pl->ell[(size_t)pl->strag[0]] >= 2.0 ? OPTCC_KIND_SINGLE_GE2 : OPTCC_KIND_SINGLE_LT2;
    else pl->kind = OPTCC_KIND_MULTI;

    const int64_t nq = (N + kQuantum - 1) / kQuantum;
    pl->seg.resize((size_t)k);
    pl->segdesc.resize((size_t)k);
    int64_t steps = 0, flows = 0;
    for (int g = 0; g < k; ++g) {
      const int64_t q0 = (int64_t)((__int128)g * nq / k);
      const int64_t q1 = (int64_t)((__int128)(g + 1) * nq / k);
      const int64_t lq = q1 - q0;
      int64_t dq = 0;
      if (pl->kind == OPTCC_KIND_SINGLE_LT2) {
        // App. C: D / L = (2-l) / ((p-2) l + 2), rounded to whole quanta.
        const double l = pl->ell[(size_t)pl->strag[0]];
        const double x = ((double)lq * (2.0 - l)) / ((double)(p - 2) * l + 2.0);
        dq = (int64_t)std::floor(x + 0.5);
        dq = std::max<int64_t>(0, std::min(dq, lq));
      }
      const int64_t rq = lq - dq;
      Segment &s = pl->seg[(size_t)g];
      s.begin = std::min(q0 * kQuantum, N);
      s.end = std::min(q1 * kQuantum, N);
      s.ring_begin = q0 * kQuantum;
      s.ring_end = std::min((q1 - dq) * kQuantum, N);
      s.p2p_begin = std::min((q1 - dq) * kQuantum, N);
      s.p2p_end = s.end;
      s.qbase = rq / pl->pp;
      s.nbig = rq % pl->pp;
      // Patterns (Sec. 4.2; App. D): A,B,C,D or B,D,A',C' by g mod 4.
      const int pat = g % 4;
      s.ordering = pl->m <= 1 ? ((pat == 0 || pat == 2) ? 1 : 2) : (pat <= 1 ? 2 : 1);
      SegDesc &d = pl->segdesc[(size_t)g];
      d.ring_begin = s.ring_begin;
      d.p2p_begin = s.p2p_begin;
      d.qbase = (int32_t)s.qbase;
      d.nbig = (int32_t)s.nbig;
      d.ordering = s.ordering;
      d.part = 0;
      // step and flow counts per non-empty section / chunk
      const int ns = n_side(*pl, s.ordering);
      const int fin = (pl->m >= 1 && s.ordering == 1) ? 2 : 0;  // Stage 2 + Stage 3 steps
      // non-empty sections: all with a quantum, unless the segment is cut at N
      int64_t nonempty = s.qbase > 0 ? pl->pp : s.nbig;
      if (s.ring_begin + rq * kQuantum > N) {
        nonempty = 0;
        for (int j = 0; j < pl->pp; ++j) {
          int64_t b, e;
          section_range(*pl, s, j, &b, &e);
          nonempty += e > b;
        }
      }
      steps += nonempty * ((ns > 0 ? 1 : 0) + 2 * (pl->pp - 1) + fin + ns);
      flows += nonempty * (ns + 2 * (pl->pp - 1) + fin + ns);
      if (s.p2p_end > s.p2p_begin) {
        steps += 1 + pl->pp;
        flows += 2 * pl->pp;
      }
    }
    pl->num_steps = steps;
    pl->num_flows = flows;
  } catch (const std::bad_alloc &) {
    delete pl;
    return fail(OPTCC_ENOMEM, "out of host memory");
  }
  *out = pl;
  return OPTCC_OK;
}

extern "C" int optcc_plan_servers(int q, int g, const double *sbw, int64_t N, int k,
                                  optcc_plan_t **out) {
  set_error("");
  if (!out) return fail(OPTCC_EINVAL, "out is NULL");
  if (q < 3) return fail(OPTCC_EINVAL, "q must be >= 3 servers");
  if (g < 2 || g > OPTCC_MAX_GPUS_PER_SERVER)
    return fail(OPTCC_EINVAL, "g must be in [2, OPTCC_MAX_GPUS_PER_SERVER] (g = 1 is optcc_plan)");
  if ((int64_t)q * g > OPTCC_MAX_RANKS) return fail(OPTCC_EUNSUPPORTED, "q*g exceeds OPTCC_MAX_RANKS");
  if (N < 0 || N > ((int64_t)1 << 46)) return fail(OPTCC_EINVAL, "N must be in [0, 2^46]");
  if (k < 24 || k % 8 != 0 || k > (1 << 20))
    return fail(OPTCC_EINVAL, "n_chunks must be a multiple of 8 in [24, 2^20] (App. E)");
  std::string why;
  if (!valid_bw(q, sbw, &why)) return fail(OPTCC_EINVAL, why);
  optcc_plan_t *pl = new (std::nothrow) optcc_plan_t();
  if (!pl) return fail(OPTCC_ENOMEM, "out of host memory");
  try {
    const int p = q * g;
    pl->p = p;
    pl->g = g;
    pl->q = q;
    pl->k = k;
    pl->n = N;
    pl->nseg = g * k;
    pl->nslots = OPTCC_NUM_SERVER_SLOTS;
    pl->kind = OPTCC_KIND_SERVERS;
    std::vector<double> sell;
    slowdowns(q, sbw, &sell, &pl->strag, &pl->ring);
    pl->m = (int)pl->strag.size();
    pl->pp = (int)pl->ring.size();
    if (pl->m != 1) {
      delete pl;
      return fail(OPTCC_EUNSUPPORTED, "exactly one straggler server is supported (App. E)");
    }
    pl->ell.assign((size_t)p, 1.0);
    for (int r = 0; r < p; ++r) pl->ell[(size_t)r] = sell[(size_t)(r / g)];
    const int64_t nq = (N + kQuantum - 1) / kQuantum;
    pl->seg.resize((size_t)pl->nseg);
    pl->segdesc.resize((size_t)pl->nseg);
    int64_t steps = 0;
    for (int part = 0; part < g; ++part) {
      const int64_t p0 = (int64_t)((__int128)part * nq / g);
      const int64_t lp = (int64_t)((__int128)(part + 1) * nq / g) - p0;
      for (int c = 0; c < k; ++c) {
        const int gs = part * k + c;
        const int64_t q0 = p0 + (int64_t)((__int128)c * lp / k);
        const int64_t q1 = p0 + (int64_t)((__int128)(c + 1) * lp / k);
        Segment &s = pl->seg[(size_t)gs];
        s.begin = std::min(q0 * kQuantum, N);
        s.end = std::min(q1 * kQuantum, N);
        s.ring_begin = q0 * kQuantum;
        s.ring_end = s.end;
        s.p2p_begin = s.p2p_end = s.end;
        s.qbase = (q1 - q0) / pl->pp;
        s.nbig = (q1 - q0) % pl->pp;
        s.ordering = (c % 4 == 0 || c % 4 == 2) ? 1 : 2;  // A, C: type 1; B, D: type 2
        s.part = part;
        SegDesc &d = pl->segdesc[(size_t)gs];
        d.ring_begin = s.ring_begin;
        d.p2p_begin = s.p2p_begin;
        d.qbase = (int32_t)s.qbase;
        d.nbig = (int32_t)s.nbig;
        d.ordering = s.ordering;
        d.part = part;
        int64_t nonempty = 0;
        for (int j = 0; j < pl->pp; ++j) {
          int64_t b, e;
          section_range(*pl, s, j, &b, &e);
          nonempty += e > b;
        }
        steps += nonempty * 2 * (p - 1);  // every step has one source
      }
    }
    pl->num_steps = steps;
    pl->num_flows = steps;
  } catch (const std::bad_alloc &) {
    delete pl;
    return fail(OPTCC_ENOMEM, "out of host memory");
  }
  *out = pl;
  return OPTCC_OK;
}

extern "C" int optcc_plan_info(const optcc_plan_t *pl, optcc_plan_info_t *info, int32_t *ring,
                               int32_t *strag, double *ell) {
  if (!pl || !info) return fail(OPTCC_EINVAL, "plan and info must be non-NULL");
  info->p = pl->p;
  info->k = pl->k;
  info->m = pl->m;
  info->kind = pl->kind;
  info->healthy = pl->pp;
  info->quantum = kQuantum;
  info->n = pl->n;
  info->num_steps = pl->num_steps;
  info->num_flows = pl->num_flows;
  info->g = pl->g;
  info->q = pl->q;
  info->num_segments = pl->nseg;
  info->num_slots = pl->nslots;
  if (ring) for (int i = 0; i < pl->pp; ++i) ring[i] = pl->ring[(size_t)i];
  if (strag) for (int i = 0; i < pl->m; ++i) strag[i] = pl->strag[(size_t)i];
  if (ell) for (int i = 0; i < pl->p; ++i) ell[i] = pl->ell[(size_t)i];
  return OPTCC_OK;
}

extern "C" int optcc_plan_segments(const optcc_plan_t *pl, int64_t *off, int64_t *len,
                                   int64_t *p2p) {
  if (!pl || !off || !len || !p2p) return fail(OPTCC_EINVAL, "NULL argument");
  for (int g = 0; g < pl->nseg; ++g) {
    const Segment &s = pl->seg[(size_t)g];
    off[g] = s.begin;
    len[g] = s.end - s.begin;
    p2p[g] = s.p2p_end - s.p2p_begin;
  }
  return OPTCC_OK;
}

extern "C" int64_t optcc_plan_num_flows(const optcc_plan_t *pl) {
  if (!pl) return fail(OPTCC_EINVAL, "plan is NULL");
  return pl->num_flows;
}

// The paper's stage (OPTCC_STAGE_*) of each executor slot: Sec. 4.1 stages
// S1-S4 (bubble filling rides on S2 and S3, App. C) and App. E's NVLink
// phases N1-N4.
static const int kSlotStage[OPTCC_NUM_SLOTS] = {OPTCC_STAGE_S3, OPTCC_STAGE_S1, OPTCC_STAGE_S2,
                                                OPTCC_STAGE_S3, OPTCC_STAGE_S4, OPTCC_STAGE_S2};
static const int kServerSlotStage[OPTCC_NUM_SERVER_SLOTS] = {
    OPTCC_STAGE_N3, OPTCC_STAGE_N1, OPTCC_STAGE_S3, OPTCC_STAGE_S1, OPTCC_STAGE_S2, OPTCC_STAGE_N2,
    OPTCC_STAGE_N3, OPTCC_STAGE_S3, OPTCC_STAGE_S4, OPTCC_STAGE_N4, OPTCC_STAGE_S2, OPTCC_STAGE_N2};

extern "C" int64_t optcc_plan_get_flows(const optcc_plan_t *pl, optcc_flow_t *out, int64_t cap) {
  if (!pl) return fail(OPTCC_EINVAL, "plan is NULL");
  if (cap > 0 && !out) return fail(OPTCC_EINVAL, "out is NULL");
  const int *stage_of = pl->kind == OPTCC_KIND_SERVERS ? kServerSlotStage : kSlotStage;
  int64_t nf = 0, step = 0;
  int last_slot = -1, last_seg = -1, last_sec = -2, hop = 0;
  for_each_step(*pl, [&](int slot, int g, int sec, int op, int dst, const int *srcs, int ns,
                         int64_t off, int64_t len) {
    // steps arrive grouped by (slot, segment, section), hop by hop
    if (slot == last_slot && g == last_seg && sec == last_sec) {
      ++hop;
    } else {
      hop = 0;
      last_slot = slot;
      last_seg = g;
      last_sec = sec;
    }
    for (int i = 0; i < ns; ++i, ++nf) {
      if (nf >= cap) continue;
      optcc_flow_t &f = out[nf];
      f.slot = slot;
      f.segment = g;
      f.section = sec;
      f.op = op;
      f.src = srcs[i];
      f.dst = dst;
      f.stage = stage_of[slot];
      f.hop = hop;
      f.step = step;
      f.offset = off;
      f.length = len;
    }
    ++step;
  });
  return nf;
}

extern "C" void optcc_plan_free(optcc_plan_t *pl);  // defined with the executor

extern "C" double optcc_model_time(const optcc_plan_t *pl, const double *bw) {
  if (!pl) { set_error("plan is NULL"); return NAN; }
  std::vector<double> ell = pl->ell;
  if (bw) {
    // one bandwidth per rank, or per server for a several-GPUs-per-server plan
    const int nb = pl->kind == OPTCC_KIND_SERVERS ? pl->q : pl->p;
    std::string why;
    if (!valid_bw(nb, bw, &why)) { set_error(why); return NAN; }
    std::vector<int> strag, ring;
    std::vector<double> e1;
    slowdowns(nb, bw, &e1, &strag, &ring);
    for (int i = 0; i < pl->p; ++i) ell[(size_t)i] = e1[(size_t)(i / pl->g)];
    bool same = strag == pl->strag;
    for (int i = 0; same && i < pl->p; ++i)
      same = std::fabs(ell[(size_t)i] - pl->ell[(size_t)i]) <= 1e-12 * pl->ell[(size_t)i];
    if (!same) {
      set_error("bandwidths give other stragglers or slowdowns than the plan was built for");
      return NAN;
    }
  }
  const double p = pl->p, n = (double)pl->n, k = pl->k, m = pl->m;
  if (pl->kind == OPTCC_KIND_SERVERS) {
    // App. E time analysis: k + 5.5 bodies of max{l, 2} (q-1) s = max{l, 2} n/(g k)
    const double l = ell[(size_t)(pl->strag[0] * pl->g)];
    return std::max(l, 2.0) * n * (k + 5.5) / ((double)pl->g * k);
  }
  switch (pl->kind) {
    case OPTCC_KIND_RING:
      return 2.0 * (p - 1.0) * n / p;  // T0 (Sec. 3)
    case OPTCC_KIND_SINGLE_GE2: {
      const double l = ell[(size_t)pl->strag[0]];
      return l * n * (k + 1.0) / k;  // Sec. 4.3, l >= 2
    }
    case OPTCC_KIND_SINGLE_LT2: {
      const double l = ell[(size_t)pl->strag[0]];
      return 2.0 * (p - 1.0) * l * n / ((p - 2.0) * l + 2.0) * (k + l - 1.0) / k;  // App. C
    }
    default: {
      const double l1 = ell[(size_t)pl->strag[0]];
      const double s = n / (k * (p - m));
      const double body = std::max(2.0 * (p - 1.0) * s, (l1 * (p - m) + 2.0 * (m - 1.0)) * s);
      return (k + 4.0) * body;  // App. D
    }
  }
}

extern "C" double optcc_lower_bound(int p, const double *bw, int64_t N) {
  if (p < 3 || p > OPTCC_MAX_RANKS) { set_error("p must be in [3, OPTCC_MAX_RANKS]"); return NAN; }
  if (N < 0) { set_error("N must be >= 0"); return NAN; }
  std::string why;
  if (!valid_bw(p, bw, &why)) { set_error(why); return NAN; }
  std::vector<double> ell;
  std::vector<int> strag, ring;
  slowdowns(p, bw, &ell, &strag, &ring);
  const double n = (double)N, P = p;
  const size_t m = strag.size();
  if (m == 0) return 2.0 * (P - 1.0) * n / P;
  const double l1 = ell[(size_t)strag[0]];
  if (m == 1) return std::max(2.0 * l1 * (P - 1.0) / (l1 * (P - 2.0) + 2.0), l1) * n;
  double inv = 0.0;
  for (int r : strag) inv += 1.0 / ell[(size_t)r];
  return std::max(2.0 * (P - 1.0) / (P - (double)m + inv), l1) * n;
}

extern "C" double optcc_lower_bound_servers(int q, int g, const double *bw, int64_t N) {
  if (q < 3 || g < 1 || (int64_t)q * g > OPTCC_MAX_RANKS) {
    set_error("need q >= 3, g >= 1 and q*g <= OPTCC_MAX_RANKS");
    return NAN;
  }
  if (N < 0) { set_error("N must be >= 0"); return NAN; }
  std::string why;
  if (!valid_bw(q, bw, &why)) { set_error(why); return NAN; }
  std::vector<double> ell;
  std::vector<int> strag, ring;
  slowdowns(q, bw, &ell, &strag, &ring);
  const double n = (double)N, Q = q, G = g, P = Q * G;
  if (strag.empty()) return 2.0 * (P - 1.0) * n / (G * P);  // fault-free optimum (Sec. 3)
  if (strag.size() > 1) { set_error("more than one straggler server: no bound stated"); return NAN; }
  const double l = ell[(size_t)strag[0]];
  return n / G * std::max(2.0 * l * (Q - 1.0) / (l * (Q - 2.0) + 2.0), l);  // App. B.3
}

extern "C" int optcc_plan_traffic(const optcc_plan_t *pl, optcc_dtype_t dtype, int sb, int se,
                                  int launches, int64_t *rd, int64_t *wr) {
  if (!pl || !rd || !wr) return fail(OPTCC_EINVAL, "NULL argument");
  if (dtype != OPTCC_F32 && dtype != OPTCC_BF16 && dtype != OPTCC_I32 && dtype != OPTCC_F16)
    return fail(OPTCC_EINVAL, "unknown dtype");
  if (sb < 0 || se > pl->nslots || sb > se) return fail(OPTCC_EINVAL, "bad slot range");
  if (launches != 0 && launches != 1) return fail(OPTCC_EINVAL, "launches must be 0 or 1");
  const int64_t es = dtype == OPTCC_BF16 || dtype == OPTCC_F16 ? 2 : 4;
  int64_t r = 0, w = 0;
  auto lane = [&](int ord, bool p2p, int b, int e, int64_t *l, int64_t *s) {
    if (pl->kind == OPTCC_KIND_SERVERS) server_lane_traffic(*pl, ord, b, e, l, s);
    else lane_traffic(*pl, ord, p2p, b, e, l, s);
  };
  auto add = [&](int ord, bool p2p, int64_t len) {
    if (launches == 1) {
      int64_t l, s;
      lane(ord, p2p, sb, se, &l, &s);
      r += l * len;
      w += s * len;
    } else {
      for (int q = sb; q < se; ++q) {
        int64_t l, s;
        lane(ord, p2p, q, q + 1, &l, &s);
        r += l * len;
        w += s * len;
      }
    }
  };
  for (const Segment &s : pl->seg) {
    add(s.ordering, false, s.ring_end > s.ring_begin ? s.ring_end - std::min(s.ring_begin, s.ring_end) : 0);
    add(s.ordering, true, s.p2p_end - s.p2p_begin);
  }
  *rd = r * es;
  *wr = w * es;
  return OPTCC_OK;
}

// ------------------------------------------------------------- timeline
// Evaluation of the plan's flows in the paper's network model (Sec. 3 model;
// Sec. 4.1 flow rule; App. B.1 time weighting).  Plans with one GPU per
// server are timed by the paper's own pattern overlay (overlay_timeline,
// below); plans with several GPUs per server, whose eight-row overlay App. E
// gives only as figures, by list scheduling (list_timeline):
//  * every rank has a send port and a receive port (full duplex), each
//    carrying at most one flow at a time;
//  * a flow of len elements between ranks a and b lasts len * max(l_a, l_b);
//  * a flow starts only after every earlier step of its section that wrote
//    its source's range, or its destination's range, has finished (a rank
//    sends only data it holds); a step finishes with its last flow;
//  * list scheduling: whenever ports free up, ready flows are started in
//    priority order if both their ports are free.  Two priority orders are
//    evaluated and the second schedule is kept only if it is shorter by more
//    than a relative 1e-9:
//      1. flow order (slot, segment, section, hop);
//      2. pattern groups: the segments taken in groups, group by group,
//         each group in flow order.  A group is four consecutive segments,
//         one of each pattern (the k/4 groups of the time analyses of
//         Sec. 4.3 and App. D); with several GPUs per server, eight
//         consecutive segments of every part (App. E: the overlay needs
//         8 | k), the parts' groups together.
// Several GPUs per server (App. E bandwidth model): a flow between two GPUs of
// one server runs over NVLink, on separate NVLink send/receive ports, at
// (g-1) times NIC speed (len/(g-1)); flows between servers use the NICs.
// Times are doubles; events closer than 1e-9 of the current time are merged.
namespace optcc {
namespace {

int list_timeline(const optcc_plan_t *pl, double *start, double *finish, int64_t cap,
                  double *makespan) {
  try {
    // steps and flows in execution order
    std::vector<int32_t> st_dst, f_src, f_dst;  // flows: send and receive port ids
    std::vector<int64_t> st_first, f_step;
    std::vector<double> f_dur;
    std::vector<std::vector<int64_t>> deps;
    std::unordered_map<uint64_t, int64_t> last_writer;  // (rank, seg, sec) -> step
    auto key = [](int rank, int seg, int sec) {
      return ((uint64_t)(uint32_t)rank << 40) | ((uint64_t)(uint32_t)seg << 12) | (uint64_t)(sec + 1);
    };
    std::vector<int32_t> f_group;  // pattern group of the flow's segment
    for_each_step(*pl, [&](int, int g, int sec, int, int dst, const int *srcs, int ns,
                           int64_t, int64_t len) {
      const int64_t sid = (int64_t)st_dst.size();
      st_dst.push_back(dst);
      st_first.push_back((int64_t)f_src.size());
      std::vector<int64_t> d;
      auto dep = [&](int rank) {
        auto it = last_writer.find(key(rank, g, sec));
        if (it != last_writer.end() && std::find(d.begin(), d.end(), it->second) == d.end())
          d.push_back(it->second);
      };
      for (int i = 0; i < ns; ++i) dep(srcs[i]);
      dep(dst);
      deps.push_back(std::move(d));
      for (int i = 0; i < ns; ++i) {
        // port 2r: rank r's NIC; port 2r+1: its NVLink lane (same server only)
        const bool nvl = pl->g > 1 && srcs[i] / pl->g == dst / pl->g;
        f_src.push_back(2 * srcs[i] + (nvl ? 1 : 0));
        f_dst.push_back(2 * dst + (nvl ? 1 : 0));
        f_step.push_back(sid);
        f_group.push_back(pl->g > 1 ? (g % pl->k) / 8 : g / 4);
        f_dur.push_back(nvl ? (double)len / (double)(pl->g - 1)
                            : (double)len * std::max(pl->ell[(size_t)srcs[i]], pl->ell[(size_t)dst]));
      }
      last_writer[key(dst, g, sec)] = sid;
    });
    st_first.push_back((int64_t)f_src.size());
    const int64_t nst = (int64_t)st_dst.size(), nfl = (int64_t)f_src.size();
    std::vector<std::vector<int64_t>> dependents((size_t)nst);
    for (int64_t s = 0; s < nst; ++s)
      for (int64_t d : deps[(size_t)s]) dependents[(size_t)d].push_back(s);
    const int p = 2 * pl->p;  // ports
    // One list schedule: rk[f] = position of flow f in the priority order.
    // Returns the makespan; fs/ff receive every flow's start and finish.
    auto simulate = [&](const std::vector<int64_t> &rk, std::vector<double> &fs,
                        std::vector<double> &ff) -> double {
      std::vector<int64_t> order((size_t)nfl);
      for (int64_t f = 0; f < nfl; ++f) order[(size_t)rk[(size_t)f]] = f;
      std::vector<int32_t> pending((size_t)nst), left((size_t)nst);
      for (int64_t s = 0; s < nst; ++s) {
        pending[(size_t)s] = (int32_t)deps[(size_t)s].size();
        left[(size_t)s] = (int32_t)(st_first[(size_t)s + 1] - st_first[(size_t)s]);
      }
      fs.assign((size_t)nfl, -1.0);
      ff.assign((size_t)nfl, -1.0);
      std::vector<char> send_busy((size_t)p, 0), recv_busy((size_t)p, 0);
      // Ready flows by (sender, receiver), held as priority positions.  Flows
      // of one pair share both ports, so only the first of them in priority
      // order can be the next to start.  cand holds priority positions too.
      std::vector<std::unordered_map<int, std::set<int64_t>>> out_ready((size_t)p);
      std::vector<std::set<int>> in_partners((size_t)p);
      using Ev = std::pair<double, int64_t>;
      std::priority_queue<Ev, std::vector<Ev>, std::greater<Ev>> ev;
      std::vector<int64_t> cand;
      std::vector<int> freed_send, freed_recv;
      auto make_ready = [&](int64_t s) {
        for (int64_t f = st_first[(size_t)s]; f < st_first[(size_t)s + 1]; ++f) {
          const int a = f_src[(size_t)f], b = f_dst[(size_t)f];
          out_ready[(size_t)a][b].insert(rk[(size_t)f]);
          in_partners[(size_t)b].insert(a);
          cand.push_back(rk[(size_t)f]);
        }
      };
      for (int64_t s = 0; s < nst; ++s)
        if (pending[(size_t)s] == 0) make_ready(s);
      double t = 0.0, last = 0.0;
      int64_t done = 0;
      while (done < nfl) {
        // candidates: newly ready flows and the head of every ready pair that
        // touches a port freed at t; start them in priority order
        for (int a : freed_send)
          for (auto &kv : out_ready[(size_t)a])
            if (!recv_busy[(size_t)kv.first]) cand.push_back(*kv.second.begin());
        for (int b : freed_recv)
          for (int a : in_partners[(size_t)b])
            if (!send_busy[(size_t)a]) cand.push_back(*out_ready[(size_t)a][b].begin());
        freed_send.clear();
        freed_recv.clear();
        std::sort(cand.begin(), cand.end());
        cand.erase(std::unique(cand.begin(), cand.end()), cand.end());
        for (int64_t r : cand) {
          const int64_t f = order[(size_t)r];
          if (fs[(size_t)f] >= 0.0) continue;
          const int a = f_src[(size_t)f], b = f_dst[(size_t)f];
          if (send_busy[(size_t)a] || recv_busy[(size_t)b]) continue;
          auto &q = out_ready[(size_t)a][b];
          if (q.empty() || *q.begin() != r) continue;  // an earlier flow of the pair is waiting
          fs[(size_t)f] = t;
          ff[(size_t)f] = t + f_dur[(size_t)f];
          send_busy[(size_t)a] = 1;
          recv_busy[(size_t)b] = 1;
          q.erase(q.begin());
          if (q.empty()) {
            out_ready[(size_t)a].erase(b);
            in_partners[(size_t)b].erase(a);
          }
          ev.push({ff[(size_t)f], f});
        }
        cand.clear();
        if (ev.empty()) return -1.0;  // no flow can start: a dependency cycle
        t = ev.top().first;
        const double tol = 1e-9 * std::max(1.0, t);
        while (!ev.empty() && ev.top().first <= t + tol) {
          const int64_t f = ev.top().second;
          ev.pop();
          ++done;
          last = std::max(last, ff[(size_t)f]);
          const int a = f_src[(size_t)f], b = f_dst[(size_t)f];
          send_busy[(size_t)a] = 0;
          recv_busy[(size_t)b] = 0;
          freed_send.push_back(a);
          freed_recv.push_back(b);
          const int64_t s = f_step[(size_t)f];
          if (--left[(size_t)s] == 0)
            for (int64_t d : dependents[(size_t)s])
              if (--pending[(size_t)d] == 0) make_ready(d);
        }
      }
      return last;
    };
    // 1. flow order; 2. pattern groups (a stable counting sort of the flows
    // by group).  The two schedules share only read-only inputs, so the
    // second runs on a thread of its own.
    std::vector<int64_t> rk((size_t)nfl), rk2;
    for (int64_t f = 0; f < nfl; ++f) rk[(size_t)f] = f;
    const int ng = 1 + (nfl ? *std::max_element(f_group.begin(), f_group.end()) : 0);
    if (ng > 1) {
      std::vector<int64_t> pos((size_t)ng + 1, 0);
      for (int64_t f = 0; f < nfl; ++f) ++pos[(size_t)f_group[(size_t)f] + 1];
      for (int i = 0; i < ng; ++i) pos[(size_t)i + 1] += pos[(size_t)i];
      rk2.resize((size_t)nfl);
      for (int64_t f = 0; f < nfl; ++f) rk2[(size_t)f] = pos[(size_t)f_group[(size_t)f]]++;
    }
    std::vector<double> fs, ff, fs2, ff2;
    std::future<double> second;
    if (ng > 1) second = std::async(std::launch::async, [&] { return simulate(rk2, fs2, ff2); });
    double best = simulate(rk, fs, ff);
    const double mk2 = ng > 1 ? second.get() : -1.0;  // rethrows the thread's exception
    if (best < 0.0) return fail(OPTCC_EINVAL, "timeline: no flow can start (dependency cycle)");
    if (ng > 1) {
      if (mk2 >= 0.0 && mk2 < best * (1.0 - 1e-9)) {
        best = mk2;
        fs.swap(fs2);
        ff.swap(ff2);
      }
    }
    for (int64_t f = 0; f < std::min(cap, nfl); ++f) {
      start[f] = fs[(size_t)f];
      finish[f] = ff[(size_t)f];
    }
    *makespan = best;
  } catch (const std::bad_alloc &) {
    return fail(OPTCC_ENOMEM, "out of host memory");
  } catch (const std::exception &e) {  // e.g. no thread for the second schedule
    return fail(OPTCC_ENOMEM, std::string("timeline: ") + e.what());
  }
  return OPTCC_OK;
}

// The paper's pattern overlay (Sec. 4.2 for one straggler, App. D for
// several, Sec. 4.3 and App. C for the timing) as an explicit timetable;
// the flow grids of the paper are figures, so the layout below is rebuilt
// from the text:
//  * a parallel body has W = P' + m - 1 windows (App. D: p - 1 windows per
//    body, p - m - 1 of them with ring flows and m with straggler traffic,
//    per rank).  Straggler s_i (i = 1 the worst) takes windows i-1 ..
//    i-1+P'-1: in window w it receives from healthy rank R[w-i+1] and sends
//    to the next one, R[w-i+2], so the ring edges R[e] -> R[e+1] with
//    w-m+1 <= e <= w carry nothing in window w;
//  * ring stages: each body holds Stage 1 or Stage 4 of two segments, one per
//    sub-slot, earlier segment first; the h-th window in which an edge
//    carries ring flows carries hop h of the chain that crosses it at hop h;
//  * stage bodies per pattern (segment g = pattern g mod 4 of group g div 4,
//    offsets from body 4 (g div 4)): one straggler A = S1 S2 S3 S4 at
//    0..3, B = S3 S1 S4 S2 at 0..3, C and D the same one body later (k + 1
//    bodies, Sec. 4.3); several stragglers B = S3 S1 S4 S2 at 0..3, D at
//    2..5, A' with S1 at 1, C' with S1 at 3 (S2, S3, S4 in the next bodies),
//    the non-finalising stragglers' raw values two bodies before Stage 1 and
//    the global sum to them in the Stage 4 body (k + 4 bodies, App. D);
//  * bubble filling (App. C): segment g's point-to-point chunk goes up in
//    body g after the Stage 2 flow of the same sender and window, and down
//    in body g + 1 after the Stage 3 flow;
//  * windows run one after another; a window lasts as long as its longest
//    lane (an edge's two sub-slots, or a straggler's receive or send flows
//    back to back).
// Without straggler the ring takes its segments one after another, Stage 1
// then Stage 4, one hop per window (T0 exactly).  The timeline returned runs
// that timetable without its window boundaries: every port takes its flows
// in the timetable's order (window, lane, position), each as soon as both its
// ports are free and the steps it depends on are done, which is never later
// than the windowed timetable (with equal sections the two agree on the
// closed forms of Sec. 4.3 and App. C; the section sizes' rounding to whole
// quanta makes windows wait for their longest lane).
int overlay_timeline(const optcc_plan_t &pl, double *start, double *finish, int64_t cap,
                     double *makespan) {
  constexpr int X = INT32_MIN;  // the pattern has no such slot
  static const int kOne[4][OPTCC_NUM_SLOTS] = {
      {X, 0, 1, 2, 3, X}, {0, 1, X, X, 2, 3}, {X, 1, 2, 3, 4, X}, {1, 2, X, X, 3, 4}};
  static const int kMulti[4][OPTCC_NUM_SLOTS] = {
      {0, 1, X, X, 2, 3}, {2, 3, X, X, 4, 5}, {-1, 1, 2, 3, 4, 4}, {1, 3, 4, 5, 6, 6}};
  try {
    const int pp = pl.pp, m = pl.m;
    const int64_t W = m > 0 ? pp + m - 1 : pp - 1;
    std::vector<int> ring_pos((size_t)pl.p, -1), strag_no((size_t)pl.p, 0);
    for (int i = 0; i < pp; ++i) ring_pos[(size_t)pl.ring[(size_t)i]] = i;
    for (int i = 0; i < m; ++i) strag_no[(size_t)pl.strag[(size_t)i]] = i + 1;
    const auto &tab = m == 1 ? kOne : kMulti;
    struct Place {
      int64_t cell;   // body * W + window (bodies shifted to start at 0)
      int32_t lane;   // ring edge e, or pp + 2(i-1) (+1 for sends) for straggler i
      int32_t order;  // within the lane: the segment (ring) or 0/1 (straggler)
      int64_t flow;
      double dur;
    };
    std::vector<Place> pl_of;
    pl_of.reserve((size_t)pl.num_flows);
    // per flow: sender, receiver, step; per step: the steps it depends on
    // (earlier steps of its section that last wrote its sources or its
    // destination)
    std::vector<int32_t> f_src, f_dst;
    std::vector<int64_t> f_step, dep_first(1, 0), dep_list;
    f_src.reserve((size_t)pl.num_flows);
    f_dst.reserve((size_t)pl.num_flows);
    f_step.reserve((size_t)pl.num_flows);
    std::unordered_map<uint64_t, int64_t> last_writer;  // (rank, seg, sec) -> step
    auto wkey = [](int rank, int seg, int sec) {
      return ((uint64_t)(uint32_t)rank << 40) | ((uint64_t)(uint32_t)seg << 12) | (uint64_t)(sec + 1);
    };
    int64_t nf = 0, nsteps = 0;
    int last_slot = -1, last_seg = -1, last_sec = -2, hop = 0;
    const int64_t shift = m >= 2 ? 1 : 0;  // the head body of A' is body -1
    for_each_step(pl, [&](int slot, int g, int sec, int, int dst, const int *srcs, int ns,
                          int64_t, int64_t len) {
      if (slot == last_slot && g == last_seg && sec == last_sec) {
        ++hop;
      } else {
        hop = 0;
        last_slot = slot;
        last_seg = g;
        last_sec = sec;
      }
      const int64_t sid = nsteps++;
      const size_t d0 = dep_list.size();
      auto dep = [&](int rank) {
        auto it = last_writer.find(wkey(rank, g, sec));
        if (it != last_writer.end() &&
            std::find(dep_list.begin() + (ptrdiff_t)d0, dep_list.end(), it->second) == dep_list.end())
          dep_list.push_back(it->second);
      };
      for (int i = 0; i < ns; ++i) dep(srcs[i]);
      dep(dst);
      dep_first.push_back((int64_t)dep_list.size());
      last_writer[wkey(dst, g, sec)] = sid;
      for (int i = 0; i < ns; ++i, ++nf) {
        const int src = srcs[i];
        f_src.push_back(src);
        f_dst.push_back(dst);
        f_step.push_back(sid);
        Place q;
        q.flow = nf;
        q.dur = (double)len * std::max(pl.ell[(size_t)src], pl.ell[(size_t)dst]);
        int64_t body, window;
        if (m == 0) {  // the ring: segment by segment, Stage 1 then Stage 4
          body = 2 * (int64_t)g + (slot == 1 ? 0 : 1);
          window = hop;
          q.lane = ring_pos[(size_t)src];
          q.order = 0;
        } else if (sec < 0) {  // bubble filling
          if (slot == 2) {
            body = g;
            window = ring_pos[(size_t)src];
            q.lane = pp;
          } else {
            body = (int64_t)g + 1;
            window = (ring_pos[(size_t)dst] + pp - 1) % pp;
            q.lane = pp + 1;
          }
          q.order = 1;
        } else if (slot == 1 || slot == 4) {  // ring stages
          const int e = ring_pos[(size_t)src];
          body = 4 * (int64_t)(g / 4) + tab[g % 4][slot];
          window = hop < e ? hop : hop + m;
          q.lane = e;
          q.order = g;
        } else {  // straggler traffic
          body = 4 * (int64_t)(g / 4) + tab[g % 4][slot];
          if (strag_no[(size_t)dst] > 0) {  // received by s_i from R[a]
            const int si = strag_no[(size_t)dst], a = ring_pos[(size_t)src];
            window = a + si - 1;
            q.lane = pp + 2 * (si - 1);
          } else {  // sent by s_i to R[b]
            const int si = strag_no[(size_t)src], b = ring_pos[(size_t)dst];
            window = (b + pp - 1) % pp + si - 1;
            q.lane = pp + 2 * (si - 1) + 1;
          }
          q.order = 0;
        }
        q.cell = (body + shift) * W + window;
        pl_of.push_back(q);
      }
    });
    std::sort(pl_of.begin(), pl_of.end(), [](const Place &x, const Place &y) {
      if (x.cell != y.cell) return x.cell < y.cell;
      if (x.lane != y.lane) return x.lane < y.lane;
      return x.order < y.order;
    });
    // The timetable's order is a valid execution order (every port's flows
    // in sequence, every step after the steps it depends on): run it with
    // each flow starting as soon as it can.
    std::vector<double> fs((size_t)nf), ff((size_t)nf), send_free((size_t)pl.p, 0.0),
        recv_free((size_t)pl.p, 0.0), step_end((size_t)nsteps, 0.0);
    double t = 0.0;
    for (const Place &q : pl_of) {
      const int64_t f = q.flow, sid = f_step[(size_t)f];
      const int a = f_src[(size_t)f], b = f_dst[(size_t)f];
      double x = std::max(send_free[(size_t)a], recv_free[(size_t)b]);
      for (int64_t d = dep_first[(size_t)sid]; d < dep_first[(size_t)sid + 1]; ++d)
        x = std::max(x, step_end[(size_t)dep_list[(size_t)d]]);
      fs[(size_t)f] = x;
      ff[(size_t)f] = x + q.dur;
      send_free[(size_t)a] = recv_free[(size_t)b] = ff[(size_t)f];
      step_end[(size_t)sid] = std::max(step_end[(size_t)sid], ff[(size_t)f]);
      t = std::max(t, ff[(size_t)f]);
    }
    for (int64_t f = 0; f < std::min(cap, nf); ++f) {
      start[f] = fs[(size_t)f];
      finish[f] = ff[(size_t)f];
    }
    *makespan = t;
  } catch (const std::bad_alloc &) {
    return fail(OPTCC_ENOMEM, "out of host memory");
  }
  return OPTCC_OK;
}

}  // namespace
}  // namespace optcc

extern "C" int optcc_plan_timeline(const optcc_plan_t *pl, double *start, double *finish,
                                   int64_t cap, double *makespan) {
  if (!pl || !makespan) return fail(OPTCC_EINVAL, "plan and makespan must be non-NULL");
  if (cap > 0 && (!start || !finish)) return fail(OPTCC_EINVAL, "start/finish are NULL");
  if (pl->num_flows > ((int64_t)1 << 26))
    return fail(OPTCC_EUNSUPPORTED, "timeline limited to 2^26 flows");
  if (pl->kind == OPTCC_KIND_SERVERS) return list_timeline(pl, start, finish, cap, makespan);
  return overlay_timeline(*pl, start, finish, cap, makespan);
}
