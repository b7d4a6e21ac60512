/*
 * OptCC oracle: plain serial CPU reference of the schedule-driven
 * reduce-and-forward data movement.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may include, link,
 * load or call this file.  It shares no code, header, table or constant with
 * the GPU library; both are written independently from the paper and from
 * the same readings of the points the paper leaves open (its pattern figures
 * are not available):
 *   - the healthy ring is the healthy ranks in ascending order; section j's
 *     chain starts at ring[j] and ends at its holder ring[j-1]; Stage 3
 *     returns the sum to the holder and Stage 4 starts there;
 *   - in ordering 2 the stragglers' raw values are added at the chain start
 *     before Stage 1, in straggler order;
 *   - bubble filling: per segment one point-to-point chunk after the
 *     sections; the straggler adds its own value first, then ring[0..P'-1];
 *   - m >= 2, patterns A'/C': the worst straggler finalises as in ordering 1,
 *     the others add their raw values at the chain start and receive the sum
 *     after Stage 4 (read literally the printed text is not an AllReduce);
 *   - one rounding per step; sizes in whole quanta of 64 elements.
 *
 * orc_run executes the steps serially; orc_run_parallel gives the same bits
 * on several host threads (OpenMP over segments, each segment's steps in
 * serial order), for timing the oracle on all host cores.
 *
 * Pins (tests outside this file): exact int32 sums against the definition of
 * the result; contributor sets (nobody counted twice, everybody counted);
 * the fp error bound of recursive summation; a chain's association order
 * against a sequential cumulative sum, for every plan kind; flow counts and
 * split sizes against the paper's worked examples; the lemmas' traffic
 * volumes.  The paper does not fix the order of the additions, so the exact
 * fp32/bf16 bit patterns follow from the readings above; given them, the
 * cumulative-sum pins fix every fp32 bit.
 *
 * Source of every rule below (paper: "Don't Let a Few Network Failures Slow
 * the Entire AllReduce"):
 *   - problem setting, slowdown factor l = 1/b, correctness = every rank ends
 *     with the elementwise sum .......................... Sec. 3 (problem setting)
 *   - k segments of p-1 sections of s = n/(k(p-1)) ........ Sec. 4.1
 *   - Stage 1 reduce-scatter chain on the healthy ring, Stage 2 upload,
 *     Stage 3 download, Stage 4 allgather ................. Sec. 4.1 (Stages 1-4)
 *   - the two valid stage orderings (1) S1-S2-S3-S4 and
 *     (2) S3-S1-S4-S2 ...................................... Sec. 4.1 (stage ordering)
 *   - patterns A/C (ordering 1), B/D (ordering 2), k/4
 *     segments per pattern ................................. Sec. 4.2 (four patterns, pipelining)
 *   - bubble filling for l < 2: per segment p-1 sections of s' and one
 *     point-to-point allreduce chunk of D = (2-l)s'/l, with
 *     s' = n l / (k((p-2)l+2)) ............................ Sec. 4.2 (bubble filling), App. C
 *   - m >= 2 stragglers: p-m sections of s = n/(k(p-m)),
 *     patterns B, D, A', C' ................................ App. D
 *
 * Step model.  One step writes one destination range of one rank:
 *   COPY   : dst <- src
 *   REDUCE : acc = widen(dst); acc = acc + widen(src_i) for each source in
 *            listed order; dst <- narrow(acc)
 * widen/narrow are the identity for fp32 and int32 (int32 adds wrap modulo
 * 2^32); for bf16, widen is the exact 16-bit shift to fp32 and narrow rounds
 * fp32 to bf16 to nearest, ties to even; for fp16 (IEEE 754 binary16) widen
 * is exact and narrow rounds to nearest, ties to even, with subnormals kept
 * and overflow to infinity.  Every step rounds once, so a chain of hops
 * rounds at every hop, as a 16-bit wire would.
 *
 * Steps carry a slot number 0..5 that orders the stages of every section:
 *   0 straggler raw values folded into the chain start (ordering 2's Stage 3,
 *     and the non-finalising stragglers of A'/C')
 *   1 Stage 1 chain            2 Stage 2 upload (ordering 1) / P2P up
 *   3 Stage 3 download (ordering 1) / P2P down
 *   4 Stage 4 allgather        5 G sent to the remaining stragglers
 *                                (ordering 2's Stage 2, A'/C' non-finalisers)
 * Running all steps of slot 0, then slot 1, ... is one valid serial order:
 * segments never share coordinates, and within a section the slot order is
 * the section's own stage order.
 *
 * Several GPUs per server (App. E): q servers of g GPUs, ranks numbered
 * server-major (rank = server * g + local index); one bandwidth per server
 * (PXN pools a server's NICs, Sec. 2).  The vector is split into g parts,
 * part i led by local GPU i of every server; each part runs the schedule
 * above among the leaders, with NVLink phases around the NIC stages:
 * collect = a reduce chain along the server's local ring backwards onto the
 * leader, distribute = a copy chain forwards from the leader.  Slots 0..11:
 *   0 N3 collect at the straggler (type 2)   1 N1 collect at healthy servers
 *   2 S3 straggler sum into the chain start (type 2)   3 S1 chain of leaders
 *   4 S2 holder -> straggler leader, which adds its own value (type 1)
 *   5 N2 fold: forward reduce chain on the straggler (type 1)
 *   6 N3 copy back: backward copy chain on the straggler (type 1)
 *   7 S3 straggler leader -> holder (type 1)   8 S4 allgather of leaders
 *   9 N4 distribute on healthy servers   10 S2 holder -> straggler (type 2)
 *   11 N2 distribute on the straggler (type 2)
 * Patterns A, C use type 1 (S1-S2-S3-S4), B, D type 2 (S3-S1-S4-S2).
 *
 * Build:  gcc -O2 -std=c99 -ffp-contract=off -fno-fast-math -shared -fPIC
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_F32 0
#define ORC_BF16 1
#define ORC_I32 2
#define ORC_F16 3

#define ORC_COPY 0
#define ORC_REDUCE 1

/* Plan kinds. */
#define ORC_RING 0       /* no straggler: textbook ring */
#define ORC_SINGLE_GE2 1 /* one straggler, l >= 2 */
#define ORC_SINGLE_LT2 2 /* one straggler, 1 < l < 2: bubble filling */
#define ORC_MULTI 3      /* m >= 2 stragglers */
#define ORC_SERVERS 4    /* g >= 2 GPUs per server, one straggler server */
#define ORC_MAX_SLOTS 12

/* Split quantum in elements: every section and P2P chunk is a whole number
 * of quanta (the last quantum of the vector may be partial). */
#define ORC_QUANTUM 64

typedef struct {
  int32_t slot, seg, sec, op, dst, nsrc;
  int64_t src_at; /* index into the source pool */
  int64_t off, len;
} orc_step;

typedef struct {
  int p, k, m, kind, pp; /* pp = P' = number of healthy ranks (servers when g > 1) */
  int g, q, nseg;        /* GPUs per server, servers, segments in total */
  int64_t n;
  double ell[1024];      /* l_i = max_b / b_i */
  int ring[1024];        /* healthy ranks, ascending */
  int strag[1024];       /* stragglers sorted by l descending, ties lower rank */
  int seg_lo, seg_hi;    /* segments whose steps were built */
  /* per-segment split (all k segments) */
  int64_t *seg_off, *seg_len, *p2p_len;
  int64_t nsteps, cap_steps, nsrcpool, cap_srcpool;
  orc_step *steps;
  int32_t *srcpool;
} orc_sched;

static const char *g_err = "";
const char *orc_last_error(void) { return g_err; }

/* ---------------------------------------------------------------- steps */

static int push_step(orc_sched *s, int slot, int seg, int sec, int op, int dst,
                     const int *srcs, int nsrc, int64_t off, int64_t len) {
  if (len <= 0) return 0; /* an empty section moves nothing */
  if (s->nsteps == s->cap_steps) {
    int64_t nc = s->cap_steps ? 2 * s->cap_steps : 1024;
    orc_step *ns = (orc_step *)realloc(s->steps, (size_t)nc * sizeof(orc_step));
    if (!ns) return -2;
    s->steps = ns;
    s->cap_steps = nc;
  }
  while (s->nsrcpool + nsrc > s->cap_srcpool) {
    int64_t nc = s->cap_srcpool ? 2 * s->cap_srcpool : 4096;
    int32_t *np = (int32_t *)realloc(s->srcpool, (size_t)nc * sizeof(int32_t));
    if (!np) return -2;
    s->srcpool = np;
    s->cap_srcpool = nc;
  }
  orc_step *st = &s->steps[s->nsteps++];
  st->slot = slot;
  st->seg = seg;
  st->sec = sec;
  st->op = op;
  st->dst = dst;
  st->nsrc = nsrc;
  st->src_at = s->nsrcpool;
  st->off = off;
  st->len = len;
  for (int i = 0; i < nsrc; ++i) s->srcpool[s->nsrcpool++] = srcs[i];
  return 0;
}

/* Healthy-ring position arithmetic: R[(j + t) mod P']. */
static int ring_at(const orc_sched *s, int j, int t) {
  int pp = s->pp;
  int idx = ((j + t) % pp + pp) % pp;
  return s->ring[idx];
}

/* The steps of one ring section j of segment g, covering [off, off+len).
 * ordering: 1 = S1-S2-S3-S4, 2 = S3-S1-S4-S2 (Sec. 4.1).  For m >= 2 the
 * ordering-1 segments (A', C') let the worst straggler finalise and fold the
 * others in at the chain start, the exact reading of App. D. */
static int section_steps(orc_sched *s, int g, int j, int ordering, int64_t off,
                         int64_t len) {
  int pp = s->pp, m = s->m, rc = 0;
  int holder = ring_at(s, j, pp - 1); /* R[j-1]: where Stage 1 ends */
  int one[1];
  int *pre = (int *)malloc(sizeof(int) * (size_t)(m > 0 ? m : 1));
  if (!pre) return -2;

  /* slot 0: stragglers' raw values join at the chain start R[j]. */
  int npre = 0;
  if (m >= 1 && ordering == 2)
    for (int i = 0; i < m; ++i) pre[npre++] = s->strag[i];
  if (m >= 2 && ordering == 1)
    for (int i = 1; i < m; ++i) pre[npre++] = s->strag[i];
  if (npre > 0) rc |= push_step(s, 0, g, j, ORC_REDUCE, ring_at(s, j, 0), pre, npre, off, len);

  /* slot 1, Stage 1: P'-1 hops; the receiver adds its own value. */
  for (int t = 1; t <= pp - 1; ++t) {
    one[0] = ring_at(s, j, t - 1);
    rc |= push_step(s, 1, g, j, ORC_REDUCE, ring_at(s, j, t), one, 1, off, len);
  }

  if (m >= 1 && ordering == 1) {
    int fin = s->strag[0];
    /* slot 2, Stage 2: the holder uploads its partial; the straggler adds its
     * own value and so holds the global sum. */
    one[0] = holder;
    rc |= push_step(s, 2, g, j, ORC_REDUCE, fin, one, 1, off, len);
    /* slot 3, Stage 3: the global sum goes back to the holder. */
    one[0] = fin;
    rc |= push_step(s, 3, g, j, ORC_COPY, holder, one, 1, off, len);
  }

  /* slot 4, Stage 4: allgather from the holder along the ring. */
  for (int t = 0; t <= pp - 2; ++t) {
    one[0] = ring_at(s, j, t - 1);
    rc |= push_step(s, 4, g, j, ORC_COPY, ring_at(s, j, t), one, 1, off, len);
  }

  /* slot 5: the global sum reaches the stragglers that did not finalise. */
  if (m >= 1) {
    int first = (ordering == 1) ? 1 : 0;
    for (int i = first; i < m; ++i) {
      one[0] = holder;
      rc |= push_step(s, 5, g, j, ORC_COPY, s->strag[i], one, 1, off, len);
    }
  }
  free(pre);
  return rc;
}

/* The point-to-point allreduce chunk of a segment (bubble filling, Sec. 4.2):
 * every healthy rank sends its own chunk to the straggler, which sums its own
 * value first and then R[0..P'-1] in ring order; the sum is broadcast back. */
static int p2p_steps(orc_sched *s, int g, int64_t off, int64_t len) {
  int rc = 0, one[1];
  int st = s->strag[0];
  rc |= push_step(s, 2, g, -1, ORC_REDUCE, st, s->ring, s->pp, off, len);
  for (int i = 0; i < s->pp; ++i) {
    one[0] = st;
    rc |= push_step(s, 3, g, -1, ORC_COPY, s->ring[i], one, 1, off, len);
  }
  return rc;
}

/* ------------------------------------------------------------- building */

void orc_free(orc_sched *s) {
  if (!s) return;
  free(s->steps);
  free(s->srcpool);
  free(s->seg_off);
  free(s->seg_len);
  free(s->p2p_len);
  free(s);
}


/* Serial order: by slot, keeping build order (segment, section, hop) within
 * a slot (a stable counting sort). */
static int sort_by_slot(orc_sched *s) {
  int64_t cnt[ORC_MAX_SLOTS + 1] = {0};
  for (int64_t i = 0; i < s->nsteps; ++i) cnt[s->steps[i].slot + 1]++;
  for (int q = 0; q < ORC_MAX_SLOTS; ++q) cnt[q + 1] += cnt[q];
  orc_step *sorted = (orc_step *)malloc((size_t)(s->nsteps ? s->nsteps : 1) * sizeof(orc_step));
  if (!sorted) return -2;
  for (int64_t i = 0; i < s->nsteps; ++i) sorted[cnt[s->steps[i].slot]++] = s->steps[i];
  free(s->steps);
  s->steps = sorted;
  s->cap_steps = s->nsteps;
  return 0;
}

/* Build the schedule for segments [seg_lo, seg_hi) (all segments when
 * seg_hi <= 0).  Returns 0, or a negative status with orc_last_error set. */
int orc_build(int p, const double *bw, int64_t n, int k, int seg_lo, int seg_hi,
              orc_sched **out) {
  *out = NULL;
  if (p < 3 || p > 1024) { g_err = "p must be in [3, 1024]"; return -1; }
  if (n < 0) { g_err = "N must be >= 0"; return -1; }
  if (k < 4 || k % 4 != 0) { g_err = "n_chunks must be a positive multiple of 4"; return -1; }
  double bmax = 0.0;
  for (int i = 0; i < p; ++i) {
    if (!(bw[i] > 0.0) || !isfinite(bw[i])) { g_err = "bandwidths must be finite and > 0"; return -1; }
    if (bw[i] > bmax) bmax = bw[i];
  }
  orc_sched *s = (orc_sched *)calloc(1, sizeof(orc_sched));
  if (!s) return -2;
  s->p = p;
  s->n = n;
  s->k = k;
  s->g = 1;
  s->q = p;
  s->nseg = k;
  for (int i = 0; i < p; ++i) s->ell[i] = bmax / bw[i];

  /* Stragglers: ranks slower than the fastest, by l descending, then rank. */
  int m = 0, pp = 0;
  for (int i = 0; i < p; ++i) {
    if (bw[i] < bmax) s->strag[m++] = i;
    else s->ring[pp++] = i;
  }
  for (int a = 1; a < m; ++a) { /* insertion sort, stable on rank */
    int v = s->strag[a], b = a - 1;
    while (b >= 0 && s->ell[s->strag[b]] < s->ell[v]) { s->strag[b + 1] = s->strag[b]; --b; }
    s->strag[b + 1] = v;
  }
  s->m = m;
  s->pp = pp;
  if (pp < 2) { orc_free(s); g_err = "fewer than 2 healthy ranks"; return -3; }
  if (m == 0) s->kind = ORC_RING;
  else if (m == 1) s->kind = (s->ell[s->strag[0]] >= 2.0) ? ORC_SINGLE_GE2 : ORC_SINGLE_LT2;
  else s->kind = ORC_MULTI;

  /* Segment split: NQ quanta, segment g owns quanta [g NQ / k, (g+1) NQ / k). */
  s->seg_off = (int64_t *)calloc((size_t)k, sizeof(int64_t));
  s->seg_len = (int64_t *)calloc((size_t)k, sizeof(int64_t));
  s->p2p_len = (int64_t *)calloc((size_t)k, sizeof(int64_t));
  if (!s->seg_off || !s->seg_len || !s->p2p_len) { orc_free(s); return -2; }
  int64_t nq = (n + ORC_QUANTUM - 1) / ORC_QUANTUM;
  if (seg_hi <= 0 || seg_hi > k) seg_hi = k;
  if (seg_lo < 0) seg_lo = 0;
  s->seg_lo = seg_lo;
  s->seg_hi = seg_hi;

  for (int g = 0; g < k; ++g) {
    int64_t q0 = (int64_t)g * nq / k, q1 = (int64_t)(g + 1) * nq / k;
    int64_t lq = q1 - q0;
    /* Bubble filling: the P2P chunk holds D/L = (2-l)/((p-2)l+2) of the
     * segment, rounded to whole quanta (App. C data accounting). */
    int64_t dq = 0;
    if (s->kind == ORC_SINGLE_LT2) {
      double l = s->ell[s->strag[0]];
      double x = ((double)lq * (2.0 - l)) / ((double)(p - 2) * l + 2.0);
      dq = (int64_t)floor(x + 0.5);
      if (dq < 0) dq = 0;
      if (dq > lq) dq = lq;
    }
    int64_t rq = lq - dq; /* quanta on the ring path */
    int64_t qb = rq / pp, big = rq % pp;
    int64_t seg_b = q0 * ORC_QUANTUM < n ? q0 * ORC_QUANTUM : n;
    int64_t seg_e = q1 * ORC_QUANTUM < n ? q1 * ORC_QUANTUM : n;
    s->seg_off[g] = seg_b;
    s->seg_len[g] = seg_e - seg_b;
    int64_t pb = (q1 - dq) * ORC_QUANTUM, pe = q1 * ORC_QUANTUM;
    if (pb > n) pb = n;
    if (pe > n) pe = n;
    s->p2p_len[g] = pe - pb;
    if (g < seg_lo || g >= seg_hi) continue;

    /* Pattern of segment g: A,B,C,D for one straggler, B,D,A',C' for several;
     * A, C, A', C' use ordering 1 and B, D use ordering 2. */
    int pat = g % 4, ordering;
    if (m <= 1) ordering = (pat == 0 || pat == 2) ? 1 : 2;
    else ordering = (pat <= 1) ? 2 : 1;

    int64_t qcur = q0;
    for (int j = 0; j < pp; ++j) {
      int64_t ql = qb + (j < big ? 1 : 0);
      int64_t b = qcur * ORC_QUANTUM, e = (qcur + ql) * ORC_QUANTUM;
      if (b > n) b = n;
      if (e > n) e = n;
      if (section_steps(s, g, j, ordering, b, e - b)) { orc_free(s); g_err = "out of memory"; return -2; }
      qcur += ql;
    }
    if (dq > 0 && p2p_steps(s, g, pb, pe - pb)) { orc_free(s); g_err = "out of memory"; return -2; }
  }

  if (sort_by_slot(s)) { orc_free(s); return -2; }
  *out = s;
  return 0;
}


/* --------------------------------------------------- several GPUs per server */

/* Rank of local ring position d (0 = leader) of server sv in part i. */
static int srank(const orc_sched *s, int sv, int part, int d) {
  return sv * s->g + (part + d) % s->g;
}

static int chain_server(const orc_sched *s, int j, int t) {
  int pp = s->pp;
  return s->ring[((j + t) % pp + pp) % pp];
}

/* The steps of section j of a segment of part `part` (App. E, NVLink phases
 * N1-N4 around Stages S1-S4).  type 1: S1-S2-S3-S4, type 2: S3-S1-S4-S2. */
static int server_section_steps(orc_sched *s, int seg, int part, int j, int type,
                                 int64_t off, int64_t len) {
  int g = s->g, pp = s->pp, sv = s->strag[0], rc = 0, one[1];
  int last = pp - 1; /* chain position of the holder */
  /* N1: every healthy server collects its local values onto its leader. */
  for (int h = 0; h < pp; ++h)
    for (int d = g - 2; d >= 0; --d) {
      one[0] = srank(s, s->ring[h], part, d + 1);
      rc |= push_step(s, 1, seg, j, ORC_REDUCE, srank(s, s->ring[h], part, d), one, 1, off, len);
    }
  if (type == 2) {
    /* N3 (type 2): the straggler server collects onto its leader ... */
    for (int d = g - 2; d >= 0; --d) {
      one[0] = srank(s, sv, part, d + 1);
      rc |= push_step(s, 0, seg, j, ORC_REDUCE, srank(s, sv, part, d), one, 1, off, len);
    }
    /* ... S3: and sends its sum to the chain start, which adds it. */
    one[0] = srank(s, sv, part, 0);
    rc |= push_step(s, 2, seg, j, ORC_REDUCE, srank(s, chain_server(s, j, 0), part, 0), one, 1, off, len);
  }
  /* S1: reduce-scatter chain over the healthy leaders. */
  for (int t = 1; t <= pp - 1; ++t) {
    one[0] = srank(s, chain_server(s, j, t - 1), part, 0);
    rc |= push_step(s, 3, seg, j, ORC_REDUCE, srank(s, chain_server(s, j, t), part, 0), one, 1, off, len);
  }
  int holder = srank(s, chain_server(s, j, last), part, 0);
  if (type == 1) {
    /* S2: the straggler leader adds the healthy partial to its own value. */
    one[0] = holder;
    rc |= push_step(s, 4, seg, j, ORC_REDUCE, srank(s, sv, part, 0), one, 1, off, len);
    /* N2 (type 1): forward along the local ring, each GPU adding its own. */
    for (int d = 1; d <= g - 1; ++d) {
      one[0] = srank(s, sv, part, d - 1);
      rc |= push_step(s, 5, seg, j, ORC_REDUCE, srank(s, sv, part, d), one, 1, off, len);
    }
    /* N3 (type 1): the global sum travels back to the leader. */
    for (int d = g - 2; d >= 0; --d) {
      one[0] = srank(s, sv, part, d + 1);
      rc |= push_step(s, 6, seg, j, ORC_COPY, srank(s, sv, part, d), one, 1, off, len);
    }
    /* S3: straggler leader -> holder. */
    one[0] = srank(s, sv, part, 0);
    rc |= push_step(s, 7, seg, j, ORC_COPY, holder, one, 1, off, len);
  }
  /* S4: allgather over the healthy leaders from the holder. */
  for (int t = 0; t <= pp - 2; ++t) {
    one[0] = srank(s, chain_server(s, j, t - 1), part, 0);
    rc |= push_step(s, 8, seg, j, ORC_COPY, srank(s, chain_server(s, j, t), part, 0), one, 1, off, len);
  }
  /* N4: every healthy leader distributes along its local ring. */
  for (int h = 0; h < pp; ++h)
    for (int d = 1; d <= g - 1; ++d) {
      one[0] = srank(s, s->ring[h], part, d - 1);
      rc |= push_step(s, 9, seg, j, ORC_COPY, srank(s, s->ring[h], part, d), one, 1, off, len);
    }
  if (type == 2) {
    /* S2 (type 2): holder -> straggler leader; N2: distribute there. */
    one[0] = holder;
    rc |= push_step(s, 10, seg, j, ORC_COPY, srank(s, sv, part, 0), one, 1, off, len);
    for (int d = 1; d <= g - 1; ++d) {
      one[0] = srank(s, sv, part, d - 1);
      rc |= push_step(s, 11, seg, j, ORC_COPY, srank(s, sv, part, d), one, 1, off, len);
    }
  }
  return rc;
}

/* Schedule for q servers of g GPUs with one bandwidth per server, exactly
 * one straggler server (App. E covers the single-straggler case).  k is the
 * number of segments per part: 8 | k and k >= 24 (App. E notation). */
int orc_build_servers(int q, int g, const double *sbw, int64_t n, int k, int seg_lo,
                      int seg_hi, orc_sched **out) {
  *out = NULL;
  if (q < 3 || g < 2 || (int64_t)q * g > 1024) { g_err = "need q >= 3 servers, g >= 2, q*g <= 1024"; return -1; }
  if (n < 0) { g_err = "N must be >= 0"; return -1; }
  if (k < 24 || k % 8 != 0) { g_err = "n_chunks must be a multiple of 8 and >= 24"; return -1; }
  double bmax = 0.0;
  for (int i = 0; i < q; ++i) {
    if (!(sbw[i] > 0.0) || !isfinite(sbw[i])) { g_err = "bandwidths must be finite and > 0"; return -1; }
    if (sbw[i] > bmax) bmax = sbw[i];
  }
  orc_sched *s = (orc_sched *)calloc(1, sizeof(orc_sched));
  if (!s) return -2;
  s->p = q * g;
  s->q = q;
  s->g = g;
  s->n = n;
  s->k = k;
  s->nseg = g * k;
  s->kind = ORC_SERVERS;
  int m = 0, pp = 0;
  for (int sv = 0; sv < q; ++sv) {
    if (sbw[sv] < bmax) s->strag[m++] = sv;
    else s->ring[pp++] = sv;
    for (int l = 0; l < g; ++l) s->ell[sv * g + l] = bmax / sbw[sv];
  }
  s->m = m;
  s->pp = pp;
  if (m != 1) { orc_free(s); g_err = "exactly one straggler server is supported"; return -3; }
  s->seg_off = (int64_t *)calloc((size_t)s->nseg, sizeof(int64_t));
  s->seg_len = (int64_t *)calloc((size_t)s->nseg, sizeof(int64_t));
  s->p2p_len = (int64_t *)calloc((size_t)s->nseg, sizeof(int64_t));
  if (!s->seg_off || !s->seg_len || !s->p2p_len) { orc_free(s); return -2; }
  if (seg_hi <= 0 || seg_hi > s->nseg) seg_hi = s->nseg;
  if (seg_lo < 0) seg_lo = 0;
  s->seg_lo = seg_lo;
  s->seg_hi = seg_hi;
  int64_t nq = (n + ORC_QUANTUM - 1) / ORC_QUANTUM;
  for (int part = 0; part < g; ++part) {
    int64_t p0 = (int64_t)part * nq / g, p1 = (int64_t)(part + 1) * nq / g, lp = p1 - p0;
    for (int sg = 0; sg < k; ++sg) {
      int gs = part * k + sg;
      int64_t q0 = p0 + (int64_t)sg * lp / k, q1 = p0 + (int64_t)(sg + 1) * lp / k;
      int64_t b0 = q0 * ORC_QUANTUM < n ? q0 * ORC_QUANTUM : n;
      int64_t e0 = q1 * ORC_QUANTUM < n ? q1 * ORC_QUANTUM : n;
      s->seg_off[gs] = b0;
      s->seg_len[gs] = e0 - b0;
      if (gs < seg_lo || gs >= seg_hi) continue;
      int type = (sg % 4 == 0 || sg % 4 == 2) ? 1 : 2;
      int64_t rq = q1 - q0, qb = rq / pp, big = rq % pp, qcur = q0;
      for (int j = 0; j < pp; ++j) {
        int64_t ql = qb + (j < big ? 1 : 0);
        int64_t b = qcur * ORC_QUANTUM, e = (qcur + ql) * ORC_QUANTUM;
        if (b > n) b = n;
        if (e > n) e = n;
        if (server_section_steps(s, gs, part, j, type, b, e - b)) { orc_free(s); g_err = "out of memory"; return -2; }
        qcur += ql;
      }
    }
  }
  if (sort_by_slot(s)) { orc_free(s); return -2; }
  *out = s;
  return 0;
}

/* ------------------------------------------------------------ accessors */

int orc_info(const orc_sched *s, int64_t *out12, int *ring, int *strag, double *ell) {
  out12[0] = s->p; out12[1] = s->k; out12[2] = s->m; out12[3] = s->kind;
  out12[4] = s->pp; out12[5] = s->n; out12[6] = s->nsteps; out12[7] = s->nsrcpool;
  out12[8] = s->g; out12[9] = s->q; out12[10] = s->nseg; out12[11] = 0;
  for (int i = 0; i < s->pp; ++i) ring[i] = s->ring[i];
  for (int i = 0; i < s->m; ++i) strag[i] = s->strag[i];
  for (int i = 0; i < s->p; ++i) ell[i] = s->ell[i];
  return 0;
}

void orc_segments(const orc_sched *s, int64_t *off, int64_t *len, int64_t *p2p) {
  for (int g = 0; g < s->nseg; ++g) { off[g] = s->seg_off[g]; len[g] = s->seg_len[g]; p2p[g] = s->p2p_len[g]; }
}

/* Export the steps as parallel arrays: ints[i*6 + .] = slot, seg, sec, op,
 * dst, nsrc; offs[i*3 + .] = src_at, off, len; pool = source ranks. */
void orc_steps(const orc_sched *s, int32_t *ints, int64_t *offs, int32_t *pool) {
  for (int64_t i = 0; i < s->nsteps; ++i) {
    const orc_step *st = &s->steps[i];
    int32_t *a = ints + 6 * i;
    a[0] = st->slot; a[1] = st->seg; a[2] = st->sec; a[3] = st->op; a[4] = st->dst; a[5] = st->nsrc;
    int64_t *b = offs + 3 * i;
    b[0] = st->src_at; b[1] = st->off; b[2] = st->len;
  }
  memcpy(pool, s->srcpool, (size_t)s->nsrcpool * sizeof(int32_t));
}

/* ------------------------------------------------------------ arithmetic */

static float bf16_widen(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

/* fp32 -> bf16, round to nearest, ties to even (NaN stays NaN, quietened). */
static uint16_t bf16_narrow(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u);
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7fffu + lsb;
  return (uint16_t)(u >> 16);
}

/* binary16 -> fp32, exact.  Layout: sign, 5-bit exponent (bias 15), 10-bit
 * fraction; exponent 0 holds zeros and subnormals (fraction * 2^-24), 31
 * infinities and NaNs (returned quiet, payload kept). */
static float f16_widen(uint16_t h) {
  const uint32_t sign = (uint32_t)(h & 0x8000u) << 16;
  const uint32_t e = (h >> 10) & 0x1fu, m = h & 0x3ffu;
  uint32_t u;
  if (e == 0) {
    float f = ldexpf((float)m, -24);  /* exact: m < 2^10 */
    memcpy(&u, &f, 4);
    u |= sign;
  } else if (e == 31) {
    u = sign | 0x7f800000u | (m ? 0x00400000u | (m << 13) : 0u);
  } else {
    u = sign | ((e - 15u + 127u) << 23) | (m << 13);
  }
  float f;
  memcpy(&f, &u, 4);
  return f;
}

/* fp32 -> binary16, round to nearest, ties to even.  |f| >= 65520 (the
 * midpoint between the largest finite value 65504 and 2^16) becomes
 * infinity; values below 2^-14 become subnormals (units of 2^-24), and
 * |f| <= 2^-25 (a tie with zero at most) becomes zero. */
static uint16_t f16_narrow(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  const uint16_t sign = (uint16_t)((u >> 16) & 0x8000u);
  const uint32_t a = u & 0x7fffffffu;
  if (a > 0x7f800000u) return (uint16_t)(sign | 0x7e00u | ((a >> 13) & 0x3ffu));  /* NaN */
  if (a >= 0x477ff000u) return (uint16_t)(sign | 0x7c00u);  /* >= 65520: infinity */
  if (a >= 0x38800000u) {  /* normal result: keep 10 of the 23 fraction bits */
    const uint32_t e = (a >> 23) - 127u + 15u;
    uint32_t h = (e << 10) | ((a >> 13) & 0x3ffu);
    const uint32_t rem = a & 0x1fffu;
    if (rem > 0x1000u || (rem == 0x1000u && (h & 1u))) h += 1u;  /* may carry into e */
    return (uint16_t)(sign | h);
  }
  if (a <= 0x33000000u) return sign;  /* |f| <= 2^-25 */
  /* subnormal result: m = |f| / 2^-24 rounded; |f| = mm * 2^(e - 150) */
  const uint32_t e = a >> 23, mm = (a & 0x7fffffu) | 0x800000u;
  const uint32_t sh = 126u - e;  /* 14 .. 24 */
  uint32_t m = mm >> sh;
  const uint32_t rem = mm & ((1u << sh) - 1u), half = 1u << (sh - 1u);
  if (rem > half || (rem == half && (m & 1u))) m += 1u;
  return (uint16_t)(sign | m);
}

uint16_t orc_bf16_round(float f) { return bf16_narrow(f); }

void orc_f16_round_array(const float *x, uint16_t *y, int64_t n) {
  for (int64_t i = 0; i < n; ++i) y[i] = f16_narrow(x[i]);
}

void orc_f16_widen_array(const uint16_t *x, float *y, int64_t n) {
  for (int64_t i = 0; i < n; ++i) y[i] = f16_widen(x[i]);
}

void orc_bf16_round_array(const float *x, uint16_t *y, int64_t n) {
  for (int64_t i = 0; i < n; ++i) y[i] = bf16_narrow(x[i]);
}

/* One step applied to element c of every involved buffer. */
static void apply_elem(int dtype, const orc_step *st, const int32_t *srcs, void **bufs,
                       int64_t c) {
  if (dtype == ORC_F32) {
    float **b = (float **)bufs;
    if (st->op == ORC_COPY) { b[st->dst][c] = b[srcs[0]][c]; return; }
    float acc = b[st->dst][c];
    for (int i = 0; i < st->nsrc; ++i) acc = acc + b[srcs[i]][c];
    b[st->dst][c] = acc;
  } else if (dtype == ORC_BF16) {
    uint16_t **b = (uint16_t **)bufs;
    if (st->op == ORC_COPY) { b[st->dst][c] = b[srcs[0]][c]; return; }
    float acc = bf16_widen(b[st->dst][c]);
    for (int i = 0; i < st->nsrc; ++i) acc = acc + bf16_widen(b[srcs[i]][c]);
    b[st->dst][c] = bf16_narrow(acc);
  } else if (dtype == ORC_F16) {
    uint16_t **b = (uint16_t **)bufs;
    if (st->op == ORC_COPY) { b[st->dst][c] = b[srcs[0]][c]; return; }
    float acc = f16_widen(b[st->dst][c]);
    for (int i = 0; i < st->nsrc; ++i) acc = acc + f16_widen(b[srcs[i]][c]);
    b[st->dst][c] = f16_narrow(acc);
  } else {
    uint32_t **b = (uint32_t **)bufs;
    if (st->op == ORC_COPY) { b[st->dst][c] = b[srcs[0]][c]; return; }
    uint32_t acc = b[st->dst][c];
    for (int i = 0; i < st->nsrc; ++i) acc = acc + b[srcs[i]][c];
    b[st->dst][c] = acc;
  }
}

/* Execute every step with slot in [slot_lo, slot_hi), serially, in order,
 * over whole rank buffers (p host pointers of N elements). */
int orc_run(const orc_sched *s, int dtype, void **bufs, int slot_lo, int slot_hi) {
  if (dtype < 0 || dtype > 3) { g_err = "bad dtype"; return -1; }
  for (int64_t i = 0; i < s->nsteps; ++i) {
    const orc_step *st = &s->steps[i];
    if (st->slot < slot_lo || st->slot >= slot_hi) continue;
    const int32_t *srcs = s->srcpool + st->src_at;
    for (int64_t c = st->off; c < st->off + st->len; ++c) apply_elem(dtype, st, srcs, bufs, c);
  }
  return 0;
}

/* Same result as orc_run, bit for bit, on `nthreads` host threads (OpenMP).
 * Every step reads and writes coordinates of its own segment only, and a
 * coordinate's steps run in serial order whatever the thread: the segments
 * are shared out among the threads, and each runs its segment's steps in
 * the serial order of orc_run.  So every coordinate sees exactly the
 * operations of orc_run, in the same order. */
int orc_run_parallel(const orc_sched *s, int dtype, void **bufs, int slot_lo, int slot_hi,
                     int nthreads) {
  if (dtype < 0 || dtype > 3) { g_err = "bad dtype"; return -1; }
  if (nthreads < 1) { g_err = "nthreads must be >= 1"; return -1; }
  int nseg = s->nseg;
  /* step indices grouped by segment, each group in serial order */
  int64_t *start = (int64_t *)calloc((size_t)nseg + 1, sizeof(int64_t));
  int64_t *order = (int64_t *)malloc((size_t)(s->nsteps ? s->nsteps : 1) * sizeof(int64_t));
  if (!start || !order) { free(start); free(order); g_err = "out of memory"; return -2; }
  for (int64_t i = 0; i < s->nsteps; ++i) start[s->steps[i].seg + 1]++;
  for (int g = 0; g < nseg; ++g) start[g + 1] += start[g];
  int64_t *fill = (int64_t *)malloc(((size_t)nseg + 1) * sizeof(int64_t));
  if (!fill) { free(start); free(order); g_err = "out of memory"; return -2; }
  memcpy(fill, start, ((size_t)nseg + 1) * sizeof(int64_t));
  for (int64_t i = 0; i < s->nsteps; ++i) order[fill[s->steps[i].seg]++] = i;
  free(fill);
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
  for (int g = 0; g < nseg; ++g) {
    for (int64_t a = start[g]; a < start[g + 1]; ++a) {
      const orc_step *st = &s->steps[order[a]];
      if (st->slot < slot_lo || st->slot >= slot_hi) continue;
      const int32_t *srcs = s->srcpool + st->src_at;
      for (int64_t c = st->off; c < st->off + st->len; ++c) apply_elem(dtype, st, srcs, bufs, c);
    }
  }
  free(start);
  free(order);
  return 0;
}

/* Same as orc_run restricted to the sorted coordinates coords[0..S): cols
 * holds p host pointers to S values each (column i of rank r is coordinate
 * coords[i]).  Used to check full-size runs at sampled coordinates. */
int orc_run_sampled(const orc_sched *s, int dtype, void **cols, const int64_t *coords,
                    int64_t S, int slot_lo, int slot_hi) {
  if (dtype < 0 || dtype > 3) { g_err = "bad dtype"; return -1; }
  for (int64_t i = 1; i < S; ++i)
    if (coords[i] <= coords[i - 1]) { g_err = "coords must be strictly increasing"; return -1; }
  for (int64_t i = 0; i < s->nsteps; ++i) {
    const orc_step *st = &s->steps[i];
    if (st->slot < slot_lo || st->slot >= slot_hi) continue;
    const int32_t *srcs = s->srcpool + st->src_at;
    /* first sampled coordinate >= st->off */
    int64_t lo = 0, hi = S;
    while (lo < hi) {
      int64_t mid = lo + (hi - lo) / 2;
      if (coords[mid] < st->off) lo = mid + 1; else hi = mid;
    }
    for (int64_t a = lo; a < S && coords[a] < st->off + st->len; ++a)
      apply_elem(dtype, st, srcs, cols, a);
  }
  return 0;
}
