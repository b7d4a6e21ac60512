/*
 * optcc.h - C ABI of the OptCC schedule-execution library for MI355X (gfx950).
 *
 * OptCC ("Don't Let a Few Network Failures Slow the Entire AllReduce") is a
 * four-stage pipelined AllReduce for clusters in which a few ranks' NICs are
 * slower (stragglers).  This library builds its schedule and executes every
 * step of it on one GPU, where the p logical ranks are p buffers in HBM:
 * after optcc_allreduce_emulate every buffer holds the elementwise sum of all
 * p inputs (Sec. 3, problem setting: correctness conditions (i) and (ii)).
 *
 * Conventions for every entry point:
 *   - status codes: OPTCC_OK (0) or a negative OPTCC_E* value; the message of
 *     the last failure on the calling thread is returned by optcc_last_error.
 *   - the library never aborts and never allocates on behalf of the caller
 *     except where stated.
 *   - device memory (bufs) is caller-owned.  A plan is host memory owned by
 *     the caller (optcc_plan / optcc_plan_free); it lazily owns one small
 *     read-only device copy of its step tables per device it has run on.
 *   - "stream" is a hipStream_t (NULL = the default stream).  Emulation calls
 *     are asynchronous and return once the kernels are enqueued.  The first
 *     call of a plan on a device with elements of a given size (2 or 4 bytes)
 *     uploads its tables (hipMalloc + hipMemcpy) and so may not be captured
 *     into a HIP graph (made during a capture, it fails with OPTCC_EINVAL
 *     before touching the device and the capture stays valid); every later
 *     call only launches kernels and may be captured.
 */
#ifndef OPTCC_H
#define OPTCC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OPTCC_OK 0
#define OPTCC_EINVAL (-1)      /* bad argument, or arguments that disagree with the plan */
#define OPTCC_ENOMEM (-2)      /* host or device allocation failed */
/* outside the method's domain (p < 3, fewer than 2 healthy ranks) or this
 * library's limits */
#define OPTCC_EUNSUPPORTED (-3)
#define OPTCC_EDEVICE (-4)     /* a HIP runtime call failed; the message names it */

#define OPTCC_MAX_RANKS 1024        /* largest p a plan accepts */
#define OPTCC_MAX_EMULATE_RANKS 256 /* largest p the GPU executor accepts */
#define OPTCC_NUM_SLOTS 6           /* stage slots of a one-GPU-per-server plan */
#define OPTCC_NUM_SERVER_SLOTS 12   /* stage slots of a several-GPUs-per-server plan */
#define OPTCC_MAX_GPUS_PER_SERVER 64 /* largest g optcc_plan_servers accepts */
#define OPTCC_QUANTUM 64            /* split quantum in elements */

typedef struct optcc_plan optcc_plan_t;

typedef enum { OPTCC_F32 = 0, OPTCC_BF16 = 1, OPTCC_I32 = 2, OPTCC_F16 = 3 } optcc_dtype_t;

typedef enum {
  OPTCC_KIND_RING = 0,       /* no straggler: the ring of Sec. 3 (T0) */
  OPTCC_KIND_SINGLE_GE2 = 1, /* one straggler with l >= 2 (Sec. 4.3, first case) */
  OPTCC_KIND_SINGLE_LT2 = 2, /* one straggler with l < 2: bubble filling (Sec. 4.2, App. C) */
  OPTCC_KIND_MULTI = 3,      /* m >= 2 stragglers (App. D) */
  OPTCC_KIND_SERVERS = 4     /* g >= 2 GPUs per server, one straggler server (App. E) */
} optcc_kind_t;

/*
 * optcc_plan - build the OptCC schedule for p ranks (Sec. 4.1-4.2, App. C, App. D).
 *
 *   p               number of ranks, 3 <= p <= OPTCC_MAX_RANKS (Sec. 3 needs p >= 3)
 *   link_bandwidths host array of p finite values > 0, any unit.  Slowdowns
 *                   are l_i = max(b) / b_i; every rank slower than the fastest
 *                   is a straggler, sorted by l descending, ties to lower rank.
 *   N               elements per rank, N >= 0
 *   n_chunks        k, the number of segments: a positive multiple of 4
 *                   (Sec. 4.2: k/4 segments per pattern)
 *   out             receives the plan; untouched on failure
 *
 * Split: quanta of OPTCC_QUANTUM elements; segment g owns quanta
 * [floor(g*NQ/k), floor((g+1)*NQ/k)) with NQ = ceil(N/64).  For one straggler
 * with l < 2 each segment ends with a point-to-point chunk of
 * floor(Lq*(2-l)/((p-2)*l+2) + 0.5) quanta (App. C: D = (2-l)s'/l); the rest
 * is split over the P' = p - m healthy ranks' sections, the first (rem)
 * sections one quantum larger.  Ranges are clipped at N.
 * Errors: OPTCC_EINVAL (bad p/N/k/bandwidths), OPTCC_EUNSUPPORTED (p > limit,
 * fewer than 2 healthy ranks), OPTCC_ENOMEM.  No device call is made.
 */
int optcc_plan(int p, const double *link_bandwidths, int64_t N, int n_chunks,
               optcc_plan_t **out);

/*
 * optcc_plan_servers - build the OptCC schedule for q servers of g GPUs each
 * with one straggler server (App. E: NVLink phases N1-N4 around the four NIC
 * stages, two schedule types, no bubble filling).
 *
 *   q, g              servers and GPUs per server: q >= 3, 2 <= g <=
 *                     OPTCC_MAX_GPUS_PER_SERVER, p = q*g <= OPTCC_MAX_RANKS.
 *                     Ranks are numbered server-major: rank = server*g + local
 *                     index.
 *   server_bandwidths host array of q finite values > 0: one NIC bandwidth per
 *                     server (PXN pools a server's NICs, Sec. 2, so all its
 *                     GPUs share one slowdown l = max(b)/b).  Exactly one
 *                     server must be slower than the fastest.
 *   N                 elements per rank, N >= 0
 *   n_chunks          k, segments per part: a multiple of 8 and >= 24 (App. E
 *                     notation: the pattern overlay needs 8 | k and k >= 24)
 *   out               receives the plan; untouched on failure
 *
 * Split: the vector's NQ = ceil(N/64) quanta form g parts, part i =
 * [floor(i*NQ/g), floor((i+1)*NQ/g)), led by local GPU i of every server;
 * each part is cut into k segments like optcc_plan (segment index part*k + c),
 * and each segment into q-1 sections (one per healthy server), the first
 * (rem) one quantum larger.  Segment c of a part uses schedule type 1
 * (S1-S2-S3-S4, patterns A and C) when c mod 4 is 0 or 2, type 2
 * (S3-S1-S4-S2, patterns B and D) otherwise.  Local ring of part i on every
 * server: position d is local GPU (i + d) mod g; collect phases run it
 * backwards onto the leader (d = 0), distribute phases forwards.
 * The plan's ring[] and stragglers[] hold server indices.
 * Errors: OPTCC_EINVAL (bad q/g/N/k/bandwidths), OPTCC_EUNSUPPORTED (no or
 * several straggler servers, p over the limit), OPTCC_ENOMEM.  No device call.
 */
int optcc_plan_servers(int q, int g, const double *server_bandwidths, int64_t N, int n_chunks,
                       optcc_plan_t **out);

/* Free a plan and its device tables (the plan was built by optcc_plan or
 * optcc_plan_servers, whose passages define it).  The caller guarantees that
 * no emulation using it is still running on any stream, and that every HIP
 * graph that captured an emulation call of this plan has been destroyed
 * first: a graph keeps the addresses of the plan's device tables, so
 * replaying it after the free would read freed memory.  NULL is ignored. */
void optcc_plan_free(optcc_plan_t *plan);

/*
 * optcc_allreduce_emulate - execute every step of the plan, in place, as one
 * fused launch on `stream` (Sec. 4.1 Stages 1-4 for every section in its
 * pattern's stage ordering, plus App. C bubble filling and App. D's
 * stragglers).  On completion every buffer holds the elementwise sum.
 *
 *   bufs   host array of p device pointers; bufs[r] holds rank r's N elements
 *          of `dtype`, aligned to the element size.  Buffers must not overlap.
 *          16-byte alignment of every pointer enables the vector path;
 *          128-byte (cache-line) alignment gives full speed (16-byte-only
 *          alignment costs 3-24 %, element alignment 1.4-3.6x).
 *   p, N   must equal the plan's
 *   dtype  OPTCC_F32 (fp32 adds), OPTCC_BF16 and OPTCC_F16 (IEEE binary16)
 *          (fp32 accumulation, one round-to-nearest-even per step; fp16
 *          keeps subnormals and overflows to infinity), OPTCC_I32 (adds
 *          modulo 2^32)
 *
 * Every step writes its destination rank's buffer; a partial sum that the
 * next step of the same section consumes is kept in registers.  The result is
 * bitwise deterministic.  With N = 0 (or an empty slot range) nothing is
 * read or written and the pointers are not inspected.  Errors: OPTCC_EINVAL
 * (mismatch with the plan, NULL or misaligned pointers, overlapping buffers
 * or buffers that would run past the end of the address space, a first call
 * on a device made while `stream` is being captured), OPTCC_EUNSUPPORTED
 * (p > OPTCC_MAX_EMULATE_RANKS, or a segment whose ring sections hold 2^31
 * or more quanta: the device tables index a segment's quanta in 32 bits;
 * that is N of about 2^39 elements per rank at k = 4, beyond one GPU's HBM),
 * OPTCC_EDEVICE, OPTCC_ENOMEM (first use of the plan on a device allocates
 * its tables).  These checks are made before any device call.
 *
 * Launch order of the tiles (never the result): plans of more than 32
 * healthy ranks with one GPU per server whose tiles outnumber 2,048
 * (4,096 with fewer than 90 healthy ranks; a tile is one 16-byte vector per
 * lane, 1,024 elements for 32-bit types, for these plans), and plans of 90
 * or more ranks with several GPUs per server whose tiles (2,048 elements
 * here) outnumber 4,096 (2,048 from 120 ranks) and whose buffers are
 * 16-byte aligned,
 * run a grid of the resident workgroups that take tiles from a device
 * counter.  Each such call takes its own 64-byte counter block from a ring
 * of 4,096 per plan and device (256 KiB, allocated and zeroed by the plan's
 * first such call on the device; if that fails the call keeps the static
 * order), and
 * its last workgroup sets the block back to zero.  So at most 4,096 of
 * these calls of one plan may be queued or running at once on one device,
 * over all streams; beyond that two could share a block.  Calls captured
 * into a HIP graph keep the static order.
 */
int optcc_allreduce_emulate(void *const *bufs, int p, int64_t N, optcc_dtype_t dtype,
                            const optcc_plan_t *plan, void *stream);

/*
 * optcc_allreduce_emulate_slots - execute only the steps whose stage slot is
 * in [slot_begin, slot_end), either fused in one launch (launches = 1) or as
 * one launch per slot (launches = 0), same buffers and errors as above.
 * Slots of a one-GPU-per-server plan (each section uses a subset, always in
 * increasing order):
 *   0  stragglers' raw values folded into the chain start (ordering 2, Sec. 4.1;
 *      the non-finalising stragglers of A'/C', App. D)
 *   1  Stage 1 reduce-scatter chain        2  Stage 2 upload; P2P up (App. C)
 *   3  Stage 3 download; P2P down          4  Stage 4 allgather
 *   5  global sum to the stragglers that did not finalise (ordering 2 Stage 2)
 * Slots of a several-GPUs-per-server plan (App. E; "leader" = local ring
 * position 0 of the section's part, type = schedule type of the segment):
 *   0  N3 collect onto the straggler server's leader (type 2)
 *   1  N1 collect onto every healthy server's leader
 *   2  S3: the straggler leader's sum added into the chain start (type 2)
 *   3  S1 reduce-scatter chain over the healthy leaders
 *   4  S2: the straggler leader adds the holder's partial (type 1)
 *   5  N2 fold: forward along the straggler's local ring, each GPU adding
 *      its own value (type 1)
 *   6  N3: the global sum copied back along the straggler's ring (type 1)
 *   7  S3: straggler leader -> holder (type 1)
 *   8  S4 allgather over the healthy leaders
 *   9  N4 distribute on every healthy server
 *   10 S2: holder -> straggler leader (type 2)
 *   11 N2 distribute on the straggler server (type 2)
 * After [0, s) the buffers equal the state after the first s slots of every
 * section; [0, 6) (or [0, 12)) is the whole AllReduce.
 */
int optcc_allreduce_emulate_slots(void *const *bufs, int p, int64_t N, optcc_dtype_t dtype,
                                  const optcc_plan_t *plan, int slot_begin, int slot_end,
                                  int launches, void *stream);

/*
 * optcc_allreduce_emulate_noalloc - optcc_allreduce_emulate for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Same arguments, result (bit for
 * bit) and errors as optcc_allreduce_emulate, and the caller still passes the
 * buffers.  It calls no hipMalloc, hipFree or other allocating routine: the
 * plan's step tables (32 bytes per segment, rounded up to 256, plus 16 bytes
 * per tile of 1024-8192 elements) are copied on `stream`, on every call, into
 * a static device array of OPTCC_NOALLOC_SCRATCH_BYTES that the library holds
 * on each GPU it runs on until the process ends; a plan whose tables need
 * more is refused with OPTCC_EUNSUPPORTED before any device call (about 2^29
 * elements per rank at 2048-element tiles fit).  Every call on one GPU shares
 * that GPU's array, which keeps the last call's tables (nothing in it must
 * start at zero): calls on one GPU that overlap in time (on different
 * streams, or from several host threads without ordering) race and give
 * undefined results.  The plan must stay alive until the call's work on
 * `stream` has completed (its host tables are the copies' source).  Tiles
 * always run in the static order here (no device counters), so the long
 * plans that optcc_allreduce_emulate runs with work stealing take a few per
 * cent longer through this entry point; the result is the same.
 */
#define OPTCC_NOALLOC_SCRATCH_BYTES (4 << 20)
int optcc_allreduce_emulate_noalloc(void *const *bufs, int p, int64_t N, optcc_dtype_t dtype,
                                    const optcc_plan_t *plan, void *stream);

/*
 * optcc_model_time - completion time of the plan's schedule in the paper's
 * bandwidth-bound model (a healthy NIC moves one element per time unit; Sec. 3),
 * for N elements per rank, in fp64:
 *   no straggler      T0 = 2(p-1)N/p
 *   one, l >= 2       l N (k+1)/k                                   (Sec. 4.3)
 *   one, l < 2        2(p-1) l N/((p-2)l+2) * (k+l-1)/k             (Sec. 4.3, App. C)
 *   m >= 2            (k+4) max{2(p-1)s, (l_1(p-m)+2(m-1))s}, s = N/(k(p-m))  (App. D)
 *   g GPUs/server     max{l, 2} N (k+5.5)/(g k)                     (App. E time analysis)
 * link_bandwidths may be NULL (use the plan's) or must give the same
 * stragglers and slowdowns (relative difference <= 1e-12): p entries, or q
 * (one per server) for a server plan.  Returns NaN on error, with
 * optcc_last_error set.
 */
double optcc_model_time(const optcc_plan_t *plan, const double *link_bandwidths);

/*
 * optcc_lower_bound - best known lower bound on any correct AllReduce for
 * this profile and N, in the same unit (App. A, best lower bounds):
 *   no straggler  T0;  one straggler  max{2l(p-1)/(l(p-2)+2), l} N  (tight bound, App. B.1);
 *   m >= 2        max{2(p-1)/(p-m+sum 1/l_i), l_1} N  (Theorem 2).
 * Returns NaN on invalid input (p < 3, bad bandwidths, N < 0).
 */
double optcc_lower_bound(int p, const double *link_bandwidths, int64_t N);

/*
 * optcc_lower_bound_servers - best known lower bound for q servers of g GPUs
 * with one straggler server, same unit (tight multi-GPU bound, App. B.3):
 *   (N/g) max{2l(q-1)/(l(q-2)+2), l};  without a straggler the fault-free
 *   optimum 2(p-1)N/(g p) with p = q g (Sec. 3).
 * Returns NaN on invalid input (q < 3, g < 1, bad bandwidths, N < 0, or more
 * than one straggler server).
 */
double optcc_lower_bound_servers(int q, int g, const double *server_bandwidths, int64_t N);

/*
 * optcc_narrow_f32 - round n fp32 values to dtype (OPTCC_BF16 or OPTCC_F16)
 * with the rule every reduce step of the executor applies to its fp32 sum:
 * round to nearest, ties to even; bf16 NaNs stay NaN (quietened, payload
 * kept in the top bits), fp16 keeps subnormals and overflows to infinity.
 * This is the per-step rounding of 16-bit data (Sec. 3 result applied to a
 * 16-bit wire, one rounding per step), exposed so that it can be checked
 * against an independent implementation over every fp32 pattern.
 *   src    device array of n floats (4-byte aligned)
 *   dst    device array of n 16-bit results (2-byte aligned); may not
 *          overlap src
 * Asynchronous on `stream`.  Errors: OPTCC_EINVAL (n < 0, NULL, misaligned or
 * overlapping pointers with n > 0, an array that would run past the end of
 * the address space, other dtypes), OPTCC_EDEVICE.
 */
int optcc_narrow_f32(const float *src, void *dst, int64_t n, optcc_dtype_t dtype, void *stream);

/* Message of the last failure on the calling thread ("" if none).  Library
 * plumbing, not part of the method: every entry point above sets it when it
 * returns an error status (or NaN) and clears it on entry to an emulation. */
const char *optcc_last_error(void);

/* ------------------------------------------------------------ introspection
 * Plan data for tests and reports.  No code is shared with any checker. */

typedef struct {
  int32_t p, k, m, kind;
  int32_t healthy;  /* P' = p - m (healthy servers q - 1 for a server plan) */
  int32_t quantum;  /* OPTCC_QUANTUM */
  int64_t n;
  int64_t num_steps; /* steps: one destination write each */
  int64_t num_flows; /* flows: one per (step, source rank) */
  int32_t g, q;          /* GPUs per server (1 for optcc_plan) and servers */
  int32_t num_segments;  /* k, or g*k for a server plan */
  int32_t num_slots;     /* OPTCC_NUM_SLOTS or OPTCC_NUM_SERVER_SLOTS */
} optcc_plan_info_t;

/* Fill info and, when non-NULL, ring[P'] (healthy ranks in ring order; server
 * indices for a server plan), stragglers[m] (sorted; servers likewise) and
 * slowdowns[p] (per rank). */
int optcc_plan_info(const optcc_plan_t *plan, optcc_plan_info_t *info, int32_t *ring,
                    int32_t *stragglers, double *slowdowns);

/* Per segment (num_segments entries each): element offset, length, and
 * length of the trailing point-to-point chunk (0 unless bubble filling). */
int optcc_plan_segments(const optcc_plan_t *plan, int64_t *offset, int64_t *length,
                        int64_t *p2p_length);

/* The paper's stage of a flow.  Sec. 4.1 splits every section's AllReduce
 * into four NIC stages: S1 reduce-scatter over the healthy ring, S2 upload
 * to the straggler, S3 download from the straggler, S4 allgather over the
 * healthy ring (ordering 2 runs them S3-S1-S4-S2, so S3 is then the
 * straggler's raw value going out first).  Bubble filling enlarges the S2
 * and S3 flows with a point-to-point chunk (App. C), so its up and down
 * flows carry S2 and S3.  App. E adds the NVLink phases N1 collect, N2
 * distribute or fold, N3 collect or copy back, N4 distribute around them.
 * Stage of each executor slot:
 *   one GPU per server:   slot 0 S3, 1 S1, 2 S2, 3 S3, 4 S4, 5 S2
 *   several per server:   slot 0 N3, 1 N1, 2 S3, 3 S1, 4 S2, 5 N2, 6 N3,
 *                         7 S3, 8 S4, 9 N4, 10 S2, 11 N2 */
#define OPTCC_STAGE_S1 1
#define OPTCC_STAGE_S2 2
#define OPTCC_STAGE_S3 3
#define OPTCC_STAGE_S4 4
#define OPTCC_STAGE_N1 5
#define OPTCC_STAGE_N2 6
#define OPTCC_STAGE_N3 7
#define OPTCC_STAGE_N4 8

/* One flow: one section (or one bubble-filling chunk) moved from one rank
 * to another (Sec. 4.1's unit of transfer; App. E
 * adds NVLink flows between the GPUs of one server).  A step is one
 * destination write: a reduce step with several sources has one flow per
 * source, all with the same step index. */
typedef struct {
  int32_t slot;    /* 0..num_slots-1, see optcc_allreduce_emulate_slots */
  int32_t segment; /* 0..num_segments-1 */
  int32_t section; /* 0..P'-1, or -1 for the point-to-point chunk */
  int32_t op;      /* 0 copy, 1 reduce (dst += src) */
  int32_t src, dst;
  int32_t stage;   /* OPTCC_STAGE_*: the paper's stage the flow belongs to */
  int32_t hop;     /* position of the step among its section's steps in this
                      slot, from 0 (the hop along a chain: S1 and S4, the
                      NVLink rings) */
  int64_t step;    /* index of the step: the sources of a multi-source reduce
                      share it and are listed in accumulation order */
  int64_t offset, length; /* element range */
} optcc_flow_t;

/* Number of flows, and the flows in execution order (slot, segment, section,
 * hop).  get_flows writes min(cap, total) entries and returns the total, or a
 * negative status. */
int64_t optcc_plan_num_flows(const optcc_plan_t *plan);
int64_t optcc_plan_get_flows(const optcc_plan_t *plan, optcc_flow_t *out, int64_t cap);

/*
 * optcc_plan_traffic - algorithmic HBM bytes of one emulation call over
 * [slot_begin, slot_end) with `launches` as above, for `dtype`: the loads the
 * executor issues (each input value once, plus, per launch, the state the
 * launch starts from) into *read_bytes and one write per step into
 * *write_bytes.  Partial sums a step hands to the next step of the same
 * section inside one launch stay in registers and are not counted as reads.
 * Errors: OPTCC_EINVAL (NULL pointers, unknown dtype, bad slot range).
 */
int optcc_plan_traffic(const optcc_plan_t *plan, optcc_dtype_t dtype, int slot_begin,
                       int slot_end, int launches, int64_t *read_bytes,
                       int64_t *write_bytes);

/*
 * optcc_plan_timeline - evaluate the plan's schedule in the paper's network
 * model: start and finish time of every flow (in optcc_plan_get_flows order)
 * and the makespan, in the unit of optcc_model_time.  Model (Sec. 3, Sec. 4.1,
 * App. B.1): every rank has one send and one receive port, each carrying one
 * flow at a time (full duplex); a flow of len elements between ranks a and b
 * lasts len * max(l_a, l_b); a flow starts after the earlier steps of its
 * section that wrote its source's or its destination's range.
 *   - one GPU per server: the paper's pattern overlay (Sec. 4.2, App. C,
 *     App. D) as an explicit timetable of parallel bodies of P' + m - 1
 *     windows: straggler s_i (worst first) receives from R[w-i+1] and sends to
 *     R[w-i+2] in window w, every ring edge carries hop h of its chains in the
 *     h-th window it is free, and each stage of a segment sits in the body
 *     its pattern gives (one straggler: A and B from body 4q, C and D one body
 *     later, k + 1 bodies; several: B, D, A', C' in k + 4 bodies; bubble
 *     filling in the straggler windows).  With equal sections the windowed
 *     timetable takes exactly the closed forms of Sec. 4.3 and App. C, and
 *     App. D's body count.  The times returned run that timetable without
 *     window boundaries: each port takes its flows in the timetable's order,
 *     each as soon as both ports and its data are ready (never later).
 *     Without straggler: the ring, one hop per window, T0 exactly.
 *   - several GPUs per server (App. E, whose eight-row overlay is given only
 *     as figures): work-conserving list scheduling in flow order and in
 *     groups of eight segments per part, the shorter kept; a flow between
 *     two GPUs of one server runs on their NVLink ports at (g-1) times NIC
 *     speed (len/(g-1)).
 * start/finish may be NULL when cap = 0.  Errors: OPTCC_EINVAL,
 * OPTCC_EUNSUPPORTED (more than 2^26 flows), OPTCC_ENOMEM.
 */
int optcc_plan_timeline(const optcc_plan_t *plan, double *start, double *finish, int64_t cap,
                        double *makespan);

#ifdef __cplusplus
}
#endif

#endif /* OPTCC_H */
