/*
 * ar_plan.h -- C ABI of the MI355X AllReduce-plan executor.
 *
 * The library executes AllReduce plans in the sense of "Revisiting the Time
 * Cost Model of AllReduce" (GenModel / GenTree, arXiv 2409.04202) for n
 * emulated processors whose buffers of N elements all live in the memory of
 * one GPU.
 *
 *   AllReduce: every processor ends with the element-wise sum of all
 *   processors' data (Section 1; Section 2.1).  A *plan* is an ordering of
 *   data-movement and reduce steps (Section 2.1).  The ReduceScatter /
 *   AllGather plans split the data into n blocks, each processor reduces one
 *   share, then the shares are sent back to everyone (Section 2.1).
 *
 * A plan is expanded on the host into an explicit list of steps grouped in
 * phases.  A step is
 *
 *   reduce:  x_dst[b, e) <- x_srcs[0][b, e) + ... + x_srcs[k-1][b, e),
 *            folded left to right (the k-way sum of Section 3.1, which costs
 *            k reads and one write per element, the memory term of GenModel)
 *   copy:    x_dst[b, e) <- x_src[b, e)
 *
 * Every step of a phase reads the buffers as they were when the phase
 * started; the library checks at creation that no step of a phase reads or
 * writes a range another step of the same phase writes, so the steps of a
 * phase may run in any order or all at once.  Phases run in order.
 *
 * Arithmetic (fixed, so a plan has one exact result):
 *   AR_F32   IEEE binary32 adds, round to nearest even, no contraction,
 *            denormals kept, in the step's source order;
 *   AR_I32   two's-complement wrap-around adds;
 *   AR_BF16  buffers hold bfloat16; each reduce step widens its inputs to
 *            fp32, folds them in fp32 in source order and rounds the result
 *            once to bf16 (round to nearest even).
 *
 * Conventions for every call:
 *   - Every function returns an ar_status; AR_OK is 0.  No C++ exception
 *     crosses this interface.  On failure a description is available from
 *     ar_last_error() (per thread, valid until the next call on the thread).
 *   - Out-parameters are written only on success; on failure a plan/timer
 *     out-pointer is set to NULL.
 *   - Plan creation and introspection make no GPU call and work without a
 *     GPU.  Execution needs a gfx950 device.
 */
#ifndef AR_PLAN_H
#define AR_PLAN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum ar_status {
    AR_OK = 0,
    AR_ERR_INVALID_ARG = 1,  /* bad pointer, size, index or plan shape      */
    AR_ERR_UNSUPPORTED = 2,  /* valid request the library does not handle    */
    AR_ERR_OOM = 3,          /* host or device allocation failed             */
    AR_ERR_HIP = 4,          /* a HIP runtime call or kernel launch failed   */
    AR_ERR_INTERNAL = 5
} ar_status;

typedef enum ar_dtype { AR_F32 = 0, AR_I32 = 1, AR_BF16 = 2 } ar_dtype;

/* Plan kinds (Section 2.1 and Section 3.3, Tables 1 and 2):
 *  AR_RING  Ring: 2(n-1) steps; in step j processor i receives block
 *           (i - j) mod n from processor i - 1 and, in the first n - 1 steps,
 *           adds its own block to it (reduce step with srcs {i, i-1}); in
 *           the last n - 1 steps it stores it (copy).  After the
 *           ReduceScatter half processor i owns block (i + 2) mod n.
 *  AR_RHD   Recursive halving-doubling: for n a power of two, in halving
 *           step j processor r pairs with r XOR 2^j, keeps the lower half of
 *           the range it holds if bit j of r is 0 and the upper half
 *           otherwise, and reduces it over the pair (2^-(j+1) of the data in
 *           step j); the doubling steps run the halving steps backwards as
 *           copies.  Otherwise, with p the largest power of two below n, two
 *           steps are added (2 ceil(log2 n) in all): processor q >= p first
 *           reduces its whole buffer into q - p, ranks 0..p-1 run the
 *           power-of-two plan on p blocks, and q finally copies the result
 *           from q - p (ranks >= p then own nothing).
 *  AR_CPS   Co-located PS: processor p reduces block p over all n inputs in
 *           one n-way step, then the n - 1 others copy it.
 *  AR_TREE  Hierarchical co-located PS on a symmetric tree, i.e. the GenTree
 *           basic sub-plan of Algorithm 1 for a tree whose switches at level
 *           l all have fanin[l] children (fanin[0] = servers per bottom
 *           switch).  n must equal the product of the fan-ins.  Rank r has
 *           digits d_l = (r / (f_0...f_{l-1})) mod f_l.  ReduceScatter level
 *           l reduces, over the f_l ranks that differ from r only in digit
 *           l (ascending), the part of r's previous range that r owns;
 *           AllGather runs the levels in reverse as copies.  Rank r owns
 *           after level l the n/(f_0...f_l) blocks starting at block
 *           o_l(r) * n/(f_0...f_l), o_l = o_{l-1} * f_l + d_l, o_{-1} = 0
 *           (the bottom-up placement of Algorithm 1).  Levels with fan-in 1
 *           add no phase.
 *  AR_RB    Reduce-Broadcast (parameter server): rank 0 reduces all n full
 *           buffers in one n-way step, then the others copy the result.
 *
 * Block split: block b of the n-way split covers [b*q + min(b, rem),
 * (b+1)*q + min(b+1, rem)) with q = N / n, rem = N mod n (the floor share,
 * one more for the first rem blocks, as in Algorithm 1).
 */
typedef enum ar_kind {
    AR_RING = 0, AR_RHD = 1, AR_CPS = 2, AR_TREE = 3, AR_RB = 4,
    AR_GENTREE = 5   /* only through ar_plan_create_gentree */
} ar_kind;

typedef enum ar_op { AR_OP_REDUCE = 0, AR_OP_COPY = 1 } ar_op;

typedef struct ar_topology {
    int32_t kind;          /* ar_kind                                       */
    int32_t num_levels;    /* AR_TREE: number of fan-in levels (>= 1)       */
    const int32_t* fanin;  /* AR_TREE: fanin[0..num_levels), innermost first;
                              ignored for other kinds; read during the call */
} ar_topology;

typedef struct ar_step {
    int32_t phase;         /* 0-based; phases execute in increasing order   */
    int32_t op;            /* ar_op                                         */
    int32_t dst;           /* processor written, 0 <= dst < n               */
    int32_t nsrc;          /* number of sources (copy: exactly 1)           */
    const int32_t* srcs;   /* nsrc processor indices, folded in this order  */
    int64_t begin;         /* element range [begin, end), 0 <= b <= e <= N  */
    int64_t end;
} ar_step;

typedef struct ar_plan ar_plan;
typedef struct ar_timer ar_timer;

/* ---------------------------------------------------------------- plans */

/* Expand a plan of kind topo->kind for n processors of N elements of dtype.
 * n >= 1, N >= 0 (n = 1 or N = 0 gives a plan with no work; N < n gives
 * empty blocks, which are kept as empty steps).  n <= 65536.
 * Errors: AR_ERR_INVALID_ARG (NULL out/topo, n < 1, N < 0, unknown dtype or
 * kind, tree fan-in < 1, missing fan-ins or product != n, N * element size
 * overflowing int64), AR_ERR_UNSUPPORTED (more than 2^26 steps), AR_ERR_OOM.  The plan owns all its memory; free it with ar_plan_destroy. */
ar_status ar_plan_create(int32_t n, int64_t N, int32_t dtype,
                         const ar_topology* topo, ar_plan** out);

/* GenTree's basic plan on an arbitrary tree (Section 4.2, Algorithm 1).  The
 * tree is given in preorder: nchild[i] is the number of children of node i
 * (0 for a server), for num_nodes nodes; the list must describe exactly one
 * tree.  Servers are the processors, numbered in that (depth-first) order;
 * n is their number (<= 65536).
 *   Placement: bottom-up, after the ReduceScatter below a switch every
 *   server under it owns floor(n / s) of the n blocks, s being the number of
 *   servers under the switch, and the first (n mod s) in child order own one
 *   more; a server takes, in order, the first blocks of its own list (the
 *   blocks it owned under its child; a server child's list is every block)
 *   that no earlier server under the switch took.  Where this leaves a
 *   block unplaced (it can on asymmetric trees), the block goes to the
 *   server holding it in the first child that holds it.
 *   Steps: each switch reduces every block placed on a server over one
 *   holder per child (in child order) -- a co-located PS when the children
 *   are alike, the asymmetric co-located PS otherwise -- with consecutive
 *   blocks of one server and the same holders in one step; switches of one
 *   height share a phase; the AllGather reverses the ReduceScatter level by
 *   level.  On a symmetric tree this is exactly AR_TREE.  A switch with one
 *   child adds nothing.  A plan choice inside a switch (e.g. m x k
 *   hierarchical CPS) is expressed as an extra level of switches.
 * ar_plan_owner gives the root-level owner range, or AR_ERR_UNSUPPORTED when
 * a processor's blocks there are not contiguous.  Errors: AR_ERR_INVALID_ARG
 * (malformed list, N < 0, unknown dtype, more than 65536 servers),
 * AR_ERR_UNSUPPORTED (children x servers summed over the nodes > 2^28). */
ar_status ar_plan_create_gentree(int64_t N, int32_t dtype, int32_t num_nodes,
                                 const int32_t* nchild, ar_plan** out);

/* Build a plan from an explicit step list (any order; steps are grouped by
 * phase, phases must be numbered 0..P-1 without gaps).  Each step is
 * validated (indices, ranges, copy has one source, reduce at least one) and
 * each phase is checked for hazards: AR_ERR_INVALID_ARG if a step writes a
 * range that another step of the same phase reads or writes.  The arrays
 * are copied; the caller keeps ownership of `steps`.  Such a plan has no
 * owner map (ar_plan_owner returns AR_ERR_UNSUPPORTED). */
ar_status ar_plan_create_custom(int32_t n, int64_t N, int32_t dtype,
                                const ar_step* steps, int64_t nsteps,
                                ar_plan** out);

/* Free a plan and the device memory it holds.  NULL is a no-op.  Must not be
 * called while an execution of the plan may still be running. */
ar_status ar_plan_destroy(ar_plan* plan);

/* ------------------------------------------------------------ execution */

/* Execute the plan in place on bufs[0..n): n device pointers on the current
 * device, each to at least N * element-size bytes, pairwise non-overlapping
 * (checked on the host: AR_ERR_INVALID_ARG for NULL or overlapping
 * buffers).  `stream` is a hipStream_t (NULL = the default stream).  The
 * call is asynchronous and stream-ordered: it enqueues about one kernel
 * launch per phase (see ar_plan_num_launches) and returns; when the stream
 * reaches that point every buffer holds the AllReduce result, bit for bit
 * the result of running the steps phase by phase as listed.  The
 * pointer array is read during the call only.  Any pointer alignment works;
 * 16-byte-aligned buffers take the vector path.  The first call on a device
 * uploads the plan's tile tables; the first call with a new buffer set
 * builds that set's step records (each executed step's range and resolved
 * buffer pointers, (4 + k + d) * 8 bytes rounded up to 16 for a step with
 * k sources and d destinations) on the host and uploads them; the plan keeps
 * the records of its 4 most recently used buffer sets per device (device and
 * pinned host memory owned by the plan), so repeated executes on the same
 * buffers only launch kernels.  Such a call may therefore be captured in a
 * HIP graph (stream capture records its kernel launches only); the first
 * call on a device or with a new buffer set allocates, copies and records
 * an event, so it must run before capture starts.  Executions of one plan
 * must be ordered (one stream, or synchronised).  Distinct plans are
 * independent.  Errors: AR_ERR_INVALID_ARG, AR_ERR_OOM, AR_ERR_HIP. */
ar_status ar_plan_execute(ar_plan* plan, void* const* bufs, void* stream);

/* Same, with buffer p at (char*)base + p * stride_bytes; stride_bytes must
 * be >= N * element size. */
ar_status ar_plan_execute_strided(ar_plan* plan, void* base,
                                  int64_t stride_bytes, void* stream);

/* ar_plan_execute that also records a pair of HIP events on `stream`
 * around every kernel launch into `timer` (appended; AR_ERR_INVALID_ARG
 * when the timer is full).  Results are read with ar_timer_read. */
ar_status ar_plan_execute_timed(ar_plan* plan, void* const* bufs,
                                void* stream, ar_timer* timer);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * ar_plan_execute without any device allocation.  Same arguments, same
 * launches and the same result bits as ar_plan_execute; no call makes a
 * device allocation or calls hipMalloc, hipFree or any other allocating HIP
 * routine.  The plan's device-side tables and the step records of the buffer
 * set (the staging ar_plan_execute allocates per plan) live instead in one
 * array of AR_NOALLOC_MAX_BYTES bytes that the library holds on every device
 * it runs on, from that device's first such call until the process ends.
 *   - Every call on a device shares that device's array, which keeps the last
 *     call's contents: the call copies the plan's tables and records into it
 *     (hipMemcpyAsync from host memory the plan owns, on `stream`) unless the
 *     last call on the device used the same plan, options and buffer set.
 *     Calls that may overlap on one device (other streams, other host
 *     threads without ordering) race on the array and must be ordered by
 *     the caller.
 *   - The first call with a plan (and after each option change) builds the
 *     plan's host-side image of the tables (host memory, freed with the
 *     plan).
 *   - A call whose plan and buffer set are those of the last call on the
 *     device enqueues kernel launches only; so a caller capturing the call
 *     into a HIP graph makes one uncaptured call with the same plan and
 *     buffers first, and does not interleave calls with other plans or
 *     buffer sets on the device between the replays.
 *   - AR_ERR_UNSUPPORTED, with the size in ar_last_error(), when the plan's
 *     tables and records exceed AR_NOALLOC_MAX_BYTES (their size grows with
 *     the number of steps and, for a resident launch, with N: 40 bytes per
 *     256-element tile; RHD n = 8 at 2^26 fp32 takes about 10 MiB).
 *   Errors otherwise as ar_plan_execute. */
#define AR_NOALLOC_MAX_BYTES (32u << 20)
ar_status ar_plan_execute_noalloc(ar_plan* plan, void* const* bufs, void* stream);

/* Executor options (ar_plan_set_option).
 *  AR_OPT_FUSE (default 1): let the executor merge steps where that removes
 *  memory traffic without changing any result bit:
 *   - copies of one phase that read the same range of the same buffer run
 *     as one step that reads it once and stores it to every destination;
 *   - a copy of a range that a reduce step of the previous phase has just
 *     produced is absorbed into that reduce step, which stores its result to
 *     the copy's destination too (where the last ReduceScatter phase meets
 *     the first AllGather phase), provided no other step of that phase
 *     touches the absorbed destination range.
 *  With 0, every plan step runs as listed, one launch per phase and source
 *  count.  Changing an option drops the plan's device state; it must not
 *  be done while an execution of the plan may still be running. */
/*  AR_OPT_SLICE (default 2): sliced launches.  A sliced launch runs a run of
 *  consecutive phases in one launch in which each wavefront carries a fixed
 *  tile of element positions through those phases in order, running each
 *  step on its tile, so that no barrier or launch separates the phases
 *  (every step is element-wise and the steps of a phase are independent, so
 *  a position only depends on what earlier phases did at that position).
 *  Every step still reads and writes the buffers in memory as listed.
 *  0: never; 1: the whole plan as one sliced launch whenever possible;
 *  2: the runs of phases a cost model predicts faster as sliced launches,
 *  among phases that each write at most 256 MiB (what one phase hands to the
 *  next then fits the last-level cache either way) for a plain sliced launch,
 *  of any size for a resident one.  A run is possible when
 *  every boundary of its steps is a multiple of 16 bytes; sliced launches
 *  are used only with 16-byte aligned buffers (otherwise every phase runs
 *  as its phase launches, those reported with AR_OPT_SLICE = 0). */
/*  AR_OPT_RESIDENT (default 1): a sliced launch may run resident instead:
 *  each workgroup keeps its tile of element positions in on-chip memory
 *  (LDS) for the whole run, loading each buffer's tile once, before the
 *  run's first read of it, and storing each tile the run writes once, with
 *  its final value, so that the run's intermediate values stay on chip.
 *  With n <= 64 buffers the tile of every buffer has its own LDS row; with
 *  more (streamed form) the run's values share up to 64 LDS slots, each
 *  value held from its load or computation to its last use, the folds
 *  computed depth first and the loads issued ahead.  Every step still folds
 *  the same values with the plan's sources in their listed order, so
 *  results are the same bits.  With AR_OPT_SLICE = 2 the cost model picks
 *  the plain or the resident form per run (n <= 64), or (n > 64) runs the
 *  whole plan as one streamed launch when it predicts that faster than the
 *  runs it chose; with AR_OPT_SLICE = 1 the whole plan runs resident.
 *  0: sliced launches always run plain. */
typedef enum ar_option { AR_OPT_FUSE = 0, AR_OPT_SLICE = 1, AR_OPT_RESIDENT = 2 } ar_option;
ar_status ar_plan_set_option(ar_plan* plan, int32_t option, int64_t value);

/* The kernel launches one execution on 16-byte aligned buffers issues (host
 * only, no GPU call): their number, and for launch i the plan phase its
 * steps come from (-1 for a sliced launch, -2 for a resident one, -3 for a
 * streamed resident one), their
 * source count (the
 * largest, for a sliced launch), the most destinations any of its
 * steps stores to, its number of steps and its algorithmic bytes:
 * (k + destinations) * len * e summed over its steps (each source read
 * once, each destination written once); for a resident launch, the bytes
 * of the buffer tiles it loads and stores (each once; a whole AllReduce
 * run resident moves 2 * n * N * e).  Any out-pointer may be NULL. */
ar_status ar_plan_num_launches(const ar_plan* plan, int32_t* count);
ar_status ar_plan_launch_info(const ar_plan* plan, int32_t i, int32_t* phase,
                              int32_t* nsrc, int32_t* max_dst,
                              int64_t* num_steps, int64_t* bytes);

/* The kernel launch i (as in ar_plan_launch_info) runs on 16-byte aligned
 * buffers: AR_KERNEL_PHASE, one wavefront per wave tile of its steps;
 * AR_KERNEL_SPLIT, a workgroup per wave tile, each wavefront storing the
 * folded tile to a share of the step's destinations (a launch of few tiles
 * whose steps store to many buffers; on unaligned buffers it runs as
 * AR_KERNEL_PHASE); AR_KERNEL_SLICED, AR_KERNEL_RESIDENT and AR_KERNEL_STREAM
 * for the sliced, resident and streamed resident launches (phase -1, -2 and
 * -3 above).  Host only, no GPU call.  AR_ERR_INVALID_ARG for a NULL plan or
 * kernel, or i out of range. */
typedef enum ar_kernel {
    AR_KERNEL_PHASE = 0, AR_KERNEL_SPLIT = 1, AR_KERNEL_SLICED = 2,
    AR_KERNEL_RESIDENT = 3, AR_KERNEL_STREAM = 4
} ar_kernel;
ar_status ar_plan_launch_kernel(const ar_plan* plan, int32_t i, int32_t* kernel);

/* -------------------------------------------------------- introspection */

/* Shape of the plan: any out-pointer may be NULL. */
ar_status ar_plan_info(const ar_plan* plan, int32_t* n, int64_t* N,
                       int32_t* dtype, int32_t* num_phases,
                       int64_t* num_steps);

/* Step i (0 <= i < num_steps) in execution order (by phase).  out->srcs
 * points into the plan and stays valid until ar_plan_destroy. */
ar_status ar_plan_get_step(const ar_plan* plan, int64_t i, ar_step* out);

/* Phase p: `op` is AR_OP_REDUCE if any step reduces, else AR_OP_COPY;
 * steps [first_step, first_step + num_steps); `bytes` is the phase's
 * algorithmic traffic: (k + 1) * len * e per k-way reduce step, 2 * len * e
 * per copy step (GenModel's memory term for reduces, Section 3.1; a copy
 * reads and writes each element once).  Any out-pointer may be NULL. */
ar_status ar_plan_phase_info(const ar_plan* plan, int32_t phase, int32_t* op,
                             int64_t* first_step, int64_t* num_steps,
                             int64_t* bytes);

/* Range [begin, end) that processor p holds fully reduced once the
 * ReduceScatter phases are done (empty for processors that own nothing,
 * e.g. non-root ranks of AR_RB).  AR_ERR_UNSUPPORTED for custom plans. */
ar_status ar_plan_owner(const ar_plan* plan, int32_t p, int64_t* begin,
                        int64_t* end);

/* Total algorithmic bytes of all reduce steps and of all copy steps (same
 * rule as ar_plan_phase_info).  Either out-pointer may be NULL. */
ar_status ar_plan_bytes(const ar_plan* plan, int64_t* reduce_bytes,
                        int64_t* copy_bytes);

/* ------------------------------------------------------------- GenModel */

/* GenModel (Section 3) with the terms one GPU has, for predicting a plan's
 * time and choosing a plan (Section 3.4 fits the model from co-located PS
 * runs; Algorithm 2 picks the plan of smallest predicted time).  The
 * predicted time of a plan is the dot product of AR_GENMODEL_TERMS
 * parameters with its terms:
 *   terms[0] A   rounds: the plan's phases (the alpha term of Tables 1-2);
 *   terms[1] K   the sum over phases of the largest source count of a step
 *                of the phase (a k-way step waits for k dependent loads per
 *                element: a per-phase latency growing with k);
 *   terms[2] Dh, terms[3] Dc   the reduce steps' memory traffic, (k + 1) *
 *                len * e per k-way step (the delta term, Section 3.1), split
 *                by where each access is served;
 *   terms[4] Bh, terms[5] Bc   the copy steps' traffic, 2 * len * e each,
 *                split the same way.
 * An access is counted as served from the last-level cache of cache_bytes
 * (the "c" terms) when the plan's whole footprint n * N * e fits it, when it
 * reads a range an earlier step of the same phase read, or when it reads a
 * range the previous phase wrote and that phase wrote at most cache_bytes;
 * otherwise from HBM (the "h" terms).  Host only, no GPU call.  Errors:
 * AR_ERR_INVALID_ARG (NULL argument, cache_bytes < 0). */
#define AR_GENMODEL_TERMS 6
ar_status ar_genmodel_terms(const ar_plan* plan, int64_t cache_bytes, double* terms);

/* The plan of smallest predicted time (params . terms, with the terms of
 * ar_genmodel_terms for cache_bytes) for n processors of N elements of
 * dtype, among: Ring, co-located PS, RHD, and AR_TREE for every ordered
 * factorisation of n into 2..max_levels fan-ins >= 2 (innermost first; the
 * factorisations in increasing order of their first fan-in, depth first).
 * Ties go to the earlier candidate.  Candidates too large to expand are
 * skipped.  Out: *kind (ar_kind), *num_levels and fanin[0..*num_levels)
 * (fanin has room for max_levels entries; 0 levels for the non-tree
 * kinds), *seconds the predicted time.  Host only.  Errors:
 * AR_ERR_INVALID_ARG (NULL argument, n < 1, N < 0, cache_bytes < 0,
 * max_levels outside [2, 32], unknown dtype), AR_ERR_UNSUPPORTED (no
 * candidate could be expanded), AR_ERR_OOM. */
ar_status ar_genmodel_select(int32_t n, int64_t N, int32_t dtype, const double* params,
                             int64_t cache_bytes, int32_t max_levels, int32_t* kind,
                             int32_t* num_levels, int32_t* fanin, double* seconds);

/* The same terms with several cache tiers: cache_bytes[0..tiers) the tiers'
 * sizes, strictly decreasing (say the last-level cache, then the L2 caches
 * together), 1 <= tiers <= AR_GENMODEL_MAX_TIERS.  An access is served from
 * the smallest tier under whose size the rule of ar_genmodel_terms classes
 * it as cached, else from HBM.  terms has 4 + 2 * tiers entries: A, K, the
 * reduce bytes from HBM, from tier 0, ..., from tier tiers-1, then the copy
 * bytes the same way.  With one tier the terms are ar_genmodel_terms'.  Host
 * only.  Errors: AR_ERR_INVALID_ARG (NULL plan or terms, a bad tier count or
 * list), AR_ERR_OOM. */
#define AR_GENMODEL_MAX_TIERS 4
ar_status ar_genmodel_terms_tiered(const ar_plan* plan, int32_t tiers, const int64_t* cache_bytes,
                                   double* terms);

/* ar_genmodel_select with the tiered terms: params has 4 + 2 * tiers
 * entries, one per term of ar_genmodel_terms_tiered.  ar_genmodel_select is
 * this with one tier.  Errors as ar_genmodel_select's, and a bad tier count
 * or list is AR_ERR_INVALID_ARG. */
ar_status ar_genmodel_select_tiered(int32_t n, int64_t N, int32_t dtype, const double* params,
                                    int32_t tiers, const int64_t* cache_bytes, int32_t max_levels,
                                    int32_t* kind, int32_t* num_levels, int32_t* fanin,
                                    double* seconds);

/* --------------------------------------------------------------- timing */

/* A timer holds up to `capacity` launch records (capacity >= 1).  Its HIP
 * events are created on first use, on the device current at that time. */
ar_status ar_timer_create(int64_t capacity, ar_timer** out);
ar_status ar_timer_reset(ar_timer* timer);          /* forget all records */
/* Wait for the recorded events and copy out up to `cap` records: launch[i]
 * is the index (as in ar_plan_launch_info) of the launch record i timed and
 * ms[i] its duration in milliseconds (begin-to-end event time on the launch
 * stream).  *count receives the number of records copied.  launch or ms may
 * be NULL. */
ar_status ar_timer_read(ar_timer* timer, int64_t cap, int64_t* count,
                        int32_t* launch, float* ms);
ar_status ar_timer_destroy(ar_timer* timer);        /* NULL is a no-op */

/* -------------------------------------------------------------- errors */

const char* ar_status_string(ar_status s);  /* static string, never NULL   */
const char* ar_last_error(void);            /* "" when there is none       */

#ifdef __cplusplus
}
#endif

#endif /* AR_PLAN_H */
