/*
 * bfs.h -- barrier-free synchronization of loop-nested multi-engine kernels
 * on one MI355X (gfx950) GPU.
 *
 * The library takes what the paper's allocation pass takes -- a structured
 * program (a tree of loops over blocks of per-engine instructions) plus a
 * dependency graph of (producer, consumer, offset) triples (Section 1 and
 * Appendix A.1) -- and produces the synchronization that enforces it:
 *
 *   - barrier-free mode (Sections 5.1-5.5): every dependency becomes one wait
 *     on a monotone counter owned by (producer's loop, producer's engine),
 *     against the threshold
 *         isGT(rhat_S, k) * max(N * expr - (N - K), 0)           (Eq. 2, Eq. 5)
 *     with expr = r_P - k when the producer sits directly in the shared loop
 *     S (case C1), and expr = r_P when it is nested deeper (C2: forward,
 *     k = 0; C3: backward, k = 1) (Section 5.2).  r_l counts every entry
 *     (iteration start) of loop l and is never reset; rhat_l counts the
 *     entries in the current trip and is reset when l's loop statement is
 *     reached (Section 5.1).
 *   - barrier mode (Section 3.4): all engines synchronize before every
 *     non-top loop statement and at the end of every iteration of a non-top
 *     loop (drain, barrier, counter reset, barrier); inside a region a
 *     consumer waits for the producer's static ordinal on its engine.
 *
 * On the GPU an engine is a group of wavefronts of one workgroup; a counter
 * is a 32-bit LDS word per (counter slot, producer wave); the loop registers
 * live in scalar registers.  The datapath is a hand-written HIP kernel
 * family selected by bfs_program.kernel.
 *
 * Conventions for every entry point:
 *   - Returns a bfs_status.  Out-parameters are written only on BFS_OK.
 *     bfs_last_error() then describes the most recent failure of the calling
 *     thread.
 *   - Input descriptors are caller-owned and copied; the caller may free them
 *     when the call returns.
 *   - Device pointers are caller-owned and must stay valid until the work
 *     enqueued on the stream has completed.
 */
#ifndef BFS_H
#define BFS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

struct ihipStream_t;                      /* hipStream_t is struct ihipStream_t* */

typedef struct bfs_plan bfs_plan;         /* opaque, library-owned */

typedef enum {
  BFS_OK = 0,
  BFS_E_INVALID = 1,          /* malformed program, bad id, bad argument */
  BFS_E_ORDER = 2,            /* producer not before consumer where offset 0 requires it */
  BFS_E_NOT_ALLOCATABLE = 3,  /* dependency outside the cases of Section 5.2 */
  BFS_E_RESOURCE = 4,         /* exceeds LDS / wave / counter limits */
  BFS_E_DEVICE = 5,           /* HIP runtime error */
  BFS_E_DEADLOCK = 6,         /* a device wait exceeded the watchdog */
  BFS_E_UNSUPPORTED = 7       /* program does not match the kernel family */
} bfs_status;

typedef enum { BFS_MODE_BARRIER_FREE = 0, BFS_MODE_BARRIER = 1 } bfs_mode;

/* Flags of bfs_plan_create.
 *
 * BFS_PLAN_BARRIER_FALLBACK: a dependency outside the allocatable cases of
 * Section 5.2 (a producer nested below the shared loop S with an offset other
 * than 0 forward or 1 backward) is kept instead of failing with
 * BFS_E_NOT_ALLOCATABLE and falls back to the barrier scheme, as Section 5.2
 * prescribes: every engine drains its in-flight instructions and meets the
 * others at the end of every iteration of S (no counter is reset, so the
 * monotone semaphores of the other dependencies stay valid).  Such a
 * dependency gets no counter and no wait.  When S is the top-level loop the
 * dependency is never owed (its single iteration has rhat_S = 1 <= k) and no
 * barrier is placed.  Only the interpreter family executes these barriers;
 * bfs_run of another family's plan that has one returns BFS_E_UNSUPPORTED. */
#define BFS_PLAN_BARRIER_FALLBACK 1u

/* Semaphore granularity (Section 5.4 per-instruction, Section 5.5 per-loop,
 * Section 6.1 per-engine).
 *
 * BFS_ALLOC_PER_ENGINE: one counter per producer engine, incremented at the
 * retirement of every instruction of that engine; in-order retirement makes
 * its value the number of the engine's instructions retired so far.  A
 * dependency's threshold is that counter's value right after the producer
 * instance Eq. 1 requires: the number of the producer engine's instructions
 * up to that instance in program order.  Section 6.1 gives it as a sum of
 * loop-entry terms along the producer's path and caches the outer partial
 * sums; here the sum is carried incrementally, in its cached form, by the
 * consumer engine, which walks every loop: it keeps, per producer engine,
 * the running count of that engine's instructions up to its own position
 * (program-order counts of each block, added as it walks), and takes a
 * snapshot of it at the producer's position.  A dependency at offset k on
 * the producer's own loop S keeps the snapshots of the last k + 1
 * iterations of S (indexed by r_S); a producer nested below S (C2, C3) keeps
 * the latest one.  The threshold is the snapshot of iteration r_S - k, or
 * the latest one, under the isGT(rhat_S, k) mask of Eq. 5 (no mask for a
 * linearized offset, which reads r_S over all trips): one register read and
 * the mask per issue.  Exact wherever per-loop counters are (the same Eq. 1
 * requirement, certified on a coarser counter).  Barrier-free plans of the
 * interpreter family only; other families return BFS_E_UNSUPPORTED at
 * bfs_run. */
typedef enum { BFS_ALLOC_PER_LOOP = 0, BFS_ALLOC_PER_INSTR = 1, BFS_ALLOC_PER_ENGINE = 2 } bfs_alloc;

/* Datapath kernel families. */
typedef enum {
  BFS_KERNEL_INTERP = 0,      /* generic tile-machine interpreter, one wave per engine */
  BFS_KERNEL_STREAM3 = 1,     /* load / add / store stream over a 3-level nest */
  BFS_KERNEL_GEMM = 2,        /* bf16 GEMM + bias + GELU, load / MFMA / epilogue engines */
  BFS_KERNEL_ATTN = 3,        /* variable-length attention forward */
  BFS_KERNEL_MOE = 4,         /* MoE grouped GEMM with runtime per-expert trip counts */
  BFS_KERNEL_RMSNORM = 5,     /* RMSNorm + per-row FP8 (E4M3) quantization, load / vector / store engines */
  BFS_KERNEL_ADAMW = 6,       /* AdamW step over fp32 parameter chunks, load / vector / store engines */
  BFS_KERNEL_CHAIN = 7        /* two-engine chain: tiles loaded into an LDS ring, scaled and accumulated */
} bfs_kernel;

/*
 * The program (the statement tree of Section 7.1 with the block streams of
 * Appendix A.1), as flat int32 arrays:
 *
 *   loops        loop 0 is the top level (parent -1, runs once).  Every other
 *                loop l has loop_parent[l] and appears exactly once in its
 *                parent's body.  loop_is_cond[l] marks a conditional (a loop
 *                whose trip count is 0 or 1).
 *   body         CSR: loop l's body is items body_off[l] .. body_off[l+1]-1,
 *                in program order; item i is a block (body_kind 0) or a loop
 *                (body_kind 1) with id body_id[i].
 *   blocks       CSR: block b lists instruction ids block_instrs[block_off[b]
 *                .. block_off[b+1]-1] in one sequential program order; each
 *                engine's stream is the projection onto that engine.
 *   instrs       instr_engine[i], instr_opcode[i] and instr_args[8*i .. 8*i+7]
 *                (datapath opcode and operands; meaning set by the family).
 *   deps         deps[3*d .. 3*d+2] = producer, consumer, offset k >= 0, with
 *                k the distance on the innermost loop enclosing both.
 *   dep_linear   NULL, or per dependency 0 (the relation of Section 4.2) or
 *                1: EXTENSION, not in the paper.  The offset counts
 *                iterations of S since the start of the workgroup, across
 *                trips of S: the consumer's iteration with monotone count
 *                r_S needs the producer's iterations up to r_S - k, also
 *                those of earlier trips (no underflow at a trip start).  It
 *                lets a ring indexed by a monotone register, (r_S - 1) % R,
 *                be protected against reuse across trip boundaries by one
 *                dependency.  Allowed only with the producer directly in S
 *                (its threshold is Eq. 5 of C1 without the isGT mask).
 *   tile machine tile_elems fp32 values per tile (multiple of 64, <= 256),
 *                ring_slots[r] slots in LDS ring r (0 = unused), n_accs
 *                accumulator tiles.
 */
typedef struct {
  int32_t kernel;                  /* bfs_kernel */
  int32_t n_engines;               /* 1..8 */
  int32_t waves_per_engine[8];
  int32_t n_loops;
  const int32_t *loop_parent;
  const int32_t *loop_is_cond;
  const int32_t *body_off;
  const int32_t *body_kind;
  const int32_t *body_id;
  int32_t n_blocks;
  const int32_t *block_off;
  const int32_t *block_instrs;
  int32_t n_instrs;
  const int32_t *instr_engine;
  const int32_t *instr_opcode;
  const int32_t *instr_args;
  int32_t n_deps;
  const int32_t *deps;
  int32_t tile_elems;
  int32_t ring_slots[4];
  int32_t n_accs;
  const int32_t *dep_linear;       /* NULL, or [n_deps]: see above */
} bfs_program;

/* One dependency's barrier-free wait (Eq. 5). */
typedef struct {
  int32_t dep;
  int32_t kase;          /* 1 = C1 (P == S), 2 = C2 (nested, forward), 3 = C3 (nested, backward),
                            4 = barrier fallback (BFS_PLAN_BARRIER_FALLBACK; counter -1, no wait,
                            ordered by the barriers at the end of every iteration of loop_S),
                            6 = linearized offset (extension, dep_linear; producer in S, no mask) */
  int32_t loop_S;        /* innermost loop enclosing producer and consumer */
  int32_t loop_P;        /* producer's parent loop */
  int32_t k;             /* offset on S */
  int32_t expr_sub;      /* k for C1, 0 for C2 / C3 */
  int32_t N, K;          /* decode of the shared counter: N instructions, producer is the K-th */
  int32_t needs_mask;    /* k > 0: multiply by isGT(rhat_S, k) */
  int32_t counter;       /* counter slot the consumer polls */
  int32_t prd_engine;
  int32_t cns_engine;
  int32_t forward;       /* producer precedes consumer in S's body */
  int32_t snap_slots;    /* BFS_ALLOC_PER_ENGINE: snapshots the consumer keeps (k + 1 when the
                            producer is directly in S, else 1; N and K are then 0); 0 otherwise */
} bfs_formula;

/* One dependency's barrier-mode wait (Section 3.4). */
typedef struct {
  int32_t dep;
  int32_t same_region;   /* 0: a barrier always separates them, no wait */
  int32_t prd_engine;
  int32_t ordinal;       /* producer's position on its engine since the last barrier */
} bfs_static_wait;

/* Resource figures (Table alloc-resources / Table alloc-sema-combined columns). */
typedef struct {
  int32_t n_counters;            /* semaphores used */
  int32_t regs_per_engine;       /* loop registers r, rhat plus the wait register; per-engine:
                                    plus the running counts and snapshots (most of any engine) */
  int32_t salu_ops_per_wait;     /* 5 per-loop, 3 per-instruction, 3 per-engine (index, mask,
                                    read), 0 barrier */
  int32_t n_waits;               /* waits emitted */
  int32_t n_sync_points;         /* barrier mode: loop statements + iteration ends in the tree;
                                    barrier-free: loops whose iteration ends carry a fallback barrier */
  int32_t n_fallback;            /* dependencies handled by the barrier fallback */
} bfs_stats;

/* Options of one launch; NULL selects the defaults. */
typedef struct {
  uint64_t watchdog_polls;       /* polls before a wait gives up (0 = default, about 1 s) */
  int32_t fault_dep;             /* test knob: dependency whose threshold is raised (-1 = none) */
  int32_t fault_delta;           /* amount added to that threshold */
  uint64_t *dev_stats;           /* NULL, or n_wg * W * 8 uint64 per-wave counters (W = waves per
                                    workgroup), in 100 MHz ticks: [0] wave run time, [1] time
                                    blocked in waits, [2] blocked waits, [3] time in barriers,
                                    [4] time waiting for own loads to land, [5] polls, [6-7] 0 */
  int32_t k_unroll;              /* GEMM family: iterations of the static-trip K loop per
                                    loop-body copy, also in instrumented launches, whose debug
                                    log then records the unrolled bodies' waits (0 or 1: none,
                                    2, 4, 8; unrolled bodies see their thresholds as fixed
                                    offsets of one loop-invariant value, the code-size versus
                                    regOp trade-off of static loops); other families ignore it.
                                    Other values: BFS_E_INVALID */
  uint32_t flags;                /* 0 or BFS_RUN_* bits below; other bits: BFS_E_INVALID */
} bfs_run_opts;

/* bfs_run_opts.flags.
 *
 * BFS_RUN_PER_INSTANCE: stream family, barrier-free, uninstrumented: every
 * trip of the innermost loop runs one instance at a time (one wait, one tile
 * moved and one counter add per instance), the loop the barrier mode runs,
 * instead of the batches of up to four consecutive instances that
 * uninstrumented launches take otherwise.  The schedule is then the same in
 * both modes and only the synchronization differs (the isolation of the
 * allocation that Section 8.2 asks for).  Other families ignore it.
 *
 * BFS_RUN_LOG_BATCHED: stream family, barrier-free, with a debug log: the
 * engines run the batched loop of uninstrumented launches and log one entry
 * per batch wait, for the instance whose threshold the batch waits for (the
 * batch's last instance, or in a pair of M iterations the last instance of
 * the trip that holds the larger threshold).  Without it an instrumented
 * launch logs every instance from the per-instance loop.  Ignored with an
 * injected fault (fault_dep >= 0), which always runs the per-instance loop. */
#define BFS_RUN_PER_INSTANCE 1u
#define BFS_RUN_LOG_BATCHED 2u

/*
 * Plan the synchronization of prog (Sections 5.2-5.5, or Section 3.4 in
 * barrier mode).  Validates the tree, classifies every dependency, assigns
 * counter slots and computes N, K and the barrier ordinals.  Host only; needs
 * no GPU.  flags: 0 or BFS_PLAN_BARRIER_FALLBACK (other bits: BFS_E_INVALID).
 * Errors: BFS_E_INVALID, BFS_E_ORDER (offset 0 with the producer not before
 * the consumer, or a nested backward producer at offset 0),
 * BFS_E_NOT_ALLOCATABLE (nested producer with another offset, without
 * BFS_PLAN_BARRIER_FALLBACK; a linearized dependency whose producer is not
 * directly in S), BFS_E_RESOURCE.
 */
bfs_status bfs_plan_create(const bfs_program *prog, bfs_mode mode, bfs_alloc alloc, uint32_t flags,
                           bfs_plan **out);

/* Formula table (one entry per dependency, in dependency order).  The array
 * is owned by the plan and valid until bfs_plan_destroy. */
bfs_status bfs_plan_formulas(const bfs_plan *plan, const bfs_formula **out, int32_t *n);

/* Barrier-mode waits (one per dependency); owned by the plan. */
bfs_status bfs_plan_static_waits(const bfs_plan *plan, const bfs_static_wait **out, int32_t *n);

bfs_status bfs_plan_stats(const bfs_plan *plan, bfs_stats *out);

/*
 * Host evaluation of dependency dep's threshold for the consumer engine's
 * registers r_P (entries of the producer's parent loop) and rhat_S (entries of
 * the shared loop in its current trip): Eq. 5 in barrier-free mode, the static
 * ordinal (or 0) in barrier mode, 0 for a barrier-fallback dependency.  This
 * is the value the device computes.  BFS_E_UNSUPPORTED for a per-engine plan
 * (its thresholds are snapshots of the walk, not a function of r_P, rhat_S).
 */
bfs_status bfs_eval_threshold(const bfs_plan *plan, int32_t dep, uint32_t r_P, uint32_t rhat_S,
                              uint32_t *out);

/* Frees the plan and its device images.  NULL-safe. */
void bfs_plan_destroy(bfs_plan *plan);

/*
 * Enqueue one execution of the planned program on stream (asynchronous): the
 * engines run the program with the synchronization the plan emitted, the
 * counter waits with Eq. 5's thresholds on the engines' loop registers
 * (Section 5.1, entries and per-trip entries per loop; Section 5.5, one
 * counter per loop and producer engine, or Eq. 3 per instruction, or the
 * per-engine counters of Section 6.1) in barrier-free mode, the all-engine
 * barriers and static ordinals of Section 3.4 in barrier mode; each
 * instruction's counter is incremented when it retires.
 *
 *   dev_buffers  family-specific device pointers, n_buffers of them
 *                (interp / stream3: [0] int64 per-workgroup tile base,
 *                [1] fp32 input tiles, [2] fp32 output; see the family notes
 *                in the implementation files for gemm / attn / moe).  The
 *                library does not know buffer lengths: the caller owns the
 *                buffers and must size them for the trip tables it passes
 *                (attn: the work list holds tile t of workgroup w at row
 *                w + t * n_wg for every t below w's T trip).
 *   dev_trips    int32 trip counts; dev_trip_off int64 [n_wg][n_loops]: the
 *                j-th execution of loop l in workgroup w runs
 *                dev_trips[dev_trip_off[w*n_loops + l] + j] iterations.
 *   n_wg         workgroups.
 *   dev_debug_log  NULL, or a uint32 buffer of n_wg * W * (1 + 4 * debug_capacity)
 *                words (W = waves per workgroup): per (workgroup, wave) the
 *                number of waits released, then up to debug_capacity entries
 *                {dependency, consumer instance, threshold, observed counter}.
 *                Logging is for tests; timed runs pass NULL.
 *   opts         NULL for defaults.
 * The first launch of a plan on a device uploads its tables (one allocation
 * per plan and device).  Device-side deadlock is reported by bfs_run_status.
 * BFS_E_UNSUPPORTED: a barrier-free plan with barrier-fallback dependencies
 * of a family other than the interpreter.
 */
bfs_status bfs_run(const bfs_plan *plan, const void *const *dev_buffers, int32_t n_buffers,
                   const int32_t *dev_trips, const int64_t *dev_trip_off, int32_t n_wg,
                   struct ihipStream_t *stream, uint32_t *dev_debug_log, int64_t debug_capacity,
                   const bfs_run_opts *opts);

/*
 * bfs_run without any device allocation, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Same arguments, kernels and results as bfs_run.
 *
 * bfs_run keeps each plan's device tables and error words in an allocation
 * of its own (made at the plan's first launch on a device).  This entry
 * point places them instead in one fixed array of BFS_NOALLOC_MAX_IMAGE_BYTES
 * bytes in the library's code object: each device holds its own copy from
 * the library's load until the process ends, and every plan on that device
 * shares it.  It calls no allocation routine (no hipMalloc, no hipFree).
 *
 *   - A plan whose tables exceed the array: BFS_E_RESOURCE (nothing is
 *     launched).  Only the interpreter family reads the tables: the first
 *     launch of an interpreter plan after another plan's writes them into
 *     the array with an asynchronous host-to-device copy on stream (the plan
 *     must stay alive until that work has completed); the other families read
 *     only the error words.
 *   - The error words are shared by every plan on the device: a device-side
 *     error (watchdog, rejected trip count) stays recorded until
 *     bfs_run_status of a plan that used this entry point on the device
 *     reports and clears it.
 *   - The array keeps the last call's contents.  Calls that overlap on one
 *     device (several streams or threads at once) race on it.
 */
#define BFS_NOALLOC_MAX_IMAGE_BYTES (256u * 1024u)
bfs_status bfs_run_noalloc(const bfs_plan *plan, const void *const *dev_buffers, int32_t n_buffers,
                           const int32_t *dev_trips, const int64_t *dev_trip_off, int32_t n_wg,
                           struct ihipStream_t *stream, uint32_t *dev_debug_log, int64_t debug_capacity,
                           const bfs_run_opts *opts);

/* Synchronizes stream, then reports (and clears) the plan's error words --
 * those of its own allocation (bfs_run) and, if the plan has used
 * bfs_run_noalloc on the current device, the fixed array's:
 * BFS_E_DEADLOCK if any wait gave up since the last call, BFS_E_INVALID if a
 * workgroup rejected a run-time input (a trip count beyond its work item, a
 * trip table that disagrees with a loop the kernel runs statically, a load
 * offset beyond 32 bits, a trip count beyond the ring-slot reuse the
 * program's dependencies order); the first error since the last call is
 * reported.  Allocates nothing. */
bfs_status bfs_run_status(const bfs_plan *plan, struct ihipStream_t *stream);

const char *bfs_status_string(bfs_status s);
const char *bfs_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* BFS_H */
