/*
 * pat.h -- C-ABI of the PAT (Parallel Aggregated Trees) all-gather and
 * reduce-scatter library for AMD Instinct MI355X (gfx950).
 *
 * Operations follow S. Jeaugey, "PAT: a new algorithm for all-gather and
 * reduce-scatter operations at scale" (arXiv:2506.20252):
 *   - the operations and their buffer rules: section "All-gather and
 *     reduce-scatter algorithms" (MPI semantics: the send buffer is never
 *     written; the reduce-scatter receive buffer is small);
 *   - the algorithm: sections "Binomial-tree based algorithms" (shifted
 *     binomial trees, farthest dimension first, truncated trees for any rank
 *     count), "The PAT algorithm" (intermediate buffers of bounded size,
 *     aggregation limited to T parallel sub-trees, far-first linear schedule)
 *     and "Conversion to reduce-scatter operations" (reversed trees, close
 *     dimensions first, accumulation buffers).
 *
 * One GPU emulates N virtual ranks.  Every rank's send buffer, receive buffer
 * and intermediate buffers ("slots") live in this GPU's memory, and each
 * network transfer of the paper is a device-local copy into the receiving
 * rank's slot or receive buffer.  Nothing crosses between GPUs.
 *
 * Conventions for every entry point:
 *   - Status codes only; nothing is thrown across this boundary.
 *   - `sendbufs` / `recvbufs` are HOST arrays of `nranks` DEVICE pointers,
 *     read during the call only (the library copies them into a device
 *     table it owns).  The buffers themselves are owned by the caller and
 *     must stay valid until `stream` has finished the operation.
 *   - Calls are asynchronous with respect to the host and ordered on
 *     `stream`.  Calls that use the same (operation, nranks, count, dtype,
 *     buffer budget) share library-owned intermediate buffers: they must be
 *     ordered on one stream (or otherwise serialised by the caller).
 *   - Pointers must be aligned to the element size.  When every pointer is
 *     16-byte aligned and count * sizeof(element) is a multiple of 16, the
 *     kernels move 128-bit vectors.  Otherwise they still move 128-bit
 *     vectors, at element-aligned addresses, as long as every piece of a
 *     chunk holds at least one (16 bytes; bf16 reduce-scatter: 4 elements):
 *     a piece's last, partial vector is moved back to end where the piece
 *     ends and stores only its own elements.  Pieces under one vector move
 *     single elements (correct, slower).
 *   - In place is allowed only in the MPI/NCCL form given per operation;
 *     any other overlap between a receive buffer and another buffer is
 *     PAT_ERR_INVALID_ARGUMENT.  Send buffers may overlap each other.
 *   - The library is thread-safe; plans are cached per device.
 */
#ifndef PAT_H_
#define PAT_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PAT_OK = 0,
  PAT_ERR_INVALID_ARGUMENT = 1, /* bad pointer, size, alignment or overlap */
  PAT_ERR_UNSUPPORTED = 2,      /* dtype / op / mode not provided */
  PAT_ERR_OUT_OF_MEMORY = 3,    /* intermediate buffers could not be allocated */
  PAT_ERR_HIP = 4,              /* a HIP runtime call failed; see pat_last_hip_error() */
  PAT_ERR_TIMEOUT = 5,          /* a persistent kernel's step barrier gave up waiting */
  PAT_ERR_INTERNAL = 6,         /* a plan failed its own consistency checks */
  PAT_ERR_TOO_LARGE = 7         /* pat_reducescatter_noalloc: the operation needs more than
                                   PAT_NOALLOC_SCRATCH_BYTES of tables and intermediate buffers */
} pat_status_t;

typedef enum {
  PAT_INT32 = 0,   /* reduce-scatter sums wrap modulo 2^32 */
  PAT_FLOAT32 = 1, /* IEEE float32 adds, round to nearest even */
  PAT_BFLOAT16 = 2 /* reduce-scatter: partial sums carried in float32, rounded
                      to bfloat16 (nearest even) once, at the owning rank */
} pat_dtype_t;

typedef enum { PAT_SUM = 0 } pat_op_t;

typedef enum {
  PAT_ALLGATHER = 0,
  PAT_REDUCESCATTER = 1
} pat_collective_t;

typedef enum {
  /* One launch per operation.  Workgroups take per-step work from device
   * counters in step order, and step s starts only when every piece of step
   * s - 1 is done.  It needs no co-residency, so any grid size is safe; the
   * grid is 2, 4 or all workgroups per compute unit by bytes per step
   * (PAT_PERSISTENT_BLOCKS_PER_CU overrides).  Each step costs a few
   * microseconds of device-scope synchronisation, more than a kernel
   * boundary, so the stream mode is faster on MI355X. */
  PAT_EXEC_PERSISTENT = 0,
  /* One kernel per step, captured once per plan (and vector width) into a
   * HIP graph and replayed. */
  PAT_EXEC_GRAPH = 1,
  /* One kernel per step, launched directly on the stream.  The default: as
   * fast as the graph for large operations, and without the graph launch's
   * fixed cost for small ones. */
  PAT_EXEC_STREAM = 2,
  /* Dataflow: one launch per piece, no step barrier.  Workgroups take work
   * in step order as in the persistent mode, but a work item (one tile of
   * one chunk-edge) waits only for the two buffers it touches: per (rank,
   * slot) counters of completed tiles -- the receiver's slot emptied by every
   * earlier reader before it is refilled, the sender's slot filled before it
   * is read (all-gather); the child's accumulator complete, the receiver's
   * earlier additions done (reduce-scatter).  Ranks and trees run ahead of
   * one another as far as their own buffers allow (section "Future work":
   * the linear part).  Waits are bounded like the persistent mode's
   * (PAT_ERR_TIMEOUT).  Needs N x (slot entries per rank + 1) 4-byte counters,
   * at most 256 MiB (else PAT_ERR_UNSUPPORTED). */
  PAT_EXEC_DATAFLOW = 3
} pat_exec_mode_t;

/*
 * All-gather (section "All-gather and reduce-scatter algorithms"):
 *   recvbufs[r][x * count + i] = sendbufs[x][i]   for all ranks r, x and i < count.
 *   sendbufs[x]: `count` elements.   recvbufs[r]: nranks * count elements.
 * Steps: the all-gather steps of section "The PAT algorithm".
 * In place: sendbufs[r] == recvbufs[r] + r * count (the own chunk is then not copied).
 * count == 0: PAT_OK, nothing is launched.  nranks == 1: a plain copy.
 */
pat_status_t pat_allgather(const void* const* sendbufs, void* const* recvbufs, size_t count,
                           pat_dtype_t dtype, int nranks, hipStream_t stream);

/*
 * Reduce-scatter, sum (sections "All-gather and reduce-scatter algorithms" and
 * "Conversion to reduce-scatter operations"):
 *   recvbufs[R][i] = sum over x of sendbufs[x][R * count + i]   for i < count.
 *   sendbufs[x]: nranks * count elements.   recvbufs[R]: `count` elements.
 * Summation order: the reversed binomial tree of chunk R rooted at rank R;
 * with the far-first linear order children are added nearest first and the
 * order does not depend on the buffer budget.
 * In place: recvbufs[r] == sendbufs[r] + r * count.
 * count == 0: PAT_OK, nothing is launched.  nranks == 1: a plain copy.
 */
pat_status_t pat_reducescatter(const void* const* sendbufs, void* const* recvbufs, size_t count,
                               pat_dtype_t dtype, pat_op_t op, int nranks, hipStream_t stream);

/*
 * Reduce-scatter that allocates nothing, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation.  Same operation, arguments, summation order, buffer
 * budget, linear order and fusion settings as pat_reducescatter, and the same
 * bits; it always runs as per-step kernels on `stream` (the execution-mode
 * setting does not apply).
 *
 * Instead of the plan cache's device memory, every table, intermediate buffer
 * and float32 root accumulator lives in a fixed array of
 * PAT_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * until the process ends.  The call makes no hipMalloc / hipFree / host
 * pinning and creates no event, stream or graph; its host-side schedule
 * tables are built in ordinary host memory.  When the plan or the pointer
 * set differs from the previous call's on this GPU, the tables are first
 * copied into the array with host-to-device copies on `stream`; repeated
 * calls with the same plan and buffers launch kernels only.
 *
 * Every call on a GPU shares that GPU's array, which keeps the last call's
 * contents (nothing in it must start at zero): calls that may overlap on one
 * GPU -- on different streams, or from several host threads without ordering
 * -- race and give undefined results.  Order them on one stream.
 *
 * Errors: as pat_reducescatter, plus PAT_ERR_TOO_LARGE (nothing is launched)
 * when the plan's slots (slot_bytes_total of pat_plan_info) and tables
 * exceed the array.
 */
#define PAT_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)
pat_status_t pat_reducescatter_noalloc(const void* const* sendbufs, void* const* recvbufs, size_t count,
                                       pat_dtype_t dtype, pat_op_t op, int nranks, hipStream_t stream);

/*
 * Intermediate-buffer budget B, in bytes per slot (section "The PAT
 * algorithm": the aggregation is limited to what the buffer holds).  A rank
 * holds at most ceil(log2 nranks) slots of at most B bytes each.  The plan
 * uses T = 2^t parallel sub-trees, the largest power of two <= 2^(L-1) whose
 * largest step fits B; a chunk larger than B is processed in pieces of at
 * most B bytes.  0 restores the default (8 MiB, or the PAT_BUFFER_BYTES
 * environment variable).  Affects plans created afterwards.
 */
pat_status_t pat_set_buffer_bytes(size_t bytes_per_slot);
size_t pat_get_buffer_bytes(void);

/*
 * Order of the linear part inside the T parallel sub-trees (section "The PAT
 * algorithm"): far-first, the paper's main schedule and the default, or
 * close-first, the alternative the paper allows.  Both drain every slot before
 * its distance is used again, so both keep <= T chunks per slot; the step
 * count is the same.  The reduce-scatter summation order follows the chosen
 * walk.  Default: far-first, or the PAT_LINEAR_ORDER environment variable
 * (far | close).  Affects plans created afterwards.
 */
typedef enum { PAT_LINEAR_FAR_FIRST = 0, PAT_LINEAR_CLOSE_FIRST = 1 } pat_linear_order_t;
pat_status_t pat_set_linear_order(int order);
int pat_get_linear_order(void);

/*
 * Aggregation rule (section "The PAT algorithm": as many parallel sub-trees
 * as the buffer permits).  PAT_AGGREGATION_POW2, the default, takes T = 2^t
 * sub-trees, the largest power of two whose steps fit the budget, as in the
 * paper's examples.  PAT_AGGREGATION_BUDGET lets a step carry any number
 * K = floor(B / chunk bytes) of chunks: where K is not a power of two (or the
 * rank count is not), a list schedule -- still one peer per step, each node
 * forwarding farthest child first, at most K chunks per slot -- may need
 * fewer steps, and replaces the power-of-two schedule then (never with
 * pieces).  The reduce-scatter's summation order is the same either way.  A
 * list schedule runs without fused launches (its slot entries pass between
 * trees).  Default: PAT_AGGREGATION_POW2, or the PAT_AGGREGATION environment
 * variable (pow2 | budget).  Affects plans created afterwards.
 */
typedef enum { PAT_AGGREGATION_POW2 = 0, PAT_AGGREGATION_BUDGET = 1 } pat_aggregation_t;
pat_status_t pat_set_aggregation(int mode);
int pat_get_aggregation(void);

/* Execution mode (pat_exec_mode_t).  Default: PAT_EXEC_STREAM, or the
 * PAT_EXEC_MODE environment variable (persistent | graph | stream | dataflow). */
pat_status_t pat_set_exec_mode(int mode);
int pat_get_exec_mode(void);

/*
 * Fusion of the schedule's top part (stream and graph modes).  In the top t
 * steps (the fully aggregated distances, section "The PAT algorithm") every
 * intermediate-buffer entry serves a single tree, so one workgroup per (tree,
 * tile of its chunk) can run all of them with workgroup barriers instead of
 * one kernel per step.  When the sub-trees span at most 4 (T >= 2^(L-2)) the
 * same holds for the whole schedule, whose linear steps then join the
 * fusable range: a linear-part node keeps its chunk at index p / 4 of its
 * distance's slot, used by position p alone, and leaves keep nothing.  The
 * edges, bytes and summation order are unchanged.  A workgroup runs its
 * tree's steps one after another, so wide steps (many chunks per rank) are
 * better left to one kernel each.  AUTO (the default, or the PAT_TOP_FUSION
 * environment variable: auto | on | off) fuses the far end of the fusable
 * range, the steps that move at most 128 MiB and in which one tree's edges
 * over one tile of its chunk amount to at most 2048 vectors, when there are
 * two or more such steps; ON
 * fuses the whole fusable range whenever it has two or more steps.  Neither
 * fuses a chunk that is split into pieces.  A tile is the smallest power of
 * two from 32 to 256 vectors that keeps the launch within 1024 workgroups.
 */
typedef enum { PAT_FUSION_AUTO = 0, PAT_FUSION_OFF = 1, PAT_FUSION_ON = 2 } pat_fusion_t;
pat_status_t pat_set_top_fusion(int mode);
int pat_get_top_fusion(void);

/* Wall-clock limit of one wait of the persistent kernel for the previous step,
 * in microseconds (0 = default, 10 s).  When exceeded the kernel records a
 * timeout (see pat_check_device_status) and exits instead of waiting forever;
 * the operation's result is then undefined. */
pat_status_t pat_set_barrier_timeout_us(uint32_t microseconds);

/* Plan summary.  Host-only: needs no GPU. */
typedef struct {
  int nranks;
  int L;                      /* ceil(log2 nranks) */
  int t;                      /* T = 2^t parallel sub-trees */
  int T;
  int steps;                  /* communication steps per piece */
  int pieces;                 /* pieces a chunk is split into (1 unless chunk > budget) */
  int max_chunks_per_step;    /* largest number of chunks a rank sends in one step */
  int vector_path;            /* path taken with 16-byte-aligned pointers: 1 aligned 128-bit
                                 vectors; 2 128-bit vectors with a partial last vector per piece
                                 (also the path of element-aligned pointers whenever it is not 0);
                                 0 single elements (a piece under one vector) */
  size_t count;               /* elements per chunk */
  size_t piece_elems;         /* elements per piece */
  size_t slot_elem_bytes;     /* 4 for bf16 reduce-scatter (float32 partials) */
  int slot_dims;              /* distinct slot dimensions a rank uses */
  int slot_chunks_per_rank;   /* chunk-sized slot entries per rank */
  size_t slot_bytes_per_rank; /* intermediate memory per rank */
  size_t slot_bytes_total;    /* all ranks, plus the float32 root accumulators */
  double alg_bytes;           /* memory bytes the steps must read + write per operation */
  double bus_bytes_per_rank;  /* (nranks - 1) * count * sizeof(dtype) */
  int fused_steps;            /* steps run as one fused launch (stream/graph modes, current setting) */
  int launches_per_op;        /* kernel launches per operation in stream mode (path vector_path) */
  int streaming;              /* 1: nontemporal loads and stores (operations of >= 1e9 algorithmic bytes) */
  int xcd_run;                /* step kernels: each XCD takes runs of this many consecutive work items
                                 (0: a contiguous eighth of each step; all-gather 0, reduce-scatter 32) */
  int list_schedule;          /* 1: the list schedule of PAT_AGGREGATION_BUDGET (T = chunks per step) */
} pat_plan_info_t;

pat_status_t pat_plan_info(pat_collective_t coll, int nranks, size_t count, pat_dtype_t dtype,
                           pat_plan_info_t* out);

/*
 * Step table of a plan (one piece), host-only.  For step s (in execution
 * order) step_d[s] is the distance d and step_k[s] the number of chunks each
 * rank handles; the entries of step s follow those of step s-1.  Entry j:
 *   pos[j]   tree position p (all-gather: the sender; reduce-scatter: the receiver);
 *   a[j], b[j], c[j]  slot indices (chunk entries of a rank's slot area) or markers:
 *     all-gather:     a = source slot or -1 (own send buffer),
 *                     b = slot written at the receiver or -1 (receive buffer only),
 *                     c = -1 (unused);
 *     reduce-scatter: a = child's slot or -1 (child's raw input),
 *                     b = own accumulator slot, -1 (own raw input), -2 (root accumulator),
 *                     c = destination slot, -2 (root accumulator), -3 (root, last receive).
 * Arrays must hold max_steps / max_entries elements; *nsteps / *nentries get
 * the sizes (PAT_ERR_INVALID_ARGUMENT if they do not fit).
 */
pat_status_t pat_plan_steps(pat_collective_t coll, int nranks, size_t count, pat_dtype_t dtype,
                            int32_t* step_d, int32_t* step_k, int max_steps, int32_t* pos,
                            int32_t* a, int32_t* b, int32_t* c, int max_entries, int* nsteps,
                            int* nentries);

/*
 * Launch tracing, for measurement (stream mode only; graph and persistent
 * modes and pat_reducescatter_noalloc record nothing).  pat_trace_start
 * creates 2 * max_launches HIP events and arms the trace: the following
 * operations record one event on their stream right before and one right
 * after each kernel launch, until max_launches launches are recorded.
 * pat_trace_read waits for the recorded events and returns, per launch in
 * launch order: its duration in milliseconds (ms), the algorithmic bytes it
 * moves by the plan's byte model (bytes; summed over an operation's launches
 * they give pat_plan_info's alg_bytes), its kernel (kind: 0 one step, 1 a
 * fused range of steps) and its first launch-level step (step).  Any output
 * array may be NULL; each must hold `max` entries.  *n gets the number of
 * launches recorded; if it exceeds max, PAT_ERR_INVALID_ARGUMENT and the trace
 * stays armed.  Otherwise the events are destroyed and the trace disarmed.
 * max_launches: 1 .. 2^20.
 */
pat_status_t pat_trace_start(int max_launches);
pat_status_t pat_trace_read(float* ms, double* bytes, int32_t* kind, int32_t* step, int max, int* n);

/*
 * Step clock of fused launches (measurement; stream mode).  When the
 * environment variable PAT_STEP_CLOCK is 1 as a plan is made, every fused
 * launch of that plan (the range of steps one workgroup per (tree, tile) runs
 * with workgroup barriers in between) records, per workgroup, the device wall
 * clock before its first step and after each step: step k of workgroup w took
 * stamps[w * per_workgroup + k + 1] - stamps[w * per_workgroup + k] ticks
 * (*ticks_per_us per microsecond).  pat_step_clock waits for the plan's last
 * operation and copies the stamps of its last fused launch (the plan of the
 * current device, buffer budget and linear order).  *workgroups and
 * *per_workgroup are set whenever such stamps exist; `stamps` must hold
 * their product (else PAT_ERR_INVALID_ARGUMENT).  PAT_ERR_INVALID_ARGUMENT
 * too when the plan has none (no such plan, the variable was off, or no
 * fused launch ran in stream mode).  Off by default: the fused kernel then
 * records nothing.
 */
pat_status_t pat_step_clock(pat_collective_t coll, int nranks, size_t count, pat_dtype_t dtype, uint64_t* stamps,
                            size_t max, int* workgroups, int* per_workgroup, double* ticks_per_us);

/* Cached plans: their number and the device memory they hold, all devices.
 * Plans are cached per (operation, nranks, count, dtype, budget, linear
 * order, device).  When a new plan would take a device's cached plans past
 * PAT_PLAN_CACHE_BYTES (default 32 GiB), the least recently used plans of that
 * device are released first, each after its last operation has finished on
 * its stream; an allocation failure releases every other plan of the device
 * and retries once.  Host-only. */
pat_status_t pat_cache_stats(int* plans, size_t* bytes);

/* Waits for `stream`, then reports (and clears) a barrier timeout recorded by
 * a persistent kernel on the current device: PAT_OK or PAT_ERR_TIMEOUT. */
pat_status_t pat_check_device_status(hipStream_t stream);

/* Last hipError_t seen by a call that returned PAT_ERR_HIP (0 if none). */
int pat_last_hip_error(void);

const char* pat_status_string(pat_status_t status);

/* Frees every plan, intermediate buffer and graph on every device.  Waits for
 * the devices first.  Later calls rebuild what they need. */
pat_status_t pat_finalize(void);

#ifdef __cplusplus
}
#endif

#endif /* PAT_H_ */
