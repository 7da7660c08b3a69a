/*
 * hoccl.h -- C ABI of libhoccl, an MI355X (gfx950) implementation of the
 * hot path behind HOCCL's collectives: the chunked data movement and the
 * element-wise reduction of ring reduce-scatter, all-gather and all-reduce,
 * point-to-point send/recv and all-to-all(v).
 *
 * Setting.  One process drives one GPU.  A collective runs across R "virtual
 * ranks" whose buffers all live in that GPU's memory: rank r's buffer is
 * simply the r-th pointer of an array.  The paper's setting spans many GPUs;
 * here every ring hop, every point-to-point flow and every all-to-all block
 * becomes a copy or a reduction between two regions of one HBM.
 *
 * Two execution paths, as in the paper's design (System Design, Overview):
 *   - pure-copy steps go to the SDMA copy engines, so they occupy no compute
 *     unit (the zero-SM point-to-point executor, here "zero-CU"): a CPU
 *     proxy thread issues them on chosen engines through ROCr;
 *   - reduction steps, which the paper leaves to SM-side execution
 *     (Limitations), run as gfx950 HIP kernels with an explicit workgroup
 *     budget.
 * Operator order with the caller's stream is kept by a stream manager
 * (Stream Manager section): the start/finish flag handshake through host
 * memory for the engine proxy, and HIP event fork/join for the copies the
 * HIP runtime issues (HOCCL_COPY_HIP).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers.  `send` and `recv` are HOST arrays of R DEVICE pointers.  The
 *   arrays are read during the call only; the device buffers are owned by the
 *   caller, must stay valid until the operation completes on `stream`, and
 *   are never retained by the library after that.
 * Counts are in elements of `dtype`.  For copy-only collectives the dtype
 *   only sets the element size (4 bytes for int32/fp32, 2 for bf16, 1 for
 *   uint8) and the bytes are moved bit for bit.
 * Asynchrony.  Every call returns once the work is enqueued.  The operation
 *   starts after all work previously enqueued on `stream` and all work
 *   enqueued on `stream` afterwards sees its results.  No call synchronises
 *   the host with the device except where stated (workspace growth).  The
 *   HIP runtime itself makes the enqueueing thread wait once too much work
 *   is pending behind unfinished work: on MI355X about 1000 of this
 *   library's kernel launches (some 150 ring reduce-scatters at R = 8),
 *   or 32 of the HIP runtime's own copies of 1 MiB or more on the
 *   HOCCL_COPY_HIP path.  The engine proxy admits 512 operations in flight
 *   and waits up to its timeout for a free one.
 * Errors.  Every function returns a hoccl_status_t and never throws.
 *   Argument errors are detected before anything is enqueued.  A failing HIP
 *   or HSA call returns HOCCL_ERR_HIP; hoccl_last_error_string() describes
 *   it.  Faults of the device work itself surface at the caller's own
 *   synchronisation.  `count == 0` is a successful no-op.  The only error
 *   that outlives its call is the SDMA proxy's watchdog: copies of an
 *   earlier call that made no progress for proxy_timeout_ms are reported
 *   once, as HOCCL_ERR_TIMEOUT, by the next SDMA call (which then
 *   enqueues nothing).
 * Threads.  Calls from several host threads on one device take turns: each
 *   holds a per-device lock while it plans and enqueues (not while the
 *   work runs), and calls run in the order they take it.  Statistics and
 *   error strings are per thread.  hoccl_finalize must not overlap other
 *   calls.  Collectives issued on different streams that overlap in time are
 *   ordered by the library where they share its workspace or its internal
 *   copy / handshake streams, in the order the calls were issued: a call
 *   must not wait, through the caller's own stream dependencies, for a call
 *   issued after it.
 * Stream capture.  A call on a stream that is capturing into a HIP graph
 *   records its kernels, events and copies (never a memset) and allocates
 *   no device memory.  Engine-proxy copies are recorded as a host node that
 *   issues them on the SDMA engines at every replay and returns once they
 *   have completed (no GPU code); this needs the host-function handshake,
 *   so while a profiler is loaded AUTO records the HIP runtime's copies
 *   instead.  A call returns HOCCL_ERR_UNSUPPORTED, enqueuing nothing, as
 *   the first call on a device (which creates the library's streams and
 *   probes the engines), when it needs a larger workspace than the library
 *   holds, or when copy_path is SDMA with the handshake kernel
 *   (proxy_handshake 0 or 1).  Make the same call once outside capture
 *   first.  The copy lists of recorded host nodes stay allocated until
 *   hoccl_finalize.  A workspace a graph captured stays
 *   allocated until hoccl_finalize, after which the graph must not be
 *   replayed.  Replays share it with the device's other workspace users
 *   (ring reduce-scatter and all-reduce over more than two ranks) and are
 *   not ordered with them by the library: a replay must not overlap another
 *   such call or replay.  Kernel timing skips captured calls.
 * In-place forms (the only allowed overlaps between send and recv):
 *   all-reduce      send[r] == recv[r];
 *   all-gather      send[r] == recv[r] + r * sendcount elements;
 *   reduce-scatter  recv[r] == send[r] + r * recvcount elements.
 *   All other collectives are out-of-place only.
 * Alignment.  Any element-aligned pointer is accepted; 16-byte aligned
 *   buffers take the vectorised fast path.
 */
#ifndef HOCCL_H
#define HOCCL_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    HOCCL_OK = 0,
    HOCCL_ERR_INVALID_ARG = 1, /* bad pointer, count, R, dtype, peer map or overlap */
    HOCCL_ERR_UNSUPPORTED = 2, /* valid request the library cannot serve here     */
    HOCCL_ERR_HIP = 3,         /* a HIP / HSA runtime call failed                   */
    HOCCL_ERR_NO_MEMORY = 4,   /* workspace or host allocation failed               */
    HOCCL_ERR_TIMEOUT = 5,     /* the copy proxy's watchdog, or a mailbox wait, expired */
    HOCCL_ERR_INTERNAL = 6
} hoccl_status_t;

/* Element types.  INT32, FP32 and BF16 are the reduction types.  UINT8 is
 * for the copy-only collectives (all-gather, send/recv, all-to-all(v)),
 * which move bits and use the dtype only for the element size: it lets a
 * caller move any byte count.  The reductions (all-reduce,
 * reduce-scatter, ring hop) return HOCCL_ERR_INVALID_ARG for it. */
typedef enum { HOCCL_INT32 = 0, HOCCL_FP32 = 1, HOCCL_BF16 = 2, HOCCL_UINT8 = 3 } hoccl_dtype_t;

/* Where pure-copy steps run.  AUTO, SDMA and KERNEL keep the values 0, 1
 * and 2; the HIP runtime's own copy is appended as 3. */
typedef enum {
    HOCCL_COPY_AUTO = 0,   /* SDMA, the path that keeps copies off the compute
                              units; HIP when the engines cannot be driven,
                              or while capturing under a profiler           */
    HOCCL_COPY_SDMA = 1,   /* a CPU proxy thread issues each chunk on an
                              explicitly chosen SDMA engine (ROCr,
                              hsa_amd_memory_async_copy_on_engine) and
                              releases the stream by flag handshake
                              (proxy_handshake); with chunk_bytes 0 and fewer
                              chains than engines it cuts every copy into
                              engines/chains equal pieces of at least
                              512 KiB.  Its copies finish while every CU is
                              busy (Zero-SM Point-to-Point Executor)       */
    HOCCL_COPY_KERNEL = 2, /* CU copy kernel with workgroups_per_step
                              workgroups (comparator / fallback)           */
    HOCCL_COPY_HIP = 3     /* hipMemcpyAsync(DeviceToDeviceNoCU) on the
                              library's copy streams.  Where the copy runs is
                              the HIP runtime's choice: in the runtime
                              PyTorch bundles it runs on the compute units
                              (it cannot finish while every CU is busy), in
                              ROCm 7.2's on one SDMA engine.
                              Graph-capturable                             */
} hoccl_copy_path_t;

/* How reduce-scatter / all-reduce reduce.  Every choice folds in the same
 * order, so the results are identical bit for bit. */
typedef enum {
    HOCCL_REDUCE_RING = 0,   /* R-1 ring steps (or fused_hops steps per
                                launch), one kernel launch per step over all
                                ranks; fp32 partials for bf16 (bf16 ones
                                with bf16_partials)                        */
    HOCCL_REDUCE_DIRECT = 1, /* one launch folds all R inputs in the ring
                                order (fewer HBM bytes)                    */
    HOCCL_REDUCE_AUTO = 2    /* DIRECT where the one-GPU fold is faster:
                                up to direct_max_ranks ranks, whatever the
                                size; RING otherwise.  The choice made is
                                reported in hoccl_stats_t.reduce_algo_used */
} hoccl_reduce_algo_t;

/* The first seven fields are the core configuration; the rest extend it. */
typedef struct {
    int workgroups_per_step;    /* workgroups per reduce / CU-copy launch;
                                   0 = automatic (fills the chip)              */
    int threads_per_workgroup;  /* 64..1024, multiple of 64; 0 = 256           */
    size_t chunk_bytes;         /* split copies into pieces of this size
                                   (>= 4096); 0 = no split, or the automatic
                                   split of the SDMA copy path                 */
    int copy_streams;           /* copy streams of the HIP path, 1..16; 0 = 8  */
    hoccl_copy_path_t copy_path;
    int allgather_direct;       /* 1 (default): every rank copies each shard
                                   from its owner, the all-pairs traffic
                                   matrix; 0: ring forwarding r -> r+1         */
    int allreduce_chunk_groups; /* split each all-reduce ring chunk into this
                                   many groups so the gather of group g
                                   overlaps the reduction of group g+1 (on
                                   the SDMA path the proxy issues group g's
                                   copies once an event the stream records
                                   after its reduction has completed);
                                   0 = automatic: 2 on the SDMA path outside
                                   graph capture when each rank holds at
                                   least 32 MiB and the engine budget is 8
                                   or more (with fewer engines the gather
                                   dwarfs the reduction it would overlap),
                                   else 1 (plan dumps assume the SDMA
                                   path)                                       */
    /* ---- extensions ---- */
    int sdma_engines;           /* engines the SDMA path may use, 1..32 (at
                                   most those available, 16 on MI355X);
                                   0 = automatic: 4, the most whose copies
                                   cost a concurrent bf16 GEMM at most 2%
                                   (the copies run about 3x slower than on
                                   all 16; set 16 where no compute runs
                                   beside them)                                */
    hoccl_reduce_algo_t reduce_algo;
    int kernel_timing;          /* 1: record HIP events around every reduce /
                                   copy kernel launch (hoccl_get_kernel_times) */
    unsigned int proxy_timeout_ms; /* watchdog of the SDMA proxy: an operation
                                   whose copies make no progress (none
                                   issued, none completed) for this long is
                                   reported; 0 = 10000                      */
    int proxy_handshake;        /* the stream side of the SDMA path's
                                   start/finish flag handshake (Stream
                                   Manager, CPU-GPU handshake protocol):
                                   -1 (default): 2, or 0 while a ROCm
                                   profiler is loaded;
                                   0: a one-lane kernel on the caller's
                                   stream that waits on a CU while the
                                   copies run (4 KiB send/recv: 23 us);
                                   1: that kernel on a private CU-masked
                                   stream with a hardware queue of its own,
                                   joined to the caller's stream by events
                                   (86 us), so the wait never holds back the
                                   caller's hardware queue;
                                   2: a host function on the caller's stream
                                   (hipLaunchHostFunc): no GPU code waits and
                                   no CU is used (4 KiB send/recv: 57 us),
                                   but the HIP runtime's callback thread is
                                   blocked while the copies run.  With a
                                   ROCm profiler loaded (rocprofiler-sdk
                                   preloaded, or HSA_TOOLS_LIB set) an
                                   explicit 2 returns HOCCL_ERR_UNSUPPORTED */
    size_t ring_group_bytes;    /* ring reduce-scatter / all-reduce run their
                                   R-1 steps group by group over slices of
                                   every chunk, one group's partials
                                   taking at most this many bytes, so they
                                   stay in the 256 MB last-level cache from
                                   step to step (same fold order, same bits).
                                   0 = the library default; SIZE_MAX = one
                                   group                                       */
    unsigned int proxy_wait_limit_us; /* the handshake kernel stops waiting
                                   after this long, so its dispatch always
                                   ends; the proxy then reports
                                   HOCCL_ERR_TIMEOUT at the next SDMA call.
                                   0 = 2 * proxy_timeout_ms + 1 s              */
    int fused_hops;             /* ring reduce-scatter / all-reduce: ring hops
                                   folded per reduction launch, 0..64 (0 and
                                   1: one hop per launch; at most 8 per
                                   launch are used).  A fused launch adds its
                                   hops' contributions to the partial in
                                   registers, in the ring's order (same
                                   bits), and reads and writes the partial
                                   once instead of once per hop; R-1 hops
                                   fold the whole chunk in one launch      */
    int a2a_schedule;           /* all-to-all(v) copy schedule:
                                   0 (default): every flow a chain of its
                                   own, chains balanced over the engines by
                                   bytes and interleaved by flow size;
                                   1: the stages of the collective
                                   scheduler's Birkhoff-like decomposition
                                   of the traffic matrix (Collective
                                   Scheduler, Algorithm 1): each stage a
                                   matching (every rank sends and receives
                                   at most one piece), the engines' queues
                                   in stage order;
                                   2: as 1, the stages run one after another
                                   (the CU copy kernel launches stage by
                                   stage; on the SDMA path this returns
                                   HOCCL_ERR_UNSUPPORTED, enqueuing
                                   nothing).  The HIP path ignores stages  */
    size_t proxy_slice_bytes;   /* balanced issue on the SDMA path, for
                                   operations whose copies wait for no
                                   other (send/recv, direct all-gather,
                                   all-to-all(v)): instead of issuing every
                                   copy at once on its scheduled engine,
                                   the proxy lets the engines take pieces
                                   in the schedule's order as they have
                                   room (two pieces, or twice this many
                                   bytes, in flight each).  An engine's
                                   first piece is a whole copy if that is
                                   no more than its share of the total;
                                   later ones are the unissued bytes over
                                   the engine count, at least this many
                                   bytes.  An
                                   engine takes a piece only if it would
                                   finish it before the operation's
                                   projected end or about as early as any
                                   engine, from rates measured on its
                                   completed pieces; so an engine slowed by
                                   other work (for a while after a large
                                   device free, engine 1) costs only its
                                   share (flow-size-aware chunk
                                   scheduling).  A multiple of 4096,
                                   >= 64 KiB.  0 = automatic: 4 MiB with 8
                                   or more engines for operations of at
                                   least 64 MiB per engine, every copy at
                                   once otherwise (the automatic 4 engines,
                                   which the release does not slow, where
                                   balanced issue raised a concurrent
                                   GEMM's loss by about half a point, and
                                   smaller operations, where it cost more
                                   than a slowed engine could);
                                   SIZE_MAX = every copy at once.  Copies
                                   that wait for others (the ring
                                   all-gather, the reduce-scatter /
                                   all-reduce gathers) and graph captures
                                   are always issued at once               */
    int bf16_partials;          /* bf16 reduce-scatter / all-reduce partials:
                                   0 (default): the partial sums travel in
                                   fp32 and each output is rounded to bf16
                                   once, after its last addition (the
                                   result is the sum in ring order rounded
                                   once);
                                   1: every addition's result is rounded to
                                   bf16 (round to nearest, ties to even)
                                   before the next one, as when each rank
                                   of the ring forwards its partial in the
                                   collective's own element type: the ring
                                   step moves 6 bytes per element instead
                                   of 8 to 10 and its workspace is half the
                                   size, at up to R-1 roundings of error
                                   instead of one.  The same ring order and the
                                   same roundings on the ring, fused hops,
                                   the direct fold and every grouping.
                                   Other dtypes ignore it.  hoccl_ring_hop
                                   is unaffected: its HOCCL_HOP_ONLY is the
                                   bf16-partial hop                         */
} hoccl_config_t;

/* The first eight fields are the core statistics; the rest extend them. */
typedef struct {
    int reduce_launches;        /* reduction kernel launches enqueued          */
    int copy_ops;               /* copy commands issued to the engine proxy
                                   or the HIP runtime                          */
    int workgroups_per_step;    /* workgroups per launch actually used         */
    int cus_available;          /* compute units of the device                 */
    int cus_used_max;           /* upper bound on CUs occupied by this call:
                                   min(workgroups, CUs) when kernels run; at
                                   least 1 when the SDMA handshake is the
                                   one-lane kernel; all CUs when copies go
                                   through the HIP runtime (HOCCL_COPY_HIP),
                                   which may run them as a kernel of its own;
                                   0 for copy-only calls on the SDMA path
                                   with the host-function handshake            */
    hoccl_copy_path_t copy_path_used;
    unsigned long long hbm_bytes_algorithmic; /* bytes every step must read
                                   and write in HBM, summed over the call      */
    double host_enqueue_us;     /* host time spent inside the call             */
    /* ---- extensions ---- */
    int copy_kernel_launches;   /* CU copy kernel launches enqueued            */
    hoccl_reduce_algo_t reduce_algo_used; /* RING or DIRECT (never AUTO)       */
    unsigned long long copy_bytes;             /* bytes moved by copy steps   */
} hoccl_stats_t;

/* ---- set-up and configuration ------------------------------------------
 * The paper switches a training job between NCCL and its library with one
 * environment variable (Implementation); here HOCCL_* variables configure
 * the library the same way.
 *
 * Initialise the library on `device` (the current HIP device if < 0):
 * creates the internal copy streams, the event pool and, when the SDMA
 * engines can be driven directly, the proxy thread and its flag pool.
 * Reads HOCCL_* environment variables into the configuration:
 *   HOCCL_WG_PER_STEP, HOCCL_THREADS_PER_WG, HOCCL_CHUNK_BYTES,
 *   HOCCL_COPY_STREAMS, HOCCL_SDMA_ENGINES, HOCCL_AG_DIRECT,
 *   HOCCL_AR_GROUPS, HOCCL_KERNEL_TIMING, HOCCL_PROXY_HANDSHAKE,
 *   HOCCL_PROXY_WAIT_LIMIT_US, HOCCL_RING_GROUP_BYTES, HOCCL_FUSED_HOPS,
 *   HOCCL_A2A_SCHEDULE, HOCCL_PROXY_SLICE_BYTES, HOCCL_BF16_PARTIALS
 *   (the fields of the same meaning),
 *   HOCCL_COPY_PATH = auto | sdma (or engines) | kernel | hip,
 *   HOCCL_REDUCE_ALGO = ring | direct | auto,
 *   HOCCL_DEBUG = 1 (log every executed plan as JSON to stderr),
 *   HOCCL_SDMA_ENGINE_IDS = "i,j,..." (the SDMA engines the SDMA
 *   proxy may use, in that order; read when the proxy is created),
 *   HOCCL_PROXY_SCHEDULE = round_robin (ablation: chain c on engine c mod E
 *   in plan order, instead of the byte-balanced, flow-size-interleaved
 *   schedule).
 * A set of values that fails validation falls back to the defaults.
 * Optional: every collective initialises lazily on the current device. */
hoccl_status_t hoccl_init(int device);

/* Waits for the device, then releases streams, events, workspace, the proxy
 * thread and the flag pool.  A later call re-initialises. */
hoccl_status_t hoccl_finalize(void);

/* Replace / read the configuration.  Invalid fields give
 * HOCCL_ERR_INVALID_ARG and leave the configuration unchanged. */
hoccl_status_t hoccl_set_config(const hoccl_config_t *cfg);
hoccl_status_t hoccl_get_config(hoccl_config_t *cfg);

/* Statistics of the most recent collective call on this thread: launches,
 * copies, workgroups and CUs, the quantities the paper's communication
 * benchmark reports per configuration (Evaluation, Communication Benchmark:
 * bandwidth against the number of SMs a collective may use). */
hoccl_status_t hoccl_get_last_stats(hoccl_stats_t *stats);

/* With kernel_timing on, every kernel launch of every collective call is
 * bracketed by a pair of timing events on the stream it is launched on (at
 * most 65536 launches between two reads; later ones go untimed).
 * This returns the durations in milliseconds of all launches recorded since
 * the previous read, in launch order, waits for those launches to finish and
 * clears the record.  *n receives the number of launches; at most `cap`
 * durations are written.  With cap == 0 it only reports the count and keeps
 * the record. */
hoccl_status_t hoccl_get_kernel_times(float *ms, int cap, int *n);

const char *hoccl_status_string(hoccl_status_t status);
const char *hoccl_last_error_string(void);

/* Number of SDMA engines the library can drive directly (0 if none): the
 * copy engines of the Background's DMA Engines section, each executing one
 * copy at a time. */
int hoccl_sdma_engine_count(void);

/* ---- collectives --------------------------------------------------------
 * Reductions are sums.  The paper leaves reductions to SM-side execution and
 * fixes no order, so the library defines one: ring direction r -> r+1, and
 * the fold for chunk j starts at rank j+1 and ends at rank j,
 *     out = ((x[j+1] + x[j+2]) + ...) + x[j]      (rank indices mod R).
 * int32 adds wrap modulo 2^32; fp32 adds are IEEE binary32 round-to-nearest-
 * even; bf16 inputs are widened exactly to fp32, summed in fp32 in the same
 * order and rounded once to bf16 (round to nearest even).  Every path
 * (ring or direct, any workgroup count, any chunk grouping) follows this
 * order, so results are identical bit for bit. */

/* all-reduce of `count` elements per rank.  A reduction collective, which
 * the paper leaves to SM-side execution (Limitations); here the reduction
 * runs on a chosen number of workgroups and the gather on the SDMA path.
 * The ring splits count into R
 * chunks of c = ceil(count / R) elements (the last may be short or empty);
 * rank j's reduced chunk j is then forwarded around the ring by copy steps.
 * send[r], recv[r]: count elements each. */
hoccl_status_t hoccl_allreduce(const void *const *send, void *const *recv,
                               size_t count, hoccl_dtype_t dtype, int R,
                               hipStream_t stream);

/* reduce-scatter: send[r] holds R * recvcount elements; rank r receives
 * block r (recvcount elements) of the element-wise sum.  A reduction
 * collective (Limitations): it runs as reduction kernels only, with no copy
 * step. */
hoccl_status_t hoccl_reduce_scatter(const void *const *send, void *const *recv,
                                    size_t recvcount, hoccl_dtype_t dtype,
                                    int R, hipStream_t stream);

/* For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The same
 * operation, arguments and results as hoccl_reduce_scatter, bit for bit,
 * but the call allocates nothing and creates no stream or event.  Where the
 * ring keeps partials (bf16 over more than two ranks; int32 / fp32 in
 * place) they live in a static device array of 128 MiB that every device
 * the library runs on holds from initialisation until the process ends.  A
 * call that needs more (R * recvcount * 4 bytes, or 2 for bf16 with
 * bf16_partials, beyond 128 MiB) returns
 * HOCCL_ERR_INVALID_ARG and enqueues nothing; the reduction the
 * configuration picks decides whether any is needed (the direct fold needs
 * none).  The library must already be initialised on the current device
 * (hoccl_init, or any earlier call), else HOCCL_ERR_UNSUPPORTED.  Kernel
 * timing is off for these calls and a one-rank copy runs as a CU copy
 * kernel.  Every such call on a device shares that device's array: calls
 * whose executions overlap on one GPU (on different streams, or in graph
 * replays) race and give wrong results, so the caller orders them. */
hoccl_status_t hoccl_reduce_scatter_noalloc(const void *const *send, void *const *recv,
                                            size_t recvcount, hoccl_dtype_t dtype, int R,
                                            hipStream_t stream);

/* all-gather: send[r] holds sendcount elements; every recv[r] receives the
 * R shards in rank order (R * sendcount elements).  As a traffic matrix
 * (Collective Scheduler, traffic matrix abstraction) C[s][d] = sendcount
 * for every pair: copy-only, moved by the configured copy path (the SDMA
 * engines by default). */
hoccl_status_t hoccl_allgather(const void *const *send, void *const *recv,
                               size_t sendcount, hoccl_dtype_t dtype, int R,
                               hipStream_t stream);

/* point-to-point send/recv, the primitive of the Zero-SM Point-to-Point
 * Executor (intra-node communication: the sender's copy engine writes
 * straight into the receiver's buffer): rank r sends its count elements to rank
 * peers[r] (a host array of R ints; -1 = rank r sends nothing).  A receiver
 * named twice is an argument error; a rank may send to itself (local copy).
 * recv[d] of a rank nobody sends to may be NULL and is left untouched. */
hoccl_status_t hoccl_sendrecv(const void *const *send, void *const *recv,
                              const int *peers, size_t count,
                              hoccl_dtype_t dtype, int R, hipStream_t stream);

/* all-to-all with uniform blocks: block d of send[s] (count elements at
 * offset d * count) lands at block s of recv[d].  The traffic matrix
 * (Collective Scheduler, traffic matrix abstraction) has C[s][d] = count
 * for every pair. */
hoccl_status_t hoccl_alltoall(const void *const *send, void *const *recv,
                              size_t count, hoccl_dtype_t dtype, int R,
                              hipStream_t stream);

/* all-to-all(v): the paper's origin traffic matrix C (Collective
 * Scheduler, traffic matrix abstraction) given directly:
 * C[s][d] = sendcounts[s * R + d]
 * elements move from send[s] + sdispls[s * R + d] to
 * recv[d] + rdispls[s * R + d] (all in elements; host arrays of R*R).
 * Destination ranges must not overlap. */
hoccl_status_t hoccl_alltoallv(const void *const *send,
                               const size_t *sendcounts, const size_t *sdispls,
                               void *const *recv, const size_t *rdispls,
                               hoccl_dtype_t dtype, int R, hipStream_t stream);

/* One ring hop of one rank (a reduction step, Limitations):
 * out[i] = partial[i] + local[i] for i < count,
 * in the arithmetic of the ring fold above, with `partial` the earlier
 * ranks' sum (or, on the first hop, the previous rank's own element) and
 * `local` this rank's contribution.  This is the step each GPU runs per hop
 * when the ranks are GPUs (each hop of the ring reduce-scatter of the
 * paper's collective set), exposed on its own so that one rank's share can
 * be run and timed; the collectives above run it for all R ranks in one
 * launch.  `hop` selects the operand types of a bf16 fold:
 *   HOCCL_HOP_FIRST   partial bf16, out fp32
 *   HOCCL_HOP_MIDDLE  partial fp32, out fp32
 *   HOCCL_HOP_LAST    partial fp32, out bf16 (rounded to nearest even)
 *   HOCCL_HOP_ONLY    partial bf16, out bf16 (a two-rank fold, rounded once)
 * `local` is bf16 throughout.  For int32 and fp32 every operand has the
 * dtype and the four hops compute the same thing.  All three are device
 * pointers of count elements, any alignment (16-byte aligned runs at full
 * speed).  `out` may be `partial` or `local` itself when its element size
 * is the same (the in-place update of a partial); any other overlap is
 * HOCCL_ERR_INVALID_ARG.  Launch shape from workgroups_per_step and
 * threads_per_workgroup as for the collectives; no workspace, no copies,
 * no allocation, so the call may be captured into a graph.  Statistics as
 * for a collective (one reduction launch). */
typedef enum {
    HOCCL_HOP_FIRST = 0,
    HOCCL_HOP_MIDDLE = 1,
    HOCCL_HOP_LAST = 2,
    HOCCL_HOP_ONLY = 3
} hoccl_hop_t;

hoccl_status_t hoccl_ring_hop(const void *partial, const void *local, void *out,
                              size_t count, hoccl_dtype_t dtype, hoccl_hop_t hop,
                              hipStream_t stream);

/* ---- several processes on one device ------------------------------------
 * The paper's runtime IPC-handle exchange (Zero-SM Point-to-Point Executor,
 * intra-node communication): a process exports the allocation holding one
 * of its device buffers, another process on the same device opens it and
 * can then pass the buffer to the collectives above as one of its R
 * pointers.  The handles travel out of band (the PyTorch backend posts
 * them in a mailbox, below).  The exporter must not free the allocation while an
 * importer has it open.
 *
 * Export the allocation that contains device pointer `ptr`: `handle`
 * receives 64 bytes, *offset ptr's byte offset in the allocation and
 * *alloc_bytes its size.  HOCCL_ERR_INVALID_ARG if ptr is not device memory
 * of an allocation; HOCCL_ERR_UNSUPPORTED for allocations of 2 GiB or more,
 * which are not shared. */
hoccl_status_t hoccl_ipc_export(const void *ptr, void *handle, size_t *offset, size_t *alloc_bytes);

/* Open a handle another process exported (each handle is opened once and
 * cached: later calls with the same handle reuse the mapping) and return
 * in *ptr the device address of byte `offset` of that allocation.
 * Allocations of 2 GiB or more are refused (HOCCL_ERR_UNSUPPORTED). */
hoccl_status_t hoccl_ipc_open(const void *handle, size_t offset, size_t alloc_bytes, void **ptr);

/* Close every handle this process opened. */
hoccl_status_t hoccl_ipc_close_all(void);

/* Cross-process mailboxes: the paper's CPU-based cross-process
 * synchronisation (Zero-SM Point-to-Point Executor, intra-node), by which
 * processes that share buffers tell each other that inputs are ready and
 * operations have completed.  A mailbox is a POSIX shared-memory object of
 * `slots` slots, each a 32-bit sequence number plus up to `slot_bytes` of
 * payload.  Host memory only: no device is touched, and these calls work
 * without a GPU.
 *
 * Protocol: a writer posts a payload into a slot with a sequence number;
 * a reader waits until the slot's number has reached the one it expects
 * (numbers compare modulo 2^32, so a slot's numbers should only grow), then
 * reads the payload.  The payload written before the number is visible to
 * any reader that has seen the number.  A slot's writer must not post again
 * until every reader of the previous payload is done with it; the caller's
 * protocol orders that (the PyTorch backend lets a rank post call k + 1
 * only after it has seen call k complete).  Every slot starts at 0.
 *
 * hoccl_mailbox_create makes the object `name` ("/name", as shm_open) and
 * maps it; it fails if the name exists.  hoccl_mailbox_open maps an
 * existing one and takes its geometry from it.  hoccl_mailbox_unlink
 * removes the name (mappings stay valid, so once every process has opened
 * it nothing is left behind when they exit).  hoccl_mailbox_close unmaps
 * and frees the handle.  The handle is owned by the caller; one handle may
 * be used from several threads, but not to post into one slot at once.
 *
 * hoccl_mailbox_wait polls briefly, then sleeps on the slot (a futex on
 * the shared word); it returns HOCCL_ERR_TIMEOUT after timeout_ms.  With
 * timeout_ms 0 it looks once and returns at once (HOCCL_OK or
 * HOCCL_ERR_TIMEOUT), without setting an error string.
 * hoccl_mailbox_read copies the payload into buf (cap bytes) and stores its
 * length in *len; HOCCL_ERR_INVALID_ARG if it does not fit.  Bad names,
 * slots or sizes are HOCCL_ERR_INVALID_ARG; hoccl_last_error_string() says
 * which. */
typedef struct hoccl_mailbox hoccl_mailbox_t;
hoccl_status_t hoccl_mailbox_create(const char *name, unsigned slots, size_t slot_bytes,
                                    hoccl_mailbox_t **box);
hoccl_status_t hoccl_mailbox_open(const char *name, hoccl_mailbox_t **box);
hoccl_status_t hoccl_mailbox_unlink(const char *name);
hoccl_status_t hoccl_mailbox_close(hoccl_mailbox_t *box);
hoccl_status_t hoccl_mailbox_post(hoccl_mailbox_t *box, unsigned slot, unsigned seq,
                                  const void *data, size_t len);
hoccl_status_t hoccl_mailbox_wait(hoccl_mailbox_t *box, unsigned slot, unsigned seq,
                                  unsigned timeout_ms);
hoccl_status_t hoccl_mailbox_read(hoccl_mailbox_t *box, unsigned slot, void *buf, size_t cap,
                                  size_t *len);

/* ---- introspection (tests and tools) ------------------------------------
 * The planner's schedule for a collective: its traffic matrix turned into
 * copy chains and reduction steps (Collective Scheduler, from C to the
 * DMA-engine work queues).  Writes it as JSON into buf
 * (NUL-terminated, truncated to len).  op: 0 all-reduce, 1 reduce-scatter,
 * 2 all-gather, 3 send/recv (peers r -> r+1, last rank sends nothing),
 * 4 all-to-all.  Buffers are named symbolically ("send", "recv", "ws" with
 * rank and byte offset), so no device is needed.  Uses the current
 * configuration.  *needed receives the full length including the NUL
 * (`needed` may be NULL). */
hoccl_status_t hoccl_debug_plan_json(int op, size_t count, hoccl_dtype_t dtype,
                                     int R, char *buf, size_t len,
                                     size_t *needed);

/* The paper's collective scheduler (Collective Scheduler section) on a
 * described multi-node topology, host only.  G GPUs; C: G*G row-major
 * traffic matrix in bytes (C[u*G+v] = bytes from GPU u to GPU v; the
 * diagonal is ignored); node[u]: intra-node (NVLink/xGMI) domain of GPU u;
 * peer[u]: its symmetric peer (-1: none); bw_intra / bw_inter: bandwidth of
 * an intra-node / inter-node edge.  Writes JSON {"T": expanded traffic
 * matrix with forwarding copies (Eq. 2-5), "stages": stage matrices T^s from
 * the Birkhoff-like decomposition (Algorithm 1), "tau": stage durations
 * (Eq. 9-10), "total": their sum (Eq. 11)}.  Buffer conventions as for
 * hoccl_debug_plan_json. */
hoccl_status_t hoccl_debug_schedule_json(int G, const double *C, const int *node, const int *peer,
                                         double bw_intra, double bw_inter, char *buf, size_t len,
                                         size_t *needed);

/* Flow-size-aware chunk order on one DMA engine (Collective Scheduler,
 * flow-size-aware chunk scheduling): flows of bytes[i] are cut
 * into chunk_bytes pieces and order[k] receives the flow of the k-th chunk
 * (at most cap entries); *n receives the total number of chunks. */
hoccl_status_t hoccl_debug_interleave(int nflows, const double *bytes, double chunk_bytes, int *order,
                                      size_t cap, size_t *n);

/* Streaming ceilings of the memory system, the rates the collectives'
 * kernels are read against (the paper reports bandwidth against what the
 * hardware moves, Evaluation, Communication Benchmark).  One launch over
 * `bytes` bytes per operand: mode 0 reads a; 1 writes c; 2 copies a to c;
 * 3 writes c = a + b (fp32); 4 adds 1 to c in place (fp32); 5 and 6 are
 * modes 2 and 3 with non-temporal stores (faster to HBM once the data
 * outgrows the Infinity Cache, slower while it fits).  Device
 * pointers, 16-byte aligned, `bytes` a multiple of 16; mode 0 needs c as a
 * 4-byte sink it never writes in practice.  Launch shape from
 * workgroups_per_step and threads_per_workgroup (automatic: about 4
 * vectors per thread).  Statistics report the bytes moved. */
hoccl_status_t hoccl_debug_stream_ceiling(int mode, const void *a, const void *b, void *c, size_t bytes,
                                          hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* HOCCL_H */
