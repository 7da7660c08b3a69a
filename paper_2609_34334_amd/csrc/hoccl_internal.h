// Internal types shared by the planner, the executor and the kernels.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/hoccl.h"

namespace hoccl {

enum class Op : int {
    AllReduce = 0,
    ReduceScatter = 1,
    AllGather = 2,
    SendRecv = 3,
    AllToAll = 4,
    AllToAllV = 5
};

// A symbolic buffer position: which buffer (send[rank], recv[rank] or the
// library workspace) and a byte offset into it.  Plans are built on these so
// the planner never touches device memory and can be dumped and replayed on
// the host.
enum BufKind : uint8_t { BUF_NONE = 0, BUF_SEND = 1, BUF_RECV = 2, BUF_WS = 3 };

struct BufRef {
    uint8_t kind = BUF_NONE;
    int rank = 0;
    size_t off = 0;  // bytes
};

// Element types a reduction step reads and writes.  The local contribution
// (in1) is always of the collective's dtype; in0 and out are either the
// dtype itself or the accumulator type (fp32 for bf16, the dtype otherwise).
enum Phase : int {
    PH_FIRST = 0,   // in0 = x[j+1] (dtype),  in1 = x[j+2],  out = partial (acc)
    PH_MIDDLE = 1,  // in0 = partial (acc),   in1 = x[r],    out = partial (acc)
    PH_LAST = 2,    // in0 = partial (acc),   in1 = x[j],    out = recv (dtype)
    PH_ONLY = 3     // R == 2: in0 = x[j+1],  in1 = x[j],    out = recv (dtype)
};

struct ReduceSeg {
    BufRef in0, in1, out;
    std::vector<BufRef> more;  // further contributions, added after in1 in order
    size_t n = 0;  // elements
};

// One ring step: every rank adds its contribution to the partial it
// received; one kernel launch covers all ranks' segments of the step.  A
// fused step folds `hops` consecutive ring hops in one launch: each segment
// adds in1 and then the `more` contributions to its partial, which stays in
// registers between the adds.
struct ReduceStep {
    Phase phase = PH_MIDDLE;
    int group = 0;
    int step = 0;   // the first ring hop the launch performs
    int hops = 1;
    std::vector<ReduceSeg> segs;
};

// Ring hops one fused launch may fold (contributions per segment).
constexpr int kMaxHops = 8;

// Direct reduction: one launch folds all R inputs of every chunk in the ring
// order.  Chunk j spans elements [j*c, min(total, (j+1)*c)) of the inputs;
// its result goes to recv[j] at out_off(j) (reduce-scatter) or to every
// recv[r] at the chunk's own offset (all-reduce, write_all).
struct FoldStep {
    size_t c = 0;        // chunk length in elements
    size_t total = 0;    // input elements per rank covered by the fold
    bool write_all = false;
    bool out_at_chunk = false;  // reduce-scatter: recv[j] at 0; else j*c
};

// One copy: `bytes` from src to dst.  Copies with the same chain run in
// order (the ring hops of one chunk); different chains are independent.  A
// copy with group >= 0 may only start once the reduction of that group has
// finished (all-reduce's gather phase).  `level` is the copy's position in
// its chain, used to batch independent copies into one CU-copy launch.
struct CopyOp {
    BufRef dst, src;
    size_t bytes = 0;
    int chain = 0;
    int group = -1;
    int level = 0;
    int stage = -1;  // all-to-all stage of the collective scheduler, or -1
};

struct Plan {
    Op op = Op::AllReduce;
    hoccl_dtype_t dtype = HOCCL_FP32;
    int R = 1;
    size_t count = 0;
    int ngroups = 1;
    std::vector<ReduceStep> reduce_steps;  // in launch order, grouped
    bool has_fold = false;
    FoldStep fold;
    std::vector<CopyOp> copies;            // in issue order
    int nchains = 0;
    size_t ws_bytes = 0;                   // workspace the plan needs
    bool bf16_partials = false;            // bf16 partials, rounded at every add
    unsigned long long hbm_bytes = 0;      // algorithmic HBM bytes
    unsigned long long copy_bytes = 0;
};

struct PlanOptions {
    bool allgather_direct = false;
    int allreduce_groups = 1;  // 0: automatic (plan_allreduce)
    size_t chunk_bytes = 0;
    bool in_place = false;
    hoccl_reduce_algo_t algo = HOCCL_REDUCE_RING;
    // Ring reductions run group by group, each group's fp32 partials taking
    // at most this many bytes (0: one group), so that they stay in the
    // last-level cache from one step to the next.
    size_t group_partial_bytes = 0;
    // Ring hops per reduction launch (0 or 1: one; at most kMaxHops).
    int fused_hops = 1;
    // All-to-all(v) copy schedule (hoccl_config_t.a2a_schedule): 0 byte-
    // balanced chains; 1 and 2 the stages of the collective scheduler's
    // decomposition (copies tagged with their stage; 2 runs them serially).
    int a2a_schedule = 0;
    // bf16 reductions keep their partials in bf16, rounding every addition
    // (hoccl_config_t.bf16_partials).
    bool bf16_partials = false;
};

// HOCCL_REDUCE_AUTO folds directly up to this many ranks.  On one GPU the
// fold moves (R+1) elements per reduce-scatter output element against the
// ring's 2(R-1) (plus the fp32 partials of bf16), so it is the faster
// schedule at every size measured; beyond this rank count the ring is used.
constexpr int kDirectMaxRanks = 64;
bool use_direct(hoccl_reduce_algo_t algo, int R);

size_t dtype_size(hoccl_dtype_t dt);
// Bytes of one partial-sum element: 4 (fp32 for bf16), 2 for bf16 with
// bf16 partials.
size_t acc_size(hoccl_dtype_t dt, bool bf16_partials = false);

// Planner entry points (plan.cpp); pure host code.
Plan plan_allreduce(size_t count, hoccl_dtype_t dt, int R, const PlanOptions &o);
Plan plan_reduce_scatter(size_t recvcount, hoccl_dtype_t dt, int R, const PlanOptions &o);
Plan plan_allgather(size_t sendcount, hoccl_dtype_t dt, int R, const PlanOptions &o);
Plan plan_sendrecv(size_t count, hoccl_dtype_t dt, int R, const int *peers,
                   const PlanOptions &o);
Plan plan_alltoall(size_t count, hoccl_dtype_t dt, int R, const PlanOptions &o);
Plan plan_alltoallv(const size_t *counts, const size_t *sdispls, const size_t *rdispls,
                    hoccl_dtype_t dt, int R, const PlanOptions &o);

// Assigns each chain of a plan to one of `queues` queues so that the bytes
// per queue are balanced (largest chain first, onto the least loaded queue).
std::vector<int> assign_chains(const Plan &p, int queues);

std::string plan_to_json(const Plan &p);

// ---- kernels (kernels.hip) -------------------------------------------------

constexpr int kMaxReduceSegs = 64;
constexpr int kMaxCopySegs = 128;
constexpr int kMaxRanks = 64;

// Each kernel's argument struct has a fixed number of slots.  The executor
// fills the largest form; the launchers pass the smallest form that holds the
// launch's segments.  The HIP runtime stages the arguments of every launch
// that has not started yet, and the enqueueing thread waits once about 1 MB
// of them is pending (measured on MI355X).  With 2 KiB of slots, some 450
// launches queued behind unfinished work stall the caller; an 8-rank ring
// step passes 264 bytes (plus the runtime's own 256 bytes of hidden
// arguments), and about 1000 fit.
struct RSegArg {
    const void *in0;
    const void *in1;
    void *out;
    uint64_t n;
};
template <int CAP>
struct ReduceArgsT {
    RSegArg seg[CAP];
    int nseg;
};
using ReduceArgs = ReduceArgsT<kMaxReduceSegs>;

// A fused step's segment: the partial (or first operand) in0, then nloc
// contributions loc[0..nloc) added in order, into out.
struct MSegArg {
    const void *in0;
    const void *loc[kMaxHops];
    void *out;
    uint64_t n;
    int nloc;
};
constexpr int kMaxMultiSegs = 32;  // 32 segments: 3.1 KiB of arguments
template <int CAP>
struct MultiArgsT {
    MSegArg seg[CAP];
    int nseg;
};
using MultiArgs = MultiArgsT<kMaxMultiSegs>;

struct CSegArg {
    const void *src;
    void *dst;
    uint64_t bytes;
};
template <int CAP>
struct CopyArgsT {
    CSegArg seg[CAP];
    int nseg;
};
using CopyArgs = CopyArgsT<kMaxCopySegs>;

template <int CAP>
struct FoldArgsT {
    const void *in[CAP];
    void *out[CAP];
    uint64_t c;
    uint64_t total;
    int R;
    int write_all;
    int out_at_chunk;
};
using FoldArgs = FoldArgsT<kMaxRanks>;

// The stream side of one proxy operation's start/finish handshake.  The
// three flags are host memory mapped for the device.
struct HandshakeArgs {
    uint32_t *start;        // the kernel writes start_value; the proxy clears it
    uint32_t *finish;       // the proxy writes finish_value; the kernel clears it
    uint32_t *status;       // the kernel writes 1 here if it gave up waiting
    uint32_t start_value;
    uint32_t finish_value;
    uint64_t limit_ticks;   // give up after this many device wall-clock ticks
};

// bf16_partials: a bf16 step keeps every operand and result in bf16 (the
// middle and last phases read, and the first and middle write, bf16
// partials); a bf16 fold, or fused step, rounds after every addition.
hipError_t launch_reduce_step(hoccl_dtype_t dt, Phase ph, const ReduceArgs &a, int wg,
                              int threads, hipStream_t s, bool bf16_partials = false);
hipError_t launch_fold(hoccl_dtype_t dt, const FoldArgs &a, int wg, int threads,
                       hipStream_t s, bool bf16_partials = false);
hipError_t launch_multihop(hoccl_dtype_t dt, Phase ph, const MultiArgs &a, int wg, int threads,
                           hipStream_t s, bool bf16_partials = false);
hipError_t launch_copy(const CopyArgs &a, int wg, int threads, hipStream_t s);

// Work one thread does in one pass of each kernel's main loop (elements of
// the collective's dtype, or bytes for the copy kernel).
size_t reduce_step_elems_per_thread(hoccl_dtype_t dt, Phase ph, bool bf16_partials = false);
size_t fold_elems_per_thread(hoccl_dtype_t dt);
size_t multihop_elems_per_thread(hoccl_dtype_t dt);
size_t copy_bytes_per_thread();
hipError_t launch_handshake(const HandshakeArgs &a, hipStream_t s);

// The static device scratch of hoccl_reduce_scatter_noalloc (scratch.hip):
// its size, and this device's address of it (call with the device current).
constexpr size_t kScratchBytes = (size_t)128 << 20;
hipError_t scratch_address(void **out);

}  // namespace hoccl
