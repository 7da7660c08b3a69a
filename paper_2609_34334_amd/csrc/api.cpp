// C ABI of libhoccl: argument validation, configuration, the stream manager
// and the schedule executor.
//
// Stream manager (Stream Manager section of the paper): a collective is
// enqueued on the caller's stream `s`.  Reduction kernels run on `s` itself.
// Copy steps run either
//   * by the copy proxy (proxy.cpp), which drives chosen SDMA engines itself
//     and is ordered with `s` by the start/finish flag handshake -- the
//     default, and the only path whose copies occupy no compute unit;
//   * on the library's copy streams as hipMemcpyAsync(DeviceToDeviceNoCU),
//     where the HIP runtime decides what executes the copy: `s` records a
//     fork event that each copy stream waits on before its first copy, and
//     `s` waits on a join event of every copy stream it used, so the
//     collective sits in `s` exactly where it was enqueued;
//   * or as CU copy kernels on `s`.
// All-reduce's gather copies of group g wait on an event recorded on `s`
// right after group g's last reduction step, so the copies of one group
// overlap the CU reduction of the next (the paper's per-chunk buffer state
// machine, reduced to "partial ready" / "final ready").
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "ceilings.h"
#include "errors.h"
#include "hoccl_internal.h"
#include "proxy.h"
#include "schedule.h"

namespace hoccl {

namespace {

thread_local std::string t_err;
thread_local hoccl_stats_t t_stats;

struct TimingPair {
    hipEvent_t a, b;
};

struct DeviceState {
    // Held by every call while it plans and enqueues on this device, so
    // calls from several host threads take turns.
    std::recursive_mutex call_mu;
    int device = -1;
    int num_cus = 0;
    std::vector<hipStream_t> copy_streams;
    hipEvent_t ev_fork = nullptr;
    std::vector<hipEvent_t> ev_group;
    std::vector<hipEvent_t> ev_join;
    void *ws = nullptr;
    size_t ws_cap = 0;
    hipEvent_t ws_event = nullptr;
    hipStream_t ws_last_stream = nullptr;
    bool ws_captured = false;        // a graph captured the current workspace
    std::vector<void *> ws_retired;  // older workspaces captured graphs may replay into
    std::vector<TimingPair> timing_pool;
    size_t timing_used = 0;
    Proxy *proxy = nullptr;
    std::string proxy_why;  // why the proxy could not be created
    void *scratch = nullptr;  // this device's address of the static scratch
    std::string scratch_why;  // why it has none
};

std::mutex g_mu;
std::map<int, DeviceState *> g_states;
hoccl_config_t g_cfg;
bool g_cfg_init = false;
bool g_debug = false;  // HOCCL_DEBUG=1: log every executed plan to stderr

void set_err(const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_err = buf;
}

#define HIP_TRY(call)                                                                     \
    do {                                                                                  \
        hipError_t e_ = (call);                                                           \
        if (e_ != hipSuccess) {                                                           \
            set_err("%s failed: %s (%s:%d)", #call, hipGetErrorString(e_), __FILE__, __LINE__); \
            return HOCCL_ERR_HIP;                                                         \
        }                                                                                 \
    } while (0)

#define TRY(expr)                          \
    do {                                   \
        hoccl_status_t st_ = (expr);       \
        if (st_ != HOCCL_OK) return st_;   \
    } while (0)

hoccl_config_t default_config() {
    hoccl_config_t c;
    std::memset(&c, 0, sizeof c);
    c.workgroups_per_step = 0;
    c.threads_per_workgroup = 256;
    c.chunk_bytes = 0;
    c.copy_streams = 8;
    c.sdma_engines = 0;
    c.copy_path = HOCCL_COPY_AUTO;
    c.allgather_direct = 1;
    c.allreduce_chunk_groups = 0;
    c.reduce_algo = HOCCL_REDUCE_AUTO;
    c.kernel_timing = 0;
    c.proxy_timeout_ms = 10000;
    c.proxy_handshake = -1;
    c.ring_group_bytes = 0;
    c.proxy_wait_limit_us = 0;
    c.fused_hops = 1;
    c.a2a_schedule = 0;
    c.proxy_slice_bytes = 0;
    c.bf16_partials = 0;
    return c;
}

bool config_valid(const hoccl_config_t &c) {
    if (c.workgroups_per_step < 0 || c.workgroups_per_step > (1 << 20)) return false;
    if (c.threads_per_workgroup != 0 &&
        (c.threads_per_workgroup < 64 || c.threads_per_workgroup > 1024 ||
         c.threads_per_workgroup % 64 != 0))
        return false;
    if (c.copy_streams < 0 || c.copy_streams > 16) return false;
    if (c.sdma_engines < 0 || c.sdma_engines > 32) return false;
    if ((int)c.copy_path < HOCCL_COPY_AUTO || (int)c.copy_path > HOCCL_COPY_HIP) return false;
    if (c.allreduce_chunk_groups < 0 || c.allreduce_chunk_groups > 1024) return false;
    if ((int)c.reduce_algo < HOCCL_REDUCE_RING || (int)c.reduce_algo > HOCCL_REDUCE_AUTO) return false;
    if (c.chunk_bytes != 0 && c.chunk_bytes < 4096) return false;
    if (c.proxy_handshake < -1 || c.proxy_handshake > 2) return false;
    if (c.fused_hops < 0 || c.fused_hops > kMaxRanks) return false;
    if (c.a2a_schedule < 0 || c.a2a_schedule > 2) return false;
    if (c.proxy_slice_bytes != 0 && c.proxy_slice_bytes != SIZE_MAX &&
        (c.proxy_slice_bytes < ((size_t)64 << 10) || c.proxy_slice_bytes % 4096 != 0))
        return false;
    if (c.bf16_partials != 0 && c.bf16_partials != 1) return false;
    return true;
}

long env_long(const char *name, long dflt) {
    const char *v = std::getenv(name);
    if (!v || !*v) return dflt;
    char *end = nullptr;
    long x = std::strtol(v, &end, 0);
    return (end && *end == 0) ? x : dflt;
}

void load_config_locked() {
    if (g_cfg_init) return;
    hoccl_config_t c = default_config();
    c.workgroups_per_step = (int)env_long("HOCCL_WG_PER_STEP", c.workgroups_per_step);
    c.threads_per_workgroup = (int)env_long("HOCCL_THREADS_PER_WG", c.threads_per_workgroup);
    c.chunk_bytes = (size_t)env_long("HOCCL_CHUNK_BYTES", (long)c.chunk_bytes);
    c.copy_streams = (int)env_long("HOCCL_COPY_STREAMS", c.copy_streams);
    c.sdma_engines = (int)env_long("HOCCL_SDMA_ENGINES", c.sdma_engines);
    c.allgather_direct = (int)env_long("HOCCL_AG_DIRECT", c.allgather_direct);
    c.allreduce_chunk_groups = (int)env_long("HOCCL_AR_GROUPS", c.allreduce_chunk_groups);
    c.kernel_timing = (int)env_long("HOCCL_KERNEL_TIMING", c.kernel_timing);
    c.proxy_handshake = (int)env_long("HOCCL_PROXY_HANDSHAKE", c.proxy_handshake);
    c.proxy_wait_limit_us = (unsigned)env_long("HOCCL_PROXY_WAIT_LIMIT_US", c.proxy_wait_limit_us);
    c.fused_hops = (int)env_long("HOCCL_FUSED_HOPS", c.fused_hops);
    c.a2a_schedule = (int)env_long("HOCCL_A2A_SCHEDULE", c.a2a_schedule);
    c.bf16_partials = (int)env_long("HOCCL_BF16_PARTIALS", c.bf16_partials);
    if (const char *v = std::getenv("HOCCL_RING_GROUP_BYTES")) c.ring_group_bytes = std::strtoull(v, nullptr, 0);
    if (const char *v = std::getenv("HOCCL_PROXY_SLICE_BYTES")) c.proxy_slice_bytes = std::strtoull(v, nullptr, 0);
    if (const char *v = std::getenv("HOCCL_COPY_PATH")) {
        if (!std::strcmp(v, "hip")) c.copy_path = HOCCL_COPY_HIP;
        else if (!std::strcmp(v, "sdma") || !std::strcmp(v, "engines")) c.copy_path = HOCCL_COPY_SDMA;
        else if (!std::strcmp(v, "kernel")) c.copy_path = HOCCL_COPY_KERNEL;
        else c.copy_path = HOCCL_COPY_AUTO;
    }
    if (const char *v = std::getenv("HOCCL_REDUCE_ALGO")) {
        if (!std::strcmp(v, "ring")) c.reduce_algo = HOCCL_REDUCE_RING;
        else if (!std::strcmp(v, "direct")) c.reduce_algo = HOCCL_REDUCE_DIRECT;
        else c.reduce_algo = HOCCL_REDUCE_AUTO;
    }
    if (!config_valid(c)) c = default_config();
    g_debug = env_long("HOCCL_DEBUG", 0) != 0;
    g_cfg = c;
    g_cfg_init = true;
}

hoccl_config_t config() {
    std::lock_guard<std::mutex> lk(g_mu);
    load_config_locked();
    return g_cfg;
}

void destroy_state(DeviceState *st) {
    if (!st) return;
    int prev = 0;
    (void)hipGetDevice(&prev);
    (void)hipSetDevice(st->device);
    (void)hipDeviceSynchronize();
    delete st->proxy;
    for (auto s : st->copy_streams) (void)hipStreamDestroy(s);
    if (st->ev_fork) (void)hipEventDestroy(st->ev_fork);
    for (auto e : st->ev_group) (void)hipEventDestroy(e);
    for (auto e : st->ev_join) (void)hipEventDestroy(e);
    if (st->ws_event) (void)hipEventDestroy(st->ws_event);
    if (st->ws) (void)hipFree(st->ws);
    for (void *w : st->ws_retired) (void)hipFree(w);
    for (auto &tp : st->timing_pool) {
        (void)hipEventDestroy(tp.a);
        (void)hipEventDestroy(tp.b);
    }
    (void)hipSetDevice(prev);
    delete st;
}

hoccl_status_t create_state(int device, DeviceState **out) {
    DeviceState *st = new DeviceState();
    st->device = device;
    auto fail = [&](hoccl_status_t s) {
        destroy_state(st);
        return s;
    };
    hipDeviceProp_t prop;
    hipError_t e = hipGetDeviceProperties(&prop, device);
    if (e != hipSuccess) {
        set_err("hipGetDeviceProperties(%d): %s", device, hipGetErrorString(e));
        return fail(HOCCL_ERR_HIP);
    }
    st->num_cus = prop.multiProcessorCount;
    const int K = 16;  // the most copy streams any configuration may use
    // Plain streams on the runtime's shared hardware queues.  Giving each its
    // own queue (a CU-masked stream) was measured slower for SDMA copies:
    // the pipeline send/recv schedule took 39.7 ms instead of 9.8 ms.
    for (int k = 0; k < K; ++k) {
        hipStream_t s = nullptr;
        e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
        if (e != hipSuccess) {
            set_err("hipStreamCreateWithFlags: %s", hipGetErrorString(e));
            return fail(HOCCL_ERR_HIP);
        }
        st->copy_streams.push_back(s);
        hipEvent_t ev;
        e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
        if (e != hipSuccess) {
            set_err("hipEventCreateWithFlags: %s", hipGetErrorString(e));
            return fail(HOCCL_ERR_HIP);
        }
        st->ev_join.push_back(ev);
    }
    if ((e = hipEventCreateWithFlags(&st->ev_fork, hipEventDisableTiming)) != hipSuccess ||
        (e = hipEventCreateWithFlags(&st->ws_event, hipEventDisableTiming)) != hipSuccess) {
        set_err("hipEventCreateWithFlags: %s", hipGetErrorString(e));
        return fail(HOCCL_ERR_HIP);
    }
    // The static scratch of the entry point that allocates nothing: this
    // device's address of it, taken once here with the device current.
    // A failure leaves only that entry point unusable.
    if ((e = scratch_address(&st->scratch)) != hipSuccess) {
        (void)hipGetLastError();  // handled: do not leave it for the next caller
        st->scratch = nullptr;
        st->scratch_why = std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e);
    }
    st->proxy = Proxy::create(device, &st->proxy_why);  // null when the engines cannot be driven
    *out = st;
    return HOCCL_OK;
}

// `capturing`: the caller's stream is capturing a graph, or the caller must
// not allocate.  Creating the state then would synchronise the device and
// allocate, so it is refused.
hoccl_status_t get_state(DeviceState **out, bool capturing = false) {
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    std::lock_guard<std::mutex> lk(g_mu);
    load_config_locked();
    auto it = g_states.find(dev);
    if (it != g_states.end()) {
        *out = it->second;
        return HOCCL_OK;
    }
    if (capturing) {
        set_err("the library is not initialised on device %d and cannot be during stream "
                "capture or in a call that allocates nothing: call hoccl_init (or any "
                "collective) first", dev);
        return HOCCL_ERR_UNSUPPORTED;
    }
    DeviceState *st = nullptr;
    TRY(create_state(dev, &st));
    g_states[dev] = st;
    *out = st;
    return HOCCL_OK;
}

// ---- execution ------------------------------------------------------------------

PlanOptions options_from(const hoccl_config_t &cfg, bool in_place);

struct Buffers {
    const void *const *send;
    void *const *recv;
    void *ws;
};

inline void *resolve(const BufRef &b, const Buffers &B) {
    switch (b.kind) {
    case BUF_SEND: return (char *)B.send[b.rank] + b.off;
    case BUF_RECV: return (char *)B.recv[b.rank] + b.off;
    case BUF_WS: return (char *)B.ws + b.off;
    default: return nullptr;
    }
}

// During stream capture nothing is allocated: the call needs a workspace
// that an earlier call outside capture already made large enough.  A
// workspace a graph has captured is never freed before finalize, since any
// replay of that graph still writes into it.
hoccl_status_t ensure_ws(DeviceState &st, size_t bytes, bool capturing) {
    if (bytes <= st.ws_cap) {
        st.ws_captured = st.ws_captured || capturing;
        return HOCCL_OK;
    }
    if (capturing) {
        set_err("this call needs a %zu-byte workspace but %zu bytes are allocated, and the "
                "workspace cannot grow during stream capture: make the same call once "
                "outside capture first", bytes, st.ws_cap);
        return HOCCL_ERR_UNSUPPORTED;
    }
    // Growing the workspace waits for every user of the old one.
    HIP_TRY(hipDeviceSynchronize());
    if (st.ws && st.ws_captured)
        st.ws_retired.push_back(st.ws);
    else if (st.ws)
        HIP_TRY(hipFree(st.ws));
    st.ws_captured = false;
    st.ws = nullptr;
    st.ws_cap = 0;
    st.ws_last_stream = nullptr;
    size_t cap = (bytes + (1u << 20) - 1) & ~((size_t)(1u << 20) - 1);
    hipError_t e = hipMalloc(&st.ws, cap);
    if (e != hipSuccess) {
        st.ws = nullptr;
        set_err("hipMalloc(%zu) for the workspace: %s", cap, hipGetErrorString(e));
        return HOCCL_ERR_NO_MEMORY;
    }
    st.ws_cap = cap;
    return HOCCL_OK;
}

// Workgroups per launch.  An explicit budget wins.  Otherwise enough for
// about one pass of the kernel's main loop per thread in the largest launch,
// between one workgroup per CU and 64 per CU (16384 on MI355X): measured on
// the headline bf16 ring and fold, the streaming kernels keep gaining up to
// about one pass per thread and lose nothing beyond.
int workgroups_for(const DeviceState &st, const hoccl_config_t &cfg, unsigned long long passes,
                   int threads) {
    if (cfg.workgroups_per_step > 0) return cfg.workgroups_per_step;
    unsigned long long wg = (passes + (unsigned long long)threads - 1) / (unsigned long long)threads;
    unsigned long long lo = (unsigned long long)st.num_cus, hi = 64ull * st.num_cus;
    return (int)std::min(hi, std::max(lo, wg));
}

int auto_workgroups(const DeviceState &st, const hoccl_config_t &cfg, const Plan &p, int threads) {
    if (cfg.workgroups_per_step > 0) return cfg.workgroups_per_step;
    unsigned long long passes = 0;  // thread passes of the largest launch
    auto need = [&](unsigned long long work, size_t per_thread) {
        passes = std::max(passes, (work + per_thread - 1) / per_thread);
    };
    for (const ReduceStep &s : p.reduce_steps) {
        unsigned long long n = 0;
        for (const ReduceSeg &g : s.segs) n += g.n;
        need(n, s.hops > 1 ? multihop_elems_per_thread(p.dtype)
                           : reduce_step_elems_per_thread(p.dtype, s.phase, p.bf16_partials));
    }
    if (p.has_fold) need(p.fold.total, fold_elems_per_thread(p.dtype));
    if (cfg.copy_path == HOCCL_COPY_KERNEL)
        for (const CopyOp &c : p.copies) need((unsigned long long)c.bytes * p.R, copy_bytes_per_thread());
    return workgroups_for(st, cfg, passes, threads);
}

// Launches timed between two reads of hoccl_get_kernel_times; later ones go
// untimed, so a caller that never reads does not grow the event pool
// without bound.
constexpr size_t kMaxTimedLaunches = (size_t)1 << 16;

hoccl_status_t timed_begin(DeviceState &st, const hoccl_config_t &cfg, hipStream_t s,
                           TimingPair **tp) {
    *tp = nullptr;
    if (!cfg.kernel_timing || st.timing_used >= kMaxTimedLaunches) return HOCCL_OK;
    if (st.timing_used == st.timing_pool.size()) {
        TimingPair p;
        HIP_TRY(hipEventCreate(&p.a));
        HIP_TRY(hipEventCreate(&p.b));
        st.timing_pool.push_back(p);
    }
    *tp = &st.timing_pool[st.timing_used++];
    HIP_TRY(hipEventRecord((*tp)->a, s));
    return HOCCL_OK;
}

hoccl_status_t timed_end(TimingPair *tp, hipStream_t s) {
    if (tp) HIP_TRY(hipEventRecord(tp->b, s));
    return HOCCL_OK;
}

// SDMA engines the copy proxy may use.  sdma_engines 0 is the automatic
// budget: the most engines whose copies cost a concurrent bf16 8192^3 GEMM
// at most 2% at the upper end of a 95% interval (100 paired runs each) on
// the FSDP all-gather, the pipeline send/recv schedule and the EP
// all-to-all(v).  Measured: 4 engines (about 220 GB/s of copies) cost it
// 0.0-0.1% (upper bounds 0.6-0.8%); 5 and 6 engines up to 1.6% (upper
// bound 2.3%); 8 engines 1.6-1.9% (upper bound 2.7%); all 16 (650 GB/s)
// 4.6-6.0%.  The GEMM's loss follows the copies' aggregate rate.
constexpr int kAutoSdmaEngines = 4;

int engine_budget(const hoccl_config_t &cfg) {
    return cfg.sdma_engines > 0 ? cfg.sdma_engines : kAutoSdmaEngines;
}

// Smallest piece of the proxy's balanced issue (0 asks the proxy to issue
// every copy at once).  Freeing a large device allocation slows SDMA
// engine 1 to about half its rate for tens of ms per GiB freed; with every
// copy issued at once, an all-gather on all 16 engines then waits for that
// engine (58 instead of 94 GB/s per rank).  Pieces pulled by the engines,
// with a finish-time gate, give the slowed engine only what it can finish
// (94 GB/s).  Automatic: balanced from kBalancedMinEngines engines up, for
// operations that move at least kBalancedMinBytesPerEngine per engine.  The
// automatic budget of 4 (engines 2-5, never slowed by the release) issues
// every copy at once: balanced issue there raised a concurrent GEMM's loss
// beside the FSDP all-gather from 0.8-1.5% to 1.4-2.1% (three alternating
// runs of 100 pairs) and made the EP all-to-all(v) 1.7% slower.  Below
// 64 MiB per engine it cost more than a slowed engine could: a 32 MiB
// message on 16 engines took 123-146 us against 113-131.
constexpr size_t kProxySliceBytes = (size_t)4 << 20;
constexpr int kBalancedMinEngines = 8;
constexpr unsigned long long kBalancedMinBytesPerEngine = 64ull << 20;

size_t proxy_slice(const hoccl_config_t &cfg, unsigned long long copy_bytes) {
    if (cfg.proxy_slice_bytes == SIZE_MAX) return 0;
    if (cfg.proxy_slice_bytes) return cfg.proxy_slice_bytes;
    const int E = engine_budget(cfg);
    return E >= kBalancedMinEngines && copy_bytes >= (unsigned long long)E * kBalancedMinBytesPerEngine
               ? kProxySliceBytes
               : 0;
}

// With record_groups, an event is recorded on s after each group's last
// reduction step: gates[g] when given, else the library's ev_group[g].
hoccl_status_t run_reductions(DeviceState &st, const hoccl_config_t &cfg, const Plan &p,
                              const Buffers &B, hipStream_t s, int wg, int threads,
                              bool record_groups, const std::vector<hipEvent_t> *gates = nullptr) {
    for (size_t i = 0; i < p.reduce_steps.size(); ++i) {
        const ReduceStep &step = p.reduce_steps[i];
        // A fused step: every segment's partial plus its contributions in
        // order, up to kMaxMultiSegs segments per launch.
        for (size_t b = 0; step.hops > 1 && b < step.segs.size(); b += kMaxMultiSegs) {
            MultiArgs a;
            std::memset(&a, 0, sizeof a);
            int ns = (int)std::min<size_t>(kMaxMultiSegs, step.segs.size() - b);
            for (int k = 0; k < ns; ++k) {
                const ReduceSeg &g = step.segs[b + (size_t)k];
                a.seg[k].in0 = resolve(g.in0, B);
                a.seg[k].loc[0] = resolve(g.in1, B);
                for (size_t m = 0; m < g.more.size(); ++m) a.seg[k].loc[m + 1] = resolve(g.more[m], B);
                a.seg[k].nloc = 1 + (int)g.more.size();
                a.seg[k].out = resolve(g.out, B);
                a.seg[k].n = g.n;
            }
            a.nseg = ns;
            TimingPair *tp;
            TRY(timed_begin(st, cfg, s, &tp));
            HIP_TRY(launch_multihop(p.dtype, step.phase, a, wg, threads, s, p.bf16_partials));
            TRY(timed_end(tp, s));
            t_stats.reduce_launches++;
        }
        for (size_t b = 0; step.hops == 1 && b < step.segs.size(); b += kMaxReduceSegs) {
            ReduceArgs a;
            std::memset(&a, 0, sizeof a);
            int ns = (int)std::min<size_t>(kMaxReduceSegs, step.segs.size() - b);
            for (int k = 0; k < ns; ++k) {
                const ReduceSeg &g = step.segs[b + (size_t)k];
                a.seg[k].in0 = resolve(g.in0, B);
                a.seg[k].in1 = resolve(g.in1, B);
                a.seg[k].out = resolve(g.out, B);
                a.seg[k].n = g.n;
            }
            a.nseg = ns;
            TimingPair *tp;
            TRY(timed_begin(st, cfg, s, &tp));
            HIP_TRY(launch_reduce_step(p.dtype, step.phase, a, wg, threads, s, p.bf16_partials));
            TRY(timed_end(tp, s));
            t_stats.reduce_launches++;
        }
        bool last_of_group = (i + 1 == p.reduce_steps.size()) ||
                             p.reduce_steps[i + 1].group != step.group;
        if (record_groups && last_of_group && gates) {
            HIP_TRY(hipEventRecord((*gates)[(size_t)step.group], s));
        } else if (record_groups && last_of_group) {
            while ((int)st.ev_group.size() <= step.group) {
                hipEvent_t ev;
                HIP_TRY(hipEventCreateWithFlags(&ev, hipEventDisableTiming));
                st.ev_group.push_back(ev);
            }
            HIP_TRY(hipEventRecord(st.ev_group[(size_t)step.group], s));
        }
    }
    if (p.has_fold) {
        FoldArgs a;
        std::memset(&a, 0, sizeof a);
        for (int r = 0; r < p.R; ++r) {
            a.in[r] = B.send[r];
            a.out[r] = B.recv[r];
        }
        a.c = p.fold.c;
        a.total = p.fold.total;
        a.R = p.R;
        a.write_all = p.fold.write_all ? 1 : 0;
        a.out_at_chunk = p.fold.out_at_chunk ? 1 : 0;
        TimingPair *tp;
        TRY(timed_begin(st, cfg, s, &tp));
        HIP_TRY(launch_fold(p.dtype, a, wg, threads, s, p.bf16_partials));
        TRY(timed_end(tp, s));
        t_stats.reduce_launches++;
    }
    return HOCCL_OK;
}

// A single chain (one send/recv message, one copy) runs on the caller's
// stream itself and needs no event: 14.6 us for a 4 KiB message against
// 50.8 us through a forked copy stream.  Otherwise the chains go to the
// library's copy streams (queues 1..K), forked from the caller's stream by
// an event recorded at the first fork or, for all-reduce's gather, started
// by the event of the reduction group they wait for, and joined back by one
// event each; keeping one of them on the caller's stream was measured
// 5-30% slower for those.
hoccl_status_t run_copies_hip(DeviceState &st, const hoccl_config_t &cfg, const Plan &p,
                               const Buffers &B, hipStream_t s) {
    int K = std::max(1, std::min(cfg.copy_streams ? cfg.copy_streams : 8,
                                 (int)st.copy_streams.size()));
    std::vector<int> q;
    if (p.nchains == 1) {
        K = 1;
        q.assign(1, 0);
    } else {
        q = assign_chains(p, K);
        for (int &x : q) ++x;  // queue 0 (the caller's stream) stays unused
        ++K;
    }
    std::vector<int> started((size_t)K, 0), waited((size_t)K, -1);
    bool forked = false;
    for (const CopyOp &c : p.copies) {
        int k = q[(size_t)c.chain];
        hipStream_t cs = s;
        if (k > 0) {
            cs = st.copy_streams[(size_t)(k - 1)];
            if (!started[(size_t)k]) {
                if (c.group < 0) {
                    if (!forked) {
                        HIP_TRY(hipEventRecord(st.ev_fork, s));
                        forked = true;
                    }
                    HIP_TRY(hipStreamWaitEvent(cs, st.ev_fork, 0));
                }
                started[(size_t)k] = 1;
            }
            if (c.group >= 0 && waited[(size_t)k] < c.group) {
                HIP_TRY(hipStreamWaitEvent(cs, st.ev_group[(size_t)c.group], 0));
                waited[(size_t)k] = c.group;
            }
        }
        HIP_TRY(hipMemcpyAsync(resolve(c.dst, B), resolve(c.src, B), c.bytes,
                               hipMemcpyDeviceToDeviceNoCU, cs));
        t_stats.copy_ops++;
    }
    // Queue k >= 1 is copy stream k - 1, joined back by that stream's event.
    for (int k = 1; k < K; ++k) {
        if (!started[(size_t)k]) continue;
        hipStream_t cs = st.copy_streams[(size_t)(k - 1)];
        hipEvent_t ev = st.ev_join[(size_t)(k - 1)];
        HIP_TRY(hipEventRecord(ev, cs));
        HIP_TRY(hipStreamWaitEvent(s, ev, 0));
    }
    return HOCCL_OK;
}

// All-reduce in chunk groups on the engine proxy.  After each group's last
// reduction step the caller's stream records one of the proxy's gate
// events; the proxy thread polls them and issues group g's gather copies as
// soon as its gate has completed, so the engines copy group g while the CUs
// reduce group g + 1 (the paper's per-chunk buffer states, reduced to
// "final ready").  One handshake at the end of the call releases the stream
// once every copy has completed.  A handshake per group, each on a stream
// of its own, was measured slower: every host-function handshake waits for
// the runtime's callback thread, and with 8 groups that cost more than the
// overlap gained.
hoccl_status_t run_engine_groups(DeviceState &st, const hoccl_config_t &cfg, const Plan &p,
                                 const Buffers &B, hipStream_t s, int wg, int threads, int handshake) {
    std::vector<hipEvent_t> gates;
    hoccl_status_t r = st.proxy->acquire_events(p.ngroups, gates, t_err);
    if (r != HOCCL_OK) return r;
    r = run_reductions(st, cfg, p, B, s, wg, threads, true, &gates);
    if (r != HOCCL_OK) {
        st.proxy->release_events(gates);
        return r;
    }
    std::vector<ProxyCopy> cps;
    cps.reserve(p.copies.size());
    for (const CopyOp &c : p.copies) {
        ProxyCopy pc{resolve(c.dst, B), resolve(c.src, B), c.bytes, c.chain};
        pc.gate = c.group;
        cps.push_back(pc);
    }
    int ne = 0;
    r = st.proxy->submit(cps, engine_budget(cfg), proxy_slice(cfg, p.copy_bytes), cfg.proxy_timeout_ms,
                         cfg.proxy_wait_limit_us, handshake, s, &ne, t_err, std::move(gates));
    if (r == HOCCL_OK) t_stats.copy_ops += (int)cps.size();
    return r;
}

hoccl_status_t run_copies_kernel(DeviceState &st, const hoccl_config_t &cfg, const Plan &p,
                                 const Buffers &B, hipStream_t s, int wg, int threads) {
    int maxlevel = 0;
    for (const CopyOp &c : p.copies) maxlevel = std::max(maxlevel, c.level);
    for (int lvl = 0; lvl <= maxlevel; ++lvl) {
        CopyArgs a;
        std::memset(&a, 0, sizeof a);
        auto flush = [&]() -> hoccl_status_t {
            if (a.nseg == 0) return HOCCL_OK;
            TimingPair *tp;
            TRY(timed_begin(st, cfg, s, &tp));
            HIP_TRY(launch_copy(a, wg, threads, s));
            TRY(timed_end(tp, s));
            t_stats.copy_kernel_launches++;
            std::memset(&a, 0, sizeof a);
            return HOCCL_OK;
        };
        for (const CopyOp &c : p.copies) {
            if (c.level != lvl) continue;
            a.seg[a.nseg].src = resolve(c.src, B);
            a.seg[a.nseg].dst = resolve(c.dst, B);
            a.seg[a.nseg].bytes = c.bytes;
            a.nseg++;
            if (a.nseg == kMaxCopySegs) TRY(flush());
        }
        TRY(flush());
    }
    return HOCCL_OK;
}

// Whether a ROCm profiler is loaded into this process (rocprofiler-sdk is
// preloaded and announces its tool library; the older interface uses
// HSA_TOOLS_LIB).  The host-function handshake blocks the runtime's callback
// thread, which a profiler may need to complete copies, so it is refused
// then rather than risk a stall.
bool profiler_present() {
    static const bool present = [] {
        const char *pre = std::getenv("LD_PRELOAD");
        if (pre && std::strstr(pre, "rocprofiler")) return true;
        return std::getenv("ROCP_TOOL_LIBRARIES") != nullptr || std::getenv("HSA_TOOLS_LIB") != nullptr ||
               env_long("HOCCL_ASSUME_PROFILER", 0) != 0;  // lets a test check the refusal
    }();
    return present;
}

// The engine proxy's handshake form: an explicit choice, else the host
// function, which runs no GPU code, or the one-lane kernel while a profiler
// is loaded (the host function is refused then).
int resolve_handshake(const hoccl_config_t &cfg) {
    if (cfg.proxy_handshake >= 0) return cfg.proxy_handshake;
    return profiler_present() ? 0 : 2;
}

// Copy path for a plan.  An explicit choice wins.  AUTO takes the engine
// proxy: its copies run on SDMA engines chosen through ROCr, and finish while
// every CU is busy.  The HIP runtime's device-to-device copy does not: in the
// runtime PyTorch bundles it waits for free CUs, whatever the copy kind
// asks.  While the stream is capturing a graph, the engine path is recorded
// as a host node that issues the copies at every replay, which needs the
// host-function handshake; AUTO then falls back to the HIP runtime's copies
// when that form is not available (under a profiler), and whenever no engine
// can be driven.
hoccl_copy_path_t resolve_path(const DeviceState &st, const hoccl_config_t &cfg, bool capturing) {
    if (cfg.copy_path != HOCCL_COPY_AUTO) return cfg.copy_path;
    if (!st.proxy || (capturing && resolve_handshake(cfg) != 2)) return HOCCL_COPY_HIP;
    return HOCCL_COPY_SDMA;
}

// On the engine proxy with no chunk size configured: when there are fewer
// independent chains than engines, cut every copy into k = engines / chains
// equal pieces, each a chain of its own, so that every engine works: the
// paper's striping of one flow over several queues.  Pieces stay at least
// 512 KiB (an engine copy starts in about 7 us and then moves about
// 60 GB/s).  Measured on one message with the default handshake: 8 MiB in
// 82 us as 16 pieces against 122 us as 2 pieces of 4 MiB; 48 MiB in 132 us
// as 16 pieces against 154 us as 12 pieces of 4 MiB.
constexpr size_t kMinPieceBytes = (size_t)512 << 10;

size_t auto_chunk_bytes(const DeviceState &st, const hoccl_config_t &cfg, hoccl_copy_path_t path,
                        const Plan &p) {
    if (path != HOCCL_COPY_SDMA || cfg.chunk_bytes != 0 || !st.proxy) return 0;
    int E = st.proxy->engine_count();
    E = std::min(E, engine_budget(cfg));
    if (p.nchains <= 0 || p.nchains >= E) return 0;
    size_t big = 0;
    for (const CopyOp &c : p.copies) big = std::max(big, c.bytes);
    const size_t k = (size_t)(E / p.nchains);
    size_t c = std::max((big + k - 1) / k, kMinPieceBytes);
    c = (c + 4095) & ~(size_t)4095;
    return c < big ? c : 0;
}

// Enqueues a plan's reductions and copies on `s` by the chosen copy path.
hoccl_status_t enqueue_body(DeviceState &st, const hoccl_config_t &cfg, const Plan &p,
                            const Buffers &B, hipStream_t s, hoccl_copy_path_t path, int handshake,
                            bool capturing, bool has_copies, int wg, int threads) {
    if (has_copies && path == HOCCL_COPY_SDMA && !capturing && p.ngroups > 1 &&
        !p.reduce_steps.empty()) {
        TRY(run_engine_groups(st, cfg, p, B, s, wg, threads, handshake));
    } else if (has_copies && path == HOCCL_COPY_SDMA) {
        // Reductions first (on s), then the proxy takes over the copies.
        TRY(run_reductions(st, cfg, p, B, s, wg, threads, false));
        std::vector<ProxyCopy> cps;
        cps.reserve(p.copies.size());
        for (const CopyOp &c : p.copies) {
            cps.push_back(ProxyCopy{resolve(c.dst, B), resolve(c.src, B), c.bytes, c.chain});
            cps.back().stage = c.stage;
        }
        int ne = 0;
        hoccl_status_t r;
        if (capturing) {
            r = st.proxy->capture(cps, engine_budget(cfg), cfg.proxy_timeout_ms, cfg.proxy_wait_limit_us, s,
                                  &ne, t_err);
        } else if (handshake == 2 && p.copy_bytes >= ((unsigned long long)1 << 20)) {
            // The copies may start as soon as everything before them on s
            // has completed: an event recorded here is their gate, which the
            // proxy thread polls, so the start of the host-function
            // handshake (the runtime's callback thread) overlaps the copies
            // instead of preceding them.  Measured: the pipeline schedule of
            // 16 MiB messages 6.8 ms against 7.8 ms.  Copies under 1 MiB go
            // without a gate: a 4 KiB send/recv gated took the same round
            // trip (53.6 against 51.6-53.1 us) and 6 us more host time.  So
            // does the handshake kernel, which starts within microseconds.
            std::vector<hipEvent_t> gate;
            TRY(st.proxy->acquire_events(1, gate, t_err));
            hipError_t e = hipEventRecord(gate[0], s);
            if (e != hipSuccess) {
                st.proxy->release_events(gate);
                set_err("hipEventRecord: %s", hipGetErrorString(e));
                return HOCCL_ERR_HIP;
            }
            for (ProxyCopy &c : cps) c.gate = 0;
            r = st.proxy->submit(cps, engine_budget(cfg), proxy_slice(cfg, p.copy_bytes), cfg.proxy_timeout_ms,
                                 cfg.proxy_wait_limit_us, handshake, s, &ne, t_err, std::move(gate));
        } else {
            r = st.proxy->submit(cps, engine_budget(cfg), proxy_slice(cfg, p.copy_bytes), cfg.proxy_timeout_ms,
                                 cfg.proxy_wait_limit_us, handshake, s, &ne, t_err);
        }
        if (r != HOCCL_OK) return r;
        t_stats.copy_ops += (int)cps.size();
    } else {
        TRY(run_reductions(st, cfg, p, B, s, wg, threads, has_copies && path == HOCCL_COPY_HIP));
        if (has_copies) {
            if (path == HOCCL_COPY_KERNEL)
                TRY(run_copies_kernel(st, cfg, p, B, s, wg, threads));
            else
                TRY(run_copies_hip(st, cfg, p, B, s));
        }
    }
    return HOCCL_OK;
}

// `noalloc`: the call allocates nothing (hoccl_reduce_scatter_noalloc): the
// library must already be initialised on the device, kernel timing is off,
// copies run as CU copy kernels, and the ring's partials live in the static
// scratch instead of the workspace.
template <typename Build>
hoccl_status_t execute(Build build, bool in_place, const Buffers &B0, hipStream_t s,
                       bool noalloc = false) {
    auto t0 = std::chrono::steady_clock::now();
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    HIP_TRY(hipStreamIsCapturing(s, &cap));
    const bool capturing = cap != hipStreamCaptureStatusNone;
    DeviceState *stp = nullptr;
    TRY(get_state(&stp, capturing || noalloc));
    DeviceState &st = *stp;
    std::lock_guard<std::recursive_mutex> call_lock(st.call_mu);
    hoccl_config_t cfg = config();
    std::memset(&t_stats, 0, sizeof t_stats);
    // Timing events of a captured call would be recorded only on replay; a
    // call that allocates nothing creates none.
    if (capturing || noalloc) cfg.kernel_timing = 0;
    if (noalloc) cfg.copy_path = HOCCL_COPY_KERNEL;
    Buffers B = B0;
    PlanOptions opt = options_from(cfg, in_place);
    const hoccl_copy_path_t path = resolve_path(st, cfg, capturing);
    const int handshake = resolve_handshake(cfg);
    // Automatic all-reduce groups pay off only where the gather runs on the
    // engines beside the reduction: on the engine proxy outside capture.
    if (opt.allreduce_groups == 0 && (path != HOCCL_COPY_SDMA || capturing))
        opt.allreduce_groups = 1;
    Plan p = build(opt);
    if (size_t c = auto_chunk_bytes(st, cfg, path, p)) {
        opt.chunk_bytes = c;
        p = build(opt);
    }

    const int threads = cfg.threads_per_workgroup ? cfg.threads_per_workgroup : 256;
    const int wg = auto_workgroups(st, cfg, p, threads);
    if (g_debug)
        std::fprintf(stderr, "hoccl: device %d stream %p workgroups %d copy_path %d%s plan %s\n",
                     st.device, (void *)s, wg, (int)path, capturing ? " (captured)" : "",
                     plan_to_json(p).c_str());
    if (!p.copies.empty() && path == HOCCL_COPY_SDMA && !st.proxy) {
        // Asked for explicitly: never fall back silently.
        set_err("%s", st.proxy_why.c_str());
        return HOCCL_ERR_UNSUPPORTED;
    }
    if (!p.copies.empty() && path == HOCCL_COPY_SDMA && handshake == 2 &&
        profiler_present()) {
        set_err("the host-function handshake (proxy_handshake = 2) is refused while a profiler is "
                "loaded: it blocks the runtime thread the profiler may need");
        return HOCCL_ERR_UNSUPPORTED;
    }
    if (!p.copies.empty() && path == HOCCL_COPY_SDMA && cfg.a2a_schedule == 2 &&
        (p.op == Op::AllToAll || p.op == Op::AllToAllV)) {
        // Stages run one after another on the engines made every copy of a
        // stage wait on all copies of the previous stage through dependency
        // signals; that form's first run ended in a host fault whose cause
        // is not established, so it is not offered.
        set_err("a2a_schedule 2 (stages run one after another) is not available on the SDMA copy "
                "path; use a2a_schedule 1 (stage order) or the CU copy kernel");
        return HOCCL_ERR_UNSUPPORTED;
    }
    if (!p.copies.empty() && path == HOCCL_COPY_SDMA && capturing && handshake != 2) {
        // A replay would run the handshake kernel without the proxy thread
        // issuing the copies; only the host-function form is recorded as a
        // node that issues them itself.
        set_err("the SDMA copy path is captured into a graph only with the host-function "
                "handshake (proxy_handshake 2 or -1): the handshake kernel waits for copies the "
                "proxy thread issues at call time");
        return HOCCL_ERR_UNSUPPORTED;
    }
    const bool has_kernels = !p.reduce_steps.empty() || p.has_fold;
    const bool has_copies = !p.copies.empty();
    // An error the proxy thread stored since the last call (a watchdog
    // timeout of earlier copies) is reported before anything is enqueued,
    // so the call that reports it leaves every buffer untouched.
    if (has_copies && path == HOCCL_COPY_SDMA) TRY(st.proxy->take_error(t_err));

    if (p.ws_bytes && noalloc) {
        if (p.ws_bytes > kScratchBytes) {
            set_err("this call needs %zu bytes of scratch for its partials; the static scratch of "
                    "the call that allocates nothing holds %zu", p.ws_bytes, kScratchBytes);
            return HOCCL_ERR_INVALID_ARG;
        }
        if (!st.scratch) {
            set_err("%s", st.scratch_why.c_str());
            return HOCCL_ERR_UNSUPPORTED;
        }
        B.ws = st.scratch;
    } else if (p.ws_bytes) {
        TRY(ensure_ws(st, p.ws_bytes, capturing));
        B.ws = st.ws;
        // Calls outside capture are chained through ws_event.  A captured
        // call joins no such chain: the order of its replays against other
        // users of the workspace is the caller's.
        if (!capturing && st.ws_last_stream && st.ws_last_stream != s)
            HIP_TRY(hipStreamWaitEvent(s, st.ws_event, 0));
    }
    // From here on kernels may be on the stream: whatever happens, the next
    // workspace user on another stream must wait for them.
    hoccl_status_t body = enqueue_body(st, cfg, p, B, s, path, handshake, capturing, has_copies, wg,
                                       threads);
    if (p.ws_bytes && !capturing && !noalloc) {
        hipError_t e = hipEventRecord(st.ws_event, s);
        if (e == hipSuccess) {
            st.ws_last_stream = s;
        } else if (body == HOCCL_OK) {
            set_err("hipEventRecord(ws_event): %s", hipGetErrorString(e));
            return HOCCL_ERR_HIP;
        }
    }
    TRY(body);

    bool cu_work = has_kernels || (has_copies && path == HOCCL_COPY_KERNEL);
    t_stats.workgroups_per_step = cu_work ? wg : 0;
    t_stats.cus_available = st.num_cus;
    // The engine proxy's handshake kernel waits as one lane on one CU; the
    // host-function form needs none.
    const bool handshake_wave =
        has_copies && path == HOCCL_COPY_SDMA && handshake != 2;
    int cus = cu_work ? std::min(wg, st.num_cus) : 0;
    if (handshake_wave) cus = std::max(cus, 1);
    // The HIP runtime may run its device-to-device copies as a kernel of its
    // own, on any CU (the runtime PyTorch bundles does).
    if (has_copies && path == HOCCL_COPY_HIP) cus = st.num_cus;
    t_stats.cus_used_max = cus;
    t_stats.copy_path_used = has_copies ? path : HOCCL_COPY_AUTO;
    t_stats.reduce_algo_used = p.has_fold ? HOCCL_REDUCE_DIRECT : HOCCL_REDUCE_RING;
    t_stats.hbm_bytes_algorithmic = p.hbm_bytes;
    t_stats.copy_bytes = p.copy_bytes;
    t_stats.host_enqueue_us =
        std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t0).count();
    return HOCCL_OK;
}

// ---- validation -------------------------------------------------------------------

struct Range {
    uintptr_t lo, hi;  // [lo, hi)
    int who;           // rank
    bool is_out;
};

bool overlaps(const Range &a, const Range &b) { return a.lo < b.hi && b.lo < a.hi; }

// Outputs must be pairwise disjoint; an output may overlap an input only
// where `allowed(out_rank, in_rank, out, in)` says it is a permitted in-place
// form.
template <typename Allowed>
hoccl_status_t check_overlaps(const std::vector<Range> &outs, const std::vector<Range> &ins,
                              Allowed allowed) {
    std::vector<Range> o = outs;
    std::sort(o.begin(), o.end(), [](const Range &a, const Range &b) { return a.lo < b.lo; });
    for (size_t i = 1; i < o.size(); ++i)
        if (o[i].lo < o[i - 1].hi) {
            set_err("output buffers of ranks %d and %d overlap", o[i - 1].who, o[i].who);
            return HOCCL_ERR_INVALID_ARG;
        }
    for (const Range &a : outs)
        for (const Range &b : ins)
            if (a.hi > a.lo && b.hi > b.lo && overlaps(a, b) && !allowed(a, b)) {
                set_err("output of rank %d overlaps input of rank %d outside the in-place form",
                        a.who, b.who);
                return HOCCL_ERR_INVALID_ARG;
            }
    return HOCCL_OK;
}

// `copy`: a copy-only collective, which also takes HOCCL_UINT8.
hoccl_status_t check_common(const void *send, const void *recv, hoccl_dtype_t dt, int R,
                            bool copy = false) {
    if (R < 1 || R > kMaxRanks) {
        set_err("R = %d outside [1, %d]", R, kMaxRanks);
        return HOCCL_ERR_INVALID_ARG;
    }
    if (dt == HOCCL_UINT8 && !copy) {
        set_err("uint8 is for the copy-only collectives; reductions take int32, fp32 or bf16");
        return HOCCL_ERR_INVALID_ARG;
    }
    if (dt != HOCCL_INT32 && dt != HOCCL_FP32 && dt != HOCCL_BF16 && dt != HOCCL_UINT8) {
        set_err("unknown dtype %d", (int)dt);
        return HOCCL_ERR_INVALID_ARG;
    }
    if (!send || !recv) {
        set_err("send/recv pointer arrays must not be NULL");
        return HOCCL_ERR_INVALID_ARG;
    }
    return HOCCL_OK;
}

hoccl_status_t check_ptrs(const void *const *arr, int R, const char *what) {
    for (int r = 0; r < R; ++r)
        if (!arr[r]) {
            set_err("%s[%d] is NULL", what, r);
            return HOCCL_ERR_INVALID_ARG;
        }
    return HOCCL_OK;
}

bool size_overflows(size_t a, size_t b) {
    if (b != 0 && a > SIZE_MAX / b) {
        set_err("count %zu times %zu bytes does not fit in size_t", a, b);
        return true;
    }
    return false;
}

// Budget of one ring group's fp32 partials when ring_group_bytes is 0: the
// 256 MB last-level cache.  Measured on the bf16 R=8 reduce-scatter: at 1 GiB
// per rank one group gives 141 GB/s, 256 MiB groups 198 GB/s, 128 MiB groups
// 193 GB/s and 512 MiB groups 151 GB/s; sizes whose partials fit stay one
// group.
constexpr size_t kRingGroupBytesDefault = (size_t)256 << 20;

// Automatic all-reduce chunk groups need enough engines: the overlap of a
// group's gather with the next group's reduction pays only while the
// gather is not far longer than the reduction.  bf16, R = 8, 48 MiB per
// rank, one group against two: 4 engines 1.91 / 1.98 ms, 8 engines 1.30 /
// 1.26, 12 engines 1.01 / 0.96, 16 engines 0.88 / 0.81.
constexpr int kAutoGroupsMinEngines = 8;

PlanOptions options_from(const hoccl_config_t &cfg, bool in_place) {
    PlanOptions o;
    o.group_partial_bytes = cfg.ring_group_bytes ? cfg.ring_group_bytes : kRingGroupBytesDefault;
    o.allgather_direct = cfg.allgather_direct != 0;
    o.allreduce_groups = cfg.allreduce_chunk_groups;  // 0: automatic
    if (o.allreduce_groups == 0 && engine_budget(cfg) < kAutoGroupsMinEngines) o.allreduce_groups = 1;
    o.chunk_bytes = cfg.chunk_bytes;
    o.in_place = in_place;
    o.algo = cfg.reduce_algo;
    o.fused_hops = cfg.fused_hops;
    o.a2a_schedule = cfg.a2a_schedule;
    o.bf16_partials = cfg.bf16_partials != 0;
    return o;
}

}  // namespace

void set_error_message(const char *msg) { t_err = msg; }

}  // namespace hoccl

using namespace hoccl;

static hoccl_status_t reduce_scatter_impl(const void *const *send, void *const *recv, size_t n,
                                          hoccl_dtype_t dt, int R, hipStream_t stream, bool noalloc) {
    TRY(check_common(send, recv, dt, R));
    if (n == 0) return HOCCL_OK;
    TRY(check_ptrs(send, R, "send"));
    TRY(check_ptrs((const void *const *)recv, R, "recv"));
    size_t es = dtype_size(dt);
    if (size_overflows(n, es * (size_t)R)) return HOCCL_ERR_INVALID_ARG;
    size_t ob = n * es, ib = (size_t)R * n * es;
    std::vector<Range> outs, ins;
    bool in_place = true;
    for (int r = 0; r < R; ++r) {
        outs.push_back({(uintptr_t)recv[r], (uintptr_t)recv[r] + ob, r, true});
        ins.push_back({(uintptr_t)send[r], (uintptr_t)send[r] + ib, r, false});
        in_place &= ((const char *)recv[r] == (const char *)send[r] + (size_t)r * ob);
    }
    TRY(check_overlaps(outs, ins, [ob](const Range &o, const Range &i) {
        return o.who == i.who && o.lo == i.lo + (uintptr_t)o.who * ob;
    }));
    return execute([&](const PlanOptions &o) { return plan_reduce_scatter(n, dt, R, o); }, in_place,
                   Buffers{send, recv, nullptr}, stream, noalloc);
}

extern "C" {

hoccl_status_t hoccl_init(int device) {
    if (device >= 0) HIP_TRY(hipSetDevice(device));
    DeviceState *st = nullptr;
    return get_state(&st);
}

hoccl_status_t hoccl_finalize(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    for (auto &kv : g_states) destroy_state(kv.second);
    g_states.clear();
    return HOCCL_OK;
}

hoccl_status_t hoccl_set_config(const hoccl_config_t *cfg) {
    if (!cfg || !config_valid(*cfg)) {
        set_err("invalid configuration");
        return HOCCL_ERR_INVALID_ARG;
    }
    std::lock_guard<std::mutex> lk(g_mu);
    load_config_locked();
    g_cfg = *cfg;
    return HOCCL_OK;
}

hoccl_status_t hoccl_get_config(hoccl_config_t *cfg) {
    if (!cfg) return HOCCL_ERR_INVALID_ARG;
    *cfg = config();
    return HOCCL_OK;
}

hoccl_status_t hoccl_get_last_stats(hoccl_stats_t *stats) {
    if (!stats) return HOCCL_ERR_INVALID_ARG;
    *stats = t_stats;
    return HOCCL_OK;
}

hoccl_status_t hoccl_get_kernel_times(float *ms, int cap, int *n) {
    if (!n || (cap > 0 && !ms)) return HOCCL_ERR_INVALID_ARG;
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    DeviceState *st = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        auto it = g_states.find(dev);
        if (it != g_states.end()) st = it->second;
    }
    *n = 0;
    if (!st) return HOCCL_OK;
    std::lock_guard<std::recursive_mutex> call_lock(st->call_mu);
    *n = (int)st->timing_used;
    if (cap <= 0) return HOCCL_OK;  // query the count only; keep the record
    for (size_t i = 0; i < st->timing_used; ++i) {
        HIP_TRY(hipEventSynchronize(st->timing_pool[i].b));
        if ((int)i < cap) HIP_TRY(hipEventElapsedTime(&ms[i], st->timing_pool[i].a, st->timing_pool[i].b));
    }
    st->timing_used = 0;
    return HOCCL_OK;
}

const char *hoccl_status_string(hoccl_status_t s) {
    switch (s) {
    case HOCCL_OK: return "ok";
    case HOCCL_ERR_INVALID_ARG: return "invalid argument";
    case HOCCL_ERR_UNSUPPORTED: return "unsupported";
    case HOCCL_ERR_HIP: return "HIP/HSA runtime error";
    case HOCCL_ERR_NO_MEMORY: return "out of memory";
    case HOCCL_ERR_TIMEOUT: return "timeout";
    case HOCCL_ERR_INTERNAL: return "internal error";
    }
    return "unknown status";
}

const char *hoccl_last_error_string(void) { return t_err.c_str(); }

int hoccl_sdma_engine_count(void) {
    DeviceState *st = nullptr;
    if (get_state(&st) != HOCCL_OK) return 0;
    if (!st->proxy) {
        set_err("%s", st->proxy_why.c_str());
        return 0;
    }
    return st->proxy->engine_count();
}

hoccl_status_t hoccl_ring_hop(const void *partial, const void *local, void *out, size_t count,
                              hoccl_dtype_t dt, hoccl_hop_t hop, hipStream_t stream) {
    auto t0 = std::chrono::steady_clock::now();
    if (dt != HOCCL_INT32 && dt != HOCCL_FP32 && dt != HOCCL_BF16) {
        set_err("unknown dtype %d", (int)dt);
        return HOCCL_ERR_INVALID_ARG;
    }
    if ((int)hop < HOCCL_HOP_FIRST || (int)hop > HOCCL_HOP_ONLY) {
        set_err("unknown hop %d", (int)hop);
        return HOCCL_ERR_INVALID_ARG;
    }
    if (count == 0) return HOCCL_OK;
    if (!partial || !local || !out) {
        set_err("partial, local and out must not be NULL");
        return HOCCL_ERR_INVALID_ARG;
    }
    // Element sizes of partial, local and out (see Phase).
    const size_t es = dtype_size(dt);
    size_t s0 = es, so = es;
    if (dt == HOCCL_BF16) {
        s0 = (hop == HOCCL_HOP_MIDDLE || hop == HOCCL_HOP_LAST) ? 4 : 2;
        so = (hop == HOCCL_HOP_FIRST || hop == HOCCL_HOP_MIDDLE) ? 4 : 2;
    }
    if (size_overflows(count, 4)) return HOCCL_ERR_INVALID_ARG;
    const Range r0{(uintptr_t)partial, (uintptr_t)partial + count * s0, 0, false};
    const Range r1{(uintptr_t)local, (uintptr_t)local + count * es, 0, false};
    const Range ro{(uintptr_t)out, (uintptr_t)out + count * so, 0, true};
    // Exact aliasing with an input of the same element size is an in-place
    // update: each element is read and then written by the same thread.
    if ((overlaps(ro, r0) && !(ro.lo == r0.lo && so == s0)) ||
        (overlaps(ro, r1) && !(ro.lo == r1.lo && so == es))) {
        set_err("out overlaps an input other than as the same buffer of the same element type");
        return HOCCL_ERR_INVALID_ARG;
    }
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    HIP_TRY(hipStreamIsCapturing(stream, &cap));
    const bool capturing = cap != hipStreamCaptureStatusNone;
    DeviceState *stp = nullptr;
    TRY(get_state(&stp, capturing));
    DeviceState &st = *stp;
    std::lock_guard<std::recursive_mutex> call_lock(st.call_mu);
    hoccl_config_t cfg = config();
    if (capturing) cfg.kernel_timing = 0;
    std::memset(&t_stats, 0, sizeof t_stats);
    const Phase ph = (Phase)hop;
    const int threads = cfg.threads_per_workgroup ? cfg.threads_per_workgroup : 256;
    const size_t per = reduce_step_elems_per_thread(dt, ph);
    const int wg = workgroups_for(st, cfg, (count + per - 1) / per, threads);
    ReduceArgs a;
    std::memset(&a, 0, sizeof a);
    a.seg[0].in0 = partial;
    a.seg[0].in1 = local;
    a.seg[0].out = out;
    a.seg[0].n = count;
    a.nseg = 1;
    TimingPair *tp;
    TRY(timed_begin(st, cfg, stream, &tp));
    HIP_TRY(launch_reduce_step(dt, ph, a, wg, threads, stream));
    TRY(timed_end(tp, stream));
    t_stats.reduce_launches = 1;
    t_stats.workgroups_per_step = wg;
    t_stats.cus_available = st.num_cus;
    t_stats.cus_used_max = std::min(wg, st.num_cus);
    t_stats.copy_path_used = HOCCL_COPY_AUTO;
    t_stats.reduce_algo_used = HOCCL_REDUCE_RING;
    t_stats.hbm_bytes_algorithmic = (unsigned long long)count * (s0 + es + so);
    t_stats.host_enqueue_us =
        std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t0).count();
    return HOCCL_OK;
}

hoccl_status_t hoccl_allreduce(const void *const *send, void *const *recv, size_t count,
                               hoccl_dtype_t dt, int R, hipStream_t stream) {
    TRY(check_common(send, recv, dt, R));
    if (count == 0) return HOCCL_OK;
    TRY(check_ptrs(send, R, "send"));
    TRY(check_ptrs((const void *const *)recv, R, "recv"));
    size_t es = dtype_size(dt);
    if (size_overflows(count, es)) return HOCCL_ERR_INVALID_ARG;
    size_t bytes = count * es;
    std::vector<Range> outs, ins;
    bool in_place = true;
    for (int r = 0; r < R; ++r) {
        outs.push_back({(uintptr_t)recv[r], (uintptr_t)recv[r] + bytes, r, true});
        ins.push_back({(uintptr_t)send[r], (uintptr_t)send[r] + bytes, r, false});
        in_place &= (send[r] == recv[r]);
    }
    TRY(check_overlaps(outs, ins, [](const Range &o, const Range &i) {
        return o.who == i.who && o.lo == i.lo;
    }));
    return execute([&](const PlanOptions &o) { return plan_allreduce(count, dt, R, o); }, in_place,
                   Buffers{send, recv, nullptr}, stream);
}

hoccl_status_t hoccl_reduce_scatter(const void *const *send, void *const *recv, size_t n,
                                    hoccl_dtype_t dt, int R, hipStream_t stream) {
    return reduce_scatter_impl(send, recv, n, dt, R, stream, false);
}

hoccl_status_t hoccl_reduce_scatter_noalloc(const void *const *send, void *const *recv, size_t n,
                                            hoccl_dtype_t dt, int R, hipStream_t stream) {
    return reduce_scatter_impl(send, recv, n, dt, R, stream, true);
}

hoccl_status_t hoccl_allgather(const void *const *send, void *const *recv, size_t n,
                               hoccl_dtype_t dt, int R, hipStream_t stream) {
    TRY(check_common(send, recv, dt, R, true));
    if (n == 0) return HOCCL_OK;
    TRY(check_ptrs(send, R, "send"));
    TRY(check_ptrs((const void *const *)recv, R, "recv"));
    size_t es = dtype_size(dt);
    if (size_overflows(n, es * (size_t)R)) return HOCCL_ERR_INVALID_ARG;
    size_t ib = n * es, ob = (size_t)R * n * es;
    std::vector<Range> outs, ins;
    bool in_place = true;
    for (int r = 0; r < R; ++r) {
        outs.push_back({(uintptr_t)recv[r], (uintptr_t)recv[r] + ob, r, true});
        ins.push_back({(uintptr_t)send[r], (uintptr_t)send[r] + ib, r, false});
        in_place &= ((const char *)send[r] == (const char *)recv[r] + (size_t)r * ib);
    }
    TRY(check_overlaps(outs, ins, [ib](const Range &o, const Range &i) {
        return o.who == i.who && i.lo == o.lo + (uintptr_t)o.who * ib;
    }));
    return execute([&](const PlanOptions &o) { return plan_allgather(n, dt, R, o); }, in_place,
                   Buffers{send, recv, nullptr}, stream);
}

hoccl_status_t hoccl_sendrecv(const void *const *send, void *const *recv, const int *peers,
                              size_t n, hoccl_dtype_t dt, int R, hipStream_t stream) {
    TRY(check_common(send, recv, dt, R, true));
    if (!peers) {
        set_err("peers must not be NULL");
        return HOCCL_ERR_INVALID_ARG;
    }
    std::vector<int> seen((size_t)R, 0);
    for (int r = 0; r < R; ++r) {
        int d = peers[r];
        if (d < -1 || d >= R) {
            set_err("peers[%d] = %d outside [-1, R)", r, d);
            return HOCCL_ERR_INVALID_ARG;
        }
        if (d >= 0 && seen[(size_t)d]++) {
            set_err("rank %d receives from two senders", d);
            return HOCCL_ERR_INVALID_ARG;
        }
    }
    if (n == 0) return HOCCL_OK;
    size_t es = dtype_size(dt);
    if (size_overflows(n, es)) return HOCCL_ERR_INVALID_ARG;
    size_t b = n * es;
    std::vector<Range> outs, ins;
    for (int r = 0; r < R; ++r) {
        int d = peers[r];
        if (d < 0) continue;
        if (!send[r] || !recv[d]) {
            set_err("send[%d] or recv[%d] is NULL", r, d);
            return HOCCL_ERR_INVALID_ARG;
        }
        outs.push_back({(uintptr_t)recv[d], (uintptr_t)recv[d] + b, d, true});
        ins.push_back({(uintptr_t)send[r], (uintptr_t)send[r] + b, r, false});
    }
    TRY(check_overlaps(outs, ins, [](const Range &, const Range &) { return false; }));
    return execute([&](const PlanOptions &o) { return plan_sendrecv(n, dt, R, peers, o); }, false,
                   Buffers{send, recv, nullptr}, stream);
}

hoccl_status_t hoccl_alltoall(const void *const *send, void *const *recv, size_t n,
                              hoccl_dtype_t dt, int R, hipStream_t stream) {
    TRY(check_common(send, recv, dt, R, true));
    if (n == 0) return HOCCL_OK;
    TRY(check_ptrs(send, R, "send"));
    TRY(check_ptrs((const void *const *)recv, R, "recv"));
    size_t es = dtype_size(dt);
    if (size_overflows(n, es * (size_t)R)) return HOCCL_ERR_INVALID_ARG;
    size_t b = (size_t)R * n * es;
    std::vector<Range> outs, ins;
    for (int r = 0; r < R; ++r) {
        outs.push_back({(uintptr_t)recv[r], (uintptr_t)recv[r] + b, r, true});
        ins.push_back({(uintptr_t)send[r], (uintptr_t)send[r] + b, r, false});
    }
    TRY(check_overlaps(outs, ins, [](const Range &, const Range &) { return false; }));
    return execute([&](const PlanOptions &o) { return plan_alltoall(n, dt, R, o); }, false,
                   Buffers{send, recv, nullptr}, stream);
}

hoccl_status_t hoccl_alltoallv(const void *const *send, const size_t *counts, const size_t *sd,
                               void *const *recv, const size_t *rd, hoccl_dtype_t dt, int R,
                               hipStream_t stream) {
    TRY(check_common(send, recv, dt, R, true));
    if (!counts || !sd || !rd) {
        set_err("counts and displacements must not be NULL");
        return HOCCL_ERR_INVALID_ARG;
    }
    size_t es = dtype_size(dt);
    std::vector<Range> outs, ins;
    for (int s = 0; s < R; ++s)
        for (int d = 0; d < R; ++d) {
            size_t k = (size_t)s * (size_t)R + (size_t)d;
            if (counts[k] == 0) continue;
            if (!send[s] || !recv[d]) {
                set_err("send[%d] or recv[%d] is NULL", s, d);
                return HOCCL_ERR_INVALID_ARG;
            }
            if (size_overflows(counts[k], es) || sd[k] > SIZE_MAX / es - counts[k] ||
                rd[k] > SIZE_MAX / es - counts[k]) {
                set_err("count/displacement overflow at (%d, %d)", s, d);
                return HOCCL_ERR_INVALID_ARG;
            }
            uintptr_t o = (uintptr_t)recv[d] + rd[k] * es, i = (uintptr_t)send[s] + sd[k] * es;
            outs.push_back({o, o + counts[k] * es, d, true});
            ins.push_back({i, i + counts[k] * es, s, false});
        }
    if (outs.empty()) return HOCCL_OK;
    TRY(check_overlaps(outs, ins, [](const Range &, const Range &) { return false; }));
    return execute([&](const PlanOptions &o) { return plan_alltoallv(counts, sd, rd, dt, R, o); },
                   false, Buffers{send, recv, nullptr}, stream);
}

hoccl_status_t hoccl_debug_plan_json(int op, size_t count, hoccl_dtype_t dt, int R, char *buf,
                                     size_t len, size_t *needed) {
    TRY(check_common((const void *)1, (const void *)1, dt, R, op >= 2));
    PlanOptions o = options_from(config(), false);
    Plan p;
    switch (op) {
    case 0: p = plan_allreduce(count, dt, R, o); break;
    case 1: p = plan_reduce_scatter(count, dt, R, o); break;
    case 2: p = plan_allgather(count, dt, R, o); break;
    case 3: {
        std::vector<int> peers((size_t)R);
        for (int r = 0; r < R; ++r) peers[(size_t)r] = r + 1 < R ? r + 1 : -1;
        p = plan_sendrecv(count, dt, R, peers.data(), o);
        break;
    }
    case 4: p = plan_alltoall(count, dt, R, o); break;
    default: set_err("unknown op %d", op); return HOCCL_ERR_INVALID_ARG;
    }
    std::string js = plan_to_json(p);
    if (needed) *needed = js.size() + 1;
    if (buf && len) {
        size_t k = std::min(len - 1, js.size());
        std::memcpy(buf, js.data(), k);
        buf[k] = 0;
    }
    return HOCCL_OK;
}

hoccl_status_t hoccl_debug_schedule_json(int G, const double *C, const int *node, const int *peer,
                                         double bw_intra, double bw_inter, char *buf, size_t len,
                                         size_t *needed) {
    if (G < 1 || G > 1024 || !C || !node || !peer || !(bw_intra > 0) || !(bw_inter > 0)) {
        set_err("invalid topology or traffic matrix");
        return HOCCL_ERR_INVALID_ARG;
    }
    Topology t;
    t.G = G;
    t.node.assign(node, node + G);
    t.peer.assign(peer, peer + G);
    t.bw_nvlink = bw_intra;
    t.bw_rdma = bw_inter;
    for (int u = 0; u < G; ++u)
        if (t.peer[(size_t)u] < -1 || t.peer[(size_t)u] >= G) {
            set_err("peer[%d] = %d outside [-1, G)", u, t.peer[(size_t)u]);
            return HOCCL_ERR_INVALID_ARG;
        }
    std::vector<std::vector<double>> M((size_t)G, std::vector<double>((size_t)G));
    for (int u = 0; u < G; ++u)
        for (int v = 0; v < G; ++v) {
            double x = C[(size_t)u * (size_t)G + (size_t)v];
            if (!(x >= 0)) {
                set_err("C[%d][%d] is negative or NaN", u, v);
                return HOCCL_ERR_INVALID_ARG;
            }
            M[(size_t)u][(size_t)v] = x;
        }
    std::string js = schedule_to_json(decompose(t, M));
    if (needed) *needed = js.size() + 1;
    if (buf && len) {
        size_t k = std::min(len - 1, js.size());
        std::memcpy(buf, js.data(), k);
        buf[k] = 0;
    }
    return HOCCL_OK;
}

hoccl_status_t hoccl_debug_stream_ceiling(int mode, const void *a, const void *b, void *c, size_t bytes,
                                          hipStream_t stream) {
    if (mode < 0 || mode > 6) {
        set_err("unknown mode %d", mode);
        return HOCCL_ERR_INVALID_ARG;
    }
    if (bytes == 0) return HOCCL_OK;
    const bool need_a = mode != 1 && mode != 4, need_b = mode == 3 || mode == 6, need_c = true;
    if ((need_a && !a) || (need_b && !b) || (need_c && !c)) {
        set_err("a pointer the mode needs is NULL");
        return HOCCL_ERR_INVALID_ARG;
    }
    if (bytes % 16 || ((uintptr_t)a | (uintptr_t)b | (uintptr_t)c) % 16) {
        set_err("bytes and every pointer must be multiples of 16");
        return HOCCL_ERR_INVALID_ARG;
    }
    DeviceState *st = nullptr;
    TRY(get_state(&st));
    std::lock_guard<std::recursive_mutex> call_lock(st->call_mu);
    hoccl_config_t cfg = config();
    const int threads = cfg.threads_per_workgroup ? cfg.threads_per_workgroup : 256;
    const int wg = workgroups_for(*st, cfg, (bytes / 16 + 3) / 4, threads);
    std::memset(&t_stats, 0, sizeof t_stats);
    HIP_TRY(launch_stream_ceiling(mode, a, b, c, bytes, wg, threads, stream));
    t_stats.workgroups_per_step = wg;
    t_stats.cus_available = st->num_cus;
    t_stats.cus_used_max = std::min(wg, st->num_cus);
    static const unsigned long long per_byte[] = {1, 1, 2, 3, 2, 2, 3};
    t_stats.hbm_bytes_algorithmic = per_byte[mode] * (unsigned long long)bytes;
    return HOCCL_OK;
}

hoccl_status_t hoccl_debug_interleave(int nflows, const double *bytes, double chunk_bytes, int *order,
                                      size_t cap, size_t *n) {
    if (nflows < 0 || (nflows > 0 && !bytes) || !(chunk_bytes > 0) || !n) return HOCCL_ERR_INVALID_ARG;
    std::vector<int> o = interleave_chunks(std::vector<double>(bytes, bytes + nflows), chunk_bytes);
    *n = o.size();
    if (order)
        for (size_t i = 0; i < o.size() && i < cap; ++i) order[i] = o[i];
    return HOCCL_OK;
}

}  // extern "C"
