// Copy proxy: the paper's CPU-driven DMA path with its stream handshake.
//
// The paper drives the copy engines from a CPU proxy thread and keeps them
// in order with the surrounding kernels through two flags per operation in
// host memory, written and awaited by the GPU stream with stream memory
// operations (Stream Manager: CPU-GPU handshake synchronization protocol):
//
//   stream:  write start := START;  wait start == 0;     <- start path
//            wait finish == FINISH; write finish := 0;   <- completion path
//   proxy:   see start == START, write start := 0 (acknowledge),
//            run the copies, write finish := FINISH, see finish == 0.
//
// The stream's side of the handshake takes one of three forms
// (hoccl_config_t.proxy_handshake; by default 2, or 0 while a profiler is
// loaded):
//   0            one dispatch of a one-lane handshake kernel on the caller's
//                stream, performing all four flag operations in order and
//                sleeping between polls.  HIP's own stream memory operations
//                are separate spinning kernels here, one dispatch each.
//                While the copies run, that lane holds a wave slot on one CU.
//   1            the same kernel on a private stream created with a CU mask,
//                which gets a hardware queue of its own; the caller's stream
//                joins it through HIP events (fork before the start path,
//                join after the completion path).
//   2            a host function (hipLaunchHostFunc) that performs the four
//                steps on the runtime's callback thread: no GPU code waits.
//                It blocks that thread while the copies run, and a profiler
//                may need the same thread to complete copies, so the library
//                refuses this form while a profiler is loaded.
// Every form gives up after a bounded time, so the stream always drains.
//
// Copy gates: an operation's copies may also be tied to events the caller
// records on its stream before the handshake (an all-reduce's gather of
// chunk group g behind group g's reduction).  The proxy thread polls those
// events and issues each gate's copies as soon as it completes, before the
// stream reaches the handshake; the handshake still releases the stream
// only once every copy of the operation has completed.
#include "proxy.h"
#include "hoccl_internal.h"
#include "schedule.h"

#include <hip/hip_runtime.h>
#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <deque>
#include <mutex>
#include <numeric>
#include <thread>

namespace hoccl {

namespace {

constexpr uint32_t kStartValue = 0x53544152u;   // written by the stream
constexpr uint32_t kFinishValue = 0x46494e49u;  // written by the proxy
// Operations that may be in flight at once: a caller that enqueues many
// collectives ahead of the GPU (a pipeline schedule of 32 send/recv rounds,
// several times over) waits for a free slot only beyond this many.
constexpr int kSlots = 512;
constexpr size_t kLine = 64;  // one cache line per flag
constexpr int kFlagsPerSlot = 3;  // start, finish, status

struct FindAgent {
    uint32_t bdf;
    bool found;
    hsa_agent_t agent;
};

hsa_status_t find_agent_cb(hsa_agent_t a, void *data) {
    FindAgent *f = (FindAgent *)data;
    hsa_device_type_t t;
    if (hsa_agent_get_info(a, HSA_AGENT_INFO_DEVICE, &t) != HSA_STATUS_SUCCESS) return HSA_STATUS_SUCCESS;
    if (t != HSA_DEVICE_TYPE_GPU) return HSA_STATUS_SUCCESS;
    uint32_t bdf = 0;
    if (hsa_agent_get_info(a, (hsa_agent_info_t)HSA_AMD_AGENT_INFO_BDFID, &bdf) != HSA_STATUS_SUCCESS)
        return HSA_STATUS_SUCCESS;
    if ((bdf >> 3) == (f->bdf >> 3)) {  // bus and device; any function
        f->agent = a;
        f->found = true;
        return HSA_STATUS_INFO_BREAK;
    }
    return HSA_STATUS_SUCCESS;
}

// Runs a 256-byte device-to-device copy on each of the first 16 engine ids and
// returns the mask of those that completed within 200 ms.  The scratch
// buffer is leaked if a copy is still outstanding, so no late write can land
// in freed memory.
uint32_t probe_engines(hsa_agent_t agent) {
    constexpr int kIds = 16;
    constexpr size_t kStep = 512;
    char *buf = nullptr;
    if (hipMalloc(&buf, 2 * kIds * kStep) != hipSuccess) return 0;
    if (hipMemset(buf, 0x5a, 2 * kIds * kStep) != hipSuccess || hipDeviceSynchronize() != hipSuccess) {
        (void)hipFree(buf);
        return 0;
    }
    hsa_signal_t sig;
    if (hsa_signal_create(1, 0, nullptr, &sig) != HSA_STATUS_SUCCESS) {
        (void)hipFree(buf);
        return 0;
    }
    uint32_t ok = 0;
    bool outstanding = false;
    for (int e = 0; e < kIds && !outstanding; ++e) {
        hsa_signal_store_screlease(sig, 1);
        char *src = buf + (size_t)e * kStep, *dst = buf + (size_t)(kIds + e) * kStep;
        if (hsa_amd_memory_async_copy_on_engine(dst, agent, src, agent, 256, 0, nullptr, sig,
                                                (hsa_amd_sdma_engine_id_t)(1u << e), true) !=
            HSA_STATUS_SUCCESS)
            continue;
        auto t0 = std::chrono::steady_clock::now();
        while (hsa_signal_load_scacquire(sig) != 0) {
            if (std::chrono::steady_clock::now() - t0 > std::chrono::milliseconds(200)) {
                outstanding = true;
                break;
            }
            std::this_thread::yield();
        }
        if (!outstanding) ok |= 1u << e;
    }
    if (!outstanding) {
        hsa_signal_destroy(sig);
        (void)hipFree(buf);
    }
    return ok;
}

inline uint32_t load_flag(volatile uint32_t *p) {
    return __atomic_load_n((uint32_t *)p, __ATOMIC_ACQUIRE);
}
inline void store_flag(volatile uint32_t *p, uint32_t v) {
    __atomic_store_n((uint32_t *)p, v, __ATOMIC_RELEASE);
}

}  // namespace

struct ProxyOp {
    enum State { ACTIVE, WAIT_ACK };
    int slot = -1;
    std::vector<ProxyCopy> copies;  // in issue order: the gates' blocks, then the ungated
    std::vector<uint32_t> engine;   // engine id bit per copy
    std::vector<std::vector<int>> deps;  // earlier copies each copy waits for
    std::vector<hsa_signal_t> sig;
    std::vector<hipEvent_t> gates;  // copy gates (taken from the pool)
    std::vector<char> gate_open;
    size_t next = 0;                // copies issued so far
    bool start_seen = false;        // the stream reached the handshake
    State state = ACTIVE;
    std::chrono::steady_clock::time_point since;  // last issue
    unsigned timeout_ms = 10000;
    bool timed_out = false;
    bool copy_failed = false;
    size_t ended = 0;               // copies seen ended so far
    // Balanced issue (Proxy::submit) over the engines of the budget: the
    // scheduled copies are cut into pieces as engines take them; `pieces`
    // and `sig` grow with every piece issued.
    bool balanced = false;
    BalancedIssue bal;
    std::vector<uint32_t> slot_engine;  // engine id bit per engine slot
    std::vector<ProxyCopy> pieces;
};

struct CapturedOp;

class ProxyImpl {
  public:
    hsa_agent_t agent{};
    std::vector<uint32_t> engines;  // id bits of usable engines
    uint32_t *flags = nullptr;      // kSlots * kFlagsPerSlot flags, one per cache line
    uint64_t ticks_per_ms = 100000;  // device wall clock
    hipStream_t hs = nullptr;       // private CU-masked stream for handshake form 1
    hipEvent_t ev_fork = nullptr, ev_join = nullptr;
    std::mutex mu;
    std::condition_variable cv_work, cv_slot;
    std::deque<ProxyOp *> incoming;
    std::vector<int> free_slots;
    std::vector<hsa_signal_t> free_signals;
    std::vector<hipEvent_t> free_events;  // pool for copy gates
    bool stop = false;
    std::thread th;
    hoccl_status_t sticky = HOCCL_OK;
    std::string sticky_msg;
    std::vector<CapturedOp *> captured;  // kept until the proxy is destroyed

    volatile uint32_t *flag(int s, int k) {
        return (volatile uint32_t *)((char *)flags + (size_t)(kFlagsPerSlot * s + k) * kLine);
    }
    volatile uint32_t *start_flag(int s) { return flag(s, 0); }
    volatile uint32_t *finish_flag(int s) { return flag(s, 1); }
    volatile uint32_t *status_flag(int s) { return flag(s, 2); }

    void fail(hoccl_status_t st, const char *msg) {
        std::lock_guard<std::mutex> lk(mu);
        if (sticky == HOCCL_OK) {
            sticky = st;
            sticky_msg = msg;
        }
    }

    // Issues copy i on `engine` behind the copies it depends on (their
    // signals were armed at submission, so a copy waits for a predecessor
    // even if issued first).  A failure is stored and false returned.
    bool issue_copy(ProxyOp &op, size_t i, uint32_t engine) {
        const ProxyCopy &c = op.copies[i];
        std::vector<hsa_signal_t> deps;
        for (int d : op.deps[i]) deps.push_back(op.sig[(size_t)d]);
        hsa_status_t e = hsa_amd_memory_async_copy_on_engine(
            c.dst, agent, c.src, agent, c.bytes, (uint32_t)deps.size(), deps.empty() ? nullptr : deps.data(),
            op.sig[i], (hsa_amd_sdma_engine_id_t)engine, true);
        if (e == HSA_STATUS_SUCCESS) return true;
        char buf[160];
        std::snprintf(buf, sizeof buf, "hsa_amd_memory_async_copy_on_engine failed (%d)", (int)e);
        fail(HOCCL_ERR_HIP, buf);
        return false;
    }

    // Issues copy op.next on its scheduled engine.
    void issue_next(ProxyOp &op) {
        const size_t i = op.next++;
        if (!issue_copy(op, i, op.engine[i])) {
            // Retire the copies that were never issued so the op completes.
            for (size_t k = i; k < op.copies.size(); ++k) hsa_signal_store_screlease(op.sig[k], 0);
            op.next = op.copies.size();
        }
    }

    // A completion signal for a new piece, from the pool or created; armed
    // (value 1) before the piece is issued.
    bool piece_signal(hsa_signal_t &sg) {
        {
            std::lock_guard<std::mutex> lk(mu);
            if (!free_signals.empty()) {
                sg = free_signals.back();
                free_signals.pop_back();
                hsa_signal_store_screlease(sg, 1);
                return true;
            }
        }
        if (hsa_signal_create(1, 0, nullptr, &sg) == HSA_STATUS_SUCCESS) return true;
        fail(HOCCL_ERR_HIP, "hsa_signal_create failed");
        return false;
    }

    // Issues a piece of the operation's copy pc.copy on `engine`.
    bool issue_piece(ProxyOp &op, const Piece &pc, uint32_t engine) {
        hsa_signal_t sg;
        if (!piece_signal(sg)) return false;
        ProxyCopy c = op.copies[(size_t)pc.copy];
        c.dst = (char *)c.dst + pc.offset;
        c.src = (const char *)c.src + pc.offset;
        c.bytes = pc.bytes;
        op.pieces.push_back(c);
        op.sig.push_back(sg);
        const hsa_status_t e = hsa_amd_memory_async_copy_on_engine(c.dst, agent, c.src, agent, c.bytes, 0, nullptr,
                                                                   sg, (hsa_amd_sdma_engine_id_t)engine, true);
        if (e == HSA_STATUS_SUCCESS) return true;
        hsa_signal_store_screlease(sg, 0);  // never issued: counts as ended
        char buf[160];
        std::snprintf(buf, sizeof buf, "hsa_amd_memory_async_copy_on_engine failed (%d)", (int)e);
        fail(HOCCL_ERR_HIP, buf);
        return false;
    }

    // One pass of balanced issue.  After a failed issue nothing more is
    // issued, and the operation completes once the issued pieces have.
    bool issue_balanced(ProxyOp &op) {
        const double now_us =
            std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now().time_since_epoch()).count();
        return op.bal.pass(
            now_us, [&](int i) { return copy_ended(op, (size_t)i); },
            [&](int e, const Piece &pc) { return issue_piece(op, pc, op.slot_engine[(size_t)e]); });
    }

    // Whether the copies behind gate g may go: its event has completed (a
    // failed query opens it and is reported, so the operation still ends).
    bool gate_open(ProxyOp &op, int g) {
        if (op.gate_open[(size_t)g]) return true;
        hipError_t e = hipEventQuery(op.gates[(size_t)g]);
        if (e == hipErrorNotReady) return false;
        if (e != hipSuccess) fail(HOCCL_ERR_HIP, "hipEventQuery on a copy gate failed");
        op.gate_open[(size_t)g] = 1;
        return true;
    }

    // A copy's completion signal drops from 1 to 0 when it completes; ROCr
    // sets it negative when the copy fails.  A failed copy counts as ended
    // (so the operation still completes) and is reported once.
    bool copy_ended(ProxyOp &op, size_t i) {
        const hsa_signal_value_t v = hsa_signal_load_scacquire(op.sig[i]);
        if (v < 0 && !op.copy_failed) {
            op.copy_failed = true;
            char buf[160];
            std::snprintf(buf, sizeof buf, "an SDMA copy of %zu bytes reported an error (%lld)",
                          (op.balanced ? op.pieces[i] : op.copies[i]).bytes, (long long)v);
            fail(HOCCL_ERR_HIP, buf);
        }
        return v <= 0;
    }

    size_t copies_ended(ProxyOp &op) {
        size_t n = 0;
        for (size_t i = 0; i < op.sig.size(); ++i) n += copy_ended(op, i);
        return n;
    }

    void report_timeout(ProxyOp &op) {
        size_t ended = 0;
        for (size_t i = 0; i < op.sig.size(); ++i) ended += hsa_signal_load_scacquire(op.sig[i]) <= 0;
        char buf[200];
        if (op.balanced)
            std::snprintf(buf, sizeof buf,
                          "SDMA copies did not complete within the proxy timeout (balanced issue of %zu copies: "
                          "%zu pieces issued, %zu ended%s)",
                          op.copies.size(), op.bal.issued(), ended, op.bal.all_issued() ? "" : ", more to issue");
        else
            std::snprintf(buf, sizeof buf,
                          "SDMA copies did not complete within the proxy timeout (%zu of %zu copies issued, "
                          "%zu ended)",
                          op.next, op.copies.size(), ended);
        fail(HOCCL_ERR_TIMEOUT, buf);
    }

    void release(ProxyOp *op) {
        std::lock_guard<std::mutex> lk(mu);
        for (auto &s : op->sig) free_signals.push_back(s);
        for (auto &e : op->gates) free_events.push_back(e);
        free_slots.push_back(op->slot);
        cv_slot.notify_all();
        delete op;
    }

    bool started(ProxyOp &op) {
        if (load_flag(start_flag(op.slot)) != kStartValue) return false;
        store_flag(start_flag(op.slot), 0);  // acknowledge
        return true;
    }

    void loop() {
        std::vector<ProxyOp *> active;
        for (;;) {
            {
                std::unique_lock<std::mutex> lk(mu);
                if (active.empty())
                    cv_work.wait(lk, [&] { return stop || !incoming.empty(); });
                while (!incoming.empty()) {
                    active.push_back(incoming.front());
                    incoming.pop_front();
                }
                if (stop && active.empty()) return;
            }
            bool progress = false;
            auto now = std::chrono::steady_clock::now();
            for (size_t i = 0; i < active.size();) {
                ProxyOp *op = active[i];
                bool retired = false;
                switch (op->state) {
                case ProxyOp::ACTIVE:
                    // The stream reached the handshake: everything before it,
                    // including every gate, has completed.
                    if (!op->start_seen && started(*op)) {
                        op->start_seen = true;
                        progress = true;
                    }
                    if (op->balanced) {
                        // All copies share one gate (or none: the stream's start).
                        const int g = op->copies[0].gate;
                        const bool may_go = g < 0 ? op->start_seen : gate_open(*op, g);
                        if (may_go && !op->bal.all_issued()) {
                            if (issue_balanced(*op)) {
                                op->since = now;
                                progress = true;
                            } else if (!op->timed_out && now - op->since >
                                                             std::chrono::milliseconds(op->timeout_ms)) {
                                // Copies in flight that never complete hold back the rest.
                                op->timed_out = true;
                                report_timeout(*op);
                            }
                        }
                        if (!op->bal.all_issued() || !op->start_seen) break;
                    } else {
                        // Issue in order what may go: a gated copy once its
                        // gate is open, an ungated one once the stream has
                        // started.
                        while (op->next < op->copies.size()) {
                            const int g = op->copies[op->next].gate;
                            if (g < 0 ? !op->start_seen : !gate_open(*op, g)) break;
                            issue_next(*op);
                            op->since = now;
                            progress = true;
                        }
                        if (op->next < op->copies.size() || !op->start_seen) break;
                    }
                    {
                        // The watchdog runs on progress: a copy issued or
                        // completed restarts it.
                        const size_t ended = copies_ended(*op);
                        if (ended == op->sig.size()) {
                            progress = true;
                            store_flag(finish_flag(op->slot), kFinishValue);
                            op->state = ProxyOp::WAIT_ACK;
                            op->since = now;
                        } else if (ended > op->ended) {
                            op->ended = ended;
                            op->since = now;
                        } else if (!op->timed_out &&
                                   now - op->since > std::chrono::milliseconds(op->timeout_ms)) {
                            op->timed_out = true;
                            report_timeout(*op);
                        }
                    }
                    break;
                case ProxyOp::WAIT_ACK:
                    // The stream reset `finish`: the slot may be reused.  If
                    // the handshake kernel gave up waiting it never will;
                    // the slot is free then too, and the error is reported.
                    if (load_flag(finish_flag(op->slot)) == 0) {
                        release(op);
                        retired = true;
                        progress = true;
                    } else if (load_flag(status_flag(op->slot)) != 0) {
                        fail(HOCCL_ERR_TIMEOUT, "the stream stopped waiting for the SDMA copies "
                                                "before they completed");
                        release(op);
                        retired = true;
                        progress = true;
                    }
                    break;
                }
                if (retired) {
                    active[i] = active.back();
                    active.pop_back();
                } else {
                    ++i;
                }
            }
            if (!progress) std::this_thread::yield();
        }
    }
};

Proxy *Proxy::create(int device, std::string *why) {
    auto fail = [&](const char *msg, long code) -> Proxy * {
        if (why) {
            char buf[200];
            std::snprintf(buf, sizeof buf, "SDMA engine proxy unavailable: %s (%ld)", msg, code);
            *why = buf;
        }
        return nullptr;
    };
    int bus = 0, dev = 0;
    hipError_t he;
    if ((he = hipDeviceGetAttribute(&bus, hipDeviceAttributePciBusId, device)) != hipSuccess ||
        (he = hipDeviceGetAttribute(&dev, hipDeviceAttributePciDeviceId, device)) != hipSuccess)
        return fail("PCI location query failed", (long)he);
    hsa_status_t hs = hsa_init();
    if (hs != HSA_STATUS_SUCCESS) return fail("hsa_init failed", (long)hs);
    FindAgent f{(uint32_t)((bus << 8) | (dev << 3)), false, {}};
    hsa_iterate_agents(find_agent_cb, &f);
    if (!f.found) {
        hsa_shut_down();
        return fail("no HSA GPU agent at the HIP device's PCI location", (long)f.bdf);
    }
    uint32_t mask = 0;
    hs = hsa_amd_memory_copy_engine_status(f.agent, f.agent, &mask);
    if (hs != HSA_STATUS_SUCCESS || mask == 0) {
        // Some ROCr builds do not answer this query for same-device copies
        // although they execute them; find the usable engines by running one
        // small copy on each.
        mask = probe_engines(f.agent);
    }
    if (mask == 0) {
        hsa_shut_down();
        return fail("no SDMA engine accepts device-to-device copies", (long)hs);
    }
    ProxyImpl *p = new ProxyImpl();
    p->agent = f.agent;
    // Engines 0 and 1 also serve the runtime's own host transfers: use them
    // last.  HOCCL_SDMA_ENGINE_IDS ("3,0,7") restricts the proxy to the
    // listed usable engines, in that order.
    if (const char *ids = std::getenv("HOCCL_SDMA_ENGINE_IDS")) {
        for (const char *c = ids; *c;) {
            char *end = nullptr;
            long b = std::strtol(c, &end, 10);
            if (end == c) break;
            if (b >= 0 && b < 32 && (mask & (1u << b))) p->engines.push_back(1u << b);
            c = (*end == ',') ? end + 1 : end;
        }
    } else {
        for (int b = 2; b < 32; ++b)
            if (mask & (1u << b)) p->engines.push_back(1u << b);
        for (int b = 0; b < 2; ++b)
            if (mask & (1u << b)) p->engines.push_back(1u << b);
    }
    if (p->engines.empty()) {
        delete p;
        hsa_shut_down();
        return fail("HOCCL_SDMA_ENGINE_IDS names no usable engine", (long)mask);
    }
    void *fl = nullptr;
    he = hipHostMalloc(&fl, kSlots * kFlagsPerSlot * kLine, hipHostMallocCoherent | hipHostMallocMapped);
    if (he != hipSuccess || !fl) {
        delete p;
        hsa_shut_down();
        return fail("hipHostMalloc of the flag pool failed", (long)he);
    }
    std::memset(fl, 0, kSlots * kFlagsPerSlot * kLine);
    p->flags = (uint32_t *)fl;
    int khz = 0;
    if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, device) == hipSuccess && khz > 0)
        p->ticks_per_ms = (uint64_t)khz;
    // A CU-masked stream owns a hardware queue.  The runtime accepts masks
    // only with at least one CU in every XCD; logical CUs 0-7 are one per
    // XCD on MI355X, so the mask is 0xff (the wait kernel itself is a single
    // thread on one of them).
    uint32_t cu_mask[8] = {0xffu, 0, 0, 0, 0, 0, 0, 0};
    if (hipExtStreamCreateWithCUMask(&p->hs, 8, cu_mask) != hipSuccess ||
        hipEventCreateWithFlags(&p->ev_fork, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&p->ev_join, hipEventDisableTiming) != hipSuccess) {
        (void)hipGetLastError();  // handled: do not leave it for the next caller
        if (p->hs) (void)hipStreamDestroy(p->hs);
        p->hs = nullptr;  // the handshake then runs on the caller's stream
    }
    for (int s = kSlots - 1; s >= 0; --s) p->free_slots.push_back(s);
    p->th = std::thread([p] { p->loop(); });
    return new Proxy(p);
}

// A copy operation recorded into a HIP graph.  The graph holds a host node
// that runs `run_captured` at every replay: it issues the operation's
// copies on their engines itself and returns once they have completed, so
// the stream waits without GPU code and without the proxy thread, which
// only ever sees operations submitted at call time.  The copy list and its
// completion signals stay allocated until the proxy is destroyed
// (hoccl_finalize), after which such a graph must not be replayed.
struct CapturedOp {
    ProxyImpl *P = nullptr;
    std::vector<ProxyCopy> copies;
    std::vector<uint32_t> engine;
    std::vector<std::vector<int>> deps;
    std::vector<hsa_signal_t> sig;
    std::chrono::microseconds limit{0};
};

// Runs on the HIP runtime's callback thread, so it calls no HIP function.
// A failure is reported by the next call into the proxy, and the function
// always returns within `limit`, so the stream drains.
void run_captured(void *arg) {
    CapturedOp &op = *(CapturedOp *)arg;
    ProxyImpl &P = *op.P;
    size_t issued = 0;
    for (size_t i = 0; i < op.copies.size(); ++i, ++issued) {
        const ProxyCopy &c = op.copies[i];
        hsa_signal_store_screlease(op.sig[i], 1);
        std::vector<hsa_signal_t> deps;
        for (int d : op.deps[i]) deps.push_back(op.sig[(size_t)d]);
        if (hsa_amd_memory_async_copy_on_engine(c.dst, P.agent, c.src, P.agent, c.bytes, (uint32_t)deps.size(),
                                                deps.empty() ? nullptr : deps.data(), op.sig[i],
                                                (hsa_amd_sdma_engine_id_t)op.engine[i], true) != HSA_STATUS_SUCCESS) {
            hsa_signal_store_screlease(op.sig[i], 0);
            P.fail(HOCCL_ERR_HIP, "hsa_amd_memory_async_copy_on_engine failed in a graph replay");
            break;
        }
    }
    const auto t0 = std::chrono::steady_clock::now();
    for (size_t i = 0; i < issued; ++i)
        while (hsa_signal_load_scacquire(op.sig[i]) != 0) {
            if (std::chrono::steady_clock::now() - t0 > op.limit) {
                P.fail(HOCCL_ERR_TIMEOUT, "SDMA copies of a graph replay did not complete in time");
                return;
            }
            std::this_thread::yield();
        }
}

Proxy::~Proxy() {
    {
        std::lock_guard<std::mutex> lk(impl_->mu);
        impl_->stop = true;
    }
    impl_->cv_work.notify_all();
    if (impl_->th.joinable()) impl_->th.join();
    for (CapturedOp *op : impl_->captured) {
        for (auto &sg : op->sig) hsa_signal_destroy(sg);
        delete op;
    }
    for (auto &s : impl_->free_signals) hsa_signal_destroy(s);
    for (auto &e : impl_->free_events) (void)hipEventDestroy(e);
    if (impl_->flags) (void)hipHostFree(impl_->flags);
    if (impl_->hs) (void)hipStreamDestroy(impl_->hs);
    if (impl_->ev_fork) (void)hipEventDestroy(impl_->ev_fork);
    if (impl_->ev_join) (void)hipEventDestroy(impl_->ev_join);
    delete impl_;
    hsa_shut_down();
}

int Proxy::engine_count() const { return (int)impl_->engines.size(); }

hoccl_status_t Proxy::take_error(std::string &err) {
    std::lock_guard<std::mutex> lk(impl_->mu);
    hoccl_status_t st = impl_->sticky;
    if (st != HOCCL_OK) {
        err = impl_->sticky_msg;
        impl_->sticky = HOCCL_OK;
        impl_->sticky_msg.clear();
    }
    return st;
}

// The stream side of the handshake run as a host function: the HIP runtime
// holds every later operation of the stream until it returns, so the stream
// waits without any GPU code.  It performs the same four flag steps as the
// handshake kernel, on the runtime's callback thread, and gives up (status
// = 1) after the same bounded time.  It must not call into HIP.
struct HostSide {
    volatile uint32_t *start, *finish, *status;
    std::chrono::microseconds limit;
};

void host_side_handshake(void *arg) {
    HostSide *h = (HostSide *)arg;
    const auto t0 = std::chrono::steady_clock::now();
    auto wait = [&](volatile uint32_t *f, uint32_t want) {
        while (load_flag(f) != want) {
            if (std::chrono::steady_clock::now() - t0 > h->limit) return false;
            std::this_thread::yield();
        }
        return true;
    };
    store_flag(h->start, kStartValue);
    if (!wait(h->start, 0) || !wait(h->finish, kFinishValue))
        store_flag(h->status, 1);
    else
        store_flag(h->finish, 0);
    delete h;
}

// The copies of one operation in issue order, each with its engine and the
// earlier copy of its chain it must wait for.  Chains are balanced over at
// most `max_engines` engines by bytes, largest first onto the least loaded;
// the chains sharing an engine are interleaved copy by copy in proportion
// to their length (flow-size-aware chunk scheduling), each chain keeping
// its own order.
struct EngineSchedule {
    std::vector<ProxyCopy> copies;
    std::vector<uint32_t> engine;         // engine id bit per copy
    std::vector<std::vector<int>> deps;   // copies each copy waits for
    int engines_used = 0;
};

// The collective scheduler's stages on the engines (Collective Scheduler,
// Algorithm 1).  Every stage's copies go to the engines largest first onto
// the least loaded by bytes so far, each engine's queue in stage order,
// issued stage by stage and one copy per engine in turn; only the engines'
// own order keeps the stages apart (no copy waits for another).
EngineSchedule schedule_stages(const ProxyImpl &P, const std::vector<ProxyCopy> &copies, int max_engines) {
    int E = (int)P.engines.size();
    if (max_engines > 0) E = std::min(E, max_engines);
    int nst = 0;
    for (auto &c : copies) nst = std::max(nst, c.stage + 1);
    std::vector<std::vector<size_t>> of_stage((size_t)nst);
    for (size_t i = 0; i < copies.size(); ++i) of_stage[(size_t)copies[i].stage].push_back(i);
    std::vector<unsigned long long> load((size_t)E, 0);
    std::vector<std::vector<size_t>> per_engine((size_t)E);
    std::vector<int> eng(copies.size(), 0);
    for (auto &st : of_stage) {
        std::vector<size_t> q = st;
        std::stable_sort(q.begin(), q.end(), [&](size_t a, size_t b) { return copies[a].bytes > copies[b].bytes; });
        for (size_t i : q) {
            size_t best = 0;
            for (size_t k = 1; k < load.size(); ++k)
                if (load[k] < load[best]) best = k;
            load[best] += copies[i].bytes;
            per_engine[best].push_back(i);
            eng[i] = (int)best;
        }
    }
    // Issue order: stage by stage, and within a stage one copy per engine in
    // turn, so every copy is issued after every copy it may wait for.
    EngineSchedule out;
    std::vector<int> pos(copies.size(), -1);
    for (int sidx = 0; sidx < nst; ++sidx) {
        std::vector<size_t> next((size_t)E, 0);
        bool more = true;
        while (more) {
            more = false;
            for (int e = 0; e < E; ++e) {
                auto &q = per_engine[(size_t)e];
                while (next[(size_t)e] < q.size() && copies[q[next[(size_t)e]]].stage < sidx) ++next[(size_t)e];
                if (next[(size_t)e] < q.size() && copies[q[next[(size_t)e]]].stage == sidx) {
                    size_t i = q[next[(size_t)e]++];
                    pos[i] = (int)out.copies.size();
                    out.copies.push_back(copies[i]);
                    out.engine.push_back(P.engines[(size_t)e]);
                    more = true;
                }
            }
        }
    }
    out.deps.assign(out.copies.size(), {});
    for (auto l : load) out.engines_used += l > 0;
    return out;
}

EngineSchedule schedule_copies(const ProxyImpl &P, const std::vector<ProxyCopy> &copies,
                               int max_engines) {
    if (!copies.empty() && copies[0].stage >= 0) return schedule_stages(P, copies, max_engines);
    int E = (int)P.engines.size();
    if (max_engines > 0) E = std::min(E, max_engines);
    // Balance bytes per engine: largest chain first onto the least loaded.
    int nch = 0;
    for (auto &c : copies) nch = std::max(nch, c.chain + 1);
    std::vector<unsigned long long> cb((size_t)nch, 0);
    for (auto &c : copies) cb[(size_t)c.chain] += c.bytes;
    std::vector<int> order((size_t)nch);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return cb[(size_t)a] > cb[(size_t)b]; });
    std::vector<unsigned long long> load((size_t)E, 0);
    std::vector<int> eng_of_chain((size_t)nch, 0);
    // HOCCL_PROXY_SCHEDULE=round_robin is the ablation baseline: chain c on
    // engine c mod E, each engine's copies in plan order.
    static const bool round_robin = [] {
        const char *v = std::getenv("HOCCL_PROXY_SCHEDULE");
        return v && std::strcmp(v, "round_robin") == 0;
    }();
    for (int ch : order) {
        size_t best = 0;
        if (round_robin) {
            best = (size_t)(ch % E);
        } else {
            for (size_t k = 1; k < load.size(); ++k)
                if (load[k] < load[best]) best = k;
        }
        eng_of_chain[(size_t)ch] = (int)best;
        load[best] += cb[(size_t)ch];
    }
    // Order per engine: the chains sharing an engine are interleaved copy by
    // copy in proportion to their length (flow-size-aware chunk scheduling),
    // each chain keeping its own order.
    std::vector<std::vector<size_t>> of_chain((size_t)nch);
    for (size_t i = 0; i < copies.size(); ++i) of_chain[(size_t)copies[i].chain].push_back(i);
    std::vector<std::vector<size_t>> per_engine((size_t)E);
    for (int e = 0; e < E; ++e) {
        std::vector<size_t> &q = per_engine[(size_t)e];
        std::vector<int> chains;
        std::vector<double> len;
        for (int ch = 0; ch < nch; ++ch)
            if (eng_of_chain[(size_t)ch] == e && !of_chain[(size_t)ch].empty()) {
                chains.push_back(ch);
                len.push_back((double)of_chain[(size_t)ch].size());
            }
        std::vector<size_t> next(chains.size(), 0);
        if (round_robin) {
            for (size_t k = 0; k < chains.size(); ++k)
                for (size_t i : of_chain[(size_t)chains[k]]) q.push_back(i);
            continue;
        }
        for (int k : interleave_chunks(len, 1.0)) {
            int ch = chains[(size_t)k];
            q.push_back(of_chain[(size_t)ch][next[(size_t)k]++]);
        }
    }
    // Issue order: one copy per engine in turn, so that every engine has work
    // after the first E host calls instead of the last engine waiting for
    // all the others' copies to be issued (each issue costs the proxy thread
    // some microseconds).  Each engine's own order is kept.
    std::vector<size_t> issue;
    issue.reserve(copies.size());
    for (size_t r = 0; issue.size() < copies.size(); ++r)
        for (int e = 0; e < E; ++e)
            if (r < per_engine[(size_t)e].size()) issue.push_back(per_engine[(size_t)e][r]);
    EngineSchedule out;
    out.copies.reserve(copies.size());
    for (size_t i : issue) out.copies.push_back(copies[i]);
    std::vector<int> last((size_t)nch, -1);
    out.engine.resize(out.copies.size());
    out.deps.assign(out.copies.size(), {});
    for (size_t i = 0; i < out.copies.size(); ++i) {
        int ch = out.copies[i].chain;
        out.engine[i] = P.engines[(size_t)eng_of_chain[(size_t)ch]];
        if (last[(size_t)ch] >= 0) out.deps[i].push_back(last[(size_t)ch]);
        last[(size_t)ch] = (int)i;
    }
    for (auto l : load) out.engines_used += l > 0;
    return out;
}

hoccl_status_t Proxy::acquire_events(int n, std::vector<hipEvent_t> &out, std::string &err) {
    ProxyImpl &P = *impl_;
    out.clear();
    {
        std::lock_guard<std::mutex> lk(P.mu);
        while ((int)out.size() < n && !P.free_events.empty()) {
            out.push_back(P.free_events.back());
            P.free_events.pop_back();
        }
    }
    while ((int)out.size() < n) {
        hipEvent_t e = nullptr;
        hipError_t he = hipEventCreateWithFlags(&e, hipEventDisableTiming);
        if (he != hipSuccess) {
            err = std::string("hipEventCreateWithFlags: ") + hipGetErrorString(he);
            release_events(out);
            return HOCCL_ERR_HIP;
        }
        out.push_back(e);
    }
    return HOCCL_OK;
}

void Proxy::release_events(std::vector<hipEvent_t> &events) {
    std::lock_guard<std::mutex> lk(impl_->mu);
    for (hipEvent_t e : events) impl_->free_events.push_back(e);
    events.clear();
}

// Whether an operation's copies may be issued balanced: one gate for all,
// and no copy waits for another (every chain a single copy, or stage-tagged
// copies, which the stage schedule never makes wait).
bool balance_eligible(const std::vector<ProxyCopy> &copies) {
    if (copies.empty()) return false;
    std::vector<int> chains;
    chains.reserve(copies.size());
    for (const ProxyCopy &c : copies) {
        if (c.gate != copies[0].gate) return false;
        chains.push_back(c.chain);
    }
    if (copies[0].stage >= 0) return true;
    std::sort(chains.begin(), chains.end());
    return std::adjacent_find(chains.begin(), chains.end()) == chains.end();
}

hoccl_status_t Proxy::submit(const std::vector<ProxyCopy> &copies_in, int max_engines, size_t slice_bytes,
                             unsigned timeout_ms, unsigned wait_limit_us, int handshake,
                             hipStream_t s, int *engines_used, std::string &err,
                             std::vector<hipEvent_t> gates) {
    ProxyImpl &P = *impl_;
    for (const ProxyCopy &c : copies_in)
        if (c.gate >= (int)gates.size()) {
            err = "a copy names a gate that was not given";
            release_events(gates);
            return HOCCL_ERR_INTERNAL;
        }
    const std::vector<ProxyCopy> &copies = copies_in;
    const bool balanced = slice_bytes > 0 && balance_eligible(copies);
    ProxyOp *op = new ProxyOp();
    op->timeout_ms = timeout_ms ? timeout_ms : 10000;
    op->since = std::chrono::steady_clock::now();
    {
        // Each gate's copies are scheduled as a block of their own, the
        // gates in order and the ungated copies last, so a gate's block goes
        // out as soon as the gate opens.
        int used = 0;
        const int ng = (int)gates.size();
        for (int k = 0; k <= ng; ++k) {
            const int g = k < ng ? k : -1;
            std::vector<ProxyCopy> part;
            for (const ProxyCopy &c : copies)
                if (c.gate == g) part.push_back(c);
            if (part.empty()) continue;
            EngineSchedule sch = schedule_copies(P, part, max_engines);
            const int base = (int)op->copies.size();
            for (size_t i = 0; i < sch.copies.size(); ++i) {
                op->copies.push_back(sch.copies[i]);
                op->engine.push_back(sch.engine[i]);
                std::vector<int> d = sch.deps[i];
                for (int &x : d) x += base;
                op->deps.push_back(std::move(d));
            }
            used = std::max(used, sch.engines_used);
        }
        if (engines_used) *engines_used = used;
    }
    if (balanced) {
        // The schedule's issue order (byte-balanced, flow-size interleaved,
        // or stage by stage) is the order in which the engines of the
        // budget take pieces of the copies.
        int E = (int)P.engines.size();
        if (max_engines > 0) E = std::min(E, max_engines);
        std::vector<size_t> bytes;
        for (const ProxyCopy &c : op->copies) bytes.push_back(c.bytes);
        op->balanced = true;
        op->slot_engine.assign(P.engines.begin(), P.engines.begin() + E);
        op->bal = BalancedIssue(E, slice_bytes, 2 * slice_bytes, bytes);
        if (engines_used) *engines_used = std::min(E, (int)op->copies.size());
    }
    op->gates = std::move(gates);
    op->gate_open.assign(op->gates.size(), 0);
    const size_t sig_wanted = op->balanced ? 0 : op->copies.size();
    // Signals and a flag slot.
    {
        std::unique_lock<std::mutex> lk(P.mu);
        if (!P.cv_slot.wait_for(lk, std::chrono::milliseconds(op->timeout_ms),
                                [&] { return !P.free_slots.empty(); })) {
            for (hipEvent_t e : op->gates) P.free_events.push_back(e);
            delete op;
            err = "no free handshake slot within the proxy timeout";
            return HOCCL_ERR_TIMEOUT;
        }
        op->slot = P.free_slots.back();
        P.free_slots.pop_back();
        while (op->sig.size() < sig_wanted && !P.free_signals.empty()) {
            op->sig.push_back(P.free_signals.back());
            P.free_signals.pop_back();
        }
    }
    auto give_back = [&]() {
        std::lock_guard<std::mutex> lk(P.mu);
        for (auto &x : op->sig) P.free_signals.push_back(x);
        for (hipEvent_t e : op->gates) P.free_events.push_back(e);
        P.free_slots.push_back(op->slot);
        delete op;
    };
    while (op->sig.size() < sig_wanted) {
        hsa_signal_t sg;
        if (hsa_signal_create(1, 0, nullptr, &sg) != HSA_STATUS_SUCCESS) {
            err = "hsa_signal_create failed";
            give_back();
            return HOCCL_ERR_HIP;
        }
        op->sig.push_back(sg);
    }
    // Every copy's signal is armed before any is issued: a copy waits on its
    // chain predecessor's signal, which must read "pending" until that copy
    // has been issued and has completed.  (Balanced pieces take and arm
    // their signals as they are issued.)
    for (auto &sg : op->sig) hsa_signal_store_screlease(sg, 1);
    // The handshake kernel runs on the caller's stream, or on the private
    // CU-masked stream when asked for (and that stream exists).
    hipStream_t hs = s;
    if (handshake == 1 && P.hs) {
        hipError_t e = hipEventRecord(P.ev_fork, s);
        if (e == hipSuccess) e = hipStreamWaitEvent(P.hs, P.ev_fork, 0);
        if (e != hipSuccess) {
            err = std::string("fork to the handshake stream failed: ") + hipGetErrorString(e);
            give_back();
            return HOCCL_ERR_HIP;
        }
        hs = P.hs;
    }
    // One dispatch carries the stream's whole side of the handshake.  It
    // stops waiting after wait_limit_us, by default twice the proxy timeout
    // plus a second, so the stream drains even if the proxy never answers
    // (the proxy's own watchdog reports first).  A free slot belongs to the
    // proxy; its flags are cleared here because a handshake that gave up
    // leaves FINISH set, which must never release a later wait early.
    store_flag(P.start_flag(op->slot), 0);
    store_flag(P.finish_flag(op->slot), 0);
    store_flag(P.status_flag(op->slot), 0);
    if (handshake == 2) {
        HostSide *h = new HostSide{P.start_flag(op->slot), P.finish_flag(op->slot),
                                   P.status_flag(op->slot),
                                   std::chrono::microseconds(
                                       wait_limit_us ? (uint64_t)wait_limit_us
                                                     : (2ull * op->timeout_ms + 1000ull) * 1000ull)};
        hipError_t e = hipLaunchHostFunc(s, host_side_handshake, h);
        if (e != hipSuccess) {
            delete h;
            (void)hipGetLastError();
            err = std::string("hipLaunchHostFunc failed: ") + hipGetErrorString(e);
            give_back();
            return HOCCL_ERR_HIP;
        }
        {
            std::lock_guard<std::mutex> lk(P.mu);
            P.incoming.push_back(op);
        }
        P.cv_work.notify_one();
        return HOCCL_OK;
    }
    HandshakeArgs ha;
    ha.start = (uint32_t *)P.start_flag(op->slot);
    ha.finish = (uint32_t *)P.finish_flag(op->slot);
    ha.status = (uint32_t *)P.status_flag(op->slot);
    ha.start_value = kStartValue;
    ha.finish_value = kFinishValue;
    ha.limit_ticks = wait_limit_us
                         ? std::max<uint64_t>(1, (uint64_t)wait_limit_us * P.ticks_per_ms / 1000)
                         : (2ull * op->timeout_ms + 1000ull) * P.ticks_per_ms;
    hipError_t e = launch_handshake(ha, hs);
    if (e != hipSuccess) {
        // Nothing of the handshake reached a stream: give everything back.
        (void)hipGetLastError();
        err = std::string("handshake launch failed: ") + hipGetErrorString(e);
        give_back();
        return HOCCL_ERR_HIP;
    }
    if (hs != s && ((e = hipEventRecord(P.ev_join, hs)) != hipSuccess ||
                    (e = hipStreamWaitEvent(s, P.ev_join, 0)) != hipSuccess)) {
        // Whatever part of the handshake reached the stream, the proxy must
        // still see the op through, so hand it over regardless and report.
        err = std::string("stream memory operation failed: ") + hipGetErrorString(e);
    }
    {
        std::lock_guard<std::mutex> lk(P.mu);
        P.incoming.push_back(op);
    }
    P.cv_work.notify_one();
    return e == hipSuccess ? HOCCL_OK : HOCCL_ERR_HIP;
}

hoccl_status_t Proxy::capture(const std::vector<ProxyCopy> &copies, int max_engines,
                              unsigned timeout_ms, unsigned wait_limit_us, hipStream_t s,
                              int *engines_used, std::string &err) {
    ProxyImpl &P = *impl_;
    CapturedOp *op = new CapturedOp();
    op->P = &P;
    {
        EngineSchedule sch = schedule_copies(P, copies, max_engines);
        op->copies = std::move(sch.copies);
        op->engine = std::move(sch.engine);
        op->deps = std::move(sch.deps);
        if (engines_used) *engines_used = sch.engines_used;
    }
    const uint64_t t = timeout_ms ? timeout_ms : 10000;
    op->limit = std::chrono::microseconds(wait_limit_us ? (uint64_t)wait_limit_us : (2 * t + 1000) * 1000);
    auto drop = [&]() {
        for (auto &sg : op->sig) hsa_signal_destroy(sg);
        delete op;
    };
    while (op->sig.size() < op->copies.size()) {
        hsa_signal_t sg;
        if (hsa_signal_create(0, 0, nullptr, &sg) != HSA_STATUS_SUCCESS) {
            err = "hsa_signal_create failed";
            drop();
            return HOCCL_ERR_HIP;
        }
        op->sig.push_back(sg);
    }
    hipError_t e = hipLaunchHostFunc(s, run_captured, op);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        err = std::string("capturing the copy host function failed: ") + hipGetErrorString(e);
        drop();
        return HOCCL_ERR_HIP;
    }
    std::lock_guard<std::mutex> lk(P.mu);
    P.captured.push_back(op);
    return HOCCL_OK;
}

}  // namespace hoccl
