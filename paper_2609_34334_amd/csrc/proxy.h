// Copy proxy: a CPU thread that drives chosen SDMA engines directly and is
// ordered with a HIP stream by the paper's start/finish flag handshake.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstddef>
#include <string>
#include <vector>

#include "../../include/hoccl.h"

namespace hoccl {

struct ProxyCopy {
    void *dst;
    const void *src;
    size_t bytes;
    int chain;      // copies of one chain run in order; chains are independent
    int gate = -1;  // index into submit's `gates`, or -1: wait for the stream
    int stage = -1; // collective-scheduler stage (all-to-all), or -1
};

class ProxyImpl;

class Proxy {
  public:
    // Null when the device's SDMA engines cannot be driven directly; *why
    // then says which step failed.
    static Proxy *create(int device, std::string *why);
    ~Proxy();

    int engine_count() const;

    // The error the proxy thread stored since the last call (a watchdog
    // timeout, a failed copy issue), cleared by this call; HOCCL_OK if none.
    // The executor takes it before it enqueues anything, so a call that
    // reports it has enqueued nothing.
    hoccl_status_t take_error(std::string &err);

    // Events for submit's `gates`, taken from the proxy's pool.  They return
    // to it when the operation that uses them retires, or by
    // release_events if the caller does not submit after all.
    hoccl_status_t acquire_events(int n, std::vector<hipEvent_t> &out, std::string &err);
    void release_events(std::vector<hipEvent_t> &events);

    // Enqueues the handshake on `s` and hands the copies to the proxy
    // thread; returns once enqueued.  Copies run on at most `max_engines`
    // engines (0 = all), balanced by bytes per engine.  A copy with gate
    // g >= 0 is issued as soon as gates[g] (recorded by the caller on `s`
    // before the handshake) has completed, which the proxy thread polls;
    // the others when the stream reaches the handshake.  The handshake
    // releases the stream once every copy has completed.  The operation
    // takes the gate events over, also when it fails.
    // The stream side of the start/finish flag handshake (`handshake`, as
    // hoccl_config_t.proxy_handshake): 0, a one-lane kernel on `s`; 1, that
    // kernel on the proxy's private CU-masked stream joined to `s` by
    // events; 2, a host function on `s` run by the HIP runtime's callback
    // thread.  It stops waiting after wait_limit_us (0: twice the timeout
    // plus a second).
    // Copies tagged with stages (all of them, or none) are scheduled stage
    // by stage instead: each stage's copies over the engines by bytes, every
    // engine's queue in stage order.
    // With slice_bytes > 0, an operation whose copies wait for no other copy
    // and share one gate is issued balanced (BalancedIssue): the scheduled
    // copies, in their issue order, are cut into guided pieces as the
    // engines take them (an engine's first piece whole where it fits its
    // share; then the unissued bytes over the engine count, at least
    // slice_bytes).  An engine takes a piece while it holds fewer than two
    // or the piece fits within 2 * slice_bytes with those it holds, and only
    // if, at the engines' measured rates, it would finish the piece before
    // the operation's projected end or about as early as any engine could.
    // Otherwise (and with slice_bytes 0) every copy is issued at once on its
    // scheduled engine.
    hoccl_status_t submit(const std::vector<ProxyCopy> &copies, int max_engines, size_t slice_bytes,
                          unsigned timeout_ms, unsigned wait_limit_us, int handshake,
                          hipStream_t s, int *engines_used, std::string &err,
                          std::vector<hipEvent_t> gates = {});

    // For a stream that is capturing a graph: records a host node on `s`
    // that, at every replay, issues the copies on their engines and returns
    // once they have completed (no GPU code, no proxy thread).  The copy
    // list stays allocated until the proxy is destroyed.
    hoccl_status_t capture(const std::vector<ProxyCopy> &copies, int max_engines,
                           unsigned timeout_ms, unsigned wait_limit_us, hipStream_t s,
                           int *engines_used, std::string &err);

  private:
    explicit Proxy(ProxyImpl *impl) : impl_(impl) {}
    ProxyImpl *impl_;
};

}  // namespace hoccl
