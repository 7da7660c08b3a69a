// Host replay of every plan shape under AddressSanitizer and UBSan.
//
// Each rank's send and receive buffer is its own heap allocation of exactly
// the size the C ABI documents for the collective (in-place forms alias
// them the documented way), so a plan that reads or writes one byte outside
// a caller buffer or the workspace it asked for is reported by the sanitizer.
// The replay touches exactly the bytes the kernels and copies would: every
// reduction segment element by element with the element sizes of its phase,
// the direct fold with its chunk indexing, every copy with memmove.  The
// values are not checked here (the plan-replay tests compare them with the
// oracle); the arithmetic is a byte mix so that every byte is really read.
// The collective scheduler (stage decomposition and chunk interleave) runs
// here too, on random multi-node traffic, for its indexing.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "../../paper_2609_34334_amd/csrc/hoccl_internal.h"
#include "../../paper_2609_34334_amd/csrc/schedule.h"

using namespace hoccl;

namespace {

struct Bufs {
    std::vector<char *> send, recv, own;  // own: allocations to free
    char *ws = nullptr;
};

char *alloc(size_t n) {
    char *p = (char *)std::malloc(n ? n : 1);
    for (size_t i = 0; i < n; ++i) p[i] = (char)(i * 131 + 7);
    return p;
}

char *at(const BufRef &b, const Bufs &B) {
    switch (b.kind) {
    case BUF_SEND: return B.send[(size_t)b.rank] + b.off;
    case BUF_RECV: return B.recv[(size_t)b.rank] + b.off;
    case BUF_WS: return B.ws + b.off;
    default: std::fprintf(stderr, "bad buffer kind\n"); std::abort();
    }
}

void mix(char *out, const char *a, const char *b, size_t eo, size_t ea, size_t eb) {
    unsigned char t[8] = {0};
    for (size_t k = 0; k < ea; ++k) t[k % 8] ^= (unsigned char)a[k];
    for (size_t k = 0; k < eb; ++k) t[k % 8] += (unsigned char)b[k];
    std::memcpy(out, t, eo);
}

void replay(const Plan &p, const Bufs &B) {
    const size_t es = dtype_size(p.dtype), as = acc_size(p.dtype, p.bf16_partials);
    for (const ReduceStep &st : p.reduce_steps) {
        size_t e0 = (st.phase == PH_FIRST || st.phase == PH_ONLY) ? es : as;
        size_t eo = (st.phase == PH_LAST || st.phase == PH_ONLY) ? es : as;
        for (const ReduceSeg &g : st.segs) {
            char *in0 = at(g.in0, B), *in1 = at(g.in1, B), *out = at(g.out, B);
            std::vector<char *> more;
            for (const BufRef &m : g.more) more.push_back(at(m, B));
            for (size_t i = 0; i < g.n; ++i) {
                // the partial is read first; a fused step's further
                // contributions are read before the output is written
                char acc[8] = {0};
                mix(acc, in0 + i * e0, in1 + i * es, eo, e0, es);
                for (char *m : more) mix(acc, acc, m + i * es, eo, eo, es);
                std::memcpy(out + i * eo, acc, eo);
            }
        }
    }
    if (p.has_fold) {
        const FoldStep &f = p.fold;
        for (int j = 0; j < p.R; ++j) {
            size_t s0 = (size_t)j * f.c;
            if (s0 >= f.total) continue;
            size_t n = std::min(f.c, f.total - s0);
            size_t oe = f.out_at_chunk ? 0 : s0;
            for (size_t i = 0; i < n; ++i) {
                char acc[4] = {0};
                for (int k = 0; k < p.R; ++k) {
                    const char *x = B.send[(size_t)((j + 1 + k) % p.R)] + (s0 + i) * es;
                    mix(acc, acc, x, es, es, es);
                }
                int nout = f.write_all ? p.R : 1;
                for (int q = 0; q < nout; ++q)
                    std::memcpy(B.recv[(size_t)(f.write_all ? q : j)] + (oe + i) * es, acc, es);
            }
        }
    }
    for (const CopyOp &c : p.copies) std::memmove(at(c.dst, B), at(c.src, B), c.bytes);
}

int checked = 0;

void run(const Plan &p, int R, size_t send_bytes, size_t recv_bytes, int in_place) {
    Bufs B;
    B.send.resize((size_t)R);
    B.recv.resize((size_t)R);
    for (int r = 0; r < R; ++r) {
        if (in_place == 1) {            // all-gather: send[r] = recv[r] + r * sendcount
            B.recv[(size_t)r] = alloc(recv_bytes);
            B.own.push_back(B.recv[(size_t)r]);
            B.send[(size_t)r] = B.recv[(size_t)r] + (size_t)r * send_bytes;
        } else if (in_place == 2) {     // reduce-scatter: recv[r] = send[r] + r * recvcount
            B.send[(size_t)r] = alloc(send_bytes);
            B.own.push_back(B.send[(size_t)r]);
            B.recv[(size_t)r] = B.send[(size_t)r] + (size_t)r * recv_bytes;
        } else if (in_place == 3) {     // all-reduce: send[r] == recv[r]
            B.send[(size_t)r] = B.recv[(size_t)r] = alloc(send_bytes);
            B.own.push_back(B.send[(size_t)r]);
        } else {
            B.send[(size_t)r] = alloc(send_bytes);
            B.recv[(size_t)r] = alloc(recv_bytes);
            B.own.push_back(B.send[(size_t)r]);
            B.own.push_back(B.recv[(size_t)r]);
        }
    }
    if (p.ws_bytes) B.ws = alloc(p.ws_bytes);
    replay(p, B);
    std::free(B.ws);
    for (char *x : B.own) std::free(x);
    ++checked;
}

}  // namespace

int main() {
    const int Rs[] = {1, 2, 3, 4, 5, 8, 13, 64};
    const hoccl_dtype_t dts[] = {HOCCL_INT32, HOCCL_FP32, HOCCL_BF16, HOCCL_UINT8};
    for (int R : Rs)
        for (hoccl_dtype_t dt : dts) {
            const size_t es = dtype_size(dt);
            const bool sums = dt != HOCCL_UINT8;  // bytes: copy collectives only
            const size_t counts[] = {1, 7, (size_t)R * 5 + 3, 1000};
            for (size_t n : counts)
                for (int ip = 0; ip < 2; ++ip)
                    for (int algo = 0; algo < 2; ++algo)
                        for (int groups : {1, 3})
                            for (size_t chunk : {(size_t)0, (size_t)4096}) {
                                PlanOptions o;
                                o.in_place = ip != 0;
                                o.algo = (hoccl_reduce_algo_t)algo;
                                o.allreduce_groups = groups;
                                o.chunk_bytes = chunk;
                                for (int direct = 0; direct < 2; ++direct) {
                                    o.allgather_direct = direct != 0;
                                    if (sums) run(plan_allreduce(n, dt, R, o), R, n * es, n * es, ip ? 3 : 0);
                                    run(plan_allgather(n, dt, R, o), R, n * es, (size_t)R * n * es, ip ? 1 : 0);
                                }
                                if (sums)
                                    run(plan_reduce_scatter(n, dt, R, o), R, (size_t)R * n * es, n * es, ip ? 2 : 0);
                                if (algo == 0 && sums)
                                    for (int hops : {3, 64}) {  // fused ring hops
                                        PlanOptions f = o;
                                        f.fused_hops = hops;
                                        run(plan_allreduce(n, dt, R, f), R, n * es, n * es, ip ? 3 : 0);
                                        run(plan_reduce_scatter(n, dt, R, f), R, (size_t)R * n * es, n * es,
                                            ip ? 2 : 0);
                                    }
                                if (algo == 0 && dt == HOCCL_BF16) {  // bf16 partials (fused hops ignored)
                                    PlanOptions b = o;
                                    b.bf16_partials = true;
                                    b.fused_hops = 3;
                                    run(plan_allreduce(n, dt, R, b), R, n * es, n * es, ip ? 3 : 0);
                                    run(plan_reduce_scatter(n, dt, R, b), R, (size_t)R * n * es, n * es, ip ? 2 : 0);
                                }
                                if (ip) continue;
                                std::vector<int> shift((size_t)R), rev((size_t)R);
                                for (int r = 0; r < R; ++r) {
                                    shift[(size_t)r] = r + 1 < R ? r + 1 : -1;
                                    rev[(size_t)r] = R - 1 - r;
                                }
                                run(plan_sendrecv(n, dt, R, shift.data(), o), R, n * es, n * es, 0);
                                run(plan_sendrecv(n, dt, R, rev.data(), o), R, n * es, n * es, 0);
                                run(plan_alltoall(n, dt, R, o), R, (size_t)R * n * es, (size_t)R * n * es, 0);
                                PlanOptions st = o;  // the collective scheduler's stages
                                st.a2a_schedule = 1;
                                run(plan_alltoall(n, dt, R, st), R, (size_t)R * n * es, (size_t)R * n * es, 0);
                                // all-to-all(v): counts s->d from a fixed pattern, packed displacements
                                std::vector<size_t> C((size_t)R * R), sd((size_t)R * R), rd((size_t)R * R);
                                for (int s = 0; s < R; ++s)
                                    for (int d = 0; d < R; ++d)
                                        C[(size_t)s * R + d] = (size_t)((s * 7 + d * 3 + (int)n) % 11);
                                size_t smax = 0, rmax = 0;
                                for (int s = 0; s < R; ++s) {
                                    size_t off = 0;
                                    for (int d = 0; d < R; ++d) {
                                        sd[(size_t)s * R + d] = off;
                                        off += C[(size_t)s * R + d];
                                    }
                                    smax = std::max(smax, off);
                                }
                                for (int d = 0; d < R; ++d) {
                                    size_t off = 0;
                                    for (int s = 0; s < R; ++s) {
                                        rd[(size_t)s * R + d] = off;
                                        off += C[(size_t)s * R + d];
                                    }
                                    rmax = std::max(rmax, off);
                                }
                                run(plan_alltoallv(C.data(), sd.data(), rd.data(), dt, R, o), R, smax * es,
                                    rmax * es, 0);
                                run(plan_alltoallv(C.data(), sd.data(), rd.data(), dt, R, st), R, smax * es,
                                    rmax * es, 0);
                            }
        }
    // Scheduler: G GPUs in nodes of 2, 4 or 8, each GPU's symmetric peer the
    // neighbour in its own node (as in the paper's worked example), random
    // traffic with zeros, then the chunk interleave of a row.
    unsigned long long seed = 12345;
    auto rnd = [&]() {
        seed = seed * 6364136223846793005ull + 1442695040888963407ull;
        return (double)((seed >> 33) % 1000);
    };
    int schedules = 0;
    for (int G : {2, 4, 8, 16})
        for (int per : {2, 4, 8}) {
            if (per > G || G % per) continue;
            Topology t;
            t.G = G;
            t.bw_nvlink = 8.0;
            t.bw_rdma = 1.0;
            for (int g = 0; g < G; ++g) t.node.push_back(g / per);
            for (int g = 0; g < G; ++g) t.peer.push_back((g / per) * per + ((g % per) ^ 1));
            for (int rep = 0; rep < 5; ++rep) {
                std::vector<std::vector<double>> C((size_t)G, std::vector<double>((size_t)G, 0.0));
                for (int u = 0; u < G; ++u)
                    for (int v = 0; v < G; ++v) {
                        double x = rnd();
                        C[(size_t)u][(size_t)v] = (u != v && x > 300) ? x : 0.0;
                    }
                Schedule sc = decompose(t, C);
                (void)schedule_to_json(sc);
                std::vector<int> order = interleave_chunks(C[0], 64.0);
                (void)order;
                ++schedules;
            }
        }
    std::printf("plans replayed: %d, schedules: %d\n", checked, schedules);
    return 0;
}
