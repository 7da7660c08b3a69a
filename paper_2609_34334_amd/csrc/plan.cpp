// Planner: turns a collective call into a schedule of reduction steps and
// copies over symbolic buffers.
//
// The paper's collective scheduler turns a collective into a traffic matrix
// C of point-to-point flows and then into stages and DMA-engine chunk queues
// (Collective Scheduler: traffic matrix abstraction, Eq. 6-11 constraints,
// flow-size-aware chunk scheduling).  Here every virtual rank shares one
// HBM, so there is a single domain and no forwarding traffic: the flows of C
// become copies directly, each flow may be cut into fixed-size chunks, and
// the chunks are spread over the copy queues in proportion to their bytes.
// Reductions (outside the paper's scope) follow the ring: R-1 steps, and in
// step s rank r adds its element of chunk (r-s-2) mod R to the partial it
// received from rank r-1, so chunk j's fold starts at rank j+1 and ends at
// rank j.
#include <algorithm>
#include <cstdio>
#include <numeric>
#include <sstream>

#include "hoccl_internal.h"
#include "schedule.h"

namespace hoccl {

size_t dtype_size(hoccl_dtype_t dt) { return dt == HOCCL_BF16 ? 2 : dt == HOCCL_UINT8 ? 1 : 4; }
size_t acc_size(hoccl_dtype_t dt, bool bf16_partials) {
    return dt == HOCCL_BF16 && bf16_partials ? 2 : 4;
}

static inline int mod(int a, int R) { return ((a % R) + R) % R; }

bool use_direct(hoccl_reduce_algo_t algo, int R) {
    return algo == HOCCL_REDUCE_DIRECT || (algo == HOCCL_REDUCE_AUTO && R <= kDirectMaxRanks);
}

static BufRef ref(uint8_t kind, int rank, size_t off) {
    BufRef b;
    b.kind = kind;
    b.rank = rank;
    b.off = off;
    return b;
}

// Bytes one reduction segment must move: two reads and one write.
static unsigned long long seg_bytes(hoccl_dtype_t dt, bool bf16p, Phase ph, size_t n) {
    size_t e = dtype_size(dt), a = acc_size(dt, bf16p);
    switch (ph) {
    case PH_FIRST: return (unsigned long long)n * (e + e + a);
    case PH_MIDDLE: return (unsigned long long)n * (a + e + a);
    case PH_LAST: return (unsigned long long)n * (a + e + e);
    case PH_ONLY: return (unsigned long long)n * (e + e + e);
    }
    return 0;
}

// Appends `bytes` from src to dst, cut into pieces of at most chunk_bytes.
// Piece p of a chain becomes chain (chain * pieces + p) so that the pieces of
// one hop are independent while each piece still follows its own ring order.
static void add_copy(Plan &p, BufRef dst, BufRef src, size_t bytes, int chain, int group,
                     int level, size_t chunk_bytes, int pieces_per_chain) {
    if (bytes == 0) return;
    if (chunk_bytes == 0 || bytes <= chunk_bytes) {
        CopyOp c;
        c.dst = dst;
        c.src = src;
        c.bytes = bytes;
        c.chain = chain * pieces_per_chain;
        c.group = group;
        c.level = level;
        p.copies.push_back(c);
        p.copy_bytes += bytes;
        p.hbm_bytes += 2ull * bytes;
        return;
    }
    size_t off = 0;
    int piece = 0;
    while (off < bytes) {
        size_t b = std::min(chunk_bytes, bytes - off);
        CopyOp c;
        c.dst = dst;
        c.dst.off += off;
        c.src = src;
        c.src.off += off;
        c.bytes = b;
        c.chain = chain * pieces_per_chain + piece;
        c.group = group;
        c.level = level;
        p.copies.push_back(c);
        p.copy_bytes += b;
        p.hbm_bytes += 2ull * b;
        off += b;
        ++piece;
    }
}

static int pieces_for(size_t bytes, size_t chunk_bytes) {
    if (chunk_bytes == 0 || bytes <= chunk_bytes) return 1;
    return (int)((bytes + chunk_bytes - 1) / chunk_bytes);
}

static void finish_chains(Plan &p) {
    int m = -1;
    for (auto &c : p.copies) m = std::max(m, c.chain);
    // compact chain ids to 0..nchains-1 in first-appearance order
    std::vector<int> remap((size_t)(m + 1), -1);
    int next = 0;
    for (auto &c : p.copies) {
        if (remap[(size_t)c.chain] < 0) remap[(size_t)c.chain] = next++;
        c.chain = remap[(size_t)c.chain];
    }
    p.nchains = next;
}

// Ring reduction over the element range [e0, e0 + len) of every chunk j,
// where chunk j of rank r's send buffer starts at element j * stride.  The
// partial of element e lives at workspace element e (a mirror of the input
// index space) so it keeps the inputs' vector alignment.  Rank j's result
// goes to recv[j] at element out_base(j) + (e - j * stride).
//
// With H hops per launch, one launch performs ring hops s0 .. s0+H-1 for
// every chunk: chunk j's operands in fold order are x[j+1], x[j+2], ...,
// x[j] (rank indices mod R); hop s adds operand s+1 (rank j+s+2), the
// addition rank j+s+2 performs in the ring.  So a fused launch reads the
// partial once (on the first hop: x[j+1] itself), adds its H operands in
// that order and writes once.  H = 1 is the ring step itself; H >= R-1 folds
// every operand in one launch.
static void ring_reduce(Plan &p, hoccl_dtype_t dt, int R, size_t stride,
                        const std::vector<size_t> &chunk_len, size_t g0, size_t glen,
                        int group, bool out_at_chunk, int H) {
    size_t es = dtype_size(dt), as = acc_size(dt, p.bf16_partials);
    for (int s0 = 0; s0 <= R - 2; s0 += H) {
        const int s1 = std::min(s0 + H, R - 1);  // hops s0 .. s1-1
        const bool first = s0 == 0, last = s1 == R - 1;
        ReduceStep st;
        st.group = group;
        st.step = s0;
        st.hops = s1 - s0;
        st.phase = first ? (last ? PH_ONLY : PH_FIRST) : (last ? PH_LAST : PH_MIDDLE);
        // Segments in chunk order: launch block b serves segment b mod R
        // and lands on XCD b mod 8, so at R = 8 chunk j's partial is
        // written and read again by the same XCD at every step.
        for (int j = 0; j < R; ++j) {
            // The rank performing hop s0 of chunk j is r = j + s0 + 2.
            int r = mod(j + s0 + 2, R);
            size_t L = chunk_len[(size_t)j];
            if (g0 >= L) continue;
            size_t n = std::min(glen, L - g0);
            size_t e = (size_t)j * stride + g0;  // first element (input index space)
            ReduceSeg sg;
            sg.n = n;
            sg.in1 = ref(BUF_SEND, r, e * es);
            for (int h = s0 + 1; h < s1; ++h) sg.more.push_back(ref(BUF_SEND, mod(j + h + 2, R), e * es));
            if (first)
                sg.in0 = ref(BUF_SEND, mod(r - 1, R), e * es);
            else
                sg.in0 = ref(BUF_WS, 0, e * as);
            if (last) {
                size_t oe = out_at_chunk ? g0 : e;
                sg.out = ref(BUF_RECV, j, oe * es);
            } else {
                sg.out = ref(BUF_WS, 0, e * as);
            }
            p.hbm_bytes += seg_bytes(dt, p.bf16_partials, st.phase, n) +
                           (unsigned long long)n * es * sg.more.size();
            st.segs.push_back(std::move(sg));
        }
        if (!st.segs.empty()) p.reduce_steps.push_back(std::move(st));
    }
}

// Hops per ring launch from the option (0 and 1: one), at most kMaxHops.
static int hops_per_launch(const PlanOptions &o) {
    return std::max(1, std::min(o.fused_hops, kMaxHops));
}

// Groups a ring reduction over chunks of c elements is split into so that
// one group's partials (R chunk slices of acc-size elements) take at most
// `limit` bytes.  Two ranks keep no partials.
static int cache_groups(int R, size_t c, hoccl_dtype_t dt, bool bf16p, size_t limit) {
    if (limit == 0 || R <= 2 || c == 0) return 1;
    unsigned long long bytes = (unsigned long long)R * c * acc_size(dt, bf16p);
    unsigned long long G = (bytes + limit - 1) / limit;
    if (G > c) G = c;
    return (int)std::max(1ull, std::min(G, 1ull << 20));
}

Plan plan_reduce_scatter(size_t n, hoccl_dtype_t dt, int R, const PlanOptions &o) {
    Plan p;
    p.op = Op::ReduceScatter;
    p.dtype = dt;
    p.R = R;
    p.count = n;
    p.bf16_partials = o.bf16_partials && dt == HOCCL_BF16;
    if (n == 0) return p;
    size_t es = dtype_size(dt);
    if (R == 1) {
        if (!o.in_place)
            add_copy(p, ref(BUF_RECV, 0, 0), ref(BUF_SEND, 0, 0), n * es, 0, -1, 0,
                     o.chunk_bytes, pieces_for(n * es, o.chunk_bytes));
        finish_chains(p);
        return p;
    }
    if (use_direct(o.algo, R)) {
        p.has_fold = true;
        p.fold.c = n;
        p.fold.total = (size_t)R * n;
        p.fold.write_all = false;
        p.fold.out_at_chunk = true;
        p.hbm_bytes = (unsigned long long)R * n * (R * es + es);
        return p;
    }
    std::vector<size_t> len((size_t)R, n);
    const int G = cache_groups(R, n, dt, p.bf16_partials, o.group_partial_bytes);
    const size_t gl = (n + (size_t)G - 1) / (size_t)G;
    p.ngroups = G;
    const int H = hops_per_launch(o);
    for (int g = 0; g < G; ++g) ring_reduce(p, dt, R, n, len, (size_t)g * gl, gl, g, true, H);
    // Partials cross launches only when the hops take more than one.
    p.ws_bytes = (R - 1 > H) ? (size_t)R * n * acc_size(dt, p.bf16_partials) : 0;
    return p;
}

Plan plan_allreduce(size_t count, hoccl_dtype_t dt, int R, const PlanOptions &o) {
    Plan p;
    p.op = Op::AllReduce;
    p.dtype = dt;
    p.R = R;
    p.count = count;
    p.bf16_partials = o.bf16_partials && dt == HOCCL_BF16;
    if (count == 0) return p;
    size_t es = dtype_size(dt);
    if (R == 1) {
        if (!o.in_place)
            add_copy(p, ref(BUF_RECV, 0, 0), ref(BUF_SEND, 0, 0), count * es, 0, -1, 0,
                     o.chunk_bytes, pieces_for(count * es, o.chunk_bytes));
        finish_chains(p);
        return p;
    }
    size_t c = (count + (size_t)R - 1) / (size_t)R;
    std::vector<size_t> len((size_t)R);
    for (int j = 0; j < R; ++j) {
        size_t b = (size_t)j * c;
        len[(size_t)j] = b >= count ? 0 : std::min(c, count - b);
    }
    if (use_direct(o.algo, R)) {
        p.has_fold = true;
        p.fold.c = c;
        p.fold.total = count;
        p.fold.write_all = true;
        p.fold.out_at_chunk = false;
        p.hbm_bytes = (unsigned long long)count * (R * es + R * es);
        return p;
    }
    // allreduce_groups 0 is automatic: two groups once each rank holds at
    // least 32 MiB, so that the engine proxy's gather of group 0 overlaps
    // the reduction of group 1 (bf16, R = 8: 0.80 against 0.89 ms at 48 MiB
    // per rank), else one (2 MiB per rank: 0.18 ms with one, 0.24 with two).
    const int want = o.allreduce_groups > 0 ? o.allreduce_groups
                                            : (count * es >= ((size_t)32 << 20) ? 2 : 1);
    int G = std::max(want, cache_groups(R, c, dt, p.bf16_partials, o.group_partial_bytes));
    if ((size_t)G > c) G = (int)c;
    size_t cg = (c + (size_t)G - 1) / (size_t)G;
    p.ngroups = G;
    const int H = hops_per_launch(o);
    for (int g = 0; g < G; ++g) ring_reduce(p, dt, R, c, len, (size_t)g * cg, cg, g, false, H);
    // Gather phase: chunk j (group g) travels j -> j+1 -> ... -> j-1.
    int maxp = 1;
    for (int g = 0; g < G; ++g)
        for (int j = 0; j < R; ++j) {
            size_t L = len[(size_t)j];
            size_t g0 = (size_t)g * cg;
            if (g0 >= L) continue;
            maxp = std::max(maxp, pieces_for(std::min(cg, L - g0) * es, o.chunk_bytes));
        }
    for (int g = 0; g < G; ++g)
        for (int j = 0; j < R; ++j) {
            size_t L = len[(size_t)j];
            size_t g0 = (size_t)g * cg;
            if (g0 >= L) continue;
            size_t n = std::min(cg, L - g0);
            size_t off = ((size_t)j * c + g0) * es;
            for (int s = 0; s <= R - 2; ++s) {
                int src = o.allgather_direct ? j : mod(j + s, R);
                int dst = mod(j + s + 1, R);
                // ring: one chain per chunk (each hop reads the previous
                // hop's output); direct: every copy is its own chain.
                int chain = o.allgather_direct ? (g * R + j) * R + s : g * R + j;
                add_copy(p, ref(BUF_RECV, dst, off), ref(BUF_RECV, src, off), n * es, chain, g,
                         o.allgather_direct ? 0 : s, o.chunk_bytes, maxp);
            }
        }
    p.ws_bytes = (R - 1 > H) ? (size_t)R * c * acc_size(dt, p.bf16_partials) : 0;
    finish_chains(p);
    return p;
}

Plan plan_allgather(size_t n, hoccl_dtype_t dt, int R, const PlanOptions &o) {
    Plan p;
    p.op = Op::AllGather;
    p.dtype = dt;
    p.R = R;
    p.count = n;
    if (n == 0) return p;
    size_t es = dtype_size(dt), bytes = n * es;
    int P = pieces_for(bytes, o.chunk_bytes);
    // chain j carries shard j around the ring; the owner's own placement
    // (out-of-place only) is the first copy of the chain.
    for (int j = 0; j < R; ++j) {
        size_t off = (size_t)j * bytes;
        int level = 0;
        if (!o.in_place)
            add_copy(p, ref(BUF_RECV, j, off), ref(BUF_SEND, j, 0), bytes, j * R, -1, level++,
                     o.chunk_bytes, P);
        for (int s = 0; s <= R - 2; ++s) {
            int dst = mod(j + s + 1, R);
            BufRef src;
            if (o.allgather_direct || s == 0)
                src = ref(BUF_SEND, j, 0);
            else
                src = ref(BUF_RECV, mod(j + s, R), off);
            int chain = o.allgather_direct ? j * R + s + 1 : j * R;
            add_copy(p, ref(BUF_RECV, dst, off), src, bytes, chain, -1,
                     o.allgather_direct ? 0 : level + s, o.chunk_bytes, P);
        }
    }
    finish_chains(p);
    return p;
}

Plan plan_sendrecv(size_t n, hoccl_dtype_t dt, int R, const int *peers, const PlanOptions &o) {
    Plan p;
    p.op = Op::SendRecv;
    p.dtype = dt;
    p.R = R;
    p.count = n;
    if (n == 0) return p;
    size_t bytes = n * dtype_size(dt);
    int P = pieces_for(bytes, o.chunk_bytes);
    for (int r = 0; r < R; ++r) {
        int d = peers[r];
        if (d < 0) continue;
        add_copy(p, ref(BUF_RECV, d, 0), ref(BUF_SEND, r, 0), bytes, r, -1, 0, o.chunk_bytes, P);
    }
    finish_chains(p);
    return p;
}

// All-to-all(v) by the collective scheduler's stages (Collective
// Scheduler, Algorithm 1).  The traffic matrix C (bytes, one memory domain:
// every rank in one node, no symmetric peers, so no forwarding traffic) is
// decomposed into stages, each a matching: every rank sends at most one
// piece and receives at most one.  Flow (s, d) is cut into the pieces its
// stages carry, in stage order, each piece a chain of its own tagged with
// its stage (and, for the CU copy kernel, launched stage by stage through
// `level`).  The ranks' copies to themselves, which the decomposition
// leaves out, form one last stage.
static void plan_a2a_stages(Plan &p, const size_t *counts, const size_t *sd, const size_t *rd, int R,
                            size_t es) {
    Topology t;
    t.G = R;
    t.node.assign((size_t)R, 0);
    t.peer.assign((size_t)R, -1);
    std::vector<std::vector<double>> C((size_t)R, std::vector<double>((size_t)R, 0.0));
    for (int s = 0; s < R; ++s)
        for (int d = 0; d < R; ++d)
            if (s != d) C[(size_t)s][(size_t)d] = (double)(counts[(size_t)s * R + d] * es);
    Schedule sch = decompose(t, C);
    std::vector<size_t> done((size_t)R * R, 0);  // bytes of each flow planned so far
    int chain = 0;
    auto piece = [&](int s, int d, size_t bytes, int stage) {
        size_t k = (size_t)s * R + d;
        CopyOp c;
        c.dst = ref(BUF_RECV, d, rd[k] * es + done[k]);
        c.src = ref(BUF_SEND, s, sd[k] * es + done[k]);
        c.bytes = bytes;
        c.chain = chain++;
        c.stage = stage;
        c.level = stage;
        p.copies.push_back(c);
        p.copy_bytes += bytes;
        p.hbm_bytes += 2ull * bytes;
        done[k] += bytes;
    };
    int stage = 0;
    for (const auto &S : sch.stages) {
        bool any = false;
        for (int s = 0; s < R; ++s)
            for (int d = 0; d < R; ++d) {
                if (s == d || !(S[(size_t)s][(size_t)d] > 0.0)) continue;
                size_t k = (size_t)s * R + d, left = counts[k] * es - done[k];
                // The stage amounts are sums and differences of whole flow
                // sizes, so they are exact in double; clamp all the same.
                size_t b = std::min(left, (size_t)(S[(size_t)s][(size_t)d] + 0.5));
                if (b) {
                    piece(s, d, b, stage);
                    any = true;
                }
            }
        if (any) ++stage;
    }
    // Whatever a stage did not carry (none, as the decomposition is
    // complete) and the copies to self go last.
    bool any = false;
    for (int s = 0; s < R; ++s)
        for (int d = 0; d < R; ++d) {
            size_t k = (size_t)s * R + d, left = counts[k] * es - done[k];
            if (left) {
                piece(s, d, left, stage);
                any = true;
            }
        }
    (void)any;
    p.nchains = chain;
}

Plan plan_alltoall(size_t n, hoccl_dtype_t dt, int R, const PlanOptions &o) {
    Plan p;
    p.op = Op::AllToAll;
    p.dtype = dt;
    p.R = R;
    p.count = n;
    if (n == 0) return p;
    size_t bytes = n * dtype_size(dt);
    if (o.a2a_schedule != 0) {
        std::vector<size_t> counts((size_t)R * R, n), sd((size_t)R * R), rd((size_t)R * R);
        for (int s = 0; s < R; ++s)
            for (int d = 0; d < R; ++d) {
                sd[(size_t)s * R + d] = (size_t)d * n;
                rd[(size_t)s * R + d] = (size_t)s * n;
            }
        plan_a2a_stages(p, counts.data(), sd.data(), rd.data(), R, dtype_size(dt));
        return p;
    }
    int P = pieces_for(bytes, o.chunk_bytes);
    for (int s = 0; s < R; ++s)
        for (int d = 0; d < R; ++d)
            add_copy(p, ref(BUF_RECV, d, (size_t)s * bytes), ref(BUF_SEND, s, (size_t)d * bytes),
                     bytes, s * R + d, -1, 0, o.chunk_bytes, P);
    finish_chains(p);
    return p;
}

Plan plan_alltoallv(const size_t *counts, const size_t *sd, const size_t *rd, hoccl_dtype_t dt,
                    int R, const PlanOptions &o) {
    Plan p;
    p.op = Op::AllToAllV;
    p.dtype = dt;
    p.R = R;
    size_t es = dtype_size(dt);
    size_t total = 0;
    int P = 1;
    for (int k = 0; k < R * R; ++k) {
        total += counts[k];
        P = std::max(P, pieces_for(counts[k] * es, o.chunk_bytes));
    }
    p.count = total;
    if (o.a2a_schedule != 0) {
        plan_a2a_stages(p, counts, sd, rd, R, es);
        return p;
    }
    for (int s = 0; s < R; ++s)
        for (int d = 0; d < R; ++d) {
            size_t k = (size_t)s * R + d;
            add_copy(p, ref(BUF_RECV, d, rd[k] * es), ref(BUF_SEND, s, sd[k] * es), counts[k] * es,
                     (int)k, -1, 0, o.chunk_bytes, P);
        }
    finish_chains(p);
    return p;
}

std::vector<int> assign_chains(const Plan &p, int queues) {
    std::vector<unsigned long long> bytes((size_t)p.nchains, 0);
    for (auto &c : p.copies) bytes[(size_t)c.chain] += c.bytes;
    std::vector<int> order((size_t)p.nchains);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(),
                     [&](int a, int b) { return bytes[(size_t)a] > bytes[(size_t)b]; });
    std::vector<unsigned long long> load((size_t)std::max(1, queues), 0);
    std::vector<int> q((size_t)p.nchains, 0);
    for (int ch : order) {
        size_t best = 0;
        for (size_t k = 1; k < load.size(); ++k)
            if (load[k] < load[best]) best = k;
        q[(size_t)ch] = (int)best;
        load[best] += bytes[(size_t)ch];
    }
    return q;
}

static const char *kind_name(uint8_t k) {
    switch (k) {
    case BUF_SEND: return "send";
    case BUF_RECV: return "recv";
    case BUF_WS: return "ws";
    default: return "none";
    }
}

static void put_ref(std::ostringstream &os, const BufRef &b) {
    os << "[\"" << kind_name(b.kind) << "\"," << b.rank << "," << b.off << "]";
}

std::string plan_to_json(const Plan &p) {
    static const char *phases[] = {"first", "middle", "last", "only"};
    std::ostringstream os;
    os << "{\"op\":" << (int)p.op << ",\"dtype\":" << (int)p.dtype << ",\"R\":" << p.R
       << ",\"count\":" << p.count << ",\"ngroups\":" << p.ngroups << ",\"ws_bytes\":" << p.ws_bytes
       << ",\"hbm_bytes\":" << p.hbm_bytes << ",\"copy_bytes\":" << p.copy_bytes
       << ",\"nchains\":" << p.nchains << ",\"bf16_partials\":" << (p.bf16_partials ? 1 : 0)
       << ",\"reduce_steps\":[";
    for (size_t i = 0; i < p.reduce_steps.size(); ++i) {
        const auto &s = p.reduce_steps[i];
        if (i) os << ",";
        os << "{\"phase\":\"" << phases[s.phase] << "\",\"group\":" << s.group
           << ",\"step\":" << s.step << ",\"hops\":" << s.hops << ",\"segs\":[";
        for (size_t k = 0; k < s.segs.size(); ++k) {
            const auto &g = s.segs[k];
            if (k) os << ",";
            os << "{\"in0\":";
            put_ref(os, g.in0);
            os << ",\"in1\":";
            put_ref(os, g.in1);
            os << ",\"more\":[";
            for (size_t m = 0; m < g.more.size(); ++m) {
                if (m) os << ",";
                put_ref(os, g.more[m]);
            }
            os << "],\"out\":";
            put_ref(os, g.out);
            os << ",\"n\":" << g.n << "}";
        }
        os << "]}";
    }
    os << "],\"fold\":";
    if (p.has_fold)
        os << "{\"c\":" << p.fold.c << ",\"total\":" << p.fold.total
           << ",\"write_all\":" << (p.fold.write_all ? 1 : 0)
           << ",\"out_at_chunk\":" << (p.fold.out_at_chunk ? 1 : 0) << "}";
    else
        os << "null";
    os << ",\"copies\":[";
    for (size_t i = 0; i < p.copies.size(); ++i) {
        const auto &c = p.copies[i];
        if (i) os << ",";
        os << "{\"dst\":";
        put_ref(os, c.dst);
        os << ",\"src\":";
        put_ref(os, c.src);
        os << ",\"bytes\":" << c.bytes << ",\"chain\":" << c.chain << ",\"group\":" << c.group
           << ",\"level\":" << c.level << ",\"stage\":" << c.stage << "}";
    }
    os << "]}";
    return os.str();
}

}  // namespace hoccl
