// The paper's collective scheduler for a described multi-node topology
// (Collective Scheduler section): the forwarding expansion of the traffic
// matrix, the Birkhoff-like stage decomposition (Algorithm 1) and the
// flow-size-aware interleaving of chunks on a DMA engine.
//
// On one GPU every flow stays inside one HBM, so the executor needs none of
// this; it is the planning layer a multi-node deployment would run before
// the point-to-point executor, kept host-only and checked against the
// paper's worked example and its constraints.
#include <algorithm>
#include <cmath>
#include <sstream>
#include <vector>

#include "schedule.h"

namespace hoccl {

namespace {

inline bool same_node(const Topology &t, int u, int v) { return t.node[(size_t)u] == t.node[(size_t)v]; }
inline bool is_rdma(const Topology &t, int u, int v) { return u != v && !same_node(t, u, v); }
inline bool is_forward_edge(const Topology &t, int u, int v) { return u != v && t.peer[(size_t)u] == v; }

using Mat = std::vector<std::vector<double>>;

Mat zeros(int G) { return Mat((size_t)G, std::vector<double>((size_t)G, 0.0)); }

}  // namespace

// Eq. 2-5: an inter-node flow f = C[u,v] becomes f' on (u, peer(u)), the
// RDMA transfer f on (u, v) and f'' on (peer(v), v).  A_u sums the f' of
// u's inter-node flows, B_v the f'' of the flows v receives from other
// nodes, and the NVLink edge between symmetric peers (u, peer(u)) carries
// C[u, peer(u)] + A_u + B_peer(u).  Every other entry keeps C.
std::vector<std::vector<double>> expand_traffic(const Topology &t, const std::vector<std::vector<double>> &C) {
    const int G = t.G;
    std::vector<double> A((size_t)G, 0.0), B((size_t)G, 0.0);
    for (int u = 0; u < G; ++u)
        for (int v = 0; v < G; ++v)
            if (is_rdma(t, u, v)) {
                A[(size_t)u] += C[(size_t)u][(size_t)v];
                B[(size_t)v] += C[(size_t)u][(size_t)v];
            }
    Mat T = C;
    for (int u = 0; u < G; ++u) {
        T[(size_t)u][(size_t)u] = 0.0;
        int v = t.peer[(size_t)u];
        if (v >= 0 && v != u && same_node(t, u, v)) T[(size_t)u][(size_t)v] += A[(size_t)u] + B[(size_t)v];
    }
    return T;
}

// Stage duration (Eq. 9-10): the slowest domain decides.  A domain's load is
// its largest entry in the stage; the NVLink domains share one bandwidth.
double stage_time(const Topology &t, const std::vector<std::vector<double>> &S) {
    double lr = 0.0, ln = 0.0;
    for (int u = 0; u < t.G; ++u)
        for (int v = 0; v < t.G; ++v) {
            double x = S[(size_t)u][(size_t)v];
            if (x <= 0.0) continue;
            if (is_rdma(t, u, v))
                lr = std::max(lr, x);
            else
                ln = std::max(ln, x);
        }
    return std::max(lr / t.bw_rdma, ln / t.bw_nvlink);
}

// Algorithm 1.  Readings where the paper is silent:
//  * the contention-free RDMA matching of a stage is built greedily from the
//    largest residual RDMA entries, taking an entry only if its sender has
//    no outgoing and its receiver no incoming RDMA flow yet (Eq. 8);
//  * "the largest removable portion" is the smallest residual entry of that
//    matching, so each stage empties at least one RDMA entry (the peeling
//    step of a Birkhoff-von Neumann decomposition);
//  * the forwarding copies of the moved portion go into the same stage, on
//    (u, peer(u)) and (peer(v), v);
//  * native NVLink traffic is split beforehand, per NVLink domain, into
//    matchings (each GPU at most one native send and one native receive),
//    again by greedy peeling; a stage is then topped up from those
//    components as far as every touched entry stays within the stage's
//    duration at NVLink bandwidth (the "slack");
//  * once RDMA traffic is exhausted, the remaining native components form
//    stages of their own.
Schedule decompose(const Topology &t, const std::vector<std::vector<double>> &C) {
    const int G = t.G;
    const double eps = 1e-9;
    Schedule out;
    out.T = expand_traffic(t, C);
    // residual RDMA flows and native (non-forwarding) NVLink flows
    Mat rdma = zeros(G), native = zeros(G);
    for (int u = 0; u < G; ++u)
        for (int v = 0; v < G; ++v) {
            if (u == v) continue;
            if (is_rdma(t, u, v))
                rdma[(size_t)u][(size_t)v] = C[(size_t)u][(size_t)v];
            else
                native[(size_t)u][(size_t)v] = C[(size_t)u][(size_t)v];
        }
    // Step 2: native NVLink traffic -> matching components.
    struct Component {
        std::vector<std::pair<int, int>> edges;
        std::vector<double> left;  // per edge
    };
    std::vector<Component> comps;
    {
        Mat r = native;
        for (;;) {
            std::vector<std::pair<double, std::pair<int, int>>> cand;
            for (int u = 0; u < G; ++u)
                for (int v = 0; v < G; ++v)
                    if (r[(size_t)u][(size_t)v] > eps) cand.push_back({r[(size_t)u][(size_t)v], {u, v}});
            if (cand.empty()) break;
            std::stable_sort(cand.begin(), cand.end(),
                             [](const auto &a, const auto &b) { return a.first > b.first; });
            std::vector<char> out_used((size_t)G, 0), in_used((size_t)G, 0);
            Component c;
            for (auto &e : cand) {
                int u = e.second.first, v = e.second.second;
                if (out_used[(size_t)u] || in_used[(size_t)v]) continue;
                out_used[(size_t)u] = in_used[(size_t)v] = 1;
                c.edges.push_back({u, v});
            }
            double m = 1e300;
            for (auto &e : c.edges) m = std::min(m, r[(size_t)e.first][(size_t)e.second]);
            for (auto &e : c.edges) {
                r[(size_t)e.first][(size_t)e.second] -= m;
                c.left.push_back(m);
            }
            comps.push_back(c);
        }
    }
    auto comps_left = [&]() {
        for (auto &c : comps)
            for (double x : c.left)
                if (x > eps) return true;
        return false;
    };
    auto rdma_left = [&]() {
        for (auto &row : rdma)
            for (double x : row)
                if (x > eps) return true;
        return false;
    };
    // Steps 3-9.
    while (rdma_left() || comps_left()) {
        Mat S = zeros(G);
        if (rdma_left()) {
            std::vector<std::pair<double, std::pair<int, int>>> cand;
            for (int u = 0; u < G; ++u)
                for (int v = 0; v < G; ++v)
                    if (rdma[(size_t)u][(size_t)v] > eps) cand.push_back({rdma[(size_t)u][(size_t)v], {u, v}});
            std::stable_sort(cand.begin(), cand.end(),
                             [](const auto &a, const auto &b) { return a.first > b.first; });
            std::vector<char> out_used((size_t)G, 0), in_used((size_t)G, 0);
            std::vector<std::pair<int, int>> match;
            for (auto &e : cand) {
                int u = e.second.first, v = e.second.second;
                if (out_used[(size_t)u] || in_used[(size_t)v]) continue;
                out_used[(size_t)u] = in_used[(size_t)v] = 1;
                match.push_back({u, v});
            }
            double m = 1e300;
            for (auto &e : match) m = std::min(m, rdma[(size_t)e.first][(size_t)e.second]);
            for (auto &e : match) {
                int u = e.first, v = e.second;
                rdma[(size_t)u][(size_t)v] -= m;
                S[(size_t)u][(size_t)v] += m;
                int pu = t.peer[(size_t)u], pv = t.peer[(size_t)v];
                if (pu >= 0 && pu != u && same_node(t, u, pu)) S[(size_t)u][(size_t)pu] += m;  // f'
                if (pv >= 0 && pv != v && same_node(t, pv, v)) S[(size_t)pv][(size_t)v] += m;  // f''
            }
            // Fill the NVLink slack with native matching components.
            double tau = stage_time(t, S);
            double cap = tau * t.bw_nvlink;
            for (auto &c : comps) {
                double amt = 1e300;
                bool any = false;
                for (size_t k = 0; k < c.edges.size(); ++k) {
                    if (c.left[k] <= eps) continue;
                    any = true;
                    const auto &e = c.edges[k];
                    double slack = cap - S[(size_t)e.first][(size_t)e.second];
                    amt = std::min(amt, std::min(slack, c.left[k]));
                }
                if (!any || amt <= eps) continue;
                for (size_t k = 0; k < c.edges.size(); ++k) {
                    if (c.left[k] <= eps) continue;
                    const auto &e = c.edges[k];
                    S[(size_t)e.first][(size_t)e.second] += amt;
                    c.left[k] -= amt;
                }
            }
        } else {
            // Only native NVLink traffic remains: one component per stage.
            for (auto &c : comps) {
                bool any = false;
                for (size_t k = 0; k < c.edges.size(); ++k)
                    if (c.left[k] > eps) {
                        any = true;
                        S[(size_t)c.edges[k].first][(size_t)c.edges[k].second] += c.left[k];
                        c.left[k] = 0.0;
                    }
                if (any) break;
            }
        }
        out.tau.push_back(stage_time(t, S));
        out.stages.push_back(std::move(S));
    }
    out.total = 0.0;
    for (double x : out.tau) out.total += x;
    return out;
}

// Flow-size-aware chunk order on one DMA engine: each flow is cut into
// chunks of `chunk` bytes and the next chunk always comes from the flow
// whose completed fraction after that chunk would be smallest (ties: the
// larger flow, then the lower index).  Large flows therefore get service in
// proportion to their size while small ones are revisited regularly, and
// all flows finish close together.
std::vector<int> interleave_chunks(const std::vector<double> &bytes, double chunk) {
    const size_t F = bytes.size();
    std::vector<long> total(F), done(F, 0);
    long all = 0;
    for (size_t i = 0; i < F; ++i) {
        total[i] = bytes[i] > 0 ? (long)std::ceil(bytes[i] / chunk) : 0;
        all += total[i];
    }
    std::vector<int> order;
    order.reserve((size_t)all);
    for (long k = 0; k < all; ++k) {
        int best = -1;
        double bf = 0.0;
        for (size_t i = 0; i < F; ++i) {
            if (done[i] >= total[i]) continue;
            double f = (double)(done[i] + 1) / (double)total[i];
            if (best < 0 || f < bf - 1e-12 ||
                (std::fabs(f - bf) <= 1e-12 && total[i] > total[(size_t)best])) {
                best = (int)i;
                bf = f;
            }
        }
        done[(size_t)best]++;
        order.push_back(best);
    }
    return order;
}

static void put_mat(std::ostringstream &os, const std::vector<std::vector<double>> &M) {
    os << "[";
    for (size_t u = 0; u < M.size(); ++u) {
        if (u) os << ",";
        os << "[";
        for (size_t v = 0; v < M[u].size(); ++v) {
            if (v) os << ",";
            os << M[u][v];
        }
        os << "]";
    }
    os << "]";
}

std::string schedule_to_json(const Schedule &s) {
    std::ostringstream os;
    os.precision(17);
    os << "{\"T\":";
    put_mat(os, s.T);
    os << ",\"stages\":[";
    for (size_t k = 0; k < s.stages.size(); ++k) {
        if (k) os << ",";
        put_mat(os, s.stages[k]);
    }
    os << "],\"tau\":[";
    for (size_t k = 0; k < s.tau.size(); ++k) {
        if (k) os << ",";
        os << s.tau[k];
    }
    os << "],\"total\":" << s.total << "}";
    return os.str();
}

BalancedIssue::BalancedIssue(int engines, size_t min_piece, size_t window, const std::vector<size_t> &copy_bytes)
    : min_piece_(std::max<size_t>(min_piece, 4096)), window_(window), copy_bytes_(copy_bytes),
      inflight_((size_t)std::max(engines, 1)), inflight_bytes_((size_t)std::max(engines, 1), 0),
      rate_((size_t)std::max(engines, 1), 0.0), last_done_us_((size_t)std::max(engines, 1), 0.0) {
    for (size_t b : copy_bytes) unissued_ += b;
    total_ = unissued_;
    took_.assign(inflight_.size(), 0);
    while (cur_ < copy_bytes_.size() && copy_bytes_[cur_] == 0) ++cur_;
}

size_t BalancedIssue::next_bytes(size_t e) const {
    const size_t r = copy_bytes_[cur_] - off_;
    const double E = (double)inflight_.size();
    if (!took_[e] && (double)r * E <= (double)total_) return r;
    size_t g = (size_t)std::ceil((double)unissued_ / E);
    g = std::max(min_piece_, (g + 4095) & ~(size_t)4095);
    return r <= g || r - g < min_piece_ / 2 ? r : g;
}

void BalancedIssue::advance(size_t b) {
    unissued_ -= b;
    off_ += b;
    if (off_ == copy_bytes_[cur_]) {
        off_ = 0;
        ++cur_;
        while (cur_ < copy_bytes_.size() && copy_bytes_[cur_] == 0) ++cur_;
    }
}

// The engine's oldest piece has completed (seen at now_us): it started when
// it was issued or when the engine's previous piece completed, whichever
// was later; its bytes over that time update the engine's rate (mean of the
// new and the old estimate).
void BalancedIssue::retire(size_t e, double now_us) {
    std::deque<int> &f = inflight_[e];
    const int i = f.front();
    const double start = std::max(issued_us_[(size_t)i], last_done_us_[e]);
    const double busy = now_us - start;
    if (busy > 0) {
        const double r = (double)piece_bytes_[(size_t)i] / busy;
        rate_[e] = rate_[e] > 0 ? 0.5 * (rate_[e] + r) : r;
    }
    last_done_us_[e] = now_us;
    inflight_bytes_[e] -= piece_bytes_[(size_t)i];
    inflight_total_ -= piece_bytes_[(size_t)i];
    f.pop_front();
}

// Time until engine e has run what it holds, at rate r.  The oldest piece
// has been running since it was issued or since the previous completion;
// once it is overdue, the time it has overrun counts as still to come, so
// an engine that stopped completing looks ever busier instead of idle.
double BalancedIssue::drain_us(size_t e, double now_us, double r) const {
    const std::deque<int> &f = inflight_[e];
    if (f.empty()) return 0.0;
    const int i = f.front();
    const double start = std::max(issued_us_[(size_t)i], last_done_us_[e]);
    const double expect = (double)piece_bytes_[(size_t)i] / r, ran = now_us - start;
    double t = ran < expect ? expect - ran : ran - expect;
    t += (double)(inflight_bytes_[e] - piece_bytes_[(size_t)i]) / r;
    return t;
}

// Whether engine e should take a piece of b bytes: it would finish it
// before the projected end of the operation (what all engines hold plus
// every unissued byte, over the sum of their rates), or within 5% (and
// 10 us) of the earliest finish any engine could give it.  Engines not yet
// measured are taken at the mean of the measured ones; before any
// measurement every engine qualifies.
bool BalancedIssue::earliest(size_t e, size_t b, double now_us) const {
    double sum = 0;
    int known = 0;
    for (double r : rate_)
        if (r > 0) {
            sum += r;
            ++known;
        }
    if (known == 0) return true;
    const double mean = sum / known;
    double total_rate = 0, held = 0, best = 1e300;
    for (size_t k = 0; k < inflight_.size(); ++k) {
        const double r = rate_[k] > 0 ? rate_[k] : mean;
        const double d = drain_us(k, now_us, r);
        total_rate += r;
        held += d * r;
        best = std::min(best, d + (double)b / r);
    }
    const double r = rate_[e] > 0 ? rate_[e] : mean;
    const double mine = drain_us(e, now_us, r) + (double)b / r;
    const double end = (held + (double)unissued_) / total_rate;
    return mine <= end || mine <= 1.05 * best + 10.0;
}

}  // namespace hoccl
