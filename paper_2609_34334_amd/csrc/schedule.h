// The paper's collective scheduler on a described multi-node topology.
#pragma once

#include <cstddef>
#include <deque>
#include <string>
#include <vector>

namespace hoccl {

struct Topology {
    int G = 0;
    std::vector<int> node;  // NVLink / xGMI domain of each GPU
    std::vector<int> peer;  // symmetric peer of each GPU (-1: none)
    double bw_nvlink = 1.0; // bytes per unit time of an intra-node edge
    double bw_rdma = 1.0;   // bytes per unit time of an inter-node edge
};

struct Schedule {
    std::vector<std::vector<double>> T;                   // expanded traffic
    std::vector<std::vector<std::vector<double>>> stages; // T^1 .. T^n
    std::vector<double> tau;                              // stage durations
    double total = 0.0;                                   // sum of tau
};

std::vector<std::vector<double>> expand_traffic(const Topology &t,
                                                const std::vector<std::vector<double>> &C);
double stage_time(const Topology &t, const std::vector<std::vector<double>> &S);
Schedule decompose(const Topology &t, const std::vector<std::vector<double>> &C);
std::vector<int> interleave_chunks(const std::vector<double> &bytes, double chunk);
std::string schedule_to_json(const Schedule &s);

// Balanced issue of copies that wait for no other over a set of engines
// (flow-size-aware chunk scheduling).  The copies, in their scheduled
// order, are cut into pieces as engines take them (guided self-scheduling):
// an engine's first piece is a whole copy unless the copy exceeds an
// engine's share of the total; after that a piece is the unissued bytes
// over the engine count, at least min_piece and rounded up to 4 KiB, and a
// copy's remainder goes whole when cutting would leave less than half of
// min_piece.  So a plan that is already balanced goes out as it is, and
// pieces shrink as the end nears.
//
// An engine has room while it holds fewer than two pieces (an engine whose
// queue runs dry restarts slowly, so one piece always waits behind the
// running one), or when the next piece fits within `window` bytes with
// those it holds (small pieces queue deeper).  An engine with room takes
// the piece if it would finish it before the projected end of the whole
// operation (all remaining bytes over the sum of the engines' rates, each
// measured on its completed pieces) or about as early as any engine could;
// so an engine slowed by other work keeps contributing but does not take
// the last pieces from faster ones.  An engine runs its pieces in order, so
// a pass first retires each engine's completed pieces from the front of its
// list, then deals pieces one per engine per round (every engine gets work
// before any gets a second) until no engine takes more.
struct Piece {
    int id;  // 0, 1, ... in issue order
    int copy;
    size_t offset, bytes;
};

class BalancedIssue {
  public:
    BalancedIssue() = default;
    BalancedIssue(int engines, size_t min_piece, size_t window, const std::vector<size_t> &copy_bytes);

    // One pass at time now_us (a monotonic clock, microseconds).  done(id):
    // whether issued piece id has completed.  issue(e, piece): issue the
    // piece on engine slot e, false if that failed; then nothing more is
    // issued.  Returns whether any piece completed or was issued.
    template <class Done, class Issue>
    bool pass(double now_us, Done done, Issue issue) {
        bool moved = false;
        for (size_t e = 0; e < inflight_.size(); ++e)
            while (!inflight_[e].empty() && done(inflight_[e].front())) {
                retire(e, now_us);
                moved = true;
            }
        for (bool round = true; round && !all_issued();) {
            round = false;
            for (size_t e = 0; e < inflight_.size() && !all_issued(); ++e) {
                const size_t b = next_bytes(e);
                if (inflight_[e].size() >= 2 && inflight_bytes_[e] + b > window_) continue;
                if (!earliest(e, b, now_us)) continue;
                const Piece p{(int)piece_bytes_.size(), (int)cur_, off_, b};
                round = moved = true;
                if (!issue((int)e, p)) {
                    failed_ = true;
                    return true;
                }
                advance(b);
                took_[e] = 1;
                piece_bytes_.push_back(b);
                issued_us_.push_back(now_us);
                inflight_[e].push_back(p.id);
                inflight_bytes_[e] += b;
                inflight_total_ += b;
            }
        }
        return moved;
    }

    bool all_issued() const { return cur_ == copy_bytes_.size() || failed_; }
    size_t issued() const { return piece_bytes_.size(); }
    // Measured rate of engine slot e in bytes per microsecond (0: none yet).
    double rate(size_t e) const { return rate_[e]; }

  private:
    size_t next_bytes(size_t e) const;
    void advance(size_t b);
    void retire(size_t e, double now_us);
    double drain_us(size_t e, double now_us, double r) const;
    bool earliest(size_t e, size_t b, double now_us) const;

    size_t min_piece_ = 4096, window_ = 0;
    std::vector<size_t> copy_bytes_;
    size_t cur_ = 0, off_ = 0;  // the next unissued byte: copy cur_, offset off_
    unsigned long long total_ = 0, unissued_ = 0, inflight_total_ = 0;
    std::vector<char> took_;  // per engine: whether it has taken a piece
    std::vector<size_t> piece_bytes_;
    std::vector<double> issued_us_;
    std::vector<std::deque<int>> inflight_;
    std::vector<unsigned long long> inflight_bytes_;
    std::vector<double> rate_, last_done_us_;
    bool failed_ = false;
};

}  // namespace hoccl
