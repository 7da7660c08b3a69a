// The SDMA proxy's balanced issue (BalancedIssue) against a simulation of
// engines that run their commands in order at given rates, with a fixed
// start-up cost per command, on the CPU.  Checks that the pieces cover
// every copy's bytes exactly once and in order, that an engine holding two
// pieces only takes another within its byte window, that every engine gets
// work before any gets a second piece, that the first round cuts no copy
// smaller than an engine's share, that a half-speed engine costs only its
// share of the work (against issuing every copy at once on a byte-balanced
// engine) and a
// nearly stalled one little more than the two pieces it was dealt before
// any rate was known, that equal engines lose at most a little to the
// extra commands, and that after a failed issue nothing more is issued and
// the issued pieces cover a prefix of the bytes.  Built with
// AddressSanitizer and UBSan.
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <deque>
#include <numeric>
#include <random>
#include <vector>

#include "../../paper_2609_34334_amd/csrc/schedule.h"

using hoccl::BalancedIssue;
using hoccl::Piece;

static int failures = 0;
static int cases = 0;

#define CHECK(cond, ...)                                              \
    do {                                                              \
        if (!(cond)) {                                                \
            std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
            std::fprintf(stderr, __VA_ARGS__);                        \
            std::fprintf(stderr, "\n");                               \
            ++failures;                                               \
        }                                                             \
    } while (0)

static const size_t MiB = (size_t)1 << 20;
static const double kRate = 57e3;    // about 57 GB/s per engine, in bytes per microsecond
static const double kStartUs = 7.0;  // an engine command's fixed start-up cost
static const double kDt = 2.0;       // the proxy passes every 2 us

struct Sim {
    double makespan = 0;
    size_t pieces = 0;
    std::vector<int> engines_used;
};

// Engines drain their FIFOs (start-up cost, then bytes at rate[e]); the
// proxy makes one pass every kDt.  fail_at: the issue call that fails.
static Sim run_balanced(const std::vector<double> &rate, size_t minp, size_t window,
                        const std::vector<size_t> &copies, int fail_at = -1) {
    const int E = (int)rate.size();
    BalancedIssue b(E, minp, window, copies);
    std::vector<std::deque<int>> fifo((size_t)E);
    std::vector<double> left, start;
    std::vector<size_t> bytes;
    std::vector<char> done;
    const double total = std::accumulate(copies.begin(), copies.end(), 0.0);
    size_t cur = 0, off = 0;  // the next byte the pieces must start at
    while (cur < copies.size() && copies[cur] == 0) ++cur;
    int issues = 0;
    bool failed = false, first_round = true;
    double t = 0.0;
    Sim sim;
    sim.engines_used.assign((size_t)E, 0);
    for (;;) {
        std::vector<int> got((size_t)E, 0);
        b.pass(t, [&](int i) { return done[(size_t)i] != 0; },
               [&](int e, const Piece &p) {
                   CHECK(!failed, "a piece was issued after a failed issue");
                   if (issues++ == fail_at) {
                       failed = true;
                       return false;
                   }
                   CHECK(p.id == (int)bytes.size(), "piece id %d, expected %zu", p.id, bytes.size());
                   CHECK(p.copy == (int)cur && p.offset == off, "piece of copy %d at %zu, expected copy %zu at %zu",
                         p.copy, p.offset, cur, off);
                   CHECK(p.bytes > 0 && p.offset + p.bytes <= copies[(size_t)p.copy], "piece overruns its copy");
                   if (p.offset + p.bytes < copies[(size_t)p.copy])
                       CHECK(p.bytes % 4096 == 0 && p.bytes >= minp, "inner piece of %zu bytes", p.bytes);
                   off += p.bytes;
                   if (off == copies[cur]) {
                       off = 0;
                       ++cur;
                       while (cur < copies.size() && copies[cur] == 0) ++cur;
                   }
                   std::deque<int> &f = fifo[(size_t)e];
                   double fb = (double)p.bytes;
                   for (int k : f) fb += (double)bytes[(size_t)k];
                   CHECK(f.size() < 2 || fb <= (double)window, "engine %d topped up past its window", e);
                   if (first_round) {
                       if (got[(size_t)e] > 0)
                           for (int o = 0; o < e; ++o)
                               CHECK(got[(size_t)o] > 0, "engine %d got a second piece before engine %d had one", e,
                                     o);
                       // It cuts only a copy larger than an engine's share.
                       if (got[(size_t)e] == 0)
                           CHECK(p.offset == 0 || (double)copies[(size_t)p.copy] * E > total,
                                 "the first round cut a copy of %zu bytes", copies[(size_t)p.copy]);
                   }
                   ++got[(size_t)e];
                   bytes.push_back(p.bytes);
                   left.push_back((double)p.bytes);
                   start.push_back(kStartUs);
                   done.push_back(0);
                   sim.engines_used[(size_t)e] = 1;
                   f.push_back(p.id);
                   return true;
               });
        first_round = false;
        bool busy = false;
        for (auto &f : fifo) busy |= !f.empty();
        if (b.all_issued() && !busy) break;
        for (int e = 0; e < E; ++e) {
            double budget = kDt;  // microseconds of engine time this step
            std::deque<int> &f = fifo[(size_t)e];
            while (budget > 0 && !f.empty()) {
                const int i = f.front();
                const double s = std::min(budget, start[(size_t)i]);
                start[(size_t)i] -= s;
                budget -= s;
                const double d = std::min(budget * rate[(size_t)e], left[(size_t)i]);
                left[(size_t)i] -= d;
                budget -= d / rate[(size_t)e];
                if (start[(size_t)i] <= 0 && left[(size_t)i] <= 0) {
                    done[(size_t)i] = 1;
                    f.pop_front();
                }
            }
        }
        t += kDt;
        if (t > 1e9) {
            CHECK(false, "simulation did not finish");
            break;
        }
    }
    if (fail_at < 0 || fail_at >= issues)
        CHECK(cur == copies.size(), "pieces stopped at copy %zu of %zu", cur, copies.size());
    else
        CHECK(b.all_issued() && issues == fail_at + 1, "issue went on after the failure");
    sim.makespan = t;
    sim.pieces = bytes.size();
    return sim;
}

// Every copy issued at once, copies byte-balanced over the engines
// (largest first onto the least loaded), each with its start-up cost.
static double run_static(const std::vector<double> &rate, const std::vector<size_t> &copies) {
    std::vector<size_t> order(copies.size());
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](size_t a, size_t b) { return copies[a] > copies[b]; });
    std::vector<double> load(rate.size(), 0.0), time(rate.size(), 0.0);
    for (size_t i : order) {
        size_t best = 0;
        for (size_t e = 1; e < rate.size(); ++e)
            if (load[e] < load[best]) best = e;
        load[best] += (double)copies[i];
        time[best] += kStartUs + (double)copies[i] / rate[best];
    }
    return *std::max_element(time.begin(), time.end());
}

struct Shape {
    const char *name;
    std::vector<size_t> copies;
    int engines;
};

int main() {
    const bool verbose = std::getenv("BALANCE_SIM_VERBOSE") != nullptr;
    const size_t minp = 4 * MiB, window = 2 * minp;
    // Random shapes and rates: coverage, order and the window.
    std::mt19937_64 g(7);
    for (int rep = 0; rep < 120; ++rep) {
        std::vector<size_t> copies;
        const int n = 1 + (int)(g() % 40);
        for (int c = 0; c < n; ++c) copies.push_back(g() % 5 == 0 ? (size_t)(g() % 70000) : 1 + g() % (96 * MiB));
        const int E = 1 + (int)(g() % 16);
        std::vector<double> rate((size_t)E);
        for (double &r : rate) r = kRate * (0.05 + (double)(g() % 100) / 100.0);
        const size_t mp = (size_t)(1 + g() % 64) << 16;
        run_balanced(rate, mp, 2 * mp, copies);
        ++cases;
    }
    std::vector<Shape> shapes = {
        {"FSDP all-gather, 64 x 48 MiB on 16 engines", std::vector<size_t>(64, 48 * MiB), 16},
        {"1 GiB all-gather, 64 x 128 MiB on 16 engines", std::vector<size_t>(64, 128 * MiB), 16},
        {"FSDP all-gather on 4 engines", std::vector<size_t>(64, 48 * MiB), 4},
        {"64 MiB send/recv cut into 16 pieces on 16 engines", std::vector<size_t>(16, 4 * MiB), 16},
        {"64 MiB send/recv cut into 4 pieces on 4 engines", std::vector<size_t>(4, 16 * MiB), 4},
        {"7 messages of 32 MiB on 4 engines", std::vector<size_t>(7, 32 * MiB), 4},
    };
    for (const Shape &sh : shapes) {
        const double total = std::accumulate(sh.copies.begin(), sh.copies.end(), 0.0);
        std::vector<double> rate((size_t)sh.engines, kRate);
        Sim eq = run_balanced(rate, minp, window, sh.copies);
        const double st = run_static(rate, sh.copies);
        CHECK(eq.makespan <= 1.03 * st + 4 * kDt, "%s, equal engines: balanced %.0f us against static %.0f us",
              sh.name, eq.makespan, st);
        // Few commands: the copies plus a few per engine at the end.
        CHECK(eq.pieces <= sh.copies.size() + 6 * (size_t)sh.engines, "%s: %zu pieces", sh.name, eq.pieces);
        if (sh.copies.size() >= (size_t)sh.engines)
            CHECK(std::accumulate(eq.engines_used.begin(), eq.engines_used.end(), 0) == sh.engines,
                  "%s: an engine never ran", sh.name);
        if (verbose)
            std::printf("%s: %zu pieces, balanced %.0f us, static %.0f us\n", sh.name, eq.pieces, eq.makespan, st);
        if (total < 512.0 * MiB) {
            ++cases;
            continue;
        }
        for (int slow = 0; slow < sh.engines; slow += 5) {
            rate.assign((size_t)sh.engines, kRate);
            rate[(size_t)slow] = kRate / 2;
            const double ideal = total / std::accumulate(rate.begin(), rate.end(), 0.0);
            Sim bal = run_balanced(rate, minp, window, sh.copies);
            const double sst = run_static(rate, sh.copies);
            CHECK(bal.makespan <= 1.06 * ideal, "%s, engine %d at half rate: balanced %.0f us against ideal %.0f us",
                  sh.name, slow, bal.makespan, ideal);
            CHECK(sst >= 1.3 * bal.makespan, "%s, engine %d at half rate: static %.0f us, balanced %.0f us",
                  sh.name, slow, sst, bal.makespan);
            if (verbose)
                std::printf("%s, engine %d at half rate: balanced %.0f us, static %.0f us, ideal %.0f us\n", sh.name,
                            slow, bal.makespan, sst, ideal);
        }
        // One engine at a twentieth of the rate: the others take over all
        // but the two pieces it was dealt before its rate was known.
        rate.assign((size_t)sh.engines, kRate);
        rate[0] = kRate / 20;
        const double ideal = total / std::accumulate(rate.begin(), rate.end(), 0.0);
        const double first = (double)(sh.copies[0] + sh.copies[(size_t)sh.engines]) / rate[0];
        Sim bal = run_balanced(rate, minp, window, sh.copies);
        CHECK(bal.makespan <= std::max(1.15 * ideal, first + 4 * kStartUs + 4 * kDt),
              "%s, engine 0 at 1/20 rate: balanced %.0f us against ideal %.0f us", sh.name, bal.makespan, ideal);
        if (verbose)
            std::printf("%s, engine 0 at 1/20 rate: balanced %.0f us, ideal %.0f us, its first pieces %.0f us\n",
                        sh.name, bal.makespan, ideal, first);
        ++cases;
    }
    // Small copies (an EP all-to-all's 56 blocks of 64 KiB on 4 engines):
    // everything goes out in the first pass, as when issued at once.
    {
        BalancedIssue b(4, minp, window, std::vector<size_t>(56, (size_t)64 << 10));
        int n = 0;
        b.pass(0.0, [](int) { return false; }, [&](int, const Piece &) { ++n; return true; });
        CHECK(n == 56 && b.all_issued(), "small copies: %d of 56 issued in the first pass", n);
        ++cases;
    }
    // One engine, any sizes, zero-byte copies among them.
    {
        std::vector<size_t> copies = {0, 1, 4096, 9 * MiB, 0, 12345, 3 * MiB, 0};
        run_balanced({kRate}, minp, window, copies);
        ++cases;
    }
    // A failed issue: nothing more is issued, and what was issued is an
    // exact prefix of the bytes (checked inside run_balanced).
    for (int fail_at : {0, 1, 9, 31, 95}) {
        run_balanced(std::vector<double>(6, kRate), MiB, 2 * MiB, std::vector<size_t>(96, 2 * MiB), fail_at);
        ++cases;
    }
    std::printf("balance cases: %d\n", cases);
    return failures ? 1 : 0;
}
