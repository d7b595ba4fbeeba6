// Host-compiled simulation of the one-pass geometry build's look-back, using
// the same status rules as the kernel (lookback.h).  Rows take tickets in
// order, run concurrently under a random schedule, publish their size, look
// back over 64 predecessors per step exactly as the kernel's lanes do, and
// give up after `spin_limit` failed polls.  Checked, over many schedules:
//   * with a large limit no row gives up and the stripped row_ptr is the
//     exclusive scan of the sizes;
//   * with limit 0 rows do give up; every row that is not poisoned still has
//     its exact offset; a row whose look-back reaches a poisoned prefix is
//     poisoned; and the stripped total row_ptr[R] is negative exactly when
//     some row is poisoned.
// Prints one line per case and exits 0 when every check holds.
#include <cstdint>
#include <cstdio>
#include <random>
#include <vector>

#include "lookback.h"

namespace lb = ris::lookback;

struct Row {
    int state = 0;          // 0 waiting for its ticket, 1 building, 2 looking back, 3 done
    int64_t count = 0;
    int64_t j = 0;          // look-back position (rows below j are still to be summed)
    int64_t prefix = 0;
    uint32_t spins = 0;
    int build_left = 0;
    bool poisoned = false;
    bool met_poison = false;
};

struct Result {
    bool ok = true;
    int64_t poisoned = 0;
};

static Result simulate(int64_t R, uint32_t spin_limit, unsigned seed) {
    std::mt19937_64 rng(seed);
    std::vector<int64_t> status(R + 1, 0);   // status of row r in status[r + 1]
    std::vector<Row> rows(R);
    std::vector<int64_t> truth(R + 1, 0);
    for (int64_t r = 0; r < R; ++r) {
        rows[r].count = (int64_t)(rng() % 2000);
        rows[r].build_left = (int)(rng() % 6);
        truth[r + 1] = truth[r] + rows[r].count;
    }
    int64_t next_ticket = 0, done = 0;
    std::vector<int64_t> active;
    const size_t width = 1 + rng() % 48;     // rows in flight
    while (done < R) {
        while (active.size() < width && next_ticket < R) {
            rows[next_ticket].state = 1;
            rows[next_ticket].j = next_ticket;
            active.push_back(next_ticket++);
        }
        const size_t pick = rng() % active.size();
        const int64_t r = active[pick];
        Row& w = rows[r];
        if (w.state == 1) {
            if (w.build_left-- > 0) continue;
            status[r + 1] = lb::aggregate(w.count);
            w.state = 2;
            continue;
        }
        // one look-back step: "lane" i reads the status of row j - 1 - i
        bool finished = false;
        if (w.j == 0) {
            finished = true;
        } else {
            int64_t v[64];
            uint64_t inc = 0, ready = 0;
            for (int i = 0; i < 64; ++i) {
                const int64_t idx = w.j - i;
                v[i] = idx > 0 ? status[idx] : lb::inclusive(0, false);
                if (lb::is_inclusive(v[i])) inc |= 1ull << i;
                if (lb::is_ready(v[i])) ready |= 1ull << i;
            }
            const int first = lb::step_end(inc, ready);
            if (first < 0) {
                if (w.spins++ >= spin_limit) { w.poisoned = true; finished = true; }
            } else {
                int64_t part = 0;
                for (int i = 0; i < first && i < 64; ++i) part += lb::value(v[i]);
                if (first < 64) {
                    if (lb::is_poisoned(v[first])) {
                        w.poisoned = true;
                        w.met_poison = true;
                    } else {
                        part += lb::value(v[first]);
                    }
                }
                if (!w.poisoned) w.prefix += part;
                if (first < 64) finished = true;
                else w.j -= 64;
            }
        }
        if (finished) {
            status[r + 1] = lb::inclusive(w.prefix + w.count, w.poisoned);
            w.state = 3;
            ++done;
            active.erase(active.begin() + pick);
        }
    }
    // strip, as k_strip_status does
    Result res;
    std::vector<int64_t> row_ptr(R + 1, 0);
    bool any = false;
    for (int64_t i = 1; i <= R; ++i) {
        any |= lb::is_poisoned(status[i]);
        row_ptr[i] = lb::stripped(status[i]);
    }
    if (any) row_ptr[R] = -1;
    for (int64_t r = 0; r < R; ++r) {
        const Row& w = rows[r];
        if (w.poisoned) {
            ++res.poisoned;
            if (row_ptr[r + 1] != -1) res.ok = false;
        } else {
            if (w.prefix != truth[r]) res.ok = false;            // exact offset
            if (r + 1 < R && row_ptr[r + 1] != truth[r + 1]) res.ok = false;
        }
    }
    if ((row_ptr[R] < 0) != (res.poisoned > 0)) res.ok = false;
    if (res.poisoned == 0 && row_ptr[R] != truth[R]) res.ok = false;
    return res;
}

int main() {
    bool ok = true;
    int64_t poisoned_runs = 0, runs = 0;
    for (unsigned seed = 0; seed < 200; ++seed) {
        const int64_t R = 1 + (int64_t)(seed * 37 % 700);
        const Result big = simulate(R, 1u << 20, seed);
        if (!big.ok || big.poisoned) {
            std::printf("FAIL large limit: seed %u R %lld poisoned %lld\n", seed, (long long)R,
                        (long long)big.poisoned);
            ok = false;
        }
        const Result zero = simulate(R, 0, seed + 1000);
        if (!zero.ok) {
            std::printf("FAIL limit 0: seed %u R %lld\n", seed, (long long)R);
            ok = false;
        }
        poisoned_runs += zero.poisoned > 0;
        ++runs;
    }
    std::printf("large limit: %lld runs clean; limit 0: %lld of %lld runs poisoned\n", (long long)runs,
                (long long)poisoned_runs, (long long)runs);
    if (poisoned_runs == 0) {
        std::printf("FAIL: limit 0 never gave up\n");
        ok = false;
    }
    std::printf(ok ? "OK\n" : "FAILED\n");
    return ok ? 0 : 1;
}
