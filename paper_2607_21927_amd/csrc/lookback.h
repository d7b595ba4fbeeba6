// Status words of the one-pass geometry build's decoupled look-back.
//
// Row r of the build publishes its status in row_ptr[r + 1] while the build
// runs; the flags are stripped afterwards.  A status is
//   0                     nothing known yet,
//   kAgg | count          the row's own size is known,
//   kInc | prefix         the inclusive prefix (offset of the next row) is known,
//   kInc | kPoison        the row gave up waiting for its predecessors, or its
//                         look-back met a poisoned prefix: its offset is
//                         unknown and it wrote no keys.
// A row looks back over up to 64 predecessors at a time (nearest first) and
// stops at the nearest one whose inclusive prefix is known, once every row
// between is at least aggregate-ready.  Poison is carried by inclusive words
// only, so a row whose look-back reaches a poisoned prefix is poisoned in turn;
// a row that passed a predecessor while that one was only aggregate-ready
// still finds its offset correctly (aggregate counts are always exact).  After
// the build, any poisoned row makes the total row_ptr[R] negative: the CSR is
// then incomplete and must not be used.
//
// Pure bit rules, shared by the kernel and by a host-compiled simulation.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define RIS_HD __host__ __device__
#else
#define RIS_HD
#endif

namespace ris {
namespace lookback {

constexpr int64_t kPoison = 1ll << 60;
constexpr int64_t kAgg = 1ll << 61;
constexpr int64_t kInc = 1ll << 62;
constexpr int64_t kValue = kPoison - 1;   // sizes and offsets stay below 2^60

// Status with the row's own size known.
RIS_HD inline int64_t aggregate(int64_t count) { return kAgg | count; }

// Final status of a row: its inclusive prefix, or poison.
RIS_HD inline int64_t inclusive(int64_t prefix_plus_count, bool poisoned) {
    return poisoned ? (kInc | kPoison) : (kInc | prefix_plus_count);
}

RIS_HD inline bool is_inclusive(int64_t s) { return (s & kInc) != 0; }
RIS_HD inline bool is_ready(int64_t s) { return (s & (kInc | kAgg)) != 0; }
RIS_HD inline bool is_poisoned(int64_t s) { return (s & kPoison) != 0; }
RIS_HD inline int64_t value(int64_t s) { return s & kValue; }

// One look-back step over a window of predecessor statuses, given as two
// masks over the window's slots (slot i = the i-th nearest predecessor;
// slots past the first row hold an inclusive 0): `inc` marks inclusive
// statuses, `ready` those at least aggregate-ready.  Returns the slot of the
// nearest inclusive status (64 if none) when every slot up to it is ready,
// and -1 when the step must wait.
RIS_HD inline int step_end(uint64_t inc, uint64_t ready) {
    const int first = inc ? __builtin_ctzll(inc) : 64;
    const uint64_t need = first >= 63 ? ~0ull : ((1ull << (first + 1)) - 1ull);
    return (ready & need) == need ? first : -1;
}

// The flags stripped: the row's end offset, or -1 for a poisoned row.
RIS_HD inline int64_t stripped(int64_t s) { return is_poisoned(s) ? -1 : value(s); }

}  // namespace lookback
}  // namespace ris
