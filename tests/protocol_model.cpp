// protocol_model.cpp -- a CPU model of the library's inter-workgroup
// protocols, for tests only (nothing here is linked into the library).
//
// Workgroups become std::threads and workspace words become std::atomic
// words.  The rules modelled are the ones the HIP kernels follow:
//  * tile tickets: one 64-bit header word [epoch:32 | next ticket:32],
//    fetch-and-add per workgroup; the workgroup that takes ticket nwg - 1
//    stores (epoch + 1) << 32, so the next launch starts at ticket 0;
//  * status words [state:2 | epoch:30 | value:32], state X (nothing yet),
//    A (tile aggregate) or P (inclusive prefix); a word whose epoch tag is
//    not the reader's reads as X;
//  * decoupled look-back (Section 2.1; Merrill and Garland): a tile
//    publishes A, then one 64-lane window after another reads the 64
//    nearest predecessors; a window in which an X lies at or before the
//    nearest P is read again; otherwise the values up to that P (all of the
//    window if it holds no P) are summed; the first tile of a segment
//    publishes P directly.  Every wait is bounded and raises the error flag;
//  * the epoch wrap: in the launch whose 30-bit tag is all ones, every
//    workgroup counts itself in the header's done counter after its last
//    status access, and the last one zeroes every status word;
//  * the per-row arrival count: a row's tiles store their tagged sums
//    [001 | value] and count themselves in a tagged counter by
//    compare-and-swap (an untagged word counts as zero); the row's last
//    arrival waits (bounded) until every sum is tagged, computes the row's
//    result, and clears the sums and the counter.
//
// A launch runs on `slots` worker threads that take workgroups from a
// dispatch order (a random permutation of the block indices, or block order
// with one "XCD" of eight held back), so workgroups start out of order and
// fewer of them than the grid are resident at once.  Random pauses sit where
// the kernels' adversarial build pauses.  What the model checks:
//  * every launch ends (a wait that cannot end trips the spin limit);
//  * every scan equals the serial scan (uint32, wrapping), every row result
//    the serial one;
//  * the error flag and the done counter are 0 after every launch;
//  * the workspace invariant after every launch: each word outside the header
//    is 0, or a count/sum with the top two bits clear that no row op left
//    tagged, or a status word (state A or P) of an epoch no later than the
//    current one.
// It models the protocol's logic (which word may hold what when, and who
// waits for whom), not the GPU memory model: the kernels order a store
// before the count that announces it by waiting for its acknowledgement, and
// the model by program order on atomics.
//
// Usage: protocol_model [--mutation NAME] [--seed S] [--quick] [--scenario NAME]
// Exit status 0 when every check holds; 1 with a message naming the first
// failure otherwise.  A mutation plants one protocol mistake, which some
// check must catch.

#include <atomic>
#include <chrono>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <string>
#include <thread>
#include <vector>

namespace {

// ---------------------------------------------------------------- mutations
enum class Mut {
    None,
    BlockIdxTiles,     // tile = block index instead of a ticket
    NoTicketReset,     // the last ticket does not restart the count
    IgnoreEpoch,       // stale status words read as current
    NoWrapClear,       // the wrap launch does not zero the status words
    XAsZero,           // an unpublished predecessor counts as zero
    DropPLane,         // the nearest P's value is left out of the sum
    WindowFromSelf,    // the first window starts at the tile itself
    RowPlainCount,     // the row counter counts whatever the word holds
    RowNoClearCounter, // the last arrival leaves the row counter set
    XcdTickets,        // one ticket counter per XCD: tile = 8 * ticket + xcd
    PersistentResetAtTiles,  // persistent grid: the count restarts at the last tile's ticket
};
Mut g_mut = Mut::None;

struct MutName { const char* name; Mut m; };
const MutName kMutations[] = {
    {"none", Mut::None},
    {"blockidx_tiles", Mut::BlockIdxTiles},
    {"no_ticket_reset", Mut::NoTicketReset},
    {"ignore_epoch", Mut::IgnoreEpoch},
    {"no_wrap_clear", Mut::NoWrapClear},
    {"x_as_zero", Mut::XAsZero},
    {"drop_p_lane", Mut::DropPLane},
    {"window_from_self", Mut::WindowFromSelf},
    {"row_plain_count", Mut::RowPlainCount},
    {"row_no_clear_counter", Mut::RowNoClearCounter},
    {"xcd_tickets", Mut::XcdTickets},
    {"persistent_reset_at_tiles", Mut::PersistentResetAtTiles},
};

[[noreturn]] void fail(const std::string& what) {
    std::fprintf(stderr, "FAIL: %s\n", what.c_str());
    std::fflush(stderr);
    std::exit(1);
}

// ---------------------------------------------------------------- words
constexpr int kWave = 64;
constexpr uint64_t kStateShift = 62;
constexpr uint64_t kStateMask = 3ull << kStateShift;
constexpr uint64_t kX = 0, kA = 1ull << kStateShift, kP = 2ull << kStateShift;
constexpr uint32_t kEpochMask = (1u << 30) - 1;
constexpr uint64_t kRowTag = 1ull << 61;

uint64_t status_word(uint64_t state, uint32_t epoch, uint32_t v) {
    return state | ((uint64_t)(epoch & kEpochMask) << 32) | v;
}
uint64_t status_state(uint64_t w, uint32_t epoch) {
    if (g_mut == Mut::IgnoreEpoch) return w & kStateMask;
    return ((uint32_t)(w >> 32) & kEpochMask) == (epoch & kEpochMask) ? (w & kStateMask) : kX;
}
bool row_word(uint64_t w) { return (w >> 61) == 1; }

struct Workspace {
    std::atomic<uint64_t> ticket{0};
    std::atomic<uint32_t> done{0};
    std::atomic<uint32_t> error{0};
    std::atomic<uint64_t> xcd_ticket[8];
    std::vector<std::atomic<uint64_t>> words;
    explicit Workspace(size_t n) : words(n) {
        for (auto& w : words) w.store(0, std::memory_order_relaxed);
        for (auto& t : xcd_ticket) t.store(0, std::memory_order_relaxed);
    }
    uint32_t epoch() const { return (uint32_t)(ticket.load() >> 32); }
};

// ---------------------------------------------------------------- timing
thread_local uint64_t t_rng = 1;
uint32_t rnd() {  // xorshift64*
    t_rng ^= t_rng >> 12;
    t_rng ^= t_rng << 25;
    t_rng ^= t_rng >> 27;
    return (uint32_t)((t_rng * 2685821657736338717ull) >> 32);
}
void seed_thread(uint64_t s) { t_rng = s * 0x9E3779B97F4A7C15ull + 0x632BE59BD9B4E019ull; }

int g_pause_per_mille = 200;
void pause_point() {
    const uint32_t r = rnd() % 1000;
    if (r >= (uint32_t)g_pause_per_mille) return;
    if (r % 8 == 0)
        std::this_thread::sleep_for(std::chrono::microseconds(20 + rnd() % 200));
    else
        std::this_thread::yield();
}

// A bounded wait: gives up after kSpinSeconds (a deadlock in the model), or
// at once once any wait has given up.
constexpr double kSpinSeconds = 2.0;
struct Spin {
    std::chrono::steady_clock::time_point t0 = std::chrono::steady_clock::now();
    uint32_t n = 0;
    bool give_up(Workspace& ws) {
        if (ws.error.load(std::memory_order_relaxed)) return true;
        if ((++n & 255) == 0 &&
            std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count() > kSpinSeconds) {
            ws.error.store(1);
            return true;
        }
        std::this_thread::yield();
        return false;
    }
};

// ---------------------------------------------------------------- launches
// Runs body(block) for every block of the grid on `slots` threads; `order`
// is the dispatch order.  `xcd_held`: block order, but blocks of XCD 0 (block
// % 8 == 0) wait until every other block has been dispatched -- a legal
// schedule when another kernel holds that XCD's slots.
void launch(uint32_t nwg, int slots, const std::vector<uint32_t>& order,
            const std::function<void(uint32_t)>& body, uint64_t seed) {
    std::atomic<uint32_t> next{0};
    std::vector<std::thread> th;
    for (int s = 0; s < slots; ++s)
        th.emplace_back([&, s] {
            seed_thread(seed * 1315423911u + (uint64_t)s);
            while (true) {
                const uint32_t i = next.fetch_add(1);
                if (i >= nwg) break;
                body(order[i]);
            }
        });
    for (auto& t : th) t.join();
}

std::vector<uint32_t> dispatch_order(uint32_t nwg, int kind, uint64_t seed) {
    std::vector<uint32_t> o(nwg);
    for (uint32_t i = 0; i < nwg; ++i) o[i] = i;
    if (kind == 0) {  // random permutation
        seed_thread(seed);
        for (uint32_t i = nwg; i > 1; --i) std::swap(o[i - 1], o[rnd() % i]);
    } else if (kind == 1) {  // reversed
        for (uint32_t i = 0; i < nwg; ++i) o[i] = nwg - 1 - i;
    } else {  // block order with XCD 0's blocks last
        std::vector<uint32_t> a, b;
        for (uint32_t i = 0; i < nwg; ++i) (i % 8 == 0 ? b : a).push_back(i);
        o = a;
        o.insert(o.end(), b.begin(), b.end());
    }
    return o;
}

// ---------------------------------------------------------------- tickets
struct Ticket { uint32_t tile, epoch; };

Ticket take_ticket(Workspace& ws, uint32_t nwg, uint32_t block) {
    if (g_mut == Mut::XcdTickets) {
        // tiles 8k + x go to XCD x's k-th workgroup (block % 8 plays the XCD)
        const uint32_t x = block % 8;
        const uint32_t k = (uint32_t)ws.xcd_ticket[x].fetch_add(1, std::memory_order_relaxed);
        const uint64_t old = ws.ticket.fetch_add(1, std::memory_order_relaxed);
        if ((uint32_t)old == nwg - 1) {
            ws.ticket.store((uint64_t)((uint32_t)(old >> 32) + 1) << 32, std::memory_order_relaxed);
            for (auto& t : ws.xcd_ticket) t.store(0, std::memory_order_relaxed);
        }
        pause_point();
        return {8 * k + x, (uint32_t)(old >> 32)};
    }
    const uint64_t old = ws.ticket.fetch_add(1, std::memory_order_relaxed);
    Ticket t{(uint32_t)old, (uint32_t)(old >> 32)};
    if (t.tile == nwg - 1 && g_mut != Mut::NoTicketReset)
        ws.ticket.store((uint64_t)(t.epoch + 1) << 32, std::memory_order_relaxed);
    if (g_mut == Mut::BlockIdxTiles) t.tile = block;
    pause_point();
    return t;
}

// ---------------------------------------------------------------- look-back
// The exclusive prefix of `tile` (including `base` from the segment's first
// tile), publishing A first and P at the end; tiles [first, tile) precede it.
uint32_t lookback(Workspace& ws, std::atomic<uint64_t>* status, uint32_t tile, uint32_t first,
                  uint32_t agg, uint32_t base, uint32_t epoch) {
    pause_point();
    if (tile == first) {
        status[tile].store(status_word(kP, epoch, base + agg), std::memory_order_relaxed);
        return base;
    }
    status[tile].store(status_word(kA, epoch, agg), std::memory_order_relaxed);
    uint32_t excl = 0;
    int64_t end = g_mut == Mut::WindowFromSelf ? (int64_t)tile : (int64_t)tile - 1;
    Spin spin;
    while (true) {
        uint64_t s[kWave], st[kWave];
        uint64_t pmask = 0, xmask = 0;
        for (int lane = 0; lane < kWave; ++lane) {
            const int64_t idx = end - lane;
            s[lane] = 0;
            st[lane] = kP;  // past the segment start: an empty prefix
            if (idx >= (int64_t)first) {
                s[lane] = status[idx].load(std::memory_order_relaxed);
                st[lane] = status_state(s[lane], epoch);
            }
            if (st[lane] == kP) pmask |= 1ull << lane;
            if (st[lane] == kX) xmask |= 1ull << lane;
        }
        const uint64_t upto = pmask ? (((pmask & (~pmask + 1)) << 1) - 1) : ~0ull;
        if ((xmask & upto) && g_mut != Mut::XAsZero) {
            if (spin.give_up(ws)) break;
            continue;
        }
        uint64_t take = upto;
        if (g_mut == Mut::DropPLane && pmask) take = upto >> 1;
        for (int lane = 0; lane < kWave; ++lane)
            if ((take >> lane) & 1) excl += (uint32_t)s[lane];
        end -= kWave;
        if (pmask) break;
    }
    pause_point();
    status[tile].store(status_word(kP, epoch, excl + agg), std::memory_order_relaxed);
    return excl;
}

void finish_epoch(Workspace& ws, uint32_t epoch, uint32_t nwg, std::atomic<uint64_t>* status,
                  size_t nwords) {
    if ((epoch & kEpochMask) != kEpochMask) return;
    const uint32_t d = ws.done.fetch_add(1, std::memory_order_acq_rel);
    if (d != nwg - 1) return;
    if (g_mut != Mut::NoWrapClear)
        for (size_t i = 0; i < nwords; ++i) status[i].store(0, std::memory_order_relaxed);
    ws.done.store(0, std::memory_order_release);
}

// One segmented inclusive scan launch: `segs` tiles of `tile_len` per row
// (a 1-D scan is one row), `carry` added to row 0's first tile.  Tiles are
// taken by ticket, row-major, as the row and 1-D look-back kernels do.
void scan_launch(Workspace& ws, const std::vector<uint32_t>& x, std::vector<uint32_t>& y,
                 uint32_t rows, uint32_t segs, uint32_t tile_len, uint32_t carry, int slots,
                 int order_kind, uint64_t seed) {
    const uint32_t nwg = rows * segs;
    const uint32_t len = (uint32_t)(x.size() / rows);
    std::atomic<uint64_t>* status = ws.words.data();
    const size_t nwords = ws.words.size();
    auto body = [&](uint32_t block) {
        const Ticket t = take_ticket(ws, nwg, block);
        if (t.tile >= nwg) {  // the kernels' guard for a workspace never zero-filled
            ws.error.store(1);
            return;
        }
        const uint32_t row = t.tile / segs, seg = t.tile % segs;
        const uint64_t lo = (uint64_t)row * len + (uint64_t)seg * tile_len;
        const uint64_t hi = (uint64_t)row * len + std::min<uint64_t>((uint64_t)(seg + 1) * tile_len, len);
        uint32_t agg = 0;
        for (uint64_t i = lo; i < hi; ++i) agg += x[i];
        const uint32_t base = (t.tile == 0) ? carry : 0;
        const uint32_t excl = lookback(ws, status, t.tile, row * segs, agg, base, t.epoch);
        uint32_t run = excl;
        for (uint64_t i = lo; i < hi; ++i) y[i] = (run += x[i]);
        finish_epoch(ws, t.epoch, nwg, status, nwords);
    };
    launch(nwg, slots, dispatch_order(nwg, order_kind, seed), body, seed);
}

// The same scan by a persistent grid of `grid` workgroups, each holding the
// ticket of its next tile while it finishes the current one (its next
// tile's loads in flight meanwhile): take a ticket; while it is a tile, take
// the next ticket, then scan the tile.  Every workgroup takes exactly one
// ticket past the last tile, so the count restarts at ticket ntiles + grid - 1.
void scan_launch_persistent(Workspace& ws, const std::vector<uint32_t>& x, std::vector<uint32_t>& y,
                            uint32_t ntiles, uint32_t tile_len, uint32_t carry, uint32_t grid,
                            int slots, uint64_t seed) {
    const uint32_t len = (uint32_t)x.size();
    std::atomic<uint64_t>* status = ws.words.data();
    const size_t nwords = ws.words.size();
    const uint32_t reset_at = g_mut == Mut::PersistentResetAtTiles ? ntiles : ntiles + grid;
    auto body = [&](uint32_t block) {
        Ticket cur = take_ticket(ws, reset_at, block);
        while (cur.tile < ntiles) {
            const Ticket next = take_ticket(ws, reset_at, block);
            const uint64_t lo = (uint64_t)cur.tile * tile_len;
            const uint64_t hi = std::min<uint64_t>(lo + tile_len, len);
            uint32_t agg = 0;
            for (uint64_t i = lo; i < hi; ++i) agg += x[i];
            const uint32_t base = cur.tile == 0 ? carry : 0;
            const uint32_t excl = lookback(ws, status, cur.tile, 0, agg, base, cur.epoch);
            uint32_t run = excl;
            for (uint64_t i = lo; i < hi; ++i) y[i] = (run += x[i]);
            if (next.epoch != cur.epoch) {  // a ticket of a later launch: the protocol is broken
                ws.error.store(1);
                break;
            }
            cur = next;
        }
        if (cur.tile >= reset_at && g_mut != Mut::PersistentResetAtTiles) ws.error.store(1);
        finish_epoch(ws, cur.epoch, grid, status, nwords);
    };
    launch(grid, slots, dispatch_order(grid, 0, seed), body, seed);
}

// ---------------------------------------------------------------- row arrivals
uint32_t row_arrive(std::atomic<uint64_t>* counter) {
    pause_point();
    if (g_mut == Mut::RowPlainCount) return (uint32_t)counter->fetch_add(1, std::memory_order_relaxed);
    uint64_t old = counter->load(std::memory_order_relaxed);
    while (true) {
        const uint32_t before = row_word(old) ? (uint32_t)old : 0u;
        uint64_t expected = old;
        if (counter->compare_exchange_strong(expected, kRowTag | (before + 1u),
                                             std::memory_order_relaxed, std::memory_order_relaxed))
            return before;
        old = expected;
    }
}

// rows x segs tiles (block = row * segs + seg, no ticket: nothing waits on a
// tile that has not stored yet); the row's last arrival writes out[row] =
// (row sum, first tile whose inclusive sum reaches thr[row], else segs).
void row_launch(Workspace& ws, const std::vector<uint32_t>& x, std::vector<uint64_t>& out,
                const std::vector<uint32_t>& thr, uint32_t rows, uint32_t segs, uint32_t tile_len,
                int slots, int order_kind, uint64_t seed) {
    const uint32_t nwg = rows * segs;
    const uint32_t len = (uint32_t)(x.size() / rows);
    std::atomic<uint64_t>* sums = ws.words.data();
    std::atomic<uint64_t>* arrivals = sums + nwg;
    auto body = [&](uint32_t block) {
        const uint32_t row = block / segs, seg = block % segs;
        const uint64_t lo = (uint64_t)row * len + (uint64_t)seg * tile_len;
        const uint64_t hi = (uint64_t)row * len + std::min<uint64_t>((uint64_t)(seg + 1) * tile_len, len);
        uint32_t agg = 0;
        for (uint64_t i = lo; i < hi; ++i) agg += x[i] & 0xFFFFu;  // sums below 2^31
        sums[block].store(kRowTag | agg, std::memory_order_relaxed);
        if (row_arrive(&arrivals[row]) != segs - 1) return;
        uint32_t total = 0, first = segs;
        for (uint32_t s = 0; s < segs; ++s) {
            uint64_t w;
            Spin spin;
            while (!row_word(w = sums[row * segs + s].load(std::memory_order_relaxed)))
                if (spin.give_up(ws)) break;
            total += (uint32_t)w;
            if (first == segs && total >= thr[row]) first = s;
        }
        out[row] = ((uint64_t)total << 32) | first;
        for (uint32_t s = 0; s < segs; ++s) sums[row * segs + s].store(0, std::memory_order_relaxed);
        if (g_mut != Mut::RowNoClearCounter) arrivals[row].store(0, std::memory_order_relaxed);
    };
    launch(nwg, slots, dispatch_order(nwg, order_kind, seed), body, seed);
}

// ---------------------------------------------------------------- checks
void check_after_launch(Workspace& ws, const std::string& what) {
    if (ws.error.load()) fail(what + ": error flag set (a wait gave up or a ticket was out of range)");
    if (ws.done.load()) fail(what + ": done counter left at " + std::to_string(ws.done.load()));
    const uint32_t cur = ws.epoch() & kEpochMask;
    for (size_t i = 0; i < ws.words.size(); ++i) {
        const uint64_t w = ws.words[i].load();
        const uint64_t st = w & kStateMask;
        if (st == 0) {
            if (row_word(w)) fail(what + ": a row word left tagged at " + std::to_string(i));
            continue;
        }
        if (st == kStateMask) fail(what + ": a word with state 11 at " + std::to_string(i));
        const uint32_t e = (uint32_t)(w >> 32) & kEpochMask;
        if (e > cur) fail(what + ": a status word of a later epoch at " + std::to_string(i));
    }
}

std::vector<uint32_t> make_input(size_t n, uint64_t seed) {
    seed_thread(seed);
    std::vector<uint32_t> x(n);
    for (auto& v : x) v = rnd();
    return x;
}

void check_scan(const std::vector<uint32_t>& x, const std::vector<uint32_t>& y, uint32_t rows,
                uint32_t carry, const std::string& what) {
    const size_t len = x.size() / rows;
    for (uint32_t r = 0; r < rows; ++r) {
        uint32_t run = r == 0 ? carry : 0;
        for (size_t i = 0; i < len; ++i) {
            run += x[r * len + i];
            if (y[r * len + i] != run)
                fail(what + ": scan differs at row " + std::to_string(r) + " index " + std::to_string(i));
        }
    }
}

struct Runner {
    Workspace& ws;
    uint64_t seed;
    int launches = 0;

    void scan(uint32_t rows, uint32_t segs, uint32_t tile_len, int slots, int order_kind,
              bool ragged = true) {
        seed_thread(seed * 7919 + launches);
        const uint32_t len = segs * tile_len - (ragged ? rnd() % tile_len : 0);
        const uint32_t carry = rnd();
        auto x = make_input((size_t)rows * len, seed * 104729 + launches);
        std::vector<uint32_t> y(x.size(), 0xDEADBEEFu);
        const std::string what = "scan launch " + std::to_string(launches) + " (rows " +
                                 std::to_string(rows) + ", tiles/row " + std::to_string(segs) +
                                 ", slots " + std::to_string(slots) + ", epoch " +
                                 std::to_string(ws.epoch()) + ")";
        scan_launch(ws, x, y, rows, segs, tile_len, carry, slots, order_kind, seed + launches);
        ++launches;
        check_after_launch(ws, what);
        check_scan(x, y, rows, carry, what);
    }

    void persistent(uint32_t ntiles, uint32_t tile_len, uint32_t grid, int slots) {
        seed_thread(seed * 7907 + launches);
        const uint32_t len = ntiles * tile_len - rnd() % tile_len;
        const uint32_t carry = rnd();
        auto x = make_input(len, seed * 104723 + launches);
        std::vector<uint32_t> y(x.size(), 0xDEADBEEFu);
        const std::string what = "persistent launch " + std::to_string(launches) + " (tiles " +
                                 std::to_string(ntiles) + ", grid " + std::to_string(grid) +
                                 ", slots " + std::to_string(slots) + ", epoch " +
                                 std::to_string(ws.epoch()) + ")";
        scan_launch_persistent(ws, x, y, ntiles, tile_len, carry, grid, slots, seed + launches);
        ++launches;
        check_after_launch(ws, what);
        check_scan(x, y, 1, carry, what);
    }

    void rows(uint32_t nrows, uint32_t segs, uint32_t tile_len, int slots, int order_kind) {
        const uint32_t len = segs * tile_len - rnd() % tile_len;
        auto x = make_input((size_t)nrows * len, seed * 15485863 + launches);
        std::vector<uint32_t> thr(nrows);
        std::vector<uint64_t> out(nrows, ~0ull);
        for (uint32_t r = 0; r < nrows; ++r) {
            uint64_t tot = 0;
            for (uint32_t i = 0; i < len; ++i) tot += x[(size_t)r * len + i] & 0xFFFFu;
            thr[r] = (uint32_t)(tot * (rnd() % 1100) / 1000);
        }
        const std::string what = "row launch " + std::to_string(launches) + " (rows " +
                                 std::to_string(nrows) + ", tiles/row " + std::to_string(segs) + ")";
        row_launch(ws, x, out, thr, nrows, segs, tile_len, slots, order_kind, seed + launches);
        ++launches;
        check_after_launch(ws, what);
        for (uint32_t r = 0; r < nrows; ++r) {
            uint32_t total = 0, first = segs;
            for (uint32_t s = 0; s < segs; ++s) {
                uint32_t agg = 0;
                for (uint32_t i = s * tile_len; i < std::min((s + 1) * tile_len, len); ++i)
                    agg += x[(size_t)r * len + i] & 0xFFFFu;
                total += agg;
                if (first == segs && total >= thr[r]) first = s;
            }
            if (out[r] != (((uint64_t)total << 32) | first))
                fail(what + ": row " + std::to_string(r) + (out[r] == ~0ull ? " never finished" : " wrong"));
        }
    }
};

// ---------------------------------------------------------------- scenarios
// Back-to-back scans of varying grid on one workspace, random dispatch.
void scenario_scans(uint64_t seed, bool quick) {
    Workspace ws(1 << 14);
    Runner r{ws, seed};
    const int slot_sets[] = {1, 2, 7, 16, 48};
    const int n = quick ? 12 : 40;
    for (int i = 0; i < n; ++i) {
        seed_thread(seed * 31 + i);
        const uint32_t segs = 1 + rnd() % (i % 3 == 0 ? 600 : 90);
        r.scan(1, segs, 1 + rnd() % 40, slot_sets[i % 5], i % 2);
    }
}

// Segmented (row) scans, 1-D scans and row arrivals interleaved on one
// workspace whose words start as leftovers of earlier calls.
void scenario_mixed(uint64_t seed, bool quick) {
    Workspace ws(1 << 13);
    ws.ticket.store((uint64_t)5 << 32);
    seed_thread(seed);
    for (auto& w : ws.words) {  // words earlier calls may leave: old status words, counts, zeros
        const uint32_t k = rnd() % 4;
        w.store(k == 0 ? status_word(kA, rnd() % 5, rnd())
                : k == 1 ? status_word(kP, rnd() % 5, rnd())
                : k == 2 ? (uint64_t)(rnd() & 0x3FFFFFFF) : 0);
    }
    Runner r{ws, seed};
    const int n = quick ? 10 : 30;
    for (int i = 0; i < n; ++i) {
        seed_thread(seed * 131 + i);
        switch (i % 3) {
            case 0: r.scan(1 + rnd() % 20, 1 + rnd() % 30, 1 + rnd() % 25, 1 + (int)(rnd() % 24), 0); break;
            case 1: r.rows(1 + rnd() % 40, 1 + rnd() % 40, 1 + rnd() % 30, 1 + (int)(rnd() % 24), 0); break;
            default: r.scan(1, 1 + rnd() % 400, 1 + rnd() % 16, 1 + (int)(rnd() % 32), 1); break;
        }
    }
}

// Across the 30-bit epoch wrap, the workspace full of words tagged with
// epoch 0 (written 2^30 calls before the wrap); the launches after the wrap
// use more tiles than those before it.
void scenario_wrap(uint64_t seed, bool) {
    Workspace ws(1 << 13);
    seed_thread(seed);
    for (auto& w : ws.words) w.store(status_word(kP, 0, rnd()));
    ws.ticket.store((uint64_t)(kEpochMask - 2) << 32);
    Runner r{ws, seed};
    for (int i = 0; i < 3; ++i) r.scan(1, 40 + 10 * i, 8, 12, 0);  // epochs 2^30 - 3 .. 2^30 - 1
    if (ws.epoch() != kEpochMask + 1) fail("wrap: epoch did not advance once per launch");
    for (int i = 0; i < 4; ++i) r.scan(1, 400 + 900 * i, 3, 12, 0);
}

// Dispatch that holds one XCD's blocks back (block order otherwise), few
// slots: the single ticket counter must still make progress.
void scenario_held_xcd(uint64_t seed, bool) {
    Workspace ws(1 << 13);
    Runner r{ws, seed};
    for (int i = 0; i < 4; ++i) r.scan(1, 257 + 64 * i, 5, 24, 2, false);
}

// Persistent grids (each workgroup holding its next tile's ticket) between
// ordinary launches on one workspace, across the epoch wrap; grids larger
// than the resident slots start late and still finish.
void scenario_persistent(uint64_t seed, bool quick) {
    Workspace ws(1 << 13);
    ws.ticket.store((uint64_t)(kEpochMask - 4) << 32);
    Runner r{ws, seed};
    const int n = quick ? 6 : 14;
    for (int i = 0; i < n; ++i) {
        seed_thread(seed * 733 + i);
        const uint32_t grid = 1 + rnd() % 40;
        r.persistent(1 + rnd() % 700, 1 + rnd() % 12, grid, 1 + (int)(rnd() % 40));
        if (i % 3 == 2) r.scan(1, 1 + rnd() % 200, 1 + rnd() % 9, 8, 0);
    }
}

struct Scenario { const char* name; void (*run)(uint64_t, bool); };
const Scenario kScenarios[] = {
    {"scans", scenario_scans},
    {"mixed", scenario_mixed},
    {"wrap", scenario_wrap},
    {"held_xcd", scenario_held_xcd},
    {"persistent", scenario_persistent},
};

}  // namespace

int main(int argc, char** argv) {
    uint64_t seed = 1;
    bool quick = false;
    std::string only;
    for (int i = 1; i < argc; ++i) {
        const std::string a = argv[i];
        if (a == "--mutation" && i + 1 < argc) {
            const std::string m = argv[++i];
            bool found = false;
            for (const auto& mn : kMutations)
                if (m == mn.name) g_mut = mn.m, found = true;
            if (!found) { std::fprintf(stderr, "unknown mutation %s\n", m.c_str()); return 2; }
        } else if (a == "--seed" && i + 1 < argc) {
            seed = std::strtoull(argv[++i], nullptr, 10);
        } else if (a == "--quick") {
            quick = true;
        } else if (a == "--scenario" && i + 1 < argc) {
            only = argv[++i];
        } else if (a == "--list-mutations") {
            for (const auto& mn : kMutations) std::printf("%s\n", mn.name);
            return 0;
        } else {
            std::fprintf(stderr, "usage: %s [--mutation NAME] [--seed S] [--quick] [--scenario NAME]\n", argv[0]);
            return 2;
        }
    }
    for (const auto& s : kScenarios) {
        if (!only.empty() && only != s.name) continue;
        s.run(seed, quick);
        std::printf("ok %s\n", s.name);
        std::fflush(stdout);
    }
    std::printf("MODEL_OK\n");
    return 0;
}
