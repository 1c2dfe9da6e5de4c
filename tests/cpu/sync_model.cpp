// CPU model of the step kernel's cross-workgroup protocols, run under
// ThreadSanitizer: one host thread per workgroup, std::atomic in place of the
// device-coherent atomics, and the protocol arithmetic of the library itself
// (kl_sync.h, compiled here for the host).
//
// The device code orders its data before a signal by completing its stores
// (s_waitcnt vmcnt(0)) before the relaxed arrival atomic is issued, and a
// waiter issues its data loads only after its poll has seen the count; in the
// C++ memory model that is a release on the arrival and an acquire on the
// poll, which is what the model uses.  Tagged words need no ordering at all:
// value and tag travel in one atomic 8-byte access (relaxed here).
//
// Checks, each over several launches in a row (counters never reset):
//   1. grid barrier: no thread passes barrier k before every thread has
//      written its slot for k; launches recover their epoch from their own
//      group's counter (uneven group sizes: 20 threads on 16 counters);
//   2. watchdog: a launch in which one thread never arrives ends in every
//      thread with the error flag set, instead of hanging;
//   3. tagged hand-offs: readers accept exactly the current layer's values,
//      never an earlier layer's or step's, across the tag wrap;
//   4. a missing tagged writer trips the watchdog too.
// Prints "sync model OK" and exits 0, else prints the failure and exits 1.
// With --plant-early-barrier it runs check 1 with a planted off-by-one barrier
// target, which the check (or ThreadSanitizer) must report.
#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <string>
#include <thread>
#include <vector>

#include "kl_sync.h"

using namespace kl;

namespace {

// polls before a wait gives up (the device allows 2^22 polls of about a
// microsecond each; here every poll past the first 64 yields the CPU)
constexpr int kSpin = 1 << 18;

int g_fail = 0;
int g_plant = 0;   // 1: a planted mistake (barrier k waits for barrier k - 1's target)
void check(bool ok, const char *what) {
    if (!ok) {
        std::fprintf(stderr, "FAIL: %s\n", what);
        g_fail = 1;
    }
}

struct Grid {
    int nwg, ng;
    std::vector<std::atomic<unsigned long long>> cnt;   // one per group
    std::atomic<int> err{0};
    explicit Grid(int n) : nwg(n), ng(bar_group_count(n)), cnt(bar_group_count(n)) {
        for (auto &c : cnt) c.store(0);
    }
};

// One workgroup's view of a launch: bases recovered from its own group.
struct Launch {
    Grid &G;
    int w;
    std::vector<unsigned long long> base;
    Launch(Grid &g, int w_) : G(g), w(w_), base(g.ng) {
        const int own = w % G.ng;
        const unsigned long long c = G.cnt[own].load(std::memory_order_acquire);
        for (int g = 0; g < G.ng; ++g) base[g] = bar_launch_base(c, G.nwg, G.ng, own, g);
    }
    void arrive() { G.cnt[w % G.ng].fetch_add(1, std::memory_order_release); }
    // false when the wait gave up (the error flag is then set)
    bool wait(int k) {
        for (int spins = 1;; ++spins) {
            bool done = true;
            for (int g = 0; g < G.ng; ++g)
                done = done && bar_reached(G.cnt[g].load(std::memory_order_acquire),
                                           bar_target(base[g], k - g_plant, G.nwg, G.ng, g));
            if (done) return true;
            if ((spins & 63) == 0 && G.err.load(std::memory_order_relaxed)) return false;
            if (spins >= kSpin) {
                G.err.store(1, std::memory_order_relaxed);
                return false;
            }
            if (spins > 64) std::this_thread::yield();
        }
    }
};

template <class F>
void run_threads(int n, F &&f) {
    std::vector<std::thread> t;
    for (int w = 0; w < n; ++w) t.emplace_back(f, w);
    for (auto &x : t) x.join();
}

// 1. barriers over several launches; plain (non-atomic) data, ordered by the
// barrier alone: TSan reports a race if the protocol lets a reader through early
void test_barrier(int nwg, int launches, int nbar) {
    Grid G(nwg);
    std::vector<int> slot(nwg * nbar, -1);
    for (int L = 0; L < launches; ++L) {
        run_threads(nwg, [&](int w) {
            Launch me(G, w);
            for (int k = 0; k < nbar; ++k) {
                slot[k * nwg + w] = L * 1000 + k;
                me.arrive();
                if (!me.wait(k)) return;
                for (int v = 0; v < nwg; ++v)
                    if (slot[k * nwg + v] != L * 1000 + k) G.err.store(2);
            }
        });
        check(G.err.load() == 0, "barrier: a thread passed before every slot was written");
    }
    for (int g = 0; g < G.ng; ++g)
        check(G.cnt[g].load() ==
                  (unsigned long long)launches * nbar * bar_group_size(nwg, G.ng, g),
              "barrier: counters end at launches x barriers x group size");
}

// 2. a missing arrival ends the launch through the watchdog
void test_watchdog(int nwg) {
    Grid G(nwg);
    run_threads(nwg, [&](int w) {   // a clean launch first (2 barriers)
        Launch me(G, w);
        for (int k = 0; k < 2; ++k) {
            me.arrive();
            me.wait(k);
        }
    });
    check(G.err.load() == 0, "watchdog: clean launch");
    std::atomic<int> returned{0};
    run_threads(nwg, [&](int w) {
        Launch me(G, w);
        me.arrive();
        me.wait(0);
        if (w != 3) me.arrive();   // workgroup 3 never arrives on barrier 1
        me.wait(1);
        returned.fetch_add(1);
    });
    check(G.err.load() == 1, "watchdog: a missing arrival sets the error flag");
    check(returned.load() == nwg, "watchdog: every thread returned");
}

// 3. tagged hand-offs: per step and layer, writers publish words, readers
// (after the barrier that separates uses of the buffer, as in the kernel) poll
// until current and check the value
void test_tagged(int nwg, int steps, int layers, unsigned first_epoch) {
    Grid G(nwg);
    const int nwords = 3 * nwg;
    std::vector<std::atomic<unsigned long long>> buf(nwords);
    for (auto &x : buf) x.store(0);   // cleared memory: tag 0, never current
    unsigned epoch = first_epoch;
    for (int s = 0; s < steps; ++s) {
        const unsigned e = epoch;
        check(e != 0 && e + (unsigned)layers - 1u >= e, "tags: a step's range holds no 0, no wrap");
        run_threads(nwg, [&](int w) {
            Launch me(G, w);
            for (int l = 0; l < layers; ++l) {
                const unsigned tag = e + (unsigned)l;
                for (int i = w; i < nwords; i += nwg)   // write my words of layer l
                    buf[i].store(ll_word((unsigned)(s * 7919 + l * 131 + i), tag),
                                 std::memory_order_relaxed);
                // read every word of layer l (written by others)
                for (int i = 0; i < nwords; ++i) {
                    unsigned long long v = 0;
                    for (int spins = 1;; ++spins) {
                        v = buf[i].load(std::memory_order_relaxed);
                        if (ll_current(v, tag)) break;
                        if (spins >= kSpin || G.err.load(std::memory_order_relaxed)) {
                            G.err.store(1);
                            return;
                        }
                        if (spins > 64) std::this_thread::yield();
                    }
                    if (ll_value(v) != (unsigned)(s * 7919 + l * 131 + i)) G.err.store(3);
                }
                // the kernel separates a buffer's reuse by a grid barrier
                me.arrive();
                if (!me.wait(l)) return;
            }
        });
        check(G.err.load() == 0, "tags: every value read is the current layer's");
        const unsigned next = ll_next_epoch(e, layers);
        check(next == 1u || next == e + (unsigned)layers, "tags: the next range follows or restarts");
        check(next + (unsigned)layers - 1u >= next, "tags: the next range does not wrap");
        epoch = next;
    }
}

// 4. a word that is never written trips the watchdog
void test_tagged_missing_writer() {
    std::atomic<unsigned long long> word{ll_word(5, 41)};   // last step's tag
    std::atomic<int> err{0};
    std::thread t([&] {
        for (int spins = 1;; ++spins) {
            if (ll_current(word.load(std::memory_order_relaxed), 42)) return;
            if (spins >= kSpin) {
                err.store(1);
                return;
            }
        }
    });
    t.join();
    check(err.load() == 1, "tags: a stale word is never taken as current");
}

}  // namespace

int main(int argc, char **argv) {
    if (argc > 1 && std::string(argv[1]) == "--plant-early-barrier") {
        // the model must catch a barrier that lets threads through one early
        g_plant = 1;
        test_barrier(20, 2, 5);
        return g_fail ? 1 : 0;
    }
    // group sizes: 20 threads on 16 counters (sizes 2 and 1); 5 on 5
    test_barrier(20, 4, 5);
    test_barrier(5, 3, 7);
    test_watchdog(20);
    test_tagged(12, 4, 3, 1u);
    // near the top of the tag space: the range restarts at 1 instead of wrapping
    test_tagged(12, 4, 3, 0xFFFFFFFFu - 8u);
    test_tagged_missing_writer();
    // the epoch arithmetic on its own
    check(ll_next_epoch(0, 32) == 1, "epoch: 0 restarts at 1");
    check(ll_next_epoch(1, 32) == 33, "epoch: consecutive ranges");
    check(ll_next_epoch(0xFFFFFFFFu - 63u, 32) == 1, "epoch: restart before the top");
    check(bar_launch_base(7, 20, 16, 3, 0) == 6 && bar_launch_base(7, 20, 16, 3, 5) == 3,
          "barrier: base from the own group's count (sizes 2 and 1)");
    if (g_fail) return 1;
    std::printf("sync model OK\n");
    return 0;
}
