// Arithmetic of the step kernel's cross-workgroup protocols, shared by the
// device code and by the CPU model of the protocols in the tests (compiled
// there with KL_HD defined empty).  Nothing here touches memory.
//
// Grid barrier.  nwg workgroups arrive on ng = min(kBarGroups, nwg) monotonic
// 64-bit counters, workgroup w on counter w % ng, which therefore counts
// group_size(g) arrivals per barrier.  The counters are never reset: after E
// complete barriers counter g holds E * group_size(g).  At launch start a
// workgroup reads its own group's counter c and recovers E = c / size (its
// own group cannot have completed barrier E before it arrives, so c is below
// (E + 1) size); barrier k of the launch is then complete when every counter
// g has reached (E + k + 1) group_size(g).
//
// Tagged hand-offs.  A value crossing workgroups travels in one 8-byte word
// with the tag of the step and layer that wrote it (value in the low 32
// bits, tag in the high 32 bits); a reader accepts a word whose tag is the
// current one.  Step s uses tags epoch_s .. epoch_s + L - 1 for its L layers;
// the next step's range starts right after, and restarts at 1 before it
// would reach 2^32, so no step's range contains 0, the tag of cleared memory.
// (The epoch lives in device memory: read at launch start, advanced by the
// step's last phase.)
#pragma once

#include <stdint.h>

#ifndef KL_HD
#define KL_HD __host__ __device__
#endif

namespace kl {

constexpr int kSyncBarGroups = 16;   // first level of the grid barrier

KL_HD inline int bar_group_count(int nwg) { return nwg < kSyncBarGroups ? nwg : kSyncBarGroups; }

// Arrivals per barrier on counter g (workgroups w with w % ng == g).
KL_HD inline unsigned bar_group_size(int nwg, int ng, int g) {
    return (unsigned)(nwg / ng + (g < nwg % ng ? 1 : 0));
}

// The value counter g starts this launch at, from the own group's counter c
// (own group og).
KL_HD inline unsigned long long bar_launch_base(unsigned long long own_count, int nwg, int ng,
                                               int og, int g) {
    const unsigned long long epoch = own_count / bar_group_size(nwg, ng, og);
    return epoch * bar_group_size(nwg, ng, g);
}

// Counter g's value once barrier k of the launch is complete.
KL_HD inline unsigned long long bar_target(unsigned long long base, int k, int nwg, int ng,
                                          int g) {
    return base + (unsigned long long)(k + 1) * bar_group_size(nwg, ng, g);
}

// Wrap-safe "counter has reached target" for monotonic 64-bit counters.
KL_HD inline bool bar_reached(unsigned long long count, unsigned long long target) {
    return (long long)(count - target) >= 0;
}

KL_HD inline unsigned long long ll_word(unsigned value, unsigned tag) {
    return ((unsigned long long)tag << 32) | value;
}
KL_HD inline bool ll_current(unsigned long long word, unsigned tag) {
    return (unsigned)(word >> 32) == tag;
}
KL_HD inline unsigned ll_value(unsigned long long word) { return (unsigned)word; }

// The first tag of the step after one whose range started at 'prev', for a
// model of n_layers layers (0 < n_layers < 2^30).
KL_HD inline unsigned ll_next_epoch(unsigned prev, int n_layers) {
    const unsigned L = (unsigned)n_layers;
    if (prev == 0 || prev > 0xFFFFFFFFu - 2u * L) return 1u;   // restart before wrapping
    return prev + L;
}

}  // namespace kl
