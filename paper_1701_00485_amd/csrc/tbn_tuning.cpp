// tbn_tuning.cpp -- the test and tuning knobs of tbn_tuning.h: process-wide atomics,
// unset (-1) at load.  Kernel selection reads them through tbn::knob().
#include <atomic>

#include "tbn_tuning.h"
#include "tbn_kernels.h"

namespace {
std::atomic<int32_t> g_knobs[TBN_KNOB_COUNT] = {{-1}, {-1}, {-1}, {-1}, {-1}, {-1}, {-1}, {-1}};
}  // namespace

namespace tbn {
int knob(int which) {
    if (which < 0 || which >= TBN_KNOB_COUNT) return -1;
    return g_knobs[which].load(std::memory_order_relaxed);
}
}  // namespace tbn

extern "C" tbn_status tbn_tuning_set(tbn_knob k, int32_t value) {
    if ((int)k < 0 || (int)k >= TBN_KNOB_COUNT) return TBN_ERR_SHAPE;
    g_knobs[k].store(value, std::memory_order_relaxed);
    return TBN_OK;
}

extern "C" int32_t tbn_tuning_get(tbn_knob k) { return tbn::knob((int)k); }
