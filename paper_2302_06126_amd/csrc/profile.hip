// Optional per-kernel timing (include/tag_profile.h): HIP event pairs
// recorded on the launch stream around every launch of one kernel stage.
#include <vector>

#include "../../include/tag_profile.h"
#include "tag_internal.hpp"

namespace tag {
namespace {
struct ProfState {
    int stage = -1;
    int cap = 0;
    int n = 0;
    bool open = false;
    std::vector<hipEvent_t> b, e;
};
ProfState g_prof;

void release() {
    for (hipEvent_t ev : g_prof.b) (void)hipEventDestroy(ev);
    for (hipEvent_t ev : g_prof.e) (void)hipEventDestroy(ev);
    g_prof = ProfState();
}
}  // namespace

void prof_begin(int stage, hipStream_t s) {
    if (stage != g_prof.stage || g_prof.n >= g_prof.cap || g_prof.open) return;
    if (hipEventRecord(g_prof.b[g_prof.n], s) == hipSuccess) g_prof.open = true;
}

void prof_end(int stage, hipStream_t s) {
    if (stage != g_prof.stage || !g_prof.open) return;
    if (hipEventRecord(g_prof.e[g_prof.n], s) == hipSuccess) g_prof.n++;
    g_prof.open = false;
}
}  // namespace tag

using namespace tag;

extern "C" tag_status tag_profile_begin(int32_t stage, int32_t capacity) {
    clear_error();
    if (stage < 0 || stage >= TAG_STAGE_COUNT) TAG_FAIL(TAG_EINVAL, "unknown stage");
    if (capacity < 1 || capacity > (1 << 20)) TAG_FAIL(TAG_EINVAL, "capacity must be in [1, 2^20]");
    release();
    g_prof.b.resize(capacity);
    g_prof.e.resize(capacity);
    for (int i = 0; i < capacity; ++i) {
        if (hipEventCreate(&g_prof.b[i]) != hipSuccess || hipEventCreate(&g_prof.e[i]) != hipSuccess) {
            g_prof.b.resize(i);
            g_prof.e.resize(i);
            release();
            TAG_FAIL(TAG_EHIP, "hipEventCreate failed");
        }
    }
    g_prof.cap = capacity;
    g_prof.stage = stage;
    return TAG_OK;
}

extern "C" tag_status tag_profile_end(double *total_ms, int32_t *n_launches) {
    clear_error();
    if (!total_ms || !n_launches) TAG_FAIL(TAG_EINVAL, "outputs must be non-NULL");
    double tot = 0.0;
    const int n = g_prof.n;
    for (int i = 0; i < n; ++i) {
        float ms = 0.f;
        if (hipEventSynchronize(g_prof.e[i]) != hipSuccess ||
            hipEventElapsedTime(&ms, g_prof.b[i], g_prof.e[i]) != hipSuccess) {
            release();
            TAG_FAIL(TAG_EHIP, "reading profile events failed");
        }
        tot += ms;
    }
    *total_ms = tot;
    *n_launches = n;
    release();
    return TAG_OK;
}
