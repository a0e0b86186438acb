// profile.cpp -- thread-local per-kernel timing (see profile.h) and its C ABI.
#include "profile.h"

#include <string.h>

#include <vector>

#include "../../include/sbp.h"

namespace sbpi {

namespace {
struct Profile {
    bool active = false;
    int count = 0;
    std::vector<ProfileSlot> slots;
};
thread_local Profile g_prof;
}  // namespace

ProfileSlot *profile_next() {
    Profile &p = g_prof;
    if (!p.active || p.count >= (int)p.slots.size()) return nullptr;
    return &p.slots[p.count++];
}

}  // namespace sbpi

extern "C" {

int sbp_profile_begin(int capacity) {
    if (capacity < 0) return SBP_ERR_SHAPE;
    sbpi::Profile &p = sbpi::g_prof;
    // grow the event pool if needed (events are reused across profiles)
    while ((int)p.slots.size() < capacity) {
        sbpi::ProfileSlot s;
        memset(&s, 0, sizeof(s));
        hipError_t e = hipEventCreate(&s.start);
        if (e == hipSuccess) e = hipEventCreate(&s.stop);
        if (e != hipSuccess) return SBP_ERR_HIP;
        p.slots.push_back(s);
    }
    p.count = 0;
    p.active = true;
    return SBP_OK;
}

int sbp_profile_end(float *us, char *names, int name_len) {
    sbpi::Profile &p = sbpi::g_prof;
    p.active = false;
    for (int i = 0; i < p.count; ++i) {
        hipError_t e = hipEventSynchronize(p.slots[i].stop);
        float ms = 0.f;
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.slots[i].start, p.slots[i].stop);
        if (e != hipSuccess) return SBP_ERR_HIP;
        if (us) us[i] = ms * 1000.f;
        if (names && name_len > 0) {
            strncpy(names + (size_t)i * name_len, p.slots[i].name, name_len - 1);
            names[(size_t)i * name_len + name_len - 1] = 0;
        }
    }
    return p.count;
}

}  // extern "C"
