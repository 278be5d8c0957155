// Host-only parts of the library: the per-layer cache plan and the expert packing.
// No HIP calls here, so this file also builds into a CPU-only library for tests.
#include <algorithm>
#include <cstring>
#include <vector>

#include "common.h"

namespace {

struct Cand {
    int expert;
    int count;      // tokens whose prefetched set holds the expert
    int best;       // smallest position the expert takes in those sets
};

}  // namespace

extern "C" size_t apex_expert_bytes(int d, int I) {
    if (d <= 0 || I <= 0) return 0;
    return size_t(6) * size_t(d) * size_t(I);
}

extern "C" apex_status apex_pack_expert(const uint16_t *w1, const uint16_t *w3,
                                        const uint16_t *w2, int d, int I, uint16_t *out) {
    APEX_REQUIRE(w1 && w3 && w2 && out, "apex_pack_expert: NULL pointer");
    APEX_REQUIRE(d > 0 && I > 0, "apex_pack_expert: d=%d I=%d must be positive", d, I);
    const size_t D = size_t(d), N = size_t(I);
    for (size_t i = 0; i < N; ++i) {
        std::memcpy(out + i * 2 * D, w1 + i * D, D * sizeof(uint16_t));
        std::memcpy(out + i * 2 * D + D, w3 + i * D, D * sizeof(uint16_t));
    }
    std::memcpy(out + 2 * N * D, w2, N * D * sizeof(uint16_t));
    return APEX_OK;
}

extern "C" apex_status apex_plan_residency(int E, int C, const int32_t *pf_idx,
                                           const int32_t *pf_count, int B, int k_max,
                                           int64_t step, int32_t *expert_of_slot,
                                           int64_t *last_used, int32_t *copy_expert,
                                           int32_t *copy_slot, int *n_copies) {
    APEX_REQUIRE(E >= 1 && E <= APEX_MAX_EXPERTS, "apex_plan_residency: E=%d out of [1,64]", E);
    APEX_REQUIRE(C >= 1, "apex_plan_residency: C=%d must be >= 1", C);
    APEX_REQUIRE(B >= 0 && k_max >= 1, "apex_plan_residency: B=%d k_max=%d", B, k_max);
    APEX_REQUIRE(expert_of_slot && last_used && copy_expert && copy_slot && n_copies,
                 "apex_plan_residency: NULL table pointer");
    APEX_REQUIRE(B == 0 || (pf_idx && pf_count), "apex_plan_residency: NULL route pointer");

    // validate inputs before touching any output
    int slot_of[APEX_MAX_EXPERTS];
    std::fill(slot_of, slot_of + E, -1);
    for (int s = 0; s < C; ++s) {
        const int e = expert_of_slot[s];
        APEX_REQUIRE(e >= -1 && e < E, "apex_plan_residency: expert_of_slot[%d]=%d", s, e);
        if (e >= 0) {
            APEX_REQUIRE(slot_of[e] < 0, "apex_plan_residency: expert %d in two slots", e);
            slot_of[e] = s;
        }
    }
    int count[APEX_MAX_EXPERTS] = {0};
    int best[APEX_MAX_EXPERTS];
    std::fill(best, best + E, 1 << 30);
    for (int b = 0; b < B; ++b) {
        const int m = pf_count[b];
        APEX_REQUIRE(m >= 0 && m <= k_max, "apex_plan_residency: pf_count[%d]=%d", b, m);
        for (int j = 0; j < m; ++j) {
            const int e = pf_idx[size_t(b) * k_max + j];
            APEX_REQUIRE(e >= 0 && e < E, "apex_plan_residency: pf_idx[%d,%d]=%d", b, j, e);
            count[e] += 1;
            best[e] = std::min(best[e], j);
        }
    }

    // target set T: the first C candidates by (count desc, best rank asc, id asc)
    std::vector<Cand> cand;
    for (int e = 0; e < E; ++e)
        if (count[e] > 0) cand.push_back({e, count[e], best[e]});
    std::sort(cand.begin(), cand.end(), [](const Cand &a, const Cand &b) {
        if (a.count != b.count) return a.count > b.count;
        if (a.best != b.best) return a.best < b.best;
        return a.expert < b.expert;
    });
    if (int(cand.size()) > C) cand.resize(C);
    bool in_target[APEX_MAX_EXPERTS] = {false};
    for (const Cand &c : cand) in_target[c.expert] = true;

    // free slots: empty ones ascending, then residents outside T by (last use, id)
    std::vector<int> free_slots;
    for (int s = 0; s < C; ++s)
        if (expert_of_slot[s] < 0) free_slots.push_back(s);
    std::vector<int> evictable;
    for (int s = 0; s < C; ++s) {
        const int e = expert_of_slot[s];
        if (e >= 0 && !in_target[e]) evictable.push_back(e);
    }
    std::sort(evictable.begin(), evictable.end(), [&](int a, int b) {
        if (last_used[a] != last_used[b]) return last_used[a] < last_used[b];
        return a < b;
    });
    for (int e : evictable) free_slots.push_back(slot_of[e]);

    int n = 0;
    for (const Cand &c : cand) {
        if (slot_of[c.expert] >= 0) continue;   // already resident
        const int s = free_slots[n];            // |free| >= |T \ R| always holds
        expert_of_slot[s] = c.expert;
        copy_expert[n] = c.expert;
        copy_slot[n] = s;
        ++n;
    }
    for (const Cand &c : cand) last_used[c.expert] = step;
    *n_copies = n;
    return APEX_OK;
}
