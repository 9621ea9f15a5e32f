// Host-side expert-cache slot table (one set per covered layer; LRU, FIFO or static).
#pragma once

#include <cstdint>
#include <vector>

namespace moe {

struct Cache {
    int layers = 0, n = 0, ways = 0, top_k = 0;
    int policy = 0;                     // MOE_POLICY_*
    std::vector<int32_t> initial;       // [layers][ways] static content (MOE_POLICY_STATIC)
    std::vector<int32_t> slot_expert;   // [layers][ways], -1 empty
    std::vector<uint64_t> slot_used;    // [layers][ways], recency tick of the slot
    std::vector<uint64_t> tick;         // [layers]
    std::vector<int32_t> where;         // [layers][n], expert -> slot or -1

    bool valid_selection(const int32_t *experts, int k) const;
    void reset();
    // Step 1: slot and hit flag of each selected expert (state unchanged).
    void check(int layer, const int32_t *experts, int k, int32_t *slot_out, uint8_t *hit_out) const;
    // Policy update for one token; outputs aligned with `experts` (nullable).
    // allow (nullable, aligned with `experts`): 0 for a miss that must not be inserted.
    void step(int layer, const int32_t *experts, int k, int32_t *fill_out, int32_t *evicted_out,
              const uint8_t *allow = nullptr);
};

}  // namespace moe
