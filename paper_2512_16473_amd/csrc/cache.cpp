// Host-side slot table of the N-index, M-way expert cache (Section III-B):
// one set per covered layer, LRU replacement with every missed expert inserted so that
// later tokens hit it (Section III-A step 3). Section IV-D's comparison policies are also
// here: FIFO (a hit does not refresh its slot) and static (a fixed content, misses
// never inserted).
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <vector>

#include "cache.h"
#include "common.h"

namespace moe {

bool Cache::valid_selection(const int32_t *experts, int k) const
{
    if (k < 1 || k > top_k) return false;
    for (int a = 0; a < k; ++a) {
        if (experts[a] < 0 || experts[a] >= n) return false;
        for (int b = 0; b < a; ++b)
            if (experts[a] == experts[b]) return false;
    }
    return true;
}

void Cache::reset()
{
    std::fill(slot_expert.begin(), slot_expert.end(), -1);
    std::fill(slot_used.begin(), slot_used.end(), 0);
    std::fill(tick.begin(), tick.end(), 0);
    std::fill(where.begin(), where.end(), -1);
    if (policy == MOE_POLICY_STATIC) {
        slot_expert = initial;
        for (int l = 0; l < layers; ++l)
            for (int s = 0; s < ways; ++s) where[(size_t)l * n + initial[(size_t)l * ways + s]] = s;
    }
}

void Cache::check(int layer, const int32_t *experts, int k, int32_t *slot_out, uint8_t *hit_out) const
{
    const int32_t *map = &where[(size_t)layer * n];
    for (int j = 0; j < k; ++j) {
        const int32_t s = map[experts[j]];
        if (slot_out) slot_out[j] = s;
        if (hit_out) hit_out[j] = s >= 0 ? 1 : 0;
    }
}

void Cache::step(int layer, const int32_t *experts, int k, int32_t *fill_out, int32_t *evicted_out,
                 const uint8_t *allow)
{
    int32_t *sx = &slot_expert[(size_t)layer * ways];
    uint64_t *su = &slot_used[(size_t)layer * ways];
    int32_t *map = &where[(size_t)layer * n];
    uint64_t &clk = tick[layer];

    // Hit status of every selected expert is fixed before any change.
    bool hit[MOE_MAX_TOPK];
    for (int j = 0; j < k; ++j) hit[j] = map[experts[j]] >= 0;
    if (policy == MOE_POLICY_STATIC) {   // fixed content: nothing is stamped or inserted
        for (int j = 0; j < k; ++j) {
            if (fill_out) fill_out[j] = -1;
            if (evicted_out) evicted_out[j] = -1;
        }
        return;
    }

    // Visit the selection in ascending expert id.
    int order[MOE_MAX_TOPK];
    for (int j = 0; j < k; ++j) order[j] = j;
    std::sort(order, order + k, [&](int a, int b) { return experts[a] < experts[b]; });

    for (int q = 0; q < k; ++q) {
        const int j = order[q];
        const int32_t e = experts[j];
        ++clk;
        if (hit[j]) {
            if (policy == MOE_POLICY_LRU) su[map[e]] = clk;   // FIFO keeps the insertion stamp
            if (fill_out) fill_out[j] = -1;
            if (evicted_out) evicted_out[j] = -1;
            continue;
        }
        if (allow && !allow[j]) {   // post-fetch not issued: the miss takes no slot
            if (fill_out) fill_out[j] = -1;
            if (evicted_out) evicted_out[j] = -1;
            continue;
        }
        int victim = -1;
        for (int s = 0; s < ways; ++s)
            if (sx[s] < 0) { victim = s; break; }
        if (victim < 0) {
            uint64_t oldest = ~(uint64_t)0;
            for (int s = 0; s < ways; ++s) {
                bool current = false;
                for (int c = 0; c < k; ++c)
                    if (experts[c] == sx[s]) { current = true; break; }
                if (!current && su[s] < oldest) { oldest = su[s]; victim = s; }
            }
        }
        const int32_t old = sx[victim];
        if (old >= 0) map[old] = -1;
        sx[victim] = e;
        su[victim] = clk;
        map[e] = victim;
        if (fill_out) fill_out[j] = victim;
        if (evicted_out) evicted_out[j] = old;
    }
}

}  // namespace moe

using moe::Cache;

extern "C" {

int moe_cache_create_policy(int n_layers, int n_experts, int ways, int top_k, int policy,
                            const int32_t *static_content, moe_cache **out)
{
    MOE_GUARD_BEGIN
    MOE_REQUIRE(out, "moe_cache_create: null output handle");
    MOE_REQUIRE(n_layers >= 0, "moe_cache_create: n_layers=%d < 0", n_layers);
    MOE_REQUIRE(n_experts >= 1 && n_experts <= MOE_MAX_EXPERTS, "moe_cache_create: n_experts=%d out of [1,%d]",
                n_experts, MOE_MAX_EXPERTS);
    MOE_REQUIRE(top_k >= 1 && top_k <= MOE_MAX_TOPK, "moe_cache_create: top_k=%d out of [1,%d]", top_k,
                MOE_MAX_TOPK);
    MOE_REQUIRE(policy == MOE_POLICY_LRU || policy == MOE_POLICY_FIFO || policy == MOE_POLICY_STATIC,
                "moe_cache_create: unknown policy %d", policy);
    if (policy == MOE_POLICY_STATIC) {
        MOE_REQUIRE(ways >= 1 && ways <= n_experts, "moe_cache_create: need 1 <= ways <= n_experts (ways=%d n=%d)",
                    ways, n_experts);
        MOE_REQUIRE(n_layers == 0 || static_content, "moe_cache_create: the static policy needs its content");
        for (int l = 0; l < n_layers; ++l)
            for (int s = 0; s < ways; ++s) {
                const int32_t e = static_content[(size_t)l * ways + s];
                MOE_REQUIRE(e >= 0 && e < n_experts, "moe_cache_create: static expert %d (layer %d) out of range", e,
                            l);
                for (int q = 0; q < s; ++q)
                    MOE_REQUIRE(static_content[(size_t)l * ways + q] != e,
                                "moe_cache_create: expert %d listed twice in layer %d", e, l);
            }
    } else {
        MOE_REQUIRE(ways >= top_k && ways <= n_experts,
                    "moe_cache_create: need top_k <= ways <= n_experts (ways=%d top_k=%d n=%d)", ways, top_k,
                    n_experts);
    }
    Cache *c = new Cache();
    c->layers = n_layers;
    c->n = n_experts;
    c->ways = ways;
    c->top_k = top_k;
    c->policy = policy;
    if (policy == MOE_POLICY_STATIC) c->initial.assign(static_content, static_content + (size_t)n_layers * ways);
    c->slot_expert.assign((size_t)n_layers * ways, -1);
    c->slot_used.assign((size_t)n_layers * ways, 0);
    c->tick.assign((size_t)n_layers, 0);
    c->where.assign((size_t)n_layers * n_experts, -1);
    c->reset();
    *out = reinterpret_cast<moe_cache *>(c);
    return MOE_OK;
    MOE_GUARD_END
}

int moe_cache_create(int n_layers, int n_experts, int ways, int top_k, moe_cache **out)
{
    MOE_REQUIRE(n_layers >= 1, "moe_cache_create: n_layers=%d < 1", n_layers);
    return moe_cache_create_policy(n_layers, n_experts, ways, top_k, MOE_POLICY_LRU, nullptr, out);
}

int moe_cache_geometry(size_t budget_bytes, size_t expert_bytes, int ways, int n_layers, int *slots_out,
                       int *covered_out)
{
    MOE_REQUIRE(expert_bytes > 0 && ways >= 1 && n_layers >= 0, "moe_cache_geometry: bad arguments");
    const size_t S = budget_bytes / expert_bytes;
    const size_t N = S / (size_t)ways;
    if (slots_out) *slots_out = (int)std::min<size_t>(S, (size_t)INT32_MAX);
    if (covered_out) *covered_out = (int)std::min<size_t>(N, (size_t)n_layers);
    return MOE_OK;
}

void moe_cache_destroy(moe_cache *c) { delete reinterpret_cast<Cache *>(c); }

int moe_cache_reset(moe_cache *c)
{
    MOE_REQUIRE(c, "moe_cache_reset: null handle");
    reinterpret_cast<Cache *>(c)->reset();
    return MOE_OK;
}

int moe_cache_lookup(const moe_cache *ch, int layer, const int32_t *experts, int k, int32_t *slot_out,
                     uint8_t *hit_out)
{
    const Cache *c = reinterpret_cast<const Cache *>(ch);
    MOE_REQUIRE(c && experts, "moe_cache_lookup: null pointer");
    MOE_REQUIRE(layer >= 0 && layer < c->layers, "moe_cache_lookup: layer=%d out of [0,%d)", layer, c->layers);
    MOE_REQUIRE(c->valid_selection(experts, k),
                "moe_cache_lookup: need 1 <= k <= top_k distinct expert ids in [0,%d)", c->n);
    c->check(layer, experts, k, slot_out, hit_out);
    return MOE_OK;
}

int moe_cache_update(moe_cache *ch, int layer, const int32_t *experts, int k, int32_t *fill_slot_out,
                     int32_t *evicted_out)
{
    Cache *c = reinterpret_cast<Cache *>(ch);
    MOE_REQUIRE(c && experts, "moe_cache_update: null pointer");
    MOE_REQUIRE(layer >= 0 && layer < c->layers, "moe_cache_update: layer=%d out of [0,%d)", layer, c->layers);
    MOE_REQUIRE(c->valid_selection(experts, k),
                "moe_cache_update: need 1 <= k <= top_k distinct expert ids in [0,%d)", c->n);
    c->step(layer, experts, k, fill_slot_out, evicted_out);
    return MOE_OK;
}

int moe_cache_update_masked(moe_cache *ch, int layer, const int32_t *experts, int k, const uint8_t *insert,
                            int32_t *fill_slot_out, int32_t *evicted_out)
{
    Cache *c = reinterpret_cast<Cache *>(ch);
    MOE_REQUIRE(c && experts, "moe_cache_update_masked: null pointer");
    MOE_REQUIRE(layer >= 0 && layer < c->layers, "moe_cache_update_masked: layer=%d out of [0,%d)", layer, c->layers);
    MOE_REQUIRE(c->valid_selection(experts, k),
                "moe_cache_update_masked: need 1 <= k <= top_k distinct expert ids in [0,%d)", c->n);
    c->step(layer, experts, k, fill_slot_out, evicted_out, insert);
    return MOE_OK;
}

// Checkpoint layout (host byte order): a header of 7 int32 (magic, version, layers, n,
// ways, top_k, policy), then slot experts int32 [layers][ways], slot stamps uint64
// [layers][ways] and set clocks uint64 [layers]. The expert -> slot map is rebuilt.
namespace {
constexpr int32_t kStateMagic = 0x43454f4d;   // "MOEC"
constexpr int32_t kStateVersion = 1;
constexpr size_t kStateHeader = 7 * sizeof(int32_t);

size_t state_bytes(const Cache *c)
{
    const size_t slots = (size_t)c->layers * c->ways;
    return kStateHeader + slots * sizeof(int32_t) + slots * sizeof(uint64_t) + (size_t)c->layers * sizeof(uint64_t);
}
}  // namespace

size_t moe_cache_state_bytes(const moe_cache *ch)
{
    const Cache *c = reinterpret_cast<const Cache *>(ch);
    return c ? state_bytes(c) : 0;
}

int moe_cache_save(const moe_cache *ch, void *buf, size_t bytes)
{
    const Cache *c = reinterpret_cast<const Cache *>(ch);
    MOE_REQUIRE(c && buf, "moe_cache_save: null pointer");
    MOE_REQUIRE(bytes >= state_bytes(c), "moe_cache_save: buffer of %zu bytes, %zu needed", bytes, state_bytes(c));
    const int32_t head[7] = {kStateMagic, kStateVersion, c->layers, c->n, c->ways, c->top_k, c->policy};
    uint8_t *o = static_cast<uint8_t *>(buf);
    std::memcpy(o, head, kStateHeader);
    o += kStateHeader;
    const size_t slots = (size_t)c->layers * c->ways;
    std::memcpy(o, c->slot_expert.data(), slots * sizeof(int32_t));
    o += slots * sizeof(int32_t);
    std::memcpy(o, c->slot_used.data(), slots * sizeof(uint64_t));
    o += slots * sizeof(uint64_t);
    std::memcpy(o, c->tick.data(), (size_t)c->layers * sizeof(uint64_t));
    return MOE_OK;
}

int moe_cache_restore(moe_cache *ch, const void *buf, size_t bytes)
{
    MOE_GUARD_BEGIN
    Cache *c = reinterpret_cast<Cache *>(ch);
    MOE_REQUIRE(c && buf, "moe_cache_restore: null pointer");
    MOE_REQUIRE(bytes == state_bytes(c), "moe_cache_restore: %zu bytes, a state of this cache has %zu", bytes,
                state_bytes(c));
    const uint8_t *in = static_cast<const uint8_t *>(buf);
    int32_t head[7];
    std::memcpy(head, in, kStateHeader);
    MOE_REQUIRE(head[0] == kStateMagic && head[1] == kStateVersion, "moe_cache_restore: not a cache state");
    MOE_REQUIRE(head[2] == c->layers && head[3] == c->n && head[4] == c->ways && head[5] == c->top_k &&
                    head[6] == c->policy,
                "moe_cache_restore: state of a cache with another geometry or policy");
    const size_t slots = (size_t)c->layers * c->ways;
    std::vector<int32_t> sx(slots);
    std::vector<uint64_t> su(slots), clk((size_t)c->layers);
    std::memcpy(sx.data(), in + kStateHeader, slots * sizeof(int32_t));
    std::memcpy(su.data(), in + kStateHeader + slots * sizeof(int32_t), slots * sizeof(uint64_t));
    std::memcpy(clk.data(), in + kStateHeader + slots * (sizeof(int32_t) + sizeof(uint64_t)),
                (size_t)c->layers * sizeof(uint64_t));
    std::vector<int32_t> where((size_t)c->layers * c->n, -1);
    for (int l = 0; l < c->layers; ++l)
        for (int q = 0; q < c->ways; ++q) {
            const size_t i = (size_t)l * c->ways + q;
            const int32_t e = sx[i];
            MOE_REQUIRE(e >= -1 && e < c->n, "moe_cache_restore: expert %d in layer %d out of range", e, l);
            if (c->policy == MOE_POLICY_STATIC) {
                MOE_REQUIRE(e == c->initial[i] && su[i] == 0 && clk[l] == 0,
                            "moe_cache_restore: layer %d differs from the static content", l);
            } else if (e >= 0) {
                // a resident expert was stamped when the set's clock reached its stamp
                MOE_REQUIRE(su[i] >= 1 && su[i] <= clk[l], "moe_cache_restore: slot stamp after the clock (layer %d)",
                            l);
                for (int r = 0; r < q; ++r)
                    MOE_REQUIRE(sx[(size_t)l * c->ways + r] < 0 || su[(size_t)l * c->ways + r] != su[i],
                                "moe_cache_restore: two slots of layer %d with one stamp", l);
            }
            if (e >= 0) {
                MOE_REQUIRE(where[(size_t)l * c->n + e] < 0, "moe_cache_restore: expert %d twice in layer %d", e, l);
                where[(size_t)l * c->n + e] = q;
            }
        }
    c->slot_expert.swap(sx);
    c->slot_used.swap(su);
    c->tick.swap(clk);
    c->where.swap(where);
    return MOE_OK;
    MOE_GUARD_END
}

int moe_cache_slotmap(const moe_cache *ch, int layer, int32_t *slotmap_out)
{
    const Cache *c = reinterpret_cast<const Cache *>(ch);
    MOE_REQUIRE(c && slotmap_out, "moe_cache_slotmap: null pointer");
    MOE_REQUIRE(layer >= 0 && layer < c->layers, "moe_cache_slotmap: layer=%d out of [0,%d)", layer, c->layers);
    std::memcpy(slotmap_out, &c->where[(size_t)layer * c->n], sizeof(int32_t) * (size_t)c->n);
    return MOE_OK;
}

}  // extern "C"
