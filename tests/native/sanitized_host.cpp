// Host-side library code (cache sets and the host expert path) under AddressSanitizer
// and UndefinedBehaviorSanitizer, built by tests/test_native_sanitized.py with g++ (no
// device code; the two HIP allocation calls the host path makes are stubbed below and
// never reached). Exits 0 when every check holds; a sanitizer report aborts the run.
//
// Checks: random access traces for the three policies with plain and masked insertion
// against each set's own invariants (at most `ways` experts, no duplicates, slot ids in
// range, the selected experts resident after an LRU/FIFO step unless their insertion
// was masked, the static content never changing, lookup agreeing with the slot table
// and with the previous step's fills); checkpoint round trips and refused damaged states;
// rejected calls leave the state unchanged; reset;
// geometry; the host expert FFN identical (bit for bit) on 1, 2 and 5 threads, and zero
// for zero experts.
#include <hip/hip_runtime_api.h>

#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <set>
#include <vector>

#include "moe.h"

// ---- stand-ins for what the host sources take from the rest of the library ----
namespace moe {
static thread_local char g_msg[512];
void set_error(const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_msg, sizeof g_msg, fmt, ap);
    va_end(ap);
}
void clear_error() { g_msg[0] = 0; }
}  // namespace moe
hipError_t hipHostMalloc(void **, size_t, unsigned int) { return hipErrorOutOfMemory; }
hipError_t hipHostFree(void *) { return hipSuccess; }
const char *hipGetErrorString(hipError_t) { return "stub"; }

// ---------------------------------------------------------------------------------
static int g_failures = 0;
#define CHECK(cond, ...)                                                   \
    do {                                                                   \
        if (!(cond)) {                                                     \
            std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__);     \
            std::fprintf(stderr, __VA_ARGS__);                             \
            std::fprintf(stderr, "\n");                                    \
            if (++g_failures > 20) std::exit(1);                           \
        }                                                                  \
    } while (0)

static std::vector<int32_t> slotmap(moe_cache *c, int layer, int n)
{
    std::vector<int32_t> m(n, -7);
    CHECK(moe_cache_slotmap(c, layer, m.data()) == MOE_OK, "slotmap");
    return m;
}

static void check_set(const std::vector<int32_t> &m, int ways, const char *what)
{
    std::set<int32_t> slots;
    for (size_t e = 0; e < m.size(); ++e) {
        if (m[e] < 0) continue;
        CHECK(m[e] < ways, "%s: slot %d out of range", what, m[e]);
        CHECK(slots.insert(m[e]).second, "%s: slot %d holds two experts", what, m[e]);
    }
    CHECK((int)slots.size() <= ways, "%s: %zu experts in %d ways", what, slots.size(), ways);
}

static void trace_policy(int policy, bool masked, unsigned seed)
{
    std::mt19937 rng(seed);
    const int L = 3, n = 12, ways = 5, k = 3;
    std::vector<int32_t> content;
    if (policy == MOE_POLICY_STATIC)
        for (int l = 0; l < L; ++l)
            for (int j = 0; j < ways; ++j) content.push_back((l * 5 + j * 2) % n);
    moe_cache *c = nullptr;
    CHECK(moe_cache_create_policy(L, n, ways, k, policy, content.empty() ? nullptr : content.data(), &c) == MOE_OK,
          "create policy %d", policy);
    if (!c) return;
    for (int step = 0; step < 400; ++step) {
        const int l = (int)(rng() % L);
        // k distinct experts, biased to a window so hits and misses both happen
        std::vector<int32_t> sel;
        const int base = (int)(rng() % n);
        while ((int)sel.size() < k) {
            const int32_t e = (base + (int32_t)(rng() % 6)) % n;
            bool dup = false;
            for (int32_t s : sel) dup = dup || s == e;
            if (!dup) sel.push_back(e);
        }
        uint8_t insert[k];
        for (int j = 0; j < k; ++j) insert[j] = masked ? (uint8_t)(rng() & 1) : 1;
        const std::vector<int32_t> before = slotmap(c, l, n);
        int32_t slot[k];
        uint8_t hit[k];
        CHECK(moe_cache_lookup(c, l, sel.data(), k, slot, hit) == MOE_OK, "lookup");
        for (int j = 0; j < k; ++j) {
            CHECK(hit[j] == (before[sel[j]] >= 0), "lookup hit vs table");
            CHECK(slot[j] == before[sel[j]], "lookup slot vs table");
        }
        int32_t fill[k], ev[k];
        const int rc = masked ? moe_cache_update_masked(c, l, sel.data(), k, insert, fill, ev)
                              : moe_cache_update(c, l, sel.data(), k, fill, ev);
        CHECK(rc == MOE_OK, "update rc %d", rc);
        const std::vector<int32_t> after = slotmap(c, l, n);
        check_set(after, ways, "after update");
        for (int j = 0; j < k; ++j) {
            if (hit[j]) {
                CHECK(fill[j] == -1 && ev[j] == -1, "hit filled");
                CHECK(after[sel[j]] == before[sel[j]], "hit moved");
            } else if (policy == MOE_POLICY_STATIC || !insert[j]) {
                CHECK(fill[j] == -1 && ev[j] == -1, "non-inserted miss filled");
                CHECK(after[sel[j]] == -1, "non-inserted miss resident");
            } else {
                CHECK(fill[j] >= 0 && fill[j] < ways, "fill slot");
                CHECK(after[sel[j]] == fill[j], "filled expert not in its slot");
                if (ev[j] >= 0) {
                    CHECK(before[ev[j]] == fill[j], "evicted expert was not in the slot");
                    CHECK(after[ev[j]] == -1, "evicted expert still resident");
                    for (int32_t s : sel) CHECK(s != ev[j], "a selected expert was evicted");
                }
            }
        }
        // the other layers are untouched
        if (policy == MOE_POLICY_STATIC)
            for (int j = 0; j < ways; ++j) CHECK(after[content[l * ways + j]] == j, "static content changed");
    }
    // checkpoint round trip, and a damaged or truncated state refused
    {
        const size_t nb = moe_cache_state_bytes(c);
        std::vector<uint8_t> st(nb), st2(nb);
        CHECK(moe_cache_save(c, st.data(), nb) == MOE_OK, "save");
        moe_cache *d = nullptr;
        CHECK(moe_cache_create_policy(L, n, ways, k, policy, content.empty() ? nullptr : content.data(), &d) ==
                  MOE_OK, "create for restore");
        CHECK(moe_cache_restore(d, st.data(), nb) == MOE_OK, "restore");
        CHECK(moe_cache_save(d, st2.data(), nb) == MOE_OK && st == st2, "restored state differs");
        for (int l = 0; l < L; ++l) CHECK(slotmap(d, l, n) == slotmap(c, l, n), "restored table differs");
        CHECK(moe_cache_restore(d, st.data(), nb - 1) == MOE_EINVAL, "truncated state accepted");
        std::vector<uint8_t> bad = st;
        bad[28] = 0xff;   // first slot's expert id becomes negative and out of range
        bad[29] = 0xff;
        bad[30] = 0xff;
        bad[31] = 0x80;
        CHECK(moe_cache_restore(d, bad.data(), nb) == MOE_EINVAL, "damaged state accepted");
        CHECK(moe_cache_save(d, st2.data(), nb) == MOE_OK && st == st2, "refused restore changed the cache");
        moe_cache_destroy(d);
    }
    // rejected calls change nothing
    const std::vector<int32_t> keep = slotmap(c, 0, n);
    int32_t bad_dup[3] = {1, 1, 2}, bad_range[3] = {0, 1, n}, fill[3], ev[3];
    CHECK(moe_cache_update(c, 0, bad_dup, 3, fill, ev) == MOE_EINVAL, "duplicate ids accepted");
    CHECK(moe_cache_update(c, 0, bad_range, 3, fill, ev) == MOE_EINVAL, "id out of range accepted");
    CHECK(moe_cache_update(c, L, bad_dup, 3, fill, ev) == MOE_EINVAL, "layer out of range accepted");
    CHECK(moe_cache_update(c, 0, bad_dup, k + 1, fill, ev) == MOE_EINVAL, "k above top_k accepted");
    CHECK(slotmap(c, 0, n) == keep, "rejected update changed the set");
    CHECK(moe_cache_reset(c) == MOE_OK, "reset");
    for (int l = 0; l < L; ++l) {
        const std::vector<int32_t> m = slotmap(c, l, n);
        int resident = 0;
        for (int32_t v : m) resident += v >= 0;
        CHECK(resident == (policy == MOE_POLICY_STATIC ? ways : 0), "reset state");
    }
    moe_cache_destroy(c);
}

static void cache_arguments()
{
    moe_cache *c = nullptr;
    CHECK(moe_cache_create(1, 4, 1, 2, &c) == MOE_EINVAL && c == nullptr, "ways < top_k accepted");
    CHECK(moe_cache_create(0, 4, 2, 2, &c) == MOE_EINVAL, "no layers accepted");
    CHECK(moe_cache_create(1, MOE_MAX_EXPERTS + 1, 2, 2, &c) == MOE_EINVAL, "too many experts accepted");
    int32_t dup_content[2] = {3, 3};
    CHECK(moe_cache_create_policy(1, 4, 2, 1, MOE_POLICY_STATIC, dup_content, &c) == MOE_EINVAL,
          "static content with a duplicate accepted");
    CHECK(moe_cache_create_policy(1, 4, 2, 1, MOE_POLICY_STATIC, nullptr, &c) == MOE_EINVAL,
          "static policy without content accepted");
    CHECK(moe_cache_create_policy(0, 4, 2, 2, MOE_POLICY_LRU, nullptr, &c) == MOE_OK && c, "zero covered layers");
    moe_cache_destroy(c);
    int slots = -1, covered = -1;
    CHECK(moe_cache_geometry((size_t)56 * 1000, 1000, 4, 32, &slots, &covered) == MOE_OK && slots == 56 &&
              covered == 14, "geometry 56 slots / 4 ways");
    CHECK(moe_cache_geometry(999, 1000, 4, 32, &slots, &covered) == MOE_OK && slots == 0 && covered == 0,
          "geometry below one slot");
    CHECK(moe_cache_geometry((size_t)1 << 40, 1000, 4, 32, nullptr, &covered) == MOE_OK && covered == 32,
          "geometry capped by the layer count");
}

static uint16_t to_bf16(float v)
{
    uint32_t u;
    std::memcpy(&u, &v, 4);
    return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

static void host_path()
{
    const int d = 136, f = 72, ne = 3;   // not multiples of the vector width tails
    std::mt19937 rng(5);
    std::normal_distribution<float> nd(0.f, 0.05f);
    std::vector<std::vector<uint16_t>> slabs(ne, std::vector<uint16_t>((size_t)3 * d * f));
    for (auto &s : slabs)
        for (auto &v : s) v = to_bf16(nd(rng));
    std::vector<float> x(d), w = {0.5f, 0.3f, 0.2f};
    for (auto &v : x) v = nd(rng) * 20.f;
    const void *ptrs[ne] = {slabs[0].data(), slabs[1].data(), slabs[2].data()};
    std::vector<float> ref;
    for (int threads : {1, 2, 5}) {
        moe_host_pool *p = nullptr;
        CHECK(moe_host_pool_create(threads, &p) == MOE_OK && p, "pool %d", threads);
        if (!p) continue;
        CHECK(moe_host_pool_threads(p) == threads, "thread count");
        std::vector<float> y(d, -1.f);
        CHECK(moe_host_expert_ffn(p, x.data(), ptrs, w.data(), ne, d, f, y.data()) == MOE_OK, "host ffn");
        if (ref.empty()) ref = y;
        CHECK(std::memcmp(ref.data(), y.data(), sizeof(float) * d) == 0, "result depends on the thread count (%d)",
              threads);
        std::vector<float> z(d, -1.f);
        CHECK(moe_host_expert_ffn(p, x.data(), ptrs, w.data(), 0, d, f, z.data()) == MOE_OK, "zero experts");
        for (float v : z) CHECK(v == 0.f, "zero experts gave %g", v);
        CHECK(moe_host_expert_ffn(p, x.data(), ptrs, w.data(), MOE_MAX_TOPK + 1, d, f, z.data()) == MOE_EINVAL,
              "too many experts accepted");
        moe_host_pool_destroy(p);
    }
    void *mem = nullptr;
    CHECK(moe_host_alloc(0, &mem) == MOE_EINVAL, "zero-byte allocation accepted");
    CHECK(moe_host_alloc(64, &mem) == MOE_ENOMEM, "stubbed allocation did not report ENOMEM");
    CHECK(moe_host_free(nullptr) == MOE_OK, "free(NULL)");
}

int main()
{
    for (int policy : {MOE_POLICY_LRU, MOE_POLICY_FIFO, MOE_POLICY_STATIC})
        for (bool masked : {false, true})
            for (unsigned seed : {1u, 2u, 3u}) trace_policy(policy, masked, seed * 7 + (unsigned)policy);
    cache_arguments();
    host_path();
    if (g_failures) {
        std::fprintf(stderr, "%d check(s) failed\n", g_failures);
        return 1;
    }
    std::printf("sanitized host checks passed\n");
    return 0;
}
