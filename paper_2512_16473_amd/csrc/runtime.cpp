// One MoE layer of single-request decode, Section III-A of the paper (layers past the
// cache's covered ones, Section III-B, run every selected expert on the host):
//   step 1  cache check of the selected experts in the layer's set;
//   step 2a cache hits computed on the GPU from their cache slots;
//   step 2b the hidden state copied to the host, missed experts computed there;
//   step 3  missed experts' weights copied into the cache so later tokens find them there
//           (post-fetch), on a stream of its own (Section III-C keeps weight copies
//           off the stream that carries activations).
//
// Device side, in stream order on the compute stream: [parity mode: wait for this
// layer's earlier post-fetch, if still running] router -> gate/up/SiLU -> down ->
// reduce+combine, with no other commands between the kernels. The router kernel installs
// the layer's row of the device expert->slot mirror (copied from coherent pinned memory
// that holds the host's record of landed copies) before the hit kernels read it, and it
// hands the routing and the hidden state to the host: it writes them into coherent
// pinned memory followed by a sequence number, which the host polls (the activation
// exchange never queues behind weight copies). The host then updates the cache table,
// starts the post-fetch copies on the copy stream, runs the misses on its thread pool
// into coherent pinned memory that the reduce kernel reads directly, and enqueues the
// reduce. A post-fetched expert joins the mirror at a later call on its layer once its
// copy has landed: parity mode waits for the copy, so the hit/miss sequence does not
// depend on timing; non-blocking mode runs the expert on the host until then.
#include <immintrin.h>

#include <algorithm>
#include <chrono>
#include <deque>
#include <cstring>
#include <vector>

#include "cache.h"
#include "common.h"
#include "hostpath.h"
#include "moe_internal.h"

static_assert(MOE_MAX_TOPK_INTERNAL == MOE_MAX_TOPK, "mailbox size must match the ABI bound");

namespace {

// Events of one timed layer call. The hit count (and so the bytes) is known on the
// host only after the routing read-back; it is filled in then.
struct TimingRec {
    hipEvent_t ev[4];   // gate/up start, stop; down start, stop
    double bytes_gu;
    double bytes_dn;
};

}  // namespace

struct moe_runtime {
    moe_layer_desc desc{};
    std::vector<const void *> host_slabs;   // [L][n]
    size_t slab_bytes = 0, shared_bytes = 0;
    size_t slab_payload = 0;                // 3*d*f*2, the bytes a post-fetch copies
    moe::Cache *cache = nullptr;
    moe::HostPool *pool = nullptr;

    // device
    int32_t *d_slotmap = nullptr;   // [L][n]
    int32_t *d_idx = nullptr;       // [k]
    float *d_w = nullptr;           // [k]
    void *d_ws = nullptr;
    size_t ws_bytes = 0;
    void *d_route = nullptr;        // decode router: partial logits + arrival counter (zeroed once)

    // coherent pinned host memory shared with the kernels (host address, device address)
    moe::RouteMailbox *mbox = nullptr, *mbox_dev = nullptr;
    float *h_x = nullptr, *h_x_dev = nullptr;   // [d] hidden state of the current layer call
    float *h_y = nullptr, *h_y_dev = nullptr;   // [L][d] host-path output per layer
    std::vector<float> x_local, y_local;        // [d] cached host copies for the host FFN
    int32_t seq = 0;
    // Device mirror of the slot table. Its rows are installed by the layer's router
    // kernel from coherent host memory (h_rows), so the hit kernels of a layer call see
    // exactly the row the host decided on for that call. dev_row is the host's copy of
    // what the device holds: a slot appears there only once its post-fetch has landed.
    int32_t *h_rows = nullptr, *h_rows_dev = nullptr;   // [L][n]
    std::vector<int32_t> dev_row;                        // [L][n]
    std::vector<std::vector<std::pair<int32_t, int32_t>>> pend_fill;   // [L] (expert, slot) in flight
    std::vector<std::vector<int32_t>> pend_inval;       // [L] evicted experts to drop at the next call
    bool nonblocking = false;

    std::vector<hipEvent_t> ev_fill;   // [L] after the layer's latest slab copies
    std::vector<char> fill_pending;    // [L]

    // Bounded post-fetch: at most fill_limit slabs queued on the copy stream (0: no
    // bound). Fills complete in issue order (one stream), so a FIFO of per-call events
    // tells how many slabs are still in flight.
    int fill_limit = 0;
    std::deque<std::pair<hipEvent_t, int>> inflight;
    std::vector<hipEvent_t> fill_spare;

    bool timing = false;
    std::vector<TimingRec> pending;    // recorded, not yet resolved
    std::vector<hipEvent_t> spare;     // resolved events for reuse

    moe_runtime_stats stats{};
};

namespace {

void release(moe_runtime *rt)
{
    if (!rt) return;
    for (auto &r : rt->pending)
        for (auto e : r.ev) (void)hipEventDestroy(e);
    for (auto e : rt->spare) (void)hipEventDestroy(e);
    for (auto &q : rt->inflight) (void)hipEventDestroy(q.first);
    for (auto e : rt->fill_spare) (void)hipEventDestroy(e);
    for (auto e : rt->ev_fill)
        if (e) (void)hipEventDestroy(e);

    if (rt->d_slotmap) (void)hipFree(rt->d_slotmap);
    if (rt->d_idx) (void)hipFree(rt->d_idx);
    if (rt->d_w) (void)hipFree(rt->d_w);
    if (rt->d_ws) (void)hipFree(rt->d_ws);
    if (rt->d_route) (void)hipFree(rt->d_route);
    if (rt->mbox) (void)hipHostFree(rt->mbox);
    if (rt->h_x) (void)hipHostFree(rt->h_x);
    if (rt->h_y) (void)hipHostFree(rt->h_y);
    if (rt->h_rows) (void)hipHostFree(rt->h_rows);
    delete rt;
}

hipEvent_t take_event(moe_runtime *rt)
{
    if (!rt->spare.empty()) {
        hipEvent_t e = rt->spare.back();
        rt->spare.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// Resolve recorded timing events (the compute stream must have been synchronised).
int resolve_timing(moe_runtime *rt)
{
    for (auto &r : rt->pending) {
        float a = 0.f, b = 0.f;
        MOE_HIP(hipEventSynchronize(r.ev[3]));
        MOE_HIP(hipEventElapsedTime(&a, r.ev[0], r.ev[1]));
        MOE_HIP(hipEventElapsedTime(&b, r.ev[2], r.ev[3]));
        rt->stats.gate_up_launches += 1;
        rt->stats.gate_up_ms += a;
        rt->stats.gate_up_bytes += r.bytes_gu;
        rt->stats.down_launches += 1;
        rt->stats.down_ms += b;
        rt->stats.down_bytes += r.bytes_dn;
        for (auto e : r.ev) rt->spare.push_back(e);
    }
    rt->pending.clear();
    return MOE_OK;
}

// Slabs still being copied: retire completed entries from the front of the FIFO.
int slabs_in_flight(moe_runtime *rt)
{
    while (!rt->inflight.empty() && hipEventQuery(rt->inflight.front().first) == hipSuccess) {
        rt->fill_spare.push_back(rt->inflight.front().first);
        rt->inflight.pop_front();
    }
    (void)hipGetLastError();   // a not-ready query leaves hipErrorNotReady behind
    int n = 0;
    for (auto &q : rt->inflight) n += q.second;
    return n;
}

double now_ms()
{
    return std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now().time_since_epoch()).count();
}

}  // namespace

extern "C" {

int moe_runtime_create(const moe_layer_desc *desc, moe_runtime **out)
{
    MOE_GUARD_BEGIN
    MOE_REQUIRE(desc && out, "moe_runtime_create: null pointer");
    const moe_layer_desc &D = *desc;
    MOE_REQUIRE(D.d > 0 && D.d % 8 == 0 && D.d <= MOE_MAX_D, "moe_runtime_create: d=%d must be a multiple of 8 in [8,%d]",
                D.d, MOE_MAX_D);
    MOE_REQUIRE(D.f > 0 && D.f % 8 == 0, "moe_runtime_create: f=%d must be a positive multiple of 8", D.f);
    MOE_REQUIRE(D.f_shared >= 0 && D.f_shared % 8 == 0, "moe_runtime_create: f_shared=%d must be a multiple of 8",
                D.f_shared);
    MOE_REQUIRE(D.n >= 1 && D.n <= MOE_MAX_EXPERTS, "moe_runtime_create: n=%d out of range", D.n);
    MOE_REQUIRE(D.k >= 1 && D.k <= MOE_MAX_TOPK && D.k <= D.ways && D.ways <= D.n,
                "moe_runtime_create: need 1 <= k <= ways <= n (k=%d ways=%d n=%d)", D.k, D.ways, D.n);
    MOE_REQUIRE(D.n_layers >= 1, "moe_runtime_create: n_layers=%d < 1", D.n_layers);
    MOE_REQUIRE(D.w_router && D.host_slabs && D.cache && D.pool, "moe_runtime_create: null pointer");
    MOE_REQUIRE(D.f_shared == 0 || D.shared_pool, "moe_runtime_create: f_shared > 0 needs shared_pool");
    MOE_REQUIRE(moe::aligned16(D.w_router) && (!D.slot_pool || moe::aligned16(D.slot_pool)) &&
                    (!D.shared_pool || moe::aligned16(D.shared_pool)),
                "moe_runtime_create: device pointers must be 16-byte aligned");
    const moe::Cache *c = reinterpret_cast<const moe::Cache *>(D.cache);
    MOE_REQUIRE(c->layers <= D.n_layers && c->n == D.n && c->ways == D.ways && c->top_k == D.k,
                "moe_runtime_create: cache geometry (covered=%d n=%d ways=%d k=%d) does not fit the descriptor",
                c->layers, c->n, c->ways, c->top_k);
    MOE_REQUIRE(c->layers == 0 || D.slot_pool, "moe_runtime_create: covered layers need a slot pool");
    const size_t nh = (size_t)D.n_layers * D.n;
    for (size_t i = 0; i < nh; ++i)
        MOE_REQUIRE(D.host_slabs[i], "moe_runtime_create: host_slabs[%zu] is null", i);

    moe_runtime *rt = new moe_runtime();
    rt->desc = D;
    rt->host_slabs.assign(D.host_slabs, D.host_slabs + nh);
    rt->desc.host_slabs = rt->host_slabs.data();
    rt->slab_bytes = moe_slab_bytes(D.d, D.f);
    rt->slab_payload = (size_t)3 * D.d * D.f * 2;
    rt->shared_bytes = D.f_shared ? moe_slab_bytes(D.d, D.f_shared) : 0;
    rt->cache = reinterpret_cast<moe::Cache *>(D.cache);
    rt->pool = reinterpret_cast<moe::HostPool *>(D.pool);
    rt->x_local.assign(D.d, 0.f);
    rt->y_local.assign(D.d, 0.f);

    auto fail = [&](hipError_t e, const char *what) {
        moe::set_error("moe_runtime_create: %s failed: %s", what, hipGetErrorString(e));
        release(rt);
        return e == hipErrorOutOfMemory ? MOE_ENOMEM : MOE_EHIP;
    };
    hipError_t e;
    const int fmax = D.f > D.f_shared ? D.f : D.f_shared;
    rt->ws_bytes = moe::ffn_workspace_bytes(D.k + 1, D.d, fmax);
    if ((e = hipMalloc(&rt->d_ws, rt->ws_bytes)) != hipSuccess) return fail(e, "hipMalloc(workspace)");
    const size_t route_bytes = moe::route1_scratch_bytes(D.n, D.d);
    if ((e = hipMalloc(&rt->d_route, route_bytes)) != hipSuccess) return fail(e, "hipMalloc(router scratch)");
    if ((e = hipMemset(rt->d_route, 0, route_bytes)) != hipSuccess) return fail(e, "hipMemset(router scratch)");
    if ((e = hipMalloc((void **)&rt->d_slotmap, sizeof(int32_t) * nh)) != hipSuccess) return fail(e, "hipMalloc");
    if ((e = hipMalloc((void **)&rt->d_idx, sizeof(int32_t) * D.k)) != hipSuccess) return fail(e, "hipMalloc");
    if ((e = hipMalloc((void **)&rt->d_w, sizeof(float) * D.k)) != hipSuccess) return fail(e, "hipMalloc");
    const unsigned coherent = hipHostMallocCoherent | hipHostMallocMapped;
    if ((e = hipHostMalloc((void **)&rt->mbox, sizeof(moe::RouteMailbox), coherent)) != hipSuccess)
        return fail(e, "hipHostMalloc(mailbox)");
    if ((e = hipHostMalloc((void **)&rt->h_x, sizeof(float) * D.d, coherent)) != hipSuccess)
        return fail(e, "hipHostMalloc(x)");
    if ((e = hipHostMalloc((void **)&rt->h_y, sizeof(float) * D.d * (size_t)D.n_layers, coherent)) != hipSuccess)
        return fail(e, "hipHostMalloc(y)");
    std::memset(rt->mbox, 0, sizeof(moe::RouteMailbox));
    if ((e = hipHostGetDevicePointer((void **)&rt->mbox_dev, rt->mbox, 0)) != hipSuccess)
        return fail(e, "hipHostGetDevicePointer");
    if ((e = hipHostGetDevicePointer((void **)&rt->h_x_dev, rt->h_x, 0)) != hipSuccess)
        return fail(e, "hipHostGetDevicePointer");
    if ((e = hipHostGetDevicePointer((void **)&rt->h_y_dev, rt->h_y, 0)) != hipSuccess)
        return fail(e, "hipHostGetDevicePointer");
    if ((e = hipHostMalloc((void **)&rt->h_rows, sizeof(int32_t) * nh, coherent)) != hipSuccess)
        return fail(e, "hipHostMalloc(rows)");
    if ((e = hipHostGetDevicePointer((void **)&rt->h_rows_dev, rt->h_rows, 0)) != hipSuccess)
        return fail(e, "hipHostGetDevicePointer");
    // Slots the cache holds already (static content, warm cache) get their slabs now.
    for (int l = 0; l < c->layers; ++l)
        for (int sl = 0; sl < D.ways; ++sl) {
            const int32_t ex = c->slot_expert[(size_t)l * D.ways + sl];
            if (ex < 0) continue;
            uint8_t *dst = static_cast<uint8_t *>(D.slot_pool) + ((size_t)l * D.ways + sl) * rt->slab_bytes;
            if ((e = hipMemcpy(dst, D.host_slabs[(size_t)l * D.n + ex], rt->slab_payload, hipMemcpyHostToDevice)) !=
                hipSuccess)
                return fail(e, "hipMemcpy(initial slot)");
        }
    // Mirror of the host table as it stands now; uncovered layers map nothing.
    rt->dev_row.assign(nh, -1);
    for (int l = 0; l < c->layers; ++l)
        std::memcpy(&rt->dev_row[(size_t)l * D.n], &c->where[(size_t)l * D.n], sizeof(int32_t) * D.n);
    std::memcpy(rt->h_rows, rt->dev_row.data(), sizeof(int32_t) * nh);
    if ((e = hipMemcpy(rt->d_slotmap, rt->h_rows, sizeof(int32_t) * nh, hipMemcpyHostToDevice)) != hipSuccess)
        return fail(e, "hipMemcpy(slotmap)");
    rt->pend_fill.assign(D.n_layers, {});
    rt->pend_inval.assign(D.n_layers, {});
    rt->ev_fill.assign(D.n_layers, nullptr);
    rt->fill_pending.assign(D.n_layers, 0);
    for (int l = 0; l < D.n_layers; ++l)
        if ((e = hipEventCreateWithFlags(&rt->ev_fill[l], hipEventDisableTiming)) != hipSuccess)
            return fail(e, "event");
    *out = rt;
    return MOE_OK;
    MOE_GUARD_END
}

void moe_runtime_destroy(moe_runtime *rt)
{
    if (!rt) return;
    (void)hipDeviceSynchronize();
    release(rt);
}

int moe_layer_forward(moe_runtime *rt, int layer, const float *x_dev, float *out_dev, int32_t *idx_host,
                      float *w_host, uint8_t *hit_host, void *compute_stream, void *act_stream, void *copy_stream)
{
    MOE_GUARD_BEGIN
    MOE_REQUIRE(rt && x_dev && out_dev, "moe_layer_forward: null pointer");
    const moe_layer_desc &D = rt->desc;
    MOE_REQUIRE(layer >= 0 && layer < D.n_layers, "moe_layer_forward: layer=%d out of [0,%d)", layer, D.n_layers);
    MOE_REQUIRE(moe::aligned16(x_dev) && moe::aligned16(out_dev), "moe_layer_forward: x/out not 16-byte aligned");
    (void)act_stream;   // the router kernel hands routing and x to the host directly
    hipStream_t sc = (hipStream_t)compute_stream, sw = (hipStream_t)copy_stream;
    const int d = D.d, n = D.n, k = D.k;

    // This call's mirror row: experts evicted at the previous call leave it; post-fetches
    // into this set join it once they have landed. In parity mode an unfinished
    // post-fetch is waited for (the compute stream waits on its event); in non-blocking
    // mode its experts stay out of the row and run on the host this time.
    int32_t *row = &rt->dev_row[(size_t)layer * n];
    bool install = !rt->pend_inval[layer].empty();
    for (const int32_t v : rt->pend_inval[layer]) row[v] = -1;
    rt->pend_inval[layer].clear();
    if (rt->fill_pending[layer]) {
        const hipError_t q = hipEventQuery(rt->ev_fill[layer]);
        if (q != hipSuccess && q != hipErrorNotReady) MOE_HIP(q);
        (void)hipGetLastError();
        bool landed = q == hipSuccess;
        if (!landed && !rt->nonblocking) {
            MOE_HIP(hipStreamWaitEvent(sc, rt->ev_fill[layer], 0));
            landed = true;
        }
        if (landed) {
            for (const auto &fs : rt->pend_fill[layer]) row[fs.first] = fs.second;
            rt->pend_fill[layer].clear();
            rt->fill_pending[layer] = 0;
            install = true;
        }
    }
    int32_t *row_host = rt->h_rows + (size_t)layer * n;
    if (install) std::memcpy(row_host, row, sizeof(int32_t) * n);

    // Router; it publishes the routing and x to the host through the mailbox and
    // installs the mirror row before the hit kernels read it.
    const int32_t seq = ++rt->seq;
    const float *wr = D.w_router + (size_t)layer * n * d;
    MOE_HIP(moe::launch_route1(x_dev, wr, d, n, k, rt->d_idx, rt->d_w, rt->d_route, sc, rt->mbox_dev, rt->h_x_dev,
                               seq, install ? rt->h_rows_dev + (size_t)layer * n : nullptr,
                               rt->d_slotmap + (size_t)layer * n));

    // Hit experts on the device (slots from the device mirror of the table).
    moe::FfnParams p{};
    p.x = x_dev;
    const bool covered = layer < rt->cache->layers;
    // An uncovered layer's mirror row is all -1, so the hit kernels take no slot from it.
    p.pool = covered ? static_cast<const uint8_t *>(D.slot_pool) + (size_t)layer * D.ways * rt->slab_bytes
                     : static_cast<const uint8_t *>(D.slot_pool);
    p.slab_stride = rt->slab_bytes;
    p.sel = rt->d_idx;
    p.slotmap = rt->d_slotmap + (size_t)layer * n;
    p.w = rt->d_w;
    p.k = k;
    p.n = n;
    p.nslots = D.ways;
    p.shared = D.f_shared ? static_cast<const uint8_t *>(D.shared_pool) + (size_t)layer * rt->shared_bytes : nullptr;
    p.f_shared = D.f_shared;
    p.d = d;
    p.f = D.f;
    moe::ffn_bind_workspace(p, rt->d_ws, k + 1, d, D.f > D.f_shared ? D.f : D.f_shared);
    moe::FfnEvents ev;
    TimingRec rec{};
    if (rt->timing) {
        for (auto &e : rec.ev) {
            e = take_event(rt);
            MOE_REQUIRE(e, "moe_layer_forward: could not create timing events");
        }
        ev.gu_start = rec.ev[0];
        ev.gu_stop = rec.ev[1];
        ev.dn_start = rec.ev[2];
        ev.dn_stop = rec.ev[3];
    }
    MOE_HIP(moe::launch_ffn_stream(p, sc, rt->timing ? &ev : nullptr));

    // Step 1 on the host: wait for the routing, then check + LRU update.
    const double t0 = now_ms();
    for (uint64_t spins = 0;; ++spins) {
        if (__atomic_load_n(&rt->mbox->seq, __ATOMIC_ACQUIRE) == seq) break;
        if ((spins & 0xffff) == 0xffff && now_ms() - t0 > 60000.0) {
            moe::set_error("moe_layer_forward: routing of layer %d not published within 60 s", layer);
            return MOE_EHIP;
        }
        _mm_pause();
    }
    rt->stats.route_wait_ms += now_ms() - t0;
    int32_t sel[MOE_MAX_TOPK], fill[MOE_MAX_TOPK], evicted[MOE_MAX_TOPK];
    float wsel[MOE_MAX_TOPK];
    uint8_t hit[MOE_MAX_TOPK];
    std::memcpy(sel, rt->mbox->idx, sizeof(int32_t) * k);
    std::memcpy(wsel, rt->mbox->w, sizeof(float) * k);
    MOE_REQUIRE(rt->cache->valid_selection(sel, k), "moe_layer_forward: router returned an invalid selection");
    if (covered) {
        rt->cache->check(layer, sel, k, nullptr, hit);
        uint8_t allow[MOE_MAX_TOPK];
        const uint8_t *allow_p = nullptr;
        if (rt->fill_limit > 0) {
            // The misses the cache would insert, in its (ascending-id) order, get the
            // remaining copy budget; the others stay on the host and are not inserted.
            int budget = rt->fill_limit - slabs_in_flight(rt);
            int order[MOE_MAX_TOPK];
            for (int j = 0; j < k; ++j) order[j] = j;
            std::sort(order, order + k, [&](int a, int b) { return sel[a] < sel[b]; });
            for (int q = 0; q < k; ++q) {
                const int j = order[q];
                allow[j] = 1;
                if (!hit[j]) {
                    allow[j] = budget > 0;
                    budget -= allow[j];
                }
            }
            allow_p = allow;
        }
        rt->cache->step(layer, sel, k, fill, evicted, allow_p);
    } else {   // no cache set: every expert on the host, nothing fetched
        for (int j = 0; j < k; ++j) {
            hit[j] = 0;
            fill[j] = evicted[j] = -1;
        }
    }
    int nfill = 0;
    for (int j = 0; j < k; ++j) nfill += fill[j] >= 0;
    if (covered && rt->cache->policy != MOE_POLICY_STATIC)
        for (int j = 0; j < k; ++j) rt->stats.fills_skipped += !hit[j] && fill[j] < 0;
    // Where each expert runs: on the GPU iff this call's mirror row holds it (a cache hit
    // whose post-fetch has landed); otherwise on the host.
    for (int j = 0; j < k; ++j) {
        const bool gpu = row[sel[j]] >= 0;
        rt->stats.inflight_misses += hit[j] && !gpu;
        hit[j] = gpu;
    }

    int nmiss = 0, nhit = 0;
    const void *mslab[MOE_MAX_TOPK];
    float mw[MOE_MAX_TOPK];
    for (int j = 0; j < k; ++j) {
        if (hit[j]) {
            ++nhit;
            continue;
        }
        mslab[nmiss] = rt->host_slabs[(size_t)layer * n + sel[j]];
        mw[nmiss] = wsel[j];
        ++nmiss;
    }
    if (rt->timing) {
        const double dd = d, ff = D.f, fs = D.f_shared;
        rec.bytes_gu = nhit * (2.0 * ff * dd * 2.0 + ff * 4.0) + (fs > 0 ? 2.0 * fs * dd * 2.0 + fs * 4.0 : 0.0) + dd * 4.0;
        rec.bytes_dn = nhit * (dd * ff * 2.0 + ff * 4.0 + dd * 4.0) + (fs > 0 ? dd * fs * 2.0 + fs * 4.0 + dd * 4.0 : 0.0);
        rt->pending.push_back(rec);
    }

    // Step 3 starts first: post-fetch of the missed experts into their victim slots.
    // The slabs can land at once: no current-token expert is ever a victim, and the
    // previous token's kernels on this layer finished before this token's router.
    if (nfill) {
        uint8_t *set_base = static_cast<uint8_t *>(D.slot_pool) + (size_t)layer * D.ways * rt->slab_bytes;
        auto &pf = rt->pend_fill[layer];
        for (int j = 0; j < k; ++j) {
            if (fill[j] < 0) continue;
            // The evicted expert leaves the row at the next call, before any kernel could
            // read its slot again; a victim still in flight is simply superseded.
            if (evicted[j] >= 0) {
                rt->pend_inval[layer].push_back(evicted[j]);
                for (size_t q = 0; q < pf.size(); ++q)
                    if (pf[q].first == evicted[j]) {
                        pf.erase(pf.begin() + (ptrdiff_t)q);
                        break;
                    }
            }
            pf.emplace_back(sel[j], fill[j]);
            MOE_HIP(hipMemcpyAsync(set_base + (size_t)fill[j] * rt->slab_bytes,
                                   rt->host_slabs[(size_t)layer * n + sel[j]], rt->slab_payload,
                                   hipMemcpyHostToDevice, sw));
            rt->stats.fills += 1;
        }
    }

    // Step 2(b): misses on the host thread pool, written where the reduce reads them.
    // x and y cross through ordinary cached host memory: the coherent buffers the GPU
    // shares are not what the dot products should re-read for every weight row.
    if (nmiss) {
        const double t2 = now_ms();
        std::memcpy(rt->x_local.data(), rt->h_x, sizeof(float) * d);
        rt->pool->expert_ffn(rt->x_local.data(), mslab, mw, nmiss, d, D.f, rt->y_local.data());
        std::memcpy(rt->h_y + (size_t)layer * d, rt->y_local.data(), sizeof(float) * d);
        rt->stats.host_ffn_ms += now_ms() - t2;
    }
    MOE_HIP(moe::launch_ffn_reduce(p, nmiss ? rt->h_y_dev + (size_t)layer * d : nullptr, out_dev, sc));

    // The layer's copies are done when this event is; the next call installs them.
    if (nfill) {
        MOE_HIP(hipEventRecord(rt->ev_fill[layer], sw));
        rt->fill_pending[layer] = 1;
        if (rt->fill_limit > 0) {
            hipEvent_t fe = nullptr;
            if (!rt->fill_spare.empty()) {
                fe = rt->fill_spare.back();
                rt->fill_spare.pop_back();
            } else {
                MOE_HIP(hipEventCreateWithFlags(&fe, hipEventDisableTiming));
            }
            MOE_HIP(hipEventRecord(fe, sw));
            rt->inflight.emplace_back(fe, nfill);
        }
    }

    rt->stats.layer_calls += 1;
    rt->stats.expert_hits += nhit;
    rt->stats.expert_misses += nmiss;
    if (idx_host) std::memcpy(idx_host, sel, sizeof(int32_t) * k);
    if (w_host) std::memcpy(w_host, wsel, sizeof(float) * k);
    if (hit_host) std::memcpy(hit_host, hit, k);
    return MOE_OK;
    MOE_GUARD_END
}

int moe_decode_step(moe_runtime *rt, const float *x_dev, float *out_dev, int32_t *idx_host, float *w_host,
                    uint8_t *hit_host, void *compute_stream, void *act_stream, void *copy_stream)
{
    MOE_REQUIRE(rt && x_dev && out_dev, "moe_decode_step: null pointer");
    const moe_layer_desc &D = rt->desc;
    for (int l = 0; l < D.n_layers; ++l) {
        const size_t o = (size_t)l * D.d, q = (size_t)l * D.k;
        const int rc = moe_layer_forward(rt, l, x_dev + o, out_dev + o, idx_host ? idx_host + q : nullptr,
                                         w_host ? w_host + q : nullptr, hit_host ? hit_host + q : nullptr,
                                         compute_stream, act_stream, copy_stream);
        if (rc != MOE_OK) return rc;
    }
    return MOE_OK;
}

int moe_runtime_sync(moe_runtime *rt)
{
    MOE_REQUIRE(rt, "moe_runtime_sync: null handle");
    const int n = rt->desc.n;
    bool any = false;
    for (int l = 0; l < rt->desc.n_layers; ++l)
        any = any || rt->fill_pending[l] || !rt->pend_inval[l].empty();
    if (!any) return MOE_OK;
    // Every copy has landed once the device is idle; install what the next calls would.
    MOE_HIP(hipDeviceSynchronize());
    for (int l = 0; l < rt->desc.n_layers; ++l) {
        if (!rt->fill_pending[l] && rt->pend_inval[l].empty()) continue;
        int32_t *row = &rt->dev_row[(size_t)l * n];
        for (const int32_t v : rt->pend_inval[l]) row[v] = -1;
        for (const auto &fs : rt->pend_fill[l]) row[fs.first] = fs.second;
        rt->pend_inval[l].clear();
        rt->pend_fill[l].clear();
        rt->fill_pending[l] = 0;
        MOE_HIP(hipMemcpy(rt->d_slotmap + (size_t)l * n, row, sizeof(int32_t) * n, hipMemcpyHostToDevice));
    }
    return MOE_OK;
}

int moe_runtime_set_nonblocking(moe_runtime *rt, int enable)
{
    MOE_REQUIRE(rt, "moe_runtime_set_nonblocking: null handle");
    rt->nonblocking = enable != 0;
    return MOE_OK;
}

int moe_runtime_device_slotmap(moe_runtime *rt, int layer, int32_t *slotmap_out)
{
    MOE_REQUIRE(rt && slotmap_out, "moe_runtime_device_slotmap: null pointer");
    MOE_REQUIRE(layer >= 0 && layer < rt->desc.n_layers, "moe_runtime_device_slotmap: layer out of range");
    const int rc = moe_runtime_sync(rt);
    if (rc != MOE_OK) return rc;
    MOE_HIP(hipMemcpy(slotmap_out, rt->d_slotmap + (size_t)layer * rt->desc.n, sizeof(int32_t) * rt->desc.n,
                      hipMemcpyDeviceToHost));
    return MOE_OK;
}

int moe_runtime_set_fill_limit(moe_runtime *rt, int max_slabs_in_flight)
{
    MOE_REQUIRE(rt, "moe_runtime_set_fill_limit: null handle");
    MOE_REQUIRE(max_slabs_in_flight >= 0, "moe_runtime_set_fill_limit: %d < 0", max_slabs_in_flight);
    rt->fill_limit = max_slabs_in_flight;
    return MOE_OK;
}

int moe_runtime_set_timing(moe_runtime *rt, int enable)
{
    MOE_REQUIRE(rt, "moe_runtime_set_timing: null handle");
    const int rc = resolve_timing(rt);
    if (rc != MOE_OK) return rc;
    rt->timing = enable != 0;
    return MOE_OK;
}

int moe_runtime_get_stats(moe_runtime *rt, moe_runtime_stats *out)
{
    MOE_REQUIRE(rt && out, "moe_runtime_get_stats: null pointer");
    const int rc = resolve_timing(rt);
    if (rc != MOE_OK) return rc;
    *out = rt->stats;
    return MOE_OK;
}

int moe_runtime_reset_stats(moe_runtime *rt)
{
    MOE_REQUIRE(rt, "moe_runtime_reset_stats: null handle");
    const int rc = resolve_timing(rt);
    if (rc != MOE_OK) return rc;
    rt->stats = moe_runtime_stats{};
    return MOE_OK;
}

}  // extern "C"
