// Internal interfaces between the C ABI (host C++) and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace moe {

constexpr int kMaxJobs = 17;        // up to 16 routed experts + one shared expert
#define MOE_MAX_TOPK_INTERNAL 16
constexpr int kSegMax = 4096;       // down-projection reduction segment (elements)
constexpr int kRowsPerDownItem = 16;

// Parameters of the hit-expert FFN (gate/up/SiLU, down, reduce). A "job" is one
// expert to evaluate: routed job j < k takes its slab from the slot pool at
// slot = slotmap ? slotmap[sel[j]] : sel[j] (skipped when < 0 or when sel[j] is
// out of range, or when the slot is outside [0, nslots)); job k is the shared expert when `shared` is non-null.
struct FfnParams {
    const float *x;              // [d]
    const uint8_t *pool;         // slot pool base
    uint64_t slab_stride;        // bytes between slabs
    const int32_t *sel;          // [k]
    const int32_t *slotmap;      // [n] or null
    const float *w;              // [k] gate weights (applied in the reduce)
    int k;
    int n;                       // experts per layer (range check of sel when slotmap is used)
    int nslots;                  // slabs in the pool; slots outside [0, nslots) are inactive
    const uint8_t *shared;       // shared-expert slab or null
    int f_shared;
    int d, f;
    int32_t *jobslot;            // [kMaxJobs] slot of each job, -1 inactive (written by gate/up)
    float *h;                    // [kMaxJobs][hstride]
    int hstride;
    float *partial;              // [kMaxJobs][smax][d]
    int smax;
};

// Workspace layout helpers.
size_t ffn_workspace_bytes(int max_jobs, int d, int f_max);
void ffn_bind_workspace(FfnParams &p, void *ws, int max_jobs, int d, int f_max);

// The allocation-free hit FFN's device scratch (a static device array of this many
// bytes, one per device): noalloc_scratch returns its address on the current device.
constexpr size_t kNoAllocScratchBytes = (size_t)8 << 20;
constexpr int kMaxDevices = 64;
hipError_t noalloc_scratch(void **ptr);

// Events attached to the two weight-streaming kernel launches (null = no timing).
// They are recorded by the launch itself (start and stop of that dispatch), so their
// difference is the kernel's execution time without the dispatch gap.
struct FfnEvents {
    hipEvent_t gu_start = nullptr, gu_stop = nullptr, dn_start = nullptr, dn_stop = nullptr;
};

// Host-visible copy of one token's routing, written by the router kernel into
// coherent pinned memory: the selection, the gate weights and the hidden state, then
// `seq` (release, system scope) once everything before it is visible to the host.
struct RouteMailbox {
    int32_t seq;
    int32_t pad[15];
    int32_t idx[MOE_MAX_TOPK_INTERNAL];
    float w[MOE_MAX_TOPK_INTERNAL];
};

// Single-token decode router, one wave per (expert, 1024-float segment of its router
// row). Up to 64 such items: one work group of 1024 threads; more: one wave per item
// over many work groups, the last work group to finish (an arrival counter, which it
// resets) summing the segments in order. Either way the top-k is selected and the
// routing and x are handed to the host through the mailbox. scratch: device, >=
// route1_scratch_bytes(n, d), zero before the first call. row_src/row_dst as for
// launch_router.
size_t route1_scratch_bytes(int n, int d);
hipError_t launch_route1(const float *x, const float *wr, int d, int n, int k, int32_t *idx, float *w,
                         void *scratch, hipStream_t s, RouteMailbox *mbox, float *x_host, int32_t seq,
                         const int32_t *row_src, int32_t *row_dst);

// mbox/x_host (device addresses of host memory, nullable) are only used when T == 1.
// row_src (device address of host memory, nullable; T == 1 only): n int32 copied to
// row_dst by the kernel before it exits, i.e. before any later kernel on the stream.
hipError_t launch_router(const float *x, const float *wr, int T, int d, int n, int k,
                         int32_t *idx, float *w, hipStream_t s, RouteMailbox *mbox = nullptr,
                         float *x_host = nullptr, int32_t seq = 0, const int32_t *row_src = nullptr,
                         int32_t *row_dst = nullptr);
// gate/up/SiLU then down (split-K partials for the reduce).
hipError_t launch_ffn_stream(const FfnParams &p, hipStream_t s, const FfnEvents *ev);
// out = sum over active jobs of weight * sum of split partials (+ y_extra).
hipError_t launch_ffn_reduce(const FfnParams &p, const float *y_extra, float *out, hipStream_t s);
hipError_t launch_combine(const float *a, const float *b, const float *c, int d, float *out,
                          hipStream_t s);

// Prefill (grouped, MFMA).
struct PrefillPlan {
    int d, f, n, k, T;
    const float *wr;
    const uint8_t *pool;
    uint64_t slab_stride;
};
size_t prefill_workspace_bytes(int d, int f, int n, int k, int T);
hipError_t launch_prefill(const PrefillPlan &P, const float *X, float *OUT, int32_t *idx,
                          float *w, void *ws, hipStream_t s);

int device_cu_count();

}  // namespace moe
