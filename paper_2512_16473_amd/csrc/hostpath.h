// Host expert path: a persistent thread pool evaluating SwiGLU experts from
// bf16 weights held in host memory (the cache-miss path).
#pragma once

#include <condition_variable>
#include <cstdint>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

namespace moe {

class HostPool {
public:
    explicit HostPool(int n_threads);
    ~HostPool();
    int threads() const { return n_; }
    // Calls fn(tid, begin, end) on contiguous, near-equal ranges of [0, total),
    // one per thread (the caller is thread 0); returns when all are done.
    void parallel_for(int64_t total, const std::function<void(int, int64_t, int64_t)> &fn);
    // y = sum_j w[j] * FFN(slabs[j], x)
    void expert_ffn(const float *x, const void *const *slabs, const float *w, int ne, int d, int f, float *y);

private:
    void worker(int tid);
    int n_;
    std::vector<std::thread> th_;
    std::mutex mu_;
    std::condition_variable cv_go_, cv_done_;
    uint64_t gen_ = 0;
    int pending_ = 0;
    bool stop_ = false;
    int64_t total_ = 0;
    const std::function<void(int, int64_t, int64_t)> *fn_ = nullptr;
    std::vector<float> h_;   // [ne][f] activations, grown on demand
};

}  // namespace moe
