// A small persistent thread pool for the parameter server's SGD update (plain
// C++, no device code).
#pragma once

#include <condition_variable>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

namespace dc {

class HostPool {
  public:
    explicit HostPool(int threads);
    ~HostPool();
    // Run fn(i, n) for every i in [0, n) over the pool and the calling
    // thread; returns once every call has finished.  One caller at a time.
    void run(int n, const std::function<void(int, int)> &fn);
    int size() const { return (int)workers_.size() + 1; }

  private:
    void loop();
    std::vector<std::thread> workers_;
    std::mutex mu_;
    std::condition_variable cv_, done_cv_;
    const std::function<void(int, int)> *job_ = nullptr; // null between jobs
    int job_n_ = 0;
    int next_ = 0;    // next index of the current job to hand out
    int active_ = 0;  // workers inside the current job
    long gen_ = 0;    // job counter
    bool stop_ = false;
};

} // namespace dc
