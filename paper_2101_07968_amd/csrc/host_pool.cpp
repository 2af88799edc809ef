// HostPool: see host_pool.h.  A worker joins a job only while that job is
// still published (job_ non-null under the lock) and takes indices only
// while the job counter still names it, so a worker that wakes late never
// runs a finished job nor mixes one job's count with the next job's indices.
#include "host_pool.h"

namespace dc {

HostPool::HostPool(int threads) {
    for (int i = 1; i < threads; ++i)
        workers_.emplace_back([this] { loop(); });
}

HostPool::~HostPool() {
    {
        std::lock_guard<std::mutex> g(mu_);
        stop_ = true;
    }
    cv_.notify_all();
    for (auto &t : workers_)
        t.join();
}

void HostPool::loop() {
    long seen = 0;
    for (;;) {
        const std::function<void(int, int)> *job;
        int n;
        long gen;
        {
            std::unique_lock<std::mutex> lk(mu_);
            cv_.wait(lk, [&] { return stop_ || gen_ != seen; });
            if (stop_)
                return;
            seen = gen = gen_;
            job = job_;
            n = job_n_;
            if (!job)
                continue; // woke after that job had finished
            ++active_;
        }
        for (;;) {
            int i;
            {
                std::lock_guard<std::mutex> g(mu_);
                i = (gen_ == gen && next_ < n) ? next_++ : -1;
            }
            if (i < 0)
                break;
            (*job)(i, n);
        }
        {
            std::lock_guard<std::mutex> g(mu_);
            --active_;
        }
        done_cv_.notify_all();
    }
}

void HostPool::run(int n, const std::function<void(int, int)> &fn) {
    if (workers_.empty() || n <= 1) {
        for (int i = 0; i < n; ++i)
            fn(i, n);
        return;
    }
    long gen;
    {
        std::lock_guard<std::mutex> g(mu_);
        job_ = &fn;
        job_n_ = n;
        next_ = 0;
        gen = ++gen_;
    }
    cv_.notify_all();
    for (;;) {
        int i;
        {
            std::lock_guard<std::mutex> g(mu_);
            i = next_ < n ? next_++ : -1;
        }
        if (i < 0)
            break;
        fn(i, n);
    }
    std::unique_lock<std::mutex> lk(mu_);
    done_cv_.wait(lk, [&] { return active_ == 0 && next_ >= n; });
    // unpublish before returning: fn dies with the caller's frame
    job_ = nullptr;
    (void)gen;
}

} // namespace dc
