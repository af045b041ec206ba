// Host thread pool that splits one large memcpy between its threads: the
// host stage of the load pipeline (pageable blob -> pinned staging slot).
// Plain C++ so that it can be tested on its own under ThreadSanitizer.
#pragma once

#include <algorithm>
#include <condition_variable>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <thread>
#include <vector>

namespace ii {

// Fixed set of host threads that split one large memcpy between them.
class CopyPool {
   public:
    explicit CopyPool(uint32_t n) : n_(n) {
        for (uint32_t i = 1; i < n_; ++i) threads_.emplace_back([this, i] { worker(i); });
    }
    ~CopyPool() {
        {
            std::lock_guard<std::mutex> g(m_);
            stop_ = true;
        }
        cv_.notify_all();
        for (auto& t : threads_) t.join();
    }
    // Copy len bytes from src to dst using every thread of the pool.
    void copy(void* dst, const void* src, uint64_t len) {
        if (n_ <= 1 || len < (4u << 20)) {
            memcpy(dst, src, len);
            return;
        }
        {
            std::lock_guard<std::mutex> g(m_);
            dst_ = static_cast<uint8_t*>(dst);
            src_ = static_cast<const uint8_t*>(src);
            len_ = len;
            pending_ = n_ - 1;
            ++gen_;
        }
        cv_.notify_all();
        part(0);
        std::unique_lock<std::mutex> l(m_);
        done_.wait(l, [this] { return pending_ == 0; });
    }

   private:
    void part(uint32_t i) {
        const uint64_t per = ((len_ + n_ - 1) / n_ + 4095) & ~4095ull;
        const uint64_t b = std::min(len_, (uint64_t)i * per), e = std::min(len_, b + per);
        if (e > b) memcpy(dst_ + b, src_ + b, e - b);
    }
    void worker(uint32_t i) {
        uint64_t seen = 0;
        for (;;) {
            {
                std::unique_lock<std::mutex> l(m_);
                cv_.wait(l, [&] { return stop_ || gen_ != seen; });
                if (stop_) return;
                seen = gen_;
            }
            part(i);
            {
                std::lock_guard<std::mutex> g(m_);
                if (--pending_ == 0) done_.notify_one();
            }
        }
    }
    uint32_t n_;
    std::vector<std::thread> threads_;
    std::mutex m_;
    std::condition_variable cv_, done_;
    bool stop_ = false;
    uint64_t gen_ = 0;
    uint32_t pending_ = 0;
    uint8_t* dst_ = nullptr;
    const uint8_t* src_ = nullptr;
    uint64_t len_ = 0;
};

}  // namespace ii
