// Host thread pool that splits one large transfer between its threads: the
// host stage of the load pipeline (pageable blob -> pinned staging slot, or
// file -> pinned staging slot). Plain C++ so that it can be tested on its own
// under ThreadSanitizer.
#pragma once

#include <sys/uio.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <cerrno>
#include <condition_variable>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

namespace ii {

class CopyPool {
   public:
    explicit CopyPool(uint32_t n) : n_(n ? n : 1) {
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
    CopyPool(const CopyPool&) = delete;
    CopyPool& operator=(const CopyPool&) = delete;

    // Copies of at least this many bytes are split between the threads: one
    // thread copies about 10 GB/s, eight about 100 GB/s, so a chunk of a
    // few hundred KiB (the tail of a small model, a small chunk size) is
    // staged by all of them rather than by one.
    static constexpr uint64_t kSplitBytes = 256u << 10;

    // Copy len bytes from src to dst using every thread of the pool.
    void copy(void* dst, const void* src, uint64_t len) {
        uint8_t* d = static_cast<uint8_t*>(dst);
        const uint8_t* s = static_cast<const uint8_t*>(src);
        if (n_ <= 1 || len < kSplitBytes) {
            if (len) memcpy(d, s, len);
            return;
        }
        split(len, 4096, [d, s](uint64_t b, uint64_t e) { memcpy(d + (b), s + (b), e - b); });
    }

    // Write one byte in every 4 KiB page of [p, p + len) using every thread of
    // the pool. Pinned host memory is mapped for the CPU page by page on
    // first touch (about 3 GB/s for one thread, against about 30 GB/s once
    // mapped), so staging slots are touched when they are allocated rather
    // than during the first load.
    void touch(void* p, uint64_t len) {
        uint8_t* d = static_cast<uint8_t*>(p);
        auto piece = [d](uint64_t b, uint64_t e) {
            for (uint64_t x = b; x < e; x += 4096) reinterpret_cast<volatile uint8_t*>(d)[x] = 0;
        };
        if (n_ <= 1 || len < (4u << 20)) piece(0, len);
        else split(len, 4096, piece);
    }

    // Read file bytes [off, off + len) of fd into dst using every thread of
    // the pool; piece boundaries are multiples of `align` from off (so an
    // aligned request stays aligned for direct I/O). Only the first `need`
    // bytes must exist: a request rounded up past the end of the file may end
    // early there. Returns 0, or the errno of the first failing read (EIO if
    // the file ends before `need` bytes).
    int read(int fd, void* dst, uint64_t off, uint64_t len, uint64_t align, uint64_t need) {
        uint8_t* d = static_cast<uint8_t*>(dst);
        std::atomic<int> err{0};
        auto piece = [&](uint64_t b, uint64_t e) {
            while (b < e && !err.load(std::memory_order_relaxed)) {
                const ssize_t got = ::pread(fd, d + b, e - b, (off_t)(off + b));
                if (got < 0) {
                    if (errno == EINTR) continue;
                    err.store(errno ? errno : EIO);
                    return;
                }
                if (got == 0) {
                    if (b < need) err.store(EIO);  // end of file before the needed bytes
                    return;
                }
                b += (uint64_t)got;
            }
        };
        if (n_ <= 1 || len < (4u << 20)) piece(0, len);
        else split(len, std::max<uint64_t>(align, 4096), piece);
        return err.load();
    }

    // A gather: run r copies len[r] bytes from source offset off[r] to dst
    // + poff[r], where the runs tile [0, total) of dst in order (poff[0] = 0,
    // poff[r+1] = poff[r] + len[r]). src holds source offset `skew` at
    // src[0] (every off[r] >= skew). The threads split dst bytes evenly and
    // each finds its first run by binary search, so many small runs (rows of
    // a sharded tensor) spread like one large copy.
    void gather(uint8_t* dst, const uint8_t* src, int64_t skew, const uint32_t* off,
                const uint32_t* poff, const uint32_t* len, size_t nruns, uint64_t total) {
        if (!nruns) return;
        auto piece = [=](uint64_t b, uint64_t e) {
            size_t r = (size_t)(std::upper_bound(poff, poff + nruns, (uint32_t)b) - poff) - 1;
            for (; r < nruns && poff[r] < e; ++r) {
                const uint64_t rb = std::max<uint64_t>(b, poff[r]);
                const uint64_t re = std::min<uint64_t>(e, (uint64_t)poff[r] + len[r]);
                const uint64_t at = (uint64_t)((int64_t)off[r] - skew) + (rb - poff[r]);
                if (re > rb) memcpy(dst + rb, src + at, re - rb);
            }
        };
        if (n_ <= 1 || total < (4u << 20)) piece(0, total);
        else split(total, 64, piece);
    }

    // The same gather with the source in a file: run r reads file bytes
    // [base + off[r], +len[r]) into dst + poff[r] (buffered reads). Runs are
    // in file order; each thread reads its share of them in batches, one
    // preadv per batch: the file range from a batch's first run to its last,
    // run bytes going to their place in dst and the gaps between runs (at
    // most kMaxGap bytes each) to a scratch buffer, so that thousands of
    // short rows cost a few system calls rather than one each. Returns 0 or
    // the errno of the first failing read (EIO at end of file).
    static constexpr uint64_t kMaxGap = 256u << 10;  // larger gaps end a batch
    static constexpr int kMaxIov = 1024;              // iovecs per preadv (IOV_MAX)
    int read_gather(int fd, uint8_t* dst, uint64_t base, const uint32_t* off,
                    const uint32_t* poff, const uint32_t* len, size_t nruns, uint64_t total) {
        if (!nruns) return 0;
        std::atomic<int> err{0};
        auto piece = [&](uint64_t b, uint64_t e) {
            std::vector<uint8_t> gap_buf;
            std::vector<iovec> iov;
            iov.reserve(kMaxIov);
            size_t r = (size_t)(std::upper_bound(poff, poff + nruns, (uint32_t)b) - poff) - 1;
            while (r < nruns && poff[r] < e && !err.load(std::memory_order_relaxed)) {
                // a batch: run r from dst byte rb (the piece may start inside
                // it), then following runs while their gaps are small
                iov.clear();
                const uint64_t rb = std::max<uint64_t>(b, poff[r]);
                const uint64_t re = std::min<uint64_t>(e, (uint64_t)poff[r] + len[r]);
                const uint64_t start = base + off[r] + (rb - poff[r]);  // file offset
                iov.push_back(iovec{dst + rb, (size_t)(re - rb)});
                uint64_t fend = start + (re - rb);
                for (++r; r < nruns && poff[r] < e && (int)iov.size() + 2 <= kMaxIov; ++r) {
                    const uint64_t at = base + off[r], gap = at - fend;
                    if (gap > kMaxGap) break;
                    const uint64_t n = std::min<uint64_t>(e, (uint64_t)poff[r] + len[r]) - poff[r];
                    if (gap) {
                        if (gap_buf.size() < gap) gap_buf.resize(kMaxGap);
                        iov.push_back(iovec{gap_buf.data(), (size_t)gap});
                    }
                    iov.push_back(iovec{dst + poff[r], (size_t)n});
                    fend = at + n;
                }
                // read [start, fend) into the batch, resuming after short reads
                iovec* v = iov.data();
                int nv = (int)iov.size();
                uint64_t pos = start;
                while (pos < fend) {
                    const ssize_t got = ::preadv(fd, v, nv, (off_t)pos);
                    if (got < 0) {
                        if (errno == EINTR) continue;
                        err.store(errno ? errno : EIO);
                        return;
                    }
                    if (got == 0) {
                        err.store(EIO);
                        return;
                    }
                    pos += (uint64_t)got;
                    for (size_t g = (size_t)got; g;) {  // drop what was filled
                        if (g >= v->iov_len) {
                            g -= v->iov_len;
                            ++v;
                            --nv;
                        } else {
                            v->iov_base = static_cast<uint8_t*>(v->iov_base) + g;
                            v->iov_len -= g;
                            g = 0;
                        }
                    }
                }
            }
        };
        if (n_ <= 1 || total < (4u << 20)) piece(0, total);
        else split(total, 64, piece);
        return err.load();
    }

   private:
    // Run fn over [0, len) cut into one piece per thread, pieces aligned to
    // `align`; the calling thread takes piece 0.
    void split(uint64_t len, uint64_t align, const std::function<void(uint64_t, uint64_t)>& fn) {
        {
            std::lock_guard<std::mutex> g(m_);
            fn_ = &fn;
            len_ = len;
            align_ = align;
            pending_ = n_ - 1;
            ++gen_;
        }
        cv_.notify_all();
        part(0);
        std::unique_lock<std::mutex> l(m_);
        done_.wait(l, [this] { return pending_ == 0; });
        fn_ = nullptr;
    }
    void part(uint32_t i) {
        const uint64_t per = ((len_ + n_ - 1) / n_ + align_ - 1) / align_ * align_;
        const uint64_t b = std::min(len_, (uint64_t)i * per), e = std::min(len_, b + per);
        if (e > b) (*fn_)(b, e);
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
    const std::function<void(uint64_t, uint64_t)>* fn_ = nullptr;
    uint64_t len_ = 0, align_ = 4096;
};

}  // namespace ii

namespace ii {

// Read-ahead for direct-I/O files: R reader threads, each owning one
// page-aligned buffer; thread j reads chunks j, j + R, j + 2R, ... in turn,
// each as one block-aligned range, and refills its buffer as soon as the
// consumer has released the chunk in it. The consumer takes chunks in order
// with wait(k) / release(k). R whole-chunk reads stay in flight, which keeps a
// storage device's queue full the way a plain parallel reader does.
class ReadAhead {
   public:
    struct Range {
        uint64_t begin, end, need;  // file bytes to read; bytes that must exist
    };
    ReadAhead(int fd, uint32_t nthreads, uint64_t buf_bytes, uint32_t nchunks,
              std::function<Range(uint32_t)> range_of)
        : fd_(fd), n_(nthreads ? nthreads : 1), nchunks_(nchunks), range_of_(std::move(range_of)) {
        slots_.resize(n_);
        for (uint32_t j = 0; j < n_; ++j) {
            slots_[j].buf = static_cast<uint8_t*>(aligned_alloc(4096, (buf_bytes + 4095) & ~4095ull));
            if (!slots_[j].buf) alloc_failed_ = true;
        }
        if (!alloc_failed_)
            for (uint32_t j = 0; j < n_ && j < nchunks_; ++j)
                threads_.emplace_back([this, j] { reader(j); });
    }
    ~ReadAhead() {
        {
            std::lock_guard<std::mutex> g(m_);
            stop_ = true;
        }
        cv_.notify_all();
        for (auto& t : threads_) t.join();
        for (auto& s : slots_) free(s.buf);
    }
    ReadAhead(const ReadAhead&) = delete;
    ReadAhead& operator=(const ReadAhead&) = delete;

    bool ok() const { return !alloc_failed_; }

    // Wait until chunk k is in memory; returns its buffer (file byte
    // range_of(k).begin at offset 0), or nullptr with *err set.
    const uint8_t* wait(uint32_t k, int* err) {
        Slot& s = slots_[k % n_];
        std::unique_lock<std::mutex> l(m_);
        cv_.wait(l, [&] { return s.ready == (int64_t)k || s.err; });
        if (s.err) {
            *err = s.err;
            return nullptr;
        }
        *err = 0;
        return s.buf;
    }
    // The consumer is done with chunk k's buffer.
    void release(uint32_t k) {
        {
            std::lock_guard<std::mutex> g(m_);
            slots_[k % n_].released = (int64_t)k;
        }
        cv_.notify_all();
    }

   private:
    struct Slot {
        uint8_t* buf = nullptr;
        int64_t ready = -1;     // chunk whose bytes the buffer holds
        int64_t released = -1;  // last chunk the consumer gave back
        int err = 0;
    };
    void reader(uint32_t j) {
        Slot& s = slots_[j];
        for (uint64_t k = j; k < nchunks_; k += n_) {
            if (k >= n_) {  // the buffer still holds chunk k - n_ until it is released
                std::unique_lock<std::mutex> l(m_);
                cv_.wait(l, [&] { return stop_ || s.released == (int64_t)(k - n_); });
                if (stop_) return;
            }
            const Range r = range_of_((uint32_t)k);
            int e = 0;
            uint64_t b = 0;
            while (b < r.end - r.begin) {
                const ssize_t got =
                    ::pread(fd_, s.buf + b, r.end - r.begin - b, (off_t)(r.begin + b));
                if (got < 0) {
                    if (errno == EINTR) continue;
                    e = errno ? errno : EIO;
                    break;
                }
                if (got == 0) {
                    if (b < r.need) e = EIO;
                    break;
                }
                b += (uint64_t)got;
            }
            {
                std::lock_guard<std::mutex> g(m_);
                if (e) s.err = e;
                else s.ready = (int64_t)k;
            }
            cv_.notify_all();
            if (e) return;
        }
    }
    int fd_;
    uint32_t n_, nchunks_;
    std::function<Range(uint32_t)> range_of_;
    std::vector<Slot> slots_;
    std::vector<std::thread> threads_;
    std::mutex m_;
    std::condition_variable cv_;
    bool stop_ = false;
    bool alloc_failed_ = false;
};

}  // namespace ii
