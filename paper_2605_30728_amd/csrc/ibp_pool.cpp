// Persistent host worker pool of the runtime (host packing of gathers, large host copies).
//
// A PCIe gather call runs the pool once per staging chunk, so the time to start a run
// is on the critical path. Workers therefore spin on the generation counter for a short,
// time-bounded while after each run (a run then starts within about a microsecond) and
// only then sleep on a condition variable; the caller takes part in every run and waits
// for the workers to finish it.
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <mutex>
#include <thread>
#include <vector>

#include <immintrin.h>

#include "ibp_internal.hpp"

namespace ibp {

namespace {
// How long a worker spins for the next run before it sleeps: long enough to bridge the
// host work between the chunks of one call and between back-to-back calls, short enough
// not to take CPU time from the HIP runtime's own threads for long.
constexpr auto kSpin = std::chrono::microseconds(200);

// Spin until pred() holds or the spin time is over; returns pred().
template <class P>
bool spin_until(P pred) {
    const auto end = std::chrono::steady_clock::now() + kSpin;
    for (;;) {
        for (int i = 0; i < 64; ++i) {
            if (pred()) return true;
            _mm_pause();
        }
        if (std::chrono::steady_clock::now() >= end) return pred();
    }
}
}

struct Pool::State {
    std::vector<std::thread> workers;
    std::mutex mu;
    std::condition_variable cv;
    std::atomic<uint64_t> gen{0};
    std::atomic<uint64_t> next{0};
    std::atomic<int> pending{0};
    std::atomic<bool> stop{false};
    const std::function<void(uint64_t, uint64_t)> *fn = nullptr;
    uint64_t n = 0, block = 1;

    void work() {
        for (;;) {
            const uint64_t lo = next.fetch_add(block, std::memory_order_relaxed);
            if (lo >= n) break;
            (*fn)(lo, std::min(n, lo + block));
        }
    }

    void loop() {
        uint64_t seen = 0;
        for (;;) {
            spin_until([&] { return gen.load(std::memory_order_acquire) != seen; });
            uint64_t g = gen.load(std::memory_order_acquire);
            if (g == seen) {
                std::unique_lock<std::mutex> lk(mu);
                cv.wait(lk, [&] { return gen.load(std::memory_order_acquire) != seen; });
                g = gen.load(std::memory_order_acquire);
            }
            seen = g;
            if (stop.load(std::memory_order_acquire)) return;
            work();
            pending.fetch_sub(1, std::memory_order_acq_rel);
        }
    }
};

Pool::Pool(int threads) : st_(new State) {
    for (int i = 0; i < threads - 1; ++i) st_->workers.emplace_back([s = st_] { s->loop(); });
}

Pool::~Pool() {
    {
        std::lock_guard<std::mutex> g(st_->mu);
        st_->stop.store(true, std::memory_order_release);
        st_->gen.fetch_add(1, std::memory_order_acq_rel);
    }
    st_->cv.notify_all();
    for (auto &t : st_->workers) t.join();
    delete st_;
}

int Pool::size() const { return (int)st_->workers.size() + 1; }

void Pool::run(uint64_t n, uint64_t block, const std::function<void(uint64_t, uint64_t)> &fn) {
    if (n == 0) return;
    State &s = *st_;
    if (s.workers.empty() || n <= block) {
        fn(0, n);
        return;
    }
    // the previous run has fully ended (pending reached 0), so no worker reads these now
    s.fn = &fn;
    s.n = n;
    s.block = block;
    s.next.store(0, std::memory_order_relaxed);
    s.pending.store((int)s.workers.size(), std::memory_order_relaxed);
    {
        std::lock_guard<std::mutex> g(s.mu);
        s.gen.fetch_add(1, std::memory_order_acq_rel);
    }
    s.cv.notify_all();
    s.work();
    while (!spin_until([&] { return s.pending.load(std::memory_order_acquire) == 0; }))
        std::this_thread::yield();
    s.fn = nullptr;
}

}  // namespace ibp
