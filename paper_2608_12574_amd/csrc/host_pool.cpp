// Host worker threads for the parallel loops of the host build.
//
// Creating and joining 16 threads costs about 0.2 ms on the MI355X host, and a
// compile runs several parallel loops (a cold one, with the vocabulary tables,
// a dozen), so the workers are created once, at the first loop, and then wait
// for work.  After a loop a worker keeps checking for the next one for about
// 20 microseconds (a compile's loops follow one another closely) and then
// sleeps on a condition variable.
//
// One loop runs on the pool at a time.  A loop started while another runs (a
// compile on another host thread) gets threads of its own, as before the pool
// existed; a loop started from inside a loop runs on the calling thread.  A
// forked child starts a pool of its own (the parent's workers do not exist
// there).  A pool is never destroyed: its workers sleep until the process ends.
#include <pthread.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <exception>
#include <mutex>
#include <system_error>
#include <thread>
#include <vector>

#include "host_build.hpp"

namespace tam {

namespace {

thread_local bool t_in_loop = false;

struct Pool {
    int workers = 0;
    std::mutex busy;  // held by the caller of the loop that runs on the pool

    // The current loop.  The caller writes f, n, next, finished and error under
    // m, then hands out `tickets`: a worker joins the loop by taking a ticket
    // (decrementing a positive count), which also makes the loop's state
    // visible to it.  At the end the caller takes back the tickets left and
    // waits until every worker that joined has finished.
    std::mutex m;
    std::condition_variable wake, done;
    std::atomic<uint64_t> generation{0};
    std::atomic<int> tickets{0};
    const std::function<void(int64_t)> *f = nullptr;
    int64_t n = 0;
    std::atomic<int64_t> next{0};
    int finished = 0;
    std::exception_ptr error;

    // items of the current loop until none is left; the first exception is kept
    void work() {
        const std::function<void(int64_t)> &fn = *f;
        for (int64_t j = next.fetch_add(1); j < n; j = next.fetch_add(1)) {
            try {
                fn(j);
            } catch (...) {
                std::lock_guard<std::mutex> g(m);
                if (!error) error = std::current_exception();
                next.store(n);  // skip what is left
            }
        }
    }

    bool take_ticket() {
        int t = tickets.load();
        while (t > 0 && !tickets.compare_exchange_weak(t, t - 1)) {
        }
        return t > 0;
    }

    void worker() {
        t_in_loop = true;
        uint64_t seen = generation.load();
        for (;;) {
            const auto t0 = std::chrono::steady_clock::now();
            while (generation.load() == seen &&
                   std::chrono::steady_clock::now() - t0 < std::chrono::microseconds(20))
                __builtin_ia32_pause();
            if (generation.load() == seen) {
                std::unique_lock<std::mutex> lk(m);
                wake.wait(lk, [&] { return generation.load() != seen; });
            }
            seen = generation.load();
            if (!take_ticket()) continue;
            work();
            std::lock_guard<std::mutex> g(m);
            ++finished;
            done.notify_all();
        }
    }
};

Pool *g_pool = nullptr;
std::once_flag g_pool_once;

void fresh_pool_in_child() { g_pool = new Pool(); }  // the parent's pool is left as it was

Pool &pool() {
    std::call_once(g_pool_once, [] {
        g_pool = new Pool();
        pthread_atfork(nullptr, nullptr, fresh_pool_in_child);
    });
    return *g_pool;
}

// Threads of its own for one loop (the pool is busy).
void spawn_loop(int64_t n, int threads, const std::function<void(int64_t)> &f) {
    std::atomic<int64_t> next{0};
    std::exception_ptr error;
    std::mutex em;
    auto body = [&] {
        for (int64_t j = next.fetch_add(1); j < n; j = next.fetch_add(1)) {
            try {
                f(j);
            } catch (...) {
                std::lock_guard<std::mutex> g(em);
                if (!error) error = std::current_exception();
                next.store(n);
            }
        }
    };
    std::vector<std::thread> ts;
    try {
        for (int i = 1; i < threads; ++i)
            ts.emplace_back([&] {
                t_in_loop = true;
                body();
            });
    } catch (const std::system_error &) {  // no more threads: the ones made share the loop
    }
    t_in_loop = true;
    body();
    t_in_loop = false;
    for (auto &t : ts) t.join();
    if (error) std::rethrow_exception(error);
}

}  // namespace

void host_parallel_for(int64_t n, int threads, const std::function<void(int64_t)> &f) {
    if (threads <= 1 || n <= 1 || t_in_loop) {
        for (int64_t j = 0; j < n; ++j) f(j);
        return;
    }
    Pool &P = pool();
    std::unique_lock<std::mutex> busy(P.busy, std::try_to_lock);
    if (!busy.owns_lock()) {
        spawn_loop(n, threads, f);
        return;
    }
    try {
        while (P.workers < threads - 1) {
            std::thread([&P] { P.worker(); }).detach();
            ++P.workers;
        }
    } catch (const std::system_error &) {  // no more threads: the workers made share the loop
    }
    const int helpers = std::min(threads - 1, P.workers);
    {
        std::lock_guard<std::mutex> g(P.m);
        P.f = &f;
        P.n = n;
        P.next.store(0);
        P.finished = 0;
        P.error = nullptr;
        P.tickets.store(helpers);
        P.generation.fetch_add(1);
        P.wake.notify_all();
    }
    t_in_loop = true;
    P.work();
    t_in_loop = false;
    const int joined = helpers - P.tickets.exchange(0);
    std::exception_ptr err;
    {
        std::unique_lock<std::mutex> lk(P.m);
        P.done.wait(lk, [&] { return P.finished == joined; });
        err = P.error;
        P.error = nullptr;
        P.f = nullptr;
    }
    if (err) std::rethrow_exception(err);
}

}  // namespace tam
