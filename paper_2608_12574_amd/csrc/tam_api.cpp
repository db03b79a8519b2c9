// The C ABI of libtam (declared in include/tam.h).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cstring>
#include <exception>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <unordered_map>
#include <vector>

#include "host_build.hpp"
#include "tam_internal.hpp"
#include "trie_layout.hpp"

namespace tam {

namespace {

struct PinnedPool {
    std::mutex m;
    std::multimap<size_t, void *> idle;        // blocks ready for reuse, by size
    std::unordered_map<void *, size_t> owned;  // every block of the pool and its size
    size_t idle_bytes = 0;
};

// Never destroyed: blocks may come back from handles destroyed at exit.
PinnedPool &pinned_pool() {
    static PinnedPool *p = new PinnedPool();
    return *p;
}

thread_local bool t_pinned = false;
constexpr size_t kPinnedKeep = size_t(4) << 30;  // idle bytes kept for reuse

}  // namespace

void *pinned_take(size_t bytes) {
    if (!t_pinned || bytes < kPinnedMin) return nullptr;
    const size_t want = (bytes + kPinnedMin - 1) / kPinnedMin * kPinnedMin;
    PinnedPool &P = pinned_pool();
    {
        std::lock_guard<std::mutex> g(P.m);
        auto it = P.idle.lower_bound(want);
        if (it != P.idle.end() && it->first <= want + want / 4) {  // at most 25% larger
            void *p = it->second;
            P.idle_bytes -= it->first;
            P.idle.erase(it);
            return p;
        }
    }
    void *p = nullptr;
    if (hipHostMalloc(&p, want, hipHostMallocPortable) != hipSuccess || !p) {
        (void)hipGetLastError();
        return nullptr;
    }
    std::lock_guard<std::mutex> g(P.m);
    P.owned[p] = want;
    return p;
}

bool pinned_give(void *p) {
    PinnedPool &P = pinned_pool();
    std::lock_guard<std::mutex> g(P.m);
    auto it = P.owned.find(p);
    if (it == P.owned.end()) return false;
    const size_t size = it->second;
    if (P.idle_bytes + size > kPinnedKeep) {
        P.owned.erase(it);
        (void)hipHostFree(p);
        return true;
    }
    P.idle.emplace(size, p);
    P.idle_bytes += size;
    return true;
}

PinnedScope::PinnedScope(bool on) : prev(t_pinned) { t_pinned = on; }
PinnedScope::~PinnedScope() { t_pinned = prev; }

namespace {

constexpr int kErrSlots = 4096;

struct ErrSlots {
    std::mutex m;
    int32_t *base = nullptr;
    std::vector<int> free_slots;
    bool tried = false;
};

// Never destroyed: handles destroyed at exit hand their slots back.
ErrSlots &err_slots() {
    static ErrSlots *p = new ErrSlots();
    return *p;
}

}  // namespace

int32_t *err_slot_take() {
    ErrSlots &E = err_slots();
    std::lock_guard<std::mutex> g(E.m);
    if (!E.tried) {
        E.tried = true;
        void *p = nullptr;
        if (hipHostMalloc(&p, kErrSlots * sizeof(int32_t), hipHostMallocPortable) == hipSuccess && p) {
            E.base = static_cast<int32_t *>(p);
            for (int i = kErrSlots - 1; i >= 0; --i) E.free_slots.push_back(i);
        } else {
            (void)hipGetLastError();
        }
    }
    if (E.free_slots.empty()) return nullptr;
    int32_t *slot = E.base + E.free_slots.back();
    E.free_slots.pop_back();
    *slot = 0;
    return slot;
}

void err_slot_give(int32_t *slot) {
    if (!slot) return;
    ErrSlots &E = err_slots();
    std::lock_guard<std::mutex> g(E.m);
    E.free_slots.push_back((int)(slot - E.base));
}

}  // namespace tam

namespace {

thread_local std::string g_err;

tam_status fail(tam_status st, const std::string &msg) {
    g_err = msg;
    return st;
}

tam_status hip_fail(hipError_t e, const char *what) {
    return fail(TAM_E_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

#define TAM_HIP(expr)                                      \
    do {                                                   \
        const hipError_t e_ = (expr);                      \
        if (e_ != hipSuccess) return hip_fail(e_, #expr);  \
    } while (0)

double ms_since(std::chrono::steady_clock::time_point t0) {
    return std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
}

bool csr_ok(const int64_t *off, int64_t n) {
    if (!off || off[0] != 0) return false;
    for (int64_t i = 0; i < n; ++i)
        if (off[i + 1] < off[i]) return false;
    return true;
}

void *alloc_with(bool own, const tam_allocator &a, size_t bytes) {
    bytes = std::max<size_t>(bytes, 256);
    void *p = nullptr;
    if (own) {
        if (hipMalloc(&p, bytes) != hipSuccess) return nullptr;
    } else {
        p = a.alloc(bytes, a.ctx);
    }
    return p;
}

void free_with(bool own, const tam_allocator &a, void *p) {
    if (!p) return;
    if (own)
        (void)hipFree(p);
    else
        a.free(p, a.ctx);
}

// Sub-allocation of small tables inside one device arena.
struct Arena {
    size_t used = 0;
    template <typename T>
    size_t take(int64_t count) {
        const size_t at = used;
        used += ((size_t)std::max<int64_t>(count, 1) * sizeof(T) + 255) & ~size_t(255);
        return at;
    }
};

// ------------------------------------------------------------- vocabulary --

void vocab_release(tam_vocab *v) {
    if (!v) return;
    if (v->refs.fetch_sub(1) != 1) return;
    if (v->ready) {
        (void)hipEventSynchronize(v->ready);
        (void)hipEventDestroy(v->ready);
    }
    free_with(v->own_alloc, v->alloc, v->arena);
    delete v;
}

tam_status vocab_create(const uint8_t *tok_bytes, const int64_t *tok_off, int64_t V, uint32_t flags,
                        const tam_allocator *alloc, hipStream_t s, tam_vocab **out) {
    *out = nullptr;
    if (V <= 0) return fail(TAM_E_INVAL, "V must be >= 1");
    if (V >= INT32_MAX) return fail(TAM_E_TOOLARGE, "V must be < 2^31-1");
    if (!csr_ok(tok_off, V)) return fail(TAM_E_INVAL, "tok_off must start at 0 and be non-decreasing");
    if (!tok_bytes && tok_off[V] > 0) return fail(TAM_E_INVAL, "tok_bytes is null");
    if (alloc && (!alloc->alloc || !alloc->free)) return fail(TAM_E_INVAL, "allocator callbacks are null");
    tam_vocab *v = new (std::nothrow) tam_vocab();
    if (!v) return fail(TAM_E_NOMEM, "out of host memory");
    v->flags = flags & TAM_FLAG_HOST_ONLY;
    std::string err;
    tam_status st;
    const auto t0 = std::chrono::steady_clock::now();
    try {
        const tam::PinnedScope pinned(!(v->flags & TAM_FLAG_HOST_ONLY));  // uploaded tables: pinned blocks
        st = tam::build_vocab(tok_bytes, tok_off, V, v, &err);
    } catch (const std::bad_alloc &) {
        st = TAM_E_NOMEM;
        err = "out of host memory";
    } catch (const std::exception &x) {  // e.g. no host thread could be made
        st = TAM_E_NOMEM;
        err = std::string("host build failed: ") + x.what();
    }
    v->host_ms = ms_since(t0);
    if (st != TAM_OK) {
        delete v;
        return fail(st, err);
    }
    if (v->flags & TAM_FLAG_HOST_ONLY) {
        *out = v;
        return TAM_OK;
    }
    const auto t1 = std::chrono::steady_clock::now();
    (void)hipGetLastError();
    if (hipGetDevice(&v->device) != hipSuccess) {
        delete v;
        return fail(TAM_E_DEVICE, "no HIP device");
    }
    v->own_alloc = alloc == nullptr;
    if (alloc) v->alloc = *alloc;
    Arena a;
    const size_t o_off = a.take<uint32_t>(V + 1);
    const size_t o_blob = a.take<uint8_t>((int64_t)v->tok_blob.size());
    const size_t o_fps = a.take<uint16_t>((int64_t)v->fps.size());
    const size_t o_pay = a.take<tam::SlotPay>((int64_t)v->pay.size());
    const size_t o_pay_hi = a.take<uint64_t>((int64_t)v->pay_hi.size());
    const size_t o_short = a.take<int32_t>((int64_t)v->short_hits.size());
    const size_t o_dup = a.take<int32_t>(V);
    const size_t o_len = a.take<uint8_t>((int64_t)v->len_present.size());
    uint8_t *base = static_cast<uint8_t *>(alloc_with(v->own_alloc, v->alloc, a.used));
    if (!base) {
        delete v;
        return fail(TAM_E_NOMEM, "device allocation failed (" + std::to_string(a.used) + " bytes requested)");
    }
    v->arena = base;
    v->device_bytes = (int64_t)a.used;
    v->d_tok_off = reinterpret_cast<const uint32_t *>(base + o_off);
    v->d_tok_blob = base + o_blob;
    v->d_fps = reinterpret_cast<const uint16_t *>(base + o_fps);
    v->d_pay = reinterpret_cast<const tam::SlotPay *>(base + o_pay);
    v->d_pay_hi = reinterpret_cast<const uint64_t *>(base + o_pay_hi);
    v->d_short_hits = reinterpret_cast<const int32_t *>(base + o_short);
    v->d_dup_next = reinterpret_cast<const int32_t *>(base + o_dup);
    v->d_len_present = base + o_len;
    auto up = [&](size_t off, const void *src, size_t bytes) -> hipError_t {
        if (bytes == 0) return hipSuccess;
        return hipMemcpyAsync(base + off, src, bytes, hipMemcpyHostToDevice, s);
    };
    hipError_t e = up(o_off, v->tok_off.data(), v->tok_off.size() * 4);
    if (e == hipSuccess) e = up(o_blob, v->tok_blob.data(), v->tok_blob.size());
    if (e == hipSuccess) e = up(o_fps, v->fps.data(), v->fps.size() * sizeof(uint16_t));
    if (e == hipSuccess) e = up(o_pay, v->pay.data(), v->pay.size() * sizeof(tam::SlotPay));
    if (e == hipSuccess) e = up(o_pay_hi, v->pay_hi.data(), v->pay_hi.size() * sizeof(uint64_t));
    if (e == hipSuccess) e = up(o_short, v->short_hits.data(), v->short_hits.size() * sizeof(int32_t));
    if (e == hipSuccess) e = up(o_dup, v->dup_next.data(), v->dup_next.size() * 4);
    if (e == hipSuccess) e = up(o_len, v->len_present.data(), v->len_present.size());
    if (e == hipSuccess) e = hipEventCreateWithFlags(&v->ready, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventRecord(v->ready, s);
    v->upload_ms = ms_since(t1);
    if (e != hipSuccess) {
        st = hip_fail(e, "vocabulary upload");
        const std::string msg = g_err;
        (void)hipStreamSynchronize(s);  // copies already enqueued still read the host tables
        vocab_release(v);
        return fail(st, msg);
    }
    *out = v;
    return TAM_OK;
}

// ------------------------------------------------------------------ handle --

void *dev_alloc(tam_handle *h, size_t bytes) {
    void *p = alloc_with(h->own_alloc, h->alloc, bytes);
    if (p) h->dev_ptrs.push_back(p);
    return p;
}

void release_device(tam_handle *h) {
    if (h->work_done) (void)hipEventSynchronize(h->work_done);
    if (h->have_events) (void)hipEventSynchronize(h->ev[3]);
    for (void *p : h->dev_ptrs) free_with(h->own_alloc, h->alloc, p);
    h->dev_ptrs.clear();
    tam::err_slot_give(h->h_err);  // its last copy is behind work_done
    h->h_err = nullptr;
    h->d_err = nullptr;
    if (h->have_events)
        for (hipEvent_t &e : h->ev) (void)hipEventDestroy(e);
    if (h->work_done) (void)hipEventDestroy(h->work_done);
    h->have_events = false;
    h->work_done = nullptr;
}

// The phase events of TAM_FLAG_TIMING (created once).
hipError_t create_events(tam_handle *h) {
    if (h->have_events) return hipSuccess;
    hipError_t e = hipSuccess;
    for (hipEvent_t &ev : h->ev)
        if (e == hipSuccess) e = hipEventCreate(&ev);
    h->have_events = e == hipSuccess;
    return e;
}

void destroy_handle(tam_handle *h) {
    if (!(h->flags & TAM_FLAG_HOST_ONLY)) release_device(h);
    vocab_release(h->vocab);
    delete h;
}

// The handle keeps valid lists (all nodes without a table; with tail
// compression the tails' tokens longer than the probe window, if the vocabulary
// has any) and/or a dense table.
bool is_lazy(const tam_handle *h) { return (h->flags & TAM_FLAG_LAZY_ROWS) != 0 && h->fmt_L < 0; }

bool keeps_lists(const tam_handle *h) { return !is_lazy(h) && (!h->dt.table || h->dt.tail_long); }

unsigned default_phases(const tam_handle *h) {
    if (is_lazy(h)) return 0;                  // the cache is emptied; no rows are built
    if (h->fmt_L >= 0) return TAM_PHASE_MARK;  // k_format writes every word: no zero fill
    return (keeps_lists(h) ? unsigned(TAM_PHASE_LISTS) : 0u) | (h->dt.table ? unsigned(TAM_PHASE_TABLE) : 0u);
}

// The handle's device error count into its pinned host word (not under
// stream capture: a graph carries kernels only).
hipError_t copy_errors(const tam_handle *h, hipStream_t s, bool capturing) {
    if (!h->h_err || !h->d_err || capturing) return hipSuccess;
    return hipMemcpyAsync(h->h_err, h->d_err, sizeof(int32_t), hipMemcpyDeviceToHost, s);
}

// TAM_E_DEVICE once a copied-back count shows that the device met
// inconsistent table entries (the host build never makes them).
tam_status device_errors(const tam_handle *h) {
    const int32_t n = h->h_err ? __atomic_load_n(h->h_err, __ATOMIC_ACQUIRE) : 0;
    if (n == 0) return TAM_OK;
    return fail(TAM_E_DEVICE, "the device met " + std::to_string(n) +
                                  " inconsistent trie-table entries or cache states; results of this handle are "
                                  "not valid");
}

// The device view of one group of the probe pass under tail lists: its record
// buffer, and its blocks' region offsets and record counts.
// The device part of compile, on the caller's stream: zero fill of the table,
// the probe pass (marks into the table, counts for the lists), then the lists'
// prefix sum and fill.  Phase events are recorded only for the handle's
// default phases.
// zero_enqueued: the table's zero fill was already enqueued on `s`, with its
// events (compile starts it while the host writes the trie).
tam_status run_device_phase(tam_handle *h, unsigned phases, hipStream_t s, bool zero_enqueued = false,
                            bool lists_counted = false) {
    const tam::DevTables &t = h->dt;
    // Under stream capture (a HIP graph) only the kernels are recorded: no
    // events, which belong to eager calls.
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    TAM_HIP(hipStreamIsCapturing(s, &cap));
    const bool capturing = cap != hipStreamCaptureStatusNone;
    const unsigned counted = phases | (zero_enqueued ? unsigned(TAM_PHASE_ZERO) : 0u);
    const bool timing = h->have_events && counted == default_phases(h) && !capturing;
    if (is_lazy(h)) {  // rows built on demand: only the cache is reset
        if (timing) TAM_HIP(hipEventRecord(h->ev[0], s));
        TAM_HIP(tam::launch_lazy_reset(t, h->lazy, s));
        if (timing) {
            TAM_HIP(hipEventRecord(h->ev[1], s));
            TAM_HIP(hipEventRecord(h->ev[2], s));
            TAM_HIP(hipEventRecord(h->ev[3], s));
            h->events_recorded = true;
        }
        TAM_HIP(copy_errors(h, s, capturing));
        if (h->work_done && !capturing) TAM_HIP(hipEventRecord(h->work_done, s));
        return TAM_OK;
    }
    const bool lists = (phases & TAM_PHASE_LISTS) != 0;
    const bool count_only = !lists && (phases & TAM_PHASE_COUNT) != 0;  // the probe pass of the lists alone
    const bool zero = (phases & TAM_PHASE_ZERO) && t.table && !zero_enqueued;
    const bool mark = (phases & TAM_PHASE_MARK) && t.table;
    // lists_counted: the list counts were made group by group while the host
    // wrote the trie (events 0, 1, 4 and 2 recorded then)
    if (!lists_counted) {
        if (timing && !zero_enqueued) TAM_HIP(hipEventRecord(h->ev[0], s));
        if (zero) TAM_HIP(tam::launch_zero(t.table, t.R * t.Wp, s));
        if (timing && !zero_enqueued) TAM_HIP(hipEventRecord(h->ev[1], s));
        if (timing && zero_enqueued) TAM_HIP(hipEventRecord(h->ev[4], s));  // the probe's own start
        if (timing) h->mark_from_ev4 = zero_enqueued;
        if (lists || count_only) TAM_HIP(tam::launch_fill_i32(t.count, t.N, 0, s));
        if (t.fmt_L >= 0) {
            if (mark) TAM_HIP(tam::launch_format(t, h->pairs, s));  // every word of every row
        } else if (h->rec_groups.n > 0 && (lists || count_only)) {  // tail lists: the compile's groups
            TAM_HIP(tam::launch_probe_groups(t, h->rec_groups, 0, h->rec_groups.n, h->pairs, s));
        } else if (lists || count_only || mark) {
            TAM_HIP(tam::launch_probe(t, lists || count_only, mark, h->pairs, s));
        }
        if (timing) TAM_HIP(hipEventRecord(h->ev[2], s));
    } else if (timing) {
        h->mark_from_ev4 = true;
    }
    if (lists) {
        TAM_HIP(tam::launch_scan(t, s));
        if (h->rec_groups.n > 0) {  // the probe pass left a record of each listed hit
            TAM_HIP(tam::launch_fill_records(t, h->rec_groups, s));
        } else {
            TAM_HIP(tam::launch_fill_i32(t.cursor, t.N, 0, s));
            TAM_HIP(tam::launch_fill_lists(t, s));
        }
        h->lists_built = true;
    }
    if (timing) {
        TAM_HIP(hipEventRecord(h->ev[3], s));
        h->events_recorded = true;
    }
    TAM_HIP(copy_errors(h, s, capturing));
    if (h->work_done && !capturing) TAM_HIP(hipEventRecord(h->work_done, s));
    return TAM_OK;
}

tam_status check_device_handle(const tam_handle *h) {
    if (!h) return fail(TAM_E_INVAL, "null handle");
    if (h->flags & TAM_FLAG_HOST_ONLY) return fail(TAM_E_STATE, "handle was compiled with TAM_FLAG_HOST_ONLY");
    return TAM_OK;
}

// The trie's tables (at their offsets in the trie's allocation `tb`) and the
// vocabulary's tables in a DevTables, with the sizes they imply; no table,
// tails or lists yet.
void set_trie_tables(tam::DevTables &t, const tam_handle *h, const tam_vocab *v, uint8_t *tb, size_t o_blob,
                     size_t o_node_at, size_t o_node_pos, size_t o_depth, size_t o_child_off, size_t o_child_byte,
                     size_t o_child_node, size_t o_child_pos, size_t o_child_at) {
    t.blob = tb + o_blob;
    t.node_at = reinterpret_cast<const int32_t *>(tb + o_node_at);
    t.node_pos = reinterpret_cast<const int32_t *>(tb + o_node_pos);
    t.depth = reinterpret_cast<const int32_t *>(tb + o_depth);
    t.child_off = reinterpret_cast<const int32_t *>(tb + o_child_off);
    t.child_byte = tb + o_child_byte;
    t.child_node = reinterpret_cast<const int32_t *>(tb + o_child_node);
    t.child_pos = reinterpret_cast<const int32_t *>(tb + o_child_pos);
    t.child_at = reinterpret_cast<const uint64_t *>(tb + o_child_at);
    t.tok_off = v->d_tok_off;
    t.tok_blob = v->d_tok_blob;
    t.fps = v->d_fps;
    t.pay = v->d_pay;
    t.pay_hi = v->d_pay_hi;
    t.short_hits = v->d_short_hits;
    t.dup_next = v->d_dup_next;
    t.len_present = v->d_len_present;
    t.table = nullptr;
    t.sub_end = nullptr;
    t.tail_span = nullptr;
    t.row_of = nullptr;
    t.row_at = t.node_at;
    t.R = 0;
    t.tail_long = 0;
    t.tail_lists = 0;
    t.rec_off = nullptr;
    t.rec_cnt = nullptr;
    t.N = h->N;
    t.V = v->V;
    t.W = v->W;
    t.Wp = (v->W + 7) & ~int64_t(7);
    t.blob_bytes = h->blob_bytes;
    t.slot_mask = (uint64_t)v->fps.size() - 1;
    t.len_mask = v->len_mask;
    t.max_len = (int32_t)v->max_tok_len;
    t.terminator = h->terminator;
    t.classes = nullptr;
    t.fmt_L = -1;
}

// Compile against a built vocabulary (the handle takes one reference to it).
tam_status compile_with(const uint8_t *str_bytes, const int64_t *str_off, int64_t K, tam_vocab *vocab,
                        const int64_t *set_off, int64_t S, const tam_options *opt, const tam_allocator *alloc,
                        hipStream_t s, tam_handle **out) {
    *out = nullptr;
    if (K <= 0) return fail(TAM_E_INVAL, "K must be >= 1");
    if (!csr_ok(str_off, K)) return fail(TAM_E_INVAL, "str_off must start at 0 and be non-decreasing");
    if (!str_bytes && str_off[K] > 0) return fail(TAM_E_INVAL, "str_bytes is null");
    const int64_t one_set[2] = {0, K};
    if (!set_off || S == 0) {
        set_off = one_set;
        S = 1;
    }
    if (S < 0 || set_off[0] != 0 || set_off[S] != K) return fail(TAM_E_INVAL, "set_off must run from 0 to K");
    for (int64_t j = 0; j < S; ++j)
        if (set_off[j + 1] <= set_off[j]) return fail(TAM_E_INVAL, "every set must hold at least one string");
    tam_options o{0x22, 0, 0};
    if (opt) o = *opt;
    if (o.terminator < 0 || o.terminator > 255) return fail(TAM_E_INVAL, "terminator must be a byte value");
    if (alloc && (!alloc->alloc || !alloc->free)) return fail(TAM_E_INVAL, "allocator callbacks are null");
    const bool host_only = (o.flags & TAM_FLAG_HOST_ONLY) != 0;
    if (!host_only && (vocab->flags & TAM_FLAG_HOST_ONLY))
        return fail(TAM_E_STATE, "a device compile needs a vocabulary built without TAM_FLAG_HOST_ONLY");

    tam_handle *h = new (std::nothrow) tam_handle();
    if (!h) return fail(TAM_E_NOMEM, "out of host memory");
    h->terminator = o.terminator;
    h->flags = o.flags;
    vocab->refs.fetch_add(1);
    h->vocab = vocab;
    std::string err;
    tam_status st;
    // Device work starts before the host has finished the trie: once the trie
    // is planned its device arrays are allocated (and a full table's zero fill,
    // which needs only the node count, is enqueued); each group of sets is
    // uploaded as soon as the host has written it, so that the copies run while
    // the next group is written.
    const bool early_zero =
        !host_only && !(o.flags & (TAM_FLAG_NO_TABLE | TAM_FLAG_TAIL_LISTS | TAM_FLAG_LAZY_ROWS));
    uint64_t *early_table = nullptr;
    // blob, node_at, node_pos, depth, child_off, child_byte, child_node, sub_end,
    // and tail compression's tail_span, row_of, row_at
    uint8_t *trie_base = nullptr;
    size_t o_blob = 0, o_node_at = 0, o_node_pos = 0, o_depth = 0, o_child_off = 0, o_child_byte = 0,
           o_child_node = 0, o_child_pos = 0, o_child_at = 0, o_sub_end = 0, o_tail_span = 0, o_row_of = 0, o_row_at = 0, o_tail_rec = 0,
           o_root_rows = 0;
    // tail compression's split (with a table for the branching nodes, or with
    // sparse lists for them)
    const bool split = (o.flags & TAM_FLAG_TAIL_LISTS) && !(o.flags & TAM_FLAG_LAZY_ROWS);
    // Lists (no table): the probe pass that counts each node's list runs group
    // by group, right after each group's upload (a node's ancestors are in its
    // own set), so only the last group's counts follow the host build.
    const bool early_count =
        !host_only && (o.flags & TAM_FLAG_NO_TABLE) && !(o.flags & (TAM_FLAG_LAZY_ROWS | TAM_FLAG_TAIL_LISTS));
    // Tail compression without a table: the same, each group of sets with its
    // own records of listed hits (their regions sized on the host from the
    // group's strings).
    const bool early_tail = !host_only && (o.flags & TAM_FLAG_NO_TABLE) && (o.flags & TAM_FLAG_TAIL_LISTS) &&
                            !(o.flags & TAM_FLAG_LAZY_ROWS);
    size_t o_pairs_t = 0, o_rec_off_t = 0, o_rec_cnt_t = 0;
    int64_t next_blk = 0, next_off = 0, listed_total = 0;  // early_tail: the groups' blocks, offsets, records
    size_t o_hits = 0, o_count = 0, o_tmp = 0, o_scan_tmp = 0, o_strs = 0, o_err = 0;
    tam::DevTables te{};  // the trie and vocabulary tables the early counts read
    bool enqueued = false;  // device work that reads host tables or writes device memory
    double hook_ms = 0;     // time spent in the two hooks (allocation and enqueue)
    auto planned = [&](tam_handle *hh) -> tam_status {
        const auto t1 = std::chrono::steady_clock::now();
        (void)hipGetLastError();  // clear a stale error of an earlier, unrelated call
        if (hipGetDevice(&hh->device) != hipSuccess) {
            err = "no HIP device";
            return TAM_E_DEVICE;
        }
        if (hh->device != vocab->device) {
            err = "the vocabulary lives on another device";
            return TAM_E_STATE;
        }
        hh->own_alloc = alloc == nullptr;
        if (alloc) hh->alloc = *alloc;
        Arena ta;
        o_blob = ta.take<uint8_t>(hh->blob_bytes);
        o_node_at = ta.take<int32_t>(hh->blob_bytes);
        o_node_pos = ta.take<int32_t>(hh->N);
        o_depth = ta.take<int32_t>(hh->N);
        o_child_off = ta.take<int32_t>(hh->N + 1);
        o_child_byte = ta.take<uint8_t>(hh->edges);
        o_child_node = ta.take<int32_t>(hh->edges);
        o_child_pos = ta.take<int32_t>(hh->edges);
        o_child_at = ta.take<uint64_t>(hh->blob_bytes);
        o_sub_end = ta.take<int32_t>((hh->flags & TAM_FLAG_LAZY_ROWS) ? hh->N : 0);
        o_tail_span = ta.take<int32_t>(split ? hh->N : 0);
        o_row_of = ta.take<int32_t>(split ? hh->N : 0);
        o_row_at = ta.take<int32_t>(split ? hh->blob_bytes : 0);
        o_tail_rec = ta.take<tam::TailRec>(split ? hh->K_unique : 0);
        o_root_rows = ta.take<int32_t>(split ? 2 * hh->S : 0);
        o_hits = ta.take<int32_t>(early_count || early_tail ? tam::kWin * hh->N : 0);
        o_count = ta.take<int32_t>(early_count || early_tail ? hh->N : 0);
        // a group's blocks start a new block of nodes: at most one more block
        // than the whole range per group
        const int64_t gblocks = tam::mark_blocks(hh->N) + tam::kMaxRecGroups;
        o_pairs_t = ta.take<int32_t>(early_tail ? gblocks : 0);
        o_rec_off_t = ta.take<int32_t>(early_tail ? gblocks + tam::kMaxRecGroups : 0);  // blocks + 1 per group
        o_rec_cnt_t = ta.take<int32_t>(early_tail ? gblocks : 0);
        if (early_tail) hh->rec_off.resize((size_t)(gblocks + tam::kMaxRecGroups));
        o_strs = ta.take<tam::StrRec>(hh->K_unique);
        o_tmp = ta.take<int32_t>(hh->N);  // scratch of the child lists' build
        o_scan_tmp = ta.take<int32_t>(tam::scan_tmp_elems(hh->N));
        o_err = ta.take<int32_t>(1);
        trie_base = static_cast<uint8_t *>(dev_alloc(hh, ta.used));
        if (!trie_base) {
            err = "device allocation failed (" + std::to_string(ta.used) + " bytes requested)";
            return TAM_E_NOMEM;
        }
        hh->device_bytes = (int64_t)ta.used;
        set_trie_tables(te, hh, vocab, trie_base, o_blob, o_node_at, o_node_pos, o_depth, o_child_off, o_child_byte,
                        o_child_node, o_child_pos, o_child_at);
        hh->d_err = reinterpret_cast<int32_t *>(trie_base + o_err);
        hh->h_err = tam::err_slot_take();
        te.err = hh->d_err;
        {  // the blob's outer pads stand for the first set's root; no device error yet
            int32_t *node_at = reinterpret_cast<int32_t *>(trie_base + o_node_at);
            hipError_t e = tam::launch_fill_i32(hh->d_err, 1, 0, s);
            if (e == hipSuccess) e = tam::launch_fill_i32(node_at, tam::kBlobPad, 0, s);
            if (e == hipSuccess) e = tam::launch_fill_i32(node_at + hh->blob_bytes - tam::kBlobPad, tam::kBlobPad, 0, s);
            enqueued = true;
            if (e != hipSuccess) {
                err = std::string("trie tables: ") + hipGetErrorString(e);
                return TAM_E_DEVICE;
            }
        }
        if (early_tail) {
            te.tail_lists = 1;
            te.tail_span = reinterpret_cast<const int32_t *>(trie_base + o_tail_span);
            te.row_of = reinterpret_cast<const int32_t *>(trie_base + o_row_of);
            te.row_at = reinterpret_cast<const int32_t *>(trie_base + o_row_at);
            te.rec_off = reinterpret_cast<const int32_t *>(trie_base + o_rec_off_t);
            te.rec_cnt = reinterpret_cast<int32_t *>(trie_base + o_rec_cnt_t);
        }
        if (early_count || early_tail) {
            te.hits = reinterpret_cast<int32_t *>(trie_base + o_hits);
            te.count = reinterpret_cast<int32_t *>(trie_base + o_count);
            hipError_t e = hipStreamWaitEvent(s, vocab->ready, 0);
            const bool timing = (hh->flags & TAM_FLAG_TIMING) != 0;
            if (e == hipSuccess && timing) e = create_events(hh);
            if (e == hipSuccess && timing) e = hipEventRecord(hh->ev[0], s);
            if (e == hipSuccess && timing) e = hipEventRecord(hh->ev[1], s);  // no zero fill
            if (e == hipSuccess) e = tam::launch_fill_i32(te.count, hh->N, 0, s);
            enqueued = true;
            if (e != hipSuccess) {
                err = std::string("list counts: ") + hipGetErrorString(e);
                return TAM_E_DEVICE;
            }
        }
        if (early_zero) {
            const int64_t Wp = (vocab->W + 7) & ~int64_t(7);
            const size_t bytes = (size_t)hh->N * (size_t)Wp * sizeof(uint64_t);
            early_table = static_cast<uint64_t *>(dev_alloc(hh, bytes));
            if (!early_table) {
                err = "device allocation failed (" + std::to_string(bytes) + " bytes requested)";
                return TAM_E_NOMEM;
            }
            hh->device_bytes += (int64_t)bytes;
            hipError_t e = hipSuccess;
            const bool timing = (hh->flags & TAM_FLAG_TIMING) != 0;
            if (timing) e = create_events(hh);
            if (e == hipSuccess && timing) e = hipEventRecord(hh->ev[0], s);
            if (e == hipSuccess) e = tam::launch_zero(early_table, hh->N * Wp, s);
            enqueued = true;
            if (e == hipSuccess && timing) e = hipEventRecord(hh->ev[1], s);
            if (e != hipSuccess) {
                err = std::string("table zero fill: ") + hipGetErrorString(e);
                return TAM_E_DEVICE;
            }
        }
        hook_ms += ms_since(t1);
        return TAM_OK;
    };
    auto emitted = [&](tam_handle *hh, const tam::TrieRange &r) -> tam_status {
        const auto t1 = std::chrono::steady_clock::now();
        hipError_t e = hipSuccess;
        auto up = [&](size_t off, const void *src, int64_t lo, int64_t hi, size_t elem) {
            if (e == hipSuccess && hi > lo) {
                e = hipMemcpyAsync(trie_base + off + (size_t)lo * elem, static_cast<const uint8_t *>(src) + (size_t)lo * elem,
                                   (size_t)(hi - lo) * elem, hipMemcpyHostToDevice, s);
                enqueued = true;
            }
        };
        up(o_blob, hh->blob.data(), r.b_lo, r.b_hi, 1);
        up(o_strs, hh->strs.data(), r.s_lo, r.s_hi, sizeof(tam::StrRec));
        if (hh->flags & TAM_FLAG_LAZY_ROWS) up(o_sub_end, hh->sub_end.data(), r.n_lo, r.n_hi, 4);
        if (split) {  // the tail tables are laid out on the device from these
            up(o_tail_rec, hh->tail_rec.data(), r.s_lo, r.s_hi, sizeof(tam::TailRec));
            if (r.n_lo == 0) up(o_root_rows, hh->root_rows.data(), 0, (int64_t)hh->root_rows.size(), 4);
        }
        // the group's node_at and depth (from its strings), node positions
        // (its nodes lie in its blob range), then (lists) its counts; after the
        // last group the child lists
        int32_t *node_pos = reinterpret_cast<int32_t *>(trie_base + o_node_pos);
        if (e == hipSuccess)
            e = tam::launch_node_at(reinterpret_cast<const tam::StrRec *>(trie_base + o_strs), r.s_lo, r.s_hi,
                                    hh->blob_bytes, hh->N, reinterpret_cast<int32_t *>(trie_base + o_node_at),
                                    reinterpret_cast<int32_t *>(trie_base + o_depth), hh->d_err, s);
        if (e == hipSuccess && split)
            e = tam::launch_tail_tables(reinterpret_cast<const tam::StrRec *>(trie_base + o_strs),
                                        reinterpret_cast<const tam::TailRec *>(trie_base + o_tail_rec), r.s_lo,
                                        r.s_hi, r.n_lo == 0 ? reinterpret_cast<const int32_t *>(trie_base + o_root_rows)
                                                            : nullptr,
                                        hh->S, reinterpret_cast<const int32_t *>(trie_base + o_node_at), r.b_lo,
                                        r.b_hi, hh->N, reinterpret_cast<int32_t *>(trie_base + o_row_of),
                                        reinterpret_cast<int32_t *>(trie_base + o_tail_span),
                                        reinterpret_cast<int32_t *>(trie_base + o_row_at), hh->d_err, s);
        if (e == hipSuccess) e = tam::launch_node_pos(te, node_pos, r.n_lo, r.n_hi, r.b_lo, r.b_hi, s);
        if (early_count && e == hipSuccess) {
            const bool timing = (hh->flags & TAM_FLAG_TIMING) != 0;
            if (timing && r.n_lo == 0) e = hipEventRecord(hh->ev[4], s);  // the counts' start
            if (e == hipSuccess) e = tam::launch_count_range(te, r.n_lo, r.n_hi, s);
            if (e == hipSuccess && timing && r.n_hi == hh->N) e = hipEventRecord(hh->ev[2], s);
        }
        if (early_tail && e == hipSuccess && r.n_hi > r.n_lo) {
            // the group's record regions (sized on the host from its strings),
            // their upload, the group's record buffer, then its probe pass
            const int64_t per = tam::probe_nodes_per_block();
            const int64_t blocks = (r.n_hi - r.n_lo + per - 1) / per;
            tam::RecGroups &rg = hh->rec_groups;
            if (rg.n >= tam::kMaxRecGroups || next_blk + blocks > tam::mark_blocks(hh->N) + tam::kMaxRecGroups ||
                next_off + blocks + 1 > (int64_t)hh->rec_off.size()) {
                err = "listed-hit regions exceed the probe grid";
                return TAM_E_STATE;
            }
            const int64_t total = tam::group_regions(hh, vocab, r.s_lo, r.s_hi, r.n_lo, per, blocks,
                                                     hh->rec_off.data() + next_off);
            if (listed_total + total >= INT32_MAX) {
                err = "more than 2^31-1 valid (node, token) pairs are possible";
                return TAM_E_TOOLARGE;
            }
            const size_t rec_bytes = (size_t)(3 * std::max<int64_t>(total, 1)) * sizeof(int32_t);
            int32_t *rec = static_cast<int32_t *>(dev_alloc(hh, rec_bytes));
            if (!rec) {
                err = "device allocation failed (" + std::to_string(rec_bytes) + " bytes requested)";
                return TAM_E_NOMEM;
            }
            hh->device_bytes += (int64_t)rec_bytes;
            up(o_rec_off_t, hh->rec_off.data(), next_off, next_off + blocks + 1, 4);
            const int k = rg.n++;
            rg.n_lo[k] = r.n_lo;
            rg.n_hi[k] = r.n_hi;
            rg.blk0[k] = next_blk;
            rg.blk0[k + 1] = next_blk + blocks;
            rg.off0[k] = next_off;
            rg.rec[k] = rec;
            const bool timing = (hh->flags & TAM_FLAG_TIMING) != 0;
            if (e == hipSuccess && timing && r.n_lo == 0) e = hipEventRecord(hh->ev[4], s);  // the probe's start
            if (e == hipSuccess)
                e = tam::launch_probe_groups(te, rg, k, k + 1, reinterpret_cast<int32_t *>(trie_base + o_pairs_t), s);
            if (e == hipSuccess && timing && r.n_hi == hh->N) e = hipEventRecord(hh->ev[2], s);
            next_blk += blocks;
            next_off += blocks + 1;
            listed_total += total;
        }
        if (e == hipSuccess && r.n_hi == hh->N)
            e = tam::launch_child_lists(te, reinterpret_cast<int32_t *>(trie_base + o_child_off),
                                        reinterpret_cast<int32_t *>(trie_base + o_child_node),
                                        trie_base + o_child_byte,
                                        reinterpret_cast<int32_t *>(trie_base + o_child_pos),
                                        reinterpret_cast<uint64_t *>(trie_base + o_child_at),
                                        reinterpret_cast<int32_t *>(trie_base + o_tmp),
                                        reinterpret_cast<int32_t *>(trie_base + o_scan_tmp), s);
        hook_ms += ms_since(t1);
        if (e != hipSuccess) {
            err = std::string("upload: ") + hipGetErrorString(e);
            return TAM_E_DEVICE;
        }
        return TAM_OK;
    };
    try {
        const auto t0 = std::chrono::steady_clock::now();
        const bool lazy = (o.flags & TAM_FLAG_LAZY_ROWS) != 0;
        const tam::PinnedScope pinned(!host_only);  // the uploaded trie tables go to pinned memory
        using Planned = std::function<tam_status(tam_handle *)>;
        using Emitted = std::function<tam_status(tam_handle *, const tam::TrieRange &)>;
        st = tam::build_trie(str_bytes, str_off, K, set_off, S, o.terminator, h, &err,  // with the tail split
                             host_only ? Planned() : Planned(planned), host_only ? Emitted() : Emitted(emitted));
        h->timing.host_trie_ms = ms_since(t0) - hook_ms;
        // the lists (and their size bound) are needed without a table, or with
        // tail compression when tokens exceed the probe window
        const bool lists = !lazy && ((o.flags & TAM_FLAG_NO_TABLE) ||
                                     ((o.flags & TAM_FLAG_TAIL_LISTS) && vocab->max_tok_len > tam::kWin));
        if (st == TAM_OK && lists) {
            // tail compression without a table: the groups' record regions,
            // summed as each group was uploaded
            h->entry_bound = early_tail ? listed_total : tam::entry_upper_bound(h, vocab);
            if (h->entry_bound >= INT32_MAX) {
                st = TAM_E_TOOLARGE;
                err = "more than 2^31-1 valid (node, token) pairs are possible";
            }
        }
    } catch (const std::bad_alloc &) {
        st = TAM_E_NOMEM;
        err = "out of host memory";
    } catch (const std::exception &x) {  // e.g. no host thread could be made
        st = TAM_E_NOMEM;
        err = std::string("host build failed: ") + x.what();
    }
    if (st != TAM_OK) {
        if (enqueued) (void)hipStreamSynchronize(s);  // copies may still read the host tables
        destroy_handle(h);
        return fail(st, err);
    }
    h->V = vocab->V;
    h->W = vocab->W;
    h->Wp = (h->W + 7) & ~int64_t(7);  // rows 64-byte aligned
    if (is_lazy(h)) {
        if (o.cache_rows < 0) {
            if (enqueued) (void)hipStreamSynchronize(s);
            destroy_handle(h);
            return fail(TAM_E_INVAL, "cache_rows must be >= 0");
        }
        h->cache_rows = std::max<int64_t>(1, std::min<int64_t>(o.cache_rows ? o.cache_rows : 4096, h->N));
    }
    h->timing.dev_lists_ms = h->timing.dev_zero_ms = h->timing.dev_mark_ms = -1.f;
    h->timing.dev_total_ms = -1.f;
    if (host_only) {
        *out = h;
        return TAM_OK;
    }

    // ---- device: the remaining tables, uploads and the device phases ----
    const auto t0 = std::chrono::steady_clock::now();
    const bool lazy = is_lazy(h);
    const bool want_table = !lazy && !(h->flags & TAM_FLAG_NO_TABLE);
    const bool tails = !lazy && h->tails;
    const bool tail_long = tails && want_table && vocab->max_tok_len > tam::kWin;
    const bool tail_lists = tails && !want_table;  // branching nodes keep sparse lists
    const bool want_lists = !want_table || tail_long;
    // dense rows: every node, or the branching nodes (at least one row is kept
    // so that a tail-compressed handle always has a table)
    const int64_t R = !want_table ? 0 : tails ? std::max<int64_t>(h->dense_rows, 1) : h->N;

    Arena a;
    // the probe pass's tables (none when rows are built on demand; the hits and
    // counts of early list counts are in the trie's allocation)
    const int64_t NP = lazy ? 0 : h->N;
    const bool early = early_count || early_tail;  // hits and counts are in the trie's allocation
    const size_t o_hits_b = a.take<int32_t>(early ? 0 : tam::kWin * NP);
    const size_t o_count_b = a.take<int32_t>(early ? 0 : NP);
    const size_t o_row_ptr = a.take<int32_t>(NP + 1);
    const size_t o_cursor = a.take<int32_t>(NP);
    const size_t o_entries = a.take<int32_t>(want_lists ? std::max<int64_t>(h->entry_bound, 1) : 1);
    const size_t o_scan = a.take<int32_t>(tam::scan_tmp_elems(NP));
    // tail lists: the probe grid's pair slots are the groups' (trie allocation)
    h->npairs = lazy ? 0 : early_tail ? next_blk : tam::mark_blocks(h->N);
    const size_t o_pairs = a.take<int32_t>(early_tail ? 0 : h->npairs);
    // rows built on demand: subtree extents, the cache's bookkeeping, the
    // scratch of one group of batch rows
    const int64_t C = lazy ? h->cache_rows : 0, G = lazy ? tam::kLazyGroup : 0;
    const int64_t P = lazy ? std::min<int64_t>(C, tam::kLazyGroup) : 0;  // spare cache rows
    const size_t o_slot_of = a.take<int32_t>(lazy ? h->N : 0);
    const size_t o_node_of = a.take<int32_t>(C + P);
    const size_t o_stamp = a.take<uint32_t>(C + P);
    const size_t o_ref = a.take<uint32_t>(C + P);
    const size_t o_state = a.take<uint32_t>(3);
    const size_t o_spare = a.take<int32_t>(P);
    const size_t o_miss_free = a.take<int32_t>(G);
    const size_t o_rows_src = a.take<int32_t>(G);
    const size_t o_miss_node = a.take<int32_t>(G);
    const size_t o_miss_row = a.take<int32_t>(G);
    const size_t o_miss_off = a.take<int64_t>(G + 1);
    const size_t o_miss_dep = a.take<int32_t>(G);
    const size_t o_miss_count = a.take<int32_t>(1);

    uint8_t *base = static_cast<uint8_t *>(dev_alloc(h, a.used));
    uint64_t *table = early_table;
    const size_t table_bytes = (size_t)(lazy ? C + P : R) * (size_t)h->Wp * sizeof(uint64_t);
    if (base && (want_table || lazy) && !table) table = static_cast<uint64_t *>(dev_alloc(h, table_bytes));
    if (!base || ((want_table || lazy) && !table)) {
        (void)hipStreamSynchronize(s);  // copies may still read the host tables
        destroy_handle(h);
        return fail(TAM_E_NOMEM, "device allocation failed (" + std::to_string(a.used + table_bytes) +
                                     " bytes requested)");
    }
    h->device_bytes += (int64_t)a.used + (table && !early_table ? (int64_t)table_bytes : 0);
    h->pairs = early_tail ? reinterpret_cast<int32_t *>(trie_base + o_pairs_t)
                          : reinterpret_cast<int32_t *>(base + o_pairs);

    tam::DevTables &t = h->dt;
    set_trie_tables(t, h, vocab, trie_base, o_blob, o_node_at, o_node_pos, o_depth, o_child_off, o_child_byte,
                    o_child_node, o_child_pos, o_child_at);
    t.err = h->d_err;
    t.hits = early ? te.hits : reinterpret_cast<int32_t *>(base + o_hits_b);
    t.count = early ? te.count : reinterpret_cast<int32_t *>(base + o_count_b);
    t.row_ptr = reinterpret_cast<int32_t *>(base + o_row_ptr);
    t.cursor = reinterpret_cast<int32_t *>(base + o_cursor);
    t.entries = reinterpret_cast<int32_t *>(base + o_entries);
    t.scan_tmp = reinterpret_cast<int32_t *>(base + o_scan);
    t.table = lazy ? nullptr : table;
    t.sub_end = lazy ? reinterpret_cast<const int32_t *>(trie_base + o_sub_end) : nullptr;
    if (lazy) {
        tam::LazyDev &z = h->lazy;
        z.cache = table;
        z.slot_of = reinterpret_cast<int32_t *>(base + o_slot_of);
        z.node_of = reinterpret_cast<int32_t *>(base + o_node_of);
        z.stamp = reinterpret_cast<uint32_t *>(base + o_stamp);
        z.ref = reinterpret_cast<uint32_t *>(base + o_ref);
        z.state = reinterpret_cast<uint32_t *>(base + o_state);
        z.spare = reinterpret_cast<int32_t *>(base + o_spare);
        z.miss_free = reinterpret_cast<int32_t *>(base + o_miss_free);
        z.P = P;
        z.rows_src = reinterpret_cast<int32_t *>(base + o_rows_src);
        z.miss_node = reinterpret_cast<int32_t *>(base + o_miss_node);
        z.miss_row = reinterpret_cast<int32_t *>(base + o_miss_row);
        z.miss_off = reinterpret_cast<int64_t *>(base + o_miss_off);
        z.miss_dep = reinterpret_cast<int32_t *>(base + o_miss_dep);
        z.miss_count = reinterpret_cast<int32_t *>(base + o_miss_count);
        z.err = h->d_err;
        z.C = C;
    }
    t.tail_span = tails ? reinterpret_cast<const int32_t *>(trie_base + o_tail_span) : nullptr;
    t.row_of = tails ? reinterpret_cast<const int32_t *>(trie_base + o_row_of) : nullptr;
    t.row_at = tails ? reinterpret_cast<const int32_t *>(trie_base + o_row_at) : t.node_at;
    t.R = R;
    t.tail_long = tail_long ? 1 : 0;
    t.tail_lists = tail_lists ? 1 : 0;
    t.rec_off = early_tail ? te.rec_off : nullptr;
    t.rec_cnt = early_tail ? te.rec_cnt : nullptr;

    // the trie's tables were uploaded group by group while the host wrote them
    if (tail_lists != early_tail) {  // the listed hits' records were planned with the trie
        (void)hipStreamSynchronize(s);
        destroy_handle(h);
        return fail(TAM_E_STATE, "tail lists without their records");
    }
    hipError_t e = hipStreamWaitEvent(s, vocab->ready, 0);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&h->work_done, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventRecord(h->work_done, s);
    if (e == hipSuccess && (h->flags & TAM_FLAG_TIMING)) e = create_events(h);
    h->timing.upload_ms = hook_ms + ms_since(t0);
    if (e != hipSuccess) {
        st = hip_fail(e, "upload");
        const std::string msg = g_err;
        (void)hipStreamSynchronize(s);  // copies already enqueued still read the host tables
        destroy_handle(h);
        return fail(st, msg);
    }
    st = run_device_phase(h, default_phases(h) & ~(early_table ? unsigned(TAM_PHASE_ZERO) : 0u), s,
                          early_table != nullptr, early);
    if (st != TAM_OK) {
        const std::string msg = g_err;
        destroy_handle(h);
        return fail(st, msg);
    }
    *out = h;
    return TAM_OK;
}

// Character-position masks of a fixed-format value (see tam.h).
tam_status compile_format(const uint8_t *classes, int64_t L, tam_vocab *vocab, const tam_options *opt,
                          const tam_allocator *alloc, hipStream_t s, tam_handle **out) {
    *out = nullptr;
    if (L < 1 || L > INT32_MAX - 3) return fail(TAM_E_INVAL, "L must be in [1, 2^31-4]");
    if (!classes) return fail(TAM_E_INVAL, "classes is null");
    tam_options o{0x22, 0, 0};
    if (opt) o = *opt;
    if (o.terminator < 0 || o.terminator > 255) return fail(TAM_E_INVAL, "terminator must be a byte value");
    if (alloc && (!alloc->alloc || !alloc->free)) return fail(TAM_E_INVAL, "allocator callbacks are null");
    const int T = o.terminator;
    for (int64_t p = 0; p < L; ++p)
        if ((classes[32 * p + (T >> 3)] >> (T & 7)) & 1)
            return fail(TAM_E_TERMINATOR, "class " + std::to_string(p) + " admits the terminator byte");
    const bool host_only = (o.flags & TAM_FLAG_HOST_ONLY) != 0;
    if (!host_only && (vocab->flags & TAM_FLAG_HOST_ONLY))
        return fail(TAM_E_STATE, "a device compile needs a vocabulary built without TAM_FLAG_HOST_ONLY");

    tam_handle *h = new (std::nothrow) tam_handle();
    if (!h) return fail(TAM_E_NOMEM, "out of host memory");
    h->terminator = T;
    h->flags = o.flags & (TAM_FLAG_HOST_ONLY | TAM_FLAG_TIMING);
    vocab->refs.fetch_add(1);
    h->vocab = vocab;
    const auto t0 = std::chrono::steady_clock::now();
    const int64_t N = L + 2;
    try {
        h->fmt_L = L;
        h->classes.assign(classes, classes + 32 * L);
        h->N = N;
        h->S = 1;
        h->K_unique = 0;
        h->roots.assign(1, 0);
        h->parent.resize((size_t)N);
        h->depth.resize((size_t)N);
        h->edge.assign((size_t)N, 0);
        h->is_final.assign((size_t)N, 0);
        for (int64_t p = 0; p < N; ++p) {
            h->parent[(size_t)p] = (int32_t)(p - 1);
            h->depth[(size_t)p] = (int32_t)p;
        }
        h->edge[(size_t)(N - 1)] = (uint8_t)T;
        h->is_final[(size_t)(N - 1)] = 1;
    } catch (const std::bad_alloc &) {
        destroy_handle(h);
        return fail(TAM_E_NOMEM, "out of host memory");
    }
    h->timing.host_trie_ms = ms_since(t0);
    h->V = vocab->V;
    h->W = vocab->W;
    h->Wp = (h->W + 7) & ~int64_t(7);
    h->dense_rows = N;
    h->timing.dev_lists_ms = h->timing.dev_zero_ms = h->timing.dev_mark_ms = -1.f;
    h->timing.dev_total_ms = -1.f;
    if (host_only) {
        *out = h;
        return TAM_OK;
    }

    const auto t1 = std::chrono::steady_clock::now();
    (void)hipGetLastError();
    if (hipGetDevice(&h->device) != hipSuccess) {
        destroy_handle(h);
        return fail(TAM_E_DEVICE, "no HIP device");
    }
    if (h->device != vocab->device) {
        destroy_handle(h);
        return fail(TAM_E_STATE, "the vocabulary lives on another device");
    }
    h->own_alloc = alloc == nullptr;
    if (alloc) h->alloc = *alloc;
    h->npairs = tam::format_blocks(h->Wp);
    Arena a;
    const size_t o_cls = a.take<uint8_t>(32 * L);
    const size_t o_pairs = a.take<int32_t>(h->npairs);
    const size_t o_err = a.take<int32_t>(1);
    uint8_t *base = static_cast<uint8_t *>(dev_alloc(h, a.used));
    const size_t table_bytes = (size_t)N * (size_t)h->Wp * sizeof(uint64_t);
    uint64_t *table = base ? static_cast<uint64_t *>(dev_alloc(h, table_bytes)) : nullptr;
    if (!base || !table) {
        destroy_handle(h);
        return fail(TAM_E_NOMEM, "device allocation failed (" + std::to_string(a.used + table_bytes) +
                                     " bytes requested)");
    }
    h->device_bytes = (int64_t)(a.used + table_bytes);
    h->pairs = reinterpret_cast<int32_t *>(base + o_pairs);
    tam::DevTables &t = h->dt;
    t = tam::DevTables{};
    t.tok_off = vocab->d_tok_off;
    t.tok_blob = vocab->d_tok_blob;
    t.fps = vocab->d_fps;
    t.pay = vocab->d_pay;
    t.pay_hi = vocab->d_pay_hi;
    t.short_hits = vocab->d_short_hits;
    t.dup_next = vocab->d_dup_next;
    t.len_present = vocab->d_len_present;
    t.table = table;
    t.row_at = nullptr;
    t.N = N;
    t.V = h->V;
    t.W = h->W;
    t.Wp = h->Wp;
    t.R = N;
    t.slot_mask = (uint64_t)vocab->fps.size() - 1;
    t.len_mask = vocab->len_mask;
    t.max_len = (int32_t)vocab->max_tok_len;
    t.terminator = T;
    t.classes = base + o_cls;
    t.fmt_L = (int32_t)L;
    h->d_err = reinterpret_cast<int32_t *>(base + o_err);
    h->h_err = tam::err_slot_take();
    t.err = h->d_err;
    hipError_t e = hipStreamWaitEvent(s, vocab->ready, 0);
    if (e == hipSuccess) e = tam::launch_fill_i32(h->d_err, 1, 0, s);
    if (e == hipSuccess) e = hipMemcpyAsync(base + o_cls, h->classes.data(), h->classes.size(),
                                            hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&h->work_done, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventRecord(h->work_done, s);
    if (e == hipSuccess && (h->flags & TAM_FLAG_TIMING)) e = create_events(h);
    h->timing.upload_ms = ms_since(t1);
    tam_status st = e == hipSuccess ? TAM_OK : hip_fail(e, "upload");
    if (st == TAM_OK) st = run_device_phase(h, default_phases(h), s);
    if (st != TAM_OK) {
        const std::string msg = g_err;
        destroy_handle(h);
        return fail(st, msg);
    }
    *out = h;
    return TAM_OK;
}

// The device's trie layout on the host (tam_layout_get): the layout kernels'
// functions over the host's string records, in one pass each.
void layout_on_host(tam_handle *h) {
    const int64_t BB = h->blob_bytes, N = h->N;
    h->lay_node_at.assign((size_t)BB, 0);  // the outer pads stand for root 0, as on the device
    h->lay_depth.assign((size_t)N, -1);
    h->lay_node_pos.assign((size_t)N, -1);
    h->lay_parent.assign((size_t)N, -1);
    int32_t *node_at = h->lay_node_at.data(), *depth = h->lay_depth.data();
    int32_t *node_pos = h->lay_node_pos.data(), *parent = h->lay_parent.data();
    int64_t errors = 0;
    const int64_t K = (int64_t)h->strs.size();
    for (int64_t u = 0; u < K; ++u) errors += tam::lay_string(h->strs.data(), 0, u, BB, N, node_at, depth);
    for (int64_t g = 0; g < N; ++g) node_pos[g] = depth[g] == 0 ? -1 : INT32_MAX;
    for (int64_t p = 0; p < BB; ++p) {
        bool bad = false;
        const int32_t g = tam::lay_pos_node(node_at, depth, N, p, &bad);
        if (g >= 0 && p < node_pos[g]) node_pos[g] = (int32_t)p;
        errors += bad ? 1 : 0;
    }
    for (int64_t g = 0; g < N; ++g) {
        if (depth[g] == 0) continue;
        bool bad = false;
        parent[g] = tam::lay_parent(node_pos, node_at, N, BB, g, &bad);
        errors += bad ? 1 : 0;
    }
    h->lay_errors = errors;
}

}  // namespace

extern "C" {

tam_status tam_format_rows_noalloc(const uint8_t *classes, int64_t L, int terminator, const tam_vocab *vocab,
                                   uint64_t *out, int64_t out_stride_words, int64_t *pairs_out, void *stream) {
    g_err.clear();
    if (!classes || !vocab || !out) return fail(TAM_E_INVAL, "null argument");
    if (L < 1 || L > TAM_NOALLOC_MAX_POSITIONS)
        return fail(TAM_E_INVAL, "L must be in [1, " + std::to_string(TAM_NOALLOC_MAX_POSITIONS) +
                                     "]: the static scratch holds the class bits of at most that many positions");
    if (terminator < 0 || terminator > 255) return fail(TAM_E_INVAL, "terminator must be a byte value");
    if (out_stride_words < vocab->W) return fail(TAM_E_INVAL, "out_stride_words must be >= W");
    if ((reinterpret_cast<uintptr_t>(out) & 7) != 0 || (reinterpret_cast<uintptr_t>(pairs_out) & 7) != 0)
        return fail(TAM_E_INVAL, "out and pairs_out must be 8-byte aligned");
    for (int64_t p = 0; p < L; ++p)
        if ((classes[32 * p + (terminator >> 3)] >> (terminator & 7)) & 1)
            return fail(TAM_E_TERMINATOR, "class " + std::to_string(p) + " admits the terminator byte");
    if (vocab->flags & TAM_FLAG_HOST_ONLY) return fail(TAM_E_STATE, "the vocabulary has no device tables");
    int dev = -1;
    TAM_HIP(hipGetDevice(&dev));
    if (dev != vocab->device) return fail(TAM_E_STATE, "the vocabulary lives on another device");
    TAM_HIP(hipGetLastError());
    hipStream_t s = static_cast<hipStream_t>(stream);
    // the vocabulary's uploads, if they may still be running
    if (hipEventQuery(vocab->ready) != hipSuccess) {
        (void)hipGetLastError();
        TAM_HIP(hipStreamWaitEvent(s, vocab->ready, 0));
    }
    tam::DevTables t{};
    t.tok_off = vocab->d_tok_off;
    t.tok_blob = vocab->d_tok_blob;
    t.V = vocab->V;
    t.W = vocab->W;
    t.Wp = vocab->W;
    t.max_len = (int32_t)vocab->max_tok_len;
    t.terminator = terminator;
    t.fmt_L = (int32_t)L;
    TAM_HIP(tam::launch_format_noalloc(t, classes, out, out_stride_words, pairs_out, s));
    return TAM_OK;
}

tam_status tam_layout_get(const tam_handle *h, tam_layout *out) {
    g_err.clear();
    if (!h || !out) return fail(TAM_E_INVAL, "null argument");
    if (!(h->flags & TAM_FLAG_HOST_ONLY) || h->fmt_L >= 0)
        return fail(TAM_E_STATE, "the host layout is kept for TAM_FLAG_HOST_ONLY handles of string sets");
    tam_handle *m = const_cast<tam_handle *>(h);  // computed once, then read-only
    try {
        std::call_once(m->layout_once, [m] { layout_on_host(m); });
    } catch (const std::bad_alloc &) {
        return fail(TAM_E_NOMEM, "out of host memory");
    }
    out->blob_bytes = h->blob_bytes;
    out->blob = h->blob.data();
    out->node_at = h->lay_node_at.data();
    out->depth = h->lay_depth.data();
    out->node_pos = h->lay_node_pos.data();
    out->parent = h->lay_parent.data();
    out->errors = h->lay_errors;
    return TAM_OK;
}

const char *tam_last_error(void) { return g_err.c_str(); }

tam_status tam_vocab_create(const uint8_t *tok_bytes, const int64_t *tok_off, int64_t V, uint32_t flags,
                            const tam_allocator *alloc, void *stream, tam_vocab **out) {
    g_err.clear();
    if (!out) return fail(TAM_E_INVAL, "out is null");
    return vocab_create(tok_bytes, tok_off, V, flags, alloc, static_cast<hipStream_t>(stream), out);
}

void tam_vocab_destroy(tam_vocab *v) { vocab_release(v); }

tam_status tam_compile_vocab(const uint8_t *str_bytes, const int64_t *str_off, int64_t K,
                             const tam_vocab *vocab, const int64_t *set_off, int64_t S,
                             const tam_options *opt, const tam_allocator *alloc, void *stream,
                             tam_handle **out) {
    g_err.clear();
    if (!out) return fail(TAM_E_INVAL, "out is null");
    *out = nullptr;
    if (!vocab) return fail(TAM_E_INVAL, "vocab is null");
    return compile_with(str_bytes, str_off, K, const_cast<tam_vocab *>(vocab), set_off, S, opt, alloc,
                        static_cast<hipStream_t>(stream), out);
}

tam_status tam_compile_format(const uint8_t *classes, int64_t L, const tam_vocab *vocab,
                              const tam_options *opt, const tam_allocator *alloc, void *stream,
                              tam_handle **out) {
    g_err.clear();
    if (!out) return fail(TAM_E_INVAL, "out is null");
    *out = nullptr;
    if (!vocab) return fail(TAM_E_INVAL, "vocab is null");
    return compile_format(classes, L, const_cast<tam_vocab *>(vocab), opt, alloc, static_cast<hipStream_t>(stream),
                          out);
}

tam_status tam_compile(const uint8_t *str_bytes, const int64_t *str_off, int64_t K,
                       const uint8_t *tok_bytes, const int64_t *tok_off, int64_t V,
                       const int64_t *set_off, int64_t S, const tam_options *opt,
                       const tam_allocator *alloc, void *stream, tam_handle **out) {
    g_err.clear();
    if (!out) return fail(TAM_E_INVAL, "out is null");
    *out = nullptr;
    if (K <= 0) return fail(TAM_E_INVAL, "K must be >= 1");
    if (!csr_ok(str_off, K)) return fail(TAM_E_INVAL, "str_off must start at 0 and be non-decreasing");
    tam_options o{0x22, 0, 0};
    if (opt) o = *opt;
    tam_vocab *v = nullptr;
    hipStream_t s = static_cast<hipStream_t>(stream);
    tam_status st = vocab_create(tok_bytes, tok_off, V, o.flags, alloc, s, &v);
    if (st != TAM_OK) return st;
    st = compile_with(str_bytes, str_off, K, v, set_off, S, &o, alloc, s, out);
    if (st == TAM_OK) {
        (*out)->timing.host_vocab_ms = v->host_ms;
        (*out)->timing.upload_ms += v->upload_ms;
    }
    vocab_release(v);  // the handle keeps its own reference
    return st;
}

tam_status tam_rebuild(tam_handle *h, unsigned phases, void *stream) {
    g_err.clear();
    tam_status st = check_device_handle(h);
    if (st == TAM_OK) st = device_errors(h);
    if (st != TAM_OK) return st;
    if (is_lazy(h)) {
        if (phases != 0) return fail(TAM_E_STATE, "a handle with rows built on demand has only phase 0 (cache reset)");
        return run_device_phase(h, 0, static_cast<hipStream_t>(stream));
    }
    if (phases == 0) phases = default_phases(h);
    if (phases & ~unsigned(TAM_PHASE_LISTS | TAM_PHASE_TABLE | TAM_PHASE_COUNT))
        return fail(TAM_E_INVAL, "unknown phase bits");
    if ((phases & TAM_PHASE_TABLE) && !h->dt.table) return fail(TAM_E_STATE, "handle has no dense table");
    if ((phases & TAM_PHASE_COUNT) && (!keeps_lists(h) || !h->lists_built))
        return fail(TAM_E_STATE, "TAM_PHASE_COUNT needs a handle whose lists are built");
    if ((phases & TAM_PHASE_LISTS) && !keeps_lists(h))
        return fail(TAM_E_STATE, "valid lists are kept only with TAM_FLAG_NO_TABLE, or with "
                                 "TAM_FLAG_TAIL_LISTS and tokens longer than 16 bytes");
    return run_device_phase(h, phases, static_cast<hipStream_t>(stream));
}

tam_status tam_info_get(const tam_handle *h, tam_info *out) {
    if (!h || !out) return fail(TAM_E_INVAL, "null argument");
    out->num_nodes = h->N;
    out->num_sets = h->S;
    out->num_strings = h->K_unique;
    out->vocab_size = h->V;
    out->words_per_row = h->W;
    out->row_stride_words = h->dt.table ? h->Wp : 0;
    out->max_token_len = h->vocab->max_tok_len;
    out->device_bytes = h->device_bytes;
    out->flags = h->flags;
    out->terminator = h->terminator;
    out->roots = h->roots.data();
    out->parent = h->parent.data();
    out->depth = h->depth.data();
    out->edge_byte = h->edge.data();
    out->is_final = h->is_final.data();
    out->table = h->dt.table;
    const bool tails = h->tails;
    out->dense_rows = (h->flags & TAM_FLAG_NO_TABLE) ? 0 : tails ? h->dense_rows : h->N;
    out->dense_row = tails ? h->row_of.data() : nullptr;
    out->cache_rows = is_lazy(h) ? h->cache_rows : 0;
    out->subtree_end = h->sub_end.empty() ? nullptr : h->sub_end.data();
    out->list_capacity = h->entry_bound;
    if (is_lazy(h)) out->dense_rows = 0;
    return TAM_OK;
}

tam_status tam_apply_mask(const tam_handle *h, const int32_t *node_ids, int64_t B, void *logits,
                          int dtype, int64_t row_stride, void *stream) {
    g_err.clear();
    // argument errors first, then the handle's state
    if (!h) return fail(TAM_E_INVAL, "null handle");
    if (B < 0) return fail(TAM_E_INVAL, "B must be >= 0");
    if (dtype != TAM_DTYPE_FP32 && dtype != TAM_DTYPE_BF16) return fail(TAM_E_INVAL, "dtype must be FP32 or BF16");
    if (row_stride < h->V) return fail(TAM_E_INVAL, "row_stride must be >= V");
    const size_t elem = dtype == TAM_DTYPE_BF16 ? 2 : 4;
    if (B > 0 && (!node_ids || !logits)) return fail(TAM_E_INVAL, "null device pointer");
    if ((reinterpret_cast<uintptr_t>(logits) % elem) != 0) return fail(TAM_E_INVAL, "logits are not element-aligned");
    tam_status st = check_device_handle(h);
    if (st == TAM_OK) st = device_errors(h);
    if (st != TAM_OK || B == 0) return st;
    TAM_HIP(hipGetLastError());
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (is_lazy(h)) {  // groups of rows: cache lookup, missing rows built, masking
        const int64_t g = std::min<int64_t>(tam::kLazyGroup, h->lazy.C);
        for (int64_t r0 = 0; r0 < B; r0 += g)
            TAM_HIP(tam::launch_lazy_apply(h->dt, h->lazy, node_ids + r0, std::min(g, B - r0),
                                           static_cast<uint8_t *>(logits) + r0 * row_stride * (int64_t)elem, dtype,
                                           row_stride, s));
        return TAM_OK;
    }
    TAM_HIP(tam::launch_apply(h->dt, node_ids, B, logits, dtype, row_stride, s));
    return TAM_OK;
}

tam_status tam_advance(const tam_handle *h, const int32_t *node_ids, const int32_t *token_ids, int64_t B,
                       int32_t *out, void *stream) {
    g_err.clear();
    if (!h) return fail(TAM_E_INVAL, "null handle");
    if (B < 0) return fail(TAM_E_INVAL, "B must be >= 0");
    if (B > 0 && (!node_ids || !token_ids || !out)) return fail(TAM_E_INVAL, "null device pointer");
    tam_status st = check_device_handle(h);
    if (st == TAM_OK) st = device_errors(h);
    if (st != TAM_OK || B == 0) return st;
    TAM_HIP(hipGetLastError());
    TAM_HIP(tam::launch_advance(h->dt, node_ids, token_ids, B, out, static_cast<hipStream_t>(stream)));
    return TAM_OK;
}

tam_status tam_export_rows(const tam_handle *h, const int32_t *node_ids, int64_t n, uint64_t *out,
                           void *stream) {
    g_err.clear();
    if (!h) return fail(TAM_E_INVAL, "null handle");
    if (n < 0) return fail(TAM_E_INVAL, "n must be >= 0");
    if (n > 0 && (!node_ids || !out)) return fail(TAM_E_INVAL, "null device pointer");
    if ((reinterpret_cast<uintptr_t>(out) & 7) != 0) return fail(TAM_E_INVAL, "out must be 8-byte aligned");
    tam_status st = check_device_handle(h);
    if (st == TAM_OK) st = device_errors(h);
    if (st != TAM_OK || n == 0) return st;
    TAM_HIP(hipGetLastError());
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (is_lazy(h)) {
        for (int64_t r0 = 0; r0 < n; r0 += tam::kLazyGroup)
            TAM_HIP(tam::launch_lazy_export(h->dt, h->lazy, node_ids + r0, std::min<int64_t>(tam::kLazyGroup, n - r0),
                                            out + r0 * h->W, s));
        return TAM_OK;
    }
    if (h->dt.table) {
        TAM_HIP(tam::launch_export_dense(h->dt, node_ids, n, out, s));
    } else {
        TAM_HIP(tam::launch_rows(h->dt, node_ids, n, out, h->W, h->W, s));
        if (h->dt.tail_lists) TAM_HIP(tam::launch_export_tail(h->dt, node_ids, n, out, s));
    }
    return TAM_OK;
}

tam_status tam_valid_counts(const tam_handle *h, const int32_t *node_ids, int64_t n, int32_t *out, void *stream) {
    g_err.clear();
    if (!h) return fail(TAM_E_INVAL, "null handle");
    if (n < 0) return fail(TAM_E_INVAL, "n must be >= 0");
    if (n > 0 && (!node_ids || !out)) return fail(TAM_E_INVAL, "null device pointer");
    tam_status st = check_device_handle(h);
    if (st == TAM_OK) st = device_errors(h);
    if (st != TAM_OK) return st;
    if (is_lazy(h)) return fail(TAM_E_STATE, "rows built on demand keep no per-node valid sets");
    if (!h->dt.table && !h->lists_built) return fail(TAM_E_STATE, "the handle's valid lists are not built");
    if (n == 0) return TAM_OK;
    TAM_HIP(hipGetLastError());
    TAM_HIP(tam::launch_row_counts(h->dt, node_ids, n, out, static_cast<hipStream_t>(stream)));
    return TAM_OK;
}

tam_status tam_valid_pairs(const tam_handle *h, void *stream, int64_t *out) {
    g_err.clear();
    tam_status st = check_device_handle(h);
    if (st != TAM_OK) return st;
    if (!out) return fail(TAM_E_INVAL, "out is null");
    if (is_lazy(h)) return fail(TAM_E_STATE, "rows built on demand: no pass counts the valid pairs");
    hipStream_t s = static_cast<hipStream_t>(stream);
    // a table's marks (or, tail compression with lists, the probe pass) count
    // every pair, tails' too; plain lists count theirs
    const bool counted = h->dt.table || h->dt.tail_lists;
    std::vector<int32_t> part(counted ? (size_t)h->npairs : 0);
    int32_t listed = 0, errors = 0;
    if (counted)
        TAM_HIP(hipMemcpyAsync(part.data(), h->pairs, part.size() * sizeof(int32_t), hipMemcpyDeviceToHost, s));
    else
        TAM_HIP(hipMemcpyAsync(&listed, h->dt.row_ptr + h->N, sizeof(listed), hipMemcpyDeviceToHost, s));
    if (h->d_err) TAM_HIP(hipMemcpyAsync(&errors, h->d_err, sizeof(errors), hipMemcpyDeviceToHost, s));
    TAM_HIP(hipStreamSynchronize(s));
    if (errors != 0)
        return fail(TAM_E_DEVICE, "the device met " + std::to_string(errors) + " inconsistent trie-table entries");
    int64_t m = listed;
    for (int32_t x : part) m += x;
    *out = m;
    return TAM_OK;
}

tam_status tam_timing_get(const tam_handle *h, tam_timing *out) {
    if (!h || !out) return fail(TAM_E_INVAL, "null argument");
    *out = h->timing;
    if (h->have_events && h->events_recorded) {
        TAM_HIP(hipEventSynchronize(h->ev[3]));
        TAM_HIP(hipEventElapsedTime(&out->dev_zero_ms, h->ev[0], h->ev[1]));
        TAM_HIP(hipEventElapsedTime(&out->dev_mark_ms, h->ev[h->mark_from_ev4 ? 4 : 1], h->ev[2]));
        TAM_HIP(hipEventElapsedTime(&out->dev_lists_ms, h->ev[2], h->ev[3]));
        TAM_HIP(hipEventElapsedTime(&out->dev_total_ms, h->ev[0], h->ev[3]));
    }
    return TAM_OK;
}

void tam_destroy(tam_handle *h) {
    if (!h) return;
    destroy_handle(h);
}

}  // extern "C"
