// Internal definitions shared by the host code and the HIP kernels of libtam.
#pragma once

#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>
#include <cstdint>
#include <string>
#include <type_traits>
#include <utility>
#include <vector>

#include "../../include/tam.h"
#include "device_tables.hpp"

namespace tam {

// Large host tables of device compiles (the trie arrays that are uploaded)
// live in pinned memory taken from a process-wide pool and handed back when
// their handle is destroyed: their uploads are then direct DMA, and a compile
// that reuses a block faults no pages while filling it.  pinned_take returns
// null (ordinary memory is used) unless a PinnedScope is active on the
// calling thread, for blocks under kPinnedMin, or when pinning fails.
constexpr size_t kPinnedMin = size_t(1) << 20;
void *pinned_take(size_t bytes);
bool pinned_give(void *p);  // true if p is a pool block (now back in the pool)
struct PinnedScope {
    explicit PinnedScope(bool on);
    ~PinnedScope();
    PinnedScope(const PinnedScope &) = delete;
    PinnedScope &operator=(const PinnedScope &) = delete;
    bool prev;
};

// Pinned host words into which a handle's device error count is copied back
// (process-wide array, one slot per handle for its life); null when no slot
// is free or pinning fails, and the count is then only read back by calls
// that synchronise.
int32_t *err_slot_take();
void err_slot_give(int32_t *slot);

// An allocator whose value-initialisation (vector::resize) leaves elements of
// trivial types unset, so that large host tables are first touched by the
// threads that fill them instead of being zeroed serially beforehand.
template <typename T>
struct NoInitAlloc : std::allocator<T> {
    template <typename U>
    struct rebind {
        using other = NoInitAlloc<U>;
    };
    NoInitAlloc() = default;
    template <typename U>
    NoInitAlloc(const NoInitAlloc<U> &) noexcept {}
    T *allocate(size_t n) {
        if (n * sizeof(T) >= kPinnedMin)
            if (void *p = pinned_take(n * sizeof(T))) return static_cast<T *>(p);
        return std::allocator<T>::allocate(n);
    }
    void deallocate(T *p, size_t n) {
        if (n * sizeof(T) >= kPinnedMin && pinned_give(p)) return;
        std::allocator<T>::deallocate(p, n);
    }
    template <typename U>
    void construct(U *p) noexcept(std::is_nothrow_default_constructible<U>::value) {
        ::new ((void *)p) U;
    }
    template <typename U, typename... A>
    void construct(U *p, A &&...a) {
        ::new ((void *)p) U(std::forward<A>(a)...);
    }
};
template <typename T>
using hvec = std::vector<T, NoInitAlloc<T>>;

// Launchers (kernels.hip).  All return hipSuccess or the launch error.
hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t value, hipStream_t s);
hipError_t launch_probe(const DevTables &t, bool count, bool mark, int32_t *pairs, hipStream_t s);
// the list counts of the nodes [m0, m1) (lists only: t.table null; t.count of
// those nodes zeroed), nodes whose ancestors lie in the same range
hipError_t launch_count_range(const DevTables &t, int64_t m0, int64_t m1, hipStream_t s);
// node_at and depth of the string records [s0, s1) (records uploaded; the
// strings' earlier part-mates with shorter prefixes are in the same range)
hipError_t launch_node_at(const StrRec *strs, int64_t s0, int64_t s1, int64_t blob_bytes, int64_t N,
                          int32_t *node_at, int32_t *depth, int32_t *err, hipStream_t s);
// node_pos of the nodes [n0, n1) from the blob range [b0, b1) they were
// written in (node_at and depth of those ranges uploaded)
hipError_t launch_node_pos(const DevTables &t, int32_t *node_pos, int64_t n0, int64_t n1, int64_t b0, int64_t b1,
                           hipStream_t s);
// the child lists of every node (node_pos complete): child_off[N+1],
// child_node/child_byte/child_pos[N - roots], and child_at[blob_bytes] (the
// child range of the node at each blob position); tmp [N] and scan_tmp
// [scan_tmp_elems(N)] are scratch
hipError_t launch_child_lists(const DevTables &t, int32_t *child_off, int32_t *child_node, uint8_t *child_byte,
                              int32_t *child_pos, uint64_t *child_at, int32_t *tmp, int32_t *scan_tmp,
                              hipStream_t s);
hipError_t launch_scan(const DevTables &t, hipStream_t s);
hipError_t launch_zero(uint64_t *p, int64_t words, hipStream_t s);
int64_t mark_blocks(int64_t N);
hipError_t launch_fill_lists(const DevTables &t, hipStream_t s);
// Tail compression's row_of and tail_span of the nodes the strings [s0, s1)
// create, the roots' entries (root_rows: S (id, row) pairs; null: none) and
// row_at over the blob positions [b0, b1) (after row_of of every node there).
hipError_t launch_tail_tables(const StrRec *strs, const TailRec *trec, int64_t s0, int64_t s1,
                              const int32_t *root_rows, int64_t S, const int32_t *node_at, int64_t b0, int64_t b1,
                              int64_t N, int32_t *row_of, int32_t *tail_span, int32_t *row_at, int32_t *err,
                              hipStream_t s);
// nodes per block of the probe pass (its block b takes nodes [b * n, (b + 1) * n))
int64_t probe_nodes_per_block();
// tail compression without a table: the records of the listed hits (of
// `blocks` probe blocks) into the lists
hipError_t launch_fill_records(const DevTables &t, const RecGroups &rg, hipStream_t s);
// the probe pass's counts over nodes [m0, m1) (lists, tail lists with their
// records), with each block's valid pairs at pairs[blockIdx] (pairs may be null
// without tail lists)
// the probe pass (lists counted, records written) over groups [k0, k1) of the
// groups' grid, into pairs[blocks of those groups]
hipError_t launch_probe_groups(const DevTables &t, const RecGroups &rg, int64_t k0, int64_t k1, int32_t *pairs,
                               hipStream_t s);
hipError_t launch_rows(const DevTables &t, const int32_t *nodes, int64_t nrows, uint64_t *out,
                       int64_t out_stride_words, int64_t out_words, hipStream_t s);
hipError_t launch_apply(const DevTables &t, const int32_t *node_ids, int64_t B, void *logits,
                        int dtype, int64_t row_stride, hipStream_t s);
hipError_t launch_advance(const DevTables &t, const int32_t *node_ids, const int32_t *token_ids,
                          int64_t B, int32_t *out, hipStream_t s);
hipError_t launch_format(const DevTables &t, int32_t *pairs, hipStream_t s);
int64_t format_blocks(int64_t Wp);
// tam_format_rows_noalloc: the rows of positions 0..t.fmt_L+1 into out (stride
// words, W written per row) with the class bits staged in the static scratch;
// the pair count into *pairs_out when it is not null.  Allocates nothing.
hipError_t launch_format_noalloc(const DevTables &t, const uint8_t *classes_host, uint64_t *out, int64_t stride,
                                 int64_t *pairs_out, hipStream_t s);
hipError_t launch_export_dense(const DevTables &t, const int32_t *node_ids, int64_t n, uint64_t *out,
                               hipStream_t s);
// OR the tails' tokens (from the probe hits) into exported rows (tail compression)
hipError_t launch_export_tail(const DevTables &t, const int32_t *node_ids, int64_t n, uint64_t *out, hipStream_t s);
int64_t scan_tmp_elems(int64_t N);
// out[r] = |valid[node_ids[r]]| (0 for a dead node); not for rows built on demand
hipError_t launch_row_counts(const DevTables &t, const int32_t *node_ids, int64_t n, int32_t *out, hipStream_t s);
// one group of nb <= min(kLazyGroup, C) batch rows: cache lookup and
// replacement, rows of the misses built in the cache, then the masking
hipError_t launch_lazy_apply(const DevTables &t, const LazyDev &z, const int32_t *node_ids, int64_t nb,
                             void *logits, int dtype, int64_t row_stride, hipStream_t s);
// one group of nb <= kLazyGroup rows built straight into out[nb][W] (no cache)
hipError_t launch_lazy_export(const DevTables &t, const LazyDev &z, const int32_t *node_ids, int64_t nb,
                              uint64_t *out, hipStream_t s);
// empties the row cache
hipError_t launch_lazy_reset(const DevTables &t, const LazyDev &z, hipStream_t s);

}  // namespace tam

// ---------------------------------------------------------------------------
// A vocabulary's tables, built once per tokenizer and shared (reference
// counted) by every handle compiled against it.
// ---------------------------------------------------------------------------
struct tam_vocab {
    std::atomic<int> refs{1};
    uint32_t flags = 0;
    int device = 0;
    bool own_alloc = false;
    tam_allocator alloc{};

    int64_t V = 0, W = 0, max_tok_len = 0, device_bytes = 0;
    uint64_t len_mask = 0;
    double host_ms = 0, upload_ms = 0;

    // host tables
    tam::hvec<uint32_t> tok_off;
    tam::hvec<uint8_t> tok_blob;
    std::vector<uint8_t> len_present;
    tam::hvec<uint16_t> fps;          // the buckets, four 32-bit words each (as 16-bit halves)
    // pay / pay_hi: one entry per distinct string, by its number
    tam::hvec<tam::SlotPay> pay;
    tam::hvec<uint64_t> pay_hi;
    tam::hvec<int32_t> short_hits;
    tam::hvec<int32_t> dup_next;
    std::vector<int64_t> dup_cum;  // [max_len+1] see build_vocab (list size bound)

    // device copies (one arena)
    void *arena = nullptr;
    const uint32_t *d_tok_off = nullptr;
    const uint8_t *d_tok_blob = nullptr;
    const uint16_t *d_fps = nullptr;
    const tam::SlotPay *d_pay = nullptr;
    const uint64_t *d_pay_hi = nullptr;
    const int32_t *d_short_hits = nullptr;
    const int32_t *d_dup_next = nullptr;
    const uint8_t *d_len_present = nullptr;
    hipEvent_t ready = nullptr;  // recorded after the uploads
};

// ---------------------------------------------------------------------------
// The handle.
// ---------------------------------------------------------------------------
struct tam_handle {
    int terminator = 0x22;
    uint32_t flags = 0;
    int device = 0;
    bool own_alloc = false;
    tam_allocator alloc{};
    tam_vocab *vocab = nullptr;  // one reference held by the handle

    int64_t N = 0, S = 0, K_unique = 0, V = 0, W = 0, Wp = 0, edges = 0;
    int64_t blob_bytes = 0, entry_bound = 0, device_bytes = 0;

    // host trie tables
    tam::hvec<int32_t> roots, parent, depth;
    tam::hvec<tam::StrRec> strs;  // the blob's strings, in blob order
    tam::hvec<int32_t> sub_end;  // [N] with TAM_FLAG_LAZY_ROWS: one past the node's subtree
    tam::hvec<uint8_t> edge, is_final, blob;
    // tail compression (TAM_FLAG_TAIL_LISTS): see DevTables
    // row_of is kept on the host for the host API; tail_span and row_at only
    // for host-only handles.  A device compile lays all three out on the
    // device from tail_rec and root_rows.
    tam::hvec<int32_t> tail_span, row_of, row_at;
    bool tails = false;                  // tail compression's split is kept
    tam::hvec<tam::TailRec> tail_rec;    // [K_unique] one per blob string
    std::vector<int32_t> root_rows;      // [2 S] each set root's id and row_of
    int64_t dense_rows = 0;
    // tail compression without a table: the probe grid in the groups of nodes
    // the compile uploaded, each with its own buffer of records
    tam::RecGroups rec_groups{};
    tam::hvec<int32_t> rec_off;  // host copy of the groups' region offsets (see DevTables::rec_off)
    // character-position masks (tam_compile_format): L positions, their classes
    int64_t fmt_L = -1;
    std::vector<uint8_t> classes;
    int64_t npairs = 0;  // per-block valid-pair counters in `pairs`
    // rows built on demand (TAM_FLAG_LAZY_ROWS)
    tam::LazyDev lazy{};
    int64_t cache_rows = 0;

    std::vector<void *> dev_ptrs;  // everything allocated for this handle
    tam::DevTables dt{};

    // phase events: zero start, zero end, probe end, lists end, and probe start
    // (ev[4]) when the zero fill was enqueued earlier than the probe pass
    hipEvent_t ev[5] = {};
    bool mark_from_ev4 = false;
    int32_t *pairs = nullptr;       // device [mark_blocks(N)] per-block valid-pair counts
    bool lists_built = false;
    bool have_events = false;
    bool events_recorded = false;
    hipEvent_t work_done = nullptr;  // end of the last upload / device phase
    tam_timing timing{};
    // inconsistent table entries met on the device (DevTables::err), and the
    // pinned host word the compile and rebuild calls copy the count into
    int32_t *d_err = nullptr;
    int32_t *h_err = nullptr;
    // tam_layout_get: the position tables laid out on the host
    std::once_flag layout_once;
    tam::hvec<int32_t> lay_node_at, lay_depth, lay_node_pos, lay_parent;
    int64_t lay_errors = 0;
};
