// HIP kernels of libtam for gfx950 (CDNA4, wave64).
//
// Mask compile (Section 4.1, valid[n] for every trie node n):
//   k_zero   -- zero fill of the dense table (pure streaming stores).
//   k_probe  -- two lanes per non-root node m (in different waves), seven
//               hashed suffix lengths each: the last d <= min(depth(m), ℓ)
//               bytes of prefix(m) are hashed (read backwards from a 16-byte
//               register window) and looked up in the vocabulary table; a hit of
//               token t at d = |t| means t is valid at the ancestor d levels up,
//               because t's walk from there ends at m.  This is the paper's
//               crediting of a match to the node |t| bytes back (Section 4.2),
//               done for all nodes at once instead of along a DFS.  It keeps
//               the hits, ORs them into the zeroed table with 64-bit atomics
//               (nodes with a dense row) and, for lists, counts per node
//               (without a table under tail compression, it also records
//               each hit listed on a branching node with its rank).
//   k_scan_* -- exclusive prefix sum of the counts into row offsets.
//   k_fill   -- writes the hits' token ids into the per-node lists;
//               k_fill_records places the recorded hits instead.
//   k_rows   -- one wave per row builds rows in registers from the lists
//               (canonical rows of handles without a dense table).
// Serving (Section 2, Eq. 1 and the extended transition function):
//   k_apply  -- write-mostly masking of [B, V] logits (lists, tail rows, and
//               unaligned rows); k_apply_dense for dense-table rows, three
//               rows per block (two for small batches).
//   k_advance-- B byte walks over the child tables and along the strings of
//               the blob, one wave per row.
//   k_export_dense, k_export_tail -- canonical rows out of the dense table and
//               (tail compression) the probe's hits.
// Rows built on demand (lazy computation with a bounded cache, Appendix):
//   k_lazy_assign -- cache lookup and CLOCK replacement for a group of rows;
//               each miss takes a zero spare row, its victim becomes a spare.
//   k_lazy_probe -- the missing rows, from the suffix probes of the node's
//               subtree only, while the victims' rows are cleared; k_apply
//               then reads the cache.
// Trie tables on the device (from the blob and one record per string):
//   k_node_at, k_pos_init, k_first_pos, k_child_count, k_child_fill,
//   k_child_at, and under tail compression k_tail_nodes, k_root_rows, k_row_at.
// Fixed-format values (character-position masks):
//   k_format -- every word of the rows of positions 0..L+1, by wave ballots.
#include <hip/hip_runtime.h>

#include <climits>
#include <cstring>
#include <mutex>

#include "tam_internal.hpp"
#include "trie_layout.hpp"

namespace tam {
namespace {

constexpr int kBlock = 256;
constexpr int kWave = 64;
constexpr int kApplyUnits = 1;       // 16-byte chunks per thread in k_apply (measured best)
constexpr int kApplyRows = 3;        // rows per block of k_apply_dense (measured best on rows that change every call)
constexpr int64_t kApplyMinBlocks = 4096;  // fewer blocks than this with kApplyRows: two rows per block
// k_apply row sources: the dense table, the valid lists, or per row either
// (tail compression: dense rows for branching nodes, lists for tails)
constexpr int kApplyTable = 0, kApplyLists = 1, kApplyTail = 2;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct DevProps {
    int cus = 0;
};

DevProps props_for_current_device() {
    static DevProps cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return DevProps{256};
    if (cache[dev].cus == 0) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            cus = 256;
        cache[dev].cus = cus;
    }
    return cache[dev];
}

// p[i] = value, i < n: 16-byte stores where p is 16-byte aligned.
__global__ void __launch_bounds__(kBlock) k_fill_i32(int32_t *p, int64_t n, int32_t value) {
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    const int64_t i0 = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    int64_t done = 0;
    if ((reinterpret_cast<uintptr_t>(p) & 15) == 0) {
        const uint32_t u = (uint32_t)value;
        const u32x4 v4{u, u, u, u};
        done = n / 4;
        for (int64_t i = i0; i < done; i += stride) reinterpret_cast<u32x4 *>(p)[i] = v4;
        done *= 4;
    }
    for (int64_t i = done + i0; i < n; i += stride) p[i] = value;
}

// ---------------------------------------------------------------- probes ---

// Reversed 16-byte path window ending at blob[pos]: byte k of (lo, hi) is
// blob[pos - k].  Five aligned dword loads; the blob carries 16 zero bytes on
// both sides, so they stay inside it.
__device__ __forceinline__ void load_window(const uint8_t *blob, int64_t pos, uint64_t &lo, uint64_t &hi) {
    const int64_t ws = pos - (kWin - 1);
    const int64_t a = ws & ~int64_t(3);
    const uint32_t *w = reinterpret_cast<const uint32_t *>(blob + a);
    const uint32_t w0 = w[0], w1 = w[1], w2 = w[2], w3 = w[3], w4 = w[4];
    const uint32_t sh = (uint32_t)(ws - a) * 8u;
    const uint32_t x0 = (uint32_t)((((uint64_t)w1 << 32) | w0) >> sh);
    const uint32_t x1 = (uint32_t)((((uint64_t)w2 << 32) | w1) >> sh);
    const uint32_t x2 = (uint32_t)((((uint64_t)w3 << 32) | w2) >> sh);
    const uint32_t x3 = (uint32_t)((((uint64_t)w4 << 32) | w3) >> sh);
    lo = __builtin_bswap64(((uint64_t)x3 << 32) | x2);
    hi = __builtin_bswap64(((uint64_t)x1 << 32) | x0);
}

__device__ __forceinline__ uint32_t window_byte(uint64_t lo, uint64_t hi, int k) {
    return (uint32_t)((k < 8 ? lo >> (8 * k) : hi >> (8 * (k - 8))) & 0xffu);
}

__device__ __forceinline__ bool has_len(const DevTables &t, int d) {
    return d < 64 ? ((t.len_mask >> d) & 1ull) != 0 : t.len_present[d] != 0;
}

// The first min(d, 8) reversed bytes of a suffix of d bytes (lo) equal the slot's.
__device__ __forceinline__ bool lo_ok(uint64_t lo, const SlotPay &r, int d) {
    return (d >= 8 ? lo : (lo & (~0ull >> (64 - 8 * d)))) == r.lo;
}

// Reversed bytes 8 .. min(d, 16) - 1 of the suffix (hi) equal the slot's (d > 8).
__device__ __forceinline__ bool hi_ok(uint64_t hi, uint64_t rhi, int d) {
    return (d >= 16 ? hi : (hi & (~0ull >> (64 - 8 * (d - 8))))) == rhi;
}

__device__ __forceinline__ uint64_t home_bucket(const DevTables &t, uint64_t key) {
    return (key & t.slot_mask) / kBucket;
}

// A bucket: its kBucket fingerprints and its base, in one 16-byte load.
struct Bucket {
    u32x4 q[kBucket / 8];
};

__device__ __forceinline__ Bucket load_bucket(const DevTables &t, uint64_t b) {
    const u32x4 *p = reinterpret_cast<const u32x4 *>(t.fps + b * kBucket);
    Bucket k;
#pragma unroll
    for (int i = 0; i < kBucket / 8; ++i) k.q[i] = p[i];
    return k;
}

// The number of the bucket's first string (byte i in bits 24..31 of word i).
__device__ __forceinline__ uint32_t bucket_base(const Bucket &bk) {
    return (bk.q[0].x >> 24) | ((bk.q[0].y >> 24) << 8) | ((bk.q[0].z >> 24) << 16) | (bk.q[0].w & 0xff000000u);
}

// Bit i of *match: slot i holds fingerprint fp; bit i of *empty: slot i is empty.
__device__ __forceinline__ void bucket_masks(const Bucket &bk, uint32_t fp, uint32_t *match, uint32_t *empty) {
    uint32_t mm = 0, ee = 0;
    const uint32_t w[4] = {bk.q[0].x, bk.q[0].y, bk.q[0].z, bk.q[0].w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t a = w[i] & 0xfffu, b = (w[i] >> 12) & 0xfffu;
        mm |= ((a == fp ? 1u : 0u) | (b == fp ? 2u : 0u)) << (2 * i);
        ee |= ((a == 0u ? 1u : 0u) | (b == 0u ? 2u : 0u)) << (2 * i);
    }
    *match = mm;
    *empty = ee;
}

// The suffix of d bytes ending at blob[pos] (window (lo, hi)) equals slot s,
// whose payload m and (d > 8) pay_hi word mhi have just been read: its first 8
// reversed bytes, bytes 8..15, then (d > 16) the bytes beyond the window.
__device__ __forceinline__ bool slot_equals(const DevTables &t, const SlotPay &m, uint64_t mhi, int d, uint64_t lo,
                                            uint64_t hi, int64_t pos) {
    if ((int)m.len != d || !lo_ok(lo, m, d)) return false;
    if (d > 8 && !hi_ok(hi, mhi, d)) return false;
    if (d > kWin) {
        const uint8_t *tb = t.tok_blob + t.tok_off[m.first];
        const uint8_t *pb = t.blob + (pos - d + 1);
        for (int k = 0; k < d - kWin; ++k)
            if (tb[k] != pb[k]) return false;
    }
    return true;
}

// The hit of a suffix of d <= kShortLen bytes (last byte b0, the one before it b1).
__device__ __forceinline__ int32_t short_hit(const DevTables &t, int d, uint32_t b0, uint32_t b1) {
    return t.short_hits[short_index(d, b0, b1)];
}

// Slot (0..kBucket-1) of the first fingerprint fp in bucket bk, or -1.  The
// eight 12-bit fingerprints are compared two per word: a field of
// x = (w ^ fp:fp) & 0xffffff is zero exactly where the fingerprint matches, and
// (x - 0x001001) & ~x sets bit 11 of a zero field; a borrow out of a zero low
// field can flag the high field too, but the lowest flagged field is always a
// true match.  *open: the bucket's last slot is empty, so the bucket was never
// full and a key whose home it is lies in it (slots fill in order and are
// never cleared).
__device__ __forceinline__ int first_match(const Bucket &bk, uint32_t fp, bool *open) {
    const uint32_t fp2 = fp | (fp << 12);
    const uint32_t w[4] = {bk.q[0].x, bk.q[0].y, bk.q[0].z, bk.q[0].w};
    int s = -1;
#pragma unroll
    for (int i = 3; i >= 0; --i) {
        const uint32_t x = (w[i] ^ fp2) & 0xffffffu;
        const uint32_t z = (x - 0x001001u) & ~x & 0x800800u;
        if (z) s = 2 * i + ((z & 0x800u) ? 0 : 1);
    }
    *open = ((w[3] >> 12) & 0xfffu) == 0u;
    return s;
}

// The number of the string of d bytes that ends at blob[pos] (reversed
// window (lo, hi)), with home bucket b and fingerprint fp, or -1; its payload
// goes to *pay.  Buckets are scanned from b until one with an empty slot (load
// <= 1/4 guarantees one exists): a key sits in a later bucket only if every
// bucket before it was full when it was inserted.
__device__ __forceinline__ int32_t probe_from(const DevTables &t, uint64_t b, uint32_t fp, int d, uint64_t lo,
                                              uint64_t hi, int64_t pos, SlotPay *pay) {
    const uint64_t bmask = t.slot_mask / kBucket;
    for (;;) {
        uint32_t match, empty;
        const Bucket bk = load_bucket(t, b);
        bucket_masks(bk, fp, &match, &empty);
        const uint32_t base = bucket_base(bk);
        while (match) {
            const int i = __builtin_ctz(match);
            match &= match - 1;
            const int32_t sl = (int32_t)(base + (uint32_t)i);
            const SlotPay m = t.pay[sl];
            const uint64_t mhi = d > 8 ? t.pay_hi[sl] : 0ull;
            if (slot_equals(t, m, mhi, d, lo, hi, pos)) {
                *pay = m;
                return sl;
            }
        }
        if (empty) return -1;
        b = (b + 1) & bmask;
    }
}

// The same from the string's key (its hash).
__device__ __forceinline__ int32_t probe(const DevTables &t, uint64_t key, int d, uint64_t lo, uint64_t hi,
                                         int64_t pos, SlotPay *pay) {
    return probe_from(t, home_bucket(t, key), fingerprint(key), d, lo, hi, pos, pay);
}

// A node's suffix lengths are split over kProbeLanes lanes: lane g hashes the
// lengths kShortLen + 1 + g * kLaneLens .. kShortLen + (g + 1) * kLaneLens,
// lane 0 also reads the short ones.
constexpr int kProbeLanes = 2;
constexpr int kLaneLens = (kWin - kShortLen) / kProbeLanes;
static_assert(kLaneLens * kProbeLanes == kWin - kShortLen, "lengths split evenly over the lanes");

// The hits (hit_of_slot, or -1) of the suffixes of length d = kD0 + 1 ..
// kD0 + kLaneLens (and, for lane 0, 1 .. kShortLen) of the path ending at
// blob[pos], window (lo, hi); only d <= Lw <= kWin are probed.  hit[i] is the
// hit of length kD0 + 1 + i (lane 0: hit[kLaneLens + d - 1] for the short d).
// The hash state advances one byte per length, and the lengths are unrolled,
// so every byte extract and mask is a constant.  The home buckets of the
// lane's lengths are loaded together, then the payload (and for lengths beyond
// 8 bytes the pay_hi word) of each first fingerprint match, so the lane waits
// for two memory round trips.  Bit i of the returned mask marks a length its
// home bucket does not settle (a full bucket, or a failed first match): the
// caller probes it with the general probe.
template <int kD0>
__device__ __forceinline__ uint32_t probe_lengths(const DevTables &t, int Lw, uint64_t lo, uint64_t hi,
                                                  int32_t (&hit)[kLaneLens + kShortLen]) {
    if (kD0 == kShortLen) {
        hit[kLaneLens] = short_hit(t, 1, window_byte(lo, hi, 0), 0u);
        hit[kLaneLens + 1] = Lw >= 2 ? short_hit(t, 2, window_byte(lo, hi, 0), window_byte(lo, hi, 1)) : -1;
    } else {
        hit[kLaneLens] = hit[kLaneLens + 1] = -1;
    }
    uint32_t bidx[kLaneLens], fp[kLaneLens];
    bool act[kLaneLens];
    uint32_t h = kHashSeed;
#pragma unroll
    for (int k = 0; k < kD0 + kLaneLens; ++k) {
        h = hash_step(h, window_byte(lo, hi, k));
        if (k >= kD0) {
            const int j = k - kD0, d = k + 1;
            const uint64_t key = hash_final(h);
            bidx[j] = (uint32_t)home_bucket(t, key);
            fp[j] = fingerprint(key);
            act[j] = d <= Lw && has_len(t, d);
        }
    }
    Bucket bk[kLaneLens];
#pragma unroll
    for (int j = 0; j < kLaneLens; ++j)
        if (act[j]) bk[j] = load_bucket(t, bidx[j]);
    int32_t slot[kLaneLens];
    uint32_t pending = 0;
#pragma unroll
    for (int j = 0; j < kLaneLens; ++j) {
        slot[j] = -1;
        if (act[j]) {
            bool open;
            const int sl = first_match(bk[j], fp[j], &open);
            if (sl >= 0) slot[j] = (int32_t)(bucket_base(bk[j]) + (uint32_t)sl);
            if (sl >= 0 || !open) pending |= 1u << j;  // cleared below when the match holds
        }
    }
    SlotPay p[kLaneLens];
    uint64_t phi[kLaneLens];
#pragma unroll
    for (int j = 0; j < kLaneLens; ++j) {
        phi[j] = 0;
        if (slot[j] >= 0) {
            p[j] = t.pay[slot[j]];
            if (kD0 + j + 1 > 8) phi[j] = t.pay_hi[slot[j]];
        }
    }
#pragma unroll
    for (int j = 0; j < kLaneLens; ++j) {
        const int d = kD0 + j + 1;
        hit[j] = -1;
        if (slot[j] >= 0 && (int)p[j].len == d && lo_ok(lo, p[j], d) && (d <= 8 || hi_ok(hi, phi[j], d))) {
            hit[j] = hit_of_slot(slot[j], p[j].first, p[j].count);
            pending &= ~(1u << j);
        }
    }
    return pending;
}

// Writes the token ids of hit x (see hit_of_slot) into the list of node n.
__device__ __forceinline__ void emit(const DevTables &t, int32_t x, int32_t n) {
    if (x >= 0) {
        t.entries[t.row_ptr[n] + atomicAdd(&t.cursor[n], 1)] = x;
        return;
    }
    const SlotPay m = t.pay[-2 - x];
    const int32_t at = t.row_ptr[n] + atomicAdd(&t.cursor[n], (int32_t)m.count);
    int32_t v = m.first;
    for (int k = 0; k < (int)m.count; ++k) {
        t.entries[at + k] = v;
        v = t.dup_next[v];
    }
}

// Number of token ids of hit x.
__device__ __forceinline__ int32_t hit_count(const DevTables &t, int32_t x) {
    return x >= 0 ? 1 : (x == -1 ? 0 : (int32_t)t.pay[-2 - x].count);
}

// Calls f(hit, d) for every token string ending at node m longer than the
// window (d > 16), probing those lengths again (vocabularies rarely have them).
template <typename F>
__device__ __forceinline__ void long_hits(const DevTables &t, int64_t pos, int L, F &&f) {
    uint64_t lo, hi;
    load_window(t.blob, pos, lo, hi);
    uint32_t h = kHashSeed;
    for (int d = 1; d <= kWin; ++d) h = hash_step(h, window_byte(lo, hi, d - 1));
    for (int d = kWin + 1; d <= L; ++d) {
        h = hash_step(h, t.blob[pos - d + 1]);
        if (!has_len(t, d)) continue;
        SlotPay mt;
        const int32_t s = probe(t, hash_final(h), d, lo, hi, pos, &mt);
        if (s >= 0) f(hit_of_slot(s, mt.first, mt.count), d);
    }
}

// The group of probe block b in the groups' grid (0 without groups), and an
// entry of a group array: block-uniform selects, so that the kernel argument is
// never indexed dynamically (which would copy it to scratch memory).
__device__ __forceinline__ int group_of(const RecGroups &rg, int64_t b) {
    return (rg.n > 1 && b >= rg.blk0[1]) + (rg.n > 2 && b >= rg.blk0[2]) + (rg.n > 3 && b >= rg.blk0[3]);
}
template <typename T>
__device__ __forceinline__ T pick(const T (&a)[kMaxRecGroups], int k) {
    return k == 0 ? a[0] : k == 1 ? a[1] : k == 2 ? a[2] : a[3];
}
template <typename T>
__device__ __forceinline__ T pick(const T (&a)[kMaxRecGroups + 1], int k) {
    return k == 0 ? a[0] : k == 1 ? a[1] : k == 2 ? a[2] : a[3];
}

// Hits at distance d <= list_span(m) above node m belong to the valid lists:
// all of them with lists only, the tail ancestors of m with tail compression
// (where the lists hold only tokens longer than the window).
__device__ __forceinline__ int list_span(const DevTables &t, int64_t m) {
    if (t.tail_span) return t.tail_span[m];
    return t.table ? 0 : INT_MAX;
}

// Probe pass: kProbeLanes lanes per node m, in different waves (lane g: the
// suffix lengths of probe_lengths<kShortLen + g * kLaneLens>), all d <= min(depth, ℓ, 16) of
// prefix(m).  The suffix of length d equal to token t means t is valid at the
// ancestor d levels up, node_at[pos - d].  The hit (hit_of_slot: the token
// id, or the slot of a string with several ids, or -1) goes to hits[d-1][m];
// the tails of tail compression read their tokens back from there.  Longer
// tokens are probed again where needed (long_hits, by the last lane).  All
// loads of a lane's main path are issued before its first store or atomic
// (loads, stores and atomics share one vector-memory counter here); the rare
// lengths a home bucket does not settle follow, one at a time.
//   do_mark (a table): every hit whose ancestor has a dense row (row_at of its
//     blob position; not a tail) is OR-ed into the zeroed table with a 64-bit
//     atomic, and each block writes the number of valid (node, token) pairs its
//     hits make, tails included, into pairs[blockIdx.x].
//   kCount (lists): the listed hits are counted per node: every hit (lists
//     only); with tail compression and a table, the tails' hits of tokens
//     longer than the window; with tail compression and no table (tail_lists),
//     also every hit on a branching node, and each block then writes its
//     number of valid pairs as do_mark does.
// The grid covers the nodes [m0, m1): every node of the handle, or (lists of a
// forest) one group of whole sets, whose nodes' ancestors are in the group too.
// With tail compression and no table the groups' grid (rg) decides instead:
// this launch runs its probe blocks blk + blockIdx.x.
template <bool kCount>
__global__ void __launch_bounds__(kBlock) k_probe(DevTables t, int64_t m0, int64_t m1, int do_mark,
                                                  int32_t *__restrict__ pairs, RecGroups rg, int64_t blk) {
    constexpr int64_t kPer = kBlock / kProbeLanes;  // nodes per block
    const int64_t gb = blk + blockIdx.x;            // the block in the grid of pairs (and rec_cnt)
    const int gk = group_of(rg, gb);
    if (kCount && t.tail_lists) {
        m0 = pick(rg.n_lo, gk) + (gb - pick(rg.blk0, gk)) * kPer;
        m1 = pick(rg.n_hi, gk);
    } else {
        m0 += (int64_t)blockIdx.x * kPer;
    }
    // lane group g is uniform over a wave (so a wave runs one unrolled path):
    // wave w of the block takes lengths group w % kProbeLanes of nodes
    // (w / kProbeLanes) * 64 .. + 63 of the block's kPer
    const int wv = (int)threadIdx.x / kWave;
    const int g = wv % kProbeLanes;
    const int64_t m = m0 + (wv / kProbeLanes) * kWave + (threadIdx.x & (kWave - 1));
    int32_t found = 0;
    // tail_lists: the block's region of its group's records
    __shared__ int32_t s_rec;  // records the block has written
    int32_t *rec = nullptr;
    int32_t reg0 = 0, reg1 = 0;
    if (kCount && t.tail_lists) {
        const int64_t o = pick(rg.off0, gk) + (gb - pick(rg.blk0, gk));
        rec = pick(rg.rec, gk);
        reg0 = t.rec_off[o];
        reg1 = t.rec_off[o + 1];
        if (threadIdx.x == 0) s_rec = 0;
        __syncthreads();
    }
    const int64_t pos = m < m1 ? t.node_pos[m] : -1;  // a root ends no token
    if (pos >= 0) {
        const int L = min(t.depth[m], t.max_len);
        const int Lw = min(L, kWin);
        const int lspan = kCount ? list_span(t, m) : 0;              // listed up to here
        const int sspan = t.row_of ? 0 : lspan;                      // short hits listed up to here
        const int mspan = do_mark ? (t.tail_span ? t.tail_span[m] : 0) : INT_MAX;  // marked beyond
        const int bspan = kCount && t.tail_lists ? t.tail_span[m] : INT_MAX;      // (no table) listed beyond
        unsigned long long *table = reinterpret_cast<unsigned long long *>(t.table);
        // one hit of length d: the pairs it makes, marked at the table row of
        // its ancestor (>= 0), counted for its list node (>= 0); without a
        // table (tail_lists) a listed hit takes its rank in the node's list and
        // leaves a record in the block's region
        auto take = [&](int32_t hx, int32_t row, int32_t ln) {
            if (kCount && t.tail_lists) {
                const int32_t c = hx >= 0 ? 1 : (int32_t)t.pay[-2 - hx].count;
                found += c;
                if (ln < 0) return;
                const int32_t rank = atomicAdd(&t.count[ln], c);
                const int32_t at = reg0 + atomicAdd(&s_rec, 1);
                if (at >= reg1) {  // more records than the host's bound
                    atomicAdd(t.err, 1);
                    return;
                }
                rec[3 * (int64_t)at] = ln;
                rec[3 * (int64_t)at + 1] = rank;
                rec[3 * (int64_t)at + 2] = hx;
                return;
            }
            if (hx >= 0) {
                if (row >= 0) atomicOr(table + (int64_t)row * t.Wp + (hx >> 6), 1ull << (hx & 63));
                if (ln >= 0) atomicAdd(&t.count[ln], 1);
                ++found;
                return;
            }
            const SlotPay mt = t.pay[-2 - hx];  // a string with several token ids (rare)
            if (ln >= 0) atomicAdd(&t.count[ln], (int32_t)mt.count);
            found += mt.count;
            if (row < 0) return;
            int32_t v = mt.first;
            for (int k = 0; k < (int)mt.count; ++k) {
                atomicOr(table + (int64_t)row * t.Wp + (v >> 6), 1ull << (v & 63));
                v = t.dup_next[v];
            }
        };
        auto list_node = [&](int d) { return kCount && (d <= sspan || d > bspan) ? t.node_at[pos - d] : -1; };
        auto mark_row = [&](int d) { return d > mspan ? t.row_at[pos - d] : -1; };
        uint64_t lo, hi;
        load_window(t.blob, pos, lo, hi);
        // hit[i]: length d0 + 1 + i; hit[kLaneLens + k]: the short length k + 1 (lane 0)
        int32_t hit[kLaneLens + kShortLen];
        const int d0 = g == 0 ? kShortLen : kShortLen + kLaneLens;
        const uint32_t pending = g == 0 ? probe_lengths<kShortLen>(t, Lw, lo, hi, hit)
                                        : probe_lengths<kShortLen + kLaneLens>(t, Lw, lo, hi, hit);
        int32_t n[kLaneLens + kShortLen], r[kLaneLens + kShortLen];
#pragma unroll
        for (int k = 0; k < kLaneLens + kShortLen; ++k) {
            const int d = k < kLaneLens ? d0 + 1 + k : k - kLaneLens + 1;
            n[k] = hit[k] != -1 ? list_node(d) : -1;
            r[k] = hit[k] != -1 ? mark_row(d) : -1;
        }
        int32_t *hrow = t.hits + m;
#pragma unroll
        for (int k = 0; k < kLaneLens + kShortLen; ++k) {
            const int d = k < kLaneLens ? d0 + 1 + k : k - kLaneLens + 1;
            if (d <= Lw && (k < kLaneLens || g == 0)) hrow[(int64_t)(d - 1) * t.N] = hit[k];
        }
#pragma unroll
        for (int k = 0; k < kLaneLens + kShortLen; ++k)
            if (hit[k] != -1) take(hit[k], r[k], n[k]);
        // lengths the home bucket did not settle (rare): the general probe
        for (uint32_t pm = pending; pm; pm &= pm - 1) {
            const int d = d0 + 1 + __builtin_ctz(pm);
            uint32_t hh = kHashSeed;
            for (int k = 0; k < d; ++k) hh = hash_step(hh, window_byte(lo, hi, k));
            SlotPay mt;
            const int32_t sl = probe(t, hash_final(hh), d, lo, hi, pos, &mt);
            if (sl < 0) continue;
            const int32_t hx = hit_of_slot(sl, mt.first, mt.count);
            hrow[(int64_t)(d - 1) * t.N] = hx;
            take(hx, mark_row(d), list_node(d));
        }
        // tokens longer than the window (rare), by the last lane
        if (g == kProbeLanes - 1 && L > kWin && (do_mark || lspan > kWin || (kCount && t.tail_lists)))
            long_hits(t, pos, L, [&](int32_t hx, int d) {
                take(hx, d > mspan ? t.row_at[pos - d] : -1,
                     d <= lspan || (kCount && t.tail_lists) ? t.node_at[pos - d] : -1);
            });
    }
    if (!do_mark && !(kCount && t.tail_lists)) return;
    // block sum of the pairs
    __shared__ int32_t wsum[kBlock / kWave];
    for (int o = kWave / 2; o > 0; o >>= 1) found += __shfl_xor(found, o, kWave);
    if ((threadIdx.x & (kWave - 1)) == 0) wsum[threadIdx.x / kWave] = found;
    __syncthreads();
    if (threadIdx.x == 0) {
        int32_t total = 0;
        for (int w = 0; w < kBlock / kWave; ++w) total += wsum[w];
        pairs[gb] = total;
        if (kCount && t.tail_lists) t.rec_cnt[gb] = s_rec;
    }
}

// The records of probe block blockIdx.x of the groups' grid (tail compression
// without a table): each listed hit's ids go to its node's list at
// row_ptr[node] + rank.
__global__ void __launch_bounds__(kWave) k_fill_records(DevTables t, RecGroups rg) {
    const int64_t b = blockIdx.x;
    const int gk = group_of(rg, b);
    const int64_t o = pick(rg.off0, gk) + (b - pick(rg.blk0, gk));
    const int64_t r0 = t.rec_off[o];
    const int32_t n = min(t.rec_cnt[b], t.rec_off[o + 1] - t.rec_off[o]);
    const int32_t *rec = pick(rg.rec, gk);
    for (int32_t i = threadIdx.x; i < n; i += kWave) {
        const int32_t *r = rec + 3 * (r0 + i);
        const int32_t ln = r[0], rank = r[1], hx = r[2];
        const int64_t at = (int64_t)t.row_ptr[ln] + rank;
        if (hx >= 0) {
            t.entries[at] = hx;
            continue;
        }
        const SlotPay pm = t.pay[-2 - hx];  // a string with several token ids
        int32_t v = pm.first;
        for (int k = 0; k < (int)pm.count; ++k) {
            t.entries[at + k] = v;
            v = t.dup_next[v];
        }
    }
}

// Fill pass (lists): the hits' token ids written into the per-node lists (with
// tail compression those of tokens longer than the window, and without a
// table also those on branching nodes).
__global__ void __launch_bounds__(kBlock) k_fill(DevTables t) {
    const int64_t m = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (m >= t.N) return;
    const int64_t pos = t.node_pos[m];
    if (pos < 0) return;
    const int L = min(t.depth[m], t.max_len);
    const int Lw = min(L, kWin);
    const int span = list_span(t, m);
    const int Ls = t.row_of ? 0 : min(Lw, span);  // tail compression lists long hits only
    const int bspan = t.tail_lists ? t.tail_span[m] : INT_MAX;  // no table: branching nodes' hits too
    int32_t s[kWin];
#pragma unroll
    for (int d = 1; d <= kWin; ++d)
        s[d - 1] = d <= Lw && (d <= Ls || d > bspan) ? t.hits[(int64_t)(d - 1) * t.N + m] : -1;
#pragma unroll
    for (int d = 1; d <= kWin; ++d)
        if (s[d - 1] != -1) emit(t, s[d - 1], t.node_at[pos - d]);
    if (L > kWin && (span > kWin || t.tail_lists))
        long_hits(t, pos, L, [&](int32_t hx, int d) {
            if (d <= span || t.tail_lists) emit(t, hx, t.node_at[pos - d]);
        });
}

// Zero fill of n16 16-byte chunks: one chunk per thread, 256 threads (4 KiB)
// per block, plain stores and no grid-stride loop.  Measured on MI355X this
// shape sustains ~6.8 TB/s; more chunks per thread, non-temporal stores or a
// persistent grid-stride grid all write slower, because the blocks in flight
// then no longer sweep one compact window of memory.
__global__ void __launch_bounds__(kBlock) k_zero(u32x4 *__restrict__ p, int64_t n16) {
    const int64_t c = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (c < n16) p[c] = u32x4{0u, 0u, 0u, 0u};
}

// ------------------------------------------------------------------ scan ---

constexpr int kScanItems = 16;
constexpr int kScanTile = kBlock * kScanItems;  // elements per block

// Exclusive scan of one value per thread over the 256-thread block.
__device__ __forceinline__ int32_t block_exclusive_scan(int32_t x, int32_t *total) {
    __shared__ int32_t wave_sums[kBlock / kWave];
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    int32_t inc = x;
    for (int o = 1; o < kWave; o <<= 1) {
        const int32_t y = __shfl_up(inc, o, kWave);
        if (lane >= o) inc += y;
    }
    if (lane == kWave - 1) wave_sums[wid] = inc;
    __syncthreads();
    int32_t before = 0, all = 0;
    for (int w = 0; w < kBlock / kWave; ++w) {
        if (w < wid) before += wave_sums[w];
        all += wave_sums[w];
    }
    __syncthreads();
    *total = all;
    return before + inc - x;
}

// A thread's kScanItems consecutive values from base (0 past n): four 16-byte
// loads where the whole run is in range and aligned.
__device__ __forceinline__ void scan_load(const int32_t *in, int64_t base, int64_t n, int32_t (&v)[kScanItems]) {
    if (base + kScanItems <= n && (reinterpret_cast<uintptr_t>(in + base) & 15) == 0) {
#pragma unroll
        for (int q = 0; q < kScanItems / 4; ++q) {
            const u32x4 x = reinterpret_cast<const u32x4 *>(in + base)[q];
            v[4 * q] = (int32_t)x.x;
            v[4 * q + 1] = (int32_t)x.y;
            v[4 * q + 2] = (int32_t)x.z;
            v[4 * q + 3] = (int32_t)x.w;
        }
        return;
    }
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) v[k] = base + k < n ? in[base + k] : 0;
}

__global__ void __launch_bounds__(kBlock) k_scan_blocks(const int32_t *in, int64_t n, int32_t *sums) {
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int32_t v[kScanItems];
    scan_load(in, base, n, v);
    int32_t s = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) s += v[k];
    int32_t total;
    block_exclusive_scan(s, &total);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// One block: exclusive scan of the nb block sums in place; grand total -> *total_out.
// (Used when the block sums are more than one block of the apply pass adds up.)
__global__ void __launch_bounds__(kBlock) k_scan_top(int32_t *sums, int64_t nb, int32_t *total_out) {
    int32_t carry = 0;
    for (int64_t base = 0; base < nb; base += kScanTile) {
        const int64_t b0 = base + (int64_t)threadIdx.x * kScanItems;
        int32_t v[kScanItems];
        int32_t s = 0;
        for (int k = 0; k < kScanItems; ++k) {
            v[k] = b0 + k < nb ? sums[b0 + k] : 0;
            s += v[k];
        }
        int32_t total;
        int32_t run = carry + block_exclusive_scan(s, &total);
        for (int k = 0; k < kScanItems; ++k) {
            if (b0 + k < nb) sums[b0 + k] = run;
            run += v[k];
        }
        carry += total;
        __syncthreads();
    }
    if (threadIdx.x == 0) *total_out = carry;
}

// The scan's second pass.  own_prefix (nb <= kScanTile): each block adds up the
// block sums before its own (at most kScanTile of them, from L2) and the last
// block writes the grand total; otherwise sums holds k_scan_top's prefixes.
__global__ void __launch_bounds__(kBlock) k_scan_apply(const int32_t *in, int64_t n, const int32_t *sums,
                                                       int own_prefix, int32_t *out, int32_t *total_out) {
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int32_t v[kScanItems];
    scan_load(in, base, n, v);
    int32_t s = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) s += v[k];
    int32_t prefix, total;
    if (own_prefix) {
        int32_t p = 0;
        for (int64_t j = threadIdx.x; j < (int64_t)blockIdx.x; j += kBlock) p += sums[j];
        block_exclusive_scan(p, &prefix);
    } else {
        prefix = sums[blockIdx.x];
    }
    int32_t run = prefix + block_exclusive_scan(s, &total);
    if (own_prefix && blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) *total_out = prefix + total;
    int32_t o[kScanItems];
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        o[k] = run;
        run += v[k];
    }
    if (base + kScanItems <= n && (reinterpret_cast<uintptr_t>(out + base) & 15) == 0) {
#pragma unroll
        for (int q = 0; q < kScanItems / 4; ++q)
            reinterpret_cast<u32x4 *>(out + base)[q] =
                u32x4{(uint32_t)o[4 * q], (uint32_t)o[4 * q + 1], (uint32_t)o[4 * q + 2], (uint32_t)o[4 * q + 3]};
    } else {
#pragma unroll
        for (int k = 0; k < kScanItems; ++k)
            if (base + k < n) out[base + k] = o[k];
    }
}

// ------------------------------------------------------------ row images ---

constexpr int kRowSlots = 8;       // chunks per lane per pass
constexpr int kRowRegBatches = 4;  // 64-entry batches of a row's list held in VGPRs

// One wave per row (grid-stride over rows): the row's list (up to 256 ids) is
// loaded into VGPRs once; each pass then builds 8 chunks per lane in registers
// from it and streams them with non-temporal stores, 64 chunks (1 KiB for
// 16-byte chunks) per store instruction.  No LDS, no barriers: every wave keeps
// a whole row of stores in flight.  Row r is node nodes[r] (r if nodes is
// null), written at out + r*out_stride; a dead or out-of-range node gives a
// zero row.  CW = 64-bit words per chunk (2: 16-byte stores, 1: 8-byte).
template <int CW>
__global__ void __launch_bounds__(kBlock) k_rows(const int32_t *__restrict__ row_ptr,
                                                 const int32_t *__restrict__ entries,
                                                 const int32_t *__restrict__ nodes, int64_t nrows, int64_t N,
                                                 uint64_t *__restrict__ out, int64_t out_stride,
                                                 int64_t out_words) {
    typedef uint32_t chunk_t __attribute__((ext_vector_type(2 * CW)));
    constexpr int kBits = 64 * CW;             // tokens per chunk
    constexpr int kPass = kWave * kRowSlots;   // chunks per pass
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t nwaves = (int64_t)gridDim.x * (kBlock / kWave);
    const int64_t nchunks = out_words / CW;
    for (int64_t r = ((int64_t)blockIdx.x * kBlock + threadIdx.x) / kWave; r < nrows; r += nwaves) {
        const int64_t n = nodes ? (int64_t)nodes[r] : r;
        int32_t b = 0, e = 0;
        if (n >= 0 && n < N) {
            b = row_ptr[n];
            e = row_ptr[n + 1];
        }
        int32_t ent[kRowRegBatches];
#pragma unroll
        for (int i = 0; i < kRowRegBatches; ++i) {
            const int32_t k = b + i * kWave + lane;
            ent[i] = k < e ? entries[k] : 0;
        }
        const int32_t E = e - b;
        chunk_t *dst = reinterpret_cast<chunk_t *>(out + r * out_stride);
        for (int64_t c0 = 0; c0 < nchunks; c0 += kPass) {
            chunk_t val[kRowSlots];
#pragma unroll
            for (int k = 0; k < kRowSlots; ++k) val[k] = chunk_t(0u);
            for (int32_t j = 0; j < E; ++j) {
                int32_t v;
                if (j < kRowRegBatches * kWave) {
                    const int bi = j / kWave;
                    const int32_t src = bi == 0 ? ent[0] : bi == 1 ? ent[1] : bi == 2 ? ent[2] : ent[3];
                    v = __builtin_amdgcn_readlane(src, j % kWave);
                } else {
                    v = entries[b + j];
                }
                const int64_t rel = (int64_t)(v / kBits) - c0;
                if (rel < 0 || rel >= kPass) continue;
                const int k = (int)(rel / kWave), l = (int)(rel % kWave);
                const int dw = (v / 32) % (2 * CW);
                const uint32_t bit = lane == l ? 1u << (v % 32) : 0u;
#pragma unroll
                for (int kk = 0; kk < kRowSlots; ++kk) {
                    if (kk == k) {
#pragma unroll
                        for (int q = 0; q < 2 * CW; ++q)
                            if (q == dw) val[kk][q] |= bit;
                    }
                }
            }
#pragma unroll
            for (int k = 0; k < kRowSlots; ++k) {
                const int64_t c = c0 + k * kWave + lane;
                if (c < nchunks) __builtin_nontemporal_store(val[k], dst + c);
            }
        }
    }
}

// ----------------------------------------------------------------- apply ---

template <typename T>
struct NegInf;
template <>
struct NegInf<uint16_t> {
    static constexpr uint16_t bits = 0xFF80u;
};
template <>
struct NegInf<uint32_t> {
    static constexpr uint32_t bits = 0xFF800000u;
};

// One token id per lane (rel = id minus the first element of the block's span;
// >= kSpan: none or outside): each thread sets the bits of its own chunks.  The
// ids inside the span are few, so a ballot keeps only those.
template <int E, int kSpan>
__device__ __forceinline__ void take_ids(uint32_t rel, uint32_t (&bits)[kApplyUnits]) {
    uint64_t in_span = __ballot(rel < (uint32_t)kSpan);
    while (in_span) {
        const int j = __builtin_ctzll(in_span);
        in_span &= in_span - 1;
        const uint32_t r = (uint32_t)__builtin_amdgcn_readlane((int)rel, j);
        const uint32_t lc = r / E;
#pragma unroll
        for (int u = 0; u < kApplyUnits; ++u)
            if (lc == (uint32_t)(u * kBlock + threadIdx.x)) bits[u] |= 1u << (r % E);
    }
}

// The same for one id held by the whole wave.
template <int E, int kSpan>
__device__ __forceinline__ void set_id(uint32_t rel, uint32_t (&bits)[kApplyUnits]) {
    if (rel >= (uint32_t)kSpan) return;
    const uint32_t lc = rel / E;
#pragma unroll
    for (int u = 0; u < kApplyUnits; ++u)
        if (lc == (uint32_t)(u * kBlock + threadIdx.x)) bits[u] |= 1u << (rel % E);
}

// Grid: x = groups of kBlock*kApplyUnits chunks of one row, y = batch row.
// A chunk is 16 bytes of logits (8 bf16 or 4 fp32); thread i of a block owns
// chunks c0 + u*kBlock + i, so every store instruction covers 4 KiB per block
// contiguously (one chunk per thread writes fastest, as for the table's zero
// fill).  All mask bits of the thread are read before its first store.
// Write-mostly: a chunk without a valid token gets one non-temporal -inf store
// and no read; a fully valid chunk is skipped; a mixed chunk is read, merged and
// written (dense table), or gets -inf stores into its invalid elements only
// (lists).  List rows (kApplyLists, and the tail rows of kApplyTail): the bits
// of the block's span come from the node's valid list instead of the dense
// table (a ballot over a short list, an LDS bitmap for a long one).
// vec == 0: rows are not 16-byte aligned; go element by element.
template <typename T, int kMode>
__global__ void __launch_bounds__(kBlock) k_apply(DevTables t, const int32_t *__restrict__ node_ids,
                                                  T *__restrict__ logits, int64_t stride, int vec) {
    constexpr int E = 16 / (int)sizeof(T);
    constexpr uint32_t FULL = (1u << E) - 1u;
    constexpr T NEG = NegInf<T>::bits;
    constexpr int kSpan = kBlock * kApplyUnits * E;  // elements per block
    __shared__ uint32_t bm[kMode != kApplyTable ? kSpan / 32 : 1];

    const int64_t V = t.V;
    const int64_t b = blockIdx.y;
    const int32_t n = node_ids[b];
    const bool live = n >= 0 && (int64_t)n < t.N;
    const int64_t c0 = (int64_t)blockIdx.x * kBlock * kApplyUnits;
    const int64_t nchunks = (V + E - 1) / E;
    T *row = logits + b * stride;
    // the row's source (uniform over the block): its dense table row, its list,
    // or (a tail with tail compression) the probe's hits along its path
    const int lane = threadIdx.x & (kWave - 1);
    // With tail compression most rows are tails: the hits along the path below
    // n are loaded together with row_of[n] (lane d-1: the hit of node n+d at
    // distance d), and kept only if n turns out to be a tail.
    int32_t x_tail = -1;
    if (kMode == kApplyTail && live && lane < kWin && lane < t.max_len && (int64_t)n + lane + 1 < t.N)
        x_tail = t.hits[(int64_t)lane * t.N + n + lane + 1];
    int64_t trow = live ? n : -1;
    if (kMode == kApplyTail && live) trow = t.row_of[n];
    const bool tail_row = kMode == kApplyTail && live && trow < 0;
    // lists: every row; tail compression without a table: the branching rows
    const bool use_list = kMode == kApplyLists || (kMode == kApplyTail && !tail_row && t.table == nullptr);

    uint32_t bits[kApplyUnits];
#pragma unroll
    for (int u = 0; u < kApplyUnits; ++u) bits[u] = 0;
    const uint32_t lo = (uint32_t)(c0 * E);
    if (tail_row) {
        // lane d-1 takes the token of length d starting below the tail (the
        // path below a tail has consecutive ids, so all of them were loaded)
        const int Lt = min(min(-1 - (int)trow, kWin), (int)t.max_len);
        const int32_t x = lane < Lt ? x_tail : -1;
        take_ids<E, kSpan>(x >= 0 ? (uint32_t)x - lo : 0xffffffffu, bits);
        // strings with several token ids (rare): walk their id chains
        uint64_t multi = __ballot(x <= -2);
        while (multi) {
            const int j = __builtin_ctzll(multi);
            multi &= multi - 1;
            const SlotPay pm = t.pay[-2 - __builtin_amdgcn_readlane(x, j)];
            int32_t v = pm.first;
            for (int k = 0; k < (int)pm.count; ++k) {
                set_id<E, kSpan>((uint32_t)v - lo, bits);
                v = t.dup_next[v];
            }
        }
        if (t.tail_long || t.tail_lists) {  // tokens longer than the window: the tail's list
            const int32_t e0 = t.row_ptr[n], e1 = t.row_ptr[n + 1];
            for (int32_t k0 = e0; k0 < e1; k0 += kWave) {
                const uint32_t rel = k0 + lane < e1 ? (uint32_t)t.entries[k0 + lane] - lo : 0xffffffffu;
                take_ids<E, kSpan>(rel, bits);
            }
        }
    } else if (use_list) {
        const int32_t e0 = live ? t.row_ptr[n] : 0, e1 = live ? t.row_ptr[n + 1] : 0;
        if (e1 - e0 <= kWave) {
            // short list (block-uniform branch): every wave reads the ids into its
            // lanes, keeps those inside the block's span (a ballot), and each thread
            // picks the bits of its own chunks from the few that remain
            take_ids<E, kSpan>(lane < e1 - e0 ? (uint32_t)t.entries[e0 + lane] - lo : 0xffffffffu, bits);
        } else {
            // long list: scatter through an LDS bitmap of the block's span
            for (int i = threadIdx.x; i < kSpan / 32; i += kBlock) bm[i] = 0;
            __syncthreads();
            for (int32_t k = e0 + (int32_t)threadIdx.x; k < e1; k += kBlock) {
                const uint32_t v = (uint32_t)t.entries[k] - lo;
                if (v < (uint32_t)kSpan) atomicOr(&bm[v >> 5], 1u << (v & 31));
            }
            __syncthreads();
#pragma unroll
            for (int u = 0; u < kApplyUnits; ++u) {
                const uint32_t bit = (uint32_t)((u * kBlock + threadIdx.x) * E);
                bits[u] = (bm[bit >> 5] >> (bit & 31)) & FULL;
            }
        }
    } else {
        const uint8_t *mrow = reinterpret_cast<const uint8_t *>(t.table + (trow >= 0 ? trow * t.Wp : 0));
#pragma unroll
        for (int u = 0; u < kApplyUnits; ++u) {
            const int64_t c = c0 + u * kBlock + threadIdx.x;
            uint32_t x = 0;
            if (trow >= 0 && c < nchunks)
                x = E == 8 ? (uint32_t)mrow[c] : ((uint32_t)mrow[c >> 1] >> ((c & 1) * 4)) & FULL;
            bits[u] = x;
        }
    }

#pragma unroll
    for (int u = 0; u < kApplyUnits; ++u) {
        const int64_t c = c0 + u * kBlock + threadIdx.x;
        if (c >= nchunks) break;
        const uint32_t bu = bits[u];
        if (bu == FULL) continue;
        const int64_t e0 = c * E;
        if (vec && e0 + E <= V) {
            u32x4 *p = reinterpret_cast<u32x4 *>(row + e0);
            if (bu == 0) {
                const uint32_t w = sizeof(T) == 2 ? 0xFF80FF80u : 0xFF800000u;
                __builtin_nontemporal_store(u32x4{w, w, w, w}, p);
            } else if (use_list || tail_row) {
                // mixed, list or tail row: -inf into the invalid elements only, no
                // read (the memory side merges the partial lines; measured faster
                // for short valid lists)
                uint32_t *q = reinterpret_cast<uint32_t *>(p);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if (sizeof(T) == 2) {
                        const uint32_t two = (bu >> (2 * i)) & 3u;
                        if (two == 0)
                            q[i] = 0xFF80FF80u;
                        else if (two == 1)
                            row[e0 + 2 * i + 1] = NEG;
                        else if (two == 2)
                            row[e0 + 2 * i] = NEG;
                    } else if (!((bu >> i) & 1u)) {
                        q[i] = 0xFF800000u;
                    }
                }
            } else {
                // mixed, dense table: read, merge, write the whole chunk (measured
                // faster where valid tokens are spread over many chunks)
                u32x4 x = *p;
                T vals[E];
                __builtin_memcpy(vals, &x, 16);
#pragma unroll
                for (int i = 0; i < E; ++i)
                    if (!((bu >> i) & 1u)) vals[i] = NEG;
                __builtin_memcpy(&x, vals, 16);
                *p = x;
            }
        } else {
            const int lim = (int)min<int64_t>(E, V - e0);
            for (int i = 0; i < lim; ++i)
                if (!((bu >> i) & 1u)) row[e0 + i] = NEG;
        }
    }
}

// Dense-table rows, kApplyRows rows per block: block (x, y) takes span x (one
// chunk per thread) of the adjacent rows R y .. R y + R - 1.  All the rows'
// mask bytes are loaded first, then the logits of their mixed chunks, then the
// stores: a block keeps kApplyRows mask loads in flight, while at any moment
// the blocks still write a few compact windows of the logits.  Write-mostly as
// in k_apply (non-temporal -inf stores, read-merge-write of mixed chunks, also
// stored non-temporally).
template <typename T, int R>
__global__ void __launch_bounds__(kBlock) k_apply_dense(DevTables t, const int32_t *__restrict__ node_ids,
                                                        int64_t rows, T *__restrict__ logits, int64_t stride) {
    constexpr int E = 16 / (int)sizeof(T);
    constexpr uint32_t FULL = (1u << E) - 1u;
    constexpr T NEG = NegInf<T>::bits;
    const int64_t V = t.V, nchunks = (V + E - 1) / E;
    const int64_t c = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t e0 = c * E;
    const uint8_t *table = reinterpret_cast<const uint8_t *>(t.table);
    const int64_t row_bytes = t.Wp * 8;
    uint32_t bits[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t b = (int64_t)blockIdx.y * R + r;
        const int32_t n = b < rows ? node_ids[b] : -1;
        bits[r] = 0;  // a dead row: every token invalid
        if (n >= 0 && (int64_t)n < t.N && c < nchunks) {
            const uint8_t *mrow = table + (int64_t)n * row_bytes;
            bits[r] = E == 8 ? (uint32_t)mrow[c] : ((uint32_t)mrow[c >> 1] >> ((c & 1) * 4)) & FULL;
        }
    }
    if (c >= nchunks) return;
    const bool whole = e0 + E <= V;
    u32x4 xv[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t b = (int64_t)blockIdx.y * R + r;
        if (b < rows && whole && bits[r] != 0 && bits[r] != FULL)
            xv[r] = *reinterpret_cast<const u32x4 *>(logits + b * stride + e0);
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t b = (int64_t)blockIdx.y * R + r;
        const uint32_t bu = bits[r];
        if (b >= rows || bu == FULL) continue;
        T *row = logits + b * stride;
        if (whole) {
            u32x4 *p = reinterpret_cast<u32x4 *>(row + e0);
            if (bu == 0) {
                const uint32_t w = sizeof(T) == 2 ? 0xFF80FF80u : 0xFF800000u;
                __builtin_nontemporal_store(u32x4{w, w, w, w}, p);
            } else {
                T vals[E];
                __builtin_memcpy(vals, &xv[r], 16);
#pragma unroll
                for (int i = 0; i < E; ++i)
                    if (!((bu >> i) & 1u)) vals[i] = NEG;
                u32x4 o;
                __builtin_memcpy(&o, vals, 16);
                __builtin_nontemporal_store(o, p);
            }
        } else {
            const int lim = (int)min<int64_t>(E, V - e0);
            for (int i = 0; i < lim; ++i)
                if (!((bu >> i) & 1u)) row[e0 + i] = NEG;
        }
    }
}

// ------------------------------------------- node positions, child lists ---

// The trie's node positions and child lists, built on the device from the
// uploaded blob, node_at and depth.  The strings lie in the blob in trie
// order, so a node's first position is where the string that created it wrote
// its edge byte (node_pos), and one position before sits its parent (the pad
// byte before a string stands for the set root).  Roots have no position.

// node_at and depth from the string records [s0, s1), one thread per string
// (lay_string); a record that does not fit the tables is counted in *err.
__global__ void __launch_bounds__(kBlock) k_node_at(const StrRec *__restrict__ strs, int64_t s0, int64_t s1,
                                                    int64_t blob_bytes, int64_t N, int32_t *__restrict__ node_at,
                                                    int32_t *__restrict__ depth, int32_t *err) {
    const int64_t u = s0 + (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (u >= s1) return;
    const int32_t bad = lay_string(strs, s0, u, blob_bytes, N, node_at, depth);
    if (bad) atomicAdd(err, bad);
}

// Tail compression's tables from the string records [s0, s1), one thread per
// string: row_of and tail_span of the nodes it creates (path indices lcp ..
// len, ids first ...; see TailRec).  Ids outside [0, N) are counted in *err
// and skipped.
__global__ void __launch_bounds__(kBlock) k_tail_nodes(const StrRec *__restrict__ strs,
                                                       const TailRec *__restrict__ trec, int64_t s0, int64_t s1,
                                                       int64_t N, int32_t *__restrict__ row_of,
                                                       int32_t *__restrict__ tail_span, int32_t *err) {
    const int64_t u = s0 + (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (u >= s1) return;
    const StrRec r = strs[u];
    const TailRec tr = trec[u];
    for (int32_t i = r.lcp; i <= r.len; ++i) {
        const int64_t g = (int64_t)r.first + (i - r.lcp);
        if (g < 0 || g >= N) {
            atomicAdd(err, 1);
            return;
        }
        const bool branching = i < tr.next;
        row_of[g] = branching ? tr.row + (i - r.lcp) : -1 - (r.len - i);
        tail_span[g] = branching ? 0 : i - tr.top;
    }
}

// The set roots' entries: rr holds (root id, row) pairs.
__global__ void __launch_bounds__(kBlock) k_root_rows(const int32_t *__restrict__ rr, int64_t S, int64_t N,
                                                      int32_t *__restrict__ row_of, int32_t *__restrict__ tail_span,
                                                      int32_t *err) {
    const int64_t j = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (j >= S) return;
    const int32_t rt = rr[2 * j];
    if (rt < 0 || (int64_t)rt >= N) {
        atomicAdd(err, 1);
        return;
    }
    row_of[rt] = rr[2 * j + 1];
    tail_span[rt] = 0;
}

// row_at[p] = row_of[node_at[p]] over the blob positions [b0, b1).
__global__ void __launch_bounds__(kBlock) k_row_at(const int32_t *__restrict__ node_at,
                                                   const int32_t *__restrict__ row_of, int64_t b0, int64_t b1,
                                                   int64_t N, int32_t *__restrict__ row_at, int32_t *err) {
    const int64_t p = b0 + (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (p >= b1) return;
    const int32_t n = node_at[p];
    if (n < 0 || (int64_t)n >= N) {
        atomicAdd(err, 1);
        row_at[p] = -1;
        return;
    }
    row_at[p] = row_of[n];
}

// node_pos of the nodes [n0, n1): -1 for a root, else a large value that
// k_first_pos lowers
__global__ void __launch_bounds__(kBlock) k_pos_init(const int32_t *__restrict__ depth, int64_t n0, int64_t n1,
                                                     int32_t *__restrict__ node_pos) {
    const int64_t g = n0 + (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (g < n1) node_pos[g] = depth[g] == 0 ? -1 : INT_MAX;
}

// the first position of every non-root node in the blob range [b0, b1)
__global__ void __launch_bounds__(kBlock) k_first_pos(const int32_t *__restrict__ node_at,
                                                      const int32_t *__restrict__ depth, int64_t N, int64_t b0,
                                                      int64_t b1, int32_t *node_pos, int32_t *err) {
    const int64_t p = b0 + (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (p >= b1) return;
    bool bad = false;
    const int32_t g = lay_pos_node(node_at, depth, N, p, &bad);
    if (g >= 0) atomicMin(&node_pos[g], (int32_t)p);
    if (bad) atomicAdd(err, 1);
}

// The parent of non-root node g (lay_parent), or -1 after counting an
// inconsistent position in t.err.
__device__ __forceinline__ int32_t parent_of(const DevTables &t, int64_t g) {
    bool bad = false;
    const int32_t par = lay_parent(t.node_pos, t.node_at, t.N, t.blob_bytes, g, &bad);
    if (bad) atomicAdd(t.err, 1);
    return par;
}

// children per node (cnt zeroed before)
__global__ void __launch_bounds__(kBlock) k_child_count(DevTables t, int32_t *cnt) {
    const int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (g >= t.N || t.depth[g] == 0) return;
    const int32_t par = parent_of(t, g);
    if (par >= 0) atomicAdd(&cnt[par], 1);
}

// every non-root node into its parent's list (cursor zeroed before); the
// order inside a list is free: a lookup matches the child byte
__global__ void __launch_bounds__(kBlock) k_child_fill(DevTables t, int32_t *cursor, int32_t *child_node,
                                                       uint8_t *child_byte, int32_t *child_pos) {
    const int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (g >= t.N || t.depth[g] == 0) return;
    bool bad = false;  // counted once, by k_child_count
    const int32_t par = lay_parent(t.node_pos, t.node_at, t.N, t.blob_bytes, g, &bad);
    if (par < 0) return;
    const int32_t slot = t.child_off[par] + atomicAdd(&cursor[par], 1);
    const int32_t pos = t.node_pos[g];
    child_node[slot] = (int32_t)g;
    child_pos[slot] = pos;
    child_byte[slot] = t.blob[pos];
}

// child_at[p]: the child range of the node whose edge byte is blob[p] (the
// pads: their set's root), for walks that stop inside a string
__global__ void __launch_bounds__(kBlock) k_child_at(DevTables t, uint64_t *child_at) {
    const int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (p >= t.blob_bytes) return;
    const int32_t n = t.node_at[p];
    uint64_t r = 0;
    if (n >= 0 && (int64_t)n < t.N)
        r = (uint64_t)(uint32_t)t.child_off[n] | ((uint64_t)(uint32_t)t.child_off[n + 1] << 32);
    child_at[p] = r;
}

// ------------------------------------------------- fixed-format strings ---

// Token bytes tb[0..len) at position p of a fixed format: non-empty, within
// the L + 1 characters (the last being the terminator), every byte in its
// position's class.
__device__ __forceinline__ bool format_fits(const DevTables &t, int p, const uint8_t *tb, int len) {
    const int L = t.fmt_L;
    if (len <= 0 || p < 0 || p + len > L + 1) return false;
    for (int i = 0; i < len; ++i) {
        const int q = p + i;
        const uint32_t c = tb[i];
        const bool in = q == L ? c == (uint32_t)t.terminator
                               : ((t.classes[(int64_t)q * 32 + (c >> 3)] >> (c & 7)) & 1u) != 0;
        if (!in) return false;
    }
    return true;
}

// Character-position masks (Appendix, Constraint-Aware Dispatch Beyond Finite
// Sets), written whole: one wave per 64-token word w of every row.  Lane i
// tests token 64 w + i at each position p; the wave's ballot is word w of row p
// (lane 0 stores it at out[p * stride + w]), so no zero fill is needed, and
// words past V come out zero.  The valid (position, token) pairs are counted:
// per block into pairs[blockIdx.x], and/or added to *total.
__global__ void __launch_bounds__(kBlock) k_format(DevTables t, uint64_t *__restrict__ out, int64_t stride,
                                                   int64_t nwords, int32_t *__restrict__ pairs,
                                                   unsigned long long *total) {
    const int64_t w = ((int64_t)blockIdx.x * kBlock + threadIdx.x) / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t v = w * kWave + lane;
    int32_t found = 0;
    if (w < nwords) {
        int len = 0;
        const uint8_t *tb = t.tok_blob;
        if (v < t.V) {
            const uint32_t o = t.tok_off[v];
            len = (int)(t.tok_off[v + 1] - o);
            tb += o;
        }
        for (int p = 0; p <= t.fmt_L + 1; ++p) {
            const bool ok = format_fits(t, p, tb, len);
            const uint64_t word = __ballot(ok);
            if (lane == 0) out[(int64_t)p * stride + w] = word;
            found += ok ? 1 : 0;
        }
    }
    __shared__ int32_t wsum[kBlock / kWave];
    for (int o = kWave / 2; o > 0; o >>= 1) found += __shfl_xor(found, o, kWave);
    if (lane == 0) wsum[threadIdx.x / kWave] = found;
    __syncthreads();
    if (threadIdx.x == 0) {
        int32_t sum = 0;
        for (int k = 0; k < kBlock / kWave; ++k) sum += wsum[k];
        if (pairs) pairs[blockIdx.x] = sum;
        if (total && sum) atomicAdd(total, (unsigned long long)sum);
    }
}

// --------------------------------------------------------------- advance ---

// The extended transition function, one wave per batch row.  A child step
// compares up to 64 of the node's child bytes at once (one ballot)
// instead of a binary search.  Between child steps the walk follows the
// node's owner string (the first set string through it, stored in the blob
// right after the node's edge byte): lane j compares token byte i+j with the
// string's byte j, 64 at a time, and the walk jumps to node_at of the last
// matching position.  The run may include the owner string's terminator but
// never goes past it (the node after T has no children).  A token needs one
// child step per point where it leaves the owner string's path, usually one or
// two.
__global__ void __launch_bounds__(kBlock) k_advance(DevTables t, const int32_t *nodes, const int32_t *toks,
                                                    int64_t B, int32_t *out) {
    const int64_t b = ((int64_t)blockIdx.x * kBlock + threadIdx.x) / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    if (b >= B) return;  // uniform over the wave
    const int32_t n0 = nodes[b];
    const int32_t v = toks[b];
    int32_t n = TAM_DEAD;
    const bool ok = n0 >= 0 && (int64_t)n0 < t.N && v >= 0 && (int64_t)v < t.V;
    if (t.fmt_L >= 0) {  // character positions: p + |t| when the token fits the classes
        if (ok && lane == 0) {
            const uint32_t o = t.tok_off[v];
            const int len = (int)(t.tok_off[v + 1] - o);
            if (format_fits(t, n0, t.tok_blob + o, len)) n = n0 + len;
        }
        if (lane == 0) out[b] = n;
        return;
    }
    if (ok) {
        const int64_t a = t.tok_off[v];
        const int len = (int)(t.tok_off[v + 1] - (uint32_t)a);
        const uint32_t T = (uint32_t)t.terminator;
        int i = 0;
        n = len > 0 ? n0 : TAM_DEAD;
        int32_t lo = t.child_off[n0], hi = t.child_off[n0 + 1];  // loaded beside the token's offsets
        while (i < len && n >= 0) {
            const uint32_t c = t.tok_blob[a + i];
            // child of n along c: its child bytes, ids and blob positions, 64
            // lanes at a time, loaded together with the token byte
            int32_t nx = TAM_DEAD, px = 0;
            for (int32_t k0 = lo; k0 < hi; k0 += kWave) {
                const int32_t k = k0 + lane;
                const bool in = k < hi;
                const uint32_t cb = in ? (uint32_t)t.child_byte[k] : 0x100u;
                const int32_t cn = in ? t.child_node[k] : TAM_DEAD;
                const int32_t cp = in ? t.child_pos[k] : 0;
                const uint64_t m = __ballot(cb == c);
                if (m) {
                    const int j = (int)__builtin_ctzll(m);
                    nx = __shfl(cn, j, kWave);
                    px = __shfl(cp, j, kWave);
                    break;
                }
            }
            n = nx;
            ++i;
            if (n < 0 || i >= len) break;  // dead or done
            if (c == T) {                  // a final node: it has no children
                n = TAM_DEAD;
                break;
            }
            int64_t p = px;
            for (;;) {
                const int64_t q = p + 1 + lane;
                const uint32_t sb = q < t.blob_bytes ? (uint32_t)t.blob[q] : 0x200u;
                const uint32_t tb = i + lane < len ? (uint32_t)t.tok_blob[a + i + lane] : 0x100u;
                const uint64_t term = __ballot(sb == T);
                const uint64_t diff = ~__ballot(sb == tb);
                const int f = term ? (int)__builtin_ctzll(term) : kWave;  // first T of the window
                const int run = diff ? (int)__builtin_ctzll(diff) : kWave;
                const int k = min(run, f < kWave ? f + 1 : kWave);      // up to and including T
                p += k;
                i += k;
                if (k < kWave || i >= len || f < kWave) break;
            }
            if (i >= len) {  // the token ends inside the string: its node
                n = t.node_at[p];
                break;
            }
            // the token leaves the string at p: the child range of the node
            // there, in one load (the node itself is not needed)
            const uint64_t r = t.child_at[p];
            lo = (int32_t)(uint32_t)r;
            hi = (int32_t)(uint32_t)(r >> 32);
        }
    }
    if (lane == 0) out[b] = n;
}

// ---------------------------------------------------------------- export ---

// Rows of the nodes with a dense row; all zero for a dead node and (with tail
// compression) for a tail, whose bits k_export_tail then sets.
__global__ void __launch_bounds__(kBlock) k_export_dense(DevTables t, const int32_t *nodes, uint64_t *out) {
    const int64_t r = blockIdx.y;
    const int64_t w = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (w >= t.W) return;
    const int32_t n = nodes[r];
    const bool live = n >= 0 && (int64_t)n < t.N;
    const int64_t trow = live ? (t.row_of ? (int64_t)t.row_of[n] : (int64_t)n) : -1;
    out[r * t.W + w] = trow >= 0 ? t.table[trow * t.Wp + w] : 0ull;
}

// Tail rows (tail compression), one wave per requested row: the ids of the
// tail's hits (as in k_apply) OR-ed into the zeroed output row.
__global__ void __launch_bounds__(kBlock) k_export_tail(DevTables t, const int32_t *nodes, int64_t nrows,
                                                        uint64_t *out) {
    const int64_t r = ((int64_t)blockIdx.x * kBlock + threadIdx.x) / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    if (r >= nrows) return;
    const int32_t n = nodes[r];
    if (n < 0 || (int64_t)n >= t.N) return;
    const int32_t trow = t.row_of[n];
    if (trow >= 0) return;
    unsigned long long *row = reinterpret_cast<unsigned long long *>(out + r * t.W);
    auto set = [&](int32_t v) { atomicOr(row + (v >> 6), 1ull << (v & 63)); };
    const int Lt = min(min(-1 - trow, kWin), (int)t.max_len);
    const int32_t x = lane < Lt ? t.hits[(int64_t)lane * t.N + n + lane + 1] : -1;
    if (x >= 0) {
        set(x);
    } else if (x <= -2) {
        const SlotPay pm = t.pay[-2 - x];
        int32_t v = pm.first;
        for (int k = 0; k < (int)pm.count; ++k) {
            set(v);
            v = t.dup_next[v];
        }
    }
    if (t.tail_long)
        for (int32_t k = t.row_ptr[n] + lane; k < t.row_ptr[n + 1]; k += kWave) set(t.entries[k]);
}

// |valid[n]| of the requested nodes, one wave per node: the popcount of its
// dense row, the length of its list, or (a tail) its hits along the path plus
// its long tokens' list; 0 for a dead node.  The same sources as k_apply.
__global__ void __launch_bounds__(kBlock) k_row_counts(DevTables t, const int32_t *nodes, int64_t nrows,
                                                       int32_t *out) {
    const int64_t r = ((int64_t)blockIdx.x * kBlock + threadIdx.x) / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    if (r >= nrows) return;  // uniform over the wave
    const int32_t n = nodes[r];
    int32_t c = 0;
    if (n >= 0 && (int64_t)n < t.N) {
        const int64_t trow = t.row_of ? (int64_t)t.row_of[n] : (int64_t)n;
        const bool tail = t.row_of && trow < 0;
        if (t.table && !tail) {
            const uint64_t *row = t.table + trow * t.Wp;
            for (int64_t w = lane; w < t.W; w += kWave) c += __popcll(row[w]);
        } else {
            if (tail) {  // a tail: the token of length d starting below it is the hit of node n + d
                const int Lt = min(min(-1 - (int)trow, kWin), (int)t.max_len);
                const int32_t x = lane < Lt ? t.hits[(int64_t)lane * t.N + n + lane + 1] : -1;
                c = x >= 0 ? 1 : (x <= -2 ? (int32_t)t.pay[-2 - x].count : 0);
            }
            if ((!t.table || t.tail_long) && lane == 0) c += t.row_ptr[n + 1] - t.row_ptr[n];
        }
    }
    for (int o = kWave / 2; o > 0; o >>= 1) c += __shfl_xor(c, o, kWave);
    if (lane == 0) out[r] = c;
}

// -------------------------------------------------------- rows on demand ---

constexpr int kLazyProbeBlocks = 2048;  // grid of k_lazy_probe (grid-stride; blocks past the work exit)
constexpr int kLazyBatch = 4;           // candidates per thread and round in k_lazy_probe

// Exclusive prefix sum of one value per thread over a block of kLazyGroup
// threads; *total receives the sum.  sh holds kLazyGroup / kWave + 1 values.
// Waves scan their lanes with shuffles; wave 0 then scans the wave totals.
__device__ __forceinline__ int64_t group_scan(int64_t x, int64_t *total, int64_t *sh) {
    constexpr int kWaves = kLazyGroup / kWave;
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    int64_t inc = x;
    for (int o = 1; o < kWave; o <<= 1) {
        const int64_t y = __shfl_up(inc, o, kWave);
        if (lane >= o) inc += y;
    }
    if (lane == kWave - 1) sh[wid] = inc;
    __syncthreads();
    if (wid == 0) {
        const int64_t v = lane < kWaves ? sh[lane] : 0;
        int64_t vi = v;
        for (int o = 1; o < kWaves; o <<= 1) {
            const int64_t y = __shfl_up(vi, o, kWave);
            if (lane >= o) vi += y;
        }
        if (lane < kWaves) sh[lane] = vi - v;
        if (lane == kWaves - 1) sh[kWaves] = vi;
    }
    __syncthreads();
    const int64_t before = sh[wid];
    *total = sh[kWaves];
    __syncthreads();
    return before + inc - x;
}

// Cache words that other waves of the same block read back after a barrier:
// work-group scope (the block's waves share one CU and its L1), ordered by the
// work-group fences of __syncthreads.  Nothing outside the block reads them
// before the kernel ends.
__device__ __forceinline__ uint32_t load_wg(const uint32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void store_wg(uint32_t *p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Which rows a group of nb batch rows needs built, one block of kLazyGroup
// threads, one thread per batch row.
// kCache (tam_apply_mask):
//   1. Each live row claims its node with a compare-and-swap on slot_of: a
//      slot (>= 0) is a hit; -1 makes the row the builder of the node's row (a
//      miss); -2 - b names builder b to the other rows of that node.  A group
//      without a miss ends here, its rows' slots written.
//   2. Hits stamp their slot with the group's number, so it is not evicted.
//   3. The misses take victims by CLOCK: sweeps from the hand over windows of up
//      to kLazyGroup slots take those not used by the group and without a
//      reference bit, in order, and clear the reference bit of the others they
//      pass; the hand stops after the last slot taken.  With nb <= C at least
//      as many slots are free as there are misses, so two turns of the hand
//      suffice.
//   4. A taken slot drops its old node; each builder records its node, slot,
//      depth and candidate offset for the zero and probe passes, and every
//      batch row its slot (rows_src).
// !kCache (tam_export_rows): every live row is built, into output row b.
template <bool kCache>
__global__ void __launch_bounds__(kLazyGroup) k_lazy_assign(const int32_t *__restrict__ sub_end,
                                                            const int32_t *__restrict__ depth, int64_t N,
                                                            LazyDev z, const int32_t *__restrict__ ids,
                                                            int32_t nb) {
    __shared__ int32_t s_slot[kLazyGroup];
    __shared__ int32_t s_victim[kLazyGroup];
    __shared__ int32_t s_vold[kLazyGroup];
    __shared__ int64_t s_scan[kLazyGroup / kWave + 1];
    __shared__ uint32_t s_u[4];  // group number, -, cut, counter wrapped
    const int tid = threadIdx.x;
    const int32_t n = tid < nb ? ids[tid] : -1;
    const bool live = n >= 0 && (int64_t)n < N;
    const int64_t below = live ? (int64_t)sub_end[n] - n - 1 : 0;
    const int32_t ndep = live ? depth[n] : 0;
    int32_t slot = -1, lead = -1, freed = -1;
    bool miss = live;
    uint32_t group = 0;
    const int64_t C = z.C + z.P;  // the CLOCK sweeps every cache row and passes over the spares
    const int win = (int)min<int64_t>(C, kLazyGroup);
    int64_t hand = 0;
    if (kCache) {
        if (tid == 0) {
            uint32_t g = z.state[0] + 1u;
            s_u[3] = g == 0u ? 1u : 0u;
            if (g == 0u) g = 1u;  // 0 marks a slot never used
            z.state[0] = g;
            s_u[0] = g;
            s_u[1] = z.state[2];  // the spare ring's head
        }
        if (live) {
            const int32_t v = atomicCAS(&z.slot_of[n], -1, -2 - tid);
            miss = v == -1;
            if (v >= 0)
                slot = v;
            else if (v != -1)
                lead = -2 - v;
        }
        __syncthreads();
        group = s_u[0];
        if (s_u[3]) {  // the group counter wrapped: forget every stamp
            for (int64_t c = tid; c < C; c += kLazyGroup) store_wg(&z.stamp[c], 0u);
            __syncthreads();
        }
        if (slot >= 0) {
            store_wg(&z.stamp[slot], group);
            store_wg(&z.ref[slot], 1u);
        }
    }
    s_slot[tid] = slot;
    // no miss in the group (every live row's node is cached): only the rows'
    // slots are written
    if (kCache && !__syncthreads_or(miss ? 1 : 0)) {
        if (tid < nb) z.rows_src[tid] = slot;
        if (tid == 0) {
            z.miss_off[0] = 0;
            *z.miss_count = 0;
        }
        return;
    }
    int64_t nmiss, total;
    const int32_t rank = (int32_t)group_scan(miss ? 1 : 0, &nmiss, s_scan);
    const int64_t off = group_scan(miss ? below : 0, &total, s_scan);
    const int32_t M = (int32_t)nmiss;
    if (kCache) {
        // the hits' stamps are stored (the barrier of the scans above); each
        // window of the sweep loads its slots' stamps, reference bits and
        // nodes in one round trip
        hand = z.state[1];
        int32_t taken = 0;
        const int64_t max_sweeps = 2 * ((C + win - 1) / win) + 2;
        for (int64_t it = 0; it < max_sweeps && taken < M; ++it) {
            const bool in = tid < win;
            int64_t c = hand + tid;
            if (c >= C) c -= C;
            const uint32_t st = in ? load_wg(&z.stamp[c]) : group;
            const uint32_t rf = in ? load_wg(&z.ref[c]) : 1u;
            const int32_t old = in ? z.node_of[c] : -1;
            const bool free_slot = in && st != group && old != -2;  // spares are not victims
            const bool take = free_slot && rf == 0u;
            int64_t avail64;
            const int32_t er = (int32_t)group_scan(take ? 1 : 0, &avail64, s_scan);
            const int32_t need = M - taken, avail = (int32_t)avail64;
            if (take && er == need - 1) s_u[2] = (uint32_t)tid;
            __syncthreads();
            const int cut = avail >= need ? (int)s_u[2] : win - 1;  // last slot the hand passes
            if (tid <= cut) {
                if (take && er < need) {
                    s_victim[taken + er] = (int32_t)c;
                    s_vold[taken + er] = old;
                    store_wg(&z.stamp[c], group);
                } else if (free_slot && rf != 0u) {
                    store_wg(&z.ref[c], 0u);  // second chance
                }
            }
            taken += min(avail, need);
            hand += cut + 1;
            if (hand >= C) hand -= C;
            __syncthreads();
        }
        if (tid == 0) {
            z.state[1] = (uint32_t)hand;
            z.state[2] = (uint32_t)(((int64_t)s_u[1] + taken) % z.P);
        }
        if (miss) {
            const int32_t c = rank < taken ? s_victim[rank] : -1;
            if (c >= 0) {
                // the miss's row is the next spare (zero); its victim c becomes a
                // spare in that place, cleared by this group's build pass
                const int64_t at = ((int64_t)s_u[1] + rank) % z.P;
                const int32_t r = z.spare[at];
                z.spare[at] = c;
                freed = c;
                const int32_t old = s_vold[rank];
                if (old >= 0) z.slot_of[old] = -1;
                z.node_of[c] = -2;
                z.node_of[r] = n;
                z.slot_of[n] = r;
                store_wg(&z.stamp[r], group);
                store_wg(&z.ref[r], 1u);
                s_slot[tid] = r;
            } else {
                // not reached while nb <= C (two turns of the hand find the
                // slots); counted as an error, the rows stay fully masked
                z.slot_of[n] = -1;
                atomicAdd(z.err, 1);
                s_slot[tid] = -1;
            }
        }
        __syncthreads();
        if (tid < nb) z.rows_src[tid] = lead >= 0 ? s_slot[lead] : s_slot[tid];
    }
    if (miss) {
        z.miss_node[rank] = n;
        z.miss_row[rank] = kCache ? s_slot[tid] : tid;
        z.miss_free[rank] = freed;
        z.miss_off[rank] = off;
        z.miss_dep[rank] = ndep;
    }
    if (tid == 0) {
        z.miss_off[M] = total;
        *z.miss_count = M;
    }
}

// The hits of K independent suffixes (the one of d[k] bytes ending at blob
// position pos[k], window (lo[k], hi[k]); act[k] false: none) with their
// memory round trips issued together: short suffixes read short_hits, the
// others their home bucket, then the payload (and pay_hi) of the first
// fingerprint match; a length the home bucket does not settle falls back to
// the general probe.
template <int K>
__device__ __forceinline__ void probe_batch(const DevTables &t, const int64_t (&pos)[K], const int (&d)[K],
                                            const bool (&act)[K], const uint64_t (&lo)[K], const uint64_t (&hi)[K],
                                            int32_t (&hit)[K]) {
    uint64_t key[K];
    bool hashed[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
        hit[k] = -1;
        hashed[k] = act[k] && d[k] > kShortLen;
        key[k] = 0;
        if (act[k] && d[k] <= kShortLen) hit[k] = short_hit(t, d[k], window_byte(lo[k], hi[k], 0), window_byte(lo[k], hi[k], 1));
        if (hashed[k]) {
            uint32_t h = kHashSeed;
            for (int j = 0; j < d[k]; ++j)
                h = hash_step(h, j < kWin ? window_byte(lo[k], hi[k], j) : (uint32_t)t.blob[pos[k] - j]);
            key[k] = hash_final(h);
        }
    }
    Bucket bk[K];
#pragma unroll
    for (int k = 0; k < K; ++k)
        if (hashed[k]) bk[k] = load_bucket(t, home_bucket(t, key[k]));
    uint32_t match[K], empty[K];
    int32_t slot[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
        match[k] = empty[k] = 0;
        slot[k] = -1;
        if (hashed[k]) {
            bucket_masks(bk[k], fingerprint(key[k]), &match[k], &empty[k]);
            if (match[k]) slot[k] = (int32_t)(bucket_base(bk[k]) + (uint32_t)__builtin_ctz(match[k]));
        }
    }
    SlotPay p[K];
    uint64_t phi[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
        phi[k] = 0;
        if (slot[k] >= 0) {
            p[k] = t.pay[slot[k]];
            if (d[k] > 8) phi[k] = t.pay_hi[slot[k]];
        }
    }
#pragma unroll
    for (int k = 0; k < K; ++k) {
        if (!hashed[k]) continue;
        if (slot[k] >= 0 && slot_equals(t, p[k], phi[k], d[k], lo[k], hi[k], pos[k])) {
            hit[k] = hit_of_slot(slot[k], p[k].first, p[k].count);
        } else if (!(empty[k] != 0 && (match[k] & (match[k] - 1)) == 0)) {
            SlotPay mt;  // the home bucket does not settle it
            const int32_t sl = probe(t, key[k], d[k], lo[k], hi[k], pos[k], &mt);
            if (sl >= 0) hit[k] = hit_of_slot(sl, mt.first, mt.count);
        }
    }
}

// The candidates of misses: candidate i of miss u is node m = n + 1 + (i -
// miss_off[u]) for the misses the pass covers, a descendant d = depth(m) -
// depth(n) bytes below n (preorder: the subtree is [n, sub_end[n])).  When
// d <= max_len and the last d bytes of prefix(m), the path from n to m, are a
// token string, its ids are valid at n; every token valid at n ends its walk
// at exactly one such m.  set(row, id) records a valid id.
template <typename F>
__device__ __forceinline__ void lazy_candidates(const DevTables &t, const int64_t (&m)[kLazyBatch],
                                                const int (&dep)[kLazyBatch], bool (&act)[kLazyBatch],
                                                const int32_t (&row)[kLazyBatch], F &&set) {
    constexpr int K = kLazyBatch;
    int dm[K], d[K];
    int64_t pos[K];
#pragma unroll
    for (int k = 0; k < K; ++k) dm[k] = act[k] ? t.depth[m[k]] : 0;
#pragma unroll
    for (int k = 0; k < K; ++k) {
        d[k] = dm[k] - dep[k];
        act[k] = act[k] && row[k] >= 0 && d[k] <= t.max_len && has_len(t, d[k]);
    }
#pragma unroll
    for (int k = 0; k < K; ++k) pos[k] = act[k] ? t.node_pos[m[k]] : 0;
    uint64_t wlo[K], whi[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
        wlo[k] = whi[k] = 0;
        if (act[k]) load_window(t.blob, pos[k], wlo[k], whi[k]);
    }
    int32_t hx[K];
    probe_batch<K>(t, pos, d, act, wlo, whi, hx);
#pragma unroll
    for (int k = 0; k < K; ++k) {
        if (hx[k] == -1) continue;
        if (hx[k] >= 0) {  // one token id (the common case)
            set(row[k], hx[k]);
            continue;
        }
        const SlotPay pm = t.pay[-2 - hx[k]];  // a string with several ids
        int32_t v = pm.first;
        for (int j = 0; j < (int)pm.count; ++j) {
            set(row[k], v);
            v = t.dup_next[v];
        }
    }
}

// The grid-stride pass over the candidates of the misses miss_off covers,
// with 64-bit atomics into the zeroed rows dest + row * stride; block bx of nbx,
// kLazyBatch candidates per thread and round with their loads issued together.
// LDS of the pass: the misses' candidate offsets, nodes, rows and depths.
struct LazyMisses {
    int64_t off[kLazyGroup + 1];
    int32_t node[kLazyGroup], row[kLazyGroup], dep[kLazyGroup];
};

__device__ __forceinline__ void lazy_probe_pass(const DevTables &t, const LazyDev &z, uint64_t *dest, int64_t stride,
                                                int64_t bx, int64_t nbx, LazyMisses &sm) {
    constexpr int K = kLazyBatch;
    int64_t *s_off = sm.off;
    int32_t *s_node = sm.node, *s_row = sm.row, *s_dep = sm.dep;
    const int32_t M = *z.miss_count;
    if (M <= 0) return;
    const int64_t total = z.miss_off[M];
    const int64_t first = bx * kBlock;
    if (first >= total) return;
    for (int i = threadIdx.x; i <= M; i += kBlock) s_off[i] = z.miss_off[i];
    for (int i = threadIdx.x; i < M; i += kBlock) {
        s_node[i] = z.miss_node[i];
        s_row[i] = z.miss_row[i];
        s_dep[i] = z.miss_dep[i];
    }
    __syncthreads();
    unsigned long long *out = reinterpret_cast<unsigned long long *>(dest);
    const int64_t threads = nbx * kBlock;
    for (int64_t base = first + threadIdx.x; base < total; base += K * threads) {
        int64_t m[K];
        int32_t row[K];
        int dep[K];
        bool act[K];
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const int64_t i = base + k * threads;
            act[k] = i < total;
            row[k] = -1;
            m[k] = 0;
            dep[k] = 0;
            if (!act[k]) continue;
            int lo = 0, hi = M - 1;  // the last miss whose candidates start at or before i
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (s_off[mid] <= i)
                    lo = mid;
                else
                    hi = mid - 1;
            }
            row[k] = s_row[lo];
            m[k] = (int64_t)s_node[lo] + 1 + (i - s_off[lo]);
            dep[k] = s_dep[lo];
        }
        lazy_candidates(t, m, dep, act, row, [&](int32_t r, int32_t v) {
            atomicOr(out + (int64_t)r * stride + (v >> 6), 1ull << (v & 63));
        });
    }
}

// The rows of the group's misses, in their cache rows (spares, zero) for
// tam_apply_mask, or straight into the zeroed output rows for tam_export_rows.
// clear (tam_apply_mask): the cache rows the misses freed are zeroed first, so
// that they are zero when a later group takes them as spares.
__global__ void __launch_bounds__(kBlock) k_lazy_probe(DevTables t, LazyDev z, uint64_t *dest, int64_t stride,
                                                       int clear) {
    __shared__ LazyMisses sm;
    if (clear) {
        const int32_t M = *z.miss_count;
        const int32_t per = (int32_t)(t.Wp / 2);  // 16-byte chunks per row
        const int64_t chunks = (int64_t)M * per;
        for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < chunks; i += (int64_t)gridDim.x * kBlock) {
            const int32_t u = (int32_t)(i / per);
            const int32_t r = z.miss_free[u];
            if (r >= 0 && (int64_t)r < z.C + z.P)
                reinterpret_cast<u32x4 *>(z.cache + (int64_t)r * t.Wp)[i - (int64_t)u * per] = u32x4{0u, 0u, 0u, 0u};
        }
    }
    lazy_probe_pass(t, z, dest, stride, blockIdx.x, gridDim.x, sm);
}

// p[i] = first + i, i < n.
__global__ void __launch_bounds__(kBlock) k_iota_i32(int32_t *p, int64_t n, int32_t first) {
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i < n) p[i] = first + (int32_t)i;
}

__global__ void __launch_bounds__(kBlock) k_fill_u64(uint64_t *p, int64_t n, uint64_t value) {
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += (int64_t)gridDim.x * kBlock)
        p[i] = value;
}

inline unsigned grid_for(int64_t n, int per_block) {
    return (unsigned)((n + per_block - 1) / per_block);
}

}  // namespace

int64_t scan_tmp_elems(int64_t N) { return (N + kScanTile - 1) / kScanTile + 1; }

hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t value, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const unsigned g = (unsigned)std::min<int64_t>(grid_for(n, kBlock), 4096);
    hipLaunchKernelGGL(k_fill_i32, dim3(g), dim3(kBlock), 0, s, p, n, value);
    return hipGetLastError();
}

hipError_t launch_probe(const DevTables &t, bool count, bool mark, int32_t *pairs, hipStream_t s) {
    if (t.N <= 0) return hipSuccess;
    const int do_mark = mark && t.table ? 1 : 0;
    const dim3 grid((unsigned)mark_blocks(t.N));
    if (t.tail_lists) return hipErrorInvalidValue;  // the groups' grid (launch_probe_groups)
    const RecGroups none{};
    if (count)
        hipLaunchKernelGGL(k_probe<true>, grid, dim3(kBlock), 0, s, t, (int64_t)0, t.N, do_mark, pairs, none,
                           (int64_t)0);
    else
        hipLaunchKernelGGL(k_probe<false>, grid, dim3(kBlock), 0, s, t, (int64_t)0, t.N, do_mark, pairs, none,
                           (int64_t)0);
    return hipGetLastError();
}

// The host checks the groups' grid: consecutive node ranges within [0, N),
// each with as many blocks as its nodes need, blocks and offsets increasing.
static bool groups_ok(const DevTables &t, const RecGroups &rg) {
    if (rg.n < 1 || rg.n > kMaxRecGroups || rg.blk0[0] != 0) return false;
    for (int k = 0; k < rg.n; ++k) {
        const int64_t nodes = rg.n_hi[k] - rg.n_lo[k];
        if (rg.n_lo[k] < 0 || nodes <= 0 || rg.n_hi[k] > t.N || !rg.rec[k]) return false;
        if (rg.blk0[k + 1] - rg.blk0[k] != mark_blocks(nodes)) return false;
        if (k > 0 && (rg.n_lo[k] != rg.n_hi[k - 1] || rg.off0[k] < rg.off0[k - 1] + (rg.blk0[k] - rg.blk0[k - 1]) + 1))
            return false;
    }
    return true;
}

hipError_t launch_probe_groups(const DevTables &t, const RecGroups &rg, int64_t k0, int64_t k1, int32_t *pairs,
                               hipStream_t s) {
    if (!t.tail_lists || t.table || !pairs || !groups_ok(t, rg) || k0 < 0 || k1 > rg.n || k0 >= k1)
        return hipErrorInvalidValue;
    const int64_t b0 = rg.blk0[k0], b1 = rg.blk0[k1];
    hipLaunchKernelGGL(k_probe<true>, dim3((unsigned)(b1 - b0)), dim3(kBlock), 0, s, t, (int64_t)0, t.N, 0, pairs,
                       rg, b0);
    return hipGetLastError();
}

hipError_t launch_count_range(const DevTables &t, int64_t m0, int64_t m1, hipStream_t s) {
    if (m1 <= m0) return hipSuccess;
    if (m0 < 0 || m1 > t.N || t.table || t.tail_lists) return hipErrorInvalidValue;
    const RecGroups none{};
    hipLaunchKernelGGL(k_probe<true>, dim3((unsigned)mark_blocks(m1 - m0)), dim3(kBlock), 0, s, t, m0, m1, 0,
                       (int32_t *)nullptr, none, (int64_t)0);
    return hipGetLastError();
}

hipError_t launch_node_at(const StrRec *strs, int64_t s0, int64_t s1, int64_t blob_bytes, int64_t N,
                          int32_t *node_at, int32_t *depth, int32_t *err, hipStream_t s) {
    if (s1 <= s0) return hipSuccess;
    hipLaunchKernelGGL(k_node_at, dim3(grid_for(s1 - s0, kBlock)), dim3(kBlock), 0, s, strs, s0, s1, blob_bytes, N,
                       node_at, depth, err);
    return hipGetLastError();
}

hipError_t launch_tail_tables(const StrRec *strs, const TailRec *trec, int64_t s0, int64_t s1,
                              const int32_t *root_rows, int64_t S, const int32_t *node_at, int64_t b0, int64_t b1,
                              int64_t N, int32_t *row_of, int32_t *tail_span, int32_t *row_at, int32_t *err,
                              hipStream_t s) {
    if (s1 > s0)
        hipLaunchKernelGGL(k_tail_nodes, dim3(grid_for(s1 - s0, kBlock)), dim3(kBlock), 0, s, strs, trec, s0, s1, N,
                           row_of, tail_span, err);
    if (root_rows && S > 0)
        hipLaunchKernelGGL(k_root_rows, dim3(grid_for(S, kBlock)), dim3(kBlock), 0, s, root_rows, S, N, row_of,
                           tail_span, err);
    if (b1 > b0)
        hipLaunchKernelGGL(k_row_at, dim3(grid_for(b1 - b0, kBlock)), dim3(kBlock), 0, s, node_at, row_of, b0, b1, N,
                           row_at, err);
    return hipGetLastError();
}

hipError_t launch_node_pos(const DevTables &t, int32_t *node_pos, int64_t n0, int64_t n1, int64_t b0, int64_t b1,
                           hipStream_t s) {
    if (n0 < 0 || n1 > t.N || b0 < 0 || b1 > t.blob_bytes) return hipErrorInvalidValue;
    if (n1 > n0)
        hipLaunchKernelGGL(k_pos_init, dim3(grid_for(n1 - n0, kBlock)), dim3(kBlock), 0, s, t.depth, n0, n1, node_pos);
    if (b1 > b0)
        hipLaunchKernelGGL(k_first_pos, dim3(grid_for(b1 - b0, kBlock)), dim3(kBlock), 0, s, t.node_at, t.depth, t.N,
                           b0, b1, node_pos, t.err);
    return hipGetLastError();
}

hipError_t launch_child_lists(const DevTables &t, int32_t *child_off, int32_t *child_node, uint8_t *child_byte,
                              int32_t *child_pos, uint64_t *child_at, int32_t *tmp, int32_t *scan_tmp,
                              hipStream_t s) {
    if (t.N <= 0) return hipSuccess;
    const unsigned g = grid_for(t.N, kBlock);
    hipError_t e = launch_fill_i32(tmp, t.N, 0, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_child_count, dim3(g), dim3(kBlock), 0, s, t, tmp);
    DevTables ts = t;  // the scan: counts -> child_off[0..N], the total at N
    ts.count = tmp;
    ts.row_ptr = child_off;
    ts.scan_tmp = scan_tmp;
    e = launch_scan(ts, s);
    if (e == hipSuccess) e = launch_fill_i32(tmp, t.N, 0, s);
    if (e != hipSuccess) return e;
    DevTables tf = t;
    tf.child_off = child_off;
    hipLaunchKernelGGL(k_child_fill, dim3(g), dim3(kBlock), 0, s, tf, tmp, child_node, child_byte, child_pos);
    if (t.blob_bytes > 0)
        hipLaunchKernelGGL(k_child_at, dim3(grid_for(t.blob_bytes, kBlock)), dim3(kBlock), 0, s, tf, child_at);
    return hipGetLastError();
}

int64_t probe_nodes_per_block() { return kBlock / kProbeLanes; }

hipError_t launch_fill_records(const DevTables &t, const RecGroups &rg, hipStream_t s) {
    if (!groups_ok(t, rg)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_fill_records, dim3((unsigned)rg.blk0[rg.n]), dim3(kWave), 0, s, t, rg);
    return hipGetLastError();
}

hipError_t launch_fill_lists(const DevTables &t, hipStream_t s) {
    if (t.N <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill, dim3(grid_for(t.N, kBlock)), dim3(kBlock), 0, s, t);
    return hipGetLastError();
}

hipError_t launch_zero(uint64_t *p, int64_t words, hipStream_t s) {
    const int64_t n16 = words / 2;
    if (n16 <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_zero, dim3(grid_for(n16, kBlock)), dim3(kBlock), 0, s,
                       reinterpret_cast<u32x4 *>(p), n16);
    return hipGetLastError();
}

int64_t mark_blocks(int64_t N) { return (N * kProbeLanes + kBlock - 1) / kBlock; }

int64_t format_blocks(int64_t Wp) { return (Wp * kWave + kBlock - 1) / kBlock; }

hipError_t launch_format(const DevTables &t, int32_t *pairs, hipStream_t s) {
    hipLaunchKernelGGL(k_format, dim3((unsigned)format_blocks(t.Wp)), dim3(kBlock), 0, s, t, t.table, t.Wp, t.Wp,
                       pairs, (unsigned long long *)nullptr);
    return hipGetLastError();
}

hipError_t launch_scan(const DevTables &t, hipStream_t s) {
    const int64_t nb = grid_for(t.N, kScanTile);
    const int own = nb <= kScanTile ? 1 : 0;  // the apply pass adds up the block sums itself
    hipLaunchKernelGGL(k_scan_blocks, dim3((unsigned)nb), dim3(kBlock), 0, s, t.count, t.N, t.scan_tmp);
    if (!own) hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(kBlock), 0, s, t.scan_tmp, nb, t.row_ptr + t.N);
    hipLaunchKernelGGL(k_scan_apply, dim3((unsigned)nb), dim3(kBlock), 0, s, t.count, t.N, t.scan_tmp, own,
                       t.row_ptr, t.row_ptr + t.N);
    return hipGetLastError();
}

hipError_t launch_rows(const DevTables &t, const int32_t *nodes, int64_t nrows, uint64_t *out,
                       int64_t out_stride_words, int64_t out_words, hipStream_t s) {
    if (nrows <= 0 || out_words <= 0) return hipSuccess;
    const bool vec = (out_stride_words & 1) == 0 && (out_words & 1) == 0 &&
                     (reinterpret_cast<uintptr_t>(out) & 15) == 0;
    int per_cu = 0;
    hipError_t e = vec ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_rows<2>, kBlock, 0)
                       : hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_rows<1>, kBlock, 0);
    if (e != hipSuccess || per_cu <= 0) per_cu = 4;
    const int64_t waves_needed = nrows;
    const int64_t cap = (int64_t)props_for_current_device().cus * per_cu;
    const unsigned g = (unsigned)std::max<int64_t>(1, std::min<int64_t>(cap, grid_for(waves_needed, kBlock / kWave)));
    if (vec)
        hipLaunchKernelGGL(k_rows<2>, dim3(g), dim3(kBlock), 0, s, t.row_ptr, t.entries, nodes, nrows, t.N, out,
                           out_stride_words, out_words);
    else
        hipLaunchKernelGGL(k_rows<1>, dim3(g), dim3(kBlock), 0, s, t.row_ptr, t.entries, nodes, nrows, t.N, out,
                           out_stride_words, out_words);
    return hipGetLastError();
}

// Dense-table rows, R rows per block; grid.y (row groups) is limited to 65535
// per launch.
template <int R>
static hipError_t launch_apply_dense(const DevTables &t, const int32_t *node_ids, int64_t B, void *logits, int dtype,
                                     int64_t row_stride, int64_t gx1, hipStream_t s) {
    for (int64_t r0 = 0; r0 < B; r0 += (int64_t)65535 * R) {
        const int64_t rows = std::min<int64_t>(B - r0, (int64_t)65535 * R);
        const dim3 grid((unsigned)gx1, (unsigned)grid_for(rows, R));
        if (dtype == TAM_DTYPE_BF16)
            hipLaunchKernelGGL((k_apply_dense<uint16_t, R>), grid, dim3(kBlock), 0, s, t, node_ids + r0, rows,
                               static_cast<uint16_t *>(logits) + r0 * row_stride, row_stride);
        else
            hipLaunchKernelGGL((k_apply_dense<uint32_t, R>), grid, dim3(kBlock), 0, s, t, node_ids + r0, rows,
                               static_cast<uint32_t *>(logits) + r0 * row_stride, row_stride);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_apply(const DevTables &t, const int32_t *node_ids, int64_t B, void *logits, int dtype,
                        int64_t row_stride, hipStream_t s) {
    const int E = dtype == TAM_DTYPE_BF16 ? 8 : 4;
    const int elem = dtype == TAM_DTYPE_BF16 ? 2 : 4;
    const int64_t nchunks = (t.V + E - 1) / E;
    const unsigned gx = grid_for(nchunks, kBlock * kApplyUnits);
    const int vec = ((reinterpret_cast<uintptr_t>(logits) & 15) == 0 && ((row_stride * elem) & 15) == 0)
                        ? 1
                        : 0;
    const int mode = t.row_of ? kApplyTail : (t.table ? kApplyTable : kApplyLists);
    if (mode == kApplyTable && vec) {
        const int64_t gx1 = grid_for(nchunks, kBlock);
        // three rows per block while that keeps 16 blocks per CU in flight,
        // else two (64 fp32 rows over V = 128,256: 8.2 against 8.9 µs per call)
        if (gx1 * ((B + kApplyRows - 1) / kApplyRows) >= kApplyMinBlocks)
            return launch_apply_dense<kApplyRows>(t, node_ids, B, logits, dtype, row_stride, gx1, s);
        return launch_apply_dense<2>(t, node_ids, B, logits, dtype, row_stride, gx1, s);
    }
    // grid.y is limited to 65535 rows per launch
    for (int64_t r0 = 0; r0 < B; r0 += 65535) {
        const dim3 grid(gx, (unsigned)std::min<int64_t>(B - r0, 65535));
        const int32_t *ids = node_ids + r0;
        if (dtype == TAM_DTYPE_BF16) {
            uint16_t *p = static_cast<uint16_t *>(logits) + r0 * row_stride;
            if (mode == kApplyLists)
                hipLaunchKernelGGL((k_apply<uint16_t, kApplyLists>), grid, dim3(kBlock), 0, s, t, ids, p, row_stride, vec);
            else if (mode == kApplyTail)
                hipLaunchKernelGGL((k_apply<uint16_t, kApplyTail>), grid, dim3(kBlock), 0, s, t, ids, p, row_stride, vec);
            else
                hipLaunchKernelGGL((k_apply<uint16_t, kApplyTable>), grid, dim3(kBlock), 0, s, t, ids, p, row_stride, vec);
        } else {
            uint32_t *p = static_cast<uint32_t *>(logits) + r0 * row_stride;
            if (mode == kApplyLists)
                hipLaunchKernelGGL((k_apply<uint32_t, kApplyLists>), grid, dim3(kBlock), 0, s, t, ids, p, row_stride, vec);
            else if (mode == kApplyTail)
                hipLaunchKernelGGL((k_apply<uint32_t, kApplyTail>), grid, dim3(kBlock), 0, s, t, ids, p, row_stride, vec);
            else
                hipLaunchKernelGGL((k_apply<uint32_t, kApplyTable>), grid, dim3(kBlock), 0, s, t, ids, p, row_stride, vec);
        }
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_advance(const DevTables &t, const int32_t *node_ids, const int32_t *token_ids, int64_t B,
                          int32_t *out, hipStream_t s) {
    if (B <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_advance, dim3(grid_for(B, kBlock / kWave)), dim3(kBlock), 0, s, t, node_ids, token_ids, B,
                       out);
    return hipGetLastError();
}

hipError_t launch_lazy_apply(const DevTables &t, const LazyDev &z, const int32_t *node_ids, int64_t nb,
                             void *logits, int dtype, int64_t row_stride, hipStream_t s) {
    if (nb <= 0) return hipSuccess;
    if (nb > kLazyGroup || nb > z.C || !t.sub_end) return hipErrorInvalidValue;
    if (nb > z.P) return hipErrorInvalidValue;  // a group's misses take at most P spares
    hipLaunchKernelGGL(k_lazy_assign<true>, dim3(1), dim3(kLazyGroup), 0, s, t.sub_end, t.depth, t.N, z, node_ids,
                       (int32_t)nb);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_lazy_probe, dim3(kLazyProbeBlocks), dim3(kBlock), 0, s, t, z, z.cache, t.Wp, 1);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    // the masking reads the cache as a dense table indexed by cache row
    DevTables tc = t;
    tc.table = z.cache;
    tc.row_of = nullptr;
    tc.N = z.C + z.P;
    tc.R = z.C + z.P;
    return launch_apply(tc, z.rows_src, nb, logits, dtype, row_stride, s);
}

hipError_t launch_lazy_export(const DevTables &t, const LazyDev &z, const int32_t *node_ids, int64_t nb,
                              uint64_t *out, hipStream_t s) {
    if (nb <= 0) return hipSuccess;
    if (nb > kLazyGroup || !t.sub_end) return hipErrorInvalidValue;
    const int64_t words = nb * t.W;
    hipLaunchKernelGGL(k_fill_u64, dim3((unsigned)std::min<int64_t>(grid_for(words, kBlock), 4096)), dim3(kBlock),
                       0, s, out, words, 0ull);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_lazy_assign<false>, dim3(1), dim3(kLazyGroup), 0, s, t.sub_end, t.depth, t.N, z, node_ids,
                       (int32_t)nb);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_lazy_probe, dim3(kLazyProbeBlocks), dim3(kBlock), 0, s, t, z, out, t.W, 0);
    return hipGetLastError();
}

hipError_t launch_lazy_reset(const DevTables &t, const LazyDev &z, hipStream_t s) {
    // rows 0 .. C-1 empty, C .. C+P-1 the spares (zeroed), in ring order
    hipError_t e = launch_fill_i32(z.slot_of, t.N, -1, s);
    if (e == hipSuccess) e = launch_fill_i32(z.node_of, z.C, -1, s);
    if (e == hipSuccess) e = launch_fill_i32(z.node_of + z.C, z.P, -2, s);
    if (e == hipSuccess) e = launch_fill_i32(reinterpret_cast<int32_t *>(z.stamp), z.C + z.P, 0, s);
    if (e == hipSuccess) e = launch_fill_i32(reinterpret_cast<int32_t *>(z.ref), z.C + z.P, 0, s);
    if (e == hipSuccess) e = launch_fill_i32(reinterpret_cast<int32_t *>(z.state), 3, 0, s);
    if (e != hipSuccess || z.P <= 0) return e;
    hipLaunchKernelGGL(k_iota_i32, dim3(grid_for(z.P, kBlock)), dim3(kBlock), 0, s, z.spare, z.P, (int32_t)z.C);
    e = hipGetLastError();
    if (e == hipSuccess) e = launch_zero(z.cache + z.C * t.Wp, z.P * t.Wp, s);
    return e;
}

hipError_t launch_row_counts(const DevTables &t, const int32_t *node_ids, int64_t n, int32_t *out, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_row_counts, dim3(grid_for(n, kBlock / kWave)), dim3(kBlock), 0, s, t, node_ids, n, out);
    return hipGetLastError();
}

hipError_t launch_export_tail(const DevTables &t, const int32_t *node_ids, int64_t n, uint64_t *out, hipStream_t s) {
    if (n <= 0 || !t.row_of) return hipSuccess;
    hipLaunchKernelGGL(k_export_tail, dim3(grid_for(n, kBlock / kWave)), dim3(kBlock), 0, s, t, node_ids, n, out);
    return hipGetLastError();
}

hipError_t launch_export_dense(const DevTables &t, const int32_t *node_ids, int64_t n, uint64_t *out,
                               hipStream_t s) {
    for (int64_t r0 = 0; r0 < n; r0 += 65535) {
        const unsigned rows = (unsigned)std::min<int64_t>(n - r0, 65535);
        hipLaunchKernelGGL(k_export_dense, dim3(grid_for(t.W, kBlock), rows), dim3(kBlock), 0, s, t,
                           node_ids + r0, out + r0 * t.W);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (!t.row_of) return hipSuccess;
    hipLaunchKernelGGL(k_export_tail, dim3(grid_for(n, kBlock / kWave)), dim3(kBlock), 0, s, t, node_ids, n, out);
    return hipGetLastError();
}

// ------------------------------------------- format rows, no allocation ---

// The scratch of tam_format_rows_noalloc: a counter of the valid pairs, then
// the class bits of up to TAM_NOALLOC_MAX_POSITIONS positions, staged from the
// host through kernel arguments.  One copy per GPU, held until the process
// ends; every call on a GPU shares it (overlapping calls race).  Host code
// never names the array itself: it takes the device address that
// hipGetSymbolAddress returns (noalloc_scratch) and passes that to kernels.
constexpr size_t kScratchHeader = 256;
constexpr size_t kScratchBytes = kScratchHeader + 32 * (size_t)TAM_NOALLOC_MAX_POSITIONS;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {

constexpr int kStagePositions = 64;  // positions per staging launch (2 KiB of kernel arguments)

struct ClassChunk {
    int32_t first, count;                  // positions [first, first + count)
    uint32_t words[kStagePositions * 8];   // their class bits, 32 bytes per position
};

// Copies one chunk of class bits into the scratch (the first chunk also
// clears the pair counter).
__global__ void __launch_bounds__(kBlock) k_stage_classes(ClassChunk c, uint32_t *__restrict__ cls,
                                                          unsigned long long *counter) {
    for (int i = threadIdx.x; i < c.count * 8; i += kBlock) cls[(int64_t)c.first * 8 + i] = c.words[i];
    if (c.first == 0 && threadIdx.x == 0) *counter = 0ull;
}

__global__ void k_store_total(const unsigned long long *counter, int64_t *out) {
    if (threadIdx.x == 0) *out = (int64_t)*counter;
}

std::mutex g_scratch_mutex;
void *g_scratch_ptr[64] = {};

}  // namespace

// The device address of this GPU's scratch, looked up once per device with
// that device current.
hipError_t noalloc_scratch(uint8_t **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> g(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = static_cast<uint8_t *>(g_scratch_ptr[dev]);
    return hipSuccess;
}

hipError_t launch_format_noalloc(const DevTables &t, const uint8_t *classes_host, uint64_t *out, int64_t stride,
                                 int64_t *pairs_out, hipStream_t s) {
    const int64_t L = t.fmt_L;
    if (L < 1 || L > TAM_NOALLOC_MAX_POSITIONS || stride < t.W) return hipErrorInvalidValue;
    uint8_t *base = nullptr;
    hipError_t e = noalloc_scratch(&base);
    if (e != hipSuccess) return e;
    unsigned long long *counter = reinterpret_cast<unsigned long long *>(base);
    uint32_t *cls = reinterpret_cast<uint32_t *>(base + kScratchHeader);
    for (int64_t p0 = 0; p0 < L; p0 += kStagePositions) {
        ClassChunk c;
        c.first = (int32_t)p0;
        c.count = (int32_t)std::min<int64_t>(kStagePositions, L - p0);
        std::memset(c.words, 0, sizeof(c.words));
        std::memcpy(c.words, classes_host + 32 * p0, (size_t)c.count * 32);
        hipLaunchKernelGGL(k_stage_classes, dim3(1), dim3(kBlock), 0, s, c, cls, counter);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    DevTables tf = t;
    tf.classes = reinterpret_cast<const uint8_t *>(cls);
    hipLaunchKernelGGL(k_format, dim3((unsigned)format_blocks(t.W)), dim3(kBlock), 0, s, tf, out, stride, t.W,
                       (int32_t *)nullptr, counter);
    e = hipGetLastError();
    if (e != hipSuccess || !pairs_out) return e;
    hipLaunchKernelGGL(k_store_total, dim3(1), dim3(kWave), 0, s, counter, pairs_out);
    return hipGetLastError();
}

}  // namespace tam
