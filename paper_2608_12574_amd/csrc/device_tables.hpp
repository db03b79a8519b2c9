// Definitions shared by the HIP kernels and the host code of libtam: the
// vocabulary hash, the device view of a handle and the row cache of rows
// built on demand.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace tam {

// ---------------------------------------------------------------------------
// Vocabulary hash: keys are the token bytes read last-to-first, so that a
// suffix of a trie path can be hashed incrementally while walking backwards
// from the node where it ends.  Host (table build) and device (probe) must
// agree bit for bit, hence one definition for both.  The state is 32-bit
// FNV-1a (one multiply per byte); the key is the 64-bit product of the state
// with an odd constant, its halves swapped: the low 32 bits (the home bucket)
// are the product's well-mixed high half, the high 16 bits (the fingerprint)
// come from its low half, which is a bijection of the state.  Two strings with
// equal states share bucket and fingerprint; the payload compare tells them
// apart.
// ---------------------------------------------------------------------------
constexpr uint32_t kHashSeed = 0x811c9dc5u;

__host__ __device__ __forceinline__ uint32_t hash_step(uint32_t h, uint32_t byte) {
    return (h ^ (byte + 1u)) * 0x01000193u;
}

__host__ __device__ __forceinline__ uint64_t hash_final(uint32_t h) {
    const uint64_t p = (uint64_t)h * 0x9e3779b1ull;
    return ((p >> 32) | (p << 32)) | 1ull;  // 0 never occurs as a key
}

// Vocabulary table: open addressing over buckets of kBucket slots, one slot
// per distinct non-empty token string.  A bucket is 16 bytes (one load): four
// words, word i holding the 12-bit fingerprints of slots 2i and 2i + 1 in bits
// 0..23 and byte i of the bucket's base in bits 24..31.  The strings of the
// table are numbered bucket by bucket (a bucket's used slots come first), the
// base being the number of the bucket's first slot, so a slot's string is
// base + its index in the bucket.  That number indexes the 16-byte payloads
// (its first 8 bytes stored last byte first, its smallest token id, length and
// duplicate count), read only on a fingerprint match, with one load; bytes
// 8..15 of a longer token sit in pay_hi[number] and are read only when the
// first 8 match.  Payloads exist only for strings, not for empty slots, so the
// tables the probes read stay small.  Suffixes of at most kShortLen bytes skip
// the hash: short_hits maps them straight to their hit (short_index).
constexpr int kBucket = 8;    // fingerprints per bucket
constexpr int kWin = 16;      // path bytes a probing node keeps in registers
constexpr int kBlobPad = 32;  // zero bytes before and after the string blob (and after the token blob)
constexpr int kShortLen = 2;  // suffix lengths answered by short_hits
constexpr int kShortEntries = 256 + 65536;

__host__ __device__ __forceinline__ uint32_t fingerprint(uint64_t key) {
    return (uint32_t)(key >> 52) | 1u;  // 12 bits; 0 marks an empty slot
}

// Index in short_hits of the string of d <= kShortLen bytes whose last byte is
// `last` and (d = 2) whose first byte is `prev`.
__host__ __device__ __forceinline__ int32_t short_index(int d, uint32_t last, uint32_t prev) {
    return d == 1 ? (int32_t)last : 256 + (int32_t)((prev << 8) | last);
}

struct alignas(16) SlotPay {
    uint64_t lo;      // byte k = token byte len-1-k for k < min(len, 8), then zeros
    int32_t first;    // smallest token id with this string (-1: empty slot)
    uint16_t len;     // string length in bytes
    uint16_t count;   // number of token ids with this string
};
// pay_hi[string]: byte k - 8 = token byte len-1-k for 8 <= k < min(len, 16),
// then zeros (0 for strings of at most 8 bytes).

// What the probe pass stores per (node, suffix length): the token id when the
// string has one id, -2 - its string number when it has several, -1 when no
// token matches.
__host__ __device__ __forceinline__ int32_t hit_of_slot(int32_t slot, int32_t first, int count) {
    return count == 1 ? first : -2 - slot;
}

// One string of the trie's blob, in blob order; the device lays out node_at
// and depth from these.  at: position of its pad byte; len: its length (the
// terminator follows at at + 1 + len); lcp: its common prefix with the
// previous string of its part; first: id of the first node it creates (at
// path index lcp); psv: the nearest earlier string of its part with a shorter
// common prefix (-1: none); root: its set's root.
struct StrRec {
    int32_t at, len, lcp, first, psv, root;
};

// Tail compression: per string, what classifies the nodes it creates (path
// indices lcp .. len).  Those below index `next` (the next string's common
// prefix in its part) are branching and take dense rows row, row + 1, ... in
// order; the others are tails, with len - i nodes below them and
// tail_span = i - top (top: the path index above the string's highest tail,
// -1 when the set's root is itself a tail).
struct TailRec {
    int32_t row, next, top;
};

// ---------------------------------------------------------------------------
// Device-side view of a compiled handle (plain pointers, passed to kernels).
// ---------------------------------------------------------------------------
// Tail compression without a table: the probe grid in the groups of whole
// sets that the compile uploads one after another.  Group k covers the nodes
// [n_lo[k], n_hi[k]) with the probe blocks [blk0[k], blk0[k + 1]) (block
// blk0[k] + j holds nodes n_lo[k] + j * nodes-per-block ..), their region
// offsets at rec_off[off0[k] ..] and their records in rec[k].
constexpr int kMaxRecGroups = 4;
struct RecGroups {
    int64_t n_lo[kMaxRecGroups], n_hi[kMaxRecGroups];
    int64_t blk0[kMaxRecGroups + 1];
    int64_t off0[kMaxRecGroups];
    int32_t *rec[kMaxRecGroups];  // [3 * the group's region total]
    int32_t n;                    // groups (0: the grid is the plain one)
};

struct DevTables {
    // trie (a1)
    const uint8_t *blob;        // [pad 32][per string: pad, bytes, T][pad 32]
    const int32_t *node_at;     // [blob_bytes] node whose edge byte is that blob byte (pad: root)
    const int32_t *node_pos;    // [N] blob offset of the node's edge byte (-1 at roots)
    const int32_t *depth;       // [N]
    const int32_t *child_off;   // [N+1]
    const uint8_t *child_byte;  // [N-S]
    const int32_t *child_node;  // [N-S]
    const int32_t *child_pos;   // [N-S] node_pos of child_node[k]: where a walk goes on along its string
    const uint64_t *child_at;   // [blob_bytes] child range of node_at[p]: child_off lo | hi << 32
    // vocabulary (a2)
    const uint32_t *tok_off;    // [V+1]
    const uint8_t *tok_blob;
    const uint16_t *fps;        // [slot_mask+1] fingerprints, kBucket per bucket
    const SlotPay *pay;         // [slot_mask+1]
    const uint64_t *pay_hi;     // [slot_mask+1] bytes 8..15 of the reversed token
    const int32_t *short_hits;  // [kShortEntries] hit_of_slot of every string of <= kShortLen bytes, or -1
    const int32_t *dup_next;    // [V] next id with the same bytes, -1 at the end
    const uint8_t *len_present; // [max_len+1] 1 if some token has that length
    // valid lists (a4) and dense table
    int32_t *hits;              // [kWin][N] hit_of_slot of the suffix of length d+1 of node m, or -1
    int32_t *count;             // [N]
    int32_t *row_ptr;           // [N+1]
    int32_t *cursor;            // [N]
    int32_t *entries;           // [entry_bound]
    uint64_t *table;            // [R][Wp] or null
    // tail compression (null unless the handle has both a table and lists):
    // hits at distance d <= tail_span[m] above node m land on tail nodes (lists),
    // the others on branching nodes (dense rows row_of[node])
    const int32_t *tail_span;   // [N]
    const int32_t *row_of;      // [N] dense row of a node; a tail a: -1 - (nodes below a); null: row = node id
    const int32_t *row_at;      // [blob_bytes] row_of[node_at[p]]; equals node_at without row_of
    const int32_t *sub_end;     // [N] one past the node's subtree (rows built on demand), or null
    // tail compression without a table: each listed hit's record (node, rank
    // in the node's list, hit), written by the probe pass into its block's
    // region of its group's records (RecGroups) and placed by k_fill_records
    // once the lists' offsets are known
    const int32_t *rec_off;     // per group, its blocks + 1 region offsets, in records
    int32_t *rec_cnt;           // [probe blocks] records each probe block wrote
    int32_t *scan_tmp;          // block sums of the scan
    int32_t *err;               // [1] inconsistent table entries met on the device (0 for the host
                                // build's tables); copied back and reported by later calls
    int64_t N, V, W, Wp;
    int64_t R;                  // dense rows (N for a full table, 0 without one)
    int32_t tail_long;          // tail compression with tokens longer than kWin: their hits on
                                // tails go to the lists (row_ptr / entries)
    int32_t tail_lists;         // tail compression without a table: the branching nodes' hits go
                                // to the lists, with the tails' tokens longer than kWin
    int64_t blob_bytes;
    uint64_t slot_mask;         // slots - 1 (slots = a power of two, >= kBucket)
    uint64_t len_mask;          // bit d (d < 64): some token has length d
    int32_t max_len;
    int32_t terminator;
    // character-position masks (tam_compile_format): classes of positions 0..L-1
    const uint8_t *classes;     // [L][32] bit rows, or null for a trie handle
    int32_t fmt_L;              // L, or -1 for a trie handle
};

// Rows built on demand (TAM_FLAG_LAZY_ROWS): the row cache, and the scratch
// of one group of at most kLazyGroup batch rows.  The cache has C + P rows:
// C hold nodes' rows (or are empty), P are spares, kept in a ring.  A miss
// takes the next spare, which is zero, and its CLOCK victim becomes a spare in
// its place; the build pass of the same group clears the victims' rows while
// it builds the misses' rows, so no row is cleared and built by one launch.
constexpr int kLazyGroup = 1024;
struct LazyDev {
    uint64_t *cache;       // [C + P][Wp] cached rows
    int32_t *slot_of;      // [N] cache row holding the node's row, or -1
    int32_t *node_of;      // [C + P] node whose row a cache row holds, -1 empty, -2 spare
    uint32_t *stamp;       // [C + P] number of the group that last used the row
    uint32_t *ref;         // [C + P] CLOCK reference bit
    uint32_t *state;       // [0] groups assigned so far, [1] CLOCK hand, [2] spare ring head
    int32_t *spare;        // [P] the spare rows, zero once the group that freed them has ended
    int32_t *rows_src;     // [kLazyGroup] cache row of each batch row of the group, -1 = dead
    int32_t *miss_node;    // [kLazyGroup] nodes whose rows are built, in batch-row order
    int32_t *miss_row;     // [kLazyGroup] their destination rows (cache rows, or output rows)
    int32_t *miss_free;    // [kLazyGroup] the cache rows their misses freed (cleared by the build)
    int64_t *miss_off;     // [kLazyGroup + 1] prefix sum of their subtree sizes (minus the node)
    int32_t *miss_dep;     // [kLazyGroup] depth of each miss
    int32_t *miss_count;   // [1]
    int32_t *err;          // [1] the handle's device error count (see DevTables)
    int64_t C;             // cache rows in use (the CLOCK's capacity)
    int64_t P;             // spare rows: min(C, kLazyGroup), at least the misses of one group
};

}  // namespace tam
