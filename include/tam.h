/*
 * tam.h -- trie-automaton token masks for constrained decoding over a finite
 * set of strings, on AMD Instinct MI355X (gfx950).
 *
 * The method (Section 2, Eq. 1 and Section 4.1): a finite set E of K strings
 * is an enum constraint.  A character-level (here: byte-level) trie over E has
 * one node per distinct prefix.  For every node n the set valid[n] holds the
 * vocabulary tokens whose bytes, walked from n, stay inside the trie; decoding
 * masks the logits of every other token to -inf and then moves the state along
 * the sampled token's bytes.  Because that valid-set test only needs the walk to
 * survive (appendix "Correctness", conditions (i)-(ii)), the masks are exact,
 * not an approximation.
 *
 * This library computes, on one GPU:
 *   tam_compile    -- the trie (host) and the dense per-node bitmask table
 *                     mask[n][v] = [token v is valid at node n] (device);
 *   tam_apply_mask -- logits[b, v] = -inf where mask[node_ids[b]][v] == 0, in place;
 *   tam_advance    -- out[b] = the node reached from node_ids[b] by the bytes of
 *                     token_ids[b], or TAM_DEAD.
 *
 * Conventions fixed by this interface (the paper leaves them open):
 *   - End of a value: every string is followed by a terminator byte T
 *     (tam_options.terminator, default '"' = 0x22) inserted as an ordinary trie
 *     edge.  The node after T is final; its row is empty (a caller stops
 *     decoding there).  A token that runs past T is invalid.
 *   - A set string containing T is rejected (TAM_E_TERMINATOR).  Duplicate
 *     strings collapse; the empty string is allowed.
 *   - Node ids: the rank of the node's prefix in bytewise lexicographic order
 *     with a proper prefix before its extensions (DFS preorder, children in
 *     ascending byte order); the root of a single set is 0.  In a forest of S
 *     sets, set j occupies ids [roots[j], roots[j] + N_j) after sets 0..j-1.
 *   - TAM_DEAD (-1) is the absorbing dead state.  A node id outside [0, N) is
 *     treated as dead; a token id outside [0, V) or an empty token is never
 *     valid (empty tokens are the paper's special tokens without characters).
 *   - Canonical mask row (tam_export_rows): W = ceil(V/64) little-endian 64-bit
 *     words, token v is bit (v & 63) of word (v >> 6), bits >= V are zero.
 *
 * Memory and streams: device memory comes from the caller's allocator
 * (tam_allocator; NULL = hipMalloc/hipFree).  The large host tables of a device
 * compile (1 MiB or more) are page-locked blocks (hipHostMalloc) from a
 * process-wide pool: a destroyed handle's blocks are kept for reuse, up to
 * 4 GiB of idle blocks, so later compiles upload them by direct DMA.  Every device operation is
 * enqueued on the caller's HIP stream (`stream`, a hipStream_t passed as void*;
 * NULL = the null stream) and returns without synchronising, except where a
 * function says otherwise.  A handle is immutable after tam_compile (only
 * tam_rebuild rewrites its table in place), so apply/advance/export calls may
 * run concurrently on any streams once the compile stream has been waited on;
 * TAM_FLAG_LAZY_ROWS handles are the exception (their row cache changes).
 *
 * Errors: every entry point returns a tam_status; a negative status leaves a
 * message in tam_last_error() (thread-local).  No exception crosses the ABI.
 * Argument errors (TAM_E_INVAL) are reported before the handle's state
 * (TAM_E_STATE).  Per-row conditions on the device (dead or out-of-range ids)
 * are not errors.  An asynchronous HIP failure surfaces as TAM_E_DEVICE on a
 * later call.  The kernels that lay the trie out on the device, and the row
 * cache of TAM_FLAG_LAZY_ROWS, count any table entry or cache state that is
 * inconsistent (the library's own build makes none) instead of following it;
 * the count is copied back at the end of tam_compile and tam_rebuild (not
 * under stream capture), and once it is non-zero every later tam_apply_mask,
 * tam_advance, tam_export_rows, tam_rebuild and tam_valid_pairs call on the
 * handle returns TAM_E_DEVICE.
 */
#ifndef TAM_H
#define TAM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TAM_DEAD (-1)

typedef struct tam_handle tam_handle;
typedef struct tam_vocab tam_vocab;

typedef enum {
    TAM_OK = 0,
    TAM_E_INVAL = -1,      /* bad argument (null pointer, negative size, bad dtype, ...) */
    TAM_E_TERMINATOR = -2, /* a set string contains the terminator byte */
    TAM_E_NOMEM = -3,      /* host allocation, a host thread or the device allocator failed */
    TAM_E_DEVICE = -4,     /* a HIP call failed, or the device met inconsistent trie tables */
    TAM_E_TOOLARGE = -5,   /* sizes beyond the 32-bit index limits of the tables */
    TAM_E_STATE = -6       /* operation not available for this handle (see flags) */
} tam_status;

enum { TAM_DTYPE_FP32 = 0, TAM_DTYPE_BF16 = 1 };

enum {
    /* Build the host tables only: no HIP call, no device memory.  tam_info_get
     * works; every device entry point returns TAM_E_STATE. */
    TAM_FLAG_HOST_ONLY = 1u << 0,
    /* Keep only the sparse per-node valid lists, no dense [N, W] table: apply
     * and export then build each requested row on the fly (for forests whose
     * dense table would not fit, e.g. hundreds of per-query sets). */
    TAM_FLAG_NO_TABLE = 1u << 1,
    /* Record HIP events around each device phase of tam_compile/tam_rebuild
     * so that tam_timing_get can report per-phase times. */
    TAM_FLAG_TIMING = 1u << 2,
    /* Tail compression: dense rows only for branching nodes (two or more final
     * nodes below them).  A tail node (its subtree is one path, ending in a
     * single final node) has as valid tokens only prefixes of its one
     * remaining suffix, at most one per length (per distinct token string):
     * the short valid lists of the Appendix's memory-vs-speed trade-off.  They
     * are not stored: the path below a tail has consecutive ids, so the token
     * of length d starting below tail a is the suffix hit of node a+d, kept by
     * the probe pass; tokens longer than 16 bytes go to per-node lists.
     * Results are identical to the full table, which holds dense_rows rows
     * instead of N (c. 2.5% of the nodes of a set of 10,000 code-like
     * strings).  With TAM_FLAG_NO_TABLE there is no table at all: the
     * branching nodes keep sparse valid lists instead of dense rows (the
     * tails still read theirs from the probe hits), so a forest of many
     * per-query sets lists only 1-2% of its nodes. */
    TAM_FLAG_TAIL_LISTS = 1u << 3,
    /* Rows built on demand (the lazy computation of the Appendix's memory
     * discussion, with the matching restricted to the subtree below the
     * current node): compile computes no mask, only the trie, its subtree
     * extents and an empty cache of tam_options.cache_rows dense rows.
     * tam_apply_mask looks the rows of its nodes up in the cache; the row of a
     * node that is not there is built in that call, by suffix probes over the
     * node's subtree (every descendant at most max_token_len bytes deeper), in
     * a cache slot freed by CLOCK replacement (second chance, an approximation
     * of least-recently-used eviction).  Masks are identical to the
     * precomputed table's.  tam_apply_mask and tam_export_rows (which builds
     * the requested rows the same way, outside the cache) update device state
     * held by the handle: their calls on one handle must not overlap (use one
     * stream, or order the streams).  Takes precedence over TAM_FLAG_NO_TABLE
     * and TAM_FLAG_TAIL_LISTS. */
    TAM_FLAG_LAZY_ROWS = 1u << 4
};

/* Device allocator.  alloc returns device memory aligned to at least 256 bytes
 * (or NULL); free releases it.  Both are called on the calling thread, from
 * tam_compile and tam_destroy only. */
typedef struct {
    void *(*alloc)(size_t bytes, void *ctx);
    void (*free)(void *ptr, void *ctx);
    void *ctx;
} tam_allocator;

typedef struct {
    int terminator;      /* 0..255; default 0x22 */
    uint32_t flags;      /* TAM_FLAG_* */
    int64_t cache_rows;  /* TAM_FLAG_LAZY_ROWS: rows of the row cache; 0 = 4096; at most N is used */
} tam_options;

/* Read-only view of a compiled handle.  Host pointers stay valid until
 * tam_destroy; `table` is device memory owned by the handle. */
typedef struct {
    int64_t num_nodes;        /* N over all sets, including roots and final nodes */
    int64_t num_sets;         /* S */
    int64_t num_strings;      /* distinct strings over all sets */
    int64_t vocab_size;       /* V */
    int64_t words_per_row;    /* W = ceil(V/64), canonical row length */
    int64_t row_stride_words; /* stride of the dense table in words (>= W); 0 without a table */
    int64_t max_token_len;    /* longest token in bytes */
    int64_t device_bytes;     /* device memory held by the handle */
    uint32_t flags;
    int32_t terminator;
    const int32_t *roots;     /* [S] root id of each set */
    const int32_t *parent;    /* [N] parent id, -1 at roots */
    const int32_t *depth;     /* [N] prefix length in bytes (roots: 0) */
    const uint8_t *edge_byte; /* [N] byte on the edge into the node (roots: 0) */
    const uint8_t *is_final;  /* [N] 1 if the node is reached by the terminator */
    const uint64_t *table;    /* device [dense_rows][row_stride_words]; NULL with TAM_FLAG_NO_TABLE */
    int64_t dense_rows;       /* rows of `table`: N, or the branching nodes with TAM_FLAG_TAIL_LISTS,
                                 or 0 without a table */
    const int32_t *dense_row; /* [N] with TAM_FLAG_TAIL_LISTS: table row (or, with
                                 TAM_FLAG_NO_TABLE, number) of each branching node (>= 0);
                                 for a tail node a, -1 - (number of nodes below a).  NULL
                                 otherwise */
    int64_t cache_rows;        /* TAM_FLAG_LAZY_ROWS: rows of the row cache (else 0) */
    const int32_t *subtree_end; /* [N] with TAM_FLAG_LAZY_ROWS: one past the last node of the
                                 node's subtree (preorder ids); else NULL */
    int64_t list_capacity;     /* valid-list entries allocated: a host-computed upper bound on
                                  the listed (node, token) pairs (0 without lists) */
} tam_info;

/* Host-side wall times of the last tam_compile, and device times (HIP events,
 * only with TAM_FLAG_TIMING; else -1) of the last tam_compile/tam_rebuild that
 * ran the handle's default phases. */
typedef struct {
    double host_trie_ms;   /* dedupe, sort, preorder trie, child tables */
    double host_vocab_ms;  /* token offsets, vocabulary hash, length table */
    double upload_ms;      /* allocation + enqueue of the host-to-device copies */
    float dev_lists_ms;    /* sparse valid lists after the probe pass: prefix sum, fill */
    float dev_zero_ms;     /* zero fill of the dense table */
    float dev_mark_ms;     /* the probe pass: suffix probes, table marks, list counts */
    float dev_total_ms;    /* first device phase start to last device phase end; a compile of a
                              full table enqueues its zero fill while the host still writes the
                              trie, so this span then includes waiting for the host and uploads */
} tam_timing;

/*
 * tam_compile -- build the trie of each set and its per-node token masks
 * (Section 4.1; the valid[n] sets, precomputed once per set).
 *
 *   str_bytes, str_off  K strings in CSR form: string k is
 *                       str_bytes[str_off[k] .. str_off[k+1]); str_off has K+1
 *                       non-decreasing entries, str_off[0] = 0.  Host memory.
 *   K                   number of strings, >= 1.
 *   tok_bytes, tok_off  V vocabulary tokens in the same CSR form (token id = index).
 *                       Host memory.  Tokens may repeat (each id gets its own bit)
 *                       and may be empty (never valid).
 *   V                   vocabulary size, >= 1.
 *   set_off, S          forest: set j is strings set_off[j] .. set_off[j+1]-1
 *                       (S+1 entries, set_off[0] = 0, set_off[S] = K, every set
 *                       non-empty).  NULL / 0 = one set of all K strings.
 *   opt                 NULL = defaults (terminator '"', no flags).
 *   alloc               NULL = hipMalloc / hipFree.
 *   stream              HIP stream for the uploads and kernels.
 *   out                 receives the handle (NULL on failure).
 *
 * All host inputs are copied before return.  The device work is enqueued on
 * `stream` and may still be running when tam_compile returns; wait on the
 * stream before using the table from another stream.
 * Errors: TAM_E_INVAL, TAM_E_TERMINATOR, TAM_E_NOMEM, TAM_E_DEVICE,
 * TAM_E_TOOLARGE (N, the string bytes or the token bytes beyond 2^31-1).
 */
tam_status tam_compile(const uint8_t *str_bytes, const int64_t *str_off, int64_t K,
                       const uint8_t *tok_bytes, const int64_t *tok_off, int64_t V,
                       const int64_t *set_off, int64_t S,
                       const tam_options *opt, const tam_allocator *alloc, void *stream,
                       tam_handle **out);

/*
 * tam_vocab_create -- the vocabulary side of the masks, built once per
 * tokenizer and shared by every compile against it (the paper keeps its
 * vocabulary matcher per tokenizer and reuses it across schemas, Section 4.2
 * and the deployment paragraph of Section 5): token offsets, an exact hash of
 * every distinct token string, duplicate chains and the token-length table,
 * uploaded on `stream`.
 *
 *   tok_bytes, tok_off  V tokens in CSR form (as for tam_compile).  Host memory,
 *                       copied before return.
 *   flags               TAM_FLAG_HOST_ONLY (no device copy, for host-only
 *                       compiles) or 0; other bits are ignored.
 *   alloc               NULL = hipMalloc / hipFree; it must stay valid until the
 *                       vocabulary is freed (after its last handle).
 * The vocabulary is reference counted: every handle compiled against it holds
 * a reference, and tam_vocab_destroy drops the caller's.  Errors: TAM_E_INVAL,
 * TAM_E_NOMEM, TAM_E_DEVICE, TAM_E_TOOLARGE (V or token bytes beyond 2^31-1, a
 * token longer than 65,535 bytes, a byte string shared by more than 65,535 ids).
 */
tam_status tam_vocab_create(const uint8_t *tok_bytes, const int64_t *tok_off, int64_t V, uint32_t flags,
                            const tam_allocator *alloc, void *stream, tam_vocab **out);

/* tam_vocab_destroy -- drops the caller's reference (NULL is a no-op). */
void tam_vocab_destroy(tam_vocab *vocab);

/*
 * tam_compile_vocab -- tam_compile against a vocabulary built by
 * tam_vocab_create (same arguments otherwise, same result): per set, only the
 * trie is built on the host; the vocabulary's device tables are reused.  The
 * handle must live on the vocabulary's device; a device compile needs a
 * vocabulary built without TAM_FLAG_HOST_ONLY (else TAM_E_STATE).
 */
tam_status tam_compile_vocab(const uint8_t *str_bytes, const int64_t *str_off, int64_t K,
                             const tam_vocab *vocab, const int64_t *set_off, int64_t S,
                             const tam_options *opt, const tam_allocator *alloc, void *stream,
                             tam_handle **out);

/*
 * tam_compile_format -- character-position masks of a fixed-format value
 * (Appendix, Constraint-Aware Dispatch Beyond Finite Sets): character p
 * (0 <= p < L) of a value may be any byte of class p, and the value is then
 * closed by the terminator, as set strings are.  The handle's nodes are the
 * positions: node p = p characters written (0..L), node L+1 = after the
 * terminator (final, empty row).  Token v is valid at node p iff it is
 * non-empty, p + |t_v| <= L + 1 and byte i of t_v lies in class p+i, class L
 * being {terminator}; the advance moves to p + |t_v|, else TAM_DEAD.  Every
 * serving entry point works on the handle; tam_info_get reports parent p-1,
 * depth p, edge byte 0 (the terminator for node L+1), num_strings 0, and a
 * dense table of L+2 rows.
 *
 *   classes  host uint8[L][32]: byte c is in class p iff bit (c & 7) of
 *            classes[32 p + (c >> 3)] is set (copied).  No class may admit the
 *            terminator (TAM_E_TERMINATOR).  L >= 1.
 *   vocab    a vocabulary from tam_vocab_create (a device one unless
 *            opt->flags asks for TAM_FLAG_HOST_ONLY); the handle keeps a
 *            reference.
 *   opt      terminator; flags TAM_FLAG_HOST_ONLY and TAM_FLAG_TIMING (the
 *            representation flags do not apply).  NULL = defaults.
 *   alloc, stream, out   as for tam_compile.
 */
tam_status tam_compile_format(const uint8_t *classes, int64_t L, const tam_vocab *vocab,
                              const tam_options *opt, const tam_allocator *alloc, void *stream,
                              tam_handle **out);

enum {
    TAM_PHASE_LISTS = 1u << 0, /* sparse per-node valid lists (suffix probes, prefix sum, fill);
                                  with TAM_PHASE_MARK one probe pass serves both */
    TAM_PHASE_ZERO = 1u << 1,  /* zero fill of the dense table */
    TAM_PHASE_MARK = 1u << 2,  /* suffix probes setting the valid bits of the zeroed table */
    TAM_PHASE_TABLE = TAM_PHASE_ZERO | TAM_PHASE_MARK,
    TAM_PHASE_COUNT = 1u << 3  /* (with lists) the probe pass that writes the hits and counts the
                                  lists, without the prefix sum and fill: the lists already built
                                  stay as they are (the pass recomputes the same hits); for timing
                                  the probe pass alone */
};

/*
 * tam_rebuild -- rerun device phases of tam_compile from the handle's resident
 * device tables (bit-identical result).  `phases` is a TAM_PHASE_* mask; 0 =
 * the handle's default: TAM_PHASE_TABLE for a table (TAM_PHASE_MARK for a
 * format handle, which recomputes every word of its rows), TAM_PHASE_LISTS with
 * TAM_FLAG_NO_TABLE (with or without TAM_FLAG_TAIL_LISTS), both with
 * TAM_FLAG_TAIL_LISTS and a table when the vocabulary has tokens longer than
 * 16 bytes.  A phase the handle does not keep returns
 * TAM_E_STATE.  TAM_PHASE_MARK without TAM_PHASE_ZERO ORs the
 * same bits into the current table.  Used to time the device phase kernel by
 * kernel.  With TAM_FLAG_LAZY_ROWS the only phase is 0: it empties the row
 * cache, so that every row is built again on its next use.
 */
tam_status tam_rebuild(tam_handle *h, unsigned phases, void *stream);
/* HIP graphs: tam_rebuild, tam_apply_mask, tam_advance and tam_export_rows only
 * launch kernels on `stream`, so they may be captured into a graph (no memset
 * or event nodes are recorded; the handle must outlive every replay, and
 * tam_destroy does not wait for replays still running: synchronise first).
 * tam_valid_pairs and tam_timing_get synchronise and must not be captured. */

/* tam_info_get -- sizes and host tables of a handle (no device access).  The
 * dense table it names holds one bitmask row per node (appendix "GPU-Based
 * Masking Considerations": the masks are kept as per-node bitmasks on the GPU),
 * or per branching node with TAM_FLAG_TAIL_LISTS. */
tam_status tam_info_get(const tam_handle *h, tam_info *out);

/* Position tables of a trie as the device lays them out on a device compile
 * (Section 4.1: one node per distinct prefix, every string written once into a
 * blob in trie order).  All arrays are host memory owned by the handle. */
typedef struct {
    int64_t blob_bytes;
    const uint8_t *blob;      /* [blob_bytes]: 32 zero bytes; then for each set in order, for each
                                 of its distinct strings in node-id (trie) order, a zero pad byte,
                                 the string's bytes and the terminator; then 32 zero bytes */
    const int32_t *node_at;   /* [blob_bytes] node whose edge byte sits at that position; a pad
                                 byte stands for its set's root, the outer pads for root 0 */
    const int32_t *depth;     /* [N] prefix length (-1 for a node no record reaches) */
    const int32_t *node_pos;  /* [N] first position of the node's edge byte; -1 at roots */
    const int32_t *parent;    /* [N] node_at[node_pos - 1]; -1 at roots and unplaced nodes */
    int64_t errors;           /* inconsistent string records or positions met (0 for the
                                 library's own build; on the device the same count makes later
                                 calls return TAM_E_DEVICE) */
} tam_layout;

/*
 * tam_layout_get -- the device's trie layout computed on the host: the same
 * functions the layout kernels run on the device (node_at and depth from one
 * record per string, first positions, parents), run over the same records, so
 * that the layout can be checked without a GPU.  Only for TAM_FLAG_HOST_ONLY
 * handles of string sets (else TAM_E_STATE); computed at the first call, kept
 * until tam_destroy.  Errors: TAM_E_INVAL (null argument), TAM_E_STATE,
 * TAM_E_NOMEM.
 */
tam_status tam_layout_get(const tam_handle *h, tam_layout *out);

/*
 * tam_apply_mask -- Eq. 1 with the precomputed masks: for every row b in
 * [0, B) and token v in [0, V),
 *     logits[b * row_stride + v] = -inf   if token v is not valid at node_ids[b],
 * and the entry is left bit-for-bit unchanged otherwise (NaN payloads, -0.0 and
 * denormals survive).  A dead or out-of-range node masks the whole row.
 * Columns v >= V of a row are not touched.
 *
 *   node_ids    device int32[B].
 *   logits      device, B rows of row_stride elements, dtype TAM_DTYPE_FP32
 *               (-inf = 0xFF800000) or TAM_DTYPE_BF16 (-inf = 0xFF80).
 *   row_stride  elements between rows, >= V.
 * Rows whose base is 16-byte aligned take the vector path; any other layout is
 * still handled (element path).  B = 0 is a no-op.
 * Errors: TAM_E_INVAL (B < 0, a null pointer with B > 0, dtype not FP32 or
 * BF16, row_stride < V, logits not aligned to their element size),
 * TAM_E_STATE (host-only handle), TAM_E_DEVICE.  With TAM_FLAG_LAZY_ROWS the
 * rows of nodes missing from the row cache are built first (see the flag), in
 * groups of at most min(1024, cache rows) batch rows.
 */
tam_status tam_apply_mask(const tam_handle *h, const int32_t *node_ids, int64_t B, void *logits,
                          int dtype, int64_t row_stride, void *stream);

/*
 * tam_advance -- the state transition extended over a token's bytes
 * (Section 2, the start state moved along the characters of the output):
 *     out[b] = delta*(node_ids[b], bytes(token_ids[b]))   or TAM_DEAD.
 * node_ids, token_ids and out are device int32[B]; out may alias node_ids.
 */
tam_status tam_advance(const tam_handle *h, const int32_t *node_ids, const int32_t *token_ids,
                       int64_t B, int32_t *out, void *stream);

/*
 * tam_export_rows -- canonical mask rows of n nodes: out is device
 * uint64[n][W] (W = words_per_row); row r is the mask of node_ids[r], or all
 * zero when node_ids[r] is dead or out of range.  The canonical row is this
 * interface's reading of the appendix's "GPU-Based Masking Considerations"
 * (one bitmask per trie node, a bit per vocabulary token), whatever the
 * handle keeps internally (dense rows, tails read back from the probe hits,
 * sparse lists, or rows built on demand).
 *   node_ids  device int32[n]; out  device, 8-byte aligned, written whole.
 * Errors: TAM_E_INVAL (null pointer with n > 0, n < 0, misaligned out),
 * TAM_E_STATE (host-only handle), TAM_E_DEVICE.
 */
tam_status tam_export_rows(const tam_handle *h, const int32_t *node_ids, int64_t n, uint64_t *out,
                           void *stream);

/*
 * tam_valid_counts -- out[r] = |valid[node_ids[r]]|, the number of token ids
 * valid at that node (0 for a dead or out-of-range node): the valid-set sizes
 * the appendix tabulates by trie depth ("Valid set size distribution"), and
 * what a caller needs to choose between masking with the row and sampling
 * from a short valid list.  Counted on the device from the handle's own rows
 * (popcount of a dense row, a list's length, a tail's hits).
 *   node_ids, out  device int32[n].
 * Errors: TAM_E_INVAL, TAM_E_STATE (host-only handle, or TAM_FLAG_LAZY_ROWS:
 * no row is kept for most nodes), TAM_E_DEVICE.
 */
tam_status tam_valid_counts(const tam_handle *h, const int32_t *node_ids, int64_t n, int32_t *out, void *stream);

/*
 * tam_valid_pairs -- M = sum over all nodes of |valid[n]|, the number of
 * (node, token) pairs that are valid, as found by the last table or list
 * build.  Copies the per-block counts from the device and synchronises
 * `stream`.  TAM_E_STATE with TAM_FLAG_LAZY_ROWS (no pass over all nodes).
 */
tam_status tam_valid_pairs(const tam_handle *h, void *stream, int64_t *out);

/* tam_timing_get -- see tam_timing.  Waits for the last recorded device event. */
tam_status tam_timing_get(const tam_handle *h, tam_timing *out);

/* tam_destroy -- waits for the device work the handle enqueued itself (its
 * compile and tam_rebuild calls), then frees it.  Apply, advance and export
 * calls are the caller's: wait for their streams first.  NULL is a no-op. */
void tam_destroy(tam_handle *h);

/* Largest L that tam_format_rows_noalloc takes. */
#define TAM_NOALLOC_MAX_POSITIONS 1024

/*
 * tam_format_rows_noalloc -- for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the character-position masks of tam_compile_format written
 * straight into the caller's memory, with no handle and no allocation (no
 * hipMalloc, no allocator callback, no pageable copy: the class bits travel as
 * kernel arguments).
 *   classes     host uint8[L][32], as for tam_compile_format; 1 <= L <=
 *               TAM_NOALLOC_MAX_POSITIONS (else TAM_E_INVAL).
 *   terminator  0..255; no class may admit it (TAM_E_TERMINATOR).
 *   vocab       a device vocabulary (tam_vocab_create without
 *               TAM_FLAG_HOST_ONLY, else TAM_E_STATE) on the current device.
 *   out         device uint64[L + 2][out_stride_words], 8-byte aligned,
 *               out_stride_words >= W: row p receives the canonical row of
 *               position p (rows 0..L, then L+1 after the terminator, all zero);
 *               words W.. of each row are left as they are.
 *   pairs_out   device int64[1] for the number of valid (position, token)
 *               pairs, or NULL.
 * Scratch: the class bits and a pair counter live in a static device array of
 * 256 + 32 * TAM_NOALLOC_MAX_POSITIONS bytes per GPU, held until the process
 * ends and shared by every call on that GPU: calls that overlap on one GPU
 * (different streams, or threads without ordering) race; order them.  The
 * result equals tam_export_rows of a tam_compile_format handle, row for row.
 * Errors: TAM_E_INVAL, TAM_E_TERMINATOR, TAM_E_STATE, TAM_E_DEVICE.
 */
tam_status tam_format_rows_noalloc(const uint8_t *classes, int64_t L, int terminator, const tam_vocab *vocab,
                                   uint64_t *out, int64_t out_stride_words, int64_t *pairs_out, void *stream);

/* Message of the last failing call on this thread ("" if none). */
const char *tam_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TAM_H */
