// Host part of tam_compile: the trie of every set (Section 4.1) and the
// vocabulary tables used by the device validity kernels.
#include <algorithm>
#include <atomic>
#include <cstring>
#include <numeric>
#include <thread>

#include "host_build.hpp"

namespace tam {

namespace {

// Bytewise order of s+T against u+T, where neither s nor u contains T.
struct TerminatedLess {
    const uint8_t *bytes;
    const int64_t *off;
    uint8_t T;
    bool operator()(int64_t a, int64_t b) const {
        const uint8_t *pa = bytes + off[a], *pb = bytes + off[b];
        int64_t la = off[a + 1] - off[a], lb = off[b + 1] - off[b];
        int64_t m = std::min(la, lb);
        int c = m ? std::memcmp(pa, pb, (size_t)m) : 0;
        if (c != 0) return c < 0;
        if (la == lb) return false;
        // one string is a proper prefix of the other: the shorter continues with T
        return la < lb ? T < pb[la] : pa[lb] < T;
    }
};

// The trie of one set, with set-local node ids (root = 0) and blob offsets.
struct SetTrie {
    std::vector<int32_t> parent, depth, node_pos, node_at, child_off, child_node;
    std::vector<uint8_t> edge, is_final, blob, child_byte;
    int64_t K_unique = 0;
    tam_status st = TAM_OK;
    std::string err;
};

/*
 * Trie construction of one set (Section 4.1: insert every value one byte at a
 * time, shared prefixes merge).  Inserting the distinct terminated strings in
 * sorted order creates the new nodes of each string right after its longest
 * common prefix with the previous string, and that creation order is exactly
 * the lexicographic preorder the interface fixes.  O(N_chars) after the sort.
 * Blob layout per string: one pad byte standing for the root, the string, T.
 */
void build_one_set(const uint8_t *sb, const int64_t *so, int64_t k0, int64_t k1, uint8_t term, SetTrie &r) {
    std::vector<int64_t> order((size_t)(k1 - k0));
    std::iota(order.begin(), order.end(), k0);
    std::sort(order.begin(), order.end(), TerminatedLess{sb, so, term});
    const int64_t chars = so[k1] - so[k0];
    const size_t est = (size_t)(chars + 2 * (k1 - k0) + 1);
    r.parent.reserve(est);
    r.depth.reserve(est);
    r.edge.reserve(est);
    r.is_final.reserve(est);
    r.node_pos.reserve(est);
    r.blob.reserve(est);
    r.node_at.reserve(est);
    r.parent.push_back(-1);
    r.depth.push_back(0);
    r.edge.push_back(0);
    r.is_final.push_back(0);
    r.node_pos.push_back(-1);
    int64_t N = 1;
    std::vector<int32_t> path;
    const uint8_t *prev = nullptr;
    int64_t prev_len = -1;
    for (int64_t k : order) {
        const uint8_t *s = sb + so[k];
        const int64_t len = so[k + 1] - so[k];
        int64_t l = 0;
        if (prev) {
            const int64_t m = std::min(len, prev_len);
            while (l < m && prev[l] == s[l]) ++l;
            if (l == len && len == prev_len) continue;  // duplicate string
        }
        prev = s;
        prev_len = len;
        ++r.K_unique;
        if ((int64_t)path.size() < len + 1) path.resize((size_t)(len + 1));
        r.blob.push_back(0);
        r.node_at.push_back(0);
        for (int64_t i = 0; i <= len; ++i) {
            const uint8_t c = i < len ? s[i] : term;
            r.blob.push_back(c);
            int32_t id;
            if (i < l) {
                id = path[(size_t)i];
            } else {
                id = (int32_t)N++;
                r.parent.push_back(i == 0 ? 0 : path[(size_t)(i - 1)]);
                r.depth.push_back((int32_t)(i + 1));
                r.edge.push_back(c);
                r.is_final.push_back(i == len ? 1 : 0);
                r.node_pos.push_back((int32_t)(r.blob.size() - 1));
            }
            path[(size_t)i] = id;
            r.node_at.push_back(id);
        }
        if (N >= INT32_MAX || (int64_t)r.blob.size() >= INT32_MAX) {
            r.st = TAM_E_TOOLARGE;
            r.err = "trie exceeds 2^31-1 nodes or string bytes";
            return;
        }
    }
    // children in ascending byte order = ascending ids (preorder)
    r.child_off.assign((size_t)(N + 1), 0);
    for (int64_t m = 1; m < N; ++m) ++r.child_off[(size_t)r.parent[(size_t)m] + 1];
    for (int64_t n = 0; n < N; ++n) r.child_off[(size_t)n + 1] += r.child_off[(size_t)n];
    r.child_node.resize((size_t)(N - 1));
    r.child_byte.resize((size_t)(N - 1));
    std::vector<int32_t> fill(r.child_off.begin(), r.child_off.end() - 1);
    for (int64_t m = 1; m < N; ++m) {
        const int32_t at = fill[(size_t)r.parent[(size_t)m]]++;
        r.child_node[(size_t)at] = (int32_t)m;
        r.child_byte[(size_t)at] = r.edge[(size_t)m];
    }
}

// Runs f(j) for j in [0, n) on up to `threads` host threads.
template <typename F>
void parallel_for(int64_t n, int threads, F f) {
    if (threads <= 1 || n <= 1) {
        for (int64_t j = 0; j < n; ++j) f(j);
        return;
    }
    std::atomic<int64_t> next{0};
    std::vector<std::thread> pool;
    for (int i = 0; i < threads; ++i)
        pool.emplace_back([&] {
            for (int64_t j = next.fetch_add(1); j < n; j = next.fetch_add(1)) f(j);
        });
    for (auto &th : pool) th.join();
}

int host_threads(int64_t work_items) {
    const unsigned hw = std::max(1u, std::thread::hardware_concurrency());
    return (int)std::min<int64_t>({(int64_t)hw, (int64_t)16, work_items});
}

}  // namespace

/*
 * Tries of all sets: each set is built on its own (in parallel over host
 * threads for a forest), then the sets are laid out one after another: set j
 * takes node ids [roots[j], roots[j] + N_j) and its own range of the blob,
 * which carries kBlobPad zero bytes in front and behind so that 16-byte
 * window loads around any node never leave it.
 */
tam_status build_trie(const uint8_t *sb, const int64_t *so, int64_t K, const int64_t *set_off,
                      int64_t S, int T, tam_handle *h, std::string *err) {
    const uint8_t term = (uint8_t)T;
    const int64_t total = so[K] - so[0];
    if (total > 0) {
        const void *hit = std::memchr(sb + so[0], term, (size_t)total);
        if (hit) {
            int64_t at = (const uint8_t *)hit - sb;
            int64_t k = std::upper_bound(so, so + K + 1, at) - so - 1;
            *err = "string " + std::to_string(k) + " contains the terminator byte";
            return TAM_E_TERMINATOR;
        }
    }
    std::vector<SetTrie> sets((size_t)S);
    std::atomic<bool> oom{false};
    parallel_for(S, host_threads(S), [&](int64_t j) {
        try {
            build_one_set(sb, so, set_off[j], set_off[j + 1], term, sets[(size_t)j]);
        } catch (const std::bad_alloc &) {
            oom = true;
        }
    });
    if (oom) throw std::bad_alloc();
    std::vector<int64_t> nbase((size_t)S + 1, 0), bbase((size_t)S + 1, kBlobPad), ebase((size_t)S + 1, 0);
    h->K_unique = 0;
    for (int64_t j = 0; j < S; ++j) {
        const SetTrie &r = sets[(size_t)j];
        if (r.st != TAM_OK) {
            *err = r.err;
            return r.st;
        }
        nbase[(size_t)j + 1] = nbase[(size_t)j] + (int64_t)r.parent.size();
        bbase[(size_t)j + 1] = bbase[(size_t)j] + (int64_t)r.blob.size();
        ebase[(size_t)j + 1] = ebase[(size_t)j] + (int64_t)r.child_node.size();
        h->K_unique += r.K_unique;
    }
    const int64_t N = nbase[(size_t)S];
    const int64_t BB = bbase[(size_t)S] + kBlobPad;
    const int64_t E = ebase[(size_t)S];
    if (N >= INT32_MAX || BB >= INT32_MAX) {
        *err = "trie exceeds 2^31-1 nodes or string bytes";
        return TAM_E_TOOLARGE;
    }
    h->N = N;
    h->S = S;
    h->blob_bytes = BB;
    h->roots.resize((size_t)S);
    h->parent.resize((size_t)N);
    h->depth.resize((size_t)N);
    h->edge.resize((size_t)N);
    h->is_final.resize((size_t)N);
    h->node_pos.resize((size_t)N);
    h->child_off.resize((size_t)N + 1);
    h->child_node.assign((size_t)std::max<int64_t>(E, 1), 0);
    h->child_byte.assign((size_t)std::max<int64_t>(E, 1), 0);
    h->blob.assign((size_t)BB, 0);
    h->node_at.assign((size_t)BB, 0);
    parallel_for(S, host_threads(S), [&](int64_t j) {
        const SetTrie &r = sets[(size_t)j];
        const int32_t nb = (int32_t)nbase[(size_t)j], bb = (int32_t)bbase[(size_t)j], eb = (int32_t)ebase[(size_t)j];
        const size_t n = r.parent.size();
        h->roots[(size_t)j] = nb;
        for (size_t i = 0; i < n; ++i) {
            h->parent[nb + i] = r.parent[i] < 0 ? -1 : r.parent[i] + nb;
            h->node_pos[nb + i] = r.node_pos[i] < 0 ? -1 : r.node_pos[i] + bb;
            h->child_off[nb + i] = r.child_off[i] + eb;
        }
        std::copy(r.depth.begin(), r.depth.end(), h->depth.begin() + nb);
        std::copy(r.edge.begin(), r.edge.end(), h->edge.begin() + nb);
        std::copy(r.is_final.begin(), r.is_final.end(), h->is_final.begin() + nb);
        std::copy(r.blob.begin(), r.blob.end(), h->blob.begin() + bb);
        for (size_t i = 0; i < r.node_at.size(); ++i) h->node_at[bb + i] = r.node_at[i] + nb;
        for (size_t i = 0; i < r.child_node.size(); ++i) h->child_node[eb + i] = r.child_node[i] + nb;
        std::copy(r.child_byte.begin(), r.child_byte.end(), h->child_byte.begin() + eb);
    });
    h->child_off[(size_t)N] = (int32_t)E;
    return TAM_OK;
}

/*
 * Vocabulary tables (the paper's vocabulary decoding and its per-tokenizer
 * matcher, built here as an exact hash of every distinct token string keyed by
 * its bytes read last-to-first).  Slots live in buckets of kBucket 16-bit
 * fingerprints; a key starts at its home bucket and moves to the next bucket
 * only when the bucket is full.  Duplicate strings share a slot and chain their
 * ids in ascending order.
 */
tam_status build_vocab(const uint8_t *tb, const int64_t *to, int64_t V, tam_vocab *h,
                       std::string *err) {
    const int64_t total = to[V] - to[0];
    if (total >= INT32_MAX) {
        *err = "vocabulary bytes exceed 2^31-1";
        return TAM_E_TOOLARGE;
    }
    h->V = V;
    h->W = (V + 63) / 64;
    h->tok_off.resize((size_t)(V + 1));
    h->tok_blob.assign(tb ? tb + to[0] : nullptr, tb ? tb + to[V] : nullptr);
    h->tok_blob.insert(h->tok_blob.end(), (size_t)kBlobPad, 0);  // room for 16-byte window loads
    int64_t max_len = 0;
    for (int64_t v = 0; v <= V; ++v) h->tok_off[(size_t)v] = (uint32_t)(to[v] - to[0]);
    for (int64_t v = 0; v < V; ++v) max_len = std::max<int64_t>(max_len, to[v + 1] - to[v]);
    if (max_len > 65535) {
        *err = "a token is longer than 65535 bytes";
        return TAM_E_TOOLARGE;
    }
    h->max_tok_len = max_len;
    h->len_present.assign((size_t)(max_len + 1), 0);
    h->len_mask = 0;

    uint64_t cap = 64;
    while (cap < (uint64_t)(2 * V)) cap <<= 1;
    const uint64_t nbuckets = cap / kBucket;
    h->fps.assign(cap, (uint16_t)0);
    h->pay.assign(cap, SlotPay{0, 0, -1, 0, 0, {0, 0}});
    h->dup_next.assign((size_t)V, -1);
    std::vector<int32_t> last(cap, -1);
    const uint8_t *blob = h->tok_blob.data();
    for (int64_t v = 0; v < V; ++v) {
        const uint32_t off = h->tok_off[(size_t)v];
        const uint32_t len = h->tok_off[(size_t)v + 1] - off;
        if (len == 0) continue;
        h->len_present[len] = 1;
        if (len < 64) h->len_mask |= 1ull << len;
        uint64_t hh = kHashSeed;
        for (int64_t i = (int64_t)len - 1; i >= 0; --i) hh = hash_step(hh, blob[off + i]);
        const uint64_t key = hash_final(hh, len);
        const uint16_t fp = (uint16_t)fingerprint(key);
        uint64_t b = (key & (cap - 1)) / kBucket;
        bool placed = false;
        while (!placed) {
            for (int i = 0; i < kBucket && !placed; ++i) {
                const uint64_t s = b * kBucket + (uint64_t)i;
                if (h->fps[s] == 0) {
                    h->fps[s] = fp;
                    SlotPay r{0, 0, (int32_t)v, (uint16_t)len, 1, {0, 0}};
                    for (uint32_t k = 0; k < len && k < 16; ++k) {
                        const uint64_t c = blob[off + len - 1 - k];
                        if (k < 8)
                            r.lo |= c << (8 * k);
                        else
                            r.hi |= c << (8 * (k - 8));
                    }
                    h->pay[s] = r;
                    last[s] = (int32_t)v;
                    placed = true;
                } else if (h->fps[s] == fp && h->pay[s].len == len) {
                    const uint32_t o2 = h->tok_off[(size_t)h->pay[s].first];
                    if (std::memcmp(blob + o2, blob + off, len) == 0) {
                        if (h->pay[s].count == 65535) {
                            *err = "more than 65535 tokens share one byte string";
                            return TAM_E_TOOLARGE;
                        }
                        h->dup_next[(size_t)last[s]] = (int32_t)v;
                        last[s] = (int32_t)v;
                        ++h->pay[s].count;
                        placed = true;
                    }
                }
            }
            b = (b + 1) % nbuckets;
        }
    }
    return TAM_OK;
}

/*
 * Upper bound on the number of valid (node, token) pairs, used to size the
 * sparse lists without a device round trip: node m can end at most one distinct
 * token string of each length d <= min(depth(m), max_len), carrying at most the
 * largest duplicate count among strings of that length.
 */
int64_t entry_upper_bound(const tam_handle *h, const tam_vocab *v) {
    const int64_t L = v->max_tok_len;
    std::vector<int64_t> dup(L + 1, 0);
    for (const SlotPay &s : v->pay) {
        if (s.first < 0) continue;
        dup[(size_t)s.len] = std::max<int64_t>(dup[(size_t)s.len], s.count);
    }
    std::vector<int64_t> cum(L + 1, 0);
    for (int64_t d = 1; d <= L; ++d) cum[(size_t)d] = cum[(size_t)d - 1] + dup[(size_t)d];
    // A hit at distance d above node m lands in a list iff d <= the node's list
    // span; with tail compression only the hits longer than the probe window do
    // (the shorter ones are read straight from the probe's hits).
    const bool split = !h->tail_span.empty();
    int64_t bound = 0;
    for (int64_t m = 0; m < h->N; ++m) {
        const int64_t span = std::min<int64_t>(split ? h->tail_span[(size_t)m] : h->depth[(size_t)m], L);
        bound += cum[(size_t)span] - (split ? cum[(size_t)std::min<int64_t>(span, kWin)] : 0);
    }
    return bound;
}

/*
 * Tail compression.  A node is a tail when its subtree holds exactly one final
 * node, i.e. below it the trie is a single path; its valid tokens are then the
 * tokens equal to a prefix of that one remaining suffix.  Every other node
 * (two or more finals below) is a branching node and gets a dense table row,
 * numbered in id order; a tail a gets row_of[a] = -1 - rem(a), rem(a) being the
 * number of nodes below it.  In preorder a tail's path has consecutive ids
 * a+1 .. a+rem(a), so the token of length d starting below a is the suffix hit
 * of node a+d at distance d: tails need no stored masks.  Tails are closed
 * under descent, so above any node m the tails form the first tail_span[m]
 * ancestors: a hit at distance d above m lands on a tail iff d <= tail_span[m]
 * = depth(m) - depth(highest tail ancestor-or-self of m), and 0 when m itself
 * branches.  Every parent precedes its children: one backward pass counts the
 * finals below each node (and the path lengths below tails), one forward pass
 * finds the highest tail on each path.
 */
void split_tails(tam_handle *h) {
    const int64_t N = h->N;
    std::vector<int32_t> finals(h->is_final.begin(), h->is_final.end());
    for (int64_t n = N - 1; n > 0; --n) {
        const int32_t p = h->parent[(size_t)n];
        if (p >= 0) finals[(size_t)p] += finals[(size_t)n];
    }
    std::vector<int32_t> rem((size_t)N, 0);  // nodes below a tail (its single child is n+1)
    for (int64_t n = N - 1; n >= 0; --n)
        if (finals[(size_t)n] == 1 && !h->is_final[(size_t)n]) rem[(size_t)n] = rem[(size_t)n + 1] + 1;
    h->tail_span.assign((size_t)N, 0);
    h->row_of.assign((size_t)N, -1);
    std::vector<int32_t> top((size_t)N, -1);  // depth of the highest tail ancestor-or-self
    int32_t rows = 0;
    for (int64_t n = 0; n < N; ++n) {
        if (finals[(size_t)n] >= 2) {
            h->row_of[(size_t)n] = rows++;
            continue;
        }
        const int32_t p = h->parent[(size_t)n];
        top[(size_t)n] = (p >= 0 && top[(size_t)p] >= 0) ? top[(size_t)p] : h->depth[(size_t)n];
        h->tail_span[(size_t)n] = h->depth[(size_t)n] - top[(size_t)n];
        h->row_of[(size_t)n] = -1 - rem[(size_t)n];
    }
    h->dense_rows = rows;
    h->row_at.resize(h->node_at.size());
    for (size_t p = 0; p < h->node_at.size(); ++p) h->row_at[p] = h->row_of[(size_t)h->node_at[p]];
}

}  // namespace tam
