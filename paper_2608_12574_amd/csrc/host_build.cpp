// Host part of tam_compile: the trie of every set (Section 4.1) and the
// vocabulary tables used by the device validity kernels.
#include <algorithm>
#include <cstring>
#include <numeric>

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

}  // namespace

/*
 * Trie construction (Section 4.1: insert every value one byte at a time, shared
 * prefixes merge).  Inserting the distinct terminated strings in sorted order
 * creates the new nodes of each string right after its longest common prefix
 * with the previous string, and that creation order is exactly the
 * lexicographic preorder the interface fixes.  O(N_chars) after the sort.
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
    h->roots.assign((size_t)S, 0);
    h->parent.clear();
    h->depth.clear();
    h->edge.clear();
    h->is_final.clear();
    h->node_pos.clear();
    h->blob.clear();
    h->node_at.clear();
    h->K_unique = 0;

    int64_t reserve_nodes = total + 2 * K + S;
    h->parent.reserve((size_t)reserve_nodes);
    h->depth.reserve((size_t)reserve_nodes);
    h->edge.reserve((size_t)reserve_nodes);
    h->is_final.reserve((size_t)reserve_nodes);
    h->node_pos.reserve((size_t)reserve_nodes);
    h->blob.reserve((size_t)(total + 2 * K + 2 * kBlobPad));
    h->node_at.reserve((size_t)(total + 2 * K + 2 * kBlobPad));
    // zero pad in front, so that a node's 16-byte path window never starts before the blob
    h->blob.assign((size_t)kBlobPad, 0);
    h->node_at.assign((size_t)kBlobPad, 0);

    std::vector<int64_t> order;
    std::vector<int32_t> path;
    int64_t N = 0;
    for (int64_t j = 0; j < S; ++j) {
        const int64_t k0 = set_off[j], k1 = set_off[j + 1];
        order.resize((size_t)(k1 - k0));
        std::iota(order.begin(), order.end(), k0);
        std::sort(order.begin(), order.end(), TerminatedLess{sb, so, term});

        const int32_t root = (int32_t)N++;
        h->roots[(size_t)j] = root;
        h->parent.push_back(-1);
        h->depth.push_back(0);
        h->edge.push_back(0);
        h->is_final.push_back(0);
        h->node_pos.push_back(-1);

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
            ++h->K_unique;
            if ((int64_t)path.size() < len + 1) path.resize((size_t)(len + 1));
            // blob segment: one pad byte standing for the root, the string, T
            h->blob.push_back(0);
            h->node_at.push_back(root);
            for (int64_t i = 0; i <= len; ++i) {
                const uint8_t c = i < len ? s[i] : term;
                h->blob.push_back(c);
                int32_t id;
                if (i < l) {
                    id = path[(size_t)i];
                } else {
                    id = (int32_t)N++;
                    h->parent.push_back(i == 0 ? root : path[(size_t)(i - 1)]);
                    h->depth.push_back((int32_t)(i + 1));
                    h->edge.push_back(c);
                    h->is_final.push_back(i == len ? 1 : 0);
                    h->node_pos.push_back((int32_t)(h->blob.size() - 1));
                }
                path[(size_t)i] = id;
                h->node_at.push_back(id);
            }
            if (N >= INT32_MAX || (int64_t)h->blob.size() >= INT32_MAX) {
                *err = "trie exceeds 2^31-1 nodes or string bytes";
                return TAM_E_TOOLARGE;
            }
        }
    }
    // zero pad behind, so that aligned window loads stay inside the blob
    h->blob.insert(h->blob.end(), (size_t)kBlobPad, 0);
    h->node_at.insert(h->node_at.end(), (size_t)kBlobPad, 0);
    h->N = N;
    h->S = S;
    h->blob_bytes = (int64_t)h->blob.size();

    // children of every node, ascending bytes = ascending ids (preorder)
    h->child_off.assign((size_t)(N + 1), 0);
    for (int64_t m = 0; m < N; ++m)
        if (h->parent[(size_t)m] >= 0) ++h->child_off[(size_t)h->parent[(size_t)m] + 1];
    for (int64_t n = 0; n < N; ++n) h->child_off[(size_t)n + 1] += h->child_off[(size_t)n];
    const int64_t E = h->child_off[(size_t)N];
    h->child_node.assign((size_t)std::max<int64_t>(E, 1), 0);
    h->child_byte.assign((size_t)std::max<int64_t>(E, 1), 0);
    std::vector<int32_t> fill(h->child_off.begin(), h->child_off.end() - 1);
    for (int64_t m = 0; m < N; ++m) {
        const int32_t p = h->parent[(size_t)m];
        if (p < 0) continue;
        const int32_t at = fill[(size_t)p]++;
        h->child_node[(size_t)at] = (int32_t)m;
        h->child_byte[(size_t)at] = h->edge[(size_t)m];
    }
    return TAM_OK;
}

/*
 * Vocabulary tables (the paper's vocabulary decoding and its per-tokenizer
 * matcher, built here as an exact hash of every distinct token string keyed by
 * its bytes read last-to-first).  Slots live in buckets of kBucket 32-bit
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
    if (h->tok_blob.empty()) h->tok_blob.push_back(0);
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
    h->fps.assign(cap, 0u);
    h->srev.assign(cap, SlotRev{0, 0});
    h->smeta.assign(cap, SlotMeta{-1, 0, 0});
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
        const uint32_t fp = fingerprint(key);
        uint64_t b = (key & (cap - 1)) / kBucket;
        bool placed = false;
        while (!placed) {
            for (int i = 0; i < kBucket && !placed; ++i) {
                const uint64_t s = b * kBucket + (uint64_t)i;
                if (h->fps[s] == 0) {
                    h->fps[s] = fp;
                    SlotRev r{0, 0};
                    for (uint32_t k = 0; k < len && k < 16; ++k) {
                        const uint64_t c = blob[off + len - 1 - k];
                        if (k < 8)
                            r.lo |= c << (8 * k);
                        else
                            r.hi |= c << (8 * (k - 8));
                    }
                    h->srev[s] = r;
                    h->smeta[s] = SlotMeta{(int32_t)v, (uint16_t)len, 1};
                    last[s] = (int32_t)v;
                    placed = true;
                } else if (h->fps[s] == fp && h->smeta[s].len == len) {
                    const uint32_t o2 = h->tok_off[(size_t)h->smeta[s].first];
                    if (std::memcmp(blob + o2, blob + off, len) == 0) {
                        if (h->smeta[s].count == 65535) {
                            *err = "more than 65535 tokens share one byte string";
                            return TAM_E_TOOLARGE;
                        }
                        h->dup_next[(size_t)last[s]] = (int32_t)v;
                        last[s] = (int32_t)v;
                        ++h->smeta[s].count;
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
    for (const SlotMeta &s : v->smeta) {
        if (s.first < 0) continue;
        dup[(size_t)s.len] = std::max<int64_t>(dup[(size_t)s.len], s.count);
    }
    std::vector<int64_t> cum(L + 1, 0);
    for (int64_t d = 1; d <= L; ++d) cum[(size_t)d] = cum[(size_t)d - 1] + dup[(size_t)d];
    int64_t bound = 0;
    for (int64_t m = 0; m < h->N; ++m) bound += cum[(size_t)std::min<int64_t>(h->depth[(size_t)m], L)];
    return bound;
}

}  // namespace tam
