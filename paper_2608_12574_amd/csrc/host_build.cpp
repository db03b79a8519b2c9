// Host part of tam_compile: the trie of every set (Section 4.1) and the
// vocabulary tables used by the device validity kernels.
#include <algorithm>
#include <atomic>
#include <cstring>
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

// The sorted, distinct strings of one part (all of one set, or all of a set
// with the same first byte of s+T), planned before any node is written: each
// string's longest common prefix with the previous one fixes how many nodes
// it creates, so every part's node, edge and blob ranges are known up front
// and the parts then write straight into the handle's tables.
struct PartPlan {
    std::vector<int64_t> str;   // string indices in trie order, duplicates dropped
    std::vector<int32_t> lcp;   // common prefix with the previous string (0 for the first)
    std::vector<int32_t> psv;   // nearest earlier string with a shorter common prefix (-1: none)
    int64_t nodes = 1;          // including the part's root (its set's root)
    int64_t blob = 0;           // pad byte, bytes, T per string
    int64_t branching = 0;      // nodes other than the part root that two or more strings pass through
    tam_status st = TAM_OK;
    std::string err;
};

// The first 8 bytes of s+T, big-endian and zero-padded: terminated strings are
// prefix-free (T occurs only at their end), so two of them with different keys
// are ordered by their keys, and equal keys leave the order to the full compare.
uint64_t order_key(const uint8_t *s, int64_t len, uint8_t term) {
    uint64_t k = 0;
    for (int i = 0; i < 8; ++i) {
        const uint64_t c = i < len ? s[i] : (i == len ? term : 0);
        k = (k << 8) | c;
    }
    return k;
}

/*
 * Trie construction (Section 4.1: insert every value one byte at a time,
 * shared prefixes merge), planned: inserting the distinct terminated strings
 * in sorted order creates the new nodes of each string right after its longest
 * common prefix with the previous string, and that creation order is exactly
 * the lexicographic preorder the interface fixes.  A string of length len
 * with common prefix l creates len + 1 - l nodes.  O(N_chars) after the sort.
 */
void plan_part(const uint8_t *sb, const int64_t *so, const int64_t *idx, int64_t count, uint8_t term,
               PartPlan &r) {
    std::vector<std::pair<uint64_t, int64_t>> order((size_t)count);
    for (int64_t i = 0; i < count; ++i) {
        const int64_t k = idx[i];
        order[(size_t)i] = {order_key(sb + so[k], so[k + 1] - so[k], term), k};
    }
    const TerminatedLess less{sb, so, term};
    std::sort(order.begin(), order.end(), [&](const std::pair<uint64_t, int64_t> &a,
                                              const std::pair<uint64_t, int64_t> &b) {
        return a.first != b.first ? a.first < b.first : less(a.second, b.second);
    });
    r.str.reserve((size_t)count);
    r.lcp.reserve((size_t)count);
    const uint8_t *prev = nullptr;
    int64_t prev_len = -1;
    for (const auto &kv : order) {
        const int64_t k = kv.second;
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
        r.str.push_back(k);
        r.lcp.push_back((int32_t)l);
        r.nodes += len + 1 - l;
        r.blob += len + 2;
        if (r.nodes >= INT32_MAX || r.blob >= INT32_MAX) {
            r.st = TAM_E_TOOLARGE;
            r.err = "trie exceeds 2^31-1 nodes or string bytes";
            return;
        }
    }
    // string u creates the nodes at path indices lcp[u] .. len; the next string
    // also passes through those below index lcp[u+1] (sorted order: no later
    // string shares more of them)
    for (size_t u = 0; u < r.lcp.size(); ++u) {
        const int64_t next = u + 1 < r.lcp.size() ? r.lcp[u + 1] : 0;
        r.branching += std::max<int64_t>(0, next - r.lcp[u]);
    }
    // previous strictly smaller common prefix (a stack of increasing lcp)
    r.psv.resize(r.lcp.size());
    std::vector<int32_t> stack;
    for (size_t u = 0; u < r.lcp.size(); ++u) {
        while (!stack.empty() && r.lcp[(size_t)stack.back()] >= r.lcp[u]) stack.pop_back();
        r.psv[u] = stack.empty() ? -1 : stack.back();
        stack.push_back((int32_t)u);
    }
}

// Where a part's nodes and blob bytes go in the handle's tables.
struct PartBase {
    int32_t root;         // its set's root
    int64_t node;         // local node i >= 1 gets id node + i
    int64_t blob;         // local blob offset b goes to blob + b
    bool root_tail;       // its set has one string (the set root is then a tail)
    int64_t str0;         // blob-order index of its first string
    int64_t first_row;    // (tail split) dense row of the part's first branching node
};

/*
 * Writes a planned part into the handle: per string, a pad byte (standing for
 * the root), its bytes and T into the blob, and its record (StrRec); the nodes
 * it creates (parent, depth, edge byte, final flag); and with subtree extents,
 * the end of every node's subtree (a node's subtree ends where the first later
 * string leaves its path).  node_at, the device's depth, node positions and
 * child lists are derived on the device from the blob and the records.
 *
 * Tail split, decided when a node is created: string u creates the nodes at
 * path indices i >= lcp[u], and the next string passes through those with
 * i < lcp[u+1] (no later string shares more of them).  Those are branching
 * nodes and take the next dense rows, in creation order, which is id order.
 * The others are tails: only string u passes through them, so len - i nodes
 * lie below one, and the highest tail on the path is at index
 * max(lcp[u], lcp[u+1]) (the root itself in a set of one string).
 */
void emit_part(const uint8_t *sb, const int64_t *so, uint8_t term, const PartPlan &r, PartBase &pb,
               bool subtrees, bool tails, tam_handle *h) {
    const int64_t nstr = (int64_t)r.str.size();
    // tail_span and row_at are written here only for a host-only handle;
    // otherwise the device lays them out from the records (row_of, which the
    // host API reports, is written in both cases)
    const bool host_tables = tails && !h->tail_span.empty();
    std::vector<int32_t> path;  // global ids of the current string's nodes by depth - 1
    int64_t N = 1, B = 0, prev_len = -1;
    int32_t row = (int32_t)pb.first_row;
    // the previous string's nodes at path indices l..prev_len leave the path
    // before the next string: their subtrees end here
    auto close = [&](int64_t l) {
        if (subtrees)
            for (int64_t i = l; i <= prev_len; ++i) h->sub_end[(size_t)path[(size_t)i]] = (int32_t)(pb.node + N);
    };
    for (int64_t u = 0; u < nstr; ++u) {
        const int64_t k = r.str[(size_t)u];
        const uint8_t *s = sb + so[k];
        const int64_t len = so[k + 1] - so[k];
        const int64_t l = r.lcp[(size_t)u];
        const int64_t next = u + 1 < nstr ? r.lcp[(size_t)u + 1] : 0;
        const int64_t top = pb.root_tail ? -1 : std::max(l, next);  // index above the highest tail
        close(l);
        prev_len = len;
        if ((int64_t)path.size() < len + 1) path.resize((size_t)(len + 1));
        const int64_t at = pb.blob + B;
        const int32_t psv = r.psv[(size_t)u];
        h->strs[(size_t)(pb.str0 + u)] = StrRec{(int32_t)at, (int32_t)len, (int32_t)l, (int32_t)(pb.node + N),
                                                psv < 0 ? -1 : (int32_t)(pb.str0 + psv), pb.root};
        h->blob[(size_t)at] = 0;
        if (tails) h->tail_rec[(size_t)(pb.str0 + u)] = TailRec{row, (int32_t)next, (int32_t)top};
        if (host_tables) h->row_at[(size_t)at] = h->row_of[(size_t)pb.root];
        for (int64_t i = 0; i <= len; ++i) {
            const uint8_t c = i < len ? s[i] : term;
            const size_t pos = (size_t)(at + 1 + i);
            h->blob[pos] = c;
            if (i >= l) {
                const size_t g = (size_t)(pb.node + N++);
                h->parent[g] = (int32_t)(i == 0 ? pb.root : path[(size_t)(i - 1)]);
                h->depth[g] = (int32_t)(i + 1);
                h->edge[g] = c;
                h->is_final[g] = i == len ? 1 : 0;
                path[(size_t)i] = (int32_t)g;
                if (tails) {
                    const bool branching = i < next;
                    h->row_of[g] = branching ? row : (int32_t)(-1 - (len - i));
                    if (host_tables) h->tail_span[g] = branching ? 0 : (int32_t)(i - top);
                    if (branching) ++row;
                }
            }
            if (host_tables) h->row_at[pos] = h->row_of[(size_t)path[(size_t)i]];
        }
        B += len + 2;
    }
    close(0);
}

// Runs f(j) for j in [0, n) on up to `threads` host threads.
template <typename F>
void parallel_for(int64_t n, int threads, F f) {
    if (threads <= 1 || n <= 1) {
        for (int64_t j = 0; j < n; ++j) f(j);
        return;
    }
    host_parallel_for(n, threads, std::function<void(int64_t)>(f));
}

int host_threads(int64_t work_items) {
    const unsigned hw = std::max(1u, std::thread::hardware_concurrency());
    return (int)std::min<int64_t>({(int64_t)hw, (int64_t)16, work_items});
}

/*
 * Tail compression.  A node is a tail when its subtree holds exactly one final
 * node, i.e. below it the trie is a single path; its valid tokens are then the
 * tokens equal to a prefix of that one remaining suffix.  Every other node
 * (two or more finals below) is a branching node and gets a dense table row,
 * numbered in id order (a set's root, then its parts' nodes); a tail a gets
 * row_of[a] = -1 - rem(a), rem(a) being the number of nodes below it.  In
 * preorder a tail's path has consecutive ids a+1 .. a+rem(a), so the token of
 * length d starting below a is the suffix hit of node a+d at distance d: tails
 * need no stored masks.  Tails are closed under descent, so above any node m
 * the tails form the first tail_span[m] ancestors: a hit at distance d above m
 * lands on a tail iff d <= tail_span[m] = depth(m) - depth(highest tail
 * ancestor-or-self of m), and 0 when m itself branches.  row_at =
 * row_of[node_at] is laid along the blob.  emit_part classifies the nodes as it
 * creates them; the set roots and the first row of every part are fixed
 * before, from the planned branching counts.
 */

}  // namespace

/*
 * Tries of all sets.  A set's trie is its root plus one subtrie per distinct
 * first byte of s+T, and in preorder those subtries follow one another in byte
 * order.  The unit of host work is a part: a whole set, or (for a large set)
 * the strings of one first byte.  The parts are planned in parallel over host
 * threads (sorted, their sizes counted), laid out one after another with the
 * part roots merged into their set's root, and then written in parallel
 * straight into the handle's tables.  Set j takes node ids
 * [roots[j], roots[j] + N_j) and its own range of the blob, which carries
 * kBlobPad zero bytes in front and behind so that 16-byte window loads around
 * any node never leave it.  Every node but a root has one parent edge, so
 * the child lists (built on the device) hold N - S entries.
 */
tam_status build_trie(const uint8_t *sb, const int64_t *so, int64_t K, const int64_t *set_off,
                      int64_t S, int T, tam_handle *h, std::string *err,
                      const std::function<tam_status(tam_handle *)> &planned,
                      const std::function<tam_status(tam_handle *, const TrieRange &)> &emitted) {
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
    // parts: a set whole, or a large set cut by the first byte of s+T (its
    // strings grouped by that byte, in byte order)
    const int threads = host_threads(K);
    const int64_t split_at = std::max<int64_t>(1024, K / (2 * (int64_t)threads));
    std::vector<int64_t> idx((size_t)K);
    std::vector<int64_t> pstart;  // part p holds idx[pstart[p] .. pstart[p+1])
    std::vector<int64_t> pset;    // set of part p
    std::vector<int64_t> set_first((size_t)S + 1, 0);  // first part of each set
    {
        std::vector<int64_t> cnt(256), pos(256);
        for (int64_t j = 0; j < S; ++j) {
            set_first[(size_t)j] = (int64_t)pset.size();
            const int64_t k0 = set_off[j], k1 = set_off[j + 1];
            if (k1 - k0 < split_at) {
                for (int64_t k = k0; k < k1; ++k) idx[(size_t)k] = k;
                pstart.push_back(k0);
                pset.push_back(j);
                continue;
            }
            std::fill(cnt.begin(), cnt.end(), 0);
            for (int64_t k = k0; k < k1; ++k) ++cnt[so[k + 1] > so[k] ? sb[so[k]] : term];
            int64_t at = k0;
            for (int c = 0; c < 256; ++c) {
                pos[(size_t)c] = at;
                if (cnt[(size_t)c]) {
                    pstart.push_back(at);
                    pset.push_back(j);
                }
                at += cnt[(size_t)c];
            }
            for (int64_t k = k0; k < k1; ++k) idx[(size_t)pos[so[k + 1] > so[k] ? sb[so[k]] : term]++] = k;
        }
        set_first[(size_t)S] = (int64_t)pset.size();
        pstart.push_back(K);
    }
    const int64_t NP = (int64_t)pset.size();
    std::vector<PartPlan> parts((size_t)NP);
    std::atomic<bool> oom{false};
    parallel_for(NP, host_threads(NP), [&](int64_t p) {
        try {
            plan_part(sb, so, idx.data() + pstart[(size_t)p], pstart[(size_t)p + 1] - pstart[(size_t)p], term,
                      parts[(size_t)p]);
        } catch (const std::bad_alloc &) {
            oom = true;
        }
    });
    if (oom) throw std::bad_alloc();
    // bases: node ids (a part's local root is its set's root, the rest follow)
    // and blob offsets
    std::vector<PartBase> base((size_t)NP);
    std::vector<int64_t> root((size_t)S), set_blob((size_t)S), set_str((size_t)S);
    std::vector<int32_t> root_row((size_t)S);  // (tail split) row_of of each set root
    int64_t N = 0, BB = kBlobPad, E = 0, rows = 0;
    h->K_unique = 0;
    for (int64_t j = 0; j < S; ++j) {
        root[(size_t)j] = N++;
        set_blob[(size_t)j] = BB;
        set_str[(size_t)j] = h->K_unique;
        for (int64_t p = set_first[(size_t)j]; p < set_first[(size_t)j + 1]; ++p) {
            const PartPlan &r = parts[(size_t)p];
            if (r.st != TAM_OK) {
                *err = r.err;
                return r.st;
            }
        }
        int64_t set_strings = 0;
        for (int64_t p = set_first[(size_t)j]; p < set_first[(size_t)j + 1]; ++p)
            set_strings += (int64_t)parts[(size_t)p].str.size();
        // a set of one string: the whole path lies below its root, a tail;
        // any other set root branches and takes the set's first dense row
        const int64_t p0 = set_first[(size_t)j];
        root_row[(size_t)j] = set_strings == 1 ? (int32_t)(-1 - (parts[(size_t)p0].nodes - 1)) : (int32_t)rows++;
        for (int64_t p = set_first[(size_t)j]; p < set_first[(size_t)j + 1]; ++p) {
            const PartPlan &r = parts[(size_t)p];
            PartBase &pb = base[(size_t)p];
            pb.root_tail = set_strings == 1;
            pb.first_row = rows;
            rows += r.branching;
            pb.root = (int32_t)root[(size_t)j];
            pb.node = N - 1;
            pb.blob = BB;
            pb.str0 = h->K_unique;
            N += r.nodes - 1;
            BB += r.blob;
            E += r.nodes - 1;  // every node but a root has one parent
            h->K_unique += (int64_t)r.str.size();
            if (N >= INT32_MAX || BB >= INT32_MAX || h->K_unique >= INT32_MAX) {
                *err = "trie exceeds 2^31-1 nodes, strings or string bytes";
                return TAM_E_TOOLARGE;
            }
        }
    }
    BB += kBlobPad;
    if (BB >= INT32_MAX) {
        *err = "trie exceeds 2^31-1 nodes or string bytes";
        return TAM_E_TOOLARGE;
    }
    h->N = N;
    h->S = S;
    h->blob_bytes = BB;
    h->edges = E;
    if (planned) {  // sizes known, nothing emitted yet
        const tam_status st = planned(h);
        if (st != TAM_OK) return st;
    }
    h->roots.resize((size_t)S);
    h->parent.resize((size_t)N);
    h->depth.resize((size_t)N);
    h->edge.resize((size_t)N);
    h->is_final.resize((size_t)N);
    h->blob.resize((size_t)BB);  // the parts fill all but the outer pads
    h->strs.resize((size_t)h->K_unique);
    const bool subtrees = (h->flags & TAM_FLAG_LAZY_ROWS) != 0;
    const bool tails = (h->flags & TAM_FLAG_TAIL_LISTS) && !(h->flags & TAM_FLAG_LAZY_ROWS);
    const bool host_tables = tails && (h->flags & TAM_FLAG_HOST_ONLY);  // else laid out on the device
    h->tails = tails;
    h->sub_end.resize(subtrees ? (size_t)N : 0);
    h->row_of.resize(tails ? (size_t)N : 0);
    h->tail_span.resize(host_tables ? (size_t)N : 0);
    h->row_at.resize(host_tables ? (size_t)BB : 0);
    h->tail_rec.resize(tails ? (size_t)h->K_unique : 0);
    h->root_rows.assign(tails ? (size_t)(2 * S) : 0, 0);
    h->dense_rows = tails ? rows : 0;
    for (int64_t p = 0; p < kBlobPad; ++p) {
        h->blob[(size_t)p] = h->blob[(size_t)(BB - 1 - p)] = 0;
    }
    for (int64_t j = 0; j < S; ++j) {
        const int64_t rt = root[(size_t)j];
        h->roots[(size_t)j] = (int32_t)rt;
        h->parent[(size_t)rt] = -1;
        h->depth[(size_t)rt] = 0;
        h->edge[(size_t)rt] = 0;
        h->is_final[(size_t)rt] = 0;
        if (subtrees) h->sub_end[(size_t)rt] = (int32_t)(j + 1 < S ? root[(size_t)j + 1] : N);
        if (tails) {
            h->root_rows[(size_t)(2 * j)] = (int32_t)rt;
            h->root_rows[(size_t)(2 * j + 1)] = root_row[(size_t)j];
        }
        if (tails) h->row_of[(size_t)rt] = root_row[(size_t)j];
        if (host_tables) h->tail_span[(size_t)rt] = 0;
    }
    if (host_tables)
        for (int64_t p = 0; p < kBlobPad; ++p)  // the outer pads stand for the first set's root
            h->row_at[(size_t)p] = h->row_at[(size_t)(BB - 1 - p)] = h->row_of[0];
    // Emission in groups of whole sets (a forest of many sets: four groups, so
    // that a caller can upload a group while the next is written).
    const int64_t groups = emitted && S >= 8 ? kMaxRecGroups : 1;
    for (int64_t g = 0; g < groups; ++g) {
        const int64_t j0 = S * g / groups, j1 = S * (g + 1) / groups;
        const int64_t p0 = set_first[(size_t)j0], p1 = set_first[(size_t)j1];
        parallel_for(p1 - p0, host_threads(p1 - p0), [&](int64_t i) {
            try {
                emit_part(sb, so, term, parts[(size_t)(p0 + i)], base[(size_t)(p0 + i)], subtrees, tails, h);
            } catch (const std::bad_alloc &) {
                oom = true;
            }
        });
        if (oom) throw std::bad_alloc();
        if (emitted) {
            const TrieRange r{root[(size_t)j0], j1 < S ? root[(size_t)j1] : N,
                              g == 0 ? 0 : set_blob[(size_t)j0], j1 < S ? set_blob[(size_t)j1] : BB,
                              set_str[(size_t)j0], j1 < S ? set_str[(size_t)j1] : h->K_unique};
            const tam_status st = emitted(h, r);
            if (st != TAM_OK) return st;
        }
    }
    return TAM_OK;
}

/*
 * Vocabulary tables (the paper's vocabulary decoding and its per-tokenizer
 * matcher, built here as an exact hash of every distinct token string keyed by
 * its bytes read last-to-first).  Slots live in buckets of kBucket 12-bit
 * fingerprints; a key starts at its home bucket and moves to the next bucket
 * only when the bucket is full.  Duplicate strings share a slot and chain their
 * ids in ascending order.  Once placed, the strings are numbered bucket by
 * bucket and the payloads stored by that number (see device_tables.hpp).
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
    h->tok_blob.resize((size_t)total + kBlobPad);  // zero pad: room for 16-byte window loads
    if (total > 0) std::memcpy(h->tok_blob.data(), tb + to[0], (size_t)total);
    std::memset(h->tok_blob.data() + total, 0, (size_t)kBlobPad);
    const int64_t chunk = 1 << 14, nchunks = (V + chunk - 1) / chunk;
    std::vector<int64_t> cmax((size_t)nchunks, 0);
    parallel_for(nchunks, host_threads(nchunks), [&](int64_t c) {
        int64_t m = 0;
        for (int64_t v = c * chunk; v < std::min(V, (c + 1) * chunk); ++v) {
            h->tok_off[(size_t)v] = (uint32_t)(to[v] - to[0]);
            m = std::max<int64_t>(m, to[v + 1] - to[v]);
        }
        cmax[(size_t)c] = m;
    });
    h->tok_off[(size_t)V] = (uint32_t)(to[V] - to[0]);
    int64_t max_len = 0;
    for (int64_t m : cmax) max_len = std::max(max_len, m);
    if (max_len > 65535) {
        *err = "a token is longer than 65535 bytes";
        return TAM_E_TOOLARGE;
    }
    h->max_tok_len = max_len;
    h->len_present.assign((size_t)(max_len + 1), 0);
    h->len_mask = 0;

    // load <= 1/4 (at most 2 keys per 8-slot bucket on average): a full home
    // bucket, which sends a probe down the slower general path, stays rare
    uint64_t cap = 64;
    while (cap < (uint64_t)(4 * V)) cap <<= 1;
    const uint64_t nbuckets = cap / kBucket;
    // the tables are first touched, and set empty, in parallel
    h->fps.resize(cap);
    h->pay.resize(cap);
    h->pay_hi.resize(cap);
    h->dup_next.resize((size_t)V);
    hvec<int32_t> last(cap);
    const SlotPay empty{0, -1, 0, 0};
    const int64_t pchunk = 1 << 15, npchunks = ((int64_t)cap + pchunk - 1) / pchunk;
    parallel_for(npchunks, host_threads(npchunks), [&](int64_t c) {
        for (int64_t q = c * pchunk; q < std::min<int64_t>((int64_t)cap, (c + 1) * pchunk); ++q) {
            h->fps[(size_t)q] = 0;
            h->pay[(size_t)q] = empty;
            h->pay_hi[(size_t)q] = 0;
            last[(size_t)q] = -1;
        }
    });
    const uint8_t *blob = h->tok_blob.data();
    // keys, reversed heads and home buckets of all tokens, in parallel
    hvec<uint64_t> keys((size_t)V), heads((size_t)V * 2), home((size_t)V);
    parallel_for(nchunks, host_threads(nchunks), [&](int64_t c) {
        for (int64_t v = c * chunk; v < std::min(V, (c + 1) * chunk); ++v) {
            const uint32_t off = h->tok_off[(size_t)v];
            const uint32_t len = h->tok_off[(size_t)v + 1] - off;
            uint32_t hh = kHashSeed;
            uint64_t lo = 0, hi = 0;
            for (int64_t i = (int64_t)len - 1; i >= 0; --i) hh = hash_step(hh, blob[off + i]);
            for (uint32_t k = 0; k < len && k < 16; ++k) {
                const uint64_t ch = blob[off + len - 1 - k];
                if (k < 8)
                    lo |= ch << (8 * k);
                else
                    hi |= ch << (8 * (k - 8));
            }
            keys[(size_t)v] = len ? hash_final(hh) : 0;
            heads[(size_t)(2 * v)] = lo;
            heads[(size_t)(2 * v + 1)] = hi;
            home[(size_t)v] = (keys[(size_t)v] & (cap - 1)) / kBucket;
            h->dup_next[(size_t)v] = -1;
        }
    });
    for (int64_t v = 0; v < V; ++v) {
        const uint32_t len = h->tok_off[(size_t)v + 1] - h->tok_off[(size_t)v];
        if (len == 0) continue;
        h->len_present[len] = 1;
        if (len < 64) h->len_mask |= 1ull << len;
    }
    // Placement: token v goes to the first slot, from its home bucket on, that
    // is empty or holds its string (a duplicate joins that slot's id chain, in
    // ascending id order).  The buckets are cut into ranges placed in parallel,
    // each taking the tokens whose home bucket it holds, in id order.  A token
    // that would have to move past its range's last bucket is deferred to a
    // serial pass, in id order, over the filled table; a key therefore still
    // sits in a later bucket only if every bucket from its home to there was
    // full when it was placed, which is what the device probe relies on.
    std::atomic<bool> too_many{false};
    // place(v, b, stop, wrap): from bucket b on; with wrap, through the whole
    // table (wrapping at its end), else only up to bucket stop (exclusive).
    // False if not placed.
    auto place = [&](int64_t v, uint64_t b, uint64_t stop, bool wrap) -> bool {
        const uint32_t off = h->tok_off[(size_t)v];
        const uint32_t len = h->tok_off[(size_t)v + 1] - off;
        const uint16_t fp = (uint16_t)fingerprint(keys[(size_t)v]);  // 12 bits, never 0
        for (uint64_t n = 0; n < nbuckets; ++n) {
            for (int i = 0; i < kBucket; ++i) {
                const uint64_t sl = b * kBucket + (uint64_t)i;
                if (h->fps[sl] == 0) {
                    h->fps[sl] = fp;
                    h->pay[sl] = SlotPay{heads[(size_t)(2 * v)], (int32_t)v, (uint16_t)len, 1};
                    h->pay_hi[sl] = heads[(size_t)(2 * v + 1)];
                    last[sl] = (int32_t)v;
                    return true;
                }
                if (h->fps[sl] == fp && h->pay[sl].len == len &&
                    std::memcmp(blob + h->tok_off[(size_t)h->pay[sl].first], blob + off, len) == 0) {
                    if (h->pay[sl].count == 65535) {
                        too_many = true;
                        return true;
                    }
                    h->dup_next[(size_t)last[sl]] = (int32_t)v;
                    last[sl] = (int32_t)v;
                    ++h->pay[sl].count;
                    return true;
                }
            }
            if (!wrap && b + 1 >= stop) return false;
            b = b + 1 == nbuckets ? 0 : b + 1;
        }
        return false;  // not reached: the table is at most half full
    };
    const int64_t R = std::min<int64_t>(256, (int64_t)nbuckets);  // bucket ranges
    auto range_of = [&](uint64_t b) { return (int64_t)(b * (uint64_t)R / nbuckets); };
    auto range_start = [&](int64_t r) { return ((uint64_t)r * nbuckets + (uint64_t)R - 1) / (uint64_t)R; };
    // the non-empty tokens grouped by range, in id order: per-chunk counts, then
    // each chunk scatters its tokens after those of the chunks before it
    std::vector<int64_t> ccount((size_t)(nchunks * R), 0);
    parallel_for(nchunks, host_threads(nchunks), [&](int64_t c) {
        int64_t *cnt = ccount.data() + c * R;
        for (int64_t v = c * chunk; v < std::min(V, (c + 1) * chunk); ++v)
            if (h->tok_off[(size_t)v + 1] > h->tok_off[(size_t)v]) ++cnt[range_of(home[(size_t)v])];
    });
    std::vector<int64_t> rcount((size_t)R + 1, 0);
    for (int64_t r = 0; r < R; ++r) {
        int64_t at = rcount[(size_t)r];
        for (int64_t c = 0; c < nchunks; ++c) {
            const int64_t n = ccount[(size_t)(c * R + r)];
            ccount[(size_t)(c * R + r)] = at;
            at += n;
        }
        rcount[(size_t)r + 1] = at;
    }
    hvec<int32_t> order((size_t)rcount[(size_t)R]);
    parallel_for(nchunks, host_threads(nchunks), [&](int64_t c) {
        int64_t *at = ccount.data() + c * R;
        for (int64_t v = c * chunk; v < std::min(V, (c + 1) * chunk); ++v)
            if (h->tok_off[(size_t)v + 1] > h->tok_off[(size_t)v]) order[(size_t)at[range_of(home[(size_t)v])]++] = (int32_t)v;
    });
    std::vector<std::vector<int32_t>> deferred((size_t)R);
    parallel_for(R, host_threads(R), [&](int64_t r) {
        const uint64_t stop = r + 1 < R ? range_start(r + 1) : nbuckets;
        for (int64_t k = rcount[(size_t)r]; k < rcount[(size_t)r + 1]; ++k) {
            const int32_t v = order[(size_t)k];
            if (!place(v, home[(size_t)v], stop, false)) deferred[(size_t)r].push_back(v);
        }
    });
    std::vector<int32_t> rest;
    for (const auto &d : deferred) rest.insert(rest.end(), d.begin(), d.end());
    std::sort(rest.begin(), rest.end());
    for (int32_t v : rest) place(v, home[(size_t)v], nbuckets, true);
    if (too_many) {
        *err = "more than 65535 tokens share one byte string";
        return TAM_E_TOOLARGE;
    }
    // The strings numbered bucket by bucket (a bucket's used slots are its
    // first ones: slots fill in order), the payloads moved to that number, and
    // each bucket packed into four words: the 12-bit fingerprints of slots 2i
    // and 2i + 1 in bits 0..23 of word i, byte i of the bucket's base (its
    // first string's number) in bits 24..31.
    const int64_t bchunk = 1 << 14, nbchunks = ((int64_t)nbuckets + bchunk - 1) / bchunk;
    std::vector<int64_t> bsum((size_t)nbchunks + 1, 0);
    parallel_for(nbchunks, host_threads(nbchunks), [&](int64_t c) {
        int64_t n = 0;
        for (int64_t b = c * bchunk; b < std::min<int64_t>((int64_t)nbuckets, (c + 1) * bchunk); ++b)
            for (int i = 0; i < kBucket; ++i) n += h->fps[(size_t)(b * kBucket + i)] != 0;
        bsum[(size_t)c + 1] = n;
    });
    for (int64_t c = 0; c < nbchunks; ++c) bsum[(size_t)c + 1] += bsum[(size_t)c];
    const int64_t nstr = bsum[(size_t)nbchunks];
    hvec<SlotPay> pay_c((size_t)std::max<int64_t>(nstr, 1));
    hvec<uint64_t> pay_hi_c((size_t)std::max<int64_t>(nstr, 1), 0);
    hvec<uint16_t> packed(cap);  // the buckets' words, as 16-bit halves
    if (nstr == 0) pay_c[0] = empty;
    parallel_for(nbchunks, host_threads(nbchunks), [&](int64_t c) {
        int64_t at = bsum[(size_t)c];
        uint32_t *words = reinterpret_cast<uint32_t *>(packed.data());
        for (int64_t b = c * bchunk; b < std::min<int64_t>((int64_t)nbuckets, (c + 1) * bchunk); ++b) {
            const uint32_t base = (uint32_t)at;
            for (int i = 0; i < kBucket / 2; ++i) {
                const uint32_t f0 = h->fps[(size_t)(b * kBucket + 2 * i)], f1 = h->fps[(size_t)(b * kBucket + 2 * i + 1)];
                words[(size_t)(b * 4 + i)] = f0 | (f1 << 12) | (((base >> (8 * i)) & 0xffu) << 24);
            }
            for (int i = 0; i < kBucket; ++i) {
                const uint64_t sl = b * kBucket + (uint64_t)i;
                if (h->fps[sl] == 0) break;
                pay_c[(size_t)at] = h->pay[sl];
                pay_hi_c[(size_t)at] = h->pay_hi[sl];
                ++at;
            }
        }
    });
    h->fps.swap(packed);
    h->pay.swap(pay_c);
    h->pay_hi.swap(pay_hi_c);
    // the hits of every string of at most kShortLen bytes, indexed by its bytes
    h->short_hits.assign((size_t)kShortEntries, -1);
    for (int64_t q = 0; q < nstr; ++q) {
        const SlotPay &sp = h->pay[(size_t)q];
        if (sp.first < 0 || sp.len > kShortLen) continue;
        const uint8_t *tb = blob + h->tok_off[(size_t)sp.first];
        const int32_t at = short_index(sp.len, tb[sp.len - 1], sp.len == 2 ? tb[0] : 0u);
        h->short_hits[(size_t)at] = hit_of_slot((int32_t)q, sp.first, sp.count);
    }
    // per length d, the running sum over lengths <= d of the largest number of
    // token ids sharing one string of that length (for the list size bound)
    std::vector<int64_t> dup((size_t)max_len + 1, 0);
    {
        const int64_t nsc = (nstr + pchunk - 1) / pchunk;
        std::vector<std::vector<int64_t>> part((size_t)nsc);
        parallel_for(nsc, host_threads(nsc), [&](int64_t c) {
            std::vector<int64_t> &d = part[(size_t)c];
            d.assign((size_t)max_len + 1, 0);
            for (int64_t q = c * pchunk; q < std::min<int64_t>(nstr, (c + 1) * pchunk); ++q) {
                const SlotPay &sp = h->pay[(size_t)q];
                if (sp.first >= 0) d[(size_t)sp.len] = std::max<int64_t>(d[(size_t)sp.len], sp.count);
            }
        });
        for (const auto &d : part)
            for (int64_t l = 0; l <= max_len; ++l) dup[(size_t)l] = std::max(dup[(size_t)l], d[(size_t)l]);
    }
    h->dup_cum.assign((size_t)max_len + 1, 0);
    for (int64_t d = 1; d <= max_len; ++d) h->dup_cum[(size_t)d] = h->dup_cum[(size_t)d - 1] + dup[(size_t)d];
    return TAM_OK;
}

/*
 * Upper bound on the number of valid (node, token) pairs, used to size the
 * sparse lists without a device round trip: node m can end at most one distinct
 * token string of each length d <= min(depth(m), max_len), carrying at most the
 * largest duplicate count among strings of that length.
 */
// Sums of cum[min(x, cap)] over ranges of x, in constant time: cum is
// constant from x = cap on.
struct CumSums {
    std::vector<int64_t> pre;  // pre[x] = sum of cum[y] for y < x <= cap + 1
    int64_t cap, last;
    CumSums(const std::vector<int64_t> &cum, int64_t c) : pre((size_t)c + 2, 0), cap(c), last(cum[(size_t)c]) {
        for (int64_t y = 0; y <= c; ++y) pre[(size_t)y + 1] = pre[(size_t)y] + cum[(size_t)y];
    }
    int64_t below(int64_t n) const {  // sum over x in [0, n)
        if (n <= 0) return 0;
        return n <= cap + 1 ? pre[(size_t)n] : pre[(size_t)cap + 1] + (n - cap - 1) * last;
    }
    int64_t range(int64_t a, int64_t b) const { return b > a ? below(b) - below(a) : 0; }  // x in [a, b)
};

// Calls f(g0, g1, b) for consecutive pieces [g0, g1] of the nodes created by
// the strings [s0, s1) (every node but the roots, whose bound is 0), cut at
// base + multiples of `cut` (0: one piece per string), b being the pieces' share of
// the list bound: the ids of the hits at distance d above each node that land
// in lists (see entry_upper_bound).  A string creates nodes first, first + 1,
// ... at path indices lcp .. len; node i has depth i + 1, all = min(i + 1, L)
// and, with tail compression, tail span 0 (branching, i < next) or i - top.
// Per node: lists only cum[all]; tail compression with a table (tails'
// tokens longer than the window) cum[min(span, L)] - cum[min(span, L, kWin)];
// without a table cum[all] - cum[min(span, L, kWin)].  Each is a range sum.
template <typename F>
static void string_bounds(const tam_handle *h, const CumSums &cl, const CumSums &cw, bool split,
                          bool branching_listed, int64_t s0, int64_t s1, int64_t cut, int64_t base, F &&f) {
    for (int64_t s = s0; s < s1; ++s) {
        const StrRec &r = h->strs[(size_t)s];
        const TailRec t = split ? h->tail_rec[(size_t)s] : TailRec{0, 0, 0};
        int64_t g0 = r.first;
        const int64_t gl = (int64_t)r.first + (r.len - r.lcp);
        while (g0 <= gl) {
            const int64_t g1 = cut > 0 ? std::min(gl, base + ((g0 - base) / cut + 1) * cut - 1) : gl;
            const int64_t a = r.lcp + (g0 - r.first), b = r.lcp + (g1 - r.first);  // path indices
            int64_t sum;
            if (!split) {
                sum = cl.range(a + 1, b + 2);
            } else {
                const int64_t t0 = std::max<int64_t>(a, t.next);  // first tail of the piece
                const int64_t tails_w = t0 <= b ? cw.range(t0 - t.top, b - t.top + 1) : 0;
                if (branching_listed)
                    sum = cl.range(a + 1, b + 2) - tails_w;
                else
                    sum = (t0 <= b ? cl.range(t0 - t.top, b - t.top + 1) : 0) - tails_w;
            }
            f(g0, g1, sum);
            g0 = g1 + 1;
        }
    }
}

int64_t entry_upper_bound(const tam_handle *h, const tam_vocab *v) {
    const int64_t L = v->max_tok_len;
    const CumSums cl(v->dup_cum, L), cw(v->dup_cum, std::min<int64_t>(L, kWin));
    // Which hits at distance d above node m land in lists: all of them (lists
    // only); with tail compression and a table, those on the tails above m
    // (d <= tail_span[m]) longer than the probe window; with tail compression
    // and no table, also every hit on a branching ancestor (d > tail_span[m]).
    const bool split = h->tails;
    const bool branching_listed = split && (h->flags & TAM_FLAG_NO_TABLE);
    const int64_t K = (int64_t)h->strs.size(), chunk = 1 << 14, nchunks = (K + chunk - 1) / chunk;
    std::vector<int64_t> part((size_t)nchunks, 0);
    parallel_for(nchunks, host_threads(nchunks), [&](int64_t c) {
        int64_t b = 0;
        string_bounds(h, cl, cw, split, branching_listed, c * chunk, std::min(K, (c + 1) * chunk), 0, 0,
                      [&](int64_t, int64_t, int64_t x) { b += x; });
        part[(size_t)c] = b;
    });
    int64_t bound = 0;
    for (int64_t b : part) bound += b;
    return bound;
}

// A listed hit makes one record and at least one listed id, so a block's
// records are at most the sum of its nodes' bounds, and all regions together
// take at most entry_upper_bound records.  The blocks of a group cover its
// nodes [n0, n0 + blocks * per_block); a block's nodes may come from the
// strings of two tasks, whose sums meet in an atomic add.
int64_t group_regions(const tam_handle *h, const tam_vocab *v, int64_t s0, int64_t s1, int64_t n0,
                      int64_t per_block, int64_t blocks, int32_t *off) {
    const int64_t L = v->max_tok_len;
    const CumSums cl(v->dup_cum, L), cw(v->dup_cum, std::min<int64_t>(L, kWin));
    const bool split = h->tails;
    const bool branching_listed = split && (h->flags & TAM_FLAG_NO_TABLE);
    std::vector<int64_t> sums((size_t)blocks, 0);
    const int64_t K = s1 - s0, chunk = 1 << 12, nchunks = (K + chunk - 1) / chunk;
    parallel_for(nchunks, host_threads(nchunks), [&](int64_t c) {
        string_bounds(h, cl, cw, split, branching_listed, s0 + c * chunk, s0 + std::min(K, (c + 1) * chunk),
                      per_block, n0, [&](int64_t g0, int64_t, int64_t x) {
                          const int64_t b = (g0 - n0) / per_block;
                          if (x && b >= 0 && b < blocks) __atomic_fetch_add(&sums[(size_t)b], x, __ATOMIC_RELAXED);
                      });
    });
    int64_t run = 0;
    for (int64_t b = 0; b < blocks; ++b) {
        off[b] = (int32_t)std::min<int64_t>(run, INT32_MAX);
        run += sums[(size_t)b];
    }
    off[blocks] = (int32_t)std::min<int64_t>(run, INT32_MAX);
    return run;
}

}  // namespace tam
