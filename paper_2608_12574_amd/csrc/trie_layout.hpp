// The trie's position tables, derived from the string blob and one record per
// string (Section 4.1: one node per distinct prefix; the strings lie in the
// blob in trie order, each after a pad byte that stands for its set's root).
//
//   node_at[p]   the node whose edge byte is blob byte p (a pad: its set's root)
//   depth[g]     the prefix length of node g
//   node_pos[g]  the first blob position of non-root node g (-1 at roots)
//   parent(g)    node_at[node_pos[g] - 1]
//
// The kernels that lay these tables out on the device call the functions
// below, and the host runs the same functions over the host records so that
// the layout can be checked without a GPU.  Every write and every record read
// is range-checked: an inconsistent record, which the host build never makes,
// is counted instead of being followed, and the caller reports the count.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "device_tables.hpp"

namespace tam {

// node_at and depth of string record u (one of the records [s0, s1) of a group
// of whole sets).  String u creates the nodes first .. first + len - lcp along
// path indices lcp .. len (depth = index + 1); below index lcp its path is an
// earlier string's: index i belongs to the nearest earlier string v of the
// part with lcp[v] <= i.  Walking from u - 1 along psv (each step lowers the
// common prefix), a string whose lcp lies below the indices still open owns
// [lcp[v], open bound); one whose lcp does not is passed over.  The chain ends
// at a string with lcp 0, which owns all that is open.  Returns the number of
// inconsistent record fields met (0 for the host build's records).
__host__ __device__ inline int32_t lay_string(const StrRec *strs, int64_t s0, int64_t u, int64_t blob_bytes,
                                              int64_t N, int32_t *node_at, int32_t *depth) {
    const StrRec r = strs[u];
    if (r.at < 0 || r.len < 0 || r.lcp < 0 || r.lcp > r.len || (int64_t)r.at + 1 + r.len >= blob_bytes ||
        r.root < 0 || (int64_t)r.root >= N || r.first < 0 || (int64_t)r.first + (r.len - r.lcp) >= N)
        return 1;
    node_at[r.at] = r.root;  // the pad stands for the root
    if (r.lcp == 0) depth[r.root] = 0;
    for (int32_t i = r.lcp; i <= r.len; ++i) {
        const int32_t g = r.first + (i - r.lcp);
        node_at[r.at + 1 + i] = g;
        depth[g] = i + 1;
    }
    int32_t hi = r.lcp;  // path indices [0, hi) still open
    int64_t v = u - 1;   // lcp > 0: not the first string of its part
    while (hi > 0) {
        if (v < s0 || v >= u) return 1;  // the chain left the group, or does not go back
        const StrRec q = strs[v];
        if (q.lcp < hi) {
            if (q.lcp < 0 || q.first < 0 || (int64_t)q.first + (hi - 1 - q.lcp) >= N) return 1;
            for (int32_t i = q.lcp; i < hi; ++i) node_at[r.at + 1 + i] = q.first + (i - q.lcp);
            hi = q.lcp;
        }
        if (q.psv >= v) return 1;  // each step must go back
        v = q.psv;
    }
    return 0;
}

// The node whose first position may be blob position p: node_at[p] unless it
// is a root (a pad), else -1.  *bad is set when node_at[p] is not a node.
__host__ __device__ inline int32_t lay_pos_node(const int32_t *node_at, const int32_t *depth, int64_t N, int64_t p,
                                                bool *bad) {
    const int32_t g = node_at[p];
    if (g < 0 || (int64_t)g >= N) {
        *bad = true;
        return -1;
    }
    return depth[g] > 0 ? g : -1;
}

// The parent of non-root node g, or -1 with *bad set when g has no position
// inside the blob or the byte before it is not a node.
__host__ __device__ inline int32_t lay_parent(const int32_t *node_pos, const int32_t *node_at, int64_t N,
                                              int64_t blob_bytes, int64_t g, bool *bad) {
    const int64_t pos = node_pos[g];
    if (pos <= 0 || pos >= blob_bytes) {
        *bad = true;
        return -1;
    }
    const int32_t par = node_at[pos - 1];
    if (par < 0 || (int64_t)par >= N) {
        *bad = true;
        return -1;
    }
    return par;
}

}  // namespace tam
