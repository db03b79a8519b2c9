// Host-side table construction for tam_compile.
#pragma once

#include <functional>
#include <string>

#include "tam_internal.hpp"

namespace tam {

// Ranges of the trie tables that are complete: nodes [n_lo, n_hi), blob
// bytes [b_lo, b_hi) and string records [s_lo, s_hi).
struct TrieRange {
    int64_t n_lo, n_hi, b_lo, b_hi, s_lo, s_hi;
};

// planned (optional) runs once the trie's sizes (N, S, blob bytes, edges) are
// set in h and before any node is written.  emitted (optional) runs after each
// group of whole sets has been written (the trie's tables in those ranges,
// tail compression's included, are then final).  A non-OK status of either
// aborts the build.
tam_status build_trie(const uint8_t *str_bytes, const int64_t *str_off, int64_t K,
                      const int64_t *set_off, int64_t S, int terminator, tam_handle *h,
                      std::string *err, const std::function<tam_status(tam_handle *)> &planned = {},
                      const std::function<tam_status(tam_handle *, const TrieRange &)> &emitted = {});
tam_status build_vocab(const uint8_t *tok_bytes, const int64_t *tok_off, int64_t V, tam_vocab *h,
                       std::string *err);
int64_t entry_upper_bound(const tam_handle *h, const tam_vocab *v);
// Tail compression without a table, one group of nodes [n0, ...) created by
// the strings [s0, s1): the region of each of its probe blocks (nodes
// [n0 + b * per_block, n0 + (b + 1) * per_block)) in the group's records of
// listed hits, sized by the same bound: off[b] .. off[b + 1] for b < blocks,
// off[blocks] = the group's total, which is returned.
int64_t group_regions(const tam_handle *h, const tam_vocab *v, int64_t s0, int64_t s1, int64_t n0,
                      int64_t per_block, int64_t blocks, int32_t *off);

// Runs f(j) for every j in [0, n) on up to `threads` host threads (the caller
// and workers of a process-wide pool); rethrows the first exception of f.
void host_parallel_for(int64_t n, int threads, const std::function<void(int64_t)> &f);

}  // namespace tam
