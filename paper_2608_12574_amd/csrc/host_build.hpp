// Host-side table construction for tam_compile.
#pragma once

#include <functional>
#include <string>

#include "tam_internal.hpp"

namespace tam {

// planned (optional) runs once the trie's sizes (N, S, blob bytes) are set in
// h and before any node is written; a non-OK status aborts the build.
tam_status build_trie(const uint8_t *str_bytes, const int64_t *str_off, int64_t K,
                      const int64_t *set_off, int64_t S, int terminator, tam_handle *h,
                      std::string *err, const std::function<tam_status(tam_handle *)> &planned = {});
tam_status build_vocab(const uint8_t *tok_bytes, const int64_t *tok_off, int64_t V, tam_vocab *h,
                       std::string *err);
int64_t entry_upper_bound(const tam_handle *h, const tam_vocab *v);

}  // namespace tam
