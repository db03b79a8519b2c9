// Host-side table construction for tam_compile.
#pragma once

#include <string>

#include "tam_internal.hpp"

namespace tam {

tam_status build_trie(const uint8_t *str_bytes, const int64_t *str_off, int64_t K,
                      const int64_t *set_off, int64_t S, int terminator, tam_handle *h,
                      std::string *err);
tam_status build_vocab(const uint8_t *tok_bytes, const int64_t *tok_off, int64_t V, tam_vocab *h,
                       std::string *err);
int64_t entry_upper_bound(const tam_handle *h, const tam_vocab *v);

}  // namespace tam
