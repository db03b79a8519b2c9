// HIP kernels of libtam for gfx950 (CDNA4, wave64).
//
// Mask compile (Section 4.1, valid[n] for every trie node n):
//   k_probe<false>  count   -- every non-root node m walks back over the last
//                              d <= min(depth(m), max_len) bytes of its prefix and
//                              looks each suffix up in the vocabulary hash; a hit
//                              of token t at distance d = |t| means t is valid at
//                              the ancestor d levels up (its walk ends at m).  This
//                              is the paper's "credit the match to the node |t|
//                              bytes back" (Section 4.2), done for all nodes at
//                              once instead of along a DFS.
//   k_scan_*                -- exclusive prefix sum of the per-node counts.
//   k_probe<true>   fill    -- the same probes, writing the token ids into the
//                              per-node lists (order within a list is irrelevant).
//   k_rows                  -- one (row, tile) per work item: the tile's bits are
//                              OR-ed into an LDS image from the row's list, then
//                              the image is streamed to HBM with 16-byte
//                              non-temporal stores and cleared for the next item.
// Serving (Section 2, Eq. 1 and the extended transition function):
//   k_apply                 -- write-mostly masking of [B, V] logits.
//   k_advance               -- B byte walks over the child tables.
//   k_export_dense          -- canonical rows out of the dense table.
#include <hip/hip_runtime.h>

#include "tam_internal.hpp"

namespace tam {
namespace {

constexpr int kBlock = 256;
constexpr int kWave = 64;
constexpr int kTileWords = 4096;     // 64-bit words per LDS row image (32 KiB)
constexpr int kApplyUnits = 4;       // 16-byte chunks per thread in k_apply

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

__global__ void __launch_bounds__(kBlock) k_fill_i32(int32_t *p, int64_t n, int32_t value) {
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += (int64_t)gridDim.x * kBlock)
        p[i] = value;
}

// ---------------------------------------------------------------- probes ---

// Slot of the token string equal to blob[pos-d+1 .. pos] (key = its hash), or -1.
__device__ __forceinline__ int64_t probe(const DevTables &t, uint64_t key, int64_t pos, int d) {
    uint64_t i = key & t.slot_mask;
    for (;;) {
        const HashSlot s = t.slots[i];
        if (s.first < 0) return -1;
        if (s.key == key) {
            const uint32_t off = t.tok_off[s.first];
            const uint32_t len = t.tok_off[s.first + 1] - off;
            if (len == (uint32_t)d) {
                const uint8_t *a = t.tok_blob + off;
                const uint8_t *b = t.blob + (pos - d + 1);
                bool eq = true;
                for (int k = 0; k < d; ++k) {
                    if (a[k] != b[k]) {
                        eq = false;
                        break;
                    }
                }
                if (eq) return (int64_t)i;
            }
        }
        i = (i + 1) & t.slot_mask;
    }
}

template <bool kFill>
__global__ void __launch_bounds__(kBlock) k_probe(DevTables t) {
    const int64_t m = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (m >= t.N) return;
    const int64_t pos = t.node_pos[m];
    if (pos < 0) return;  // a root ends no token
    const int L = min(t.depth[m], t.max_len);
    uint64_t h = kHashSeed;
    for (int d = 1; d <= L; ++d) {
        h = hash_step(h, t.blob[pos - d + 1]);
        if (!t.len_present[d]) continue;
        const int64_t si = probe(t, hash_final(h, (uint32_t)d), pos, d);
        if (si < 0) continue;
        const HashSlot s = t.slots[si];
        const int32_t n = t.node_at[pos - d];  // the ancestor where the token starts
        if (!kFill) {
            atomicAdd(&t.count[n], s.count);
        } else {
            int32_t at = t.row_ptr[n] + atomicAdd(&t.cursor[n], s.count);
            int32_t v = s.first;
            for (int k = 0; k < s.count; ++k) {
                t.entries[at + k] = v;
                v = t.dup_next[v];
            }
        }
    }
}

// ------------------------------------------------------------------ scan ---

constexpr int kScanItems = 8;
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

__global__ void __launch_bounds__(kBlock) k_scan_blocks(const int32_t *in, int64_t n, int32_t *sums) {
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int32_t s = 0;
    for (int k = 0; k < kScanItems; ++k)
        if (base + k < n) s += in[base + k];
    int32_t total;
    block_exclusive_scan(s, &total);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// One block: exclusive scan of the nb block sums in place; grand total -> *total_out.
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

__global__ void __launch_bounds__(kBlock) k_scan_apply(const int32_t *in, int64_t n, const int32_t *sums,
                                                       int32_t *out) {
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    int32_t v[kScanItems];
    int32_t s = 0;
    for (int k = 0; k < kScanItems; ++k) {
        v[k] = base + k < n ? in[base + k] : 0;
        s += v[k];
    }
    int32_t total;
    int32_t run = sums[blockIdx.x] + block_exclusive_scan(s, &total);
    for (int k = 0; k < kScanItems; ++k) {
        if (base + k < n) out[base + k] = run;
        run += v[k];
    }
}

// ------------------------------------------------------------ row images ---

// Work item (r, tile): the node is nodes[r] (or r when nodes is null); the tile
// covers words [tile*kTileWords, ...) of the out_words-word row written at
// out + r*out_stride.  `vec`: rows and tiles are 16-byte aligned.
__global__ void __launch_bounds__(kBlock) k_rows(DevTables t, const int32_t *nodes, int64_t nrows,
                                                 uint64_t *out, int64_t out_stride, int64_t out_words,
                                                 int64_t ntiles, int tile_words, int vec) {
    extern __shared__ u32x4 img[];  // tile_words * 8 bytes
    uint32_t *img32 = reinterpret_cast<uint32_t *>(img);
    uint64_t *img64 = reinterpret_cast<uint64_t *>(img);
    for (int i = threadIdx.x; i < tile_words / 2; i += kBlock) img[i] = u32x4{0u, 0u, 0u, 0u};
    __syncthreads();
    const int64_t items = nrows * ntiles;
    for (int64_t it = blockIdx.x; it < items; it += gridDim.x) {
        const int64_t r = it / ntiles;
        const int64_t w0 = (it - r * ntiles) * tile_words;
        const int wn = (int)min<int64_t>(tile_words, out_words - w0);
        const int64_t n = nodes ? (int64_t)nodes[r] : r;
        if (n >= 0 && n < t.N) {
            const int32_t b = t.row_ptr[n], e = t.row_ptr[n + 1];
            const uint32_t lo = (uint32_t)(w0 * 64);
            const uint32_t span = (uint32_t)wn * 64u;
            for (int32_t k = b + (int32_t)threadIdx.x; k < e; k += kBlock) {
                const uint32_t v = (uint32_t)t.entries[k] - lo;
                if (v < span) atomicOr(&img32[v >> 5], 1u << (v & 31));
            }
        }
        __syncthreads();
        uint64_t *dst = out + r * out_stride + w0;
        if (vec) {
            u32x4 *d4 = reinterpret_cast<u32x4 *>(dst);
            for (int c = threadIdx.x; c < wn / 2; c += kBlock) {
                const u32x4 x = img[c];
                img[c] = u32x4{0u, 0u, 0u, 0u};
                __builtin_nontemporal_store(x, d4 + c);
            }
        } else {
            for (int c = threadIdx.x; c < wn; c += kBlock) {
                const uint64_t x = img64[c];
                img64[c] = 0;
                __builtin_nontemporal_store(x, dst + c);
            }
        }
        __syncthreads();
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

// Grid: x = groups of kBlock*kApplyUnits chunks of one row, y = batch row.
// A chunk is 16 bytes of logits (8 bf16 or 4 fp32).  kSparse: the mask bits of
// the block's span come from the node's valid list via an LDS bitmap instead of
// the dense table.  vec == 0: rows are not 16-byte aligned, go element by element.
template <typename T, bool kSparse>
__global__ void __launch_bounds__(kBlock) k_apply(DevTables t, const int32_t *node_ids, T *logits,
                                                  int64_t stride, int vec) {
    constexpr int E = 16 / (int)sizeof(T);
    constexpr uint32_t FULL = (1u << E) - 1u;
    constexpr T NEG = NegInf<T>::bits;
    constexpr int kSpan = kBlock * kApplyUnits * E;  // elements per block
    __shared__ uint32_t bm[kSparse ? kSpan / 32 : 1];

    const int64_t V = t.V;
    const int64_t b = blockIdx.y;
    const int32_t n = node_ids[b];
    const bool live = n >= 0 && (int64_t)n < t.N;
    const int64_t c0 = (int64_t)blockIdx.x * kBlock * kApplyUnits;
    const int64_t nchunks = (V + E - 1) / E;
    T *row = logits + b * stride;

    const uint8_t *mrow = nullptr;
    if (kSparse) {
        for (int i = threadIdx.x; i < kSpan / 32; i += kBlock) bm[i] = 0;
        __syncthreads();
        if (live) {
            const int32_t e0 = t.row_ptr[n], e1 = t.row_ptr[n + 1];
            const uint32_t lo = (uint32_t)(c0 * E);
            for (int32_t k = e0 + (int32_t)threadIdx.x; k < e1; k += kBlock) {
                const uint32_t v = (uint32_t)t.entries[k] - lo;
                if (v < (uint32_t)kSpan) atomicOr(&bm[v >> 5], 1u << (v & 31));
            }
        }
        __syncthreads();
    } else if (live) {
        mrow = reinterpret_cast<const uint8_t *>(t.table + (int64_t)n * t.Wp);
    }

#pragma unroll
    for (int u = 0; u < kApplyUnits; ++u) {
        const int64_t lc = (int64_t)u * kBlock + threadIdx.x;  // chunk within the block
        const int64_t c = c0 + lc;
        if (c >= nchunks) break;
        uint32_t bits = 0;
        if (kSparse) {
            const uint32_t bit = (uint32_t)(lc * E);
            bits = (bm[bit >> 5] >> (bit & 31)) & FULL;
        } else if (live) {
            bits = E == 8 ? (uint32_t)mrow[c] : ((uint32_t)mrow[c >> 1] >> ((c & 1) * 4)) & FULL;
        }
        if (bits == FULL) continue;
        const int64_t e0 = c * E;
        if (vec && e0 + E <= V) {
            u32x4 *p = reinterpret_cast<u32x4 *>(row + e0);
            if (bits == 0) {
                u32x4 neg;
                if (sizeof(T) == 2) {
                    const uint32_t w = 0xFF80FF80u;
                    neg = u32x4{w, w, w, w};
                } else {
                    const uint32_t w = 0xFF800000u;
                    neg = u32x4{w, w, w, w};
                }
                __builtin_nontemporal_store(neg, p);
            } else {
                u32x4 x = *p;
                T vals[E];
                __builtin_memcpy(vals, &x, 16);
#pragma unroll
                for (int i = 0; i < E; ++i)
                    if (!((bits >> i) & 1u)) vals[i] = NEG;
                __builtin_memcpy(&x, vals, 16);
                *p = x;
            }
        } else {
            const int lim = (int)min<int64_t>(E, V - e0);
            for (int i = 0; i < lim; ++i)
                if (!((bits >> i) & 1u)) row[e0 + i] = NEG;
        }
    }
}

// --------------------------------------------------------------- advance ---

__global__ void __launch_bounds__(kBlock) k_advance(DevTables t, const int32_t *nodes, const int32_t *toks,
                                                    int64_t B, int32_t *out) {
    const int64_t b = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (b >= B) return;
    const int32_t n0 = nodes[b];
    const int32_t v = toks[b];
    int32_t n = TAM_DEAD;
    if (n0 >= 0 && (int64_t)n0 < t.N && v >= 0 && (int64_t)v < t.V) {
        const uint32_t a = t.tok_off[v], e = t.tok_off[v + 1];
        if (e > a) {
            n = n0;
            for (uint32_t i = a; i < e && n >= 0; ++i) {
                const uint8_t c = t.tok_blob[i];
                int32_t lo = t.child_off[n], hi = t.child_off[n + 1];
                int32_t next = TAM_DEAD;
                while (lo < hi) {
                    const int32_t mid = (lo + hi) >> 1;
                    const uint8_t cb = t.child_byte[mid];
                    if (cb < c) {
                        lo = mid + 1;
                    } else if (cb > c) {
                        hi = mid;
                    } else {
                        next = t.child_node[mid];
                        break;
                    }
                }
                n = next;
            }
        }
    }
    out[b] = n;
}

// ---------------------------------------------------------------- export ---

__global__ void __launch_bounds__(kBlock) k_export_dense(DevTables t, const int32_t *nodes, uint64_t *out) {
    const int64_t r = blockIdx.y;
    const int64_t w = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (w >= t.W) return;
    const int32_t n = nodes[r];
    const bool live = n >= 0 && (int64_t)n < t.N;
    out[r * t.W + w] = live ? t.table[(int64_t)n * t.Wp + w] : 0ull;
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

hipError_t launch_count(const DevTables &t, hipStream_t s) {
    if (t.N <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_probe<false>, dim3(grid_for(t.N, kBlock)), dim3(kBlock), 0, s, t);
    return hipGetLastError();
}

hipError_t launch_fill_lists(const DevTables &t, hipStream_t s) {
    if (t.N <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_probe<true>, dim3(grid_for(t.N, kBlock)), dim3(kBlock), 0, s, t);
    return hipGetLastError();
}

hipError_t launch_scan(const DevTables &t, hipStream_t s) {
    const int64_t nb = grid_for(t.N, kScanTile);
    hipLaunchKernelGGL(k_scan_blocks, dim3((unsigned)nb), dim3(kBlock), 0, s, t.count, t.N, t.scan_tmp);
    hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(kBlock), 0, s, t.scan_tmp, nb, t.row_ptr + t.N);
    hipLaunchKernelGGL(k_scan_apply, dim3((unsigned)nb), dim3(kBlock), 0, s, t.count, t.N, t.scan_tmp,
                       t.row_ptr);
    return hipGetLastError();
}

hipError_t launch_rows(const DevTables &t, const int32_t *nodes, int64_t nrows, uint64_t *out,
                       int64_t out_stride_words, int64_t out_words, hipStream_t s) {
    if (nrows <= 0 || out_words <= 0) return hipSuccess;
    const int tile_words = (int)std::min<int64_t>(kTileWords, (out_words + 1) & ~int64_t(1));
    const int64_t ntiles = (out_words + tile_words - 1) / tile_words;
    const int vec = ((out_stride_words & 1) == 0 && (out_words & 1) == 0 &&
                     (reinterpret_cast<uintptr_t>(out) & 15) == 0)
                        ? 1
                        : 0;
    const size_t lds = (size_t)tile_words * 8;
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_rows, kBlock, lds) != hipSuccess ||
        per_cu <= 0)
        per_cu = 4;
    const int64_t cap = (int64_t)props_for_current_device().cus * per_cu;
    const unsigned g = (unsigned)std::min<int64_t>(nrows * ntiles, cap);
    hipLaunchKernelGGL(k_rows, dim3(g), dim3(kBlock), lds, s, t, nodes, nrows, out, out_stride_words,
                       out_words, ntiles, tile_words, vec);
    return hipGetLastError();
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
    const bool sparse = t.table == nullptr;
    // grid.y is limited to 65535 rows per launch
    for (int64_t r0 = 0; r0 < B; r0 += 65535) {
        const dim3 grid(gx, (unsigned)std::min<int64_t>(B - r0, 65535));
        const int32_t *ids = node_ids + r0;
        if (dtype == TAM_DTYPE_BF16) {
            uint16_t *p = static_cast<uint16_t *>(logits) + r0 * row_stride;
            if (sparse)
                hipLaunchKernelGGL((k_apply<uint16_t, true>), grid, dim3(kBlock), 0, s, t, ids, p, row_stride, vec);
            else
                hipLaunchKernelGGL((k_apply<uint16_t, false>), grid, dim3(kBlock), 0, s, t, ids, p, row_stride, vec);
        } else {
            uint32_t *p = static_cast<uint32_t *>(logits) + r0 * row_stride;
            if (sparse)
                hipLaunchKernelGGL((k_apply<uint32_t, true>), grid, dim3(kBlock), 0, s, t, ids, p, row_stride, vec);
            else
                hipLaunchKernelGGL((k_apply<uint32_t, false>), grid, dim3(kBlock), 0, s, t, ids, p, row_stride, vec);
        }
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_advance(const DevTables &t, const int32_t *node_ids, const int32_t *token_ids, int64_t B,
                          int32_t *out, hipStream_t s) {
    if (B <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_advance, dim3(grid_for(B, kBlock)), dim3(kBlock), 0, s, t, node_ids, token_ids, B,
                       out);
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
    return hipSuccess;
}

}  // namespace tam
