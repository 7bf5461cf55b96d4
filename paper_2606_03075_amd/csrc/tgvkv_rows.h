// Row addressing of the compacted cache, shared by compaction and decode.
//
// A (sequence, layer) keeps b_l retained rows followed by decode_reserve slots
// for the tokens decode appends.  Two layouts hold them:
//   * ContigRows: one segment per (sequence, layer) at seg_off, [H_kv][b_l + reserve][D];
//   * PagedRows:  fixed pages of 2^shift rows from a pool [n_pages][H_kv][2^shift][D],
//     row n of (sequence, layer) bl in page block_table[bl][n >> shift].
// Both give the element offset of a row, identical for the key and the value
// cache, so the kernels above them do the same arithmetic for either layout.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "tgvkv_shape.h"

namespace tgvkv {

template <int D>
struct ContigRows {
    const int64_t* seg_off;
    int reserve;
    size_t base;
    // `rows` and `lds` are unused: the segment is found from seg_off alone.
    __device__ void init(const Shape& s, int bl, int kvh, int bsz, int rows, int* lds) {
        (void)rows;
        (void)lds;
        base = ((size_t)seg_off[bl] * s.Hkv + (size_t)kvh * (bsz + reserve)) * D;
    }
    __device__ size_t row(int n) const { return base + (size_t)n * D; }
    static constexpr size_t lds_bytes(int) { return 0; }
};

// The page ids of rows [0, rows) are copied into LDS (clamped into the pool, so an
// unfilled table entry of -1 can never address outside it, and a row past the
// table's width reads its last entry) so that a row's address costs no global
// load.  init() is called by every thread and must be followed by a barrier
// before row() is used.
template <int D>
struct PagedRows {
    const int32_t* block_table;
    int max_pages, shift, n_pages;
    int hkv, kvh;
    const int* pages;
    __device__ void init(const Shape& s, int bl, int kvh_, int bsz, int rows, int* lds) {
        (void)bsz;
        hkv = s.Hkv;
        kvh = kvh_;
        const int np = min((rows + (1 << shift) - 1) >> shift, max_pages);
        for (int i = threadIdx.x; i < np; i += blockDim.x)
            lds[i] = min(max(block_table[(size_t)bl * max_pages + i], 0), n_pages - 1);
        pages = lds;
    }
    __device__ size_t row(int n) const {
        const size_t pg = (size_t)pages[min(n >> shift, max_pages - 1)];
        return (((pg * hkv + kvh) << shift) | (size_t)(n & ((1 << shift) - 1))) * D;
    }
    static constexpr size_t lds_bytes(int max_pages) { return sizeof(int) * (size_t)max_pages; }
};

}  // namespace tgvkv
