// Tile-to-tensor lookup of the int8 tensor table (bf16 plans read a
// descriptor per tile instead).
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace es {

// Index of the tensor that owns global tile `tile`: the last entry i >= t
// with first(i) <= tile, where first() is non-decreasing over the table and
// entry n (the sentinel) lies beyond every tile.  A workgroup's tiles only
// move forward, so the search starts at its current entry t: one load when
// the tile is still in the same tensor, otherwise steps of 1, 2, 4, ... and
// bisection, O(log distance) loads however many small tensors lie between
// two of its tiles.  All indices read are <= n.
template <class First>
__device__ __forceinline__ uint32_t seek_tensor(uint32_t t, uint64_t tile, uint32_t n,
                                                First first) {
    if (tile < first(t + 1)) return t;
    uint32_t lo = t + 1, hi = n, step = 1;     // first(lo) <= tile < first(hi)
    for (;;) {
        const uint32_t probe = lo + step;
        if (probe >= n) break;
        if (tile < first(probe)) {
            hi = probe;
            break;
        }
        lo = probe;
        step <<= 1;
    }
    while (hi - lo > 1) {
        const uint32_t mid = lo + (hi - lo) / 2;
        if (first(mid) <= tile) lo = mid;
        else hi = mid;
    }
    return lo;
}

}  // namespace es
