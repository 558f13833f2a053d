// Working-set bookkeeping shared by the attention kernels: which key tiles a
// query chunk visits (Sec. 3.3 deterministic visibility, Sec. 3.4 working
// set) and where each tile's rows live.
#pragma once

#include "hga_device.hpp"

namespace hga {

// Closed visible chunks D_c = [0, a) U [max(a, w0), c), a = min(F, c),
// w0 = max(0, c - W); enumerated in ascending order.
struct VisibleChunks {
    int a;      // sinks [0, a)
    int start;  // recent window [start, c)
    int count;  // |D_c|
    __host__ __device__ VisibleChunks(int c, int keep_first, int window) {
        a = keep_first < c ? keep_first : c;
        int w0 = c - window;
        if (w0 < 0) w0 = 0;
        start = w0 > a ? w0 : a;
        count = a + (c - start);
    }
    __host__ __device__ int chunk(int idx) const { return idx < a ? idx : start + (idx - a); }
};

// Kinds of key tiles.
enum TileKind { kTileVisible = 0, kTileRouted = 1, kTileCurrent = 2 };

}  // namespace hga
