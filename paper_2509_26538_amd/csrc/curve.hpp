// The Hilbert curve of a 2^order x 2^order grid (§3.1), decoded and encoded
// digit by digit.  The base-4 digits of a position d, from the least
// significant, say which quadrant of the next larger square the partial
// curve lies in and whether it is transposed (and reflected) there.
// Orientation: start (0, 0), end (side-1, 0), x = column, y = row.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hilberta {

__device__ __forceinline__ void hilbert_d2xy(int order, uint32_t d, uint32_t& x, uint32_t& y) {
    uint32_t px = 0, py = 0;
    for (int lvl = 0; lvl < order; ++lvl) {
        const uint32_t s = 1u << lvl;
        const uint32_t digit = (d >> (2 * lvl)) & 3u;
        const uint32_t rx = digit >> 1;
        const uint32_t ry = (digit ^ rx) & 1u;
        if (ry == 0) {
            if (rx) {
                px = s - 1 - px;
                py = s - 1 - py;
            }
            const uint32_t t = px;
            px = py;
            py = t;
        }
        px += s * rx;
        py += s * ry;
    }
    x = px;
    y = py;
}

// Inverse of hilbert_d2xy: peel the most significant quadrant first.
__device__ __forceinline__ uint32_t hilbert_xy2d(int order, uint32_t x, uint32_t y) {
    uint32_t d = 0;
    for (int lvl = order - 1; lvl >= 0; --lvl) {
        const uint32_t s = 1u << lvl;
        const uint32_t rx = (x >> lvl) & 1u;
        const uint32_t ry = (y >> lvl) & 1u;
        d += s * s * ((3u * rx) ^ ry);
        x &= s - 1;
        y &= s - 1;
        if (ry == 0) {
            const uint32_t t = x;
            x = y;
            y = t;
            if (rx) {
                x = s - 1 - x;
                y = s - 1 - y;
            }
        }
    }
    return d;
}

__device__ __forceinline__ int log2_side(int32_t side) { return 31 - __clz(side); }

}  // namespace hilberta
