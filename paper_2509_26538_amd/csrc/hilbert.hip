// Hilbert linearisation (§3.1) and the per-layer schedule table (§3.2, §3.3).
//
// A grid of grid_h x grid_w cells takes the curve of its enclosing square of
// side S = 2^order (the grid itself when it is a square power of two; the
// smallest enclosing power-of-two square otherwise, Appendix D).  Curve
// position d decodes to the cell (x, y), x = column, y = row; the cell is
// the grid's raster index y*grid_w + x when x < grid_w and y < grid_h, and a
// padding slot otherwise.
#include "curve.hpp"
#include "internal.hpp"

namespace hilberta {
namespace {



__global__ void __launch_bounds__(256) build_perm_kernel(int32_t side, int32_t grid_h, int32_t grid_w,
                                                         int32_t* __restrict__ perm,
                                                         int32_t* __restrict__ inv) {
    const int order = log2_side(side);
    const uint32_t n = (uint32_t)side * (uint32_t)side;
    for (uint32_t d = blockIdx.x * blockDim.x + threadIdx.x; d < n; d += gridDim.x * blockDim.x) {
        uint32_t x, y;
        hilbert_d2xy(order, d, x, y);
        const bool cell = x < (uint32_t)grid_w && y < (uint32_t)grid_h;
        const uint32_t raster = y * (uint32_t)grid_w + x;
        perm[d] = cell ? (int32_t)raster : -1;
        if (inv && cell) inv[raster] = (int32_t)d;
    }
}

// Shared runs: every cell of the central region finds its Hilbert position d
// and whether it starts a run (d-1 lies outside the region, or d = 0) or ends
// one (d+1 outside, or d = N-1).  Starts and ends are ranked separately; the
// i-th start pairs with the i-th end.  The whole workgroup calls this; the
// sorted run starts and (inclusive) ends land in LDS; returns the run count.
struct RunsLds {
    int32_t starts[kMaxSpans];
    int32_t ends[kMaxSpans];
    int32_t sorted_starts[kMaxSpans];
    int32_t sorted_ends[kMaxSpans];
    int32_t n_starts, n_ends;
};

__device__ int32_t shared_runs(RunsLds& r, int32_t side, int32_t grid_h, int32_t grid_w, int32_t shared_h,
                               int32_t shared_w, int32_t cap) {
    const int tid = threadIdx.x;
    const int order = log2_side(side);
    const uint32_t n_img = (uint32_t)side * (uint32_t)side;
    // the region is centred in the grid (which sits at the origin of the
    // enclosing square), so none of its cells is padding
    const int32_t r0 = (grid_h - shared_h) / 2;
    const int32_t c0 = (grid_w - shared_w) / 2;
    const int32_t n_cells = shared_h * shared_w;
    if (tid == 0) {
        r.n_starts = 0;
        r.n_ends = 0;
    }
    __syncthreads();
    auto inside = [&](uint32_t d) {
        uint32_t x, y;
        hilbert_d2xy(order, d, x, y);
        return (int32_t)y >= r0 && (int32_t)y < r0 + shared_h && (int32_t)x >= c0 &&
               (int32_t)x < c0 + shared_w;
    };
    for (int32_t u = tid; u < n_cells; u += blockDim.x) {
        const uint32_t y = (uint32_t)(r0 + u / shared_w);
        const uint32_t x = (uint32_t)(c0 + u % shared_w);
        const uint32_t d = hilbert_xy2d(order, x, y);
        if (d == 0 || !inside(d - 1)) {
            const int32_t i = atomicAdd(&r.n_starts, 1);
            if (i < kMaxSpans) r.starts[i] = (int32_t)d;
        }
        if (d == n_img - 1 || !inside(d + 1)) {
            const int32_t i = atomicAdd(&r.n_ends, 1);
            if (i < kMaxSpans) r.ends[i] = (int32_t)d;
        }
    }
    __syncthreads();
    int32_t n_runs = min(min(r.n_starts, r.n_ends), cap);
    n_runs = min(n_runs, kMaxSpans);
    for (int32_t i = tid; i < n_runs; i += blockDim.x) {
        int32_t rank_s = 0, rank_e = 0;
        for (int32_t j = 0; j < n_runs; ++j) {
            rank_s += r.starts[j] < r.starts[i];
            rank_e += r.ends[j] < r.ends[i];
        }
        r.sorted_starts[rank_s] = r.starts[i];
        r.sorted_ends[rank_e] = r.ends[i];
    }
    __syncthreads();
    return n_runs;
}

// The schedule in one launch.  Tiles of the slid partition: tile q holds
// the positions p of the tiled span (N tokens) with
// floor(((p + o) mod N) / N_T) = q, i.e. the cyclic range that starts at
// (q N_T - o) mod N; each carries the count of shared tokens inside it.
// Every workgroup finds the shared runs for itself (none in the moved-prefix
// layout, where the shared tokens sit in the prefix) and writes its 256
// tiles; workgroup 0 also writes the header and the runs.
__global__ void __launch_bounds__(256) schedule_kernel(ScheduleArgs a) {
    __shared__ RunsLds r;
    const int tid = threadIdx.x;
    const int32_t n_cells = a.shared_h * a.shared_w;
    const int32_t n_runs =
        a.moved || n_cells == 0 ? 0 : shared_runs(r, a.side, a.grid_h, a.grid_w, a.shared_h, a.shared_w, a.span_cap);
    if (blockIdx.x == 0) {
        int32_t* spans = a.out + 12 + 4 * a.n_tiles;
        for (int32_t i = tid; i < n_runs; i += blockDim.x) {
            spans[2 * i] = a.prefix + r.sorted_starts[i];
            spans[2 * i + 1] = r.sorted_ends[i] + 1 - r.sorted_starts[i];
        }
        for (int32_t i = n_runs + tid; i < a.span_cap; i += blockDim.x) {
            spans[2 * i] = 0;
            spans[2 * i + 1] = 0;
        }
        if (tid == 0) {
            int32_t* h = a.out;
            h[0] = 0x48424131;
            h[1] = a.prefix;
            h[2] = a.tiled;
            h[3] = a.tile;
            h[4] = a.n_tiles;
            h[5] = a.offset;
            h[6] = n_runs;
            h[7] = n_cells;
            h[8] = a.layer;
            h[9] = a.grid_h;
            h[10] = a.grid_w;
            h[11] = a.span_cap;
        }
    }
    const int32_t q = blockIdx.x * blockDim.x + tid;
    if (q >= a.n_tiles) return;
    const int32_t n_img = a.tiled;
    const int32_t start = (int32_t)(((int64_t)q * a.tile - a.offset + n_img) % n_img);
    const int32_t len1 = min(a.tile, n_img - start);
    const int32_t len2 = a.tile - len1;
    int32_t ns = 0;
    for (int32_t s = 0; s < n_runs; ++s) {
        const int32_t lo = r.sorted_starts[s];
        const int32_t hi = r.sorted_ends[s] + 1;
        ns += max(0, min(hi, start + len1) - max(lo, start));
        ns += max(0, min(hi, len2) - max(lo, 0));
    }
    int32_t* t = a.out + 12 + 4 * q;
    t[0] = a.prefix + start;
    t[1] = len1;
    t[2] = len2;
    t[3] = ns;
}

// The moved-prefix order of the image tokens: the shared tokens first, then
// the others, each part in Hilbert order.  Hilbert position d goes to slot
// c(d) if its cell is shared, else N_sh + d - c(d), where c(d) counts the
// shared cells at Hilbert positions below d (from the shared runs, which
// every workgroup finds for itself).
__global__ void __launch_bounds__(256) build_perm_moved_kernel(int32_t side, int32_t shared_h, int32_t shared_w,
                                                               int32_t* __restrict__ perm,
                                                               int32_t* __restrict__ inv) {
    __shared__ RunsLds r;
    const int32_t n_runs = shared_runs(r, side, side, side, shared_h, shared_w, kMaxSpans);
    const int order = log2_side(side);
    const uint32_t n = (uint32_t)side * (uint32_t)side;
    const int32_t n_sh = shared_h * shared_w;
    for (uint32_t d = blockIdx.x * blockDim.x + threadIdx.x; d < n; d += gridDim.x * blockDim.x) {
        int32_t below = 0;
        bool shared = false;
        for (int32_t i = 0; i < n_runs; ++i) {
            const int32_t st = r.sorted_starts[i], en = r.sorted_ends[i];
            below += max(0, min((int32_t)d, en + 1) - st);
            shared |= (int32_t)d >= st && (int32_t)d <= en;
        }
        uint32_t x, y;
        hilbert_d2xy(order, d, x, y);
        const uint32_t raster = y * (uint32_t)side + x;
        const int32_t slot = shared ? below : n_sh + (int32_t)d - below;
        perm[slot] = (int32_t)raster;
        if (inv) inv[raster] = slot;
    }
}

}  // namespace

hipError_t launch_build_perm(int32_t side, int32_t grid_h, int32_t grid_w, int32_t* perm, int32_t* inv,
                             hipStream_t s) {
    const int64_t n = (int64_t)side * side;
    const int64_t want = (n + 255) / 256;
    const int blocks = (int)(want < 65536 ? want : 65536);
    hipLaunchKernelGGL(build_perm_kernel, dim3(blocks), dim3(256), 0, s, side, grid_h, grid_w, perm, inv);
    return hipGetLastError();
}

hipError_t launch_build_perm_moved(int32_t side, int32_t shared_h, int32_t shared_w, int32_t* perm,
                                   int32_t* inv, hipStream_t s) {
    const int64_t n = (int64_t)side * side;
    const int64_t want = (n + 255) / 256;
    // every workgroup first finds the shared runs: keep the grid moderate
    const int blocks = (int)(want < 1024 ? want : 1024);
    hipLaunchKernelGGL(build_perm_moved_kernel, dim3(blocks), dim3(256), 0, s, side, shared_h, shared_w, perm, inv);
    return hipGetLastError();
}

hipError_t launch_schedule(const ScheduleArgs& a, hipStream_t s) {
    const int blocks = a.n_tiles > 256 ? (a.n_tiles + 255) / 256 : 1;
    hipLaunchKernelGGL(schedule_kernel, dim3(blocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace hilberta
