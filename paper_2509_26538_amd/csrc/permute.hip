// Token gather / scatter along the Hilbert order (§3.4):
//   gather   y[b, d, :] = x[b, perm[d], :]
//   scatter  y[b, perm[d], :] = x[b, d, :]
// Rows are copied as raw bytes.  The copy is HBM-bound: each thread moves
// kUnroll 16-byte vectors, issuing all loads before any store so that several
// requests are in flight, and consecutive threads touch consecutive vectors
// of a row so every wavefront access is one contiguous, coalesced segment.
#include "internal.hpp"

namespace hilberta {
namespace {

constexpr int kUnroll = 4;
constexpr int kCopyThreads = 256;

// I is the index type of the vector / row arithmetic: 32-bit whenever the
// sizes allow it, since 64-bit division costs far more than the copy.
template <typename V, typename I>
__global__ void __launch_bounds__(kCopyThreads) permute_kernel(PermuteArgs a, I vec_per_row,
                                                               I total_vec, I n) {
    const I first = (I)blockIdx.x * (I)(kCopyThreads * kUnroll) + (I)threadIdx.x;
    V buf[kUnroll];
    int64_t dst[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const I g = first + (I)(u * kCopyThreads);
        dst[u] = -1;
        if (g < total_vec) {
            const I row = g / vec_per_row;
            const int64_t col = (int64_t)(g - row * vec_per_row);
            const I bi = row / n;
            const int64_t b = (int64_t)bi;
            const int64_t d = (int64_t)(row - bi * n);
            const int32_t p = a.perm[d];
            if (p >= 0 && p < a.n) {
                const int64_t src_row = a.scatter ? d : p;
                const int64_t dst_row = a.scatter ? p : d;
                const char* src = a.x + b * a.x_bs + src_row * a.x_rs + col * (int64_t)sizeof(V);
                buf[u] = *reinterpret_cast<const V*>(src);
                dst[u] = b * a.y_bs + dst_row * a.y_rs + col * (int64_t)sizeof(V);
            }
        }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        if (dst[u] >= 0) *reinterpret_cast<V*>(a.y + dst[u]) = buf[u];
    }
}

template <typename V>
hipError_t launch_as(const PermuteArgs& a, hipStream_t s) {
    const int64_t vec_per_row = a.row_bytes / (int64_t)sizeof(V);
    const int64_t total = a.batch * a.n * vec_per_row;
    if (total == 0) return hipSuccess;
    const int64_t per_block = (int64_t)kCopyThreads * kUnroll;
    const int64_t blocks = (total + per_block - 1) / per_block;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    if (total + per_block < 0xffffffffLL) {
        hipLaunchKernelGGL((permute_kernel<V, uint32_t>), dim3((unsigned)blocks), dim3(kCopyThreads),
                           0, s, a, (uint32_t)vec_per_row, (uint32_t)total, (uint32_t)a.n);
    } else {
        hipLaunchKernelGGL((permute_kernel<V, int64_t>), dim3((unsigned)blocks), dim3(kCopyThreads),
                           0, s, a, vec_per_row, total, a.n);
    }
    return hipGetLastError();
}

bool aligned(const PermuteArgs& a, int64_t w) {
    return ((uintptr_t)a.x % w) == 0 && ((uintptr_t)a.y % w) == 0 && a.row_bytes % w == 0 &&
           a.x_bs % w == 0 && a.x_rs % w == 0 && a.y_bs % w == 0 && a.y_rs % w == 0;
}

}  // namespace

hipError_t launch_permute(const PermuteArgs& a, hipStream_t s) {
    if (aligned(a, 16)) return launch_as<uint4>(a, s);
    if (aligned(a, 8)) return launch_as<uint2>(a, s);
    if (aligned(a, 4)) return launch_as<uint32_t>(a, s);
    return launch_as<uint16_t>(a, s);
}

}  // namespace hilberta
