// Token gather / scatter along the Hilbert order (§3.4):
//   gather   y[b, d, :] = x[b, perm[d], :]
//   scatter  y[b, perm[d], :] = x[b, d, :]
// perm[d] < 0 marks a padding slot of a general shape (Appendix D): the
// gather writes a zero row there and the scatter skips it.  Entries >= n
// are skipped by both.
// Rows are copied as raw bytes.  The copy is HBM-bound and touches every
// byte once, so the row kernel's loads and stores are non-temporal: streamed
// through without displacing cached data, which on a cold copy is worth over
// 1.5x.  Rows of at least 64 vectors (1 KB at 16-byte vectors) go one row per
// wavefront, the row's source and destination found once in scalar
// registers and several vectors per lane in flight; shorter rows use a flat
// kernel in which consecutive threads take consecutive vectors.  Every
// wavefront access is one contiguous, coalesced segment.
#include "internal.hpp"

namespace hilberta {
namespace {

// vector types the non-temporal builtins accept
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int kUnroll = 4;
constexpr int kCopyThreads = 256;
constexpr int kRowUnroll = 4;            // vectors per lane in flight, row kernel
constexpr int64_t kMaxRowBlocks = 2048;  // about 8 workgroups per CU

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
            } else if (p < 0 && !a.scatter) {
                buf[u] = V{};
                dst[u] = b * a.y_bs + d * a.y_rs + col * (int64_t)sizeof(V);
            }
        }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        if (dst[u] >= 0) *reinterpret_cast<V*>(a.y + dst[u]) = buf[u];
    }
}


// Rows of at least one wavefront's worth of vectors: one wavefront copies a
// whole row at a time, U vectors per lane in flight, and finds the row's
// source and destination once, in scalar registers.
template <typename V, int U>
__global__ void __launch_bounds__(kCopyThreads) permute_rows_kernel(PermuteArgs a, int32_t vec_per_row,
                                                                    int64_t rows) {
    const int lane = threadIdx.x & 63;
    const int64_t wave = (int64_t)blockIdx.x * (kCopyThreads / 64) +
                         __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t n_waves = (int64_t)gridDim.x * (kCopyThreads / 64);
    for (int64_t row = wave; row < rows; row += n_waves) {
        const int64_t b = row / a.n;
        const int64_t d = row - b * a.n;
        const int32_t p = a.perm[d];
        if (p >= a.n || (p < 0 && a.scatter)) continue;
        const int64_t dst_row = a.scatter ? p : d;
        V* dst = reinterpret_cast<V*>(a.y + b * a.y_bs + dst_row * a.y_rs);
        if (p < 0) {
            // padding slot: a zero row
            for (int32_t c = lane; c < vec_per_row; c += 64) __builtin_nontemporal_store(V{}, dst + c);
            continue;
        }
        const int64_t src_row = a.scatter ? d : p;
        const V* src = reinterpret_cast<const V*>(a.x + b * a.x_bs + src_row * a.x_rs);
        for (int32_t c0 = 0; c0 < vec_per_row; c0 += 64 * U) {
            V buf[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t c = c0 + u * 64 + lane;
                if (c < vec_per_row) buf[u] = __builtin_nontemporal_load(src + c);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int32_t c = c0 + u * 64 + lane;
                if (c < vec_per_row) __builtin_nontemporal_store(buf[u], dst + c);
            }
        }
    }
}

template <typename V>
hipError_t launch_as(const PermuteArgs& a, hipStream_t s) {
    const int64_t vec_per_row = a.row_bytes / (int64_t)sizeof(V);
    const int64_t total = a.batch * a.n * vec_per_row;
    if (total == 0) return hipSuccess;
    if (vec_per_row >= 64 && vec_per_row <= 0x7fffffff) {
        const int64_t rows = a.batch * a.n;
        int64_t blocks = (rows + 3) / 4;
        if (blocks > kMaxRowBlocks) blocks = kMaxRowBlocks;
        hipLaunchKernelGGL((permute_rows_kernel<V, kRowUnroll>), dim3((unsigned)blocks), dim3(kCopyThreads), 0,
                           s, a, (int32_t)vec_per_row, rows);
        return hipGetLastError();
    }
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
    if (aligned(a, 16)) return launch_as<u32x4_t>(a, s);
    if (aligned(a, 8)) return launch_as<u32x2_t>(a, s);
    if (aligned(a, 4)) return launch_as<uint32_t>(a, s);
    return launch_as<uint16_t>(a, s);
}

}  // namespace hilberta
