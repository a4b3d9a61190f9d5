// HilbertA attention backward, fp32 path: dQ, dK and dV of the masked
// softmax attention (the gradients of §3.2-§3.4's attention), everything in
// fp32, for tight parity with the float64 oracle's gradients.
//
// The work items and lists are the bf16 path's (attn_bwd.hip): the dQ pass
// walks each query block's key list, the dK/dV pass each key block's list of
// the queries that attend it, built the same way because the mask is
// symmetric.  Dense rows are not split into key chunks.  Two lanes own one
// row, each holding half of its D columns (a dot product is the two halves'
// sum), and the arithmetic is plain fp32 on the vector ALUs: this path is
// for exactness at small sizes, not for speed.
//
// With P = exp(S - LSE) and Dlt_i = dO_i . O_i:
//   dP = dO V^T,  dS = P (dP - Dlt),  dQ = scale dS K,  dK = scale dS^T Q,
//   dV = P^T dO.
#include "bf16_stage.hpp"

namespace hilberta {
namespace {

// Dlt_i = dO_i . O_i and lse2_i = LSE_i log2(e) (0 for a row that attends
// nothing, whose probabilities are all masked anyway); one thread per row.
template <int D>
__global__ void __launch_bounds__(256) bwd_prep_f32_kernel(AttnArgs a, BwdArgs g) {
    const int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (r >= (int64_t)a.n_bh * a.n_tot) return;
    const int64_t bh = r / a.n_tot, n = r - bh * a.n_tot;
    const int64_t b = bh / a.heads, hh = bh - b * a.heads;
    const int64_t off = b * a.o_sb + hh * a.o_sh + n * a.o_sr;
    const float* o = static_cast<const float*>(a.o) + off;
    const float* d = static_cast<const float*>(g.dout) + off;
    float t = 0.f;
#pragma unroll 8
    for (int e = 0; e < D; ++e) t = fmaf(o[e], d[e], t);
    g.delta[r] = t;
    const float l = g.lse[r];
    g.lse2[r] = l == -INFINITY ? 0.f : l * 1.4426950408889634f;
}

// Item decode and list, shared by both passes: rows row0 .. row0 + 127 of
// item blockIdx.x; thread t owns row t/2, columns (t%2) D/2 .. + D/2.
struct F32Item {
    int32_t bh, bb, hh, o;
    bool dense;
    ItemList L;
    RowInfo ri;
};

template <bool PAD>
__device__ __forceinline__ F32Item f32_item(const AttnArgs& a, Spans& sp, int32_t& n_keep) {
    const int tid = threadIdx.x;
    F32Item it;
    const int32_t item = blockIdx.x;
    it.bh = item / a.items_per_bh;
    const int32_t r = item - it.bh * a.items_per_bh;
    const int32_t dense_items = a.dense_row_blocks * a.n_chunks;
    it.dense = r < dense_items;
    const int32_t chunk = it.dense ? r % a.n_chunks : 0;
    const int32_t row0 = it.dense ? (r / a.n_chunks) * kBlockM : (r - dense_items) * kBlockM;
    it.o = load_spans<kThreads>(a, sp, tid);
    const int32_t n_shared = a.sparse ? sp.cum[sp.n] : 0;
    it.L = item_list(a, it.dense, chunk, row0, it.o, n_shared, sp, n_keep, tid >> 6, tid & 63);
    it.ri = row_info(a, it.dense, row0, tid >> 1, kBlockM, it.o, n_shared, sp);
    if (!PAD) it.ri.pad = false;
    it.bb = it.bh / a.heads;
    it.hh = it.bh - it.bb * a.heads;
    return it;
}

// Row seq of a [B, H, N, D] fp32 tensor, this thread's half of the columns.
__device__ __forceinline__ const float* f32_row(const void* base, int64_t sb, int64_t sh, int64_t sr, int32_t bb,
                                                int32_t hh, int32_t seq, int half, int d) {
    return static_cast<const float*>(base) + bb * sb + hh * sh + (int64_t)seq * sr + half * (d / 2);
}

template <int D, bool PAD>
__global__ void __launch_bounds__(kThreads) bwd_dq_f32_kernel(AttnArgs a, BwdArgs g) {
    constexpr int H2 = D / 2;
    __shared__ Spans sp;
    __shared__ int32_t n_keep;
    const int half = threadIdx.x & 1;
    const F32Item it = f32_item<PAD>(a, sp, n_keep);
    const RowInfo& ri = it.ri;
    float qv[H2], dv[H2], acc[H2];
    const float* qr = f32_row(a.q, a.q_sb, a.q_sh, a.q_sr, it.bb, it.hh, ri.qseq, half, D);
    const float* dr = f32_row(g.dout, a.o_sb, a.o_sh, a.o_sr, it.bb, it.hh, ri.qseq, half, D);
#pragma unroll
    for (int e = 0; e < H2; ++e) {
        qv[e] = qr[e];
        dv[e] = dr[e];
        acc[e] = 0.f;
    }
    const int64_t row = (int64_t)it.bh * a.n_tot + ri.qseq;
    const float l2 = g.lse2[row], dl = g.delta[row];
    const float c = a.scale_log2;
    const ItemList& L = it.L;
    for (int32_t v = 0; v < L.total; ++v) {
        const int32_t seq = list_seq(v, L.b1, L.b2, L.b3, L.s0, L.sa, L.sb, sp);
        const int32_t inf = entry_info<PAD>(a, L, v, seq, it.o, sp);
        const float* kr = f32_row(a.k, a.k_sb, a.k_sh, a.k_sr, it.bb, it.hh, seq, half, D);
        const float* vr = f32_row(a.v, a.v_sb, a.v_sh, a.v_sr, it.bb, it.hh, seq, half, D);
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int e = 0; e < H2; ++e) {
            s = fmaf(qv[e], kr[e], s);
            dp = fmaf(dv[e], vr[e], dp);
        }
        s += __shfl_xor(s, 1);
        dp += __shfl_xor(dp, 1);
        const bool ok = inf == kKeyAll || inf == ri.label;
        const float p = ok ? exp2f(fmaf(s, c, -l2)) : 0.f;
        const float ds = p * (dp - dl);
#pragma unroll
        for (int e = 0; e < H2; ++e) acc[e] = fmaf(ds, kr[e], acc[e]);
    }
    if (!ri.store) return;
    const float mul = c * 0.69314718055994530942f;  // the softmax scale
    float* out = static_cast<float*>(g.dq) + it.bb * a.q_sb + it.hh * a.q_sh + (int64_t)ri.qseq * a.q_sr + half * H2;
    // a padding slot is written as zeros by selection: its sums may be inf
    // or NaN, and inf * 0 is NaN
#pragma unroll
    for (int e = 0; e < H2; ++e) out[e] = ri.pad ? 0.f : acc[e] * mul;
}

template <int D, bool PAD>
__global__ void __launch_bounds__(kThreads) bwd_dkdv_f32_kernel(AttnArgs a, BwdArgs g) {
    constexpr int H2 = D / 2;
    __shared__ Spans sp;
    __shared__ int32_t n_keep;
    const int half = threadIdx.x & 1;
    const F32Item it = f32_item<PAD>(a, sp, n_keep);
    const RowInfo& ri = it.ri;  // the key row
    float kv[H2], vv[H2], ak[H2], av[H2];
    const float* kr = f32_row(a.k, a.k_sb, a.k_sh, a.k_sr, it.bb, it.hh, ri.qseq, half, D);
    const float* vr = f32_row(a.v, a.v_sb, a.v_sh, a.v_sr, it.bb, it.hh, ri.qseq, half, D);
#pragma unroll
    for (int e = 0; e < H2; ++e) {
        kv[e] = kr[e];
        vv[e] = vr[e];
        ak[e] = 0.f;
        av[e] = 0.f;
    }
    const float c = a.scale_log2;
    const ItemList& L = it.L;
    for (int32_t v = 0; v < L.total; ++v) {
        const int32_t seq = list_seq(v, L.b1, L.b2, L.b3, L.s0, L.sa, L.sb, sp);  // a query row
        const int32_t inf = entry_info<PAD>(a, L, v, seq, it.o, sp);
        const float* qr = f32_row(a.q, a.q_sb, a.q_sh, a.q_sr, it.bb, it.hh, seq, half, D);
        const float* dr = f32_row(g.dout, a.o_sb, a.o_sh, a.o_sr, it.bb, it.hh, seq, half, D);
        const int64_t row = (int64_t)it.bh * a.n_tot + seq;
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int e = 0; e < H2; ++e) {
            s = fmaf(qr[e], kv[e], s);
            dp = fmaf(dr[e], vv[e], dp);
        }
        s += __shfl_xor(s, 1);
        dp += __shfl_xor(dp, 1);
        const bool ok = inf == kKeyAll || inf == ri.label;
        const float p = ok ? exp2f(fmaf(s, c, -g.lse2[row])) : 0.f;
        const float ds = p * (dp - g.delta[row]);
#pragma unroll
        for (int e = 0; e < H2; ++e) {
            av[e] = fmaf(p, dr[e], av[e]);
            ak[e] = fmaf(ds, qr[e], ak[e]);
        }
    }
    if (!ri.store) return;
    const float mk = c * 0.69314718055994530942f;
    float* ok_ = static_cast<float*>(g.dk) + it.bb * a.k_sb + it.hh * a.k_sh + (int64_t)ri.qseq * a.k_sr + half * H2;
    float* ov = static_cast<float*>(g.dv) + it.bb * a.v_sb + it.hh * a.v_sh + (int64_t)ri.qseq * a.v_sr + half * H2;
#pragma unroll
    for (int e = 0; e < H2; ++e) {
        ok_[e] = ri.pad ? 0.f : ak[e] * mk;
        ov[e] = ri.pad ? 0.f : av[e];
    }
}

template <int D>
hipError_t launch_bwd_f32_t(const AttnArgs& a, const BwdArgs& g, hipStream_t s) {
    if (a.n_chunks != 1) return hipErrorInvalidValue;  // dense rows are never split here
    const int64_t rows = (int64_t)a.n_bh * a.n_tot;
    const int64_t pblocks = (rows + 255) / 256;
    if (pblocks > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((bwd_prep_f32_kernel<D>), dim3((unsigned)pblocks), dim3(256), 0, s, a, g);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (a.padded) {
        hipLaunchKernelGGL((bwd_dq_f32_kernel<D, true>), dim3(a.total_items), dim3(kThreads), 0, s, a, g);
        hipLaunchKernelGGL((bwd_dkdv_f32_kernel<D, true>), dim3(a.total_items), dim3(kThreads), 0, s, a, g);
    } else {
        hipLaunchKernelGGL((bwd_dq_f32_kernel<D, false>), dim3(a.total_items), dim3(kThreads), 0, s, a, g);
        hipLaunchKernelGGL((bwd_dkdv_f32_kernel<D, false>), dim3(a.total_items), dim3(kThreads), 0, s, a, g);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bwd_f32(const AttnArgs& a, const BwdArgs& g, int head_dim, hipStream_t s) {
    if (a.total_items == 0) return hipSuccess;
    return head_dim == 128 ? launch_bwd_f32_t<128>(a, g, s) : launch_bwd_f32_t<64>(a, g, s);
}

}  // namespace hilberta
