// HilbertA attention, fp32 path and the merge of split key chunks
// (§3.2-§3.4, Appendix A, Algorithm 1), for gfx950.
//
// fp32 mode computes everything in fp32 (no reduced-precision matrix
// arithmetic) and exists for tight parity with the float64 oracle.  A
// workgroup of four wavefronts owns 128 query rows (32 per wavefront) and
// streams keys through LDS in double-buffered stages of 64, the next stage
// prefetched into registers while the current one is consumed.  Per stage,
//   S^T = K Q^T   on v_mfma_f32_32x32x2_f32, so every lane holds one query
//                 row and 32 of the 64 keys: the online softmax (Algorithm
//                 1's attn_inner: running max m, sum l, accumulator) is per
//                 lane, with one exchange between the two lane halves;
//   O^T += V^T P^T, P^T fed straight from the score registers: the MFMA's
//                 reduction index may enumerate keys in any order, so each
//                 step pairs the keys the two lane halves hold in one score
//                 register.
// The bf16 path lives in attn_bf16.hip; the work items, key segments and
// masks are shared (attn_common.hpp).
#include "attn_common.hpp"

namespace hilberta {
namespace {

constexpr int kBN = 64;  // keys per stage

template <int D>
struct alignas(16) StageF32 {
    alignas(16) float k[2][kBN][D + 1];
    alignas(16) float v[2][kBN][D + 4];
    alignas(16) int32_t info[2][kBN];
};

template <int D>
struct LoaderF32 {
    static constexpr int CH = D / 4;                 // 16-byte chunks per row
    static constexpr int PT = kBN * CH / kThreads;   // per thread, each of K and V
    f32x4 kr[PT];
    f32x4 vr[PT];
    int32_t info;
    __amdgpu_buffer_rsrc_t krs, vrs;
    int32_t krow_b, vrow_b;

    __device__ __forceinline__ static int row_of(int tid, int j) { return (tid + kThreads * j) / CH; }
    __device__ __forceinline__ static int colb_of(int tid, int j) { return ((tid + kThreads * j) % CH) * 16; }

    __device__ __forceinline__ void init(const float* kb, const float* vb, const AttnArgs& a) {
        krs = slice_rsrc(kb, a.n_tot, a.k_sr, D, 4);
        vrs = slice_rsrc(vb, a.n_tot, a.v_sr, D, 4);
        krow_b = (int32_t)(a.k_sr * 4);
        vrow_b = (int32_t)(a.v_sr * 4);
    }

    __device__ __forceinline__ void load(const Block& b, MaskCtx it, const AttnArgs& a,
                                         const Spans& sp, int tid, int32_t n_shared) {
#pragma unroll
        for (int j = 0; j < PT; ++j) {
            const int row = row_of(tid, j);
            int32_t ko, vo;
            if (b.kind != SEG_SHARED) {
                ko = (b.base + row) * krow_b;
                vo = (b.base + row) * vrow_b;
            } else {
                const int32_t seq = sp.map[min(b.first + row, n_shared - 1)];
                ko = seq * krow_b;
                vo = seq * vrow_b;
            }
            kr[j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(krs, ko + colb_of(tid, j), 0, 0));
            vr[j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(vrs, vo + colb_of(tid, j), 0, 0));
        }
        if (tid < kBN) info = b.fast ? kKeyAll : key_info(b, tid, key_seq(b, tid, sp), it, a, sp);
    }

    __device__ __forceinline__ void store(StageF32<D>& st, int buf, int tid) const {
#pragma unroll
        for (int j = 0; j < PT; ++j) {
            const int row = row_of(tid, j), col = colb_of(tid, j) / 4;
            float* kd = &st.k[buf][row][col];
            kd[0] = kr[j][0];
            kd[1] = kr[j][1];
            kd[2] = kr[j][2];
            kd[3] = kr[j][3];
            *reinterpret_cast<f32x4*>(&st.v[buf][row][col]) = vr[j];
        }
        if (tid < kBN) st.info[buf][tid] = info;
    }
};

template <int D>
struct SmemF32 {
    StageF32<D> st;
    Spans sp;
};

template <int D>
__global__ void __launch_bounds__(kThreads, 1) attn_f32_kernel(AttnArgs a) {
    __shared__ SmemF32<D> sm;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int h = lane >> 5;
    const int ql = lane & 31;

    const ItemId id = decode_item(blockIdx.x, a);
    const int32_t bh = id.bh;
    const int32_t r = id.r;
    const int32_t dense_items = a.dense_row_blocks * a.n_chunks;
    const bool dense = r < dense_items;
    MaskCtx mc{0, 0, 0, 0};
    mc.o = load_spans<kThreads>(a, sm.sp, tid);
    const int32_t n_shared = a.sparse ? sm.sp.cum[sm.sp.n] : 0;
    const int32_t chunk = dense ? r % a.n_chunks : 0;
    const int32_t row0 = dense ? (r / a.n_chunks) * kBlockM : (r - dense_items) * kBlockM;
    const Segs g = item_segments<kBN>(a, dense, chunk, row0, kBlockM, n_shared, mc);
    const int32_t lm = mc.label_mask | (a.padded ? 2 : 0);
    const RowInfo ri = row_info(a, dense, row0, wave * 32 + ql, kBlockM, mc.o, n_shared, sm.sp);

    const int32_t bb = bh / a.heads;
    const int32_t hh = bh - bb * a.heads;
    const float* qrow = reinterpret_cast<const float*>(a.q) + bb * a.q_sb + hh * a.q_sh + (int64_t)ri.qseq * a.q_sr;
    const float* kb = reinterpret_cast<const float*>(a.k) + bb * a.k_sb + hh * a.k_sh;
    const float* vb = reinterpret_cast<const float*>(a.v) + bb * a.v_sb + hh * a.v_sh;
    float q[D / 2];  // Q[row][2 kc + h]: the B operand of S^T = K Q^T
#pragma unroll
    for (int kc = 0; kc < D / 2; ++kc) q[kc] = qrow[2 * kc + h];

    f32x16 acc[D / 32];
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) acc[dt] = f32x16{};
    float m_run = -INFINITY;  // running max of the scaled logits, log2 units
    float l_run = 0.f;        // this lane's share of the running sum
    const float c = a.scale_log2;

    // Stage i is consumed from LDS buffer i&1.  At the top of iteration i the
    // registers hold stage i+1; they go to the other buffer and stage i+2 is
    // requested, so its loads are in flight while stage i is computed.
    LoaderF32<D> ld;
    ld.init(kb, vb, a);
    const int nblk = g.e3;
    ld.load(BLOCK_AT(kBN, 0, g, lm), mc, a, sm.sp, tid, n_shared);
    ld.store(sm.st, 0, tid);
    if (nblk > 1) ld.load(BLOCK_AT(kBN, 1, g, lm), mc, a, sm.sp, tid, n_shared);
    __syncthreads();
    for (int i = 0; i < nblk; ++i) {
        const int buf = i & 1;
        if (i + 1 < nblk) ld.store(sm.st, buf ^ 1, tid);
        if (i + 2 < nblk) ld.load(BLOCK_AT(kBN, i + 2, g, lm), mc, a, sm.sp, tid, n_shared);
        const Block b = BLOCK_AT(kBN, i, g, lm);
        // S^T: s[kt] holds keys 32 kt + 8 (e/4) + 4 h + e%4 against this row
        f32x16 s[2];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            f32x16 t = {};
#pragma unroll
            for (int kc = 0; kc < D / 2; ++kc)
                t = __builtin_amdgcn_mfma_f32_32x32x2f32(sm.st.k[buf][32 * kt + ql][2 * kc + h], q[kc], t, 0, 0, 0);
            s[kt] = t;
        }
        if (!b.fast) {
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int32_t inf = sm.st.info[buf][32 * kt + 8 * (e >> 2) + 4 * h + (e & 3)];
                    s[kt][e] = (inf == kKeyAll || inf == ri.label) ? s[kt][e] : -INFINITY;
                }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[kt][e]);
        mx = half_max(mx) * c;
        if (mx > m_run) {
            // exact running max in fp32 mode
            const float alpha = __builtin_amdgcn_exp2f(m_run - mx);
            m_run = mx;
            l_run *= alpha;
#pragma unroll
            for (int dt = 0; dt < D / 32; ++dt) acc[dt] *= alpha;
        }
        const float m_use = m_run == -INFINITY ? 0.f : m_run;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                s[kt][e] = __builtin_amdgcn_exp2f(fmaf(s[kt][e], c, -m_use));
                l_run += s[kt][e];
            }
        // O^T += V^T P^T; the two lane halves supply keys 4 apart
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const float v = sm.st.v[buf][32 * kt + 8 * (e >> 2) + 4 * h + (e & 3)][32 * dt + ql];
                    acc[dt] = __builtin_amdgcn_mfma_f32_32x32x2f32(v, s[kt][e], acc[dt], 0, 0, 0);
                }
        __syncthreads();
    }

    float* obase = reinterpret_cast<float*>(a.o) + bb * a.o_sb + hh * a.o_sh;
    store_row<float, D>(a, ri, bh, chunk, dense, h, m_run, l_run, acc, obase);
}

// Merge of the split key chunks of dense rows: with chunk partials
// (acc_c, m_c, l_c), M = max m_c, L = sum l_c 2^(m_c - M) and
// O = sum acc_c 2^(m_c - M) / L -- the same rescaling Algorithm 1 applies
// between key blocks, taken here chunk by chunk as an online merge.  A row
// is handled by D/4 lanes, each owning four consecutive elements (16-byte
// loads); every lane reads the (m, l) of every chunk itself (the lanes of a
// row read the same words), so no cross-lane step waits between the loads:
// the partials of four chunks are requested at once, non-temporal.
template <typename T, int D>
__global__ void __launch_bounds__(256) merge_kernel(MergeArgs m) {
    typedef float f4 __attribute__((ext_vector_type(4)));
    constexpr int LPR = D / 4;  // lanes per row
    constexpr int RPB = 256 / LPR;
    constexpr int CH = 4;       // chunks in flight
    const int sub = threadIdx.x % LPR;
    const int64_t rowid = (int64_t)blockIdx.x * RPB + threadIdx.x / LPR;
    if (rowid >= (int64_t)m.n_bh * m.n_dense_rows) return;
    const int32_t bh = (int32_t)(rowid / m.n_dense_rows);
    const int32_t r = (int32_t)(rowid - (int64_t)bh * m.n_dense_rows);
    int32_t seq = r;
    if (m.sparse && r >= m.n_txt) {
        const int32_t n_sp = min(max(m.sched[6], 0), min(m.span_cap, kMaxSpans));
        const int32_t* tab = m.sched + 12 + 4 * m.n_tiles;
        int32_t u = r - m.n_txt;
        seq = -1;
        for (int32_t s = 0; s < n_sp; ++s) {
            const int32_t st0 = min(max(tab[2 * s], m.n_txt), m.n_tot);
            const int32_t ln = min(max(tab[2 * s + 1], 0), m.n_tot - st0);
            if (u < ln) {
                seq = st0 + u;
                break;
            }
            u -= ln;
        }
        if (seq < 0) return;
    }
    const float* ml = m.ws + (int64_t)m.n_bh * m.n_chunks * m.n_dense_rows * D;
    const int64_t slot0 = (int64_t)bh * m.n_chunks * m.n_dense_rows + r;
    float M = -INFINITY, L = 0.f;
    f4 o = {0.f, 0.f, 0.f, 0.f};
    for (int32_t c0 = 0; c0 < m.n_chunks; c0 += CH) {
        float mc[CH], lc[CH];
        f4 part[CH];
#pragma unroll
        for (int k = 0; k < CH; ++k) {
            mc[k] = -INFINITY;
            lc[k] = 0.f;
            part[k] = f4{0.f, 0.f, 0.f, 0.f};
            if (c0 + k < m.n_chunks) {
                const int64_t slot = slot0 + (int64_t)(c0 + k) * m.n_dense_rows;
                mc[k] = ml[slot * 2];
                lc[k] = ml[slot * 2 + 1];
                part[k] = __builtin_nontemporal_load(reinterpret_cast<const f4*>(m.ws + slot * D) + sub);
            }
        }
#pragma unroll
        for (int k = 0; k < CH; ++k) {
            // a chunk (or the running sum) with m = -inf carries weight 0
            const float mn = fmaxf(M, mc[k]);
            const float mu = mn == -INFINITY ? 0.f : mn;
            const float wa = __builtin_amdgcn_exp2f(M - mu), wb = __builtin_amdgcn_exp2f(mc[k] - mu);
            L = L * wa + lc[k] * wb;
            o = o * wa + part[k] * wb;
            M = mn;
        }
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    const int32_t b = bh / m.heads, hh = bh - b * m.heads;
    T* orow = reinterpret_cast<T*>(m.o) + b * m.o_sb + hh * m.o_sh + (int64_t)seq * m.o_sr;
    store4<T>(orow + 4 * sub, o[0] * inv, o[1] * inv, o[2] * inv, o[3] * inv);
    if (m.lse && sub == 0)
        m.lse[(int64_t)bh * m.n_tot + seq] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
}
template <int D>
hipError_t launch_f32(const AttnArgs& a, hipStream_t s) {
    hipLaunchKernelGGL((attn_f32_kernel<D>), dim3(a.total_items), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_merge_t(const MergeArgs& m, hipStream_t s) {
    const int64_t rows = (int64_t)m.n_bh * m.n_dense_rows;
    constexpr int64_t rpb = 256 / (D / 4);
    const int64_t blocks = (rows + rpb - 1) / rpb;
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((merge_kernel<T, D>), dim3((unsigned)blocks), dim3(256), 0, s, m);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn(const AttnArgs& a, int dtype, int head_dim, hipStream_t s) {
    if (a.total_items == 0) return hipSuccess;
    if (dtype == 1) return launch_attn_bf16(a, head_dim, s);
    return head_dim == 128 ? launch_f32<128>(a, s) : launch_f32<64>(a, s);
}

hipError_t launch_merge(const MergeArgs& m, int dtype, int head_dim, hipStream_t s) {
    if (dtype == 1) return head_dim == 128 ? launch_merge_t<__bf16, 128>(m, s) : launch_merge_t<__bf16, 64>(m, s);
    return head_dim == 128 ? launch_merge_t<float, 128>(m, s) : launch_merge_t<float, 64>(m, s);
}

}  // namespace hilberta
