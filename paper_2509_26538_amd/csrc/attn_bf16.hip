// HilbertA attention, bf16 path (§3.2-§3.4, Appendix A, Algorithm 1), for
// gfx950: bf16 inputs, fp32 accumulation and softmax state, P rounded to
// bf16 for the PV product, bf16 output.
//
// A workgroup of four wavefronts owns 128 query rows (32 per wavefront); two
// workgroups share a CU, so each SIMD interleaves two wavefronts.  Keys
// stream through LDS in double-buffered stages of 64, the next stage staged
// through registers with bounds-checked buffer loads while the current one
// is consumed.  Per stage each wavefront computes
//   S^T = K Q^T    on v_mfma_f32_32x32x16_bf16: every lane holds one query
//                  row and 32 of the 64 keys, so the online softmax state
//                  (Algorithm 1's attn_inner: max m, sum l, accumulator) is
//                  per lane; the two lane halves meet through
//                  v_permlane32_swap;
//   O^T += V^T P^T with P^T straight from the score registers.  The MFMA
//                  reduction index may enumerate the 16 keys of a chunk in
//                  any order, so V^T is staged in LDS in exactly the key
//                  order the score registers hold.
// The reference max moves only when a row max grows by more than 2^8 (acc
// and l share it, so it cancels in acc / l).
#include "attn_common.hpp"

namespace hilberta {
namespace {

constexpr int kBN2 = 64;  // keys per stage
static_assert(kBlockMBf16 == 128, "four wavefronts of 32 rows");

template <int D>
struct alignas(16) Stage2 {
    alignas(16) uint16_t k[2][kBN2][D + 8];   // K rows (pitch an odd multiple of 16 B)
    alignas(16) uint16_t vt[2][D][kBN2 + 8];  // V^T, keys in score-register order
    alignas(16) int32_t info[2][kBN2];
};

template <int D>
struct Smem2 {
    Stage2<D> st;
    Spans sp;
};

template <int D>
struct Loader2 {
    static constexpr int KCH = D / 8;                     // 16-byte chunks per K row
    static constexpr int KPT = kBN2 * KCH / kThreads;     // K chunks per thread
    static constexpr int VQ = D / 4;                      // 4-element quads per V row
    static constexpr int VUNITS = 8 * VQ;                 // (8-key group, quad) pairs
    u32x4 kr[KPT];
    u32x2 vr[8];
    int32_t info;
    __amdgpu_buffer_rsrc_t krs, vrs;
    int32_t krow_b, vrow_b;

    // K piece j: row (tid + 256 j) / KCH, chunk (tid + 256 j) % KCH.
    __device__ __forceinline__ static int k_row(int tid, int j) { return (tid + kThreads * j) / KCH; }
    __device__ __forceinline__ static int k_colb(int tid, int j) { return ((tid + kThreads * j) % KCH) * 16; }
    // V group g = tid / VQ = 2 cc + hh covers keys 16 cc + 8 (j/4) + 4 hh +
    // j%4 (j < 8), which land in the eight consecutive slots 16 cc + 8 hh + j;
    // quad dq = tid % VQ.
    __device__ __forceinline__ static int v_row(int tid, int j) {
        const int g = tid / VQ, cc = g >> 1, hh = g & 1;
        return 16 * cc + 8 * (j >> 2) + 4 * hh + (j & 3);
    }
    __device__ __forceinline__ static int v_colb(int tid) { return (tid % VQ) * 8; }

    __device__ __forceinline__ void init(const __bf16* kb, const __bf16* vb, const AttnArgs& a) {
        krs = slice_rsrc(kb, a.n_tot, a.k_sr, D, 2);
        vrs = slice_rsrc(vb, a.n_tot, a.v_sr, D, 2);
        krow_b = (int32_t)(a.k_sr * 2);
        vrow_b = (int32_t)(a.v_sr * 2);
    }

    __device__ __forceinline__ void load(const Block& b, MaskCtx it, const AttnArgs& a,
                                         const Spans& sp, int tid, int32_t n_shared) {
        if (b.kind != SEG_SHARED) {
            const int32_t ks = b.base * krow_b, vs = b.base * vrow_b;
#pragma unroll
            for (int j = 0; j < KPT; ++j)
                kr[j] = __builtin_amdgcn_raw_buffer_load_b128(krs, ks + k_row(tid, j) * krow_b + k_colb(tid, j), 0, 0);
            if (tid < VUNITS) {
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    vr[j] = __builtin_amdgcn_raw_buffer_load_b64(vrs, vs + v_row(tid, j) * vrow_b + v_colb(tid), 0, 0);
            }
        } else {
            // gathered shared keys: one map lookup per staged row
#pragma unroll
            for (int j = 0; j < KPT; ++j) {
                const int32_t seq = sp.map[min(b.first + k_row(tid, j), n_shared - 1)];
                kr[j] = __builtin_amdgcn_raw_buffer_load_b128(krs, seq * krow_b + k_colb(tid, j), 0, 0);
            }
            if (tid < VUNITS) {
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int32_t seq = sp.map[min(b.first + v_row(tid, j), n_shared - 1)];
                    vr[j] = __builtin_amdgcn_raw_buffer_load_b64(vrs, seq * vrow_b + v_colb(tid), 0, 0);
                }
            }
        }
        if (tid < kBN2) info = b.fast ? kKeyAll : key_info(b, tid, key_seq(b, tid, sp), it, a, sp);
    }

    __device__ __forceinline__ void store(Stage2<D>& st, int buf, int tid) const {
#pragma unroll
        for (int j = 0; j < KPT; ++j)
            *reinterpret_cast<u32x4*>(&st.k[buf][k_row(tid, j)][k_colb(tid, j) / 2]) = kr[j];
        if (tid < VUNITS) {
            const int dq = tid % VQ, g = tid / VQ;
            const int cc = g >> 1, hh = g & 1;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                // element e of each of the 8 keys; key j goes to slot j
                const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
                u32x4 w;
#pragma unroll
                for (int j = 0; j < 8; j += 2)
                    w[j >> 1] = __builtin_amdgcn_perm(vr[j + 1][e >> 1], vr[j][e >> 1], sel);
                *reinterpret_cast<u32x4*>(&st.vt[buf][4 * dq + e][16 * cc + 8 * hh]) = w;
            }
        }
        if (tid < kBN2) st.info[buf][tid] = info;
    }
};

template <int D>
__global__ void __launch_bounds__(kThreads, 2) attn_bf16_kernel(AttnArgs a) {
    __shared__ Smem2<D> sm;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int h = lane >> 5;
    const int ql = lane & 31;

    const int item = remap_xcd(blockIdx.x, a.total_items);
    const int32_t bh = item / a.items_per_bh;
    const int32_t r = item - bh * a.items_per_bh;
    const int32_t dense_items = a.dense_row_blocks * a.n_chunks;
    const bool dense = r < dense_items;
    MaskCtx mc{0, 0, 0, 0};
    mc.o = load_spans<kThreads>(a, sm.sp, tid);
    const int32_t n_shared = a.sparse ? sm.sp.cum[sm.sp.n] : 0;
    const int32_t chunk = dense ? r % a.n_chunks : 0;
    const int32_t row0 = dense ? (r / a.n_chunks) * kBlockMBf16 : (r - dense_items) * kBlockMBf16;
    const Segs g = item_segments<kBN2>(a, dense, chunk, row0, kBlockMBf16, n_shared, mc);
    const RowInfo ri = row_info(a, dense, row0, wave * 32 + ql, kBlockMBf16, mc.o, n_shared, sm.sp);

    const int32_t bb = bh / a.heads;
    const int32_t hh = bh - bb * a.heads;
    const __bf16* qrow = reinterpret_cast<const __bf16*>(a.q) + bb * a.q_sb + hh * a.q_sh + (int64_t)ri.qseq * a.q_sr;
    const __bf16* kbase = reinterpret_cast<const __bf16*>(a.k) + bb * a.k_sb + hh * a.k_sh;
    const __bf16* vbase = reinterpret_cast<const __bf16*>(a.v) + bb * a.v_sb + hh * a.v_sh;
    // Q as the B operand of S^T = K Q^T: Q[row][16 kc + 8 h .. + 8]
    bf16x8 q[D / 16];
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) q[kc] = *reinterpret_cast<const bf16x8*>(qrow + 16 * kc + 8 * h);

    f32x16 acc[D / 32];
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) acc[dt] = f32x16{};
    float m_run = -INFINITY;  // reference max of the scaled logits, log2 units
    float l_run = 0.f;        // this lane's share of the running sum
    const float c = a.scale_log2;

    // Stage i is consumed from LDS buffer i&1.  At the top of iteration i the
    // registers hold stage i+1; they go to the other buffer and stage i+2 is
    // requested, so its loads are in flight while stage i is computed.
    Loader2<D> ld;
    ld.init(kbase, vbase, a);
    const int nblk = g.e3;
    ld.load(BLOCK_AT(kBN2, 0, g, mc.label_mask), mc, a, sm.sp, tid, n_shared);
    ld.store(sm.st, 0, tid);
    if (nblk > 1) ld.load(BLOCK_AT(kBN2, 1, g, mc.label_mask), mc, a, sm.sp, tid, n_shared);
    __syncthreads();
    for (int i = 0; i < nblk; ++i) {
        const int buf = i & 1;
        if (i + 1 < nblk) ld.store(sm.st, buf ^ 1, tid);
        if (i + 2 < nblk) ld.load(BLOCK_AT(kBN2, i + 2, g, mc.label_mask), mc, a, sm.sp, tid, n_shared);
        const Block b = BLOCK_AT(kBN2, i, g, mc.label_mask);
        // S^T: s[kt] register e holds key 32 kt + 8 (e/4) + 4 h + e%4
        f32x16 s[2];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            f32x16 t = {};
#pragma unroll
            for (int kc = 0; kc < D / 16; ++kc) {
                const bf16x8 k = *reinterpret_cast<const bf16x8*>(&sm.st.k[buf][32 * kt + ql][16 * kc + 8 * h]);
                t = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k, q[kc], t, 0, 0, 0);
            }
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
        if (__builtin_amdgcn_ballot_w64(mx > m_run + 8.f)) {
            const float m_new = fmaxf(m_run, mx);
            // a row with every key masked so far keeps -inf: leave it alone
            const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            l_run *= alpha;
#pragma unroll
            for (int dt = 0; dt < D / 32; ++dt) acc[dt] *= alpha;
        }
        const float m_use = m_run == -INFINITY ? 0.f : m_run;
        // P = exp2(S c - m), rounded to bf16 for the PV product; chunk cc of
        // 16 keys holds key 16 cc + 8 (j/4) + 4 h + j%4 in register j, i.e.
        // V^T slot 16 cc + 8 h + j
        bf16x8 p[4];
#pragma unroll
        for (int cc = 0; cc < 4; ++cc)
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float pe = __builtin_amdgcn_exp2f(fmaf(s[cc >> 1][8 * (cc & 1) + j], c, -m_use));
                l_run += pe;
                p[cc][j] = (__bf16)pe;
            }
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
            for (int cc = 0; cc < 4; ++cc) {
                const bf16x8 v = *reinterpret_cast<const bf16x8*>(&sm.st.vt[buf][32 * dt + ql][16 * cc + 8 * h]);
                acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v, p[cc], acc[dt], 0, 0, 0);
            }
        __syncthreads();
    }

    __bf16* obase = reinterpret_cast<__bf16*>(a.o) + bb * a.o_sb + hh * a.o_sh;
    store_row<__bf16, D>(a, ri, bh, chunk, dense, h, m_run, l_run, acc, obase);
}

template <int D>
hipError_t launch_t(const AttnArgs& a, hipStream_t s) {
    hipLaunchKernelGGL((attn_bf16_kernel<D>), dim3(a.total_items), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bf16(const AttnArgs& a, int head_dim, hipStream_t s) {
    return head_dim == 128 ? launch_t<128>(a, s) : launch_t<64>(a, s);
}

}  // namespace hilberta
