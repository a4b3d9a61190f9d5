// HilbertA attention backward, bf16: the gradients of the forward's masked
// softmax attention (§3.2-§3.4, Appendix A), by the chain rule.  With
// S = s Q K^T (masked), P = exp(S - LSE) the forward's probabilities, dO
// the gradient of O:
//   Dlt_i = dO_i . O_i,   dP = dO V^T,   dS = P (dP - Dlt),
//   dV = P^T dO,          dK = s dS^T Q,   dQ = s dS K.
// bf16 inputs and gradients, fp32 MFMA accumulation, P and dS rounded to
// bf16 as MFMA operands.  The launches:
//   bwd_prep_kernel  Dlt and the LSE in log2 units, one per row;
//   bwd_dq_kernel    the forward's query items and key lists: per stage
//                    S^T = K Q^T and dP^T = V dO^T with the keys as A
//                    operands, P and dS per lane (one query row per lane),
//                    dQ^T += K^T dS^T with K read transposed;
//   bwd_dkdv_kernel  key items: the list of a key block is the queries that
//                    attend it, built as a query block's key list (the mask
//                    is symmetric); S = Q K^T and dP = dO V^T with the
//                    queries as A operands (one key row per lane), then
//                    dV^T += dO^T P and dK^T += Q^T dS with Q and dO read
//                    transposed;
//   bwd_sum_kernel   after each pass, when rows are split over key (query)
//                    chunks: the sum of the chunk partials.
// No atomics: every gradient row is written once by the item that owns it,
// so the results are deterministic.  Rows that attend every key (text and
// shared rows) and keys every query attends are items of their own over the
// whole sequence.  Each stage tensor is staged once through LDS by direct
// loads, in the fk layout, whose swizzle keeps both its whole-row reads (A
// operands) and its transposing reads (Q, dO and K are read both ways)
// free of bank conflicts.
// Stages hold 32 list rows, so that two workgroups fit a CU (64-row stages
// would take 82 KB of LDS per workgroup and more than 256 registers per lane
// in the dK/dV pass) and each SIMD interleaves two wavefronts.
#include "bf16_stage.hpp"

#include <type_traits>

namespace hilberta {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

// Dlt_i = dO_i . O_i in fp32 and lse2_i = LSE_i log2(e) (0 for a row that
// attends nothing, whose probabilities are all masked anyway).  D/8 lanes
// per row, eight elements (one 16-byte load of each tensor) each; a block
// covers kPrepPasses groups of 256/(D/8) consecutive rows and requests all
// of their loads before the first sum.
constexpr int kPrepPasses = 4;

template <int D>
__global__ void __launch_bounds__(256) bwd_prep_kernel(AttnArgs a, BwdArgs g) {
    constexpr int LPR = D / 8;
    constexpr int RPP = 256 / LPR;
    typedef __bf16 bf16x8v __attribute__((ext_vector_type(8)));
    const int sub = threadIdx.x % LPR;
    const int64_t rows = (int64_t)a.n_bh * a.n_tot;
    const int64_t first = (int64_t)blockIdx.x * (RPP * kPrepPasses) + threadIdx.x / LPR;
    bf16x8v o8[kPrepPasses], d8[kPrepPasses];
#pragma unroll
    for (int u = 0; u < kPrepPasses; ++u) {
        const int64_t rowid = first + u * RPP;
        const int64_t r = rowid < rows ? rowid : 0;
        const int64_t bh = r / a.n_tot, n = r - bh * a.n_tot;
        const int64_t b = bh / a.heads, hh = bh - b * a.heads;
        const int64_t off = b * a.o_sb + hh * a.o_sh + n * a.o_sr + 8 * sub;
        o8[u] = *reinterpret_cast<const bf16x8v*>(reinterpret_cast<const __bf16*>(a.o) + off);
        d8[u] = *reinterpret_cast<const bf16x8v*>(reinterpret_cast<const __bf16*>(g.dout) + off);
    }
#pragma unroll
    for (int u = 0; u < kPrepPasses; ++u) {
        float t = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) t += (float)o8[u][e] * (float)d8[u][e];
#pragma unroll
        for (int w = LPR / 2; w > 0; w >>= 1) t += __shfl_xor(t, w, LPR);
        const int64_t r = first + u * RPP;
        if (r < rows && sub == 0) {
            g.delta[r] = t;
            const float l = g.lse[r];
            g.lse2[r] = l == -INFINITY ? 0.f : l * 1.4426950408889634f;
        }
    }
}

// One lane's gradient row, scaled by mul; a padding slot (zero) is written
// as zeros by selection, never as acc * 0: a padding row's sums may hold
// inf or NaN (its probabilities are not masked, and the caller may fill the
// slot with anything finite), and inf * 0 is NaN.
template <int D>
__device__ __forceinline__ void store_grad(__bf16* row, const f32x16 acc[D / 32], float mul, bool zero, int h) {
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int q = 0; q < 4; ++q)
            store4<__bf16>(row + 32 * dt + 8 * q + 4 * h, zero ? 0.f : acc[dt][4 * q] * mul,
                           zero ? 0.f : acc[dt][4 * q + 1] * mul, zero ? 0.f : acc[dt][4 * q + 2] * mul,
                           zero ? 0.f : acc[dt][4 * q + 3] * mul);
}

// Rows that attend every key (dQ) and keys every query attends (dK, dV) are
// split into key (query) chunks like the forward's dense rows.  Chunk c of
// dense row r writes its unscaled sums to ws[((bh C + c) R + r) 2 + t][D]
// (t = 0: dQ or dK, 1: dV), and bwd_sum_kernel adds the chunks up.
template <int D>
__device__ __forceinline__ void store_partial(const AttnArgs& a, int32_t bh, int32_t chunk, int32_t dense_row,
                                              int t, const f32x16 acc[D / 32], int h) {
    if (dense_row < 0 || dense_row >= a.n_dense_rows) return;
    const int64_t slot = ((int64_t)bh * a.n_chunks + chunk) * a.n_dense_rows + dense_row;
    float* w = a.ws + (slot * 2 + t) * D;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int q = 0; q < 4; ++q)
            *reinterpret_cast<f4*>(w + 32 * dt + 8 * q + 4 * h) =
                f4{acc[dt][4 * q], acc[dt][4 * q + 1], acc[dt][4 * q + 2], acc[dt][4 * q + 3]};
}

// Sum of the chunk partials of every dense row: dQ (pass 0) or dK and dV
// (pass 1), scaled and written in bf16 at the row's sequence position (text
// rows first, then the shared runs of the schedule table).  D/4 lanes per
// row, four elements each.
template <int D>
__global__ void __launch_bounds__(256) bwd_sum_kernel(AttnArgs a, BwdArgs g, int pass) {
    constexpr int LPR = D / 4;
    constexpr int RPB = 256 / LPR;
    const int sub = threadIdx.x % LPR;
    const int64_t rowid = (int64_t)blockIdx.x * RPB + threadIdx.x / LPR;
    if (rowid >= (int64_t)a.n_bh * a.n_dense_rows) return;
    const int32_t bh = (int32_t)(rowid / a.n_dense_rows);
    const int32_t r = (int32_t)(rowid - (int64_t)bh * a.n_dense_rows);
    int32_t seq = r;
    if (a.sparse && r >= a.n_txt) {
        const int32_t n_sp = min(max(a.sched[6], 0), min(a.span_cap, kMaxSpans));
        const int32_t* tab = a.sched + 12 + 4 * a.n_tiles;
        int32_t u = r - a.n_txt;
        seq = -1;
        for (int32_t s = 0; s < n_sp; ++s) {
            const int32_t st0 = min(max(tab[2 * s], a.n_txt), a.n_tot);
            const int32_t ln = min(max(tab[2 * s + 1], 0), a.n_tot - st0);
            if (u < ln) {
                seq = st0 + u;
                break;
            }
            u -= ln;
        }
        if (seq < 0) return;
    }
    const int32_t b = bh / a.heads, hh = bh - b * a.heads;
    const float scale = a.scale_log2 * 0.69314718055994530942f;
    for (int t = 0; t < (pass == 0 ? 1 : 2); ++t) {
        f4 acc = {0.f, 0.f, 0.f, 0.f};
        for (int32_t c = 0; c < a.n_chunks; ++c) {
            const int64_t slot = ((int64_t)bh * a.n_chunks + c) * a.n_dense_rows + r;
            acc += __builtin_nontemporal_load(reinterpret_cast<const f4*>(a.ws + (slot * 2 + t) * D) + sub);
        }
        __bf16* dst;
        float mul = scale;
        if (pass == 0) {
            dst = reinterpret_cast<__bf16*>(g.dq) + b * a.q_sb + hh * a.q_sh + (int64_t)seq * a.q_sr;
        } else if (t == 0) {
            dst = reinterpret_cast<__bf16*>(g.dk) + b * a.k_sb + hh * a.k_sh + (int64_t)seq * a.k_sr;
        } else {
            dst = reinterpret_cast<__bf16*>(g.dv) + b * a.v_sb + hh * a.v_sh + (int64_t)seq * a.v_sr;
            mul = 1.f;
        }
        store4<__bf16>(dst + 4 * sub, acc[0] * mul, acc[1] * mul, acc[2] * mul, acc[3] * mul);
    }
}

// ---------------------------------------------------------------------- dQ
constexpr int kBQ = 32;  // list rows per stage

template <int D>
struct SmemDq {
    static constexpr int SB = kBQ * Geo<D>::ROWB;
    alignas(16) uint8_t k[2][SB];   // fk: A operand of S^T, transposed A operand of dQ^T
    alignas(16) uint8_t v[2][SB];   // fk: A operand of dP^T
    alignas(16) int32_t info[2][kBQ];
    Spans sp;
    int32_t n_keep;
    int32_t slow[2];
};

template <int D, bool PAD>
__global__ void __launch_bounds__(kThreads, 2) bwd_dq_kernel(AttnArgs a, BwdArgs g) {
    using G = Geo<D>;
    constexpr int SB = SmemDq<D>::SB;
    constexpr int IPW = SB / 1024 / 4 > 0 ? SB / 1024 / 4 : 1;
    static_assert(SB == IPW * 1024 * 4, "stage of whole 1 KB loads per wavefront");
    __shared__ SmemDq<D> sm;
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
    const int32_t o = load_spans<kThreads>(a, sm.sp, tid);
    const int32_t n_shared = a.sparse ? sm.sp.cum[sm.sp.n] : 0;
    const int32_t chunk = dense ? r % a.n_chunks : 0;
    const int32_t row0 = dense ? (r / a.n_chunks) * kBlockMBf16 : (r - dense_items) * kBlockMBf16;
    const ItemList L = item_list(a, dense, chunk, row0, o, n_shared, sm.sp, sm.n_keep, wave, lane);
    const int nblk = (L.total + kBQ - 1) / kBQ;
    RowInfo ri = row_info(a, dense, row0, wave * 32 + ql, kBlockMBf16, o, n_shared, sm.sp);
    // a wavefront that stores none of its 32 rows (rows past the dense rows
    // in the last dense block, a sparse block's rows of shared tokens, which
    // dense items own, or rows past the image span) only stages its share of
    // the list: its SIMD is left to the other workgroup
    const bool idle = __builtin_amdgcn_ballot_w64(ri.store) == 0;
    if (!PAD) ri.pad = false;

    const int32_t bb = bh / a.heads;
    const int32_t hh = bh - bb * a.heads;
    __bf16* dqrow = reinterpret_cast<__bf16*>(g.dq) + bb * a.q_sb + hh * a.q_sh + (int64_t)ri.qseq * a.q_sr;
    if (PAD && !dense && !__syncthreads_or(ri.store && !ri.pad)) {
        f32x16 zero[D / 32];
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) zero[dt] = f32x16{};
        if (ri.store) store_grad<D>(dqrow, zero, 0.f, true, h);
        return;
    }
    const int64_t qoff = bb * a.q_sb + hh * a.q_sh + (int64_t)ri.qseq * a.q_sr;
    const int64_t ooff = bb * a.o_sb + hh * a.o_sh + (int64_t)ri.qseq * a.o_sr;
    bf16x8 q[D / 16], dov[D / 16];
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) {
        q[kc] = *reinterpret_cast<const bf16x8*>(reinterpret_cast<const __bf16*>(a.q) + qoff + 16 * kc + 8 * h);
        dov[kc] = *reinterpret_cast<const bf16x8*>(reinterpret_cast<const __bf16*>(g.dout) + ooff + 16 * kc + 8 * h);
    }
    const float lse2 = g.lse2[(int64_t)bh * a.n_tot + ri.qseq];
    const float dlt = g.delta[(int64_t)bh * a.n_tot + ri.qseq];
    // dP - Dlt comes out of the dP^T products: their accumulator starts at
    // -Dlt of this lane's row
    f32x16 ndlt16;
#pragma unroll
    for (int e = 0; e < 16; ++e) ndlt16[e] = -dlt;

    const __bf16* kbase = reinterpret_cast<const __bf16*>(a.k) + bb * a.k_sb + hh * a.k_sh;
    const __bf16* vbase = reinterpret_cast<const __bf16*>(a.v) + bb * a.v_sb + hh * a.v_sh;
    const __amdgpu_buffer_rsrc_t krs = slice_rsrc(kbase, a.n_tot, a.k_sr, D, 2);
    const __amdgpu_buffer_rsrc_t vrs = slice_rsrc(vbase, a.n_tot, a.v_sr, D, 2);
    const int32_t krow_b = (int32_t)(a.k_sr * 2), vrow_b = (int32_t)(a.v_sr * 2);
    // direct loads: lane l of load j fills LDS chunk p = (w IPW + j) 64 + l
    // of the stage, i.e. row p / CPR, stored chunk p % CPR, which holds
    // global chunk (p % CPR) ^ f(row)
    int32_t srow[IPW], colk[IPW], koff[IPW], voff[IPW];
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
        const int p = (wave * IPW + j) * 64 + lane;
        srow[j] = p / G::CPR;
        colk[j] = ((p % G::CPR) ^ G::fk(srow[j])) * 16;
        koff[j] = srow[j] * krow_b + colk[j];  // byte offset within a stage of consecutive rows
        voff[j] = srow[j] * vrow_b + colk[j];
    }
    const uint32_t k0 = lds_addr(&sm.k[0][wave * IPW * 1024]);
    const uint32_t v0l = lds_addr(&sm.v[0][wave * IPW * 1024]);

    auto stage_fast = [&](int32_t i) -> bool {
        const int32_t v0 = i * kBQ;
        return L.total - v0 >= kBQ && !(L.label_mask && v0 + kBQ > L.b2);
    };
    auto load_stage = [&](int32_t i, int buf) {
        const int32_t v0 = i * kBQ;
        const int32_t cnt = min(kBQ, L.total - v0);
        int32_t base = -1;
        if (v0 + cnt <= L.b1) base = L.s0 + v0;
        else if (v0 >= L.b2 && v0 + cnt <= L.b3) base = L.sa + (v0 - L.b2);
        else if (v0 >= L.b3) base = L.sb + (v0 - L.b3);
        if (PAD) {
            const int32_t v = lane < kBQ ? v0 + lane : L.total;
            const int32_t seq = v >= L.total ? 0 : base >= 0 ? base + lane
                                                            : list_seq(v, L.b1, L.b2, L.b3, L.s0, L.sa, L.sb, sm.sp);
            const int32_t inf = entry_info<true>(a, L, v, seq, o, sm.sp);
            const bool none = __builtin_amdgcn_ballot_w64(inf != kKeyInvalid) == 0;
            if (wave == 0) {
                if (lane < kBQ) sm.info[buf][lane] = inf;
                const bool slow = __builtin_amdgcn_ballot_w64(lane < kBQ && inf != kKeyAll) != 0;
                if (lane == 0) sm.slow[buf] = none ? 2 : slow ? 1 : 0;
            }
            if (none) return;
        }
        const uint32_t off = buf * SB;
        if (base >= 0 && cnt == kBQ) {
            // 32 consecutive rows inside the slice: the first row's byte
            // offset goes in the scalar offset field
#pragma unroll
            for (int j = 0; j < IPW; ++j) {
                dma16s(krs, k0 + off + j * 1024, koff[j], base * krow_b);
                dma16s(vrs, v0l + off + j * 1024, voff[j], base * vrow_b);
            }
        } else {
            // every key row first, then the loads (an asm statement with a
            // memory clobber each: a map read after one could not start
            // before it)
            int32_t key[IPW];
#pragma unroll
            for (int j = 0; j < IPW; ++j) {
                const int32_t rr = min(srow[j], cnt - 1);
                key[j] = base >= 0 ? base + rr : list_seq(v0 + rr, L.b1, L.b2, L.b3, L.s0, L.sa, L.sb, sm.sp);
            }
#pragma unroll
            for (int j = 0; j < IPW; ++j) {
                dma16(krs, k0 + off + j * 1024, key[j] * krow_b + colk[j]);
                dma16(vrs, v0l + off + j * 1024, key[j] * vrow_b + colk[j]);
            }
        }
        if (!PAD && !stage_fast(i) && tid < kBQ) {
            const int32_t v = v0 + tid;
            const int32_t seq = v >= L.total ? 0 : list_seq(v, L.b1, L.b2, L.b3, L.s0, L.sa, L.sb, sm.sp);
            sm.info[buf][tid] = entry_info<false>(a, L, v, seq, o, sm.sp);
        }
    };

    const int ka = row_base<D>(lane);
    const int va0 = tr_base<D>(lane, 0), va1 = tr_base<D>(lane, 1);
    f32x16 acc[D / 32];
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) acc[dt] = f32x16{};
    const float c = a.scale_log2;

    wait_vmcnt<0>();
    load_stage(0, 0);
    wait_vmcnt<0>();
    __syncthreads();
    // one stage; the buffer index is a compile-time constant (the loop
    // below runs stages in pairs), so LDS addresses carry it as an immediate
    auto stage = [&](int32_t i, auto buf_c) {
        constexpr int buf = decltype(buf_c)::value;
        if (i + 1 < nblk) load_stage(i + 1, buf ^ 1);
        if (!PAD || sm.slow[buf] != 2) {
            const uint8_t* kb_ = sm.k[buf];
            const uint8_t* vb_ = sm.v[buf];
            // S^T = K Q^T and dP^T = V dO^T: register e holds key
            // 8 (e/4) + 4 h + e%4 against this lane's row
            // K and V operands requested kAhead reduction steps before use
            f32x16 s = f32x16{}, dp = ndlt16;
            constexpr int kAhead = 3;
            bf16x8 rk[kAhead + 1], rv[kAhead + 1];
#pragma unroll
            for (int kc = 0; kc < kAhead; ++kc) {
                rk[kc] = *reinterpret_cast<const bf16x8*>(kb_ + (ka ^ (32 * kc)));
                rv[kc] = *reinterpret_cast<const bf16x8*>(vb_ + (ka ^ (32 * kc)));
            }
#pragma unroll
            for (int kc = 0; kc < D / 16; ++kc) {
                if (kc + kAhead < D / 16) {
                    const int ad = ka ^ (32 * (kc + kAhead));
                    rk[(kc + kAhead) % (kAhead + 1)] = *reinterpret_cast<const bf16x8*>(kb_ + ad);
                    rv[(kc + kAhead) % (kAhead + 1)] = *reinterpret_cast<const bf16x8*>(vb_ + ad);
                }
                s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(rk[kc % (kAhead + 1)], q[kc], s, 0, 0, 0);
                dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(rv[kc % (kAhead + 1)], dov[kc], dp, 0, 0, 0);
            }
            // keep that order: the scheduler would otherwise sink each read
            // to just before its product
            __builtin_amdgcn_sched_group_barrier(0x100, 2 * kAhead, 0);
#pragma unroll
            for (int kc = 0; kc < D / 16; ++kc) {
                if (kc + kAhead < D / 16) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
            }
            if (PAD ? sm.slow[buf] != 0 : !stage_fast(i)) {
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int32_t inf = sm.info[buf][8 * (e >> 2) + 4 * h + (e & 3)];
                    s[e] = (inf == kKeyAll || inf == ri.label) ? s[e] : -INFINITY;
                }
            }
            bf16x8 ds[2];
#pragma unroll
            for (int cc = 0; cc < 2; ++cc)
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int e = 8 * cc + j;
                    const float pe = __builtin_amdgcn_exp2f(fmaf(s[e], c, -lse2));
                    ds[cc][j] = (__bf16)(pe * dp[e]);
                }
            const uint8_t* ktb = sm.k[buf];
#pragma unroll
            for (int cc = 0; cc < 2; ++cc)
#pragma unroll
                for (int dt = 0; dt < D / 32; ++dt)
                    acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_operand<D>(ktb, va0, va1, cc, dt), ds[cc],
                                                                      acc[dt], 0, 0, 0);
        }
        wait_vmcnt<0>();
        __syncthreads();
    };
    if (idle) {
        for (int32_t i = 0; i < nblk; ++i) {
            if (i + 1 < nblk) load_stage(i + 1, (i + 1) & 1);
            wait_vmcnt<0>();
            __syncthreads();
        }
    } else {
        for (int32_t i = 0; i < nblk; i += 2) {
            stage(i, std::integral_constant<int, 0>{});
            if (i + 1 < nblk) stage(i + 1, std::integral_constant<int, 1>{});
        }
    }
    if (dense && a.n_chunks > 1) {
        store_partial<D>(a, bh, chunk, ri.dense_row, 0, acc, h);
        return;
    }
    if (!ri.store) return;
    store_grad<D>(dqrow, acc, a.scale_log2 * 0.69314718055994530942f, ri.pad, h);
}

// -------------------------------------------------------------------- dK dV
template <int D>
struct SmemDkdv {
    static constexpr int SB = kBQ * Geo<D>::ROWB;
    alignas(16) uint8_t q[2][SB];   // fk: A operand of S, transposed A operand of dK^T
    alignas(16) uint8_t d[2][SB];   // fk: dO, A operand of dP, transposed A operand of dV^T
    alignas(16) float lse2[2][kBQ];
    alignas(16) float ndlt[2][kBQ];  // -Dlt of the stage's queries
    alignas(16) int32_t info[2][kBQ];
    Spans sp;
    int32_t n_keep;
    int32_t slow[2];
};

template <int D, bool PAD>
__global__ void __launch_bounds__(kThreads, 2) bwd_dkdv_kernel(AttnArgs a, BwdArgs g) {
    using G = Geo<D>;
    constexpr int SB = SmemDkdv<D>::SB;
    constexpr int IPW = SB / 1024 / 4 > 0 ? SB / 1024 / 4 : 1;
    static_assert(SB == IPW * 1024 * 4, "stage of whole 1 KB loads per wavefront");
    __shared__ SmemDkdv<D> sm;
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
    const int32_t o = load_spans<kThreads>(a, sm.sp, tid);
    const int32_t n_shared = a.sparse ? sm.sp.cum[sm.sp.n] : 0;
    const int32_t chunk = dense ? r % a.n_chunks : 0;
    const int32_t row0 = dense ? (r / a.n_chunks) * kBlockMBf16 : (r - dense_items) * kBlockMBf16;
    const ItemList L = item_list(a, dense, chunk, row0, o, n_shared, sm.sp, sm.n_keep, wave, lane);
    const int nblk = (L.total + kBQ - 1) / kBQ;
    RowInfo ri = row_info(a, dense, row0, wave * 32 + ql, kBlockMBf16, o, n_shared, sm.sp);
    // a wavefront that stores none of its 32 rows (rows past the dense rows
    // in the last dense block, a sparse block's rows of shared tokens, which
    // dense items own, or rows past the image span) only stages its share of
    // the list: its SIMD is left to the other workgroup.  Not wavefront 0,
    // which also publishes each stage's row values.
    const bool idle = wave != 0 && __builtin_amdgcn_ballot_w64(ri.store) == 0;
    if (!PAD) ri.pad = false;

    const int32_t bb = bh / a.heads;
    const int32_t hh = bh - bb * a.heads;
    // output rows (formed where they are written, not held across the loop)
    auto dkrow = [&]() {
        return reinterpret_cast<__bf16*>(g.dk) + bb * a.k_sb + hh * a.k_sh + (int64_t)ri.qseq * a.k_sr;
    };
    auto dvrow = [&]() {
        return reinterpret_cast<__bf16*>(g.dv) + bb * a.v_sb + hh * a.v_sh + (int64_t)ri.qseq * a.v_sr;
    };
    if (PAD && !dense && !__syncthreads_or(ri.store && !ri.pad)) {
        f32x16 zero[D / 32];
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) zero[dt] = f32x16{};
        if (ri.store) {
            store_grad<D>(dkrow(), zero, 0.f, true, h);
            store_grad<D>(dvrow(), zero, 0.f, true, h);
        }
        return;
    }
    const int64_t koff = bb * a.k_sb + hh * a.k_sh + (int64_t)ri.qseq * a.k_sr;
    const int64_t voff = bb * a.v_sb + hh * a.v_sh + (int64_t)ri.qseq * a.v_sr;
    bf16x8 kr[D / 16], vr[D / 16];
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) {
        kr[kc] = *reinterpret_cast<const bf16x8*>(reinterpret_cast<const __bf16*>(a.k) + koff + 16 * kc + 8 * h);
        vr[kc] = *reinterpret_cast<const bf16x8*>(reinterpret_cast<const __bf16*>(a.v) + voff + 16 * kc + 8 * h);
    }

    const __bf16* qbase = reinterpret_cast<const __bf16*>(a.q) + bb * a.q_sb + hh * a.q_sh;
    const __bf16* dbase = reinterpret_cast<const __bf16*>(g.dout) + bb * a.o_sb + hh * a.o_sh;
    const __amdgpu_buffer_rsrc_t qrs = slice_rsrc(qbase, a.n_tot, a.q_sr, D, 2);
    const __amdgpu_buffer_rsrc_t drs = slice_rsrc(dbase, a.n_tot, a.o_sr, D, 2);
    const int32_t qrow_b = (int32_t)(a.q_sr * 2), drow_b = (int32_t)(a.o_sr * 2);
    const float* lse2_bh = g.lse2 + (int64_t)bh * a.n_tot;
    const float* dlt_bh = g.delta + (int64_t)bh * a.n_tot;
    const uint32_t q0 = lds_addr(&sm.q[0][wave * IPW * 1024]);
    const uint32_t d0 = lds_addr(&sm.d[0][wave * IPW * 1024]);

    float nl = 0.f, nd = 0.f;
    auto stage_fast = [&](int32_t i) -> bool {
        const int32_t v0 = i * kBQ;
        return L.total - v0 >= kBQ && !(L.label_mask && v0 + kBQ > L.b2);
    };
    auto load_stage = [&](int32_t i, int buf) {
        const int32_t v0 = i * kBQ;
        const int32_t cnt = min(kBQ, L.total - v0);
        int32_t base = -1;
        if (v0 + cnt <= L.b1) base = L.s0 + v0;
        else if (v0 >= L.b2 && v0 + cnt <= L.b3) base = L.sa + (v0 - L.b2);
        else if (v0 >= L.b3) base = L.sb + (v0 - L.b3);
        const int32_t v = lane < kBQ ? v0 + lane : L.total;
        const int32_t seq = v >= L.total ? 0 : base >= 0 ? base + lane
                                                        : list_seq(v, L.b1, L.b2, L.b3, L.s0, L.sa, L.sb, sm.sp);
        if (PAD) {
            const int32_t inf = entry_info<true>(a, L, v, seq, o, sm.sp);
            const bool none = __builtin_amdgcn_ballot_w64(inf != kKeyInvalid) == 0;
            if (wave == 0) {
                if (lane < kBQ) sm.info[buf][lane] = inf;
                const bool slow = __builtin_amdgcn_ballot_w64(lane < kBQ && inf != kKeyAll) != 0;
                if (lane == 0) sm.slow[buf] = none ? 2 : slow ? 1 : 0;
            }
            if (none) return;
        }
        if (wave == 0) {
            nl = lse2_bh[seq];
            nd = dlt_bh[seq];
        }
        const uint32_t off = buf * SB;
        // row and swizzled chunks of this lane's piece of load j, formed per
        // stage (cheaper than holding them across the loop)
        uint32_t lane_s = lane;
        asm volatile("" : "+v"(lane_s));
        int32_t srow[IPW], colk[IPW];
#pragma unroll
        for (int j = 0; j < IPW; ++j) {
            const uint32_t p = (uint32_t)(wave * IPW + j) * 64u + lane_s;
            srow[j] = (int32_t)(p / G::CPR);
            colk[j] = (int32_t)(((p % G::CPR) ^ (uint32_t)G::fk(srow[j])) * 16u);
        }
        if (base >= 0 && cnt == kBQ) {
            // 32 consecutive rows inside the slice: the first row's byte
            // offset goes in the scalar offset field
#pragma unroll
            for (int j = 0; j < IPW; ++j) {
                dma16s(qrs, q0 + off + j * 1024, srow[j] * qrow_b + colk[j], base * qrow_b);
                dma16s(drs, d0 + off + j * 1024, srow[j] * drow_b + colk[j], base * drow_b);
            }
        } else {
            // every query row first, then the loads (see the dQ pass)
            int32_t qs[IPW];
#pragma unroll
            for (int j = 0; j < IPW; ++j) {
                const int32_t rr = min(srow[j], cnt - 1);
                qs[j] = base >= 0 ? base + rr : list_seq(v0 + rr, L.b1, L.b2, L.b3, L.s0, L.sa, L.sb, sm.sp);
            }
#pragma unroll
            for (int j = 0; j < IPW; ++j) {
                dma16(qrs, q0 + off + j * 1024, qs[j] * qrow_b + colk[j]);
                dma16(drs, d0 + off + j * 1024, qs[j] * drow_b + colk[j]);
            }
        }
        if (!PAD && !stage_fast(i) && tid < kBQ) sm.info[buf][tid] = entry_info<false>(a, L, v, seq, o, sm.sp);
    };

    const int ka = row_base<D>(lane);
    const int va0 = tr_base<D>(lane, 0), va1 = tr_base<D>(lane, 1);
    f32x16 acck[D / 32], accv[D / 32];
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
        acck[dt] = f32x16{};
        accv[dt] = f32x16{};
    }
    const float c = a.scale_log2;

    wait_vmcnt<0>();
    load_stage(0, 0);
    wait_vmcnt<0>();
    if (wave == 0 && lane < kBQ) {
        sm.lse2[0][lane] = nl;
        sm.ndlt[0][lane] = -nd;
    }
    __syncthreads();
    // one stage, the buffer index a compile-time constant as in the dQ pass
    auto stage = [&](int32_t i, auto buf_c) {
        constexpr int buf = decltype(buf_c)::value;
        if (i + 1 < nblk) load_stage(i + 1, buf ^ 1);
        if (!PAD || sm.slow[buf] != 2) {
            const uint8_t* qb = sm.q[buf];
            const uint8_t* db = sm.d[buf];
            // lane bases recomputed per stage rather than held across the loop
            int ka_s = ka, va0_s = va0, va1_s = va1;
            asm volatile("" : "+v"(ka_s), "+v"(va0_s), "+v"(va1_s));
            // S = Q K^T and dP = dO V^T: register e holds query
            // 8 (e/4) + 4 h + e%4 against this lane's key.  The dP
            // accumulator starts at the queries' -Dlt, so dP - Dlt comes out
            // of the products.
            f32x16 s = f32x16{}, dp;
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4) {
                const f4 d4 = *reinterpret_cast<const f4*>(&sm.ndlt[buf][8 * g4 + 4 * h]);
#pragma unroll
                for (int t = 0; t < 4; ++t) dp[4 * g4 + t] = d4[t];
            }
#pragma unroll
            for (int kc = 0; kc < D / 16; ++kc) {
                const int ad = ka_s ^ (32 * kc);
                s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8*>(qb + ad), kr[kc], s, 0, 0, 0);
                dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8*>(db + ad), vr[kc], dp, 0, 0,
                                                             0);
            }
            if (PAD ? sm.slow[buf] != 0 : !stage_fast(i)) {
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int32_t inf = sm.info[buf][8 * (e >> 2) + 4 * h + (e & 3)];
                    s[e] = (inf == kKeyAll || inf == ri.label) ? s[e] : -INFINITY;
                }
            }
            bf16x8 pb[2], ds[2];
#pragma unroll
            for (int cc = 0; cc < 2; ++cc)
#pragma unroll
                for (int j4 = 0; j4 < 2; ++j4) {
                    const int g4 = 2 * cc + j4;
                    const f4 l4 = *reinterpret_cast<const f4*>(&sm.lse2[buf][8 * g4 + 4 * h]);
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        const int e = 4 * g4 + t;
                        const float pe = __builtin_amdgcn_exp2f(fmaf(s[e], c, -l4[t]));
                        pb[cc][4 * j4 + t] = (__bf16)pe;
                        ds[cc][4 * j4 + t] = (__bf16)(pe * dp[e]);
                    }
                }
            const uint8_t* dtb = sm.d[buf];
            const uint8_t* qtb = sm.q[buf];
            // the phase's products in a fixed order (m = 4 D/32 cc... : dV^T
            // for even m, dK^T for odd m), each A operand requested
            // kAhead products before its use
            constexpr int NM = 2 * 2 * (D / 32);
            constexpr int kAhead = 2;
            auto opnd = [&](int m) -> bf16x8 {
                return tr_operand<D>((m & 1) ? qtb : dtb, va0_s, va1_s, m / (2 * (D / 32)), (m >> 1) % (D / 32));
            };
            bf16x8 ring[kAhead + 1];
#pragma unroll
            for (int m = 0; m < kAhead; ++m) ring[m] = opnd(m);
#pragma unroll
            for (int m = 0; m < NM; ++m) {
                if (m + kAhead < NM) ring[(m + kAhead) % (kAhead + 1)] = opnd(m + kAhead);
                const int cc = m / (2 * (D / 32)), dt = (m >> 1) % (D / 32);
                if (m & 1)
                    acck[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ring[m % (kAhead + 1)], ds[cc], acck[dt], 0, 0, 0);
                else
                    accv[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ring[m % (kAhead + 1)], pb[cc], accv[dt], 0, 0, 0);
            }
        }
        wait_vmcnt<0>();
        if (wave == 0 && lane < kBQ && i + 1 < nblk) {
            sm.lse2[buf ^ 1][lane] = nl;
            sm.ndlt[buf ^ 1][lane] = -nd;
        }
        __syncthreads();
    };
    if (idle) {
        for (int32_t i = 0; i < nblk; ++i) {
            if (i + 1 < nblk) load_stage(i + 1, (i + 1) & 1);
            wait_vmcnt<0>();
            __syncthreads();
        }
    } else {
        for (int32_t i = 0; i < nblk; i += 2) {
            stage(i, std::integral_constant<int, 0>{});
            if (i + 1 < nblk) stage(i + 1, std::integral_constant<int, 1>{});
        }
    }
    if (dense && a.n_chunks > 1) {
        store_partial<D>(a, bh, chunk, ri.dense_row, 0, acck, h);
        store_partial<D>(a, bh, chunk, ri.dense_row, 1, accv, h);
        return;
    }
    if (!ri.store) return;
    store_grad<D>(dkrow(), acck, a.scale_log2 * 0.69314718055994530942f, ri.pad, h);
    store_grad<D>(dvrow(), accv, 1.f, ri.pad, h);
}

template <int D>
hipError_t launch_bwd_t(const AttnArgs& a, const BwdArgs& g, hipStream_t s) {
    const int64_t rows = (int64_t)a.n_bh * a.n_tot;
    constexpr int64_t rpb = 256 / (D / 4);
    constexpr int64_t ppb = 256 / (D / 8) * kPrepPasses;
    const int64_t pblocks = (rows + ppb - 1) / ppb;
    if (pblocks > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((bwd_prep_kernel<D>), dim3((unsigned)pblocks), dim3(256), 0, s, a, g);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t srows = (int64_t)a.n_bh * a.n_dense_rows;
    const unsigned sblocks = (unsigned)((srows + rpb - 1) / rpb);
    const bool split = a.n_chunks > 1 && srows > 0;
    if (a.padded)
        hipLaunchKernelGGL((bwd_dq_kernel<D, true>), dim3(a.total_items), dim3(kThreads), 0, s, a, g);
    else
        hipLaunchKernelGGL((bwd_dq_kernel<D, false>), dim3(a.total_items), dim3(kThreads), 0, s, a, g);
    if (split) hipLaunchKernelGGL((bwd_sum_kernel<D>), dim3(sblocks), dim3(256), 0, s, a, g, 0);
    if (a.padded)
        hipLaunchKernelGGL((bwd_dkdv_kernel<D, true>), dim3(a.total_items), dim3(kThreads), 0, s, a, g);
    else
        hipLaunchKernelGGL((bwd_dkdv_kernel<D, false>), dim3(a.total_items), dim3(kThreads), 0, s, a, g);
    if (split) hipLaunchKernelGGL((bwd_sum_kernel<D>), dim3(sblocks), dim3(256), 0, s, a, g, 1);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bwd(const AttnArgs& a, const BwdArgs& g, int head_dim, hipStream_t s) {
    if (a.total_items == 0) return hipSuccess;
    return head_dim == 128 ? launch_bwd_t<128>(a, g, s) : launch_bwd_t<64>(a, g, s);
}

}  // namespace hilberta
