// HilbertA attention, bf16 path (§3.2-§3.4, Appendix A, Algorithm 1), for
// gfx950: bf16 inputs, fp32 accumulation and softmax state, P rounded to
// bf16 for the PV product, bf16 output.
//
// A workgroup of four wavefronts owns 128 query rows (32 per wavefront); two
// workgroups share a CU, so each SIMD interleaves two wavefronts.
//
// Keys.  An item's keys form one list visited in stages of 64: for a dense
// item the contiguous keys of its chunk; for a sparse item the text keys,
// then the shared tokens that lie outside the item's own tiles (compacted
// once per item, so every shared key is valid for every row), then the
// covering tiles' range and its wrapped tail (the modular indexing of §3.2,
// two contiguous ranges addressed in place).  Only the list's last stage is
// ragged, and per-row tile masks are needed only when the rows straddle two
// tiles.
//
// Staging.  K and V rows go straight from global memory into LDS with
// bounds-checked buffer_load ... lds (no staging registers), double
// buffered: stage i+1 is requested when stage i starts.  Rows are stored
// unpadded with their 16-byte chunks XOR-swizzled by row (D = 128): K chunk
// c of row r sits at c ^ (4 (r mod 4) + (r / 4 mod 4)), a bijection on any 16
// consecutive rows, so the 16 lanes that read one 16-byte piece of 16
// consecutive rows hit 16 different bank groups; V chunk c sits at
// c ^ 4 (r mod 4), so the four rows that a transposing read touches at once
// use disjoint 64-byte quarters of the banks.
//
// Per stage each wavefront computes
//   S^T = K Q^T    on v_mfma_f32_32x32x16_bf16 with K as the A operand
//                  (ds_read_b128) and Q in registers: each lane holds one
//                  query row and 32 of the 64 keys, so the online softmax
//                  state (Algorithm 1's attn_inner: max m, sum l,
//                  accumulator) is per lane; the two lane halves meet
//                  through v_permlane32_swap;
//   O^T += V^T P^T with V^T assembled by two ds_read_b64_tr_b16 from the
//                  row-major V rows, in exactly the key order the P
//                  registers hold (the MFMA reduction index may enumerate a
//                  chunk's keys in any order), and P^T straight from the
//                  score registers.
// All K operands of a stage are requested before its QK^T MFMAs and all V
// operands before its softmax, so the LDS latency overlaps the matrix work.
// The running sum is kept in fp32 as four independent partial sums.  The
// reference max moves only when a row max grows by more than 2^8 (acc and l
// share it, so it cancels in acc / l).
//
// General shapes: when the image span holds padding positions, wavefront 0
// classifies every key of a stage while it is loaded (the curve position
// decoded to its cell) and flags the stage for the per-key masks only if a
// key is padding or needs a label; a query block made of padding rows only
// stores its empty-softmax rows without visiting any key.
#include "bf16_stage.hpp"

#include <type_traits>

namespace hilberta {
namespace {

template <int D>
struct Smem {
    alignas(16) uint8_t k[2][Geo<D>::STAGEB];
    alignas(16) uint8_t v[2][Geo<D>::STAGEB];
    alignas(16) int32_t info[2][kBN];
    Spans sp;
    int32_t n_keep;
    int32_t slow[2];  // padded spans: stage needs the per-key masks
};

// PAD: the image span holds padding positions (a general shape).  A
// separate instantiation, so that the square power-of-two path carries none
// of the padding logic.
template <int D, bool PAD>
__global__ void __launch_bounds__(kThreads, 2) attn_bf16_kernel(AttnArgs a) {
    using G = Geo<D>;
    __shared__ Smem<D> sm;
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

    // ------------------------------------------------------------ key list
    const ItemList L = item_list(a, dense, chunk, row0, o, n_shared, sm.sp, sm.n_keep, wave, lane);
    const int32_t b1 = L.b1, b2 = L.b2, b3 = L.b3, total = L.total, s0 = L.s0, sa = L.sa, sb = L.sb;
    const bool label_mask = L.label_mask;
    const int nblk = (total + kBN - 1) / kBN;
    RowInfo ri = row_info(a, dense, row0, wave * 32 + ql, kBlockMBf16, o, n_shared, sm.sp);
    // a wavefront that stores none of its 32 rows (rows past the dense rows
    // in the last dense block, a sparse block's rows of shared tokens, which
    // dense items own, or rows past the image span) only stages its share of
    // the keys: its SIMD is left to the other workgroup.  Every duty of
    // wavefront 0 beyond that lies in load_stage, which it still runs.
    const bool idle = __builtin_amdgcn_ballot_w64(ri.store) == 0;
    if (!PAD) ri.pad = false;

    const int32_t bb = bh / a.heads;
    const int32_t hh = bh - bb * a.heads;
    if (PAD && !dense && !__syncthreads_or(ri.store && !ri.pad)) {
        // nothing but padding rows (and rows stored elsewhere): no keys
        f32x16 zero[D / 32];
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) zero[dt] = f32x16{};
        __bf16* ob = reinterpret_cast<__bf16*>(a.o) + bb * a.o_sb + hh * a.o_sh;
        store_row<__bf16, D>(a, ri, bh, chunk, dense, h, -INFINITY, 0.f, zero, ob);
        return;
    }
    const __bf16* qrow = reinterpret_cast<const __bf16*>(a.q) + bb * a.q_sb + hh * a.q_sh + (int64_t)ri.qseq * a.q_sr;
    const __bf16* kbase = reinterpret_cast<const __bf16*>(a.k) + bb * a.k_sb + hh * a.k_sh;
    const __bf16* vbase = reinterpret_cast<const __bf16*>(a.v) + bb * a.v_sb + hh * a.v_sh;
    // Q as the B operand of S^T = K Q^T: Q[row][16 kc + 8 h .. + 8]
    bf16x8 q[D / 16];
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) q[kc] = *reinterpret_cast<const bf16x8*>(qrow + 16 * kc + 8 * h);

    // Direct loads: wavefront w issues IPW 1 KB loads per tensor and stage;
    // lane l of load j fills LDS chunk p = (w IPW + j) 64 + l of the stage,
    // i.e. row p / CPR, stored chunk p % CPR, which holds global chunk
    // (p % CPR) ^ f(row) of that row.
    const __amdgpu_buffer_rsrc_t krs = slice_rsrc(kbase, a.n_tot, a.k_sr, D, 2);
    const __amdgpu_buffer_rsrc_t vrs = slice_rsrc(vbase, a.n_tot, a.v_sr, D, 2);
    const int32_t krow_b = (int32_t)(a.k_sr * 2), vrow_b = (int32_t)(a.v_sr * 2);
    int32_t srow[G::IPW], kcol[G::IPW], vcol[G::IPW], koff[G::IPW], voff[G::IPW];
#pragma unroll
    for (int j = 0; j < G::IPW; ++j) {
        const int p = (wave * G::IPW + j) * 64 + lane;
        srow[j] = p / G::CPR;
        kcol[j] = ((p % G::CPR) ^ G::fk(srow[j])) * 16;
        vcol[j] = ((p % G::CPR) ^ G::fv(srow[j])) * 16;
        koff[j] = srow[j] * krow_b + kcol[j];  // byte offset within a full contiguous stage
        voff[j] = srow[j] * vrow_b + vcol[j];
    }
    const uint32_t klds0 = lds_addr(&sm.k[0][wave * G::IPW * 1024]);
    const uint32_t vlds0 = lds_addr(&sm.v[0][wave * G::IPW * 1024]);

    // does stage i need per-key masks (ragged end, or per-row tile labels)?
    auto stage_fast = [&](int32_t i) -> bool {
        const int32_t v0 = i * kBN;
        return total - v0 >= kBN && !(label_mask && v0 + kBN > b2);
    };
    auto load_stage = [&](int32_t i, int buf) {
        const int32_t v0 = i * kBN;
        const int32_t cnt = min(kBN, total - v0);
        // one contiguous segment: uniform base
        int32_t base = -1;
        if (v0 + cnt <= b1) base = s0 + v0;
        else if (v0 >= b2 && v0 + cnt <= b3) base = sa + (v0 - b2);
        else if (v0 >= b3) base = sb + (v0 - b3);
        const uint32_t kl = klds0 + buf * G::STAGEB, vl = vlds0 + buf * G::STAGEB;
        if (PAD) {
            // every wavefront classifies the stage's keys (lane = key), so
            // each knows without a barrier whether the stage holds any key
            // at all; wavefront 0 publishes the per-key masks
            const int32_t v = v0 + lane;
            const int32_t seq = v >= total ? 0 : base >= 0 ? base + lane : list_seq(v, b1, b2, b3, s0, sa, sb, sm.sp);
            const int32_t inf = entry_info<true>(a, L, v, seq, o, sm.sp);
            const bool none = __builtin_amdgcn_ballot_w64(inf != kKeyInvalid) == 0;
            if (wave == 0) {
                sm.info[buf][lane] = inf;
                const bool slow = __builtin_amdgcn_ballot_w64(inf != kKeyAll) != 0;
                if (lane == 0) sm.slow[buf] = none ? 2 : slow ? 1 : 0;
            }
            if (none) return;  // nothing but padding: not loaded, not computed
        }
        if (base >= 0 && cnt == kBN) {
            // a full stage of contiguous keys (inside the slice: every
            // segment of the list lies in [0, n_tot)): one uniform offset
            const int32_t kb0 = base * krow_b, vb0 = base * vrow_b;
#pragma unroll
            for (int j = 0; j < G::IPW; ++j) {
                dma16s(krs, kl + j * 1024, koff[j], kb0);
                dma16s(vrs, vl + j * 1024, voff[j], vb0);
            }
        } else {
            // every key row first, then the loads: each load is an asm
            // statement with a memory clobber, so a shared-token map read
            // (LDS) placed after one could not start before it
            int32_t key[G::IPW];
#pragma unroll
            for (int j = 0; j < G::IPW; ++j) {
                // absent rows of a ragged stage re-read a present row (masked)
                const int32_t rr = min(srow[j], cnt - 1);
                key[j] = base >= 0 ? base + rr : list_seq(v0 + rr, b1, b2, b3, s0, sa, sb, sm.sp);
            }
#pragma unroll
            for (int j = 0; j < G::IPW; ++j) {
                dma16(krs, kl + j * 1024, key[j] * krow_b + kcol[j]);
                dma16(vrs, vl + j * 1024, key[j] * vrow_b + vcol[j]);
            }
        }
        if (!PAD && !stage_fast(i) && tid < kBN) {
            const int32_t v = v0 + tid;
            const int32_t seq = v >= total ? 0 : list_seq(v, b1, b2, b3, s0, sa, sb, sm.sp);
            sm.info[buf][tid] = entry_info<false>(a, L, v, seq, o, sm.sp);
        }
    };

    // Operand addresses within a stage buffer.
    // K: row 32 kt + ql, chunk 2 kc + h stored at (2 kc + h) ^ fk(row); fk
    //    does not depend on kt, so the address is ka ^ (32 kc) + kt 32 ROWB.
    const int ka = ql * G::ROWB + ((h ^ G::fk(ql)) * 16);
    // V (transposing reads): lane (group gi = lane/16, j = lane%16) reads row
    //    16 cc + 8 rd + 4 h + j/4, elements 32 dt + 16 (gi%2) + 4 (j%4) .. +4,
    //    i.e. chunk 4 dt + 2 (gi%2) + (j%4)/2, half (j%4)%2; fv(row) does not
    //    depend on cc, rd: address = va ^ (64 dt) + (16 cc + 8 rd) ROWB.
    const int gi = lane >> 4, jj = lane & 15;
    const int vrow = 4 * h + (jj >> 2);
    const int va = vrow * G::ROWB + (((2 * (gi & 1) + ((jj & 3) >> 1)) ^ G::fv(vrow)) * 16) + ((jj & 3) & 1) * 8;

    f32x16 acc[D / 32];
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) acc[dt] = f32x16{};
    float m_run = -INFINITY;         // reference max of the scaled logits, log2 units
    float lp[4] = {0.f, 0.f, 0.f, 0.f};  // this lane's share of the running sum, by key chunk
    const float c = a.scale_log2;

    // Q has landed before any stage is requested: afterwards the only
    // outstanding vector-memory operations are stage loads
    wait_vmcnt<0>();
    load_stage(0, 0);
    wait_vmcnt<0>();
    __syncthreads();

    // one stage; the buffer index is a compile-time constant (the loop
    // below runs stages in pairs), so LDS addresses carry it as an immediate
    auto stage = [&](int32_t i, auto buf_c) {
        constexpr int buf = decltype(buf_c)::value;
        if (i + 1 < nblk) load_stage(i + 1, buf ^ 1);
        // padded spans: sm.slow is 0 (no masks), 1 (per-key masks) or 2
        // (only padding keys: the stage is skipped)
        if (!PAD || sm.slow[buf] != 2) {
            const uint8_t* kb_ = sm.k[buf];
            const uint8_t* vb_ = sm.v[buf];

            // S^T: s[kt] register e holds key 32 kt + 8 (e/4) + 4 h + e%4.  All
            // K operands are requested first, so the MFMAs only wait for the
            // first ones to arrive.
            bf16x8 kop[D / 16][2];
#pragma unroll
            for (int kc = 0; kc < D / 16; ++kc)
#pragma unroll
                for (int kt = 0; kt < 2; ++kt)
                    kop[kc][kt] = *reinterpret_cast<const bf16x8*>(kb_ + (ka ^ (32 * kc)) + kt * 32 * G::ROWB);
            __builtin_amdgcn_sched_barrier(0);
            f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
            for (int kc = 0; kc < D / 16; ++kc)
#pragma unroll
                for (int kt = 0; kt < 2; ++kt)
                    s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[kc][kt], q[kc], s[kt], 0, 0, 0);
            // V^T operands of the whole stage, in flight during the softmax
            bf16x8 vop[4][D / 32];
#pragma unroll
            for (int cc = 0; cc < 4; ++cc)
#pragma unroll
                for (int dt = 0; dt < D / 32; ++dt) {
                    const uint8_t* vp = vb_ + (va ^ (64 * dt)) + 16 * cc * G::ROWB;
                    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vp));
                    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vp + 8 * G::ROWB));
                    vop[cc][dt] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
                }
            __builtin_amdgcn_sched_barrier(0);
            if (PAD ? sm.slow[buf] != 0 : !stage_fast(i)) {
#pragma unroll
                for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                    for (int e = 0; e < 16; ++e) {
                        const int32_t inf = sm.info[buf][32 * kt + 8 * (e >> 2) + 4 * h + (e & 3)];
                        s[kt][e] = (inf == kKeyAll || inf == ri.label) ? s[kt][e] : -INFINITY;
                    }
            }
            // row max over the 64 keys: a tree of three-way maxima (IEEE
            // maximum, which needs no canonicalising of the MFMA results; a
            // NaN score would reach the output through exp2 either way)
            float t3[11];
#pragma unroll
            for (int g = 0; g < 5; ++g) {
                t3[g] = vmax(vmax(s[0][3 * g], s[0][3 * g + 1]), s[0][3 * g + 2]);
                t3[5 + g] = vmax(vmax(s[1][3 * g], s[1][3 * g + 1]), s[1][3 * g + 2]);
            }
            t3[10] = vmax(s[0][15], s[1][15]);
            const float u0 = vmax(vmax(t3[0], t3[1]), t3[2]);
            const float u1 = vmax(vmax(t3[3], t3[4]), t3[5]);
            const float u2 = vmax(vmax(t3[6], t3[7]), t3[8]);
            const float u3 = vmax(t3[9], t3[10]);
            const float mx = half_vmax(vmax(vmax(u0, u1), vmax(u2, u3))) * c;
            if (__builtin_amdgcn_ballot_w64(mx > m_run + 8.f)) {
                const float m_new = fmaxf(m_run, mx);
                // a row with every key masked so far keeps -inf: leave it alone
                const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
                m_run = m_new;
#pragma unroll
                for (int x = 0; x < 4; ++x) lp[x] *= alpha;
#pragma unroll
                for (int dt = 0; dt < D / 32; ++dt) acc[dt] *= alpha;
            }
            const float m_use = m_run == -INFINITY ? 0.f : m_run;
            // P = exp2(S c - m) rounded to bf16; chunk cc of 16 keys holds key
            // 16 cc + 8 (j/4) + 4 h + j%4 in register j
            bf16x8 p[4];
#pragma unroll
            for (int cc = 0; cc < 4; ++cc)
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const float pe = __builtin_amdgcn_exp2f(fmaf(s[cc >> 1][8 * (cc & 1) + j], c, -m_use));
                    lp[cc] += pe;
                    p[cc][j] = (__bf16)pe;
                }
#pragma unroll
            for (int cc = 0; cc < 4; ++cc)
#pragma unroll
                for (int dt = 0; dt < D / 32; ++dt)
                    acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[cc][dt], p[cc], acc[dt], 0, 0, 0);
        }
        // stage i+1 must have landed before anyone reads it, and every
        // wavefront must be done with this buffer before it is refilled
        wait_vmcnt<0>();
        __syncthreads();
    };
    if (idle) {
        // only this wavefront's share of every stage's loads, and the
        // barriers the other wavefronts wait at
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

    __bf16* obase = reinterpret_cast<__bf16*>(a.o) + bb * a.o_sb + hh * a.o_sh;
    const float l_run = (lp[0] + lp[1]) + (lp[2] + lp[3]);
    store_row<__bf16, D>(a, ri, bh, chunk, dense, h, m_run, l_run, acc, obase);
}

template <int D>
hipError_t launch_t(const AttnArgs& a, hipStream_t s) {
    if (a.padded)
        hipLaunchKernelGGL((attn_bf16_kernel<D, true>), dim3(a.total_items), dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL((attn_bf16_kernel<D, false>), dim3(a.total_items), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bf16(const AttnArgs& a, int head_dim, hipStream_t s) {
    return head_dim == 128 ? launch_t<128>(a, s) : launch_t<64>(a, s);
}

}  // namespace hilberta
