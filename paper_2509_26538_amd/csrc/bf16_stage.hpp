// Pieces shared by the bf16 attention kernels (forward in attn_bf16.hip,
// backward in attn_bwd.hip): the geometry of a 64-row stage of bf16 rows in
// LDS, the direct global-to-LDS loads that fill it, and the key list of a
// work item.
//
// A stage holds 64 rows of D bf16 values, unpadded, each row's 16-byte
// chunks XOR-swizzled by the row index.  fk serves rows read whole as an
// MFMA A operand and rows read with the transposing ds_read_b64_tr_b16 alike,
// so a tensor read both ways is staged once: it is a bijection on every 16
// consecutive rows (16 lanes that read one chunk each of 16 consecutive rows
// hit 16 different bank groups), and the four aligned consecutive rows that
// one transposing read touches land in disjoint quarters of the banks.  fv
// serves rows that are only read transposed (the forward's V).
#pragma once

#include "attn_common.hpp"

namespace hilberta {
namespace {

constexpr int kBN = 64;  // keys per stage
static_assert(kBlockMBf16 == 128, "four wavefronts of 32 rows");

template <int D>
struct Geo {
    static constexpr int CPR = D / 8;              // 16-byte chunks per row
    static constexpr int ROWB = D * 2;             // bytes per row
    static constexpr int STAGEB = kBN * ROWB;      // bytes per tensor and stage
    static constexpr int IPW = STAGEB / 1024 / 4;  // 1 KB direct loads per wavefront and tensor
    // chunk swizzles (XOR on the 16-byte chunk index of a row).  D = 128:
    // a row spans all 64 banks and fk puts row bits 0-1 on the quarter (chunk
    // bits 2-3), bits 2-3 on the chunk within it.  D = 64: two rows share the
    // banks (row bit 0 picks the half), fk puts row bit 1 on the quarter
    // within the half and bits 2-3 on the chunk within it.
    __device__ __forceinline__ static int fk(int row) {
        return D == 128 ? 4 * (row & 3) + ((row >> 2) & 3) : 4 * ((row >> 1) & 1) + ((row >> 2) & 3);
    }
    __device__ __forceinline__ static int fv(int row) { return D == 128 ? 4 * (row & 3) : 4 * ((row >> 1) & 1); }
};


typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// One 16-byte-per-lane buffer load straight into LDS at lds_base + 16 lane,
// bounds-checked against the resource.  Inline assembly, so that the
// compiler does not guard later LDS reads with a wait for it: the kernel
// waits for each stage explicitly before the barrier that publishes it.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rsrc, uint32_t lds_base, int32_t voff) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :
                 : "s"(lds_base), "v"(voff), "s"(rsrc)
                 : "memory", "m0");
}

// The same with a uniform byte offset in the instruction's scalar offset
// field, for a stage of contiguous rows: the per-lane offset stays fixed for
// the whole item, so issuing the stage costs no vector instruction.  The
// scalar offset is outside the buffer's range check; callers use it only
// for rows that lie inside the slice.
__device__ __forceinline__ void dma16s(__amdgpu_buffer_rsrc_t rsrc, uint32_t lds_base, int32_t voff, int32_t soff) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 :
                 : "s"(lds_base), "v"(voff), "s"(rsrc), "s"(soff)
                 : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void*)p);
}

// Sequence position of key v of the list (segment boundaries b1 <= b2 <= b3;
// segment 0 starts at s0, the shared map covers [b1, b2), segment 2 starts
// at sa and segment 3 at sb).
__device__ __forceinline__ int32_t list_seq(int32_t v, int32_t b1, int32_t b2, int32_t b3, int32_t s0,
                                            int32_t sa, int32_t sb, const Spans& sp) {
    if (v < b1) return s0 + v;
    if (v < b2) return sp.map[v - b1];
    if (v < b3) return sa + (v - b2);
    return sb + (v - b3);
}


// The list of a work item: its keys for query rows (the forward and dQ),
// or, for the key rows of dK/dV, the queries that attend them -- the mask
// is symmetric, so that list is built the same way.  Dense items take a
// contiguous chunk of the sequence; sparse items take the text, the shared
// tokens outside the rows' covering tiles (the map in LDS is compacted to
// them), then the covering tiles' range and its wrapped tail.  The whole
// workgroup calls this (it ends with a barrier on the sparse path).
struct ItemList {
    int32_t b1, b2, b3, total, s0, sa, sb;
    bool label_mask;
};

__device__ __forceinline__ ItemList item_list(const AttnArgs& a, bool dense, int32_t chunk, int32_t row0,
                                              int32_t o, int32_t n_shared, Spans& sp, int32_t& n_keep,
                                              int wave, int lane) {
    ItemList L{};
    if (dense) {
        L.s0 = chunk * a.chunk_keys;
        L.total = min(a.chunk_keys, a.n_tot - L.s0);
        L.b1 = L.b2 = L.b3 = L.total;
        return L;
    }
    const int32_t p_last = min(a.n_img, row0 + kBlockMBf16) - 1;
    const int32_t t0 = (row0 + o) % a.n_img;
    const int32_t q1 = t0 / a.tile;
    const int32_t n_lab = min(a.n_tiles, (t0 + p_last - row0) / a.tile - q1 + 1);
    L.label_mask = n_lab > 1;
    const int32_t r_start = (int32_t)(((int64_t)q1 * a.tile - o + a.n_img) % a.n_img);
    const int32_t r_len = min(n_lab * a.tile, a.n_img);
    const int32_t len_a = min(r_len, a.n_img - r_start);
    if (wave == 0) {
        int32_t w = 0;
        for (int32_t u0 = 0; u0 < n_shared; u0 += 64) {
            const int32_t u = u0 + lane;
            int32_t seq = 0;
            bool keep = false;
            if (u < n_shared) {
                seq = sp.map[u];
                // seq - n_txt and r_start lie in [0, n_img)
                int32_t rel = seq - a.n_txt - r_start;
                rel += rel < 0 ? a.n_img : 0;
                keep = rel >= r_len;
            }
            const uint64_t bal = __builtin_amdgcn_ballot_w64(keep);
            const int32_t before = __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                             __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0));
            if (keep) sp.map[w + before] = seq;
            w += __builtin_popcountll(bal);
        }
        if (lane == 0) n_keep = w;
    }
    __syncthreads();
    L.s0 = 0;
    L.b1 = a.n_txt;
    L.b2 = L.b1 + n_keep;
    L.b3 = L.b2 + len_a;
    L.total = L.b2 + r_len;
    L.sa = a.n_txt + r_start;
    L.sb = a.n_txt;
    return L;
}

// What list entry v is to the item's rows: kKeyInvalid (past the end, or a
// padding slot when PAD), kKeyAll, or its tile label when the rows straddle
// two tiles (rows of other tiles must not see it).
template <bool PAD>
__device__ __forceinline__ int32_t entry_info(const AttnArgs& a, const ItemList& L, int32_t v, int32_t seq,
                                              int32_t o, const Spans& sp) {
    if (v >= L.total) return kKeyInvalid;
    if (PAD && seq_padding(a, seq)) return kKeyInvalid;
    if (L.label_mask && v >= L.b2 && !is_shared_seq(sp, seq)) {
        // the divisors pass through an empty asm statement, so that the
        // compiler forms their reciprocals here, on this rarely taken path,
        // instead of holding them in registers across the whole stage loop
        int32_t tile = a.tile, n_img = a.n_img;
        asm volatile("" : "+s"(tile), "+s"(n_img));
        return tile_label(seq - a.n_txt, o, tile, n_img);
    }
    return kKeyAll;
}

// A operand of 32 rows x 16 columns (bf16x8 per lane) taken transposed from
// a stage in the fk layout: rows 16 cc .. 16 cc + 15 of the stage become the
// reduction index, in the order the score registers hold them (chunk cc of
// 16 list entries: register j holds entry 16 cc + 8 (j/4) + 4 h + j%4), and
// columns 32 dt .. 32 dt + 31 of the rows the 32 output rows.  The two reads
// cover rows 8 rd + 4 h + jj/4 (rd = 0, 1), whose swizzles differ, so each
// has its own lane base (tr_base); the column block dt flips only address
// bits 6-7 (the chunk index is 4 dt + c0 with c0 < 4, and fk moves whole
// quarters apart or chunks within one), and 16 rows further on is 16 ROWB
// further on (fk looks at row bits 0-3 only).
template <int D>
__device__ __forceinline__ bf16x8 tr_operand(const uint8_t* buf, int va0, int va1, int cc, int dt) {
    const int rows = 16 * cc * Geo<D>::ROWB;
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(buf + (va0 ^ (64 * dt)) + rows));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(buf + (va1 ^ (64 * dt)) + rows));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

template <int D>
__device__ __forceinline__ int tr_base(int lane, int rd) {
    const int h = lane >> 5, gi = lane >> 4, jj = lane & 15;
    const int row = 8 * rd + 4 * h + (jj >> 2);
    const int c0 = 2 * (gi & 1) + ((jj & 3) >> 1);
    return row * Geo<D>::ROWB + ((c0 ^ Geo<D>::fk(row)) * 16) + ((jj & 3) & 1) * 8;
}

// Lane base address for whole-row reads of the fk layout: row 32 kt + ql,
// chunk 2 kc + h at address (ka ^ 32 kc) + kt 32 ROWB.
template <int D>
__device__ __forceinline__ int row_base(int lane) {
    const int ql = lane & 31, h = lane >> 5;
    return ql * Geo<D>::ROWB + ((h ^ Geo<D>::fk(ql)) * 16);
}


}  // namespace
}  // namespace hilberta
