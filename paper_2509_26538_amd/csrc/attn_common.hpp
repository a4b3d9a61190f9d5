// Device-side pieces shared by the attention kernels (attn.hip: fp32 path and
// the split merge; attn_bf16.hip: the bf16 path): the key-segment walk of a
// work item, the shared-token map, per-row bookkeeping, buffer resources.
//
// Work items per (batch, head):
//   dense items  -- rows that attend every key: the text and shared rows of
//                   HilbertA (Appendix A treats both as a global prefix that
//                   attends everything), or all rows of the dense baseline.
//                   Their keys may be split into chunks whose partial
//                   (acc, m, l) are merged by a second small kernel.
//   sparse items -- consecutive image rows.  Keys: the text span, the shared
//                   tokens (gathered), and the slid tile(s) covering the
//                   rows.  A tile that runs past the end of the image span
//                   continues at its head (the modular indexing of §3.2):
//                   two contiguous segments, addressed in place.
// Each key is visited once: shared keys that also lie in the rows' tiles are
// masked in the shared segment (fp32 kernel) or left out of it (bf16
// kernel).  Rows of shared tokens inside a sparse item are computed by the
// dense items and not stored by the sparse item.
//
// General shapes (Appendix D): the image span holds every position of the
// enclosing square's curve; a position whose cell lies outside the grid is
// padding.  Padding keys are masked for every row (stages that hold one take
// the per-key mask path), and padding rows are stored as an empty softmax:
// O = 0, LSE = -inf.
#pragma once

#include "curve.hpp"
#include "internal.hpp"

namespace hilberta {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kKeyInvalid = -2;  // masked for every row
constexpr int kKeyAll = -1;      // valid for every row
enum : int32_t { SEG_CONTIG = 0, SEG_SHARED = 1, SEG_TILE = 2 };
constexpr float kLn2 = 0.69314718055994530942f;

struct Spans {
    int32_t start[kMaxSpans];    // sequence position of the run's first token
    int32_t len[kMaxSpans];
    int32_t cum[kMaxSpans + 1];  // shared tokens before the run
    int32_t n;
    int32_t map[kMaxShared];     // sequence position of the u-th shared token
};

// Uniform description of one work item's keys: at most four segments (text,
// gathered shared tokens, covering tiles, wrapped tail).  Functions below
// take these as separate scalar arguments, never through a pointer, so they
// stay in scalar registers (a field load through a selected pointer would
// pin the whole description in scratch memory).
struct Segs {
    int32_t b0, b1, b2, b3;  // sequence position of the first key (SHARED: 0)
    int32_t l0, l1, l2, l3;  // lengths
    int32_t k0, k1, k2, k3;  // kinds
    int32_t e0, e1, e2, e3;  // cumulative stage counts
};

struct Block {
    int32_t kind;
    int32_t base;   // CONTIG/TILE: sequence position of the stage's first key
    int32_t first;  // SHARED: index of the stage's first key among the shared tokens
    int32_t cnt;    // keys present in the stage (<= BN)
    bool fast;      // no per-key mask needed
};

// Per-item values the key masks need.
struct MaskCtx {
    int32_t o, r_start, r_len, label_mask;
};

// Work item of workgroup pid: its (batch, head) slice bh and its index r
// within the slice (r < dense_row_blocks * n_chunks: a dense item).  Items
// of a slice are contiguous in the logical order (dense first), and the
// logical order is dealt to the 8 XCDs in contiguous ranges, so the items of
// a slice, which share K and V, meet in one L2.  Workgroups go to the XCDs
// round-robin (pid mod 8); within its range an XCD takes every dense item
// before any sparse one: the long items start first and the short ones fill
// the end of the launch.
struct ItemId {
    int32_t bh, r;
};

__device__ __forceinline__ ItemId decode_item(int pid, const AttnArgs& a) {
    constexpr int X = 8;
    const int total = a.total_items;
    const int per = (total + X - 1) / X;
    int tall = total % X;
    if (tall == 0) tall = X;
    const int xcd = pid % X;
    const int local = pid / X;
    const int lo = xcd < tall ? xcd * per : tall * per + (xcd - tall) * (per - 1);
    const int hi = lo + (xcd < tall ? per : per - 1);
    const int ipb = a.items_per_bh;
    const int di = a.dense_row_blocks * a.n_chunks;  // dense items per slice
    const int si = ipb - di;
    // dense items before logical position x
    auto dense_before = [&](int x) { return (x / ipb) * di + min(x % ipb, di); };
    const int fl = dense_before(lo);
    const int nd = dense_before(hi) - fl;
    int item;
    if (local < nd) {  // the range holds a dense item, so di > 0
        const int k = fl + local;
        item = (k / di) * ipb + k % di;
    } else {  // and here a sparse one, so si > 0
        const int k = (lo - fl) + (local - nd);
        item = (k / si) * ipb + di + k % si;
    }
    ItemId id;
    id.bh = item / ipb;
    id.r = item - id.bh * ipb;
    return id;
}

__device__ __forceinline__ int32_t shared_seq(const Spans& sp, int32_t u) {
    return sp.map[u];  // u < cum[n] <= kMaxShared
}

// The runs are ascending and disjoint (the table's contract), so the one
// that could hold seq is the last run starting at or before it: a binary
// search over the starts.
__device__ __forceinline__ bool is_shared_seq(const Spans& sp, int32_t seq) {
    int32_t lo = 0, hi = sp.n - 1;
    if (hi < 0 || seq < sp.start[0]) return false;
    while (lo < hi) {
        const int32_t mid = (lo + hi + 1) >> 1;
        if (sp.start[mid] <= seq) lo = mid;
        else hi = mid - 1;
    }
    return seq < sp.start[lo] + sp.len[lo];
}

// Combine the two lane halves (lanes l and l^32 hold the same query row).
__device__ __forceinline__ float half_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// IEEE maximum (NaN-propagating), v_maximum_f32 / v_maximum3_f32 on gfx950
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

__device__ __forceinline__ float half_vmax(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return vmax(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float half_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ int32_t tile_label(int32_t p, int32_t o, int32_t tile, int32_t n_img) {
    return ((p + o) % n_img) / tile;
}

// Is image position p (0 <= p < n_img) a cell of the grid, not padding?
__device__ __forceinline__ bool pos_valid(const AttnArgs& a, int32_t p) {
    uint32_t x, y;
    hilbert_d2xy(a.order, (uint32_t)p, x, y);
    return x < (uint32_t)a.grid_w && y < (uint32_t)a.grid_h;
}

// Is sequence position seq a padding slot?
__device__ __forceinline__ bool seq_padding(const AttnArgs& a, int32_t seq) {
    return a.padded && seq >= a.n_txt && !pos_valid(a, seq - a.n_txt);
}

template <int BN>
__device__ __forceinline__ Block block_at(int32_t i, int32_t b0, int32_t b1, int32_t b2, int32_t b3,
                                          int32_t l0, int32_t l1, int32_t l2, int32_t l3,
                                          int32_t k0, int32_t k1, int32_t k2, int32_t k3,
                                          int32_t e0, int32_t e1, int32_t e2, int32_t label_mask) {
    const bool in0 = i < e0, in1 = i < e1, in2 = i < e2;
    const int32_t kind = in0 ? k0 : in1 ? k1 : in2 ? k2 : k3;
    const int32_t base = in0 ? b0 : in1 ? b1 : in2 ? b2 : b3;
    const int32_t len = in0 ? l0 : in1 ? l1 : in2 ? l2 : l3;
    const int32_t before = in0 ? 0 : in1 ? e0 : in2 ? e1 : e2;
    Block b;
    b.kind = kind;
    b.first = (i - before) * BN;
    b.base = base + b.first;
    b.cnt = min(BN, len - b.first);
    // label_mask bit 0: per-row tile labels; bit 1: the image span has
    // padding, so every stage takes the per-key masks
    b.fast = b.cnt == BN && !(label_mask & 2) && (kind == SEG_CONTIG || (kind == SEG_TILE && !(label_mask & 1)));
    return b;
}

#define BLOCK_AT(BN, i, g, lm)                                                                      \
    block_at<BN>((i), (g).b0, (g).b1, (g).b2, (g).b3, (g).l0, (g).l1, (g).l2, (g).l3, (g).k0,        \
                 (g).k1, (g).k2, (g).k3, (g).e0, (g).e1, (g).e2, (lm))

template <int BN>
__device__ __forceinline__ Segs make_segs(int32_t b0, int32_t l0, int32_t k0, int32_t b1, int32_t l1,
                                          int32_t k1, int32_t b2, int32_t l2, int32_t k2, int32_t b3,
                                          int32_t l3, int32_t k3) {
    Segs g;
    g.b0 = b0; g.l0 = l0; g.k0 = k0;
    g.b1 = b1; g.l1 = l1; g.k1 = k1;
    g.b2 = b2; g.l2 = l2; g.k2 = k2;
    g.b3 = b3; g.l3 = l3; g.k3 = k3;
    g.e0 = (l0 + BN - 1) / BN;
    g.e1 = g.e0 + (l1 + BN - 1) / BN;
    g.e2 = g.e1 + (l2 + BN - 1) / BN;
    g.e3 = g.e2 + (l3 + BN - 1) / BN;
    return g;
}

__device__ __forceinline__ int32_t key_seq(const Block& b, int32_t r, const Spans& sp) {
    const int32_t rr = r < b.cnt ? r : 0;  // absent keys read a present row
    if (b.kind == SEG_SHARED) return shared_seq(sp, b.first + rr);
    return b.base + rr;
}

// What key r of a stage is to the rows: kKeyInvalid (absent, or a shared key
// counted in the tile segment), kKeyAll, or the key's tile label (rows of
// other tiles must not see it).
__device__ __forceinline__ int32_t key_info(const Block& b, int32_t r, int32_t seq, MaskCtx it,
                                            const AttnArgs& a, const Spans& sp) {
    if (r >= b.cnt) return kKeyInvalid;
    if (b.kind != SEG_SHARED && seq_padding(a, seq)) return kKeyInvalid;
    if (b.kind == SEG_CONTIG) return kKeyAll;
    const int32_t p = seq - a.n_txt;
    if (b.kind == SEG_SHARED) {
        const int32_t rel = (p - it.r_start + a.n_img) % a.n_img;
        return rel < it.r_len ? kKeyInvalid : kKeyAll;
    }
    if (!it.label_mask || is_shared_seq(sp, seq)) return kKeyAll;
    return tile_label(p, it.o, a.tile, a.n_img);
}

// Loads the layer's shared runs into LDS and builds the shared-token map
// (HilbertA only); returns the slide offset o.  Ends with a barrier.
template <int NT>
__device__ __forceinline__ int32_t load_spans(const AttnArgs& a, Spans& sp, int tid) {
    int32_t o = 0;
    if (a.sparse) {
        const int32_t n_sp = min(max(a.sched[6], 0), min(a.span_cap, kMaxSpans));
        const int32_t* tab = a.sched + 12 + 4 * a.n_tiles;
        for (int s = tid; s < n_sp; s += NT) {
            const int32_t st0 = min(max(tab[2 * s], a.n_txt), a.n_tot);
            sp.start[s] = st0;
            sp.len[s] = min(max(tab[2 * s + 1], 0), a.n_tot - st0);
        }
        __syncthreads();
        if (tid == 0) {
            int32_t c = 0;
            for (int s = 0; s < n_sp; ++s) {
                sp.cum[s] = min(c, kMaxShared);
                c += sp.len[s];
            }
            sp.cum[n_sp] = min(c, kMaxShared);
            sp.n = n_sp;
        }
        __syncthreads();
        // token u belongs to the last run whose prefix count is <= u
        for (int u = tid; u < sp.cum[n_sp]; u += NT) {
            int32_t lo = 0, hi = n_sp - 1;
            while (lo < hi) {
                const int32_t mid = (lo + hi + 1) >> 1;
                if (sp.cum[mid] <= u) lo = mid;
                else hi = mid - 1;
            }
            sp.map[u] = sp.start[lo] + (u - sp.cum[lo]);
        }
        const int32_t o_raw = a.sched[5];
        o = ((o_raw % a.n_img) + a.n_img) % a.n_img;
    } else if (tid == 0) {
        sp.n = 0;
        sp.cum[0] = 0;
    }
    __syncthreads();
    return o;
}

// Key segments and mask context of an item whose first row is row0 (image
// position for sparse items), block_m rows per item, BN keys per stage.
template <int BN>
__device__ __forceinline__ Segs item_segments(const AttnArgs& a, bool dense, int32_t chunk,
                                              int32_t row0, int32_t block_m, int32_t n_shared,
                                              MaskCtx& mc) {
    if (dense) {
        const int32_t k0 = chunk * a.chunk_keys;
        return make_segs<BN>(k0, min(a.chunk_keys, a.n_tot - k0), SEG_CONTIG, 0, 0, SEG_CONTIG, 0, 0,
                             SEG_CONTIG, 0, 0, SEG_CONTIG);
    }
    const int32_t p_last = min(a.n_img, row0 + block_m) - 1;
    // tiles covering the rows: in the slid coordinate s = (p + o) mod N_img
    // the rows are the cyclic run s0 .. s0 + L - 1, which meets the labels
    // q1, q1 + 1, ... (mod T); a run as long as the image meets all T
    const int32_t s0 = (row0 + mc.o) % a.n_img;
    const int32_t run = p_last - row0 + 1;
    const int32_t q1 = s0 / a.tile;
    const int32_t n_lab = min(a.n_tiles, (s0 + run - 1) / a.tile - q1 + 1);
    mc.label_mask = n_lab > 1;
    mc.r_start = (int32_t)(((int64_t)q1 * a.tile - mc.o + a.n_img) % a.n_img);
    mc.r_len = min(n_lab * a.tile, a.n_img);
    const int32_t len_a = min(mc.r_len, a.n_img - mc.r_start);
    // segments: text, shared (gathered), covering tiles, wrapped tail
    return make_segs<BN>(0, a.n_txt, SEG_CONTIG, 0, n_shared, SEG_SHARED, a.n_txt + mc.r_start, len_a,
                         SEG_TILE, a.n_txt, mc.r_len - len_a, SEG_TILE);
}

// One query row of an item: its sequence position, whether this item
// stores it, its dense-row index (dense items) and its tile label.
struct RowInfo {
    int32_t qseq;
    int32_t dense_row;
    int32_t label;
    bool store;
    bool pad;  // a padding row: stored as O = 0, LSE = -inf
};

__device__ __forceinline__ RowInfo row_info(const AttnArgs& a, bool dense, int32_t row0,
                                            int32_t rr, int32_t block_m, int32_t o,
                                            int32_t n_shared, const Spans& sp) {
    RowInfo ri{0, -1, -3, false, false};
    if (dense) {
        ri.dense_row = row0 + rr;
        if (ri.dense_row < a.n_dense_rows) {
            if (!a.sparse || ri.dense_row < a.n_txt) {
                ri.qseq = ri.dense_row;
                ri.store = true;
            } else if (ri.dense_row - a.n_txt < n_shared) {
                ri.qseq = shared_seq(sp, ri.dense_row - a.n_txt);
                ri.store = true;
            }
        }
    } else {
        const int32_t p = row0 + rr;
        const int32_t p_last = min(a.n_img, row0 + block_m) - 1;
        const bool ok = p < a.n_img;
        const int32_t pc = ok ? p : p_last;
        ri.qseq = a.n_txt + pc;
        ri.store = ok && !is_shared_seq(sp, ri.qseq);
        ri.label = tile_label(pc, o, a.tile, a.n_img);
        ri.pad = ok && seq_padding(a, ri.qseq);
    }
    return ri;
}

// K and V rows are fetched with buffer loads: the resource holds the (batch,
// head) slice's base address and its size, each thread's byte offset of the
// rows it stages is fixed for the whole item, and a stage of contiguous keys
// adds one uniform offset.  The whole offset travels in the per-lane operand,
// which the hardware checks against the slice size: rows past the slice read
// as zero instead of touching memory outside it.
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t slice_rsrc(const void* base, int64_t rows,
                                                             int64_t row_stride, int d, int esize) {
    const int64_t bytes = ((rows - 1) * row_stride + d) * esize;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRsrcWord3);
}

template <typename T>
__device__ __forceinline__ void store4(T* dst, float a, float b, float c, float d);

template <>
__device__ __forceinline__ void store4<__bf16>(__bf16* dst, float a, float b, float c, float d) {
    typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
    bf16x4 v = {(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
    *reinterpret_cast<bf16x4*>(dst) = v;
}

template <>
__device__ __forceinline__ void store4<float>(float* dst, float a, float b, float c, float d) {
    *reinterpret_cast<f32x4*>(dst) = f32x4{a, b, c, d};
}

// Final write of one lane's row: normalised O and LSE, or (split dense
// items) the chunk's partial (acc, m, l) for the merge kernel.  acc holds
// O^T rows d = 32 dt + 8 (i/4) + 4 h + i%4 of this lane's query row.
template <typename T, int D>
__device__ __forceinline__ void store_row(const AttnArgs& a, const RowInfo& ri, int32_t bh,
                                          int32_t chunk, bool dense, int h, float m_run, float l_run,
                                          const f32x16 acc[D / 32], T* obase) {
    const float l_tot = half_sum(l_run);
    if (dense && a.n_chunks > 1) {
        if (ri.dense_row >= 0 && ri.dense_row < a.n_dense_rows) {
            const int64_t slot = ((int64_t)bh * a.n_chunks + chunk) * a.n_dense_rows + ri.dense_row;
            float* wacc = a.ws + slot * D;
#pragma unroll
            for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    *reinterpret_cast<f32x4*>(wacc + 32 * dt + 8 * g + 4 * h) =
                        f32x4{acc[dt][4 * g], acc[dt][4 * g + 1], acc[dt][4 * g + 2], acc[dt][4 * g + 3]};
            if (h == 0) {
                float* wml = a.ws + (int64_t)a.n_bh * a.n_chunks * a.n_dense_rows * D + slot * 2;
                wml[0] = m_run;
                wml[1] = l_tot;
            }
        }
        return;
    }
    if (!ri.store) return;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    T* orow = obase + (int64_t)ri.qseq * a.o_sr;
    if (ri.pad) {
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
            for (int g = 0; g < 4; ++g) store4<T>(orow + 32 * dt + 8 * g + 4 * h, 0.f, 0.f, 0.f, 0.f);
        if (a.lse && h == 0) a.lse[(int64_t)bh * a.n_tot + ri.qseq] = -INFINITY;
        return;
    }
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int g = 0; g < 4; ++g)
            store4<T>(orow + 32 * dt + 8 * g + 4 * h, acc[dt][4 * g] * inv, acc[dt][4 * g + 1] * inv,
                      acc[dt][4 * g + 2] * inv, acc[dt][4 * g + 3] * inv);
    if (a.lse && h == 0)
        a.lse[(int64_t)bh * a.n_tot + ri.qseq] = l_tot > 0.f ? (m_run + log2f(l_tot)) * kLn2 : -INFINITY;
}

}  // namespace
}  // namespace hilberta
