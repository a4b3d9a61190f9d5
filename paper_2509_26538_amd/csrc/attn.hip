// HilbertA sparse attention forward and the dense baseline (§3.2-§3.4,
// Appendix A, Algorithm 1), for gfx950.
//
// One launch covers every row of every (batch, head).  A workgroup of four
// wavefronts owns a work item: 128 query rows and an ordered list of key
// segments.  Keys stream through LDS in stages of 64 (double-buffered, the
// next stage prefetched into registers while the current one is consumed).
// Each wavefront owns 32 query rows and computes, per stage,
//   S^T = K Q^T   with the MFMA (bf16: v_mfma_f32_32x32x16_bf16,
//                 fp32: v_mfma_f32_32x32x2_f32),
// so that every lane holds one query row and 32 of the 64 keys: the online
// softmax (Algorithm 1's attn_inner: running max m, sum l, accumulator) is
// per lane, with one cross-lane exchange for the row maximum.  Then
//   O^T += V^T P^T,
// where P^T is fed straight from the score registers.  The MFMA's reduction
// index is free to enumerate the 16 keys of a chunk in any order, so V^T is
// staged in LDS in exactly the key order the score registers hold; no
// register shuffle of P is needed.
//
// Work items per (batch, head):
//   dense items  -- rows that attend every key: the text and shared rows of
//                   HilbertA (Appendix A treats both as a global prefix that
//                   attends everything), or all rows of the dense baseline.
//                   Their keys may be split into chunks whose partial
//                   (acc, m, l) are merged by a second small kernel.
//   sparse items -- 128 consecutive image rows.  Keys: the text span, the
//                   shared tokens (gathered), and the slid tile(s) covering
//                   the rows.  A tile that runs past the end of the image
//                   span continues at its head (the modular indexing of
//                   §3.2): two contiguous segments, addressed in place.
// Each key is visited once: shared keys that also lie in the rows' tiles are
// masked in the shared segment.  Rows of shared tokens inside a sparse item
// are computed by the dense items and not stored here.
#include "internal.hpp"

#include <type_traits>

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
constexpr int kMaxSegs = 4;
constexpr float kLn2 = 0.69314718055994530942f;

struct Spans {
    int32_t start[kMaxSpans];  // sequence position of the run's first token
    int32_t len[kMaxSpans];
    int32_t cum[kMaxSpans + 1];  // shared tokens before the run
    int32_t n;
    int32_t map[kMaxShared];   // sequence position of the u-th shared token
};

template <typename T, int D>
struct Stage;

template <int D>
struct alignas(16) Stage<__bf16, D> {
    alignas(16) uint16_t k[2][kBlockN][D + 8];   // K rows, padded against bank conflicts
    alignas(16) uint16_t vt[2][D][kBlockN + 8];  // V^T in the key order of the P registers
    alignas(16) int32_t info[2][kBlockN];
};

template <int D>
struct alignas(16) Stage<float, D> {
    alignas(16) float k[2][kBlockN][D + 1];
    alignas(16) float v[2][kBlockN][D + 4];
    alignas(16) int32_t info[2][kBlockN];
};

// Uniform (per-workgroup) description of one work item's keys: at most four
// segments (text, gathered shared tokens, covering tiles, wrapped tail).
// Functions below take these as separate scalar arguments, never through a
// pointer, so that they stay in scalar registers (a field load through a
// selected pointer would pin the whole description in scratch memory).
struct Segs {
    int32_t b0, b1, b2, b3;  // sequence position of the first key (SHARED: 0)
    int32_t l0, l1, l2, l3;  // lengths
    int32_t k0, k1, k2, k3;  // kinds
    int32_t e0, e1, e2, e3;  // cumulative stage counts
};

struct Block {
    int32_t kind;
    int32_t base;   // CONTIG/TILE: sequence position of the block's first key
    int32_t first;  // SHARED: index of the block's first key among the shared tokens
    int32_t cnt;    // keys present in the block (<= kBlockN)
    bool fast;      // no per-key mask needed
};

// Per-item values the key masks need.
struct MaskCtx {
    int32_t o, r_start, r_len, label_mask;
};

__device__ __forceinline__ int remap_xcd(int pid, int total) {
    // Workgroups are dealt to the 8 XCDs round-robin; give each XCD one
    // contiguous range of logical items so the items of a (batch, head),
    // which share K and V, meet in one L2.
    constexpr int X = 8;
    const int per = (total + X - 1) / X;
    int tall = total % X;
    if (tall == 0) tall = X;
    const int xcd = pid % X;
    const int local = pid / X;
    if (xcd < tall) return xcd * per + local;
    return tall * per + (xcd - tall) * (per - 1) + local;
}

__device__ __forceinline__ int32_t shared_seq(const Spans& sp, int32_t u) {
    // sequence position of the u-th shared token (u < cum[n] <= kMaxShared)
    return sp.map[u];
}

__device__ __forceinline__ bool is_shared_seq(const Spans& sp, int32_t seq) {
    bool r = false;
    for (int32_t s = 0; s < sp.n; ++s) r |= (seq >= sp.start[s]) & (seq < sp.start[s] + sp.len[s]);
    return r;
}

// Combine the two lane halves (lanes l and l^32 hold the same query row).
__device__ __forceinline__ float half_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float half_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ int32_t tile_label(int32_t p, int32_t o, int32_t tile, int32_t n_img) {
    return ((p + o) % n_img) / tile;
}

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
    b.first = (i - before) * kBlockN;
    b.base = base + b.first;
    b.cnt = min(kBlockN, len - b.first);
    b.fast = b.cnt == kBlockN && (kind == SEG_CONTIG || (kind == SEG_TILE && !label_mask));
    return b;
}

#define BLOCK_AT(i, g, lm)                                                                     \
    block_at((i), (g).b0, (g).b1, (g).b2, (g).b3, (g).l0, (g).l1, (g).l2, (g).l3, (g).k0, (g).k1, \
             (g).k2, (g).k3, (g).e0, (g).e1, (g).e2, (lm))

__device__ __forceinline__ Segs make_segs(int32_t b0, int32_t l0, int32_t k0, int32_t b1, int32_t l1,
                                           int32_t k1, int32_t b2, int32_t l2, int32_t k2, int32_t b3,
                                           int32_t l3, int32_t k3) {
    Segs g;
    g.b0 = b0; g.l0 = l0; g.k0 = k0;
    g.b1 = b1; g.l1 = l1; g.k1 = k1;
    g.b2 = b2; g.l2 = l2; g.k2 = k2;
    g.b3 = b3; g.l3 = l3; g.k3 = k3;
    g.e0 = (l0 + kBlockN - 1) / kBlockN;
    g.e1 = g.e0 + (l1 + kBlockN - 1) / kBlockN;
    g.e2 = g.e1 + (l2 + kBlockN - 1) / kBlockN;
    g.e3 = g.e2 + (l3 + kBlockN - 1) / kBlockN;
    return g;
}

__device__ __forceinline__ int32_t key_seq(const Block& b, int32_t r, const Spans& sp) {
    const int32_t rr = r < b.cnt ? r : 0;  // absent keys read a present row
    if (b.kind == SEG_SHARED) return shared_seq(sp, b.first + rr);
    return b.base + rr;
}

__device__ __forceinline__ int32_t key_info(const Block& b, int32_t r, int32_t seq, MaskCtx it,
                                   const AttnArgs& a, const Spans& sp) {
    if (r >= b.cnt) return kKeyInvalid;
    if (b.kind == SEG_CONTIG) return kKeyAll;
    const int32_t p = seq - a.n_txt;
    if (b.kind == SEG_SHARED) {
        const int32_t rel = (p - it.r_start + a.n_img) % a.n_img;
        return rel < it.r_len ? kKeyInvalid : kKeyAll;  // counted in the tile segment
    }
    if (!it.label_mask || is_shared_seq(sp, seq)) return kKeyAll;
    return tile_label(p, it.o, a.tile, a.n_img);
}

// ------------------------------------------------------------- staging
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

template <typename T, int D>
struct Loader;

template <int D>
struct Loader<__bf16, D> {
    static constexpr int KCH = D / 8;                       // 16-byte chunks per K row
    static constexpr int KPT = kBlockN * KCH / kThreads;    // per thread
    static constexpr int VQ = D / 4;                        // 4-element quads per V row
    static constexpr int VUNITS = 8 * VQ;                   // (8-key group, quad) units
    u32x4 kr[KPT];
    u32x2 vr[8];
    int32_t info;
    __amdgpu_buffer_rsrc_t krs, vrs;
    int32_t krow_b;  // bytes per K row
    int32_t vrow_b;

    // row of the block (0..63) and column byte offset each staged piece uses
    __device__ __forceinline__ static int k_row(int tid, int j) { return (tid + kThreads * j) / KCH; }
    __device__ __forceinline__ static int k_colb(int tid, int j) { return ((tid + kThreads * j) % KCH) * 16; }
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
        if (tid < kBlockN) {
            info = b.fast ? kKeyAll : key_info(b, tid, key_seq(b, tid, sp), it, a, sp);
        }
    }

    __device__ __forceinline__ void store(Stage<__bf16, D>& st, int buf, int tid) const {
#pragma unroll
        for (int j = 0; j < KPT; ++j)
            *reinterpret_cast<u32x4*>(&st.k[buf][k_row(tid, j)][k_colb(tid, j) / 2]) = kr[j];
        if (tid < VUNITS) {
            const int dq = tid % VQ, g = tid / VQ;
            const int cc = g >> 1, hh = g & 1;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                // element e of each of the 8 keys; key j goes to slot j
                u32x4 w;
#pragma unroll
                for (int j = 0; j < 8; j += 2) {
                    const uint32_t lo = vr[j][e >> 1], hi = vr[j + 1][e >> 1];
                    w[j >> 1] = __builtin_amdgcn_perm(hi, lo, (e & 1) ? 0x07060302u : 0x05040100u);
                }
                *reinterpret_cast<u32x4*>(&st.vt[buf][4 * dq + e][16 * cc + 8 * hh]) = w;
            }
        }
        if (tid < kBlockN) st.info[buf][tid] = info;
    }
};

template <int D>
struct Loader<float, D> {
    static constexpr int CH = D / 4;                     // 16-byte chunks per row
    static constexpr int PT = kBlockN * CH / kThreads;   // per thread, each of K and V
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
            int32_t ko, vo, ks = 0, vs = 0;
            if (b.kind != SEG_SHARED) {
                ko = row * krow_b;
                vo = row * vrow_b;
                ks = b.base * krow_b;
                vs = b.base * vrow_b;
            } else {
                const int32_t seq = sp.map[min(b.first + row, n_shared - 1)];
                ko = seq * krow_b;
                vo = seq * vrow_b;
            }
            kr[j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(krs, ks + ko + colb_of(tid, j), 0, 0));
            vr[j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(vrs, vs + vo + colb_of(tid, j), 0, 0));
        }
        if (tid < kBlockN) {
            info = b.fast ? kKeyAll : key_info(b, tid, key_seq(b, tid, sp), it, a, sp);
        }
    }

    __device__ __forceinline__ void store(Stage<float, D>& st, int buf, int tid) const {
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
        if (tid < kBlockN) st.info[buf][tid] = info;
    }
};

// ------------------------------------------------------------- Q operand
template <typename T, int D>
struct QOperand;

template <int D>
struct QOperand<__bf16, D> {
    bf16x8 q[D / 16];  // Q[row][16 kc + 8 h .. + 8]
    __device__ __forceinline__ void load(const __bf16* qrow, int h) {
#pragma unroll
        for (int kc = 0; kc < D / 16; ++kc)
            q[kc] = *reinterpret_cast<const bf16x8*>(qrow + 16 * kc + 8 * h);
    }
};

template <int D>
struct QOperand<float, D> {
    float q[D / 2];  // Q[row][2 kc + h]
    __device__ __forceinline__ void load(const float* qrow, int h) {
#pragma unroll
        for (int kc = 0; kc < D / 2; ++kc) q[kc] = qrow[2 * kc + h];
    }
};

// S^T for the 64 keys of a stage: s[kt] holds keys 32 kt + 8 (i/4) + 4 h + i%4
// (register i) against the lane's query row.
template <int D>
__device__ __forceinline__ void scores(const Stage<__bf16, D>& st, int buf, const QOperand<__bf16, D>& q,
                              int ql, int h, f32x16 s[2]) {
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
        f32x16 acc = {};
#pragma unroll
        for (int kc = 0; kc < D / 16; ++kc) {
            const bf16x8 a = *reinterpret_cast<const bf16x8*>(&st.k[buf][32 * kt + ql][16 * kc + 8 * h]);
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, q.q[kc], acc, 0, 0, 0);
        }
        s[kt] = acc;
    }
}

template <int D>
__device__ __forceinline__ void scores(const Stage<float, D>& st, int buf, const QOperand<float, D>& q,
                              int ql, int h, f32x16 s[2]) {
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
        f32x16 acc = {};
#pragma unroll
        for (int kc = 0; kc < D / 2; ++kc) {
            const float a = st.k[buf][32 * kt + ql][2 * kc + h];
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, q.q[kc], acc, 0, 0, 0);
        }
        s[kt] = acc;
    }
}

// O^T += V^T P^T.  acc[dt] holds O^T rows d = 32 dt + 8 (i/4) + 4 h + i%4.
template <int D>
__device__ __forceinline__ void accumulate(const Stage<__bf16, D>& st, int buf, const f32x16 p[2], int ql,
                                  int h, f32x16 acc[D / 32]) {
    bf16x8 pb[4];
#pragma unroll
    for (int cc = 0; cc < 4; ++cc) {
#pragma unroll
        for (int j = 0; j < 8; ++j) pb[cc][j] = (__bf16)p[cc >> 1][8 * (cc & 1) + j];
    }
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) {
            const bf16x8 a = *reinterpret_cast<const bf16x8*>(&st.vt[buf][32 * dt + ql][16 * cc + 8 * h]);
            acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[cc], acc[dt], 0, 0, 0);
        }
    }
}

template <int D>
__device__ __forceinline__ void accumulate(const Stage<float, D>& st, int buf, const f32x16 p[2], int ql,
                                  int h, f32x16 acc[D / 32]) {
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int key = 32 * kt + 8 * (i >> 2) + 4 * h + (i & 3);
                const float a = st.v[buf][key][32 * dt + ql];
                acc[dt] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, p[kt][i], acc[dt], 0, 0, 0);
            }
        }
    }
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
    *reinterpret_cast<float4*>(dst) = make_float4(a, b, c, d);
}

// ------------------------------------------------------------- the kernel
template <typename T, int D>
struct Smem {
    Stage<T, D> st;
    Spans sp;
};

// bf16: two workgroups per CU (LDS and registers fit twice); fp32: one.
template <typename T>
struct Occupancy {
    static constexpr int value = std::is_same<T, float>::value ? 1 : 2;
};

template <typename T, int D>
__global__ void __launch_bounds__(kThreads, Occupancy<T>::value) attn_kernel(AttnArgs a) {
    __shared__ Smem<T, D> sm;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int h = lane >> 5;
    const int ql = lane & 31;

    // ---- work item
    const int item = remap_xcd(blockIdx.x, a.total_items);
    const int32_t bh = item / a.items_per_bh;
    const int32_t r = item - bh * a.items_per_bh;
    const int32_t dense_items = a.dense_row_blocks * a.n_chunks;
    const bool dense = r < dense_items;
    MaskCtx mc{0, 0, 0, 0};

    // ---- shared runs of the layer's table (HilbertA only)
    if (a.sparse) {
        const int32_t n_sp = min(max(a.sched[6], 0), min(a.span_cap, kMaxSpans));
        const int32_t* tab = a.sched + 12 + 4 * a.n_tiles;
        for (int s = tid; s < n_sp; s += kThreads) {
            const int32_t st0 = min(max(tab[2 * s], a.n_txt), a.n_tot);
            sm.sp.start[s] = st0;
            sm.sp.len[s] = min(max(tab[2 * s + 1], 0), a.n_tot - st0);
        }
        __syncthreads();
        if (tid == 0) {
            int32_t c = 0;
            for (int s = 0; s < n_sp; ++s) {
                sm.sp.cum[s] = min(c, kMaxShared);
                c += sm.sp.len[s];
            }
            sm.sp.cum[n_sp] = min(c, kMaxShared);
            sm.sp.n = n_sp;
        }
        __syncthreads();
        // the gathered shared segment reads its keys through this map
        for (int u = tid; u < sm.sp.cum[n_sp]; u += kThreads) {
            int32_t s = 0;
            while (s + 1 < n_sp && u >= sm.sp.cum[s + 1]) ++s;
            sm.sp.map[u] = sm.sp.start[s] + (u - sm.sp.cum[s]);
        }
        const int32_t o = a.sched[5];
        mc.o = ((o % a.n_img) + a.n_img) % a.n_img;
    } else if (tid == 0) {
        sm.sp.n = 0;
        sm.sp.cum[0] = 0;
    }
    __syncthreads();
    const int32_t n_shared = a.sparse ? sm.sp.cum[sm.sp.n] : 0;

    // ---- this lane's query row and the item's key segments
    int32_t qseq = 0;        // sequence position of the row
    bool store_row = false;  // this item writes the row
    int32_t dense_row = -1;  // dense items: row index among the dense rows
    int32_t row_label = -3;
    int32_t chunk = 0;
    Segs g;
    if (dense) {
        const int32_t rb = r / a.n_chunks;
        chunk = r - rb * a.n_chunks;
        dense_row = rb * kBlockM + wave * 32 + ql;
        if (dense_row < a.n_dense_rows) {
            if (!a.sparse || dense_row < a.n_txt) {
                qseq = dense_row;
                store_row = true;
            } else if (dense_row - a.n_txt < n_shared) {
                qseq = shared_seq(sm.sp, dense_row - a.n_txt);
                store_row = true;
            }
        }
        const int32_t k0 = chunk * a.chunk_keys;
        g = make_segs(k0, min(a.chunk_keys, a.n_tot - k0), SEG_CONTIG, 0, 0, SEG_CONTIG, 0, 0,
                      SEG_CONTIG, 0, 0, SEG_CONTIG);
    } else {
        const int32_t row0 = (r - dense_items) * kBlockM;
        const int32_t p = row0 + wave * 32 + ql;
        const int32_t p_last = min(a.n_img, row0 + kBlockM) - 1;
        const bool row_ok = p < a.n_img;
        const int32_t pc = row_ok ? p : p_last;
        qseq = a.n_txt + pc;
        store_row = row_ok && !is_shared_seq(sm.sp, qseq);
        row_label = tile_label(pc, mc.o, a.tile, a.n_img);
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
        g = make_segs(0, a.n_txt, SEG_CONTIG, 0, n_shared, SEG_SHARED, a.n_txt + mc.r_start, len_a,
                      SEG_TILE, a.n_txt, mc.r_len - len_a, SEG_TILE);
    }

    const int32_t bb = bh / a.heads;
    const int32_t hh = bh - bb * a.heads;
    const T* qb = reinterpret_cast<const T*>(a.q) + bb * a.q_sb + hh * a.q_sh;
    const T* kb = reinterpret_cast<const T*>(a.k) + bb * a.k_sb + hh * a.k_sh;
    const T* vb = reinterpret_cast<const T*>(a.v) + bb * a.v_sb + hh * a.v_sh;

    QOperand<T, D> qop;
    qop.load(qb + (int64_t)qseq * a.q_sr, h);

    f32x16 acc[D / 32];
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) acc[dt] = f32x16{};
    float m_run = -INFINITY;  // reference max of the scaled logits, log2 units
    float l_run = 0.f;        // this lane's share of the running sum
    const float c = a.scale_log2;

    // ---- key stages
    // Stage i is consumed from LDS buffer i&1.  At the top of iteration i the
    // registers hold stage i+1 (loaded during iteration i-1); they go to the
    // other buffer, and stage i+2 is requested, so its global loads are in
    // flight while stage i is computed.
    Loader<T, D> ld;
    ld.init(kb, vb, a);
    const int nblk = g.e3;
    if (nblk > 0) {
        ld.load(BLOCK_AT(0, g, mc.label_mask), mc, a, sm.sp, tid, n_shared);
        ld.store(sm.st, 0, tid);
        if (nblk > 1) ld.load(BLOCK_AT(1, g, mc.label_mask), mc, a, sm.sp, tid, n_shared);
    }
    __syncthreads();
    for (int i = 0; i < nblk; ++i) {
        const int buf = i & 1;
        if (i + 1 < nblk) ld.store(sm.st, buf ^ 1, tid);
        if (i + 2 < nblk) ld.load(BLOCK_AT(i + 2, g, mc.label_mask), mc, a, sm.sp, tid, n_shared);
        const Block b = BLOCK_AT(i, g, mc.label_mask);
        f32x16 s[2];
        scores<D>(sm.st, buf, qop, ql, h, s);
        if (!b.fast) {
#pragma unroll
            for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int key = 32 * kt + 8 * (e >> 2) + 4 * h + (e & 3);
                    const int32_t inf = sm.st.info[buf][key];
                    const bool ok = inf == kKeyAll || inf == row_label;
                    s[kt][e] = ok ? s[kt][e] : -INFINITY;
                }
            }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[kt][e]);
        mx = half_max(mx) * c;
        // Lazy rescaling: the reference max only moves when some row's max
        // grew by more than 2^8; until then p <= 256 and acc and l share the
        // stale reference, which cancels in acc / l.
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
        float lsum = 0.f;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const float pe = __builtin_amdgcn_exp2f(fmaf(s[kt][e], c, -m_use));
                s[kt][e] = pe;
                lsum += pe;
            }
        l_run += lsum;
        accumulate<D>(sm.st, buf, s, ql, h, acc);
        __syncthreads();
    }

    // ---- finalize
    const float l_tot = half_sum(l_run);
    if (dense && a.n_chunks > 1) {
        // partial (acc, m, l) of this key chunk, merged by merge_kernel
        if (dense_row >= 0 && dense_row < a.n_dense_rows) {
            const int64_t slot = ((int64_t)bh * a.n_chunks + chunk) * a.n_dense_rows + dense_row;
            float* wacc = a.ws + slot * D;
#pragma unroll
            for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    *reinterpret_cast<float4*>(wacc + 32 * dt + 8 * g + 4 * h) =
                        make_float4(acc[dt][4 * g], acc[dt][4 * g + 1], acc[dt][4 * g + 2],
                                    acc[dt][4 * g + 3]);
            if (h == 0) {
                float* wml = a.ws + (int64_t)a.n_bh * a.n_chunks * a.n_dense_rows * D + slot * 2;
                wml[0] = m_run;
                wml[1] = l_tot;
            }
        }
        return;
    }
    if (!store_row) return;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    T* orow = reinterpret_cast<T*>(a.o) + bb * a.o_sb + hh * a.o_sh + (int64_t)qseq * a.o_sr;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int g = 0; g < 4; ++g)
            store4<T>(orow + 32 * dt + 8 * g + 4 * h, acc[dt][4 * g] * inv, acc[dt][4 * g + 1] * inv,
                      acc[dt][4 * g + 2] * inv, acc[dt][4 * g + 3] * inv);
    if (a.lse && h == 0) {
        a.lse[(int64_t)bh * a.n_tot + qseq] =
            l_tot > 0.f ? (m_run + log2f(l_tot)) * kLn2 : -INFINITY;
    }
}


// Merge of the split key chunks of dense rows: with chunk partials
// (acc_c, m_c, l_c), M = max m_c, L = sum l_c 2^(m_c - M) and
// O = sum acc_c 2^(m_c - M) / L -- the same rescaling Algorithm 1 applies
// between key blocks.  One wavefront per row.
template <typename T, int D>
__global__ void __launch_bounds__(256) merge_kernel(MergeArgs m) {
    constexpr int EPL = D / 64;  // elements per lane
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int64_t rowid = (int64_t)blockIdx.x * 4 + wave;
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
    float mx = -INFINITY;
    for (int c = 0; c < m.n_chunks; ++c) mx = fmaxf(mx, ml[(slot0 + (int64_t)c * m.n_dense_rows) * 2]);
    const float m_use = mx == -INFINITY ? 0.f : mx;
    float L = 0.f;
    float o[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[e] = 0.f;
    for (int c = 0; c < m.n_chunks; ++c) {
        const int64_t slot = slot0 + (int64_t)c * m.n_dense_rows;
        const float w = __builtin_amdgcn_exp2f(ml[slot * 2] - m_use);
        L += w * ml[slot * 2 + 1];
#pragma unroll
        for (int e = 0; e < EPL; ++e) o[e] += w * m.ws[slot * D + lane * EPL + e];
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    const int32_t b = bh / m.heads, hh = bh - b * m.heads;
    T* orow = reinterpret_cast<T*>(m.o) + b * m.o_sb + hh * m.o_sh + (int64_t)seq * m.o_sr;
#pragma unroll
    for (int e = 0; e < EPL; ++e) orow[lane * EPL + e] = (T)(o[e] * inv);
    if (m.lse && lane == 0)
        m.lse[(int64_t)bh * m.n_tot + seq] = L > 0.f ? (m_use + log2f(L)) * kLn2 : -INFINITY;
}

template <typename T, int D>
hipError_t launch_attn_t(const AttnArgs& a, hipStream_t s) {
    hipLaunchKernelGGL((attn_kernel<T, D>), dim3(a.total_items), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_merge_t(const MergeArgs& m, hipStream_t s) {
    const int64_t rows = (int64_t)m.n_bh * m.n_dense_rows;
    const int64_t blocks = (rows + 3) / 4;
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((merge_kernel<T, D>), dim3((unsigned)blocks), dim3(256), 0, s, m);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn(const AttnArgs& a, int dtype, int head_dim, hipStream_t s) {
    if (a.total_items == 0) return hipSuccess;
    if (dtype == 1) return head_dim == 128 ? launch_attn_t<__bf16, 128>(a, s) : launch_attn_t<__bf16, 64>(a, s);
    return head_dim == 128 ? launch_attn_t<float, 128>(a, s) : launch_attn_t<float, 64>(a, s);
}

hipError_t launch_merge(const MergeArgs& m, int dtype, int head_dim, hipStream_t s) {
    if (dtype == 1) return head_dim == 128 ? launch_merge_t<__bf16, 128>(m, s) : launch_merge_t<__bf16, 64>(m, s);
    return head_dim == 128 ? launch_merge_t<float, 128>(m, s) : launch_merge_t<float, 64>(m, s);
}

}  // namespace hilberta
