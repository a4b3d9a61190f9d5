// Internal declarations shared by the host-side C ABI (abi.cpp) and the HIP
// kernel translation units.  Nothing here is part of the public interface.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hilberta {

// ---------------------------------------------------------------- attention
// Work decomposition of one attention launch.  Per (batch, head) there are
//   dense items:  dense_row_blocks x n_chunks, rows attending every key of
//                 one key chunk (text + shared rows for HilbertA, all rows
//                 for the dense baseline);
//   sparse items: sparse_blocks query blocks of image rows (HilbertA only).
// Items of one (batch, head) are contiguous in the logical order, dense
// first, and the logical order is spread over the XCDs in contiguous ranges.
constexpr int kBlockM = 128;  // query rows per workgroup, fp32 kernel (4 waves x 32)
constexpr int kBlockMBf16 = 128;  // query rows per workgroup, bf16 kernel (4 waves x 32)
constexpr int kBlockN = 64;   // keys per pipeline stage
constexpr int kThreads = 256;
constexpr int kMaxSpans = 256;   // shared runs a workgroup can hold in LDS
constexpr int kMaxShared = 1024; // shared tokens a workgroup can map in LDS (32 x 32)

struct AttnArgs {
    const void* q;
    const void* k;
    const void* v;
    void* o;
    float* lse;      // [B*H*N_tot] or null
    float* ws;       // split-key partials (n_chunks > 1) or null
    const int32_t* sched;  // schedule table (sparse mode) or null
    int64_t q_sb, q_sh, q_sr;  // element strides: batch, head, row
    int64_t k_sb, k_sh, k_sr;
    int64_t v_sb, v_sh, v_sr;
    int64_t o_sb, o_sh, o_sr;
    float scale_log2;  // softmax scale * log2(e)
    int32_t heads;
    int32_t n_tot;
    int32_t n_txt;
    int32_t n_img;
    int32_t tile;        // N_T (sparse mode)
    int32_t n_tiles;     // T (sparse mode)
    int32_t span_cap;    // span capacity of the table (sparse mode)
    int32_t n_shared;    // shared tokens expected from the config
    int32_t n_dense_rows;
    int32_t dense_row_blocks;
    int32_t n_chunks;
    int32_t chunk_keys;  // multiple of kBlockN
    int32_t sparse_blocks;
    int32_t items_per_bh;
    int32_t total_items;
    int32_t n_bh;        // batch * heads
    int32_t sparse;      // 1: HilbertA pattern, 0: dense baseline
    // general shapes: the image span holds the 2^order x 2^order curve
    // positions of the enclosing square, those whose cell lies outside the
    // grid_h x grid_w grid being padding (masked as keys and queries)
    int32_t padded;      // 1 when some image positions are padding
    int32_t order;
    int32_t grid_h, grid_w;
};

struct MergeArgs {
    void* o;
    float* lse;
    const float* ws;
    const int32_t* sched;
    int64_t o_sb, o_sh, o_sr;
    int32_t heads;
    int32_t n_tot;
    int32_t n_txt;
    int32_t span_cap;
    int32_t n_dense_rows;
    int32_t n_chunks;
    int32_t n_bh;
    int32_t n_tiles;
    int32_t sparse;
};

// Launchers (attn.hip, attn_bf16.hip); return a hipError_t.
hipError_t launch_attn(const AttnArgs& a, int dtype, int head_dim, hipStream_t s);
hipError_t launch_attn_bf16(const AttnArgs& a, int head_dim, hipStream_t s);
hipError_t launch_merge(const MergeArgs& m, int dtype, int head_dim, hipStream_t s);

// Backward (attn_bwd.hip): the forward's AttnArgs (Q, K, V, O and their
// strides, the item decomposition without split key passes) plus these.
// dO shares O's strides, dQ Q's, dK K's and dV V's.
struct BwdArgs {
    const void* dout;
    const float* lse;   // natural-log LSE of the forward, [B*H*N_tot]
    void* dq;
    void* dk;
    void* dv;
    float* delta;       // workspace: dO . O per row, [B*H*N_tot]
    float* lse2;        // workspace: LSE in log2 units (0 for empty rows)
};
hipError_t launch_attn_bwd(const AttnArgs& a, const BwdArgs& g, int head_dim, hipStream_t s);
hipError_t launch_attn_bwd_f32(const AttnArgs& a, const BwdArgs& g, int head_dim, hipStream_t s);

// ----------------------------------------------------- permutation, schedule
// perm[d] for the side x side curve positions: the raster index of the
// grid_h x grid_w grid's cell at d, or -1 for a padding slot
hipError_t launch_build_perm(int32_t side, int32_t grid_h, int32_t grid_w, int32_t* perm, int32_t* inv,
                             hipStream_t s);
hipError_t launch_build_perm_moved(int32_t side, int32_t shared_h, int32_t shared_w, int32_t* perm,
                                   int32_t* inv, hipStream_t s);

struct ScheduleArgs {
    int32_t* out;
    int32_t grid_h, grid_w, n_txt, tile, n_tiles, shared_h, shared_w;
    int32_t side;       // side of the square the curve runs over
    int32_t prefix;     // global prefix: n_txt, plus the shared tokens when moved
    int32_t tiled;      // tokens of the tiled span: N_img, or N_img - N_sh when moved
    int32_t moved;      // 1: shared tokens gathered next to the text
    int32_t layer;
    int32_t offset;     // (layer * delta) mod tiled, computed on the host in 64 bits
    int32_t span_cap;
    int32_t words;
};
hipError_t launch_schedule(const ScheduleArgs& a, hipStream_t s);

struct PermuteArgs {
    const char* x;
    char* y;
    const int32_t* perm;
    int64_t batch, n;
    int64_t row_bytes;
    int64_t x_bs, x_rs, y_bs, y_rs;  // strides in bytes
    int32_t scatter;                  // 0 gather, 1 scatter
};
hipError_t launch_permute(const PermuteArgs& a, hipStream_t s);

}  // namespace hilberta
