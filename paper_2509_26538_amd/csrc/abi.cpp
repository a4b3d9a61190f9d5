// Host side of the C ABI declared in include/hilberta.h: argument
// validation, the work plan of an attention launch, and the launches.
// Every check runs before the first HIP call, so all error paths can be
// exercised on a machine without a GPU.
#include "hilberta.h"

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

#include "internal.hpp"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int hip_status(hipError_t e, const char* what) {
    if (e == hipSuccess) return HILBERTA_OK;
    return fail(HILBERTA_EHIP, "%s: %s", what, hipGetErrorString(e));
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

// Side of the square the curve runs over: the grid itself when it is a
// square power of two, else the smallest enclosing power-of-two square, at
// least 2 x 2 (Appendix D).  Sides must lie in [1, 32768].
int32_t enclosing_side(int32_t grid_h, int32_t grid_w) {
    const int32_t m = grid_h > grid_w ? grid_h : grid_w;
    int32_t s = 2;
    while (s < m) s *= 2;
    return s;
}

int check_grid(int32_t grid_h, int32_t grid_w) {
    if (grid_h < 1 || grid_w < 1 || grid_h > 32768 || grid_w > 32768)
        return fail(HILBERTA_EUNSUPPORTED, "grid %dx%d: each side must lie in [1, 32768]", grid_h, grid_w);
    return HILBERTA_OK;
}

int check_config(const hilberta_config* c) {
    if (!c) return fail(HILBERTA_EINVAL, "config is NULL");
    if (c->layout != HILBERTA_LAYOUT_IN_PLACE && c->layout != HILBERTA_LAYOUT_MOVED)
        return fail(HILBERTA_EINVAL, "layout %d is neither in place (0) nor moved (1)", c->layout);
    if (int rc = check_grid(c->grid_h, c->grid_w)) return rc;
    const int32_t side = enclosing_side(c->grid_h, c->grid_w);
    const bool padded = (int64_t)side * side != (int64_t)c->grid_h * c->grid_w;
    if (padded && c->layout == HILBERTA_LAYOUT_MOVED)
        return fail(HILBERTA_EUNSUPPORTED, "the moved layout needs a square power-of-two grid, not %dx%d",
                    c->grid_h, c->grid_w);
    // the image span: every position of the curve, padding included
    const int64_t n_img = (int64_t)side * side;
    if (c->n_txt < 0) return fail(HILBERTA_EINVAL, "n_txt %d < 0", c->n_txt);
    if (c->n_txt + n_img > 0x7fffffffLL)
        return fail(HILBERTA_EUNSUPPORTED, "sequence of %lld tokens is too long",
                    (long long)(c->n_txt + n_img));
    if (c->tile < 1 || (c->layout != HILBERTA_LAYOUT_MOVED && n_img % c->tile))
        return fail(HILBERTA_EUNSUPPORTED, "tile %d does not divide %lld image tokens", c->tile,
                    (long long)n_img);
    if (c->delta < 0) return fail(HILBERTA_EINVAL, "delta %d < 0", c->delta);
    if (c->shared_h < 0 || c->shared_w < 0 || c->shared_h > c->grid_h || c->shared_w > c->grid_w)
        return fail(HILBERTA_EINVAL, "shared region %dx%d outside the grid", c->shared_h, c->shared_w);
    if ((c->shared_h == 0) != (c->shared_w == 0))
        return fail(HILBERTA_EINVAL, "shared region %dx%d: both sides or neither must be zero",
                    c->shared_h, c->shared_w);
    if ((int64_t)c->shared_h * c->shared_w > hilberta::kMaxShared)
        return fail(HILBERTA_EUNSUPPORTED, "shared region %dx%d has more than %d tokens", c->shared_h,
                    c->shared_w, hilberta::kMaxShared);
    if (c->shared_h + c->shared_w > 255)
        return fail(HILBERTA_EUNSUPPORTED, "shared region %dx%d: shared_h + shared_w must be <= 255",
                    c->shared_h, c->shared_w);
    if (c->layout == HILBERTA_LAYOUT_MOVED) {
        const int64_t tiled = n_img - (int64_t)c->shared_h * c->shared_w;
        if (tiled < 1 || tiled % c->tile)
            return fail(HILBERTA_EUNSUPPORTED, "tile %d does not divide the %lld tokens outside the shared region",
                        c->tile, (long long)tiled);
    }
    return HILBERTA_OK;
}

// The sequence a valid config describes: in place, all N_img image tokens
// are tiled and the shared ones keep their slots; moved, the shared tokens
// follow the text in the global prefix and the other N_img - N_sh are tiled.
struct Geom {
    int64_t prefix, tiled, shared_in_span, cap;
};

int64_t span_len(const hilberta_config* c) {
    const int64_t side = enclosing_side(c->grid_h, c->grid_w);
    return side * side;
}

Geom geom(const hilberta_config* c) {
    const int64_t n_img = span_len(c);
    const int64_t n_sh = (int64_t)c->shared_h * c->shared_w;
    Geom g{};
    if (c->layout == HILBERTA_LAYOUT_MOVED) {
        g.prefix = c->n_txt + n_sh;
        g.tiled = n_img - n_sh;
        g.shared_in_span = 0;
        g.cap = 0;
    } else {
        g.prefix = c->n_txt;
        g.tiled = n_img;
        g.shared_in_span = n_sh;
        g.cap = n_sh ? c->shared_h + c->shared_w + 1 : 0;
    }
    return g;
}

int64_t schedule_words(const hilberta_config* c) {
    const Geom g = geom(c);
    return 12 + 4 * (g.tiled / c->tile) + 2 * g.cap;
}

struct Tensor4 {
    const void* p;
    const int64_t* s;
    const char* name;
};

int check_attn_common(const Tensor4* t, int n_t, int64_t batch, int64_t heads, int64_t n,
                      int64_t head_dim, int dtype, float scale) {
    if (batch < 0 || heads < 0) return fail(HILBERTA_EINVAL, "negative batch or heads");
    if (head_dim != 64 && head_dim != 128)
        return fail(HILBERTA_EUNSUPPORTED, "head_dim %lld not in {64, 128}", (long long)head_dim);
    if (dtype != HILBERTA_F32 && dtype != HILBERTA_BF16)
        return fail(HILBERTA_EUNSUPPORTED, "dtype %d", dtype);
    if (!(scale > 0.f) || !std::isfinite(scale))
        return fail(HILBERTA_EINVAL, "scale must be finite and > 0");
    if (batch * heads > 0x7fffffffLL) return fail(HILBERTA_EUNSUPPORTED, "too many heads");
    if (batch * heads == 0 || n == 0) return HILBERTA_OK;  // nothing is read or written
    const int64_t align = dtype == HILBERTA_BF16 ? 8 : 4;  // elements in 16 bytes
    for (int i = 0; i < n_t; ++i) {
        if (!t[i].p) return fail(HILBERTA_EINVAL, "%s is NULL", t[i].name);
        if (!t[i].s) return fail(HILBERTA_EINVAL, "%s strides are NULL", t[i].name);
        if (t[i].s[3] != 1)
            return fail(HILBERTA_EUNSUPPORTED, "%s: dim stride must be 1", t[i].name);
        for (int j = 0; j < 3; ++j) {
            if (t[i].s[j] < 0) return fail(HILBERTA_EINVAL, "%s: negative stride", t[i].name);
            if (t[i].s[j] % align)
                return fail(HILBERTA_EUNSUPPORTED, "%s: stride %lld is not a multiple of %lld elements",
                            t[i].name, (long long)t[i].s[j], (long long)align);
        }
        if ((uintptr_t)t[i].p % 16)
            return fail(HILBERTA_EUNSUPPORTED, "%s is not 16-byte aligned", t[i].name);
    }
    return HILBERTA_OK;
}

// The work plan of one attention launch (see AttnArgs).  Depends only on the
// shapes, so the workspace query and the launch agree.
struct Plan {
    int64_t n_dense_rows, dense_row_blocks, n_chunks, chunk_keys, sparse_blocks, items_per_bh,
        total_items, ws_bytes;
};

// HilbertA: dense rows (text and shared) attend every key.  Their keys are
// split into chunks only as far as needed for no dense item to run longer
// than a workgroup slot's share of the whole launch (the visited row blocks
// x keys over 512 slots, two workgroups on each of 256 CUs), and never
// shorter than twice a sparse item's key list: each XCD starts its dense
// items first and its short sparse items fill the slots behind them, and the
// partials to merge stay few.  For the dense baseline, split only when the
// rows alone would not fill the GPU a few times.
Plan make_plan(bool sparse, int64_t n_txt, int64_t n_img, int64_t n_shared, int64_t tile,
               int64_t n_tot, int64_t bh, int64_t head_dim, int dtype, bool allow_split) {
    Plan p{};
    const int64_t bn = hilberta::kBlockN;
    const int64_t bm = dtype == HILBERTA_BF16 ? hilberta::kBlockMBf16 : hilberta::kBlockM;
    int64_t chunk = round_up(n_tot, bn);
    if (sparse) {
        p.n_dense_rows = n_txt + n_shared;
        p.sparse_blocks = ceil_div(n_img, bm);
        const int64_t sparse_keys = round_up(n_txt, bn) + round_up(n_shared, bn) +
                                    round_up(tile < n_img ? tile : n_img, bn);
        const int64_t work = bh * (ceil_div(p.n_dense_rows, bm) * n_tot + p.sparse_blocks * sparse_keys);
        const int64_t share = ceil_div(work, 512);
        const int64_t k = share > 0 ? ceil_div(n_tot, share) : 1;
        chunk = round_up(ceil_div(n_tot, k), bn);
        const int64_t floor_keys = round_up(2 * (sparse_keys > 512 ? sparse_keys : 512), bn);
        if (chunk < floor_keys) chunk = floor_keys;
    } else {
        p.n_dense_rows = n_tot;
        p.sparse_blocks = 0;
        const int64_t row_items = ceil_div(n_tot, bm) * bh;
        const int64_t want = 2048;  // about four rounds of workgroups on 256 CUs
        if (row_items < want) {
            int64_t k = ceil_div(want, row_items);
            const int64_t kmax = ceil_div(n_tot, 512);
            if (k > kmax) k = kmax;
            if (k < 1) k = 1;
            chunk = round_up(ceil_div(n_tot, k), bn);
        }
    }
    if (chunk > round_up(n_tot, bn)) chunk = round_up(n_tot, bn);
    if (!allow_split || chunk < bn) chunk = round_up(n_tot, bn);
    p.chunk_keys = chunk;
    p.n_chunks = n_tot > 0 ? ceil_div(n_tot, chunk) : 1;
    if (p.n_dense_rows == 0) p.n_chunks = 1;
    p.dense_row_blocks = ceil_div(p.n_dense_rows, bm);
    p.items_per_bh = p.dense_row_blocks * p.n_chunks + p.sparse_blocks;
    p.total_items = p.items_per_bh * bh;
    p.ws_bytes = p.n_chunks > 1 ? bh * p.n_chunks * p.n_dense_rows * (head_dim + 2) * 4 : 0;
    return p;
}

// Validates what the forward and the backward share (tensors t, shapes,
// dtype, scale) and builds the launch description.  Returns OK with *empty
// set when there is nothing to read or write.
int attn_setup(bool sparse, const hilberta_config* cfg, const int32_t* sched, const Tensor4* t, int n_t,
               int64_t batch, int64_t heads, int64_t n_tot, int64_t head_dim, int dtype, float scale,
               bool allow_split, Plan& p, hilberta::AttnArgs& a, bool& empty) {
    empty = false;
    int rc = check_attn_common(t, n_t, batch, heads, n_tot, head_dim, dtype, scale);
    if (rc) return rc;
    // the attention sees a global prefix and a tiled span (see Geom)
    int64_t n_txt = 0, n_img = n_tot, n_shared = 0, tile = n_tot, n_tiles = 1, cap = 0;
    if (sparse) {
        const Geom g = geom(cfg);
        n_txt = g.prefix;
        n_img = g.tiled;
        n_shared = g.shared_in_span;
        tile = cfg->tile;
        n_tiles = n_img / tile;
        cap = g.cap;
    }
    if (n_tot > 0x7fffffffLL) return fail(HILBERTA_EUNSUPPORTED, "sequence too long");
    const int64_t bh = batch * heads;
    if (bh == 0 || n_tot == 0) {
        empty = true;
        return HILBERTA_OK;
    }
    {
        // rows staged through LDS are addressed with 32-bit byte offsets
        // from their (batch, head) slice's base: K and V, and for the
        // backward Q and dO too (t[4] is dO, which shares O's strides)
        const int64_t es = dtype == HILBERTA_BF16 ? 2 : 4;
        int64_t rs = 0;
        for (int i = 0; i < n_t; ++i) {
            if (t[i].s[2] < head_dim) return fail(HILBERTA_EINVAL, "%s: row stride smaller than head_dim", t[i].name);
            if (i == 1 || i == 2 || n_t > 4) rs = t[i].s[2] > rs ? t[i].s[2] : rs;
        }
        if (((n_tot - 1) * rs + head_dim) * es > 0x7fffffffLL)
            return fail(HILBERTA_EUNSUPPORTED, "one (batch, head) slice of a staged tensor spans more than 2 GiB");
    }
    p = make_plan(sparse, n_txt, n_img, n_shared, tile, n_tot, bh, head_dim, dtype, allow_split);
    if (p.total_items > 0x7fffffffLL) return fail(HILBERTA_EUNSUPPORTED, "too many work items");
    const int64_t* qs = t[0].s;
    const int64_t* ks = t[1].s;
    const int64_t* vs = t[2].s;
    const int64_t* os = t[3].s;
    a = hilberta::AttnArgs{};
    a.q = t[0].p;
    a.k = t[1].p;
    a.v = t[2].p;
    a.o = const_cast<void*>(t[3].p);
    a.sched = sched;
    a.q_sb = qs[0]; a.q_sh = qs[1]; a.q_sr = qs[2];
    a.k_sb = ks[0]; a.k_sh = ks[1]; a.k_sr = ks[2];
    a.v_sb = vs[0]; a.v_sh = vs[1]; a.v_sr = vs[2];
    a.o_sb = os[0]; a.o_sh = os[1]; a.o_sr = os[2];
    a.scale_log2 = scale * 1.4426950408889634f;
    a.heads = (int32_t)heads;
    a.n_tot = (int32_t)n_tot;
    a.n_txt = (int32_t)n_txt;
    a.n_img = (int32_t)n_img;
    a.tile = (int32_t)tile;
    a.n_tiles = (int32_t)n_tiles;
    a.span_cap = (int32_t)cap;
    a.n_shared = (int32_t)n_shared;
    a.n_dense_rows = (int32_t)p.n_dense_rows;
    a.dense_row_blocks = (int32_t)p.dense_row_blocks;
    a.n_chunks = (int32_t)p.n_chunks;
    a.chunk_keys = (int32_t)p.chunk_keys;
    a.sparse_blocks = (int32_t)p.sparse_blocks;
    a.items_per_bh = (int32_t)p.items_per_bh;
    a.total_items = (int32_t)p.total_items;
    a.n_bh = (int32_t)bh;
    a.sparse = sparse ? 1 : 0;
    if (sparse && (int64_t)cfg->grid_h * cfg->grid_w != span_len(cfg)) {
        a.padded = 1;
        a.order = 31 - __builtin_clz((unsigned)enclosing_side(cfg->grid_h, cfg->grid_w));
        a.grid_h = cfg->grid_h;
        a.grid_w = cfg->grid_w;
    }
    return HILBERTA_OK;
}

int check_workspace(const void* ws, int64_t ws_bytes) {
    if (ws_bytes < 0 || (ws == nullptr && ws_bytes != 0))
        return fail(HILBERTA_EINVAL, "workspace NULL with %lld bytes", (long long)ws_bytes);
    if (ws && (uintptr_t)ws % 16) return fail(HILBERTA_EUNSUPPORTED, "workspace is not 16-byte aligned");
    return HILBERTA_OK;
}

// A validated attention call: its plan and launch description.  Built on the
// host with no HIP call, so every argument error returns before anything is
// launched.
struct AttnCall {
    Plan p;
    hilberta::AttnArgs a;
    bool empty;
};

int prepare_attention(bool sparse, const hilberta_config* cfg, const int32_t* sched, const void* q,
                      const void* k, const void* v, void* o, float* lse, int64_t batch, int64_t heads,
                      int64_t n_tot, int64_t head_dim, const int64_t* qs, const int64_t* ks,
                      const int64_t* vs, const int64_t* os, int dtype, float scale, bool split,
                      AttnCall& c) {
    const Tensor4 t[4] = {{q, qs, "q"}, {k, ks, "k"}, {v, vs, "v"}, {o, os, "o"}};
    c = AttnCall{};
    int rc = attn_setup(sparse, cfg, sched, t, 4, batch, heads, n_tot, head_dim, dtype, scale, split, c.p,
                        c.a, c.empty);
    if (rc || c.empty) return rc;
    c.a.lse = lse;
    return HILBERTA_OK;
}

// The attention launch, then (split dense rows) the merge of the chunk
// partials, which live in ws (at least c.p.ws_bytes).
int launch_attention(AttnCall& c, int dtype, int64_t head_dim, void* ws, hipStream_t s) {
    hilberta::AttnArgs& a = c.a;
    a.ws = static_cast<float*>(ws);
    int rc = hip_status(hilberta::launch_attn(a, dtype, (int)head_dim, s), "attention launch");
    if (rc || c.p.n_chunks == 1) return rc;
    hilberta::MergeArgs m{};
    m.o = a.o;
    m.lse = a.lse;
    m.ws = a.ws;
    m.sched = a.sched;
    m.o_sb = a.o_sb; m.o_sh = a.o_sh; m.o_sr = a.o_sr;
    m.heads = a.heads;
    m.n_tot = a.n_tot;
    m.n_txt = a.n_txt;
    m.span_cap = a.span_cap;
    m.n_dense_rows = a.n_dense_rows;
    m.n_chunks = a.n_chunks;
    m.n_bh = a.n_bh;
    m.n_tiles = a.n_tiles;
    m.sparse = a.sparse;
    return hip_status(hilberta::launch_merge(m, dtype, (int)head_dim, s), "merge launch");
}

int run_attention(bool sparse, const hilberta_config* cfg, const int32_t* sched, const void* q,
                  const void* k, const void* v, void* o, float* lse, int64_t batch, int64_t heads,
                  int64_t n_tot, int64_t head_dim, const int64_t* qs, const int64_t* ks,
                  const int64_t* vs, const int64_t* os, int dtype, float scale, void* ws,
                  int64_t ws_bytes, void* stream) {
    int rc = check_workspace(ws, ws_bytes);
    if (rc) return rc;
    AttnCall c;
    rc = prepare_attention(sparse, cfg, sched, q, k, v, o, lse, batch, heads, n_tot, head_dim, qs, ks, vs, os,
                           dtype, scale, ws != nullptr, c);
    if (rc || c.empty) return rc;
    if (ws && ws_bytes < c.p.ws_bytes)
        return fail(HILBERTA_ECAPACITY, "workspace of %lld bytes, %lld needed", (long long)ws_bytes,
                    (long long)c.p.ws_bytes);
    return launch_attention(c, dtype, head_dim, ws, static_cast<hipStream_t>(stream));
}

// ------------------------------------------------- allocation-free forward
// hilberta_attn_fwd_noalloc keeps the split key passes' partials in this
// library-owned device array instead of a caller workspace.  Each device the
// library runs on holds its own copy from module load to the end of the
// process.  Host code never passes `scratch` itself to a kernel (on the host
// it names a stand-in, not device memory): the device address of each
// device's copy is taken once, with that device current, and kept here.
// The partials are written in full before the merge reads them, so nothing
// in the array has to start at zero.  Calls that overlap on one device share
// the array and race.
constexpr int64_t kScratchBytes = 32ll << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The scratch array's address on the device of `stream`, which must be the
// current device.
int scratch_on(void* stream, void** out) {
    int cur = 0;
    if (int rc = hip_status(hipGetDevice(&cur), "hipGetDevice")) return rc;
    int dev = cur;
    if (stream) {
        hipDevice_t d = 0;
        if (int rc = hip_status(hipStreamGetDevice(static_cast<hipStream_t>(stream), &d), "hipStreamGetDevice"))
            return rc;
        dev = d;
    }
    if (dev != cur)
        return fail(HILBERTA_EINVAL, "the stream belongs to device %d but device %d is current", dev, cur);
    if (dev < 0 || dev >= kMaxDevices) return fail(HILBERTA_EUNSUPPORTED, "device %d >= %d", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (int rc = hip_status(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)"))
            return rc;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return HILBERTA_OK;
}

// Workspace of the backward: dO . O and the base-2 LSE per row, then the
// chunk partials of the split dense rows (two D-vectors per row and chunk,
// reused by the dQ and the dK/dV passes).
int64_t bwd_rows_bytes(int64_t bh, int64_t n_tot) { return round_up(bh * n_tot * 2, 4) * 4; }

int64_t bwd_ws_bytes(const Plan& p, int64_t bh, int64_t n_tot, int64_t head_dim) {
    const int64_t part = p.n_chunks > 1 ? bh * p.n_chunks * p.n_dense_rows * 2 * head_dim * 4 : 0;
    return bwd_rows_bytes(bh, n_tot) + part;
}

int run_attention_bwd(bool sparse, const hilberta_config* cfg, const int32_t* sched, const void* q,
                      const void* k, const void* v, const void* o, const void* dout, const float* lse,
                      void* dq, void* dk, void* dv, int64_t batch, int64_t heads, int64_t n_tot,
                      int64_t head_dim, const int64_t* qs, const int64_t* ks, const int64_t* vs,
                      const int64_t* os, int dtype, float scale, void* ws, int64_t ws_bytes, void* stream) {
    const Tensor4 t[8] = {{q, qs, "q"},       {k, ks, "k"},   {v, vs, "v"},   {o, os, "o"},
                          {dout, os, "dout"}, {dq, qs, "dq"}, {dk, ks, "dk"}, {dv, vs, "dv"}};
    int rc = check_workspace(ws, ws_bytes);
    if (rc) return rc;
    if (dtype != HILBERTA_BF16 && dtype != HILBERTA_F32) return fail(HILBERTA_EUNSUPPORTED, "dtype %d", dtype);
    Plan p{};
    hilberta::AttnArgs a{};
    bool empty = false;
    // the fp32 kernels take every dense row whole (no key chunks)
    rc = attn_setup(sparse, cfg, sched, t, 8, batch, heads, n_tot, head_dim, dtype, scale, dtype == HILBERTA_BF16,
                    p, a, empty);
    if (rc || empty) return rc;
    if (!lse) return fail(HILBERTA_EINVAL, "lse is NULL");
    const int64_t need = bwd_ws_bytes(p, batch * heads, n_tot, head_dim);
    if (!ws) return fail(HILBERTA_EINVAL, "the backward needs a workspace of %lld bytes", (long long)need);
    if (ws_bytes < need)
        return fail(HILBERTA_ECAPACITY, "workspace of %lld bytes, %lld needed", (long long)ws_bytes,
                    (long long)need);
    hilberta::BwdArgs g{};
    g.dout = dout;
    g.lse = lse;
    g.dq = dq;
    g.dk = dk;
    g.dv = dv;
    g.delta = static_cast<float*>(ws);
    g.lse2 = static_cast<float*>(ws) + batch * heads * n_tot;
    a.ws = static_cast<float*>(ws) + bwd_rows_bytes(batch * heads, n_tot) / 4;  // 16-byte aligned
    const hipStream_t st = static_cast<hipStream_t>(stream);
    return hip_status(dtype == HILBERTA_BF16 ? hilberta::launch_attn_bwd(a, g, (int)head_dim, st)
                                             : hilberta::launch_attn_bwd_f32(a, g, (int)head_dim, st),
                      "backward launch");
}

int bwd_ws_query(bool sparse, const hilberta_config* cfg, int64_t batch, int64_t heads, int64_t n_tot,
                 int64_t head_dim, int dtype, int64_t* bytes) {
    if (!bytes) return fail(HILBERTA_EINVAL, "bytes is NULL");
    if (batch < 0 || heads < 0 || n_tot < 0) return fail(HILBERTA_EINVAL, "negative size");
    if (head_dim != 64 && head_dim != 128)
        return fail(HILBERTA_EUNSUPPORTED, "head_dim %lld not in {64, 128}", (long long)head_dim);
    if (dtype != HILBERTA_BF16 && dtype != HILBERTA_F32) return fail(HILBERTA_EUNSUPPORTED, "dtype %d", dtype);
    const bool split = dtype == HILBERTA_BF16;
    Plan p{};
    if (sparse) {
        const Geom g = geom(cfg);
        p = make_plan(true, g.prefix, g.tiled, g.shared_in_span, cfg->tile, n_tot, batch * heads, head_dim, dtype,
                      split);
    } else {
        p = make_plan(false, 0, n_tot, 0, n_tot, n_tot, batch * heads, head_dim, dtype, split);
    }
    *bytes = bwd_ws_bytes(p, batch * heads, n_tot, head_dim);
    return HILBERTA_OK;
}

int run_permute(bool scatter, const void* x, void* y, const int32_t* perm, int64_t batch, int64_t n,
                int64_t channels, int64_t xbs, int64_t xrs, int64_t ybs, int64_t yrs, int dtype,
                void* stream) {
    if (!x || !y || !perm) return fail(HILBERTA_EINVAL, "NULL pointer");
    if (batch < 0 || n < 0 || channels < 0) return fail(HILBERTA_EINVAL, "negative size");
    if (n > 0x7fffffffLL) return fail(HILBERTA_EUNSUPPORTED, "more than 2^31 rows");
    if (dtype != HILBERTA_F32 && dtype != HILBERTA_BF16)
        return fail(HILBERTA_EUNSUPPORTED, "dtype %d", dtype);
    if (xrs < channels || yrs < channels || xbs < 0 || ybs < 0)
        return fail(HILBERTA_EINVAL, "row stride smaller than the row");
    const int64_t es = dtype == HILBERTA_F32 ? 4 : 2;
    hilberta::PermuteArgs a{};
    a.x = static_cast<const char*>(x);
    a.y = static_cast<char*>(y);
    a.perm = perm;
    a.batch = batch;
    a.n = n;
    a.row_bytes = channels * es;
    a.x_bs = xbs * es;
    a.x_rs = xrs * es;
    a.y_bs = ybs * es;
    a.y_rs = yrs * es;
    a.scatter = scatter ? 1 : 0;
    if (batch == 0 || n == 0 || channels == 0) return HILBERTA_OK;
    return hip_status(hilberta::launch_permute(a, static_cast<hipStream_t>(stream)), "permute launch");
}

}  // namespace

extern "C" {

int hilberta_version(void) { return 100; }

const char* hilberta_last_error(void) { return g_err.c_str(); }

int hilberta_build_perm(int32_t grid_h, int32_t grid_w, int32_t* perm, int32_t* inv_or_null,
                        void* stream) {
    if (!perm) return fail(HILBERTA_EINVAL, "perm is NULL");
    if (int rc = check_grid(grid_h, grid_w)) return rc;
    return hip_status(hilberta::launch_build_perm(enclosing_side(grid_h, grid_w), grid_h, grid_w, perm,
                                                  inv_or_null, static_cast<hipStream_t>(stream)),
                      "build_perm launch");
}

int hilberta_build_perm_layout(const hilberta_config* cfg, int32_t* perm, int32_t* inv_or_null,
                               void* stream) {
    int rc = check_config(cfg);
    if (rc) return rc;
    if (!perm) return fail(HILBERTA_EINVAL, "perm is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (cfg->layout == HILBERTA_LAYOUT_MOVED && cfg->shared_h * cfg->shared_w > 0)
        return hip_status(hilberta::launch_build_perm_moved(cfg->grid_w, cfg->shared_h, cfg->shared_w, perm,
                                                            inv_or_null, s),
                          "build_perm launch");
    return hip_status(hilberta::launch_build_perm(enclosing_side(cfg->grid_h, cfg->grid_w), cfg->grid_h,
                                                  cfg->grid_w, perm, inv_or_null, s),
                      "build_perm launch");
}

int hilberta_permute(const void* x, void* y, const int32_t* perm, int64_t batch, int64_t n,
                     int64_t channels, int64_t x_batch_stride, int64_t x_row_stride,
                     int64_t y_batch_stride, int64_t y_row_stride, int dtype, void* stream) {
    return run_permute(false, x, y, perm, batch, n, channels, x_batch_stride, x_row_stride,
                       y_batch_stride, y_row_stride, dtype, stream);
}

int hilberta_unpermute(const void* x, void* y, const int32_t* perm, int64_t batch, int64_t n,
                       int64_t channels, int64_t x_batch_stride, int64_t x_row_stride,
                       int64_t y_batch_stride, int64_t y_row_stride, int dtype, void* stream) {
    return run_permute(true, x, y, perm, batch, n, channels, x_batch_stride, x_row_stride,
                       y_batch_stride, y_row_stride, dtype, stream);
}

int hilberta_schedule_words(const hilberta_config* cfg, int64_t* words) {
    int rc = check_config(cfg);
    if (rc) return rc;
    if (!words) return fail(HILBERTA_EINVAL, "words is NULL");
    *words = schedule_words(cfg);
    return HILBERTA_OK;
}

int hilberta_schedule(const hilberta_config* cfg, int32_t layer, int32_t* sched, int64_t capacity,
                      int64_t* needed, void* stream) {
    int rc = check_config(cfg);
    if (rc) return rc;
    if (layer < 0) return fail(HILBERTA_EINVAL, "layer %d < 0", layer);
    const int64_t words = schedule_words(cfg);
    if (needed) *needed = words;
    if (!sched) return fail(HILBERTA_EINVAL, "sched is NULL");
    if (capacity < words)
        return fail(HILBERTA_ECAPACITY, "schedule needs %lld words, capacity %lld", (long long)words,
                    (long long)capacity);
    const Geom g = geom(cfg);
    hilberta::ScheduleArgs a{};
    a.out = sched;
    a.grid_h = cfg->grid_h;
    a.grid_w = cfg->grid_w;
    a.side = enclosing_side(cfg->grid_h, cfg->grid_w);
    a.n_txt = cfg->n_txt;
    a.tile = cfg->tile;
    a.n_tiles = (int32_t)(g.tiled / cfg->tile);
    a.shared_h = cfg->shared_h;
    a.shared_w = cfg->shared_w;
    a.prefix = (int32_t)g.prefix;
    a.tiled = (int32_t)g.tiled;
    a.moved = cfg->layout == HILBERTA_LAYOUT_MOVED;
    a.layer = layer;
    a.offset = (int32_t)(((int64_t)layer * cfg->delta) % g.tiled);
    a.span_cap = (int32_t)g.cap;
    a.words = (int32_t)words;
    return hip_status(hilberta::launch_schedule(a, static_cast<hipStream_t>(stream)), "schedule launch");
}

int hilberta_attn_workspace_bytes(const hilberta_config* cfg, int64_t batch, int64_t heads,
                                  int64_t head_dim, int dtype, int64_t* bytes) {
    int rc = check_config(cfg);
    if (rc) return rc;
    if (!bytes) return fail(HILBERTA_EINVAL, "bytes is NULL");
    if (batch < 0 || heads < 0) return fail(HILBERTA_EINVAL, "negative batch or heads");
    if (head_dim != 64 && head_dim != 128)
        return fail(HILBERTA_EUNSUPPORTED, "head_dim %lld not in {64, 128}", (long long)head_dim);
    if (dtype != HILBERTA_F32 && dtype != HILBERTA_BF16) return fail(HILBERTA_EUNSUPPORTED, "dtype %d", dtype);
    const Geom g = geom(cfg);
    const int64_t n_tot = cfg->n_txt + span_len(cfg);
    const Plan p = make_plan(true, g.prefix, g.tiled, g.shared_in_span, cfg->tile, n_tot, batch * heads,
                             head_dim, dtype, true);
    *bytes = p.ws_bytes;
    return HILBERTA_OK;
}

int hilberta_attn_fwd(const hilberta_config* cfg, const int32_t* sched, const void* q, const void* k,
                      const void* v, void* o, float* lse_or_null, int64_t batch, int64_t heads,
                      int64_t head_dim, const int64_t q_strides[4], const int64_t k_strides[4],
                      const int64_t v_strides[4], const int64_t o_strides[4], int dtype, float scale,
                      void* workspace, int64_t workspace_bytes, void* stream) {
    int rc = check_config(cfg);
    if (rc) return rc;
    if (!sched) return fail(HILBERTA_EINVAL, "sched is NULL");
    const int64_t n_tot = cfg->n_txt + span_len(cfg);
    return run_attention(true, cfg, sched, q, k, v, o, lse_or_null, batch, heads, n_tot, head_dim,
                         q_strides, k_strides, v_strides, o_strides, dtype, scale, workspace,
                         workspace_bytes, stream);
}

int hilberta_attn_fwd_noalloc(const hilberta_config* cfg, const int32_t* sched, const void* q, const void* k,
                              const void* v, void* o, float* lse_or_null, int64_t batch, int64_t heads,
                              int64_t head_dim, const int64_t q_strides[4], const int64_t k_strides[4],
                              const int64_t v_strides[4], const int64_t o_strides[4], int dtype, float scale,
                              void* stream) {
    int rc = check_config(cfg);
    if (rc) return rc;
    if (!sched) return fail(HILBERTA_EINVAL, "sched is NULL");
    const int64_t n_tot = cfg->n_txt + span_len(cfg);
    AttnCall c;
    rc = prepare_attention(true, cfg, sched, q, k, v, o, lse_or_null, batch, heads, n_tot, head_dim, q_strides,
                           k_strides, v_strides, o_strides, dtype, scale, true, c);
    if (rc || c.empty) return rc;
    if (c.p.ws_bytes > kScratchBytes)
        return fail(HILBERTA_ECAPACITY,
                    "the split key passes need %lld bytes, more than the %lld bytes of the library's scratch",
                    (long long)c.p.ws_bytes, (long long)kScratchBytes);
    void* ws = nullptr;
    if (c.p.ws_bytes > 0) {
        rc = scratch_on(stream, &ws);
        if (rc) return rc;
    }
    return launch_attention(c, dtype, head_dim, ws, static_cast<hipStream_t>(stream));
}

int hilberta_attn_bwd_workspace_bytes(const hilberta_config* cfg, int64_t batch, int64_t heads,
                                      int64_t head_dim, int dtype, int64_t* bytes) {
    int rc = check_config(cfg);
    if (rc) return rc;
    return bwd_ws_query(true, cfg, batch, heads, cfg->n_txt + span_len(cfg), head_dim, dtype, bytes);
}

int hilberta_attn_bwd(const hilberta_config* cfg, const int32_t* sched, const void* q, const void* k,
                      const void* v, const void* o, const void* dout, const float* lse, void* dq, void* dk,
                      void* dv, int64_t batch, int64_t heads, int64_t head_dim, const int64_t q_strides[4],
                      const int64_t k_strides[4], const int64_t v_strides[4], const int64_t o_strides[4],
                      int dtype, float scale, void* workspace, int64_t workspace_bytes, void* stream) {
    int rc = check_config(cfg);
    if (rc) return rc;
    if (!sched) return fail(HILBERTA_EINVAL, "sched is NULL");
    const int64_t n_tot = cfg->n_txt + span_len(cfg);
    return run_attention_bwd(true, cfg, sched, q, k, v, o, dout, lse, dq, dk, dv, batch, heads, n_tot, head_dim,
                             q_strides, k_strides, v_strides, o_strides, dtype, scale, workspace, workspace_bytes,
                             stream);
}

int dense_attn_bwd_workspace_bytes(int64_t batch, int64_t heads, int64_t n, int64_t head_dim, int dtype,
                                   int64_t* bytes) {
    return bwd_ws_query(false, nullptr, batch, heads, n, head_dim, dtype, bytes);
}

int dense_attn_bwd(const void* q, const void* k, const void* v, const void* o, const void* dout,
                   const float* lse, void* dq, void* dk, void* dv, int64_t batch, int64_t heads, int64_t n,
                   int64_t head_dim, const int64_t q_strides[4], const int64_t k_strides[4],
                   const int64_t v_strides[4], const int64_t o_strides[4], int dtype, float scale,
                   void* workspace, int64_t workspace_bytes, void* stream) {
    if (n < 0) return fail(HILBERTA_EINVAL, "n < 0");
    return run_attention_bwd(false, nullptr, nullptr, q, k, v, o, dout, lse, dq, dk, dv, batch, heads, n, head_dim,
                             q_strides, k_strides, v_strides, o_strides, dtype, scale, workspace, workspace_bytes,
                             stream);
}

int dense_attn_workspace_bytes(int64_t batch, int64_t heads, int64_t n, int64_t head_dim, int dtype,
                               int64_t* bytes) {
    if (!bytes) return fail(HILBERTA_EINVAL, "bytes is NULL");
    if (batch < 0 || heads < 0 || n < 0) return fail(HILBERTA_EINVAL, "negative size");
    if (head_dim != 64 && head_dim != 128)
        return fail(HILBERTA_EUNSUPPORTED, "head_dim %lld not in {64, 128}", (long long)head_dim);
    if (dtype != HILBERTA_F32 && dtype != HILBERTA_BF16) return fail(HILBERTA_EUNSUPPORTED, "dtype %d", dtype);
    const Plan p = make_plan(false, 0, n, 0, n, n, batch * heads, head_dim, dtype, true);
    *bytes = p.ws_bytes;
    return HILBERTA_OK;
}

int dense_attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse_or_null,
                   int64_t batch, int64_t heads, int64_t n, int64_t head_dim,
                   const int64_t q_strides[4], const int64_t k_strides[4],
                   const int64_t v_strides[4], const int64_t o_strides[4], int dtype, float scale,
                   void* workspace, int64_t workspace_bytes, void* stream) {
    if (n < 0) return fail(HILBERTA_EINVAL, "n < 0");
    return run_attention(false, nullptr, nullptr, q, k, v, o, lse_or_null, batch, heads, n, head_dim,
                         q_strides, k_strides, v_strides, o_strides, dtype, scale, workspace,
                         workspace_bytes, stream);
}

}  // extern "C"
