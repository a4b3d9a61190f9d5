/*
 * hilberta.h -- C ABI of libhilberta.so, the HilbertA hot path on AMD
 * Instinct MI355X (gfx950).
 *
 * HilbertA (arXiv 2509.26538) orders the image tokens of a diffusion
 * transformer along a Hilbert curve, attends densely inside contiguous tiles
 * of that sequence, slides the tile boundaries by a fixed offset per layer
 * without moving any data, and lets every token attend a small central
 * shared region and the text tokens.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Ownership  The caller allocates every buffer (device memory unless stated)
 *            and keeps ownership; the library keeps no pointer after a call
 *            returns and allocates no device memory in these entry points.
 * Streams    `stream` is a hipStream_t (NULL = the default stream).  Every
 *            device-side call is asynchronous on that stream.
 * Errors     Functions return HILBERTA_OK (0) or a negative code.  Every
 *            argument is validated on the host before anything is launched,
 *            so an error leaves all outputs untouched and launches nothing.
 *            hilberta_last_error() returns a message for the calling thread's
 *            last failing call.  No C++ exception crosses this interface.
 * Sequence   The attention sequence of one (batch, head) is N_tot = n_txt +
 *            N_img tokens: text tokens at [0, n_txt), then the image span in
 *            Hilbert order at [n_txt, N_tot) (Appendix A places the text as
 *            a global prefix).  Shared-region tokens keep their Hilbert
 *            slots inside the image span (or follow the text, see layout).
 * Shapes     A grid_h x grid_w grid that is not a square power of two takes
 *            the curve of its enclosing S x S square, S the smallest power
 *            of two >= max(grid_h, grid_w) and >= 2 (Appendix D).  The image
 *            span then holds all N_img = S*S curve positions; the positions
 *            whose cell lies outside the grid are padding slots, masked out
 *            as keys and as queries.  For a square power-of-two grid,
 *            S = grid_w and N_img = grid_h*grid_w.
 * Tensors    Q, K, V, O are [B, H, N_tot, D] with element strides given as
 *            {batch, head, row, dim}; the dim stride must be 1 and the other
 *            strides multiples of 8 elements (16-byte rows for bf16).
 */
#ifndef HILBERTA_H
#define HILBERTA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HILBERTA_OK 0
#define HILBERTA_EINVAL (-1)       /* null pointer, size or stride out of range */
#define HILBERTA_EUNSUPPORTED (-2) /* valid but not supported: grid shape, D, dtype, alignment */
#define HILBERTA_ECAPACITY (-3)    /* output or workspace too small; *needed is set */
#define HILBERTA_EHIP (-4)         /* a HIP runtime call failed */

/* element types */
#define HILBERTA_F32 0
#define HILBERTA_BF16 1

/* first word of every schedule table */
#define HILBERTA_SCHEDULE_MAGIC 0x48424131

/* Sequence layouts (hilberta_config.layout). */
#define HILBERTA_LAYOUT_IN_PLACE 0 /* shared tokens keep their Hilbert slots */
#define HILBERTA_LAYOUT_MOVED 1    /* shared tokens gathered next to the text */

/*
 * Geometry of one HilbertA attention layer stack.
 *   grid_h, grid_w   latent grid, each side in [1, 32768]; N_img = S*S
 *                    image-span positions (see Shapes above)
 *   n_txt            text tokens placed before the image tokens (>= 0)
 *   tile             N_T, tokens per tile; divides N_img (§3.2)
 *   delta            per-layer advance Delta of the tile boundaries (>= 0);
 *                    the paper sets Delta = N_T / L for a slide cycle L (§3.2)
 *   shared_h/_w      central shared region (§3.3): grid rows in
 *                    [(grid_h - shared_h)/2, + shared_h) and columns in
 *                    [(grid_w - shared_w)/2, + shared_w), integer halving;
 *                    0 x 0 disables it.  At most 1024 shared tokens (32 x 32,
 *                    the largest region the paper uses) and
 *                    shared_h + shared_w <= 255.
 *   layout           HILBERTA_LAYOUT_IN_PLACE: the image span keeps all N_img
 *                    tokens in Hilbert order, the shared ones in their slots
 *                    (also global keys and dense rows), and is tiled whole.
 *                    HILBERTA_LAYOUT_MOVED (Appendix A taken literally): the
 *                    image span holds the N_sh shared tokens first, then the
 *                    others, each part in Hilbert order (see
 *                    hilberta_build_perm_layout); the global prefix is the
 *                    text and the shared tokens, and only the N_img - N_sh
 *                    others are tiled, so `tile` must divide N_img - N_sh.
 *                    Needs a square power-of-two grid (no padding).
 * The sequence must satisfy n_txt + N_img < 2^31.
 */
typedef struct hilberta_config {
    int32_t grid_h;
    int32_t grid_w;
    int32_t n_txt;
    int32_t tile;
    int32_t delta;
    int32_t shared_h;
    int32_t shared_w;
    int32_t layout;
} hilberta_config;

/* Library version (major*10000 + minor*100 + patch). Host only. */
int hilberta_version(void);

/* Message for the calling thread's last failing call ("" if none). Host only. */
const char* hilberta_last_error(void);

/*
 * hilberta_build_perm -- the Hilbert linearisation pi of §3.1.
 *   For each position d in [0, S*S) of the curve over the S x S square (S
 *   as under Shapes; the curve starts at (0, 0) and ends at (S-1, 0)),
 *   perm[d] = y*grid_w + x, where (x = column, y = row) is the cell at d,
 *   or -1 when that cell lies outside the grid (a padding slot).  If
 *   inv_or_null is not NULL, inv[y*grid_w + x] = d for every grid cell.
 *   perm: device int32[S*S]; inv: device int32[grid_h*grid_w].
 * Errors: EINVAL (perm NULL), EUNSUPPORTED (a side outside [1, 32768]).
 */
int hilberta_build_perm(int32_t grid_h, int32_t grid_w, int32_t* perm,
                        int32_t* inv_or_null, void* stream);

/*
 * hilberta_build_perm_layout -- the image-span order of cfg's layout: the
 *   Hilbert linearisation (as hilberta_build_perm) in place; moved, the
 *   shared tokens first and then the others, each part in Hilbert order
 *   (Appendix A gathers the shared tokens next to the text).  perm[d] is the
 *   raster index of the token at image-span position d (-1 at padding
 *   slots); if inv_or_null is not NULL, inv[perm[d]] = d for every grid
 *   cell.  perm: device int32[N_img]; inv: device int32[grid_h*grid_w].
 * Errors: as hilberta_schedule_words for cfg; EINVAL (perm NULL).
 */
int hilberta_build_perm_layout(const hilberta_config* cfg, int32_t* perm,
                               int32_t* inv_or_null, void* stream);

/*
 * hilberta_permute -- the token gather of §3.4, applied once at the input:
 *   y[b, d, :] = x[b, perm[d], :]   for b < batch, d < n, all `channels`.
 * hilberta_unpermute -- its inverse, applied once at the output:
 *   y[b, perm[d], :] = x[b, d, :].
 *   x, y      device tensors of `dtype`; rows of `channels` contiguous
 *             elements; strides in elements.  To leave text rows alone, pass
 *             pointers offset to the first image row.  x and y must not
 *             overlap.
 *   perm      device int32[n] (e.g. from hilberta_build_perm): a
 *             permutation of [0, n), or for a general shape an injection
 *             into the grid's raster rows with -1 at padding slots.  A
 *             negative entry makes the gather write a zero row y[b, d, :]
 *             and the scatter skip x[b, d, :]; entries >= n are skipped by
 *             both.  For a general shape, n = N_img rows of the sequence
 *             side and the raster side has grid_h*grid_w rows.
 * Errors: EINVAL (NULL pointer, negative size, row stride < channels),
 * EUNSUPPORTED (dtype).
 */
int hilberta_permute(const void* x, void* y, const int32_t* perm, int64_t batch,
                     int64_t n, int64_t channels, int64_t x_batch_stride,
                     int64_t x_row_stride, int64_t y_batch_stride,
                     int64_t y_row_stride, int dtype, void* stream);
int hilberta_unpermute(const void* x, void* y, const int32_t* perm, int64_t batch,
                       int64_t n, int64_t channels, int64_t x_batch_stride,
                       int64_t x_row_stride, int64_t y_batch_stride,
                       int64_t y_row_stride, int dtype, void* stream);

/*
 * hilberta_schedule_words -- int32 words of the schedule table for cfg.
 * Host only; validates cfg like hilberta_schedule.
 */
int hilberta_schedule_words(const hilberta_config* cfg, int64_t* words);

/*
 * hilberta_schedule -- the per-layer tile schedule of §3.2 and the shared
 * runs of §3.3, written to device memory `sched` (int32[capacity]).
 *   Layer l slides the boundaries by o = (l*delta) mod N: position p of the
 *   tiled span has tile label floor((p + l*delta)/N_T) mod T, queries and
 *   keys of equal label attend each other, and the wrap-around tile is read
 *   with modular indexing (§3.2), never copied.  In place the global prefix
 *   P is the text and the tiled span is the whole image (N = N_img); moved,
 *   P = n_txt + N_sh and N = N_img - N_sh, and there are no shared runs.
 *   Table layout (int32 words):
 *     [0] HILBERTA_SCHEDULE_MAGIC  [1] P  [2] N  [3] N_T  [4] T
 *     [5] o  [6] n_spans  [7] n_shared  [8] layer  [9] grid_h  [10] grid_w
 *     [11] span capacity C = shared_h + shared_w + 1 (0 without a region
 *          or when moved)
 *     [12 + 4q .. 12 + 4q + 3], q < T: tile q as (start, len1, len2, ns):
 *         its tokens are [start, start + len1) and, when it wraps past the
 *         end of the sequence, [P, P + len2); start is a sequence position;
 *         ns = shared tokens inside the tile (0 when moved).
 *     [12 + 4T + 2s, +1], s < C: shared run s as (start, len), sequence
 *         positions, ascending, maximal; zero past n_spans.
 *   The table has exactly hilberta_schedule_words(cfg) words.
 * Errors: EINVAL (NULL, layer < 0), EUNSUPPORTED (cfg out of range),
 * ECAPACITY (capacity too small; *needed set if needed is not NULL).
 */
int hilberta_schedule(const hilberta_config* cfg, int32_t layer, int32_t* sched,
                      int64_t capacity, int64_t* needed, void* stream);

/*
 * hilberta_attn_workspace_bytes -- device workspace hilberta_attn_fwd needs
 * for its split key passes over dense rows.  Host only.
 */
int hilberta_attn_workspace_bytes(const hilberta_config* cfg, int64_t batch,
                                  int64_t heads, int64_t head_dim, int dtype,
                                  int64_t* bytes);

/*
 * hilberta_attn_fwd -- HilbertA sparse attention forward (§3.2-§3.4,
 * Appendix A, Algorithm 1), one launch over all rows:
 *   rows of text and shared tokens attend all N_tot keys;
 *   every other image row attends the text keys, the shared keys and the
 *   keys of its own slid tile, each key once;
 *   padding slots of a general shape are no key of any row, and their own
 *   rows are written as O = 0 and lse = -inf.  Padding rows of K and V must
 *   hold finite values (hilberta_permute writes zeros there);
 *   O = softmax(scale * Q K^T restricted to those keys) V, and optionally
 *   lse = ln sum exp(scale * q.k) over the same keys (natural log).
 *   sched      device table from hilberta_schedule(cfg, layer, ...); it
 *              selects the layer.  A table for another cfg gives wrong
 *              results but no out-of-bounds access.
 *   q,k,v,o    device [batch, heads, N_tot, head_dim] with strides
 *              {batch, head, row, dim} in elements, dim stride 1; o may not
 *              overlap q, k or v.
 *   lse_or_null device float[batch*heads*N_tot] (row-major b, h, n) or NULL.
 *   head_dim   64 or 128.  dtype HILBERTA_BF16 (fp32 accumulation, P rounded
 *              to bf16 for PV, bf16 output) or HILBERTA_F32 (fp32 throughout).
 *   scale      softmax scale, usually 1/sqrt(head_dim).
 *   workspace  device scratch of at least hilberta_attn_workspace_bytes, or
 *              NULL with workspace_bytes 0 to run without split key passes.
 * With batch*heads == 0 nothing is read or written and the tensor pointers
 * may be NULL.
 * Errors: EINVAL, EUNSUPPORTED (head_dim, dtype, stride alignment),
 * ECAPACITY (workspace given but too small), EHIP.
 */
int hilberta_attn_fwd(const hilberta_config* cfg, const int32_t* sched,
                      const void* q, const void* k, const void* v, void* o,
                      float* lse_or_null, int64_t batch, int64_t heads,
                      int64_t head_dim, const int64_t q_strides[4],
                      const int64_t k_strides[4], const int64_t v_strides[4],
                      const int64_t o_strides[4], int dtype, float scale,
                      void* workspace, int64_t workspace_bytes, void* stream);

/*
 * hilberta_attn_bwd_workspace_bytes -- device workspace hilberta_attn_bwd
 * needs: 8 bytes per row of every (batch, head), for dO . O and the LSE in
 * log2 units, plus, when the rows that attend every key are split into key
 * chunks, 8 D bytes per such row, chunk and (batch, head) for the fp32
 * partial sums (of dQ in the first pass, of dK and dV in the second).
 * Host only.  Errors: as hilberta_schedule_words for cfg;
 * EUNSUPPORTED (head_dim, dtype other than bf16).
 */
int hilberta_attn_bwd_workspace_bytes(const hilberta_config* cfg, int64_t batch,
                                      int64_t heads, int64_t head_dim, int dtype,
                                      int64_t* bytes);

/*
 * hilberta_attn_fwd_noalloc -- hilberta_attn_fwd for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same kernels, results bit for bit
 * those of hilberta_attn_fwd with a workspace, but the split key passes keep
 * their partials in a device array the library owns (32 MiB per device,
 * held from the library's load to the end of the process) instead of a
 * caller workspace.  It calls no hipMalloc, hipFree or allocating library
 * routine.  Arguments as for hilberta_attn_fwd, without the workspace; the
 * stream must belong to the current device.
 * Every call on one device shares that device's array: calls that overlap
 * on one device (on different streams, or from different threads) race and
 * give undefined results.
 * Errors: as hilberta_attn_fwd; ECAPACITY when the split key passes would
 * need more than the array holds (hilberta_attn_workspace_bytes > 32 MiB;
 * the Flux.1-dev shapes need at most 19 MB, a 64 x 64 grid with 2048 text
 * tokens and 16 heads of D = 128 needs 36.6 MiB); EINVAL when the stream
 * belongs to another device than the current one.
 */
int hilberta_attn_fwd_noalloc(const hilberta_config* cfg, const int32_t* sched,
                              const void* q, const void* k, const void* v,
                              void* o, float* lse_or_null, int64_t batch,
                              int64_t heads, int64_t head_dim,
                              const int64_t q_strides[4],
                              const int64_t k_strides[4],
                              const int64_t v_strides[4],
                              const int64_t o_strides[4], int dtype,
                              float scale, void* stream);

/*
 * hilberta_attn_bwd -- gradients of hilberta_attn_fwd's output with respect
 * to Q, K and V (the backward pass that training through the sparse
 * attention needs: §4.1 fine-tunes with LoRA, the appendix on training
 * from scratch trains a DiT).  For every (batch, head), with P the forward's
 * probabilities (masked entries 0) and dO the gradient of O:
 *   dV = P^T dO,  dP = dO V^T,  dS = P (dP - rowsum(dO * O)),
 *   dQ = scale dS K,  dK = scale dS^T Q.
 * Padding slots of a general shape get zero gradients.
 *   sched      the table the forward used (same cfg and layer).
 *   q,k,v,o    the forward's inputs and output; dout shares o's strides,
 *              dq q's, dk k's and dv v's; all [batch, heads, N_tot, head_dim]
 *              device tensors as for hilberta_attn_fwd; dq, dk, dv are
 *              written completely and may not overlap the inputs.
 *   lse        the forward's natural-log LSE, device float[batch*heads*N_tot].
 *   dtype      HILBERTA_BF16: bf16 tensors, fp32 accumulation, P and dS
 *              rounded to bf16 as matrix operands.  HILBERTA_F32: fp32
 *              tensors and fp32 arithmetic throughout (for exactness at
 *              small sizes, not speed).
 *   scale      the forward's softmax scale.
 *   workspace  device scratch of at least hilberta_attn_bwd_workspace_bytes
 *              (required), 16-byte aligned.
 * Deterministic: every gradient row is written once, without atomics.
 * Errors: EINVAL (NULL pointers, no workspace), EUNSUPPORTED (head_dim,
 * dtype, stride alignment), ECAPACITY (workspace too small), EHIP.
 */
int hilberta_attn_bwd(const hilberta_config* cfg, const int32_t* sched,
                      const void* q, const void* k, const void* v, const void* o,
                      const void* dout, const float* lse, void* dq, void* dk, void* dv,
                      int64_t batch, int64_t heads, int64_t head_dim,
                      const int64_t q_strides[4], const int64_t k_strides[4],
                      const int64_t v_strides[4], const int64_t o_strides[4], int dtype,
                      float scale, void* workspace, int64_t workspace_bytes, void* stream);

/* dense_attn_bwd_workspace_bytes -- workspace for dense_attn_bwd. Host only. */
int dense_attn_bwd_workspace_bytes(int64_t batch, int64_t heads, int64_t n,
                                   int64_t head_dim, int dtype, int64_t* bytes);

/*
 * dense_attn_bwd -- gradients of dense_attn_fwd (the baseline the sparse
 * backward is measured against).  Arguments as for hilberta_attn_bwd with
 * N_tot = n and no schedule.
 */
int dense_attn_bwd(const void* q, const void* k, const void* v, const void* o,
                   const void* dout, const float* lse, void* dq, void* dk, void* dv,
                   int64_t batch, int64_t heads, int64_t n, int64_t head_dim,
                   const int64_t q_strides[4], const int64_t k_strides[4],
                   const int64_t v_strides[4], const int64_t o_strides[4], int dtype,
                   float scale, void* workspace, int64_t workspace_bytes, void* stream);

/* dense_attn_workspace_bytes -- workspace for dense_attn_fwd. Host only. */
int dense_attn_workspace_bytes(int64_t batch, int64_t heads, int64_t n,
                               int64_t head_dim, int dtype, int64_t* bytes);

/*
 * dense_attn_fwd -- full softmax attention over all n keys for every row:
 * the baseline HilbertA is measured against (Table 1's dense rows), built
 * from the same kernels and layout as hilberta_attn_fwd.  Arguments as for
 * hilberta_attn_fwd with N_tot = n and no schedule.
 */
int dense_attn_fwd(const void* q, const void* k, const void* v, void* o,
                   float* lse_or_null, int64_t batch, int64_t heads, int64_t n,
                   int64_t head_dim, const int64_t q_strides[4],
                   const int64_t k_strides[4], const int64_t v_strides[4],
                   const int64_t o_strides[4], int dtype, float scale,
                   void* workspace, int64_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* HILBERTA_H */
