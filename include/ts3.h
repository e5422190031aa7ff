/*
 * ts3.h -- C ABI of the Transolver-3 Physics-Attention layer on MI355X (gfx950).
 *
 * One layer maps point features x [N, C] to x_out [N, C] (paper section 3):
 *   w     = Softmax_per_head(Linear2(x) / tau)          slice weights, Eq. (1)
 *   s_raw = w^T x,  d = sum_i w_i                        accumulated over tiles, Eq. (4)
 *   s     = Linear1(d^-1 s_raw)                          physical states, Eq. (3) / Algorithm 1
 *   s'    = Attention(s)                                 per head, among its M tokens
 *   Z     = Linear3(s')  (no bias)                       cached state s'_out, section 3.3
 *   x_out = w Z + b3                                     full-mesh decoding, Eq. (5)
 * H heads each own M slices (H*M slice tokens) and a dh = C/H wide block of
 * Linear1's outputs / Linear3's inputs; attention runs per head with scale
 * 1/sqrt(dh).  Pass 1 (accumulate) streams tiles of x into an opaque state;
 * finalize + attention build the cached state Z; pass 2 (deslice) decodes any
 * chunk of points against it.  The slice weights w are recomputed in pass 2
 * (Eq. (5)) and never stored.
 *
 * Conventions shared by every entry point:
 *  - Pointers named x, out and every ts3_weights member are DEVICE pointers;
 *    host_dst / host_src are HOST pointers.  The caller owns all of them; they
 *    must stay valid until the work enqueued on `stream` has finished.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Every
 *    call only enqueues work and returns; ts3_state_create, ts3_state_free,
 *    ts3_state_get and ts3_state_set synchronise.
 *  - Layouts are row-major.  x and out are [n, C] of the state's io dtype
 *    (float32 or bfloat16, 16-byte aligned); weights are float32.
 *  - Every call returns a ts3_status; nothing throws or aborts.  On failure the
 *    state is unchanged unless stated, and ts3_last_error() (per thread)
 *    describes the cause.  A fault inside an enqueued kernel surfaces as
 *    TS3_ERR_HIP from a later synchronising call.
 */
#ifndef TS3_H
#define TS3_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    TS3_OK = 0,
    TS3_ERR_INVALID_ARG = 1,   /* null pointer, bad size, overlapping or misaligned tile */
    TS3_ERR_BAD_STATE = 2,     /* call out of order (see the state machine below) */
    TS3_ERR_OUT_OF_MEMORY = 3, /* device allocation failed */
    TS3_ERR_HIP = 4,           /* a HIP runtime call failed */
    TS3_ERR_UNSUPPORTED = 5    /* shape this build has no kernel for */
} ts3_status;

typedef enum { TS3_FP32 = 0, TS3_BF16 = 1 } ts3_dtype;

/* Precision of the fold of span partials (ts3_desc.accum). */
typedef enum { TS3_ACCUM_FP32 = 0, TS3_ACCUM_FP64 = 1 } ts3_accum;

/* Layer shape and numerics.
 *  C, H, M, dh : channels, heads, slices per head, head width; H*dh == C.
 *                Tuned matrix-core kernels serve (C, M) in {(64,16), (64,32),
 *                (128,16), (128,32), (128,64)}, and (256,64) with bf16
 *                storage and even H.  Any other C and M that are multiples
 *                of 16 with C <= 512 and M <= 256 run on runtime-shape
 *                vector kernels (same results up to float32 rounding order,
 *                same tiling independence, far slower; no backward).  In
 *                every case (5*M*dh + M*M) * 4 bytes <= 160 KiB (the
 *                token-attention working set); otherwise TS3_ERR_UNSUPPORTED.
 *  temperature : tau > 0 of the slice softmax; +inf gives uniform weights.
 *  eps         : added to d before the division in finalize (the paper uses 0).
 *                A slice with d + eps <= 0 has a zero mean state.
 *  io_dtype    : ts3_dtype of x and out.  TS3_BF16 stores bf16 and computes
 *                the slice-weight and contraction products on bf16 matrix
 *                cores with float32 accumulation; TS3_FP32 uses float32
 *                matrix cores throughout.  The runtime-shape kernels read
 *                either storage type and compute in float32 on vector units.
 *  group_span  : Q, points per accumulation span (1 <= Q <= 2^30).  Pass 1
 *                reduces each span to one partial and sums spans in index
 *                order, so results do not depend on how the mesh is tiled.
 *  accum       : ts3_accum, the precision of the fold of span partials (the
 *                sum over tiles of Eq. (4); Appendix A.4 on accumulating over
 *                very large meshes).  TS3_ACCUM_FP32 adds the float32 span
 *                partials in float32; TS3_ACCUM_FP64 adds them in float64 and
 *                rounds once to float32.  Each span's own partial is float32
 *                either way.  Any other value is TS3_ERR_INVALID_ARG.
 *  max_points  : largest point index + 1 the state will accumulate; sizes the
 *                span partials (ceil(max_points / Q) * H * M * (C+1) floats). */
typedef struct {
    int32_t C, H, M, dh;
    float temperature;
    float eps;
    int32_t io_dtype;
    int32_t accum;
    int64_t group_span;
    int64_t max_points;
} ts3_desc;

/* Layer weights: device pointers to row-major float32.
 *  W2 [C, H*M], b2 [H*M]   Linear2 -> slice logits; columns h*M..h*M+M-1 are head h
 *  W1 [C, H*dh], b1 [H*dh] Linear1, applied to the slice tokens
 *  Wq, Wk, Wv [H, dh, dh]  per-head token-attention projections (no bias)
 *  W3 [H*dh, C], b3 [C]    Linear3, applied to the slice tokens; b3 added per point
 * Biases may be NULL (zero). */
typedef struct {
    const float *W2, *b2;
    const float *W1, *b1;
    const float *Wq, *Wk, *Wv;
    const float *W3, *b3;
} ts3_weights;

typedef struct ts3_state ts3_state; /* opaque */

/* Gradients written by ts3_layer_backward: DEVICE pointers, float32, the
 * layouts of the matching ts3_weights members; all nine must be non-NULL.
 * They are overwritten, not accumulated into. */
typedef struct {
    float *dW2, *db2;
    float *dW1, *db1;
    float *dWq, *dWk, *dWv;
    float *dW3, *db3;
} ts3_grads;

/* Which buffer ts3_state_get / ts3_state_set address (float32, row-major). */
typedef enum {
    TS3_S_RAW = 0, /* [H, M, C]  sum_i w_i x_i            (valid after finalize; unprojected states) */
    TS3_D = 1,     /* [H, M]     sum_i w_i                (valid after finalize) */
    TS3_S = 2,     /* [H, M, dh] Linear1(d^-1 s_raw)      (valid after finalize) */
    TS3_S1 = 3,    /* [H, M, dh] Attention(s)             (valid after attention) */
    TS3_ZP = 4,    /* [H, M, C]  Linear3(s'), the cache   (valid after attention) */
    TS3_T_RAW = 5  /* [H, M, dh] sum_i w_i (x_i W1_h)     (valid after finalize; projected states) */
} ts3_buffer;

/* Allocate a state for one layer (device memory on the current HIP device) and
 * leave it reset.  *out receives the handle; it is NULL on failure. */
ts3_status ts3_state_create(const ts3_desc *desc, ts3_state **out);

/* Synchronise the device and release the state.  NULL is a no-op. */
ts3_status ts3_state_free(ts3_state *st);

/* Device bytes the state holds (for peak-memory reports). */
ts3_status ts3_state_bytes(const ts3_state *st, int64_t *bytes);

/* Whether the state accumulates projected sums (*projected = 1) or raw ones (0).
 * Eq. (2) applies Linear1 to each point before the slice sum and the form of
 * Eq. (4) after it; by linearity, sum_i w_i (x_i W1_h) = (sum_i w_i x_i) W1_h,
 * so both give the same s.  Where it needs fewer products per point (bfloat16
 * storage, C = 128, head width 16, M a multiple of 32) pass 1 sums the
 * projected rows: each span partial row is then [dh + 1] floats (t, then the
 * weight sum) instead of [C + 1], s_raw is not formed (TS3_S_RAW is
 * UNSUPPORTED; TS3_T_RAW holds the projected sums), and accumulate also needs
 * W1 (recorded at the first accumulate after reset, like W2/b2). */
ts3_status ts3_state_projected(const ts3_state *st, int32_t *projected);

/* Begin a new mesh: forget every accumulated tile.  Enqueues nothing. */
ts3_status ts3_state_reset(ts3_state *st, void *stream);

/* Pass 1 on one geometry tile (Eq. (4), Algorithm 1 tile loop): points
 * [point_offset, point_offset + n_tile) of the mesh, x_tile -> [n_tile, C].
 * point_offset must be a multiple of group_span; a tile whose end is not a
 * multiple of group_span must be the one holding the mesh's last point (no
 * later tile may start inside its last span); tiles must not overlap; the end
 * must not pass max_points.  Tiles may arrive in any order.  n_tile == 0 is a
 * no-op.  The first accumulate after reset records W2/b2 (converted once to
 * the kernel's operand format); later accumulate and deslice calls must pass
 * the same W2 and b2 pointers.  State: RESET/ACCUMULATING -> ACCUMULATING. */
ts3_status ts3_slice_accumulate(ts3_state *st, const ts3_weights *w, const void *x_tile,
                                int64_t n_tile, int64_t point_offset, void *stream);

/* Sum the span partials in index order into s_raw and d (Eq. (4)) and form
 * s = Linear1(d^-1 s_raw) per head (Algorithm 1 after the tile loop).
 * Needs W1 (b1 optional).  State: ACCUMULATING -> FINALIZED. */
ts3_status ts3_slice_finalize(ts3_state *st, const ts3_weights *w, void *stream);

/* s' = Attention(s) per head, then Z = Linear3(s') (the cached physical state
 * s'_out of section 3.3), stored with b3 for decoding.  Needs Wq, Wk, Wv, W3
 * (b3 optional).  State: FINALIZED -> ATTENDED. */
ts3_status ts3_token_attention(ts3_state *st, const ts3_weights *w, void *stream);

/* Pass 2 on one chunk (Eq. (5), Algorithm 1 deslice loop):
 * out_chunk[i] = Softmax_per_head(Linear2(x_chunk[i]) / tau) . Z + b3 for
 * i < n_chunk.  Any chunk, any number of times, any points (not only those
 * accumulated).  W2/b2 must be the pointers recorded by accumulate.
 * n_chunk == 0 is a no-op.  State: ATTENDED. */
ts3_status ts3_deslice(const ts3_state *st, const ts3_weights *w, const void *x_chunk,
                       int64_t n_chunk, void *out_chunk, void *stream);

/* Whole layer on a resident mesh (Algorithm 1): reset, accumulate tiles of
 * `tile` points, finalize, attention, deslice chunks of `chunk` points.
 * tile must be a multiple of group_span; N <= max_points.  Allocates nothing.
 * Consecutive tiles (and chunks) are enqueued alternately on `stream` and on
 * a second stream that the state owns, forked from `stream` by an event and
 * joined back into it before the call returns: work enqueued on `stream`
 * afterwards sees the whole layer.  Leaves the state ATTENDED. */
ts3_status ts3_layer_forward(ts3_state *st, const ts3_weights *w, const void *x, int64_t N,
                             int64_t tile, int64_t chunk, void *out, void *stream);

/* ts3_layer_forward for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, and hosts that forbid
 * allocation.  Same arguments and results as ts3_layer_forward (bitwise equal
 * outputs for the same desc, weights, x, N and tile), but there is no state
 * object: every buffer beyond x, out and the weights lives in one fixed
 * 64 MiB device array inside the library.  Each GPU the library runs on holds
 * its own copy of that array from the first call on that device until the
 * process ends.  The call allocates and frees nothing (no hipMalloc, no
 * stream or event creation).  All its work runs on `stream`; tiles run one
 * after another (no second stream).
 *  - Scratch needed: the span partials of one tile, ceil(tile / group_span) *
 *    H*M*(C+1) floats, plus the run sums of the mesh, ceil(ceil(N /
 *    group_span) / 64) * H*M*(C+1) floats (doubles with TS3_ACCUM_FP64), plus
 *    under 1 MiB of token-side buffers.  At C=128, H*M=512, group_span 15,625
 *    and 1M-point tiles that is about 44 MB for 100M points.  A call that needs
 *    more than 64 MiB returns TS3_ERR_INVALID_ARG before enqueuing anything.
 *  - Calls that overlap on one GPU (from several threads or streams) share the
 *    array and race: serialise them.  The array keeps the last call's
 *    contents; every region a call reads is written by that call first.
 *  - desc is validated as for ts3_state_create (max_points is not used).
 *  - N = 0 is valid: only the token-side work of an empty mesh runs and out
 *    is not touched.
 * The cached state is not retained after the call returns. */
ts3_status ts3_layer_forward_noalloc(const ts3_desc *desc, const ts3_weights *w, const void *x, int64_t N,
                                     int64_t tile, int64_t chunk, void *out, void *stream);

/* Backward of the layer (section 3.2: the training loop checkpoints every
 * tile, so the slice weights are recomputed tile by tile, never stored).
 * Given the output gradient g = dL/dx_out [N, C], writes dx = dL/dx [N, C]
 * and the weight gradients.  The state must hold the forward of the same x
 * and weights (ts3_layer_forward, or accumulate/finalize/attention over all N
 * points): it supplies s_raw, d, s, s' and Z.  Passes over the points, in
 * tiles of `tile` points (a multiple of group_span): dZ = sum_i w_i^T g_i;
 * then, after the token-side backward (Linear3, attention, Linear1, d^-1),
 * per tile dx, which also stores the softmax gradient dz of the tile's
 * points, and from the stored dz the tile's share of dW2 and db2.  Sums over
 * points are folded in index order, so the result does not depend on `tile`.
 * Float32 storage and the tuned shapes with C <= 128 only
 * (TS3_ERR_UNSUPPORTED for bfloat16 or a runtime-shape layer).  x, g, dx are
 * 16-byte aligned device pointers of N*C floats.  The dz store holds
 * min(tile, N)*H*M floats (2 GB for 1M-point tiles at H*M = 512); the first
 * call, or a later one with a larger tile, allocates it and the state keeps
 * it (ts3_state_bytes counts it; TS3_ERR_OUT_OF_MEMORY if it does not fit).
 * Leaves the state ATTENDED. */
ts3_status ts3_layer_backward(ts3_state *st, const ts3_weights *w, const void *x, const void *g, int64_t N,
                              int64_t tile, void *dx, const ts3_grads *grads, void *stream);

/* Copy a state buffer to host memory (n floats, must equal its size) after
 * synchronising `stream`.  For tests and inspection. */
ts3_status ts3_state_get(const ts3_state *st, int32_t which, float *host_dst, int64_t n,
                         void *stream);

/* Copy the span partials of spans [span0, span0 + nspan) to host memory, after
 * synchronising `stream`: [nspan][H][M][C+1] floats, where columns 0..C-1 hold
 * the sum over the span's points of w_i x_i and column C the sum of w_i.  These
 * are the per-span terms of Eq. (4) before the ordered fold (finalize sums them
 * in span order).  Every requested span must have been accumulated since the
 * last reset, and no backward may have run since (it reuses the buffer):
 * otherwise TS3_ERR_BAD_STATE.  n must equal nspan*H*M*(C+1).  A projected
 * state (ts3_state_projected) holds [nspan][H][M][dh+1] instead: columns
 * 0..dh-1 the span's sum of w_i (x_i W1_h), column dh the sum of w_i.  For
 * tests and inspection. */
ts3_status ts3_state_get_spans(const ts3_state *st, int64_t span0, int64_t nspan, float *host_dst, int64_t n,
                               void *stream);

/* Test hook: overwrite the cached state Z (which == TS3_ZP) and b3 from host
 * memory (b3 may be NULL = zero), convert it to the decoding operand format,
 * and mark the state ATTENDED, so pass 2 can be checked on its own.  The W2/b2
 * pointers used by deslice are taken from `w`.  Synchronises `stream`. */
ts3_status ts3_state_set(ts3_state *st, const ts3_weights *w, int32_t which,
                         const float *host_src, int64_t n, const float *host_b3, void *stream);

/* ------------------------------------------------------------------------
 * Transolver block stack (the model around the layer: section 3 and the
 * 8-layer configuration of Table 7).  Each block is pre-norm with residuals,
 * a form the paper does not spell out and that is taken from the Transolver
 * family:
 *     y   = x + PA(LN1(x))
 *     out = y + W_b^T GELU(W_a^T LN2(y) + b_a) + b_b
 * LayerNorm over the C channels with affine gamma/beta and eps 1e-5 (biased
 * variance); GELU in its exact form x * Phi(x) (erf evaluated to 1.5e-7).
 * Activations are bf16 [N][C]; the feed-forward products run on bf16 matrix
 * cores with float32 accumulation; each block keeps its own layer state, so
 * every block's physical state Z stays cached (section 3.3). */
typedef struct {
    ts3_weights pa;               /* Physics-Attention weights (as above) */
    const float *ln1_g, *ln1_b;   /* [C] LayerNorm before the attention */
    const float *ln2_g, *ln2_b;   /* [C] LayerNorm before the feed-forward */
    const float *Wa, *ba;         /* [C, F], [F]: first feed-forward map */
    const float *Wb, *bb;         /* [F, C], [C]: second feed-forward map */
} ts3_block_weights;               /* device float32; no pointer may be NULL
                                      except the pa biases */

typedef struct ts3_stack ts3_stack; /* opaque */

/* A stack of n_blocks blocks of layer shape `desc` (bf16 storage) with hidden
 * width `hidden` = F.  Supported (C, F): (128, 512), (256, 1024); otherwise
 * TS3_ERR_UNSUPPORTED.  Allocates n_blocks layer states plus two activation
 * buffers of max_points * C bf16 and one block's feed-forward fragments. */
ts3_status ts3_stack_create(const ts3_desc *desc, int32_t n_blocks, int32_t hidden, ts3_stack **out);
ts3_status ts3_stack_free(ts3_stack *s);
ts3_status ts3_stack_bytes(const ts3_stack *s, int64_t *bytes);

/* Block l's layer state (owned by the stack; valid until ts3_stack_free),
 * for ts3_state_get / ts3_state_set. */
ts3_status ts3_stack_layer(ts3_stack *s, int32_t l, ts3_state **layer);

/* The whole stack over a resident mesh x (bf16 [N][C], overwritten with the
 * last block's output): per block, ts3_layer_forward with `tile` and `chunk`
 * on LN1(x), then the feed-forward half.  blocks[0..n_blocks-1].  Leaves
 * every block's state ATTENDED (its cached Z).  Allocates nothing. */
ts3_status ts3_stack_forward(ts3_stack *s, const ts3_block_weights *blocks, void *x, int64_t N,
                             int64_t tile, int64_t chunk, void *stream);

/* Decoding at arbitrary query points from the cached states (section 3.3,
 * Eq. (5)): q (bf16 [n][C], overwritten) runs through every block with its
 * Physics-Attention decoded from that block's Z (ts3_deslice in chunks of
 * `chunk` points) instead of re-slicing the mesh.  Every block's state must
 * be ATTENDED (after ts3_stack_forward, or ts3_state_set on each layer).
 * n <= max_points; n == 0 is a no-op. */
ts3_status ts3_stack_decode(ts3_stack *s, const ts3_block_weights *blocks, void *q, int64_t n, int64_t chunk,
                            void *stream);

/* The feed-forward half of block l on its own: x (bf16 [n][C], overwritten)
 * becomes y + W_b^T GELU(W_a^T LN2(y) + b_a) + b_b with y = x + pa, where pa
 * is block l's Physics-Attention output for x.  If xn_next is not NULL and
 * l + 1 < n_blocks, also writes block l+1's LN1 of the result there.  The
 * block's own share of ts3_stack_forward; exposed for timing and tests. */
ts3_status ts3_stack_feedforward(ts3_stack *s, const ts3_block_weights *blocks, int32_t l, void *x,
                                 const void *pa, int64_t n, void *xn_next, void *stream);

const char *ts3_status_string(ts3_status s);
const char *ts3_last_error(void); /* thread-local detail of the last failure */

#ifdef __cplusplus
}
#endif
#endif /* TS3_H */
