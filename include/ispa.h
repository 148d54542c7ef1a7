/*
 * ispa.h -- C ABI of libispa: the data-parallel hot path of Instance-Specific
 * Parametric Absorption (ISPA, arXiv 2607.00712) on AMD Instinct MI355X
 * (gfx950).
 *
 * Three operations, each defined by the paper:
 *   ispa_attn_chunk        chunk attention of an F-Layer (full cache) or an
 *                          L-Layer (sink + sliding window), optionally both
 *                          from one pass (Sec. 2 Eq. 3; Sec. 3.4 Eq. 7-12)
 *   ispa_accum_stats       warmup statistics: residual R = y_full - y_local,
 *                          G += X^T X, C += X^T R, ||R||^2 (Sec. 3.2, Eq. 4-5
 *                          and the last paragraph of Sec. 3.2)
 *   ispa_solve_modulation  dW = (G + lambda I)^-1 C and the feasibility score
 *                          eps (Sec. 3.2, Eq. 5-6)
 * and the layer absorption that follows warmup (Sec. 3.3): ranking by eps,
 * the in-place weight update W + dW, the L-Layer cache after the permanent
 * eviction of the history, and the L-Layer's output projection.
 *
 * Conventions shared by every call
 *   - Matrices are row-major with the last dimension contiguous.
 *   - Device pointers point to device memory of the current HIP device and
 *     must be 16-byte aligned. The caller owns every buffer: the library never
 *     allocates or frees device memory and keeps no pointer beyond the work it
 *     enqueues, except the statistics workspace, which the handle uses until
 *     ispa_stats_destroy.
 *   - Work is enqueued on the caller's HIP stream (0 = the null stream) and
 *     runs asynchronously; only ispa_solve_modulation waits for the device
 *     (ispa_solve_modulation_async is its variant that does not).
 *   - Argument errors are reported before anything is enqueued, so a failing
 *     call writes nothing.
 *   - The return value is a status code (ISPA_OK or a negative ISPA_ERR_*).
 */
#ifndef ISPA_H
#define ISPA_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- status */
#define ISPA_OK                0
#define ISPA_ERR_INVALID_ARG (-1) /* null/misaligned pointer, size out of range */
#define ISPA_ERR_UNSUPPORTED (-2) /* head_dim or dtype not supported            */
#define ISPA_ERR_NOT_SPD     (-3) /* G + lambda I has a non-positive pivot      */
#define ISPA_ERR_HIP         (-4) /* a HIP launch or runtime call failed        */
#define ISPA_ERR_STATE       (-5) /* bad handle or workspace                    */
#define ISPA_ERR_SCRATCH     (-6) /* needs more than the library's fixed scratch */

/* element types of ispa_accum_stats inputs */
#define ISPA_DTYPE_BF16 0
#define ISPA_DTYPE_F32  1

/* Human-readable name of a status code (static string, never NULL). */
const char* ispa_status_string(int status);

/* ABI version of this header (major * 100 + minor). */
int ispa_abi_version(void);

/* ------------------------------------------------------------ attention */
/*
 * Attention of one chunk's queries against one layer's KV cache.
 *
 * Sec. 2, Eq. 3: Q comes from the current chunk; K and V are the cached past
 * followed by the current chunk, so the last n_q of the cache_len cached keys
 * are the current chunk, and every query sees all keys of its set (no mask
 * inside a chunk). Sec. 3.4, Eq. 7-8: the local set is the sink prefix plus the
 * most recent keys, the history is everything between them:
 *
 *   local = [0, min(sink_len, N)) U [max(N - window, 0), N)      N = cache_len
 *   hist  = [0, N) minus local
 *
 * Each set is attended with ordinary softmax attention returning the output and
 * its natural-log log-sum-exp (Eq. 9-10); full = local U hist (Eq. 11-12).
 *
 *   q          bf16 [n_q, n_heads * head_dim]   current chunk's queries
 *   k_cache    bf16 [>= cache_len, n_heads * head_dim]  keys; rows >= cache_len
 *              are never read
 *   v_cache    bf16 [>= cache_len, n_heads * head_dim]  values, same layout
 *   cache_len  N: keys in the cache, the current chunk included; n_q <= N
 *   window     w >= 1: number of most recent keys in the local set
 *              (window >= cache_len - sink_len makes the local set the full
 *              cache: an F-Layer)
 *   sink_len   s >= 0: number of leading (sink) keys in the local set
 *   n_q        >= 1 queries; n_heads >= 1; head_dim in {64, 128}
 *   scale      logit scale; <= 0 selects 1/sqrt(head_dim)
 *   out        fp32 [n_q, n_heads * head_dim]
 *   lse        fp32 [n_heads, n_q] or NULL
 *   out_local  fp32 [n_q, n_heads * head_dim] or NULL
 *   lse_local  fp32 [n_heads, n_q] or NULL (needs out_local)
 *
 * Single-stream form (out_local == NULL): out/lse receive attention over the
 * local set (an L-Layer; an F-Layer when the window covers the cache).
 * Dual-stream form (out_local != NULL, the warmup of Sec. 3.1 step 1): one pass
 * writes the local-set result to out_local/lse_local and the full-set result to
 * out/lse, which equals the LSE fusion of Eq. 11-12 of the local and history
 * branches. Outputs must not overlap the inputs or each other.
 */
int ispa_attn_chunk(const void* q, const void* k_cache, const void* v_cache,
                    int64_t cache_len, int64_t window, int64_t sink_len,
                    int32_t n_q, int32_t n_heads, int32_t head_dim, float scale,
                    float* out, float* lse, float* out_local, float* lse_local,
                    hipStream_t stream);

/*
 * ispa_attn_chunk with the work split over the whole chip. Whole work items
 * (256 queries of one head over all their keys) per workgroup can leave a
 * large part of the last round of workgroups idle (e.g. 12 heads x 19 query
 * blocks = 228 work items on 256 compute units). Split, every workgroup takes
 * an equal run of (work item, 64-key tile) units; runs that end inside a work
 * item leave a normalised partial output and LSE in the workspace, combined
 * with Eq. 11-12 in run order. At head_dim 128 the run that completes a work
 * item combines them inside the same kernel (the runs count themselves on
 * per-item counters in the workspace, which the call clears first); at
 * head_dim 64 a merge kernel combines them after the launch. The results
 * agree with ispa_attn_chunk within rounding (the merge reassociates the
 * softmax sums) and do not depend on which run finishes last.
 *
 *   segments   < 0: never split (exactly ispa_attn_chunk)
 *              0:   split when whole work items would fill the device poorly
 *              > 0: split into exactly this many runs (at most the number of
 *                   units)
 *   workspace  device, 256-byte aligned, at least ispa_attn_workspace_bytes
 *              bytes for the same arguments on the same device; may be NULL
 *              when that is 0. Used only during the call's device work.
 * Other arguments and outputs as for ispa_attn_chunk.
 */
int ispa_attn_chunk_ws(const void* q, const void* k_cache, const void* v_cache,
                       int64_t cache_len, int64_t window, int64_t sink_len,
                       int32_t n_q, int32_t n_heads, int32_t head_dim, float scale,
                       float* out, float* lse, float* out_local, float* lse_local,
                       int32_t segments, void* workspace, size_t workspace_bytes,
                       hipStream_t stream);

/* Workspace bytes ispa_attn_chunk_ws needs for these arguments on the current
 * device (dual != 0: the dual-stream form); 0 when it does not split or the
 * arguments are invalid. */
size_t ispa_attn_workspace_bytes(int64_t cache_len, int64_t window, int64_t sink_len,
                                 int32_t n_q, int32_t n_heads, int32_t head_dim,
                                 int32_t dual, int32_t segments);

/*
 * ispa_attn_chunk_ws with segments = 0 (the automatic split) for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation. The split's partial results go to a
 * scratch array that the library holds in device memory, one per GPU, for the
 * life of the process (ISPA_STATIC_SCRATCH_BYTES), instead of a caller
 * workspace; the call itself allocates and frees nothing.
 *   Arguments, outputs and results as for ispa_attn_chunk_ws (bitwise the same
 *   outputs for the same inputs).
 *   Returns ISPA_ERR_SCRATCH, before enqueueing anything, when the split needs
 *   more than ISPA_STATIC_SCRATCH_BYTES (ispa_attn_workspace_bytes with
 *   segments = 0 tells; a dual-stream chunk of 4680 queries over 7 chunks of
 *   cache that splits, e.g. with 10 heads x 128, needs 129 MiB).
 * Every call on one GPU uses the same array: calls that overlap on one GPU
 * (other streams, other threads) race and give undefined results. The array
 * needs no clearing: the call clears the counters it uses and writes every
 * partial result before it is read.
 */
#define ISPA_STATIC_SCRATCH_BYTES ((size_t)160 << 20)
int ispa_attn_chunk_noalloc(const void* q, const void* k_cache, const void* v_cache,
                            int64_t cache_len, int64_t window, int64_t sink_len,
                            int32_t n_q, int32_t n_heads, int32_t head_dim, float scale,
                            float* out, float* lse, float* out_local, float* lse_local,
                            hipStream_t stream);

/*
 * Attention over an explicit key set: one branch of the decomposable form of
 * Sec. 3.4 (Eq. 9-10), e.g. the history alone.
 *
 *   ranges     host array of n_ranges [begin, end) pairs of cache rows, each
 *              0 <= begin < end <= 2^31; the rows must exist in k_cache and
 *              v_cache. The set is their union (ranges should not overlap).
 *   n_ranges   0..3; 0 is the empty set: out = 0 and lse = -inf, the values
 *              that make ispa_attn_merge return the other branch unchanged.
 * q, k_cache, v_cache, n_q, n_heads, head_dim, scale, out, lse as for
 * ispa_attn_chunk (single-stream form).
 */
int ispa_attn_ranges(const void* q, const void* k_cache, const void* v_cache,
                     const int64_t* ranges, int32_t n_ranges,
                     int32_t n_q, int32_t n_heads, int32_t head_dim, float scale,
                     float* out, float* lse, hipStream_t stream);

/*
 * LSE fusion of two attention results over disjoint key sets (Sec. 3.4,
 * Eq. 11-12):
 *   lse = ln(e^lse_a + e^lse_b)  (evaluated as m + ln(e^(lse_a-m) + e^(lse_b-m)))
 *   out = e^(lse_a - lse) out_a + e^(lse_b - lse) out_b
 * Two empty branches (lse -inf) give out = 0, lse = -inf.
 *   out_a, out_b, out   fp32 [n_q, n_heads * head_dim]; out may be out_a or out_b
 *   lse_a, lse_b        fp32 [n_heads, n_q] (natural log)
 *   lse                 fp32 [n_heads, n_q] or NULL; must not overlap lse_a/lse_b
 *   head_dim            a positive multiple of 4
 */
int ispa_attn_merge(const float* out_a, const float* lse_a, const float* out_b, const float* lse_b,
                    int32_t n_q, int32_t n_heads, int32_t head_dim,
                    float* out, float* lse, hipStream_t stream);

/* ---------------------------------------------------------- statistics */
/*
 * Sufficient statistics of one layer's absorption problem (Sec. 3.2): the
 * method sums A_loc^T A_loc and A_loc^T R over the warmup rows and solves one
 * D x D system at the end of warmup. A handle is host-side state over a
 * caller-owned device workspace that holds every device-side quantity:
 *   G      fp32 [d_in, d_in]    sum of X^T X (lower block triangle valid)
 *   C      fp32 [d_in, d_out]   sum of X^T R
 *   s      fp64                 sum of ||R||_F^2
 *   plus staging for up to max_rows rows of bf16 X and R, and the factor of
 *   the solve.
 * A handle is not thread-safe; different handles are independent.
 */
typedef struct ispa_stats ispa_stats;

/* Bytes of device workspace a handle needs (0 if the sizes are invalid:
 * d_in, d_out in [1, 16384], d_in a multiple of 64, max_rows >= 1). */
size_t ispa_stats_workspace_bytes(int32_t d_in, int32_t d_out, int64_t max_rows);

/* Creates a handle over `workspace` (device, 256-byte aligned, at least
 * ispa_stats_workspace_bytes bytes, owned by the caller and kept alive until
 * ispa_stats_destroy) and zeroes the statistics on `stream`. */
int ispa_stats_create(ispa_stats** handle, void* workspace, size_t workspace_bytes,
                      int32_t d_in, int32_t d_out, int64_t max_rows, hipStream_t stream);

/* Zeroes G, C, s and the row count (a new warmup, e.g. the event-triggered
 * recalibration of Sec. 3.3). Asynchronous on the handle's stream. */
int ispa_stats_reset(ispa_stats* handle);

/* Releases the host handle; the workspace is the caller's to free afterwards. */
int ispa_stats_destroy(ispa_stats* handle);

/* Device addresses of G, C and s inside the workspace, and the number of rows
 * accumulated so far (host). Any output pointer may be NULL. */
int ispa_stats_views(const ispa_stats* handle, float** G, float** C, double** sq_norm_r,
                     int64_t* n_rows);

/*
 * Adds n_rows warmup rows (Sec. 3.2):
 *   R  = bf16_rne(fp32(y_full) - fp32(y_local))       [n_rows, d_out]
 *   G += X^T X,  C += X^T R,  s += ||R||_F^2,  n += n_rows
 * with X = bf16_rne(x) when x is fp32. X holds A_loc (the input of the output
 * projection, heads concatenated); y_full/y_local are the full- and local-stream
 * outputs whose difference is to be absorbed: post-projection outputs A W give
 * the paper's dW directly, the attention outputs themselves give dW' with
 * dW = dW' W.
 *   x        [n_rows, d_in]  of x_dtype  (ISPA_DTYPE_BF16 or ISPA_DTYPE_F32)
 *   y_full   [n_rows, d_out] of y_dtype
 *   y_local  [n_rows, d_out] of y_dtype
 * Any n_rows >= 0 is accepted; rows are staged max_rows at a time.
 * Enqueued on the handle's stream.
 */
int ispa_accum_stats(ispa_stats* handle, const void* x, int32_t x_dtype,
                     const void* y_full, const void* y_local, int32_t y_dtype,
                     int64_t n_rows);

/*
 * Closed-form modulation (Sec. 3.2, Eq. 5): dW = (G + lambda I)^-1 C, by a
 * Cholesky factorisation of G + lambda I and two triangular solves, in fp32.
 *   lambda    ridge weight added to the summed Gram matrix (the paper uses
 *             1e-3); lambda >= 0
 *   delta_w   fp32 [d_in, d_out] output (device)
 *   eps_out   host double or NULL: the feasibility score of Eq. 6,
 *             ||X dW - R||_F^2 = s - <dW, C> - lambda ||dW||_F^2
 * G and C are left unchanged, so the caller may solve again with another
 * lambda or keep accumulating. Waits for the handle's stream to finish; returns
 * ISPA_ERR_NOT_SPD (delta_w then unspecified) if a pivot is not positive.
 * From d_in = 4096 on (with d_out >= 128) the triangular solves of half of
 * C's columns run on a second stream that the library owns (one per device);
 * it waits for the handle's stream before it starts and the handle's stream
 * waits for it before the score, so the work stays ordered on the handle's
 * stream as seen by the caller (ISPA_SOLVE_TWO_STREAMS=0 keeps everything on
 * the handle's stream; the results are the same bits either way).
 */
int ispa_solve_modulation(ispa_stats* handle, float lambda, float* delta_w, double* eps_out);

/*
 * ispa_solve_modulation without the wait: enqueues the same work on the
 * handle's stream and returns. When it has run, eps_dev holds eps of Eq. 6
 * (the value ispa_solve_modulation reports) and status_dev holds 0, or 1 when
 * a pivot was not positive (delta_w and eps are then unspecified). For a
 * caller that reads the scores of many layers at once (the ranking of
 * Sec. 3.3) instead of waiting once per layer.
 *   eps_dev     device double (8-byte aligned) or NULL
 *   status_dev  device int32 (4-byte aligned) or NULL
 * Argument errors are returned before anything is enqueued.
 */
int ispa_solve_modulation_async(ispa_stats* handle, float lambda, float* delta_w, double* eps_dev,
                                int32_t* status_dev);

/*
 * The closed-form solves of several layers at once. At the end of warmup the
 * method computes dW and eps of every layer so that the layers can be ranked
 * by eps (Sec. 3.3); each layer's solve is the work of
 * ispa_solve_modulation_async (same arithmetic, bitwise the same results), but
 * one launch per step of the factorisation and of the sweeps covers every
 * layer, so the latency-bound chain of panel factorisations is paid once.
 *   handles     host array of n_layers statistics handles, 1 <= n_layers <=
 *               4096, with equal d_in, d_out and max_rows and equally spaced
 *               workspaces: workspace(i) = workspace(0) + i * stride, stride >=
 *               ispa_stats_workspace_bytes (handles created on consecutive
 *               equal slices of one buffer); all work is enqueued on the stream
 *               of handles[0]
 *   lambda      ridge weight, >= 0
 *   delta_w     fp32 device output: n_layers consecutive [d_in, d_out]
 *               row-major blocks, layer i at delta_w + i * d_in * d_out
 *   eps_dev     device double [n_layers] (8-byte aligned) or NULL: eps of each
 *               layer (Eq. 6)
 *   status_dev  device int32 [n_layers] (4-byte aligned) or NULL: 0, or 1 when
 *               that layer's G + lambda I had a pivot that was not positive
 * Argument errors (INVALID_ARG, or STATE for a bad handle) are returned before
 * anything is enqueued. Asynchronous; every layer's G and C are left intact.
 */
int ispa_solve_modulation_batch(ispa_stats* const* handles, int32_t n_layers, float lambda, float* delta_w,
                                double* eps_dev, int32_t* status_dev);

/*
 * Host-side check of the launch schedule of a single layer's Cholesky
 * factorisation in its look-ahead form (Sec. 3.2, Eq. 5; the solve takes that
 * form from 48 panels of 64 columns on): builds the schedule for n_panels
 * panels on n_cu compute units and walks every launch through the same
 * workgroup decode the kernel runs, checking that each 64 x 64 block on or
 * below the diagonal receives every earlier panel exactly once, in panel
 * order, after that panel was factored, that no block is written twice within
 * a launch, and that each launch finds its panel column complete. For tests;
 * touches no device. Returns 0 when the schedule is valid, a positive value
 * (the failing launch + 2, or n_panels + 1 for an incomplete block at the end)
 * otherwise, and -1 for n_panels < 1 or above 127 or n_cu < 1.
 */
int ispa_solve_lookahead_check(int32_t n_panels, int32_t n_cu);

/* ---------------------------------------------------------- absorption */
/*
 * Instance-specific layer selection (Sec. 3.3): the k layers with the lowest
 * feasibility score eps become L-Layers. Host-only (no device work).
 *   eps        host double [n_layers]
 *   k          0 <= k <= n_layers
 *   selected   host int32 [k]: layer indices in ascending eps order; ties by
 *              layer index, NaN after every number
 */
int ispa_select_layers(const double* eps, int32_t n_layers, int32_t k, int32_t* selected);

/*
 * In-place weight update of an L-Layer's output projection (Sec. 3.3):
 * W_new = W + dW, one fp32 addition per element, rounded to nearest even for a
 * bf16 weight.
 *   weight        device [d_in, d_out] (transposed == 0: the row-vector form of
 *                 Eq. 4, Y = A W) or [d_out, d_in] (transposed != 0: a linear
 *                 layer's weight, Y = A W^T, which receives dW^T); of
 *                 weight_dtype ISPA_DTYPE_BF16 or ISPA_DTYPE_F32
 *   delta_w       device fp32 [d_in, d_out], as written by ispa_solve_modulation;
 *                 must not overlap weight
 * Asynchronous on `stream`.
 */
int ispa_inject_modulation(void* weight, int32_t weight_dtype, int32_t transposed, const float* delta_w,
                           int32_t d_in, int32_t d_out, hipStream_t stream);

/*
 * The permanent eviction of an L-Layer's history (Sec. 3.3): copies the local
 * set of Eq. 7 of a cache of cache_len keys into a compact ring buffer:
 *   ring rows [0, s')            = cache rows [0, s'),  s' = min(sink_len, N)
 *   ring rows [s', s' + w')      = the last w' = min(window, N - s') cache rows
 * The ring buffers hold at least s' + window rows of `hidden` bf16 values (the
 * window part keeps growing to `window` rows as keys arrive); `*ring_rows`
 * (host, may be NULL) receives s' + w'. The window rows then form a ring whose
 * head (window keys written so far) is w'; see ispa_kv_ring_append.
 *   k_cache, v_cache, k_ring, v_ring   device bf16, rows of `hidden` elements
 *                                       (hidden a multiple of 8), 16-byte aligned;
 *                                       the ring must not overlap the cache
 * Attention over the L-Layer is then ispa_attn_chunk on the ring with
 * cache_len = the filled ring rows and window >= cache_len (key order does not
 * matter to softmax attention). Asynchronous on `stream`.
 */
int ispa_kv_evict(const void* k_cache, const void* v_cache, int64_t cache_len, int64_t window, int64_t sink_len,
                  int32_t hidden, void* k_ring, void* v_ring, int64_t* ring_rows, hipStream_t stream);

/*
 * Appends n_new keys (k_new/v_new [n_new, hidden] bf16) to an L-Layer ring:
 * window key number head + r goes to ring row sink_rows + (head + r) mod window,
 * so the ring keeps the sink rows and the most recent `window` keys (the local
 * set of Eq. 7 of the whole sequence). head = window keys written so far (w'
 * after ispa_kv_evict); afterwards the caller's head is head + n_new and the
 * filled ring rows are sink_rows + min(head + n_new, window). Only the last
 * min(n_new, window) new keys are copied. Asynchronous on `stream`.
 */
int ispa_kv_ring_append(void* k_ring, void* v_ring, int64_t sink_rows, int64_t window, int64_t head,
                        const void* k_new, const void* v_new, int64_t n_new, int32_t hidden, hipStream_t stream);

/*
 * The output projection an L-Layer applies after absorption (Sec. 3.1 step 3
 * with W_new = W + dW of Sec. 3.3; Y = A W of Eq. 4), in the linear-layer
 * layout of the weight: y = a weight^T.
 *   a        device bf16 [n_rows, d_in] (the attention output, heads concatenated)
 *   weight   device bf16 [d_out, d_in] (e.g. after ispa_inject_modulation with
 *            transposed != 0)
 *   y        device [n_rows, d_out] of y_dtype (ISPA_DTYPE_F32 or ISPA_DTYPE_BF16,
 *            rounded to nearest even); must not overlap a or weight
 *   d_in     a multiple of 32; fp32 accumulation
 * a and weight 16-byte aligned. Asynchronous on `stream`.
 */
int ispa_project(const void* a, const void* weight, int64_t n_rows, int32_t d_in, int32_t d_out, void* y,
                 int32_t y_dtype, hipStream_t stream);

/*
 * Symmetric per-row int8 quantisation for the W8A8 form of the linear layers
 * (Sec. 4 combines the method with W8A8 and reports it compatible; the scheme
 * is not stated there): for each row, scale = absmax / 127 (1 for an all-zero
 * row) and code = clamp(round_half_even(x / scale), -127, 127), the division
 * and the rounding in IEEE fp32.
 *   x       device [rows, cols] of x_dtype (ISPA_DTYPE_BF16 or ISPA_DTYPE_F32),
 *           finite values, 16-byte aligned; rows are activations (one scale
 *           per token) or the rows of a linear weight [d_out, d_in] (one
 *           scale per output channel)
 *   q       device int8 [rows, cols], 8-byte aligned
 *   scale   device fp32 [rows]
 *   cols    a multiple of 8
 * q and scale must not overlap x or each other. Asynchronous on `stream`.
 */
int ispa_quantize_rows(const void* x, int32_t x_dtype, int64_t rows, int32_t cols, int8_t* q, float* scale,
                       hipStream_t stream);

/*
 * The W8A8 form of ispa_project: y = (q_a q_w^T) * scale_a[row] * scale_w[col]
 * with the codes of ispa_quantize_rows; the product is exact in int32 and the
 * dequantisation is fp32(acc) * scale_a, then * scale_w, one fp32 rounding
 * each (and one more to bf16 for a bf16 y).
 *   q_a, scale_a   device int8 [n_rows, d_in] and fp32 [n_rows]
 *   q_w, scale_w   device int8 [d_out, d_in] and fp32 [d_out]
 *   y              device [n_rows, d_out] of y_dtype (ISPA_DTYPE_F32 or
 *                  ISPA_DTYPE_BF16); must not overlap the inputs
 *   d_in           a multiple of 64, at most 65536 (no int32 overflow)
 * q_a and q_w 16-byte aligned. Asynchronous on `stream`.
 */
int ispa_project_w8a8(const int8_t* q_a, const float* scale_a, const int8_t* q_w, const float* scale_w, int64_t n_rows,
                      int32_t d_in, int32_t d_out, void* y, int32_t y_dtype, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* ISPA_H */
