/*
 * sol_attn.h -- C ABI of the MI355X (gfx950) routed-attention library
 * (Sol-Attn forward pass: threshold routing, exact block-sparse attention and
 * proxy-score reuse fused into one online-softmax pass).
 *
 * All tensors are caller-owned, contiguous, row-major device buffers of shape
 * [B, H, N, d] (row stride d) unless stated otherwise.  Every entry point
 * validates its arguments on the host and returns a negative error code before
 * any GPU call when they are invalid; sol_attn_last_error() then describes the
 * problem.  Compute calls are asynchronous on the given HIP stream (a
 * hipStream_t passed as void*; NULL means the default stream) and do not
 * synchronise it.  GPU faults surface as SOL_ERR_HIP from a later synchronising
 * call (sol_attn_stats).
 *
 * Supported shapes: d in {64, 128}; block_k = 64; block_q in {64, 128};
 * N >= 1 with ragged last blocks (a block's statistics use only its valid
 * tokens); bf16 inputs (the hot path) and f32 inputs (a correctness-first
 * path).  The per-block routing lists live on chip, which bounds N: bf16 at
 * d = 128 up to 1,478,656 tokens (1,048,576 with a causal mask), at d = 64 up
 * to 1,971,200 (1,015,808 causal); beyond that the forward returns
 * SOL_ERR_UNSUPPORTED.  Two workgroups share a compute unit up to 245,760
 * tokens at d = 128 (causal too) and 737,280 at d = 64 (524,288 causal);
 * longer sequences run with one and take roughly twice as long per tile.  The softmax scale is 1/sqrt(d) for the exact logits and the
 * proxies alike.
 *
 * Range contract of the bf16 path (checked by nobody: outside it results are
 * undefined, typically inf/NaN, and no error code is returned):
 *   - v: every element within the f16 range (|v| <= 65504), in every mode: the
 *     value operand of the probability-times-value products is carried in f16;
 *   - q and k, in SOL_SPARSE only: every element of q and every block mean of k
 *     within the f16 range: the correction tiles multiply an f16 copy of the
 *     query rows by f16 copies of the pooled keys.
 * bf16 itself reaches 3.4e38, so these are real restrictions; attention inputs
 * of transformer layers sit far inside them.
 */
#ifndef SOL_ATTN_H
#define SOL_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Forward modes. */
enum {
    SOL_DENSE = 0,                /* softmax(QK^T/sqrt(d))V over all keys (Section 2, Eq. dense_attn) */
    SOL_SPARSE = 1,               /* routed exact blocks + zeroth-order correction
                                     (Section 3.2, Eqs. solattn_denominator and solattn_numerator) */
    SOL_SPARSE_NO_CORRECTION = 2  /* routed exact blocks only (Section 2, Eq. block_sparse_attn) */
};

/* Threshold estimator flag, OR-ed into `mode` of the forward calls and of
 * sol_attn_workspace_bytes (ignored by SOL_DENSE), or passed as the
 * threshold_mode of sol_attn_thresholds.  Without it sigma_i uses the full
 * pooled-key covariance (Eq. threshold_stats_exact); with it only the diagonal
 * v_K = mean_j(Kbar_j * Kbar_j) - mu_K * mu_K, sigma_i^2 = s^2 (Qbar_i * Qbar_i) . v_K
 * (Appendix, "Diagonal threshold estimator", Eq. appendix_diagonal_threshold). */
enum { SOL_THRESHOLD_DIAGONAL = 0x100 };

/* Element types of q, k, v and out. */
enum { SOL_BF16 = 0, SOL_F32 = 1 };

/* Return codes. */
enum {
    SOL_OK = 0,
    SOL_ERR_INVALID_ARG = -1,  /* null pointer, non-positive size, bad mode/dtype, NaN cutoff */
    SOL_ERR_UNSUPPORTED = -2,  /* valid but unsupported shape (d, block sizes, too many blocks) */
    SOL_ERR_HIP = -3,          /* a HIP runtime call failed (allocation, launch, sync) */
    SOL_ERR_WORKSPACE = -4,    /* caller workspace smaller than sol_attn_workspace_bytes() */
    SOL_ERR_NO_DATA = -5       /* sol_attn_stats: no forward wrote those counts, or B/H mismatch */
};

/*
 * Block mean pooling (Section 2, Eq. block_proxy: Qbar_i = Mean(Q_i),
 * Kbar_j = Mean(K_j); and the pooled values behind V_hat_j of Eq.
 * solattn_numerator, here as the mean, V_hat_j = n_j * Vbar_j).
 *
 * q, k, v:   [B,H,N,d] device, element type `dtype`.  A pointer may be NULL
 *            when the matching output is NULL.
 * qbar:      [B,H,ceil(N/block_q),d] f32 device, or NULL to skip.
 * kbar,vbar: [B,H,ceil(N/block_k),d] f32 device, or NULL to skip.
 * The last block of each kind averages only its n = N - (nb-1)*block valid
 * tokens.  Accumulation is in f32.
 */
int sol_attn_pool_blocks(const void* q, const void* k, const void* v,
                         float* qbar, float* kbar, float* vbar,
                         int B, int H, int N, int d, int block_q, int block_k,
                         int dtype, void* stream);

/*
 * Query-dependent thresholds from pooled inputs (Section 3.1, Eq.
 * threshold_routing with the moment form of Eq. threshold_stats_exact):
 *   mu_i    = s * Qbar_i . mean_j(Kbar_j)
 *   sigma_i = s * sqrt(Qbar_i C_K Qbar_i^T),  C_K the population covariance of
 *             the routable pooled keys (centred, accumulated in f64)
 *   tau_i   = mu_i + beta * sigma_i  (beta = -inf -> -inf, beta = +inf -> +inf)
 * with s = 1/sqrt(d).  Only the first nk_routable pooled keys take part.
 *
 * qbar: [B,H,NQ,d] f32 device; kbar: [B,H,NK,d] f32 device (NK >= nk_routable,
 * row stride d, NK rows per (b,h)).  tau (required), mu, sigma (optional):
 * [B,H,NQ] f32 device.  beta must not be NaN.  threshold_mode: 0 (exact) or
 * SOL_THRESHOLD_DIAGONAL.  Unlike the forward calls this entry point allocates
 * temporary device memory for the moments and synchronises `stream` before
 * returning.
 */
int sol_attn_thresholds(const float* qbar, const float* kbar,
                        float* tau, float* mu, float* sigma,
                        int B, int H, int NQ, int NK, int nk_routable, int d,
                        float beta, int threshold_mode, void* stream);

/*
 * Baseline routing with a materialised proxy map: the top-k and top-p selection rules
 * that Section 2 describes over the proxy row s_hat_i of Eq. block_proxy and its softmax
 * p_hat_i.  Provided to measure what the on-the-fly threshold routing of the forward
 * calls avoids; the forward never uses it.
 *
 * Writes proxies[b,h,i,j] = s * Qbar_i . Kbar_j (s = 1/sqrt(d)) for the first nk_routable
 * key blocks, then selects per query block:
 *   SOL_ROUTE_TOPK: the param = k largest proxies (1 <= k <= nk_routable, nk_routable <= 8192);
 *   SOL_ROUTE_TOPP: the shortest prefix of the blocks in decreasing proxy order whose mass
 *     under p_hat_i = Softmax(s_hat_i) reaches param = p (0 < p <= 1; a block is kept while
 *     the mass before it is below p; nk_routable <= 4096).
 * Ties go to the lower key-block index.
 *
 * qbar: [B,H,NQ,d] f32 device; kbar: [B,H,NK,d] f32 device (NK >= nk_routable);
 * proxies: [B,H,NQ,nk_routable] f32 device (written; caller-owned scratch);
 * mask_out: [B,H,NQ,ceil(nk_routable/32)] u32 device bit mask (bit j%32 of word j/32).
 * Asynchronous on `stream`.
 */
enum { SOL_ROUTE_TOPK = 0, SOL_ROUTE_TOPP = 1 };
int sol_attn_route_materialized(const float* qbar, const float* kbar, float* proxies, uint32_t* mask_out,
                                int B, int H, int NQ, int NK, int nk_routable, int d,
                                int rule, float param, void* stream);

/*
 * Routed attention forward, short form: bf16 q/k/v/out, default stream,
 * library-managed workspace, per-head counts kept for sol_attn_stats().
 * `tau` is the standardised cutoff beta of Eq. threshold_routing; mode is one
 * of SOL_DENSE, SOL_SPARSE, SOL_SPARSE_NO_CORRECTION, optionally OR-ed with
 * SOL_THRESHOLD_DIAGONAL.
 */
int sol_attn_forward(const void* q, const void* k, const void* v, void* out,
                     int B, int H, int N, int d, int block_q, int block_k,
                     float tau, int mode);

/*
 * Routed attention forward, full form.
 *
 * q, k, v (in), out (out): [B,H,N,d] device, element type `dtype`; out must not
 *   alias q, k or v.
 * tau: standardised cutoff beta (tau_i = mu_i + beta*sigma_i per query block,
 *   Eq. threshold_routing).  -INFINITY keeps every routable block (sparse modes
 *   then equal dense), +INFINITY keeps none.  Ignored by SOL_DENSE.  NaN is an
 *   error.
 * keep_tail_tokens: the last keep_tail_tokens tokens (a multiple of block_k,
 *   e.g. the text tokens of an MMDiT; Appendix, "Generation Configurations")
 *   form forced key blocks that are always computed exactly and take no part
 *   in the routing statistics or the counts.  0 for none.
 * workspace/workspace_bytes: caller device scratch of at least
 *   sol_attn_workspace_bytes(...) bytes, or NULL/0 to let the library allocate
 *   (and keep, growing on demand) its own.  It holds the pre-pass results and
 *   the fused kernel's work-queue counters, so two calls that may run at the
 *   same time (different streams) need different workspaces; calls that pass
 *   NULL share the library's one per device.
 * counts: [B,H] u32 device, or NULL for a library buffer.  After the call,
 *   counts[b*H+h] = number of (query block, routable key block) pairs selected
 *   for exact computation (all routable pairs in SOL_DENSE).
 * mask_out: [B,H,NQ,ceil(NKr/32)] u32 device bit mask of the selection (bit
 *   j%32 of word j/32 for key block j), or NULL.  Debug/parity aid; not
 *   written in SOL_DENSE.
 * mode: SOL_DENSE, SOL_SPARSE or SOL_SPARSE_NO_CORRECTION, optionally OR-ed with
 *   SOL_THRESHOLD_DIAGONAL (any other bit is an error).
 * stream: hipStream_t or NULL.
 *
 * Selection is computed on chip from f32 pooled proxies s*Qbar_i.Kbar_j and
 * never written to memory unless mask_out is given.  In the sparse modes the
 * library also orders the query blocks of each head by their pooled queries, so
 * that blocks with similar selections run together and share L2, and starts a
 * block's walk over its selected key blocks at a phase set by its place in that
 * schedule.  Neither changes which blocks are selected; the start phase changes
 * the order in which a block's exact tiles are accumulated, so results differ
 * from an increasing-order walk by rounding only.  Both are functions of the
 * inputs, so results are deterministic, and with every block selected the walk
 * starts at block 0, so tau = -INFINITY reproduces SOL_DENSE bit for bit.
 */
int sol_attn_forward_ex(const void* q, const void* k, const void* v, void* out,
                        int B, int H, int N, int d, int block_q, int block_k,
                        float tau, int mode, int dtype, int keep_tail_tokens,
                        void* workspace, size_t workspace_bytes,
                        uint32_t* counts, uint32_t* mask_out, void* stream);

/*
 * Routed attention forward under a causal mask (the row-dependent masks the
 * Appendix's error analysis names as future work: they need centring and
 * multiplicity over the valid keys).  Arguments as sol_attn_forward_ex, with no
 * forced tail, plus:
 *
 * causal_granule (G >= 1): key s is visible to query t iff
 *   s < min((t / G + 1) * G, N).  G = 1 is token-causal attention; G = the
 *   tokens of one frame gives frame-causal (autoregressive video) attention;
 *   G >= N is bidirectional attention.
 *
 * For query block i the key blocks every one of its rows sees are its routable
 * blocks: mu_i and sigma_i are the mean and population deviation of the proxies
 * over those blocks only (taken on chip from the proxies themselves), selection
 * is s_hat_ij > mu_i + beta*sigma_i among them, and an unselected one enters the
 * correction with its full valid-token count.  Key blocks only some rows see are
 * computed exactly under the token mask; blocks no row sees are skipped.
 * counts and mask_out cover the routable blocks only (mask bits of other blocks
 * are 0); sol_attn_stats divides by the routable pairs of this mask.
 * mode must not include SOL_THRESHOLD_DIAGONAL.  The workspace is the one
 * sol_attn_workspace_bytes(..., keep_tail_tokens = 0) returns.
 */
int sol_attn_forward_causal(const void* q, const void* k, const void* v, void* out,
                            int B, int H, int N, int d, int block_q, int block_k,
                            float tau, int mode, int dtype, int causal_granule,
                            void* workspace, size_t workspace_bytes,
                            uint32_t* counts, uint32_t* mask_out, void* stream);

/*
 * Routed attention forward that allocates nothing: sol_attn_forward_ex with
 * the library's built-in device scratch as the workspace.  For callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): it calls no hipMalloc/hipFree and
 * no allocating library routine.
 *
 * Arguments as sol_attn_forward_ex without the workspace; counts is required
 * (the library's own counts buffer would have to be allocated).  The scratch
 * is a 64 MiB array per GPU, held from the library's load until the process
 * ends; a shape whose sol_attn_workspace_bytes() exceeds it returns
 * SOL_ERR_WORKSPACE before any GPU call.  Every call on one GPU uses that
 * GPU's one array (everything it needs zeroed is cleared on the call's stream
 * by a fill kernel), so two calls that overlap on one GPU (different streams
 * or threads) race and give undefined results: serialise them.  The counts it
 * writes are not tracked for sol_attn_stats (tracking creates an event):
 * frac[b*H+h] = counts[b*H+h] / (NQ * NKr).
 */
int sol_attn_forward_noalloc(const void* q, const void* k, const void* v, void* out,
                             int B, int H, int N, int d, int block_q, int block_k,
                             float tau, int mode, int dtype, int keep_tail_tokens,
                             uint32_t* counts, uint32_t* mask_out, void* stream);

/* Device workspace bytes sol_attn_forward_ex needs for these arguments, or 0
 * if they are invalid/unsupported. */
size_t sol_attn_workspace_bytes(int B, int H, int N, int d, int block_q, int block_k,
                                int mode, int dtype, int keep_tail_tokens);

/*
 * Per-head selected-block fraction of a forward call (the per-head sparsity
 * counter): frac_per_head[b*H+h] = counts[b*H+h] / (routable pairs of one head),
 * NQ * NKr without a mask (host float array of B*H entries, written).
 *
 * counts: the [B,H] u32 device buffer a forward call of this library wrote
 *   (the `counts` argument of sol_attn_forward_ex / sol_attn_forward_causal),
 *   or NULL for the library's own counts buffer as written by the last forward
 *   on the calling thread that passed counts = NULL (sol_attn_forward always
 *   does).  The library remembers, per counts buffer, the shape of the forward
 *   that last wrote it, so two forwards in flight on two streams with their own
 *   counts buffers each keep their own statistics.  A caller-owned buffer must
 *   still be allocated when this is called.
 * Waits for the forward that last wrote the buffer (an event recorded on its
 * stream, so the stream itself may have been destroyed since), then copies the
 * counts to the host.  Returns SOL_ERR_NO_DATA if the buffer was not written by
 * a forward of this library, if counts is NULL and the last forward on this
 * thread used a caller-owned buffer (or there was none), or if B/H differ from
 * that forward's.
 */
int sol_attn_stats(float* frac_per_head, int B, int H, const uint32_t* counts);

/*
 * Kernel timing (profiling aid).  While enabled, every forward records a pair
 * of HIP events around its fused attention kernel on the call's stream (at most
 * 4096 launches are kept).  sol_attn_kernel_timing() waits for the recorded
 * launches, returns their total milliseconds and count, and clears them.
 */
int sol_attn_timing_enable(int enable);
int sol_attn_kernel_timing(float* total_ms, int* launches);

/* Message for the last non-zero return on the calling thread ("" if none). */
const char* sol_attn_last_error(void);

/* Free library-owned workspace and counter buffers (all devices).  The next
 * forward reallocates. */
int sol_attn_release(void);

#ifdef __cplusplus
}
#endif

#endif /* SOL_ATTN_H */
