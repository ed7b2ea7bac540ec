/*
 * xattn.h -- C ABI of the MI355X (gfx950) XAttention prefill library.
 *
 * XAttention (arXiv 2503.16428) replaces dense prefill attention by three
 * steps (Fig. 1): (1) strided antidiagonal block scoring, (2) threshold block
 * selection, (3) attention on the selected blocks only. Each step is one call
 * here, plus a dense reference mode and a chained forward.
 *
 * Conventions shared by every call
 *   - Plain C; no HIP or torch types. `stream` is a hipStream_t passed as
 *     void* (NULL = the default stream). Every call only validates its
 *     arguments on the host and enqueues kernels on `stream`: it never
 *     allocates, never synchronises and never throws. Results are ready when
 *     the caller synchronises the stream.
 *   - All array pointers are DEVICE pointers owned by the caller; the library
 *     keeps none of them after the call returns. Arrays are dense and
 *     row-major in the shapes stated below; tensors of bfloat16 values are
 *     passed as `const void*`.
 *   - Heads: query head h (0 <= h < batch*hq) reads key/value head
 *     (h / hq) * hkv + (h % hq) / (hq / hkv)  (contiguous GQA grouping).
 *   - Shapes use L = dims->seq, D = dims->head_dim, NB = L / block,
 *     HQ = batch * hq, HKV = batch * hkv.
 *   - Return value: XATTN_OK or an error code; on error nothing has been
 *     enqueued (argument errors) or the HIP launch failed (XATTN_ERR_HIP).
 *     xattn_last_error() gives a message for the calling thread.
 *   - Results are deterministic: the same inputs give bitwise equal outputs.
 *
 * Supported today: head_dim 128, block 128, stride S in {1,2,4,8,16,32,64},
 * seq a multiple of 128 and at most 262144 (NB <= 2048).
 */
#ifndef XATTN_H
#define XATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum xattn_status {
    XATTN_OK = 0,
    XATTN_ERR_ARG = 1,          /* invalid argument (null pointer, bad shape, tau <= 0 or NaN) */
    XATTN_ERR_UNSUPPORTED = 2,  /* valid but not implemented (e.g. head_dim != 128) */
    XATTN_ERR_WORKSPACE = 3,    /* workspace pointer null or smaller than required */
    XATTN_ERR_HIP = 4           /* a HIP runtime call or kernel launch failed */
};

/* Problem shape. Layouts: Q [batch][hq][seq][head_dim], K and V
 * [batch][hkv][seq][head_dim], all bfloat16. causal: 1 = query i attends to
 * keys k <= i (decoder prefill), 0 = bidirectional (e.g. video DiT). */
typedef struct xattn_dims {
    int32_t batch;
    int32_t hq;
    int32_t hkv;
    int32_t seq;
    int32_t head_dim;
    int32_t causal;
} xattn_dims;

/*
 * Step 1 -- strided antidiagonal block scoring (Sec. 3.1-3.2, Algorithm 1).
 *
 * For query head h, query block b and key block j, with nr = block / stride
 * reduced rows per block and reduced row R = b*nr + r:
 *   x[R][c]  = (1 / (sqrt(D) * S)) * sum_{t<S} q[R*S + S-1-t] . k[c*S + t]
 *              (the product of Algorithm 1's strided reshapes: the sum over
 *              the antidiagonal of every S x S sub-block of Q K^T),
 *   A[R][c]  = softmax over the valid reduced columns c (c <= R when causal),
 *   scores[h][b][j] = (1/nr) * sum_{r<nr} sum_{c in block j} A[R][c],
 * so every row sums to 1. Entries with j > b (causal) are written as 0.
 *   q        bf16 [HQ][L][D]          k  bf16 [HKV][L][D]
 *   scores   fp32 [HQ][NB][NB]        (output, fully written)
 *   workspace  device scratch of at least xattn_score_workspace_size() bytes;
 *              its contents on entry are ignored, on exit unspecified.
 * Products are bf16 x bf16 on the matrix cores with fp32 accumulation; the
 * softmax and block sums are fp32.
 */
int xattn_score_workspace_size(const xattn_dims *dims, int block, int stride,
                               size_t *bytes);
int xattn_score(const void *q, const void *k, const xattn_dims *dims, int block,
                int stride, float *scores, void *workspace, size_t workspace_bytes,
                void *stream);

/*
 * Step 1 with another sampling pattern inside each S x S sub-block (the
 * pattern ablation, Sec. 4.5, Table 4): the S summed positions are
 * (query sub-row qsub[t], key sub-row t), t < S, so
 *   X[R][c] = (1 / (S sqrt(D))) sum_{t<S} q[R*S + qsub[t]] . k[c*S + t].
 * qsub[t] = S-1-t is xattn_score (the antidiagonal); qsub[t] = t the main
 * diagonal; any other permutation (e.g. a seeded random one) the random
 * pattern, which keeps one position per sub-block row and column.
 *   qsub  host array of `stride` int32, a permutation of 0 .. stride-1; read
 *         during the call only (copied into the launch)
 * Everything else as xattn_score. XATTN_ERR_ARG if qsub is NULL or not a
 * permutation.
 */
int xattn_score_pattern(const void *q, const void *k, const xattn_dims *dims, int block,
                        int stride, const int32_t *qsub, float *scores, void *workspace,
                        size_t workspace_bytes, void *stream);

/*
 * Step 2 -- threshold block selection, find_blocks (Sec. 3.2, equation of
 * find_blocks; Algorithm 1). Per row (h, b) the candidates are j <= b
 * (causal) or all j. Each candidate's mass is taken as the integer
 * u_j = floor(clamp(scores[h][b][j], 0, 1) * 2^32); T = sum of u_j over the
 * candidates. The selected set is the shortest prefix (length >= 1) of the
 * candidates ordered by (u_j descending, j ascending) whose integer sum
 * reaches ceil(tau * T) (tau * T as one fp64 product). tau >= 1 selects every
 * candidate. Integer masses make the result independent of summation order.
 *   scores  fp32 [HQ][NB][NB]   (input; only candidate entries are read)
 *   tau     threshold, 0 < tau; values >= 1 mean "all candidates"
 *   idx     int32 [HQ][NB][NB]  (output) row (h, b): idx[h][b][0 .. cnt) are
 *           the selected key blocks in ascending order; later entries are
 *           left unchanged
 *   cnt     int32 [HQ][NB]      (output) number selected, >= 1
 */
int xattn_select(const float *scores, const xattn_dims *dims, int block, float tau,
                 int32_t *idx, int32_t *cnt, void *stream);

/*
 * Step 2 with one threshold per query head (the per-head thresholds that the
 * minimum-threshold prediction of Sec. 3.3 produces). Row (h, b) of batch
 * element n uses tau_h[h] (rows are indexed n * hq + h); otherwise exactly
 * xattn_select.
 *   tau_h  host array of dims->hq floats, each > 0 (values >= 1: all
 *          candidates); read during the call only (copied into the launch)
 * Errors: XATTN_ERR_ARG for a NULL array or a tau <= 0 / NaN,
 * XATTN_ERR_UNSUPPORTED for hq > 256.
 */
int xattn_select_heads(const float *scores, const xattn_dims *dims, int block,
                       const float *tau_h, int32_t *idx, int32_t *cnt, void *stream);

/*
 * Fixed-size block selection of the selection-strategy ablation (Sec. 4.5,
 * Table 6: Top-K and Top-Ratio against threshold selection). Per row the
 * candidates are ordered as in xattn_select, by (u_j descending, j
 * ascending) with u_j = floor(clamp(score, 0, 1) * 2^32), and the first k are
 * selected, k clamped to [1, m] for m candidates; output as xattn_select.
 *   Top-K:     k = k_h[h] key blocks (the paper quotes K in tokens: K tokens
 *              correspond to K / block blocks); host array of dims->hq
 *              int32, each >= 1
 *   Top-Ratio: k = floor(ratio_h[h] * m + 0.5) (fp32 ratio, product in
 *              fp64), at least 1; host array of dims->hq floats, each finite
 *              and > 0 (>= 1 keeps every candidate)
 * The arrays are read during the call only. Errors as xattn_select_heads.
 */
int xattn_select_topk(const float *scores, const xattn_dims *dims, int block,
                      const int32_t *k_h, int32_t *idx, int32_t *cnt, void *stream);
int xattn_select_ratio(const float *scores, const xattn_dims *dims, int block,
                       const float *ratio_h, int32_t *idx, int32_t *cnt, void *stream);

/*
 * Step 3 -- block-sparse attention (Fig. 1, right): for query i in block b of
 * head h, with K_i the keys of the listed key blocks idx[h][b][0 .. cnt)
 * (intersected with k <= i when causal):
 *   o[h][i]   = sum_{k in K_i} softmax_k(q_i . k_k / sqrt(D)) v_k
 *   lse[h][i] = log sum_{k in K_i} exp(q_i . k_k / sqrt(D))   (natural log)
 * A query with no visible key gets o = 0 and lse = -inf. Lists must hold
 * distinct ascending block indices in [0, NB); cnt in [0, NB].
 *   q  bf16 [HQ][L][D]; k, v bf16 [HKV][L][D]
 *   idx int32 [HQ][NB][NB], cnt int32 [HQ][NB]  (e.g. from xattn_select)
 *   o   bf16 [HQ][L][D] (output)
 *   lse fp32 [HQ][L] (output) or NULL
 * QK^T and PV run on the bf16 matrix cores with fp32 accumulation; the
 * online softmax is fp32 and P is rounded to bf16 for the PV product. The
 * normaliser sums the same rounded P (so o is a weighted mean of the values
 * with consistent weights); lse carries that rounding, at most 2^-8 relative
 * in the sum, i.e. below 0.004 in lse.
 */
int xattn_block_sparse_attn(const void *q, const void *k, const void *v,
                            const xattn_dims *dims, int block, const int32_t *idx,
                            const int32_t *cnt, void *o, float *lse, void *stream);

/*
 * Dense reference mode (the paper's speedup denominator, Sec. 4.3): the same
 * kernel as xattn_block_sparse_attn with every candidate block listed
 * (j <= b causal, all j otherwise), block 128. Bitwise equal to
 * xattn_block_sparse_attn on the lists xattn_select returns for tau >= 1.
 */
int xattn_dense_attn(const void *q, const void *k, const void *v,
                     const xattn_dims *dims, void *o, float *lse, void *stream);

/*
 * The three steps chained on one stream: score -> select -> sparse attention.
 * workspace: at least xattn_forward_workspace_size() bytes. It holds, in
 * order, scores fp32 [HQ][NB][NB], idx int32 [HQ][NB][NB], cnt int32 [HQ][NB]
 * (each at a 256-byte aligned offset reported by xattn_forward_layout) and
 * the scoring scratch; after the call the caller may read scores/idx/cnt there.
 */
int xattn_forward_workspace_size(const xattn_dims *dims, int block, int stride,
                                 size_t *bytes);
int xattn_forward_layout(const xattn_dims *dims, int block, int stride,
                         size_t *scores_off, size_t *idx_off, size_t *cnt_off,
                         size_t *scratch_off);
int xattn_forward(const void *q, const void *k, const void *v, const xattn_dims *dims,
                  int block, int stride, float tau, void *o, float *lse,
                  void *workspace, size_t workspace_bytes, void *stream);

/*
 * xattn_forward without allocation, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc. The workspace of xattn_forward lives in a static device
 * array of XATTN_NOALLOC_SCRATCH_BYTES bytes that the library owns (one per
 * GPU, held until the process ends; its address is looked up once per device
 * on the first call with that device current). The caller passes inputs and
 * outputs only; the call makes no allocation of any kind.
 *   Everything else as xattn_forward (o, lse and their meaning; results
 *   bitwise equal to xattn_forward's on the same inputs).
 * Errors: as xattn_forward, plus XATTN_ERR_UNSUPPORTED when the problem needs
 * more scratch than the static array holds (xattn_forward_workspace_size()
 * > XATTN_NOALLOC_SCRATCH_BYTES), and XATTN_ERR_HIP if the array's address
 * cannot be obtained.
 * Every call on one GPU shares that GPU's array, which keeps the last call's
 * contents: calls that overlap on one GPU (several streams or threads at
 * once) race and must be serialised by the caller.
 */
#define XATTN_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int xattn_forward_noalloc(const void *q, const void *k, const void *v, const xattn_dims *dims,
                          int block, int stride, float tau, void *o, float *lse, void *stream);

/*
 * Denoising-step schedule of the video-generation experiment (Sec. 4.2):
 * dense attention for the first warmup_steps steps of a diffusion sampler
 * (step < warmup_steps; the paper uses 5 of 50), XAttention from then on.
 *   step          0-based index of the current denoising step (>= 0)
 *   warmup_steps  number of leading dense steps (>= 0; 0 = never dense)
 * A dense step is exactly xattn_dense_attn (the workspace is not touched and
 * may be NULL); a later step is exactly xattn_forward with the same arguments.
 */
int xattn_forward_scheduled(const void *q, const void *k, const void *v,
                            const xattn_dims *dims, int block, int stride, float tau,
                            int step, int warmup_steps, void *o, float *lse,
                            void *workspace, size_t workspace_bytes, void *stream);

/*
 * Minimum-threshold prediction (Sec. 3.3). The paper fills a table D[h][m],
 * the best performance reachable with exactly m threshold adjustments over
 * the first h heads, each adjustment lowering one head's threshold by 10 %
 * (t <- 0.9 t); head h either keeps D[h-1][m] or takes one more adjustment on
 * top of D[h-1][m-1]. Here a head may take up to max_adjust adjustments
 * (max_adjust = 1 is the paper's recurrence) and performance is additive over
 * heads, given as a table from the caller (for instance minus each head's
 * output error at each adjusted threshold, from xattn_head_error).
 *   perf         host double [heads][max_adjust + 1]: perf[h][a] is head h's
 *                performance after a adjustments; finite
 *   adjustments  M, the total number of adjustments, 0 <= M <= heads * max_adjust
 *   adjust       host int32 [heads] (output): adjustments per head, summing
 *                to M; the threshold of head h becomes t0 * 0.9^adjust[h]
 *   best         host double (output, may be NULL): D[heads][M]
 * On equal performance a head keeps fewer adjustments. Host only (no GPU).
 * XATTN_ERR_ARG for a NULL table or adjust, heads < 1, max_adjust < 1, M
 * outside [0, heads * max_adjust] or a non-finite entry; XATTN_ERR_UNSUPPORTED
 * for tables above 2^26 entries or heads * max_adjust above 2^20.
 */
int xattn_threshold_dp(const double *perf, int heads, int max_adjust, int adjustments,
                       int32_t *adjust, double *best);

/*
 * The thresholds of the minimum-threshold prediction (Sec. 3.3): after a
 * reductions of 10 % from tau0 a head's threshold is tau0 * 0.9^a, computed
 * in fp64 and rounded once to the fp32 value the selection receives.
 *   levels  host float [max_adjust + 1] (output): levels[a] for a = 0 .. max_adjust
 * XATTN_ERR_ARG for a NULL array, tau0 <= 0 / not finite, or max_adjust < 0.
 * Host only (no GPU).
 */
int xattn_threshold_levels(double tau0, int max_adjust, float *levels);

/*
 * The whole prediction step of Sec. 3.3 on a per-head error table: the
 * dynamic program of xattn_threshold_dp with performance = minus the error
 * (the assignment of exactly `adjustments` reductions with the least total
 * error; on equal totals a head keeps fewer adjustments), followed by the
 * thresholds it implies.
 *   err        host double [heads][max_adjust + 1]: err[h][a] is head h's error
 *              after a reductions (e.g. xattn_head_error_mean at levels[a]); finite
 *   tau0       the threshold before any reduction (> 0)
 *   adjust     host int32 [heads] (output), summing to `adjustments`
 *   tau_h      host float [heads] (output): tau0 * 0.9^adjust[h] as in
 *              xattn_threshold_levels, ready for xattn_select_heads
 *   total_err  host double (output, may be NULL): the least total error
 * Errors as xattn_threshold_dp, plus XATTN_ERR_ARG for a bad tau0. Host only.
 */
int xattn_threshold_predict(const double *err, int heads, int max_adjust, int adjustments,
                            double tau0, int32_t *adjust, float *tau_h, double *total_err);

/*
 * Per-head output error, the performance proxy for xattn_threshold_dp:
 * err[h] = sum (o - o_ref)^2 / sum o_ref^2 over head h's [L][D] outputs
 * (bf16 inputs, fp64 accumulation, a fixed order: deterministic).
 *   o, o_ref   bf16 [HQ][L][D] device
 *   err        double [HQ] device (output)
 *   workspace  at least xattn_head_error_workspace_size() bytes of device memory
 */
int xattn_head_error_workspace_size(const xattn_dims *dims, size_t *bytes);
int xattn_head_error(const void *o, const void *o_ref, const xattn_dims *dims, double *err,
                     void *workspace, size_t workspace_bytes, void *stream);

/*
 * xattn_head_error averaged over the batch: err[h] for query head h < hq is
 * (1 / batch) * sum_n of the error of row n * hq + h, added in batch order
 * (the per-head table of the prediction covers heads of the model, not
 * sequences). err is double [hq] device (output); the workspace is the one
 * xattn_head_error_workspace_size() reports. Errors as xattn_head_error.
 */
int xattn_head_error_mean(const void *o, const void *o_ref, const xattn_dims *dims,
                          double *err, void *workspace, size_t workspace_bytes, void *stream);

/* Static description of a status code (never NULL). */
const char *xattn_strerror(int status);
/* Message describing the last failure on the calling thread ("" if none). */
const char *xattn_last_error(void);
/* Library ABI version: major * 10000 + minor * 100 + patch. */
int xattn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* XATTN_H */
