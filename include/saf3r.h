/*
 * saf3r.h -- C ABI of the SAF3R block-sparse global-attention hot path for
 * AMD Instinct MI355X (gfx950).
 *
 * SAF3R (Dynamic Sparse Attention for Feed-Forward 3D Reconstruction
 * Transformers) gives every attention head of a cross-view global-attention
 * layer a sparse pattern class chosen offline (Sec. 4.2) and, for dynamic
 * heads, picks the kept keys online from a cheap probe (Sec. 4.3). This
 * library runs that online stage at block granularity in three calls:
 *
 *   saf3r_estimate_blocks   pooled (mean) Q and K per 64-token block
 *   saf3r_select_blocks     kept key blocks per query block, per head class
 *   saf3r_sparse_attention  softmax attention over the kept blocks only
 *
 * plus a debug check of the kept-block lists (saf3r_validate_index).
 *
 * Tensor conventions (all calls):
 *   - Q, K, V, O are device arrays [heads, N, 64], row-major, N = frames *
 *     tokens_per_frame (tokens of frame f are [f*T, (f+1)*T)); element type
 *     is bf16 (SAF3R_BF16) or fp32 (SAF3R_F32), the same for all four.
 *   - Blocks are 64 tokens: block b holds tokens [64b, min(64b+64, N)); the
 *     last block may be partial. nb = ceil(N / 64).
 *   - Every device pointer is owned by the caller, must be valid for the
 *     sizes stated, and must not alias another argument.
 *   - Alignment: Q, K, V, O, q_pooled, the NMSE inputs and every workspace
 *     are read or written with 16-byte vector accesses and must be 16-byte
 *     aligned; k_pooled, scores and nmse_out 8-byte; block_idx, block_cnt,
 *     lse and the list check's workspace 4-byte; cosine features to their
 *     element size. A misaligned
 *     pointer returns SAF3R_ERR_INVALID_ARGUMENT. The library
 *     allocates nothing and keeps no state between calls; calls on different
 *     streams may run concurrently when their outputs do not overlap.
 *   - `problem` and `table` are host pointers read during the call only.
 *   - `stream` is a hipStream_t (NULL = the default stream). Work is enqueued
 *     asynchronously; the call returns after the launches (saf3r_validate_index
 *     alone waits for its result).
 *   - Every argument is validated on the host before anything is launched; a
 *     call that returns an error has enqueued nothing (but for
 *     SAF3R_ERR_CORRUPT_INDEX, the outcome of the list check). SAF3R_ERR_HIP
 *     reports a launch error from the HIP runtime.
 */
#ifndef SAF3R_H
#define SAF3R_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SAF3R_OK = 0,
  SAF3R_ERR_INVALID_ARGUMENT = -1, /* null or misaligned pointer, non-positive size, bad dtype */
  SAF3R_ERR_UNSUPPORTED = -2,      /* head_dim or block other than 64, sizes beyond the limits */
  SAF3R_ERR_CAPACITY = -3,         /* cap or a workspace smaller than required */
  SAF3R_ERR_HIP = -4,              /* the HIP runtime reported an error on launch */
  SAF3R_ERR_BAD_TABLE = -5,        /* unknown pattern class, or a class parameter out of range */
  SAF3R_ERR_CORRUPT_INDEX = -6     /* saf3r_validate_index found a list that breaks its form */
} saf3r_status;

typedef enum { SAF3R_F32 = 0, SAF3R_BF16 = 1 } saf3r_dtype;

/* Head pattern classes (Sec. 4.1 kernels; assignment from the offline
 * profile of Sec. 4.2). `param` is the class parameter:
 *   SAF3R_DENSE         full attention ("Full" in the ablations); param unused;
 *   SAF3R_FRAME_LOCAL   static kernel: a query block keeps every key block
 *                       that shares at least one frame with it (block
 *                       granularity, so a block straddling two frames keeps
 *                       the key blocks of both); param unused;
 *   SAF3R_TOPK          query-probe Top-K kernel (Sec. 4.3) per query block:
 *                       keep the param key blocks j with the largest score
 *                       qbar_i . kbar_j / sqrt(64), ties to the lower j;
 *                       param in [1, nb];
 *   SAF3R_ANCHOR        static kernel, anchor-frame form (Sec. 4.1): every
 *                       query block keeps the key blocks holding a token of
 *                       frame param; param in [0, frames);
 *   SAF3R_STRIDE        uniform sampling kernel (Sec. 4.1): every query
 *                       attends to key tokens 0, s, 2s, ... with s = param;
 *                       param in [1, N]; token granularity, no block list;
 *   SAF3R_GLOBAL_PROBE  query-probe Top-K as Sec. 4.3 states it: one probe
 *                       per head, the mean qbar of all N queries; keep the
 *                       param key blocks with the largest qbar . kbar_j / 8,
 *                       ties to the lower j, the same list for every query
 *                       block; param in [1, nb];
 *   SAF3R_COSINE_TOPK   DINO Top-K kernel, block-wise (Sec. 4.1, 4.3): per
 *                       frame, the param key blocks whose caller-supplied
 *                       features are most similar to the query block's;
 *                       param in [1, 64]. Lists come from
 *                       saf3r_cosine_select, once per sequence;
 *   SAF3R_SKIP          not a pattern: every call leaves the head's pooled
 *                       data, lists, counts, outputs and lse untouched. A
 *                       caller splits one layer into independent launches
 *                       (e.g. static heads on one stream while the Top-K
 *                       heads are pooled and selected on another) by
 *                       marking the other heads SKIP; param unused.
 */
typedef enum {
  SAF3R_DENSE = 0,
  SAF3R_FRAME_LOCAL = 1,
  SAF3R_TOPK = 2,
  SAF3R_ANCHOR = 3,
  SAF3R_STRIDE = 4,
  SAF3R_GLOBAL_PROBE = 5,
  SAF3R_COSINE_TOPK = 6,
  SAF3R_SKIP = 7
} saf3r_pattern;

typedef struct {
  int32_t pattern; /* saf3r_pattern */
  int32_t param;   /* class parameter, see saf3r_pattern */
} saf3r_head_cfg;  /* host array [heads] */

typedef struct {
  int32_t heads;            /* 1 .. 256 */
  int32_t frames;           /* >= 1 */
  int32_t tokens_per_frame; /* >= 1; N = frames * tokens_per_frame, 1 .. 1048576 */
  int32_t head_dim;         /* must be 64 */
  int32_t block;            /* must be 64 */
  int32_t dtype;            /* saf3r_dtype */
} saf3r_problem;

/* Number of 64-token blocks, ceil(N / 64), or a negative saf3r_status. */
int32_t saf3r_num_blocks(const saf3r_problem* problem);

/* Smallest `cap` accepted by saf3r_select_blocks / saf3r_cosine_select /
 * saf3r_sparse_attention: the longest kept-block list of any FRAME_LOCAL,
 * TOPK, ANCHOR, GLOBAL_PROBE or COSINE_TOPK head (at least 1), or a negative
 * saf3r_status. DENSE and STRIDE heads need no list. */
int32_t saf3r_index_capacity(const saf3r_problem* problem, const saf3r_head_cfg* table);

/* Block pooling (Sec. 4.3: the probe of a set of queries is their mean).
 * For every TOPK and GLOBAL_PROBE head h, block b and dimension d:
 *   q_pooled[h][b][d] = mean of Q[h][t][d] over the tokens t of block b
 *   k_pooled[h][d][b] = mean of K[h][t][d] likewise (dimension-major, so
 *                       that the scoring pass reads it coalesced)
 * in float64 (a partial last block is divided by its own token count).
 *   q, k      device, [heads, N, 64] of problem->dtype
 *   q_pooled  device, float64 [heads, nb, 64]
 *   k_pooled  device, float64 [heads, 64, nb]
 *   Entries of the other heads are left untouched.
 * Returns SAF3R_OK, or an error with nothing enqueued. */
saf3r_status saf3r_estimate_blocks(const saf3r_problem* problem, const saf3r_head_cfg* table,
                                   const void* q, const void* k,
                                   double* q_pooled, double* k_pooled, void* stream);

/* Kept key blocks per query block (Sec. 4.1 static and query-probe Top-K
 * kernels; block scores are the exact tile means of Q K^T / sqrt(64),
 * Sec. 4.3). For head h and query block i:
 *   DENSE:        block_cnt[h][i] = nb; block_idx[h][i][:] left untouched
 *                 (attention treats the head as dense);
 *   FRAME_LOCAL:  the contiguous range of key blocks sharing a frame with i;
 *   TOPK:         the param highest scores s[i][j] = qbar_i . kbar_j / 8
 *                 (computed in float64), ties to the lower j;
 *   ANCHOR:       the contiguous range of key blocks of frame param;
 *   STRIDE:       block_cnt[h][i] = ceil(ceil(N / param) / 64), the number of
 *                 64-key groups of the sampled keys; block_idx untouched;
 *   GLOBAL_PROBE: the param highest probe scores qbar . kbar_j / 8 with qbar
 *                 the mean of all N queries (float64), ties to the lower j,
 *                 the same list in every row i;
 *   COSINE_TOPK:  block_idx and block_cnt left untouched (their lists come
 *                 from saf3r_cosine_select and stay valid across layers).
 * Lists are written ascending, padded with -1 up to cap.
 *   q_pooled, k_pooled device float64, [heads, nb, 64] and [heads, 64, nb], as
 *                      written by saf3r_estimate_blocks (read for TOPK and
 *                      GLOBAL_PROBE heads only)
 *   block_idx          device int32 [heads, nb, cap]
 *   block_cnt          device int32 [heads, nb]
 *   cap                >= saf3r_index_capacity(problem, table)
 *   scores_or_null     NULL, or device float64 [heads, nb, nb]: the full score
 *                      matrix of every TOPK head; for a GLOBAL_PROBE head the
 *                      probe scores in row 0 (other rows and heads untouched)
 *   workspace_or_null  NULL: the TOPK rows are scored and selected in one
 *                      launch whose workgroups keep 16 score rows in LDS (the
 *                      library allocates nothing). Otherwise device memory,
 *                      16-byte aligned, of workspace_bytes bytes, overwritten:
 *                      the TOPK scores go there as one launch, and a second
 *                      selects one row per wave at higher occupancy (faster).
 *                      It must hold at least one TOPK head's share,
 *                      saf3r_select_workspace_bytes / (number of TOPK heads);
 *                      with less than the full size the heads are done in
 *                      batches. Both ways give the same lists.
 * Returns SAF3R_OK; SAF3R_ERR_CAPACITY for a cap or a workspace too small;
 * another error code with nothing enqueued. */
saf3r_status saf3r_select_blocks(const saf3r_problem* problem, const saf3r_head_cfg* table,
                                 const double* q_pooled, const double* k_pooled,
                                 int32_t* block_idx, int32_t* block_cnt, int32_t cap,
                                 double* scores_or_null, void* workspace_or_null,
                                 int64_t workspace_bytes, void* stream);

/* Checks the kept-block lists (a debug call, not on the hot path). For every
 * query block i of every FRAME_LOCAL, TOPK, ANCHOR, GLOBAL_PROBE and
 * COSINE_TOPK head h: 0 <= block_cnt[h][i] <= cap, and equal to param for
 * TOPK and GLOBAL_PROBE heads (Sec. 4.3 keeps exactly that many); the first
 * block_cnt[h][i] entries of block_idx[h][i] strictly ascending inside
 * [0, nb), which rules out repeats; the rest of the row -1. These are the
 * lists saf3r_select_blocks and saf3r_cosine_select write. DENSE, STRIDE and
 * SKIP heads are not read. Each row is read within its cap entries, whatever
 * it holds.
 *   block_idx, block_cnt  device, as for saf3r_sparse_attention
 *   cap                   entries per row, >= 1
 *   workspace             device, 8 bytes, 4-byte aligned, overwritten
 *   first_bad_or_null     host; on SAF3R_ERR_CORRUPT_INDEX, the lowest
 *                         failing row as h * nb + i
 * The call enqueues its check on `stream` and waits for the stream to finish
 * (it reads the result back).
 * Returns SAF3R_OK; SAF3R_ERR_CORRUPT_INDEX if a row fails; SAF3R_ERR_HIP;
 * another error code with nothing enqueued. */
saf3r_status saf3r_validate_index(const saf3r_problem* problem, const saf3r_head_cfg* table,
                                  const int32_t* block_idx, const int32_t* block_cnt, int32_t cap,
                                  int32_t* workspace, int32_t* first_bad_or_null, void* stream);

/* Workspace of saf3r_select_blocks that takes every TOPK head in one batch:
 * (TOPK heads) x nb x 64 x C x 4 bytes, C = ceil(nb / 64) rounded up to a
 * multiple of 4 (198 MB for 10 TOPK heads at nb = 2147); 0 without TOPK
 * heads; or a negative saf3r_status. */
int64_t saf3r_select_workspace_bytes(const saf3r_problem* problem, const saf3r_head_cfg* table);

/* Attention restricted to the kept keys (Sec. 4.1: compute only the scores
 * between the queries and the selected keys, softmax renormalised over
 * them). For a query token t of block i of head h, with U the tokens of the
 * blocks listed for (h, i) (all tokens for a DENSE head; tokens 0, s, 2s, ...
 * for a STRIDE head with s = param):
 *   z_u    = q_t . k_u / 8,  u in U
 *   out[t] = sum_u softmax(z)_u v_u
 *   lse[t] = log(sum_u exp(z_u))            (natural log)
 * bf16 inputs: Q K^T and P V on bf16 matrix cores with fp32 accumulation, the
 * softmax in fp32, P rounded to bf16 for P V and for the row sum that
 * normalises out and gives lse, out rounded to bf16. So on this path lse is
 * the log of the sum of the bf16-rounded weights exp(z_u - max) plus max: it
 * differs from the fp32 log-sum-exp by up to 2^-8 (bf16's relative rounding
 * of each weight), and a caller that merges lse across launches inherits that
 * bias. fp32 inputs: everything in fp32.
 *   q, k, v      device [heads, N, 64] of problem->dtype
 *   block_idx, block_cnt, cap   as written by saf3r_select_blocks; entries of
 *                DENSE and STRIDE heads are not read. A list that is not
 *                ascending, repeats a block or holds indices outside [0, nb)
 *                gives unspecified output values but no access outside the
 *                head's N rows of Q, K, V and O (saf3r_validate_index
 *                checks a set of lists beforehand): every K/V tile is read
 *                through a buffer descriptor bounded by the head's extent
 *                (an index outside [0, nb) reads a tile of zeros, and so do
 *                the rows past N of a partial last block).
 *   out          device [heads, N, 64] of problem->dtype
 *   lse_or_null  NULL, or device float32 [heads, N]
 *   workspace_or_null, workspace_bytes
 *                NULL: every query block of a head is one work item. A
 *                device buffer (16-byte aligned, workspace_bytes >= 0, else
 *                SAF3R_ERR_INVALID_ARGUMENT) of at least
 *                saf3r_attention_workspace_bytes(problem, table) bytes
 *                (else SAF3R_ERR_CAPACITY): heads of two kinds run as 4 items
 *                per query block, one per quarter of the key range (for L2
 *                locality, bf16 only: on layers of 4096 or more key blocks,
 *                list heads whose list can hold 384 or more key blocks; for
 *                load balance: list or dense heads whose query blocks walk
 *                at least 32 (bf16) or 8 (fp32) key blocks, more than twice
 *                the key blocks that all list and dense heads' query blocks
 *                walk, divided by 2048 wave slots), and a second launch merges
 *                the 4 partial softmax results per query in a fixed order
 *                (results differ from the unsplit launch only by fp32
 *                rounding and the bf16 rounding of P against each range's
 *                running max). Lists that are not ascending are still read
 *                within their row. The buffer is overwritten; launches that
 *                share one must be ordered on the GPU.
 * Returns SAF3R_OK, or an error with nothing enqueued. */
saf3r_status saf3r_sparse_attention(const saf3r_problem* problem, const saf3r_head_cfg* table,
                                    const void* q, const void* k, const void* v,
                                    const int32_t* block_idx, const int32_t* block_cnt, int32_t cap,
                                    void* out, float* lse_or_null, void* workspace_or_null,
                                    int64_t workspace_bytes, void* stream);

/* Workspace of saf3r_sparse_attention that splits its long lists:
 * (split heads) x 4 x nb x 16896 bytes, where the split heads are the heads
 * saf3r_sparse_attention describes: on a bf16 layer of nb >= 4096 key
 * blocks, the FRAME_LOCAL / TOPK / ANCHOR / GLOBAL_PROBE / COSINE_TOPK heads
 * whose list can hold 384 or more key blocks (2.9 GB for 10 such heads at
 * nb = 4294); and on any layer, list or DENSE heads whose rows are long
 * against the layer's total work (the dense head of a 10992-token layer:
 * 11.6 MB); 0 if there are none; or a negative saf3r_status. */
int64_t saf3r_attention_workspace_bytes(const saf3r_problem* problem, const saf3r_head_cfg* table);

/* Workspace bytes saf3r_cosine_select needs for features of width
 * feat_dim: (feat_dim * nb + nb * nb) * 8, or a negative saf3r_status. */
int64_t saf3r_cosine_workspace_bytes(const saf3r_problem* problem, int32_t feat_dim);

/* Per-frame cosine Top-K lists of every COSINE_TOPK head (the DINO Top-K
 * kernel of Sec. 4.1, block-wise variant of Sec. 4.3). Each token's feature
 * is scaled to unit length and averaged over its block (float64); the block
 * similarity sim[i][j] = fbar_i . fbar_j is the mean cosine similarity over
 * the tile of token pairs. For head h (param k) and query block i the kept
 * blocks are, for every frame f, the min(k, |B_f|) blocks j of
 * B_f = { j : floor(64 j / tokens_per_frame) = f } with the largest sim[i][j]
 * (ties to the lower j), written ascending and padded with -1. The lists
 * depend on the features only: the paper computes them once per sequence
 * and reuses them in every layer, and saf3r_select_blocks leaves these rows
 * untouched so a caller can do the same.
 *   features         device [N, feat_dim] of problem->dtype; every row non-zero
 *   feat_dim         1 .. 4096
 *   workspace        device, >= saf3r_cosine_workspace_bytes bytes, 8-byte
 *                    aligned; overwritten (block features, similarity matrix)
 *   block_idx, block_cnt, cap   as for saf3r_select_blocks; only rows of
 *                    COSINE_TOPK heads are written
 * Returns SAF3R_OK, or an error with nothing enqueued. */
saf3r_status saf3r_cosine_select(const saf3r_problem* problem, const saf3r_head_cfg* table,
                                 const void* features, int32_t feat_dim, void* workspace,
                                 int64_t workspace_bytes, int32_t* block_idx, int32_t* block_cnt,
                                 int32_t cap, void* stream);

/* Device workspace of saf3r_nmse in bytes (heads x 128 float64 pairs), or
 * a negative status for a bad problem. */
int64_t saf3r_nmse_workspace_bytes(const saf3r_problem* problem);

/* Approximation cost of Eq. 1 (Sec. 4.2, offline head profiling) for one
 * input: per head h,
 *   nmse_out[h] = sum (o_full - o_sparse)^2 / sum o_full^2
 * over the head's N x 64 outputs, accumulated in float64 in a fixed order
 * (the same bits on every call with the same inputs).
 *   o_full, o_sparse  device [heads, N, 64] of problem->dtype (16-byte aligned)
 *   workspace         device, >= saf3r_nmse_workspace_bytes bytes, 16-byte
 *                     aligned; overwritten with per-slice partial sums
 *   nmse_out          device float64 [heads]
 * Returns SAF3R_OK; SAF3R_ERR_INVALID_ARGUMENT for a null pointer;
 * SAF3R_ERR_CAPACITY for a workspace that is too small; nothing is enqueued
 * on an error. */
saf3r_status saf3r_nmse(const saf3r_problem* problem, const void* o_full, const void* o_sparse,
                        void* workspace, int64_t workspace_bytes, double* nmse_out,
                        void* stream);

/* saf3r_nmse without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation). The per-slice partial sums go to a 512 KB array that
 * the library holds on each GPU it runs on, until the process ends; it fits
 * every head count the library accepts (up to 256), and a problem that
 * would need more returns SAF3R_ERR_CAPACITY. Results are the same bits as
 * saf3r_nmse's. The first call on a device resolves the array's address
 * (hipGetSymbolAddress), so make it outside graph capture. Calls on one GPU
 * share the array: calls that overlap (on streams with no ordering between
 * them) race and give undefined results.
 *   o_full, o_sparse, nmse_out   as for saf3r_nmse
 * Returns SAF3R_OK; SAF3R_ERR_INVALID_ARGUMENT for a null or misaligned
 * pointer; SAF3R_ERR_HIP if the array's address cannot be resolved; nothing
 * is enqueued on an error. */
saf3r_status saf3r_nmse_noalloc(const saf3r_problem* problem, const void* o_full,
                                const void* o_sparse, double* nmse_out, void* stream);

/* Static description of a status code (never NULL). */
const char* saf3r_status_string(int32_t status);

#ifdef __cplusplus
}
#endif

#endif /* SAF3R_H */
