/*
 * polestar.h -- C ABI of the MI355X (gfx950) hot path of Polestar's cached
 * denoising step (arxiv 2607.14107): drift -> select -> sparse K/V refresh ->
 * bidirectional attention -> Polestar-Commit, for one layer of a masked
 * diffusion LLM.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All array arguments are DEVICE pointers (HIP device memory of the
 *    current device); scalars are passed by value.  The caller owns every
 *    buffer.  The library allocates nothing and keeps no mutable global
 *    state; calls are reentrant.
 *  - Arrays are dense and row-major in the index order written next to them,
 *    e.g. [batch][seq][d] means element (b, i, c) is at ((b*seq)+i)*d + c.
 *  - `dtype` selects the element type of the hidden states, weights, caches,
 *    Q/out buffers and logits: POLESTAR_FP32 (float) or POLESTAR_BF16
 *    (bfloat16 stored as uint16 bit patterns).  Reductions and softmax
 *    arithmetic are fp32; results stored in bf16 are rounded to nearest even.
 *  - Every call validates its arguments on the host first and returns
 *    POLESTAR_ERR_INVALID_ARGUMENT (nothing enqueued) for a NULL required
 *    pointer, a negative or zero size where a positive one is required, or
 *    inconsistent sizes; POLESTAR_ERR_UNSUPPORTED for shapes or alignments the
 *    kernels do not handle (all array pointers must be 16-byte aligned; bf16
 *    rows of d elements need d % 8 == 0, fp32 rows d % 4 == 0;
 *    head_dim must be 64 or 128).  It then enqueues its kernels on `stream`
 *    and returns without synchronising.  POLESTAR_ERR_LAUNCH reports a failed
 *    launch.  Faults inside kernels surface at the caller's next
 *    synchronisation.
 *  - Entry points with a `workspace` take caller-provided device scratch of
 *    at least the size returned by the matching *_workspace_size function
 *    for the same shape (POLESTAR_ERR_WORKSPACE if smaller).  Its contents
 *    need no initialisation and are garbage after the call; two calls in
 *    flight at once need two workspaces.
 */
#ifndef POLESTAR_H
#define POLESTAR_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    POLESTAR_OK = 0,
    POLESTAR_ERR_INVALID_ARGUMENT = 1,
    POLESTAR_ERR_UNSUPPORTED = 2,
    POLESTAR_ERR_LAUNCH = 3,
    POLESTAR_ERR_WORKSPACE = 4
} polestar_status;

typedef enum { POLESTAR_FP32 = 0, POLESTAR_BF16 = 1 } polestar_dtype;

/* Version of this ABI: major*10000 + minor*100 + patch. */
int polestar_version(void);

/* Static, human-readable name of a status code. */
const char* polestar_status_string(polestar_status s);

/*
 * polestar_drift -- token representation drift (Sec. 3, eq. "drift").
 *
 * The paper measures a token's drift as KL(current || previous) of its
 * distribution at two consecutive denoising steps.  Here the distribution of
 * token (b, i) is the softmax of its layer-input hidden state over the d
 * channels, so, in nats,
 *     drift[b][i] = KL( softmax(h_cur[b][i][:]) || softmax(h_prev[b][i][:]) ).
 * It is evaluated in fp32 as
 *     sum_c p_c*dl_c - log(Za / Zb),   dl = (h_cur - max h_cur) - (h_prev - max h_prev),
 * with each row's exponentials taken against its own maximum (Za, Zb its
 * softmax denominators) and Za - Zb summed term by term through expm1 where
 * the rows are close, so rows that differ by any finite amount give a finite
 * result and identical rows give exactly 0.  Tiny negative results of
 * rounding are returned as they are.
 *
 *   h_cur, h_prev : [batch][seq][d] dtype   current / cached hidden states
 *   drift         : [batch][seq] float      output
 * Requires batch, seq, d > 0.
 */
polestar_status polestar_drift(polestar_dtype dtype, int batch, int seq, int d,
                               const void* h_cur, const void* h_prev, float* drift,
                               hipStream_t stream);

/*
 * polestar_select -- stale-position selection (Alg. 1, TopK of the drift).
 *
 * Candidates of sequence b are the cached positions I = J \ J_b (Sec. 2,
 * block-wise KV caching: positions outside the active block
 * [block_start, block_start + block_len)) for which eligible[b][i] != 0
 * (eligible == NULL: every cached position).  The k candidates with the
 * largest drift are chosen; equal drift values (+0.0 and -0.0 are equal)
 * rank the lower position first.  The chosen positions are written in
 * ascending order.
 *
 *   drift       : [batch][seq] float (NaN is outside the contract)
 *   eligible    : [batch][seq] uint8 or NULL
 *   k           : per-sequence budget, 0 <= k <= seq
 *   stale_idx   : [batch][k] int32 output, ascending, padded with -1
 *   stale_count : [batch] int32 output, min(k, number of candidates)
 * Requires batch, seq > 0, 0 <= block_start, block_len >= 0,
 * block_start + block_len <= seq; stale_idx may be NULL only when k == 0.
 */
polestar_status polestar_select(int batch, int seq, const float* drift,
                                const uint8_t* eligible, int block_start, int block_len,
                                int k, int32_t* stale_idx, int32_t* stale_count,
                                hipStream_t stream);

/*
 * polestar_refresh_kv -- sparse K/V refresh (Sec. 4.1, "Measuring Drift and
 * Layer-wise KV Updates"; Corollary 1 of App. B).
 *
 * For every row r of R_b = {stale_idx[b][0 .. stale_count[b]-1]} U J_b
 * (the active block is recomputed every step, Sec. 2):
 *     k_cache[b][r] = W_k h_cur[b][r],   v_cache[b][r] = W_v h_cur[b][r]
 * with fp32 accumulation, rounded to the cache dtype.  Rows outside R_b
 * keep their bytes.  A stale index inside J_b is legal (the row is written
 * twice with the same value).
 *
 *   h_cur          : [batch][seq][d] dtype
 *   stale_idx      : [batch][k_max] int32; entries 0 .. stale_count[b]-1 are
 *                    positions in [0, seq); an entry outside [0, seq) (e.g. the
 *                    -1 padding) is skipped: no row is written for it
 *   stale_count    : [batch] int32, clamped to [0, k_max] (a negative count
 *                    refreshes only the active block)
 *   w_k, w_v       : [n_kv_heads*head_dim][d] dtype (output x input)
 *   k_cache, v_cache : [batch][seq][n_kv_heads][head_dim] dtype, in/out
 *   workspace      : >= polestar_refresh_kv_workspace_size(...) bytes
 * Requires batch, seq, d, n_kv_heads > 0, k_max >= 0, block_len >= 0,
 * block_start + block_len <= seq.  stale_idx/stale_count may be NULL only
 * when k_max == 0.  UNSUPPORTED unless d % 128 == 0 (bf16) / d % 64 == 0
 * (fp32): the projection streams rows in 256-byte steps.
 */
size_t polestar_refresh_kv_workspace_size(polestar_dtype dtype, int batch, int d,
                                          int n_kv_heads, int head_dim,
                                          int k_max, int block_len);
polestar_status polestar_refresh_kv(polestar_dtype dtype, int batch, int seq, int d,
                                    int n_kv_heads, int head_dim, const void* h_cur,
                                    const int32_t* stale_idx, const int32_t* stale_count,
                                    int k_max, int block_start, int block_len,
                                    const void* w_k, const void* w_v,
                                    void* k_cache, void* v_cache,
                                    void* workspace, size_t workspace_bytes,
                                    hipStream_t stream);

/*
 * polestar_refresh_kv_noalloc -- polestar_refresh_kv without a workspace
 * argument, for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation).
 *
 * Same arguments (minus workspace), results and validation as
 * polestar_refresh_kv; it runs the same kernels.  The scratch that
 * polestar_refresh_kv takes from its workspace (split-K partials and the row
 * map) lives instead in one array of polestar_refresh_kv_noalloc_max_bytes()
 * bytes (64 MiB) of device memory per GPU, held by the library on each GPU it
 * runs on until the process ends.  The call allocates nothing: no hipMalloc,
 * hipFree or allocating library routine.  Shapes whose refresh needs more
 * scratch than that (polestar_refresh_kv_workspace_size above the maximum)
 * return POLESTAR_ERR_WORKSPACE with nothing enqueued.  Every call on one GPU
 * shares that GPU's array: two calls whose execution overlaps on the same GPU
 * (on different streams, or from different threads) race and give undefined
 * results; calls ordered on one stream are safe.  The first call on a device
 * looks up the array's device address (POLESTAR_ERR_LAUNCH if that fails).
 */
size_t polestar_refresh_kv_noalloc_max_bytes(void);
polestar_status polestar_refresh_kv_noalloc(polestar_dtype dtype, int batch, int seq, int d,
                                            int n_kv_heads, int head_dim, const void* h_cur,
                                            const int32_t* stale_idx, const int32_t* stale_count,
                                            int k_max, int block_start, int block_len,
                                            const void* w_k, const void* w_v,
                                            void* k_cache, void* v_cache, hipStream_t stream);

/*
 * polestar_project_q -- query projection of the active block (Sec. 2, eq. 3:
 * the queries of the active positions J_b).
 *
 *   q[b][j][h][:] = W_q[h*head_dim : (h+1)*head_dim] . h_cur[b][block_start + j]
 * in fp32 accumulation, rounded to dtype (round to nearest even).  It reads
 * neither cache, so it may run on a second stream while drift, select and
 * the K/V refresh run; polestar_attend with w_q == NULL then consumes q.
 *
 *   h_cur : [batch][seq][d] dtype
 *   w_q   : [n_heads*head_dim][d] dtype
 *   q     : [batch][block_len][n_heads][head_dim] dtype (output)
 *   workspace : >= polestar_project_q_workspace_size(...) bytes (0 when
 *               batch*block_len <= 64; NULL is then allowed)
 * Requires block_len > 0, block_start + block_len <= seq; UNSUPPORTED
 * unless head_dim is 64 or 128, d % 128 == 0 (bf16) / d % 64 == 0 (fp32),
 * batch <= 65535 and every pointer is 16-byte aligned.  The workspace needs
 * no initialisation.
 */
size_t polestar_project_q_workspace_size(polestar_dtype dtype, int batch, int d,
                                         int n_heads, int head_dim, int block_len);
polestar_status polestar_project_q(polestar_dtype dtype, int batch, int seq, int d,
                                   int n_heads, int head_dim, int block_start, int block_len,
                                   const void* h_cur, const void* w_q, void* q,
                                   void* workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/*
 * polestar_attend -- bidirectional attention of the active block over the
 * whole cache (Sec. 2, eq. 3; App. B setup).
 *
 * If w_q != NULL the queries are first projected, Q = W_q h_cur[b][J_b],
 * into q_buf (fp32 accumulation, rounded to dtype); if w_q == NULL, q_buf
 * already holds Q and h_cur is not read.  Then for every query head h,
 * with KV head g = h / (n_heads / n_kv_heads) (consecutive query heads share
 * a KV head):
 *     l_j = scale * q . k_cache[b][j][g],  a = softmax_j(l),
 *     out = sum_j a_j v_cache[b][j][g]      over all seq positions j
 * with no causal or padding mask.  scale <= 0 selects 1/sqrt(head_dim).
 * lse (optional) receives the natural-log log-sum-exp of the l_j.
 *
 *   h_cur   : [batch][seq][d] dtype (read when w_q != NULL)
 *   w_q     : [n_heads*head_dim][d] dtype or NULL
 *   q_buf   : [batch][block_len][n_heads][head_dim] dtype (out if w_q, else in)
 *   k_cache, v_cache : [batch][seq][n_kv_heads][head_dim] dtype
 *   out     : [batch][block_len][n_heads][head_dim] dtype
 *   lse     : [batch][n_heads][block_len] float or NULL
 *   workspace : >= polestar_attend_workspace_size(...) bytes
 * Requires n_heads % n_kv_heads == 0, block_len > 0,
 * block_start + block_len <= seq; with w_q, d % 128 == 0 (bf16) /
 * d % 64 == 0 (fp32) as for polestar_refresh_kv.
 */
size_t polestar_attend_workspace_size(polestar_dtype dtype, int batch, int seq, int d,
                                      int n_heads, int n_kv_heads, int head_dim,
                                      int block_len);
polestar_status polestar_attend(polestar_dtype dtype, int batch, int seq, int d,
                                int n_heads, int n_kv_heads, int head_dim,
                                int block_start, int block_len,
                                const void* h_cur, const void* w_q, void* q_buf,
                                const void* k_cache, const void* v_cache, float scale,
                                void* out, float* lse,
                                void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/*
 * polestar_commit -- Polestar-Commit for the current block (Sec. 4.2,
 * Alg. 1; confidence of Sec. 2 and eq. 1).
 *
 * For every block position j of sequence b:
 *   token[b][j] = argmax over v != mask_token_id of logits[b][j][v]
 *                 (equal logits: lowest id; mask_token_id < 0: none excluded)
 *   conf[b][j]  = exp(l_token - m) / sum_v exp(l_v - m), m = max_v l_v
 *                 (softmax over the whole vocabulary)
 * and for masked positions (masked[b][j] != 0), in fp32 with this order:
 *   n     = h > 0 ? hist_len[b] : 0
 *   mu    = n > 0 ? (((hist[b][0][j] + hist[b][1][j]) + ...) + hist[b][n-1][j]) / n : 0
 *   D     = dlt_j - mu,  dlt_j = drift[b][block_start + j] (0 if drift == NULL)
 *   t     = tau_s - conf;  tau_d = (alpha * t) * t
 *   commit[b][j] = conf > tau_s || D > tau_d
 * (drift == NULL turns the drift branch off: commit = conf > tau_s).
 * If force_one != 0 and no masked position of b commits, the masked position
 * with the largest conf (lowest j on ties) commits.  Unmasked positions never
 * commit.  Finally, when h > 0 and drift != NULL, dlt is pushed into the
 * history: entries stay oldest first, at most h are kept
 * (hist_len[b] = min(n + 1, h)).
 *
 *   logits   : [batch][block_len][vocab] dtype
 *   masked   : [batch][block_len] uint8
 *   drift    : [batch][seq] float or NULL
 *   hist     : [batch][h][block_len] float, in/out (may be NULL if h == 0)
 *   hist_len : [batch] int32, in/out, values in [0, h] (NULL if h == 0)
 *   token, conf, commit : [batch][block_len] int32 / float / uint8 outputs
 *   workspace : >= polestar_commit_workspace_size(...) bytes
 * Requires block_len, vocab > 0, h >= 0, mask_token_id < vocab, and
 * block_start + block_len <= seq when drift != NULL.  UNSUPPORTED for
 * block_len > 1024, h > 16, or vocab not a whole number of 16-byte chunks.
 */
size_t polestar_commit_workspace_size(polestar_dtype dtype, int batch, int block_len,
                                      int vocab);
polestar_status polestar_commit(polestar_dtype dtype, int batch, int block_len, int vocab,
                                const void* logits, const uint8_t* masked,
                                const float* drift, int seq, int block_start,
                                float* hist, int32_t* hist_len, int h,
                                int mask_token_id, float tau_s, float alpha, int force_one,
                                int32_t* token, float* conf, uint8_t* commit,
                                void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/*
 * polestar_suffix_commit -- suffix-block commit (Sec. 4.2 "Suffix Block
 * Commit"; Alg. 1, the commit from the final layer's update packet).
 *
 * The rows are positions of the suffix window whose logits come from the
 * final layer's update packet.  For every row j of sequence b, token and conf
 * are as in polestar_commit, and
 *   commit[b][j] = masked[b][j] && eligible[b][j] && conf > tau_s
 * (drift decides which suffix positions are eligible, confidence which of
 * them commit; no history, no forced commit).
 *   logits   : [batch][n_rows][vocab] dtype
 *   masked, eligible : [batch][n_rows] uint8
 *   token, conf, commit : [batch][n_rows] int32 / float / uint8 outputs
 *   workspace : >= polestar_commit_workspace_size(dtype, batch, n_rows, vocab)
 * Requires n_rows, vocab > 0 and mask_token_id < vocab.  UNSUPPORTED for
 * n_rows > 1024 or vocab not a whole number of 16-byte chunks.
 */
polestar_status polestar_suffix_commit(polestar_dtype dtype, int batch, int n_rows, int vocab,
                                       const void* logits, const uint8_t* masked,
                                       const uint8_t* eligible, int mask_token_id, float tau_s,
                                       int32_t* token, float* conf, uint8_t* commit,
                                       void* workspace, size_t workspace_bytes,
                                       hipStream_t stream);

/*
 * Clustered proxy drift -- Polestar's own drift estimator (Sec. 4.1 "Cluster
 * and Quantize Hidden States" and "Measuring Drift and Layer-wise KV
 * Updates"; Alg. 1: SphericalKMeans at block entry, ProxyAttn, KL and TopK
 * per step).  The window's hidden states are clustered once per block; at
 * every step each cluster's proxy token attends over the cache, its drift is
 * the KL between this step's and the last step's proxy distributions, and
 * the members of the top-k clusters are the rows to refresh.  An alternative
 * to polestar_drift + polestar_select; the refresh and everything after it
 * are unchanged.
 *
 * polestar_cluster -- spherical K-means of h[b][win_idx[b][i]] (i < n_win):
 * points are the directions h/|h|; centroid j starts at the point of window
 * rank floor(j*n_win/K); `iters` rounds of (assign each point to the centroid
 * of largest cosine, lowest cluster on ties; centroid = normalised sum of its
 * members' directions, an empty cluster keeps its centroid); then every point
 * is assigned to its nearest final centroid.
 *   h         : [batch][seq][d] dtype
 *   win_idx   : [batch][n_win] int32 window positions (entries are clamped
 *               into [0, seq); positions should be distinct)
 *   labels    : out [batch][seq] int32, the cluster of each window position,
 *               -1 elsewhere
 *   sums      : out [batch][K][d] float, sum of the members' hidden states
 *   counts    : out [batch][K] int32, members per cluster
 *   centroids : out [batch][K][d] float, the unit centroids
 * K = n_clusters.  UNSUPPORTED for K > 16, n_win > 2048, K*d > 32768,
 * d not a multiple of 512 (bf16) / 256 (fp32), or h, sums, centroids not
 * 16-byte aligned.
 * Runs once per block: one workgroup per sequence.
 */
polestar_status polestar_cluster(polestar_dtype dtype, int batch, int seq, int d, const void* h,
                                 const int32_t* win_idx, int n_win, int n_clusters, int iters,
                                 int32_t* labels, float* sums, int32_t* counts, float* centroids,
                                 hipStream_t stream);

/*
 * polestar_proxy_drift -- per step: proxy token t_k = sums[b][k] / counts[b][k]
 * rounded to dtype (zero for an empty cluster); query q = W_q t_k rounded to
 * dtype; per head h (KV head g = h / (n_heads / n_kv_heads))
 *     s_(k,h,j) = scale * q_(k,h) . k_cache[b][j][g]   for every j < seq;
 * and drift[b][k] = (1/n_heads) sum_h KL(softmax_j s_(k,h,.) ||
 * softmax_j s'_(k,h,.)) in nats, s' the previous step's scores.  The new
 * scores and their log-sum-exp then replace the previous ones.
 *   sums, counts : the cluster state (polestar_cluster / _update)
 *   w_q          : [n_heads*head_dim][d] dtype
 *   k_cache      : [batch][seq][n_kv_heads][head_dim] dtype (the refreshed cache)
 *   scores       : in/out [batch][K][n_heads][seq] float
 *   lse          : in/out [batch][K][n_heads] float (natural log)
 *   first        : nonzero at block entry: no previous scores are read,
 *                  drift is 0, the scores and lse are stored
 *   drift        : out [batch][K] float
 *   workspace    : >= polestar_proxy_drift_workspace_size(...) bytes
 * scale <= 0 selects 1/sqrt(head_dim).  UNSUPPORTED unless head_dim is 64 or
 * 128, d % 128 == 0 (bf16) / d % 64 == 0 (fp32), K <= 16,
 * K * (seq + head_dim) <= 36864 (one head's scores of every cluster are held
 * on chip), and sums, W_q, k_cache and the workspace are 16-byte aligned.
 */
size_t polestar_proxy_drift_workspace_size(polestar_dtype dtype, int batch, int seq, int d,
                                           int n_heads, int head_dim, int n_clusters);
polestar_status polestar_proxy_drift(polestar_dtype dtype, int batch, int seq, int d, int n_heads,
                                     int n_kv_heads, int head_dim, int n_clusters, const float* sums,
                                     const int32_t* counts, const void* w_q, const void* k_cache,
                                     float scale, float* scores, float* lse, int first, float* drift,
                                     void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * polestar_attention_drift -- drift of the attention distributions of given
 * query rows between two steps (Alg. 1: the commit drift delta = KL of the
 * last layer's main attention of the block's tokens against the previous
 * step's; the drift functional of Sec. 3).  For every sequence b, row r and
 * query head h (KV head h / (n_heads / n_kv_heads)):
 *   s_j = scale * q[b][r][h] . k_cache[b][j][kv],  a = softmax_j(s),
 *   KL_(r,h) = sum_j a_j (log a_j - log a'_j),  a' = softmax(previous scores)
 *   drift[b][r] = mean over h of KL_(r,h)   (0 when first != 0)
 * scores[b][r][h][:] and lse[b][r][h] hold the previous step's scores and
 * natural-log normaliser on entry and this step's on return (first != 0:
 * their contents on entry are ignored).  scale <= 0 selects 1/sqrt(head_dim).
 *   q : [batch][n_rows][n_heads][head_dim] dtype;  k_cache : [batch][seq][n_kv_heads][head_dim]
 *   scores : [batch][n_rows][n_heads][seq] float;  lse : [batch][n_rows][n_heads] float
 *   drift : out [batch][n_rows] float
 *   workspace : >= polestar_attention_drift_workspace_size(...) bytes (no init)
 * UNSUPPORTED unless head_dim is 64 or 128, n_rows <= 64 and q, k_cache are
 * 16-byte aligned.  polestar_proxy_drift runs the same kernels on its proxy
 * queries.
 */
size_t polestar_attention_drift_workspace_size(int batch, int seq, int n_rows, int n_heads);
polestar_status polestar_attention_drift(polestar_dtype dtype, int batch, int seq, int n_rows, int n_heads,
                                         int n_kv_heads, int head_dim, const void* q, const void* k_cache,
                                         float scale, float* scores, float* lse, int first, float* drift,
                                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * polestar_cluster_select -- the k_top clusters of largest drift (equal
 * drift: lower cluster first) of each sequence; their member positions
 * (labels[b][p] selected) go to stale_idx[b][0..count) in ascending order,
 * the rest of the row is -1, stale_count[b] = count (at most k_max: a row
 * with more members keeps the first k_max).  Feeds polestar_refresh_kv.
 *   labels : [batch][seq] int32 (polestar_cluster), drift : [batch][K] float
 *   stale_idx : out [batch][k_max] int32, stale_count : out [batch] int32
 */
polestar_status polestar_cluster_select(int batch, int seq, const int32_t* labels, int n_clusters,
                                        const float* drift, int k_top, int32_t* stale_idx, int k_max,
                                        int32_t* stale_count, hipStream_t stream);

/*
 * polestar_cluster_update -- after the refresh of the rows in
 * stale_idx[b][0..stale_count[b]): sums[b][labels[b][p]] += h_new[b][p] -
 * h_old[b][p] for each of them that lies in the window (labels >= 0),
 * accumulated in list order (deterministic).  Labels and counts stay.
 *   h_new, h_old : [batch][seq][d] dtype;  sums : in/out [batch][K][d] float
 * UNSUPPORTED unless d % 4 == 0 and K <= 16.
 */
polestar_status polestar_cluster_update(polestar_dtype dtype, int batch, int seq, int d,
                                        const void* h_new, const void* h_old, const int32_t* labels,
                                        int n_clusters, const int32_t* stale_idx,
                                        const int32_t* stale_count, int k_max, float* sums,
                                        hipStream_t stream);

/*
 * The rest of a pre-norm layer stack, for running the denoising loop of
 * Alg. 1 on a whole model (Sec. 5.1 evaluates LLaDA- and Dream-shaped
 * models).  Layer: x += W_o Attn(RMSNorm(x)); x += W_down(silu(W_gate g) *
 * W_up g), g = RMSNorm(x).  The residual stream x is fp32; everything else
 * is stored in dtype (bf16 rounding is to nearest even).  Asynchronous on
 * `stream`; the caller owns every buffer.
 *
 * polestar_embed -- x[b][r][:] = tok_emb[ids[b][lo + r]][:] + pos_emb[lo + r][:]
 *   for r < n_rows (ids clamped into [0, vocab)).
 *   ids : [batch][seq] int32; tok_emb : [vocab][d]; pos_emb : [seq][d] dtype;
 *   x : out [batch][n_rows][d] float.  Requires lo + n_rows <= seq;
 *   UNSUPPORTED unless d % 4 == 0 and x and the tables are 16-byte aligned.
 */
polestar_status polestar_embed(polestar_dtype dtype, int batch, int seq, int d, const int32_t* ids,
                               int lo, int n_rows, const void* tok_emb, int vocab,
                               const void* pos_emb, float* x, hipStream_t stream);

/*
 * polestar_rmsnorm -- out[b][out_start + r][:] = x[b][x_start + r][:] /
 *   sqrt(mean_c x^2 + eps), unit gain, rounded to dtype, for r < n_rows.
 *   x : [batch][x_seq][d] float;  out : [batch][out_seq][d] dtype.
 * UNSUPPORTED unless d % 4 == 0, d <= 16384 and both are 16-byte aligned.
 */
polestar_status polestar_rmsnorm(polestar_dtype dtype, int batch, int n_rows, int d, const float* x,
                                 int x_seq, int x_start, float eps, void* out, int out_seq,
                                 int out_start, hipStream_t stream);

/*
 * polestar_linear -- y[b][r][:] = W x[b][row_start + r][:] for r < n_rows,
 *   fp32 accumulation on MFMA, rounded to dtype (the GEMM of the K/V
 *   refresh, dense rows in and out).
 *   x : [batch][seq][n_in]; w : [n_out][n_in]; y : out [batch][n_rows][n_out]
 *   workspace : >= polestar_linear_workspace_size(...) bytes (no init needed)
 * UNSUPPORTED unless n_in % 128 == 0 (bf16) / % 64 (fp32), n_out % 16 == 0
 * and every pointer is 16-byte aligned.
 */
size_t polestar_linear_workspace_size(polestar_dtype dtype, int batch, int n_rows, int n_out, int n_in);
polestar_status polestar_linear(polestar_dtype dtype, int batch, int seq, int n_in, int n_out,
                                int row_start, int n_rows, const void* x, const void* w, void* y,
                                void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * polestar_swiglu -- out[r][f] = silu(gate_up[r][f]) * gate_up[r][ffn + f],
 *   silu(g) = g / (1 + e^-g), fp32, rounded to dtype.
 *   gate_up : [rows][2*ffn] dtype; out : [rows][ffn] dtype.
 * UNSUPPORTED unless ffn % 4 == 0 and both are 16-byte aligned.
 */
polestar_status polestar_swiglu(polestar_dtype dtype, long rows, int ffn, const void* gate_up,
                                void* out, hipStream_t stream);

/*
 * polestar_residual_add -- x[i] += y[i] for i < n (float += dtype).
 * UNSUPPORTED unless n % 4 == 0 and both are 16-byte aligned.
 */
polestar_status polestar_residual_add(polestar_dtype dtype, long n, float* x, const void* y,
                                      hipStream_t stream);

/*
 * polestar_copy_rows -- dst[b][p][:] = src[b][p][:] for the rows that
 *   polestar_refresh_kv rewrites: the first stale_count[b] entries of
 *   stale_idx[b] (entries outside [0, seq) are skipped) and the block
 *   [block_start, block_start + block_len).  Keeps the cached hidden states
 *   H in step with the refreshed K/V (Alg. 1, Update of the cached states).
 *   src, dst : [batch][seq][d] dtype, distinct buffers.
 * UNSUPPORTED unless a row is a whole number of 16-byte chunks.
 */
polestar_status polestar_copy_rows(polestar_dtype dtype, int batch, int seq, int d, const void* src,
                                   void* dst, const int32_t* stale_idx, const int32_t* stale_count,
                                   int k_max, int block_start, int block_len, hipStream_t stream);

/*
 * Cached hidden-state residual codec (Sec. 4.1 "Cluster and Quantize Hidden
 * States"; App. C quantization format; App. D format ablation): a window
 * row is kept as its residual to its cluster's mean, quantized along the
 * channels in an OCP microscaling format -- blocks of 32 channels share one
 * E8M0 scale 2^e (byte e + 127, e = floor(log2 amax) - emax, clamped to
 * [-127, 127]); values v / 2^e rounded to nearest even and saturated:
 *   POLESTAR_MXFP4: FP4 E2M1 (emax 2, |v| <= 6), two per byte, lower
 *                   channel in the low nibble, sign in bit 3;
 *   POLESTAR_MXFP8: FP8 E4M3 (emax 8, |v| <= 448), one per byte, sign in bit 7.
 * The residual is x - mean formed in fp32; rows whose label is -1 use a zero
 * mean.  Codes [batch][seq][polestar_codec_row_bytes(fmt, d)] and scales
 * [batch][seq][d / 32] are laid out by position (rows not encoded are left
 * as they are).  UNSUPPORTED unless d % 32 == 0 and the float arrays and
 * codes are 16-byte aligned.
 *
 * polestar_cluster_means -- means[b][k] = mean over the window positions
 *   win_idx[b][0..n_win) with labels[b][p] == k of x[b][p] (fp32, summed in
 *   window order; zeros for an empty cluster).  K <= 16, d % 4 == 0.
 * polestar_codec_encode -- codes/scales of the rows idx[b][0..count[b]) of x
 *   against means[b][labels[b][p]].
 * polestar_codec_gather -- for r < count[b], p = idx[b][r]:
 *   x_out[b][r] = means[b][labels[b][p]] + decoded residual (fp32), and if
 *   h_out != NULL, h_out[b][r] = RMSNorm(x_out[b][r]) (unit gain, eps) in
 *   dtype -- the dequantisation fused into the gather that starts a packet's
 *   forward (the paper fuses it with the update-packet computation);
 *   rows r >= count[b]: zeros.  x_out [batch][k_max][d], h_out
 *   [batch][k_max][d]; d <= 16384.
 */
typedef enum { POLESTAR_MXFP4 = 0, POLESTAR_MXFP8 = 1 } polestar_codec;

size_t polestar_codec_row_bytes(int fmt, int d);
polestar_status polestar_cluster_means(int batch, int seq, int d, const float* x, const int32_t* win_idx,
                                       int n_win, const int32_t* labels, int n_clusters, float* means,
                                       hipStream_t stream);
polestar_status polestar_codec_encode(int fmt, int batch, int seq, int d, const float* x, const int32_t* idx,
                                      const int32_t* count, int k_max, const int32_t* labels, int n_clusters,
                                      const float* means, uint8_t* codes, uint8_t* scales, hipStream_t stream);
polestar_status polestar_codec_gather(int fmt, polestar_dtype dtype, int batch, int seq, int d,
                                      const uint8_t* codes, const uint8_t* scales, const int32_t* idx,
                                      const int32_t* count, int k_max, const int32_t* labels, int n_clusters,
                                      const float* means, float eps, float* x_out, void* h_out,
                                      hipStream_t stream);

/*
 * polestar_gather_rows / polestar_scatter_rows -- move the rows an update
 * packet carries (Alg. 1: the sparse forward of the selected rows and the
 * next layer's patch) between a [batch][seq] array and a compact
 * [batch][k_max] one; rows are row_bytes bytes (any element type).
 *   gather : dst[b][r] = src[b][idx[b][r]] for r < count[b]; zero rows for
 *            r in [count[b], k_max) and for entries outside [0, seq)
 *   scatter: dst[b][idx[b][r]] = src[b][r] for r < count[b]; entries
 *            outside [0, seq) are skipped (distinct entries expected)
 *   idx : [batch][k_max] int32, count : [batch] int32 (clamped to [0, k_max])
 * UNSUPPORTED unless row_bytes % 16 == 0 and src, dst are 16-byte aligned.
 */
polestar_status polestar_gather_rows(int batch, int seq, int row_bytes, const void* src,
                                     const int32_t* idx, const int32_t* count, int k_max, void* dst,
                                     hipStream_t stream);
polestar_status polestar_scatter_rows(int batch, int seq, int row_bytes, const void* src,
                                      const int32_t* idx, const int32_t* count, int k_max, void* dst,
                                      hipStream_t stream);

/*
 * polestar_step -- one whole layer step: polestar_drift, polestar_select,
 * polestar_refresh_kv, polestar_project_q, polestar_attend (queries from q)
 * and polestar_commit (with the drift branch on), with exactly their
 * definitions and results, on one stream.
 *
 * Work that does not depend on the previous launch shares launches: the
 * drift beside the vocabulary scan, the per-sequence select beside the Q
 * projection, the refresh's split-K reduction beside the Q projection's (or,
 * for a refresh large enough to run unsplit on the tile GEMM, the Q
 * projection's reduction inside the refresh launch), and the attention's
 * split merge beside the commit's finalize step, so the latency-bound pieces
 * overlap bandwidth-bound ones.  With seq > 2048, or a Q projection that is
 * neither one row tile of up to 64 rows nor two of 128 whose workgroups and
 * select's overflow one round of the 256 compute units by at most 16, select
 * and the Q projection run as launches of their own and the rest stays
 * fused; shapes outside the other fused kernels (block_len > 256, d above
 * the drift kernel's rows) run the six calls one after another.  The results
 * are the same on every path.
 *
 * All fields of polestar_step_args keep the meaning, layout and
 * requirements they have in the stand-alone calls above; eligible may be
 * NULL, lse may be NULL, h may be 0 (hist, hist_len then unused), scale <= 0
 * selects 1/sqrt(head_dim), k = 0 refreshes the active block only.
 *   workspace : >= polestar_step_workspace_size(args) bytes, no initialisation
 *   refresh_begin, refresh_end : optional events (NULL: none) recorded on the
 *       stream right before and right after the refresh launches, so that a
 *       caller can time the K/V refresh inside the step (on the fused path
 *       these launches also reduce the Q projection's partials when its plan
 *       splits K).  Events created with hipEventDisableSystemFence time the
 *       launches without the cache write-back a default event performs.
 * Returns the first non-OK status of the pieces; as with the stand-alone
 * calls, argument errors are found on the host before anything is enqueued
 * (for the fused path: every check of every piece).
 */
typedef struct polestar_step_args {
    polestar_dtype dtype;
    int batch, seq, d;
    int n_heads, n_kv_heads, head_dim;
    int block_start, block_len;
    int vocab;
    int k;               /* stale rows per sequence */
    int h;               /* drift history depth */
    int mask_token_id;
    int force_one;
    float tau_s, alpha, scale;
    const void* h_cur;   /* [batch][seq][d] */
    const void* h_prev;  /* [batch][seq][d] */
    const uint8_t* eligible;   /* [batch][seq] or NULL */
    const void* w_q;     /* [n_heads*head_dim][d] */
    const void* w_k;     /* [n_kv_heads*head_dim][d] */
    const void* w_v;     /* [n_kv_heads*head_dim][d] */
    void* k_cache;       /* [batch][seq][n_kv_heads][head_dim], in/out */
    void* v_cache;       /* [batch][seq][n_kv_heads][head_dim], in/out */
    const void* logits;  /* [batch][block_len][vocab] */
    const uint8_t* masked;     /* [batch][block_len] */
    float* hist;         /* [batch][h][block_len], in/out */
    int32_t* hist_len;   /* [batch], in/out */
    float* drift;        /* out [batch][seq] */
    int32_t* stale_idx;  /* out [batch][k] */
    int32_t* stale_count;     /* out [batch] */
    void* q;             /* out [batch][block_len][n_heads][head_dim] */
    void* out;           /* out [batch][block_len][n_heads][head_dim] */
    float* lse;          /* out [batch][n_heads][block_len] or NULL */
    int32_t* token;      /* out [batch][block_len] */
    float* conf;         /* out [batch][block_len] */
    uint8_t* commit;     /* out [batch][block_len] */
} polestar_step_args;

size_t polestar_step_workspace_size(const polestar_step_args* args);
polestar_status polestar_step(const polestar_step_args* args, void* workspace,
                              size_t workspace_bytes, hipEvent_t refresh_begin,
                              hipEvent_t refresh_end, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* POLESTAR_H */
