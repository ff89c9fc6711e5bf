/*
 * libsaki: score-aware low-rank key indexing (SAKI) on MI355X (gfx950).
 *
 * C ABI of the retrieval-index path.  For each attention head the paper
 * (Sec. 5-6, Eq. 2-4, Proposition 1) builds the optimal rank-r score map
 *     M_r = Sigma_q^{-1/2} C_r Sigma_k^{-1/2},   C = Sigma_q^{1/2} Sigma_k^{1/2},
 * stores every cached key as an r-dimensional code c_j = B_k^T (k_j - mu) and
 * scores a query q against it as (B_q^T q)^T c_j + q^T mu.  The library
 * provides the four stages of that path:
 *
 *   saki_calibrate     host, float64: moments -> clamped roots -> SVD -> B_q, B_k
 *   saki_build_index   GPU: key codes for every query head (GQA aware)
 *   saki_score_topk    GPU: query sketch, sketch scores, top-k per (query, head)
 *   saki_recall        GPU: exact float64 q.k top-k and its overlap with a
 *                      candidate top-k (recall of the true top-k, Sec. 3)
 *
 * Conventions shared by every entry point
 *   - Return value: SAKI_OK (0) or a negative saki_status; nothing throws.
 *   - Arrays are dense, row-major, and owned by the caller.  "device" means
 *     memory the GPU can read (hipMalloc / torch CUDA tensors), "host" means
 *     ordinary CPU memory.  The library never allocates device memory: GPU
 *     scratch comes in through a workspace pointer sized by the matching
 *     *_workspace_bytes helper.
 *   - GPU entry points enqueue work on `stream` (a hipStream_t passed as a
 *     plain pointer; NULL = the default stream) and return without waiting.
 *     The return value reports argument validation and launch errors only;
 *     the results are ready after the caller synchronises the stream.
 *   - Heads: H_q query heads share H_kv KV heads; query head h reads KV head
 *     g(h) = h / (H_q / H_kv) (grouped-query attention, Sec. 3).
 *   - Sizes: d = 128 on the GPU path; r in {16, 32, 64, 128}; 1 <= k <= 64;
 *     0 <= N_valid <= N_cap < 2^31.  Inputs must be finite.
 *   - Ranking: top-k lists are sorted by score descending, ties broken by the
 *     lower key index.  Rows with fewer than k candidates are padded with
 *     index -1 and score -INFINITY.
 *   - Shared state: a process-wide cache of kernel occupancies and a host
 *     worker pool (both behind mutexes), and the static scratch array of
 *     saki_score_topk_noalloc.  Every other call works only on the caller's
 *     buffers, so calls on different streams may run concurrently.
 */
#ifndef SAKI_H
#define SAKI_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SAKI_OK = 0,
  SAKI_ERR_ARG = -1,         /* null pointer, negative or inconsistent size */
  SAKI_ERR_UNSUPPORTED = -2, /* valid but unsupported (d, r, k, dtype) */
  SAKI_ERR_WORKSPACE = -3,   /* workspace / index buffer smaller than required */
  SAKI_ERR_NOMEM = -4,       /* host allocation failed or size overflows */
  SAKI_ERR_HIP = -5,         /* a HIP runtime call or kernel launch failed */
  SAKI_ERR_NUMERIC = -6      /* eigensolver did not converge / non-finite input */
} saki_status;

/* Storage type of keys (SAKI_F32, SAKI_BF16) and of key sketches (codes: all
 * three).  SAKI_FP8 is the OCP fp8 E4M3 format (bias 7, 3 mantissa bits,
 * subnormals, no infinities, largest finite value 448); quantisation
 * composes with the codes (Sec. 2), halving the bytes of a bf16 index. */
enum { SAKI_F32 = 0, SAKI_BF16 = 1, SAKI_FP8 = 2 };

/* Rank-r map used by saki_calibrate. */
enum {
  SAKI_METHOD_OPT = 0,     /* the paper's optimum M_r (Eq. 3-4), one map per query head */
  SAKI_METHOD_KEY_PCA = 1, /* baseline: P = V V^T, top-r eigenvectors of Sigma_k */
  SAKI_METHOD_SHARED = 2,  /* one map per KV group: M_r of the pooled query moment */
  SAKI_METHOD_SAP_MAP = 3, /* variant (Sec. 6): orthogonal projector on range(M_r) */
  SAKI_METHOD_SAP_SVD = 4  /* variant (Sec. 6): orthogonal projector on span(V_r) */
};

/* Human-readable description of a status code (static storage). */
const char* saki_status_string(int status);

/* ABI version of this header: 2. */
int saki_version(void);

/*
 * saki_calibrate (host) -- Sec. 6 with Eq. 2-4 and Appendix A.
 *
 * Per KV head g: mu_g = mean of k_cal[g], Sigma_k = (1/T) sum (k - mu)(k - mu)^T.
 * Per query head h: Sigma_q = (1/T) sum q q^T (uncentred).  Each moment's
 * eigenvalues below floor_rel * lambda_max are clamped to that floor (a moment
 * with lambda_max <= 0 is replaced by the identity).  C = Sigma_q^{1/2}
 * Sigma_k^{1/2} with symmetric roots; C = U diag(sigma) V^T with sigma
 * descending.  Outputs
 *     B_q = Sigma_q^{-1/2} U_r diag(sigma_r)^{1/2},
 *     B_k = Sigma_k^{-1/2} V_r diag(sigma_r)^{1/2},
 * each pair (u_i, v_i) signed so that the largest-magnitude entry of column i
 * of B_k is positive (the lowest index on ties).  The factors do not depend
 * on which square root of the moments is used: when both moments are safely
 * above the floor the library takes the Cholesky route (M = L_k^T Sigma_q L_k
 * with Sigma_k = L_k L_k^T, whose eigenvectors give the same B_q, B_k).
 * With SAKI_METHOD_SHARED the query heads of a KV group share one map (an
 * extension for GQA indexes; the paper calibrates each head alone): the
 * group's summed objective of Eq. 2 is linear in Sigma_q, so the optimum is
 * Eq. 3-4 with the pooled moment (1/G) sum_h Sigma_q^(h).  Every head of the
 * group receives the same B_q, B_k, sigma and n_clamped; an index built with
 * one code set per KV head (saki_build_index with H_q = H_kv and the group's
 * B_k) then serves all of them (index_heads = H_kv in saki_score_topk).
 * With SAKI_METHOD_KEY_PCA instead B_q = B_k = the top-r eigenvectors of
 * Sigma_k (each column's largest-magnitude entry positive), sigma = eigenvalues
 * of Sigma_k, descending.
 * The span variants of Sec. 6 give B_q = B_k = Q, an orthonormal basis of an
 * orthogonal projector P = Q Q^T, with sigma and n_clamped as for the
 * optimum: SAKI_METHOD_SAP_SVD takes Q = V_r, the top-r right singular
 * vectors of C (symmetric clamped roots); SAKI_METHOD_SAP_MAP takes the
 * Sigma_k^{1/2}-weighted span {Sigma_k^{1/2} v_i} (the range of M_r),
 * orthonormalised by Gram-Schmidt in the order of the singular values.  Each
 * column of Q is signed so that its largest-magnitude entry is positive;
 * scores depend only on P.
 *
 *   q_cal      host float [H_q, T, d]   calibration queries (pre-RoPE)
 *   k_cal      host float [H_kv, T, d]  calibration keys of the same tokens
 *   floor_rel  eigenvalue floor relative to lambda_max; the paper uses 1e-6
 *   B_q, B_k   host float [H_q, d, r]   out
 *   mu         host float [H_kv, d]     out
 *   sigma      host double [H_q, d]     out, singular values of C (or NULL)
 *   n_clamped  host int [H_q, 2]        out, clamped eigenvalues of
 *                                       (Sigma_q, Sigma_k) (or NULL)
 *   n_threads  host threads to use; 0 = min(hardware threads, 16)
 * Any d in [1, 4096] is accepted here (the GPU path needs d = 128); 1 <= r <= d.
 */
int saki_calibrate(const float* q_cal, const float* k_cal, int H_q, int H_kv,
                   int T, int d, int r, int method, double floor_rel,
                   float* B_q, float* B_k, float* mu, double* sigma,
                   int* n_clamped, int n_threads);

/*
 * saki_calibration_moments (GPU) -- the moments saki_calibrate starts from
 * (Sec. 6, Appendix A), in float64 on the GPU: Sigma_q of every query head
 * (uncentred), the mean mu and the centred Sigma_k of every KV head, all with
 * the 1/T normaliser.  Products of the float32 tokens are exact in float64;
 * only the summation order differs from the host.
 *
 *   q_cal    device float [H_q, T, d];  k_cal  device float [H_kv, T, d]
 *   Sigma_q  device double [H_q, d, d] out (full symmetric matrices)
 *   Sigma_k  device double [H_kv, d, d] out;  key_mean  device double [H_kv, d] out
 * Any d in [1, 4096] and T >= 1.
 */
int saki_calibration_moments(const float* q_cal, const float* k_cal, int H_q, int H_kv,
                             int T, int d, double* Sigma_q, double* Sigma_k,
                             double* key_mean, void* stream);

/*
 * saki_calibrate_from_moments (host) -- saki_calibrate after its moments:
 * the same factors from Sigma_q [H_q, d, d], Sigma_k [H_kv, d, d] and
 * key_mean [H_kv, d] (host float64, e.g. copied back from
 * saki_calibration_moments).  Arguments and outputs as for saki_calibrate.
 */
int saki_calibrate_from_moments(const double* Sigma_q, const double* Sigma_k,
                                const double* key_mean, int H_q, int H_kv, int d, int r,
                                int method, double floor_rel, float* B_q, float* B_k,
                                float* mu, double* sigma, int* n_clamped, int n_threads);

/*
 * saki_weight_svd_factors (host) -- the weight-SVD baseline of Table 1, read
 * as a data-blind truncation of the key projection: B_q = B_k = the top-r left
 * singular vectors of W_K^(g) (eigenvectors of W_K W_K^T), signed as above.
 *   W_K   host double [H_kv, d, D]
 *   B_q, B_k  host float [H_q, d, r] out (query head h gets its group's basis)
 */
int saki_weight_svd_factors(const double* W_K, int H_q, int H_kv, int d, int D,
                            int r, float* B_q, float* B_k);

/*
 * saki_sym_eig (host) -- the float64 symmetric eigensolver the calibration
 * uses (Householder tridiagonalisation + implicit QL).  A is n x n row-major
 * and symmetric; w receives the eigenvalues ascending and V (n x n row-major)
 * the eigenvectors as columns.  A is not modified.
 */
int saki_sym_eig(int n, const double* A, double* w, double* V);

/*
 * Size in bytes of the key-code index for B sequences x H_q query heads x
 * N_cap keys at rank r, stored as sketch_dtype.  The layout is private to the
 * library (use saki_index_export to read it).  0 on invalid arguments.
 */
size_t saki_index_bytes(int B, int H_q, int N_cap, int r, int sketch_dtype);

/*
 * saki_build_index (GPU) -- key codes c_j = B_k^(h)T (k_j - mu_g(h)) (Eq. 4)
 * for every query head h, keys j in [n_begin, n_begin + n_count).  Codes are
 * computed to float32 accuracy: k - mu in float32, every product formed from
 * three bf16 terms of each operand (what is left out is below
 * 4 * 2^-24 |k_e - mu_e| |B_k[e][m]|) and accumulated in float32.  They are
 * stored as sketch_dtype (bf16: round to nearest even; fp8: round to the
 * nearest E4M3 value, ties to the even code, magnitudes above 448 saturating
 * to 448).  Codes outside the range are left
 * untouched, so (0, N) builds the whole index and (n, 1) appends one decoded
 * token.
 *
 *   keys    device [B, H_kv, N_cap, d], key_dtype SAKI_F32 or SAKI_BF16
 *   B_k     device float [H_q, d, r];  mu  device float [H_kv, d]
 *   index   device buffer of index_bytes >= saki_index_bytes(B, H_q, N_cap, r, sketch_dtype)
 */
int saki_build_index(const void* keys, int key_dtype, int B, int H_q, int H_kv,
                     int N_cap, int d, int r, const float* B_k, const float* mu,
                     int sketch_dtype, void* index, size_t index_bytes,
                     int n_begin, int n_count, void* stream);

/*
 * saki_index_export (GPU) -- debug read-back of the codes as float
 * [B, H_q, N_cap, r] (device).  Codes never written read as whatever the
 * index buffer held.
 */
int saki_index_export(const void* index, int sketch_dtype, int B, int H_q,
                      int N_cap, int r, float* out, void* stream);

/* Workspace for saki_score_topk with these sizes (bytes; 0 on bad arguments):
 * the partial lists of a split key axis and, for Q >= 16 with N_valid below
 * 16,384 (the two-pass kernel), the query sketches z (r bf16 values per row,
 * r floats for float32 codes) and b (one float per row) of all B * H_q * Q
 * rows, formed by one kernel before the scoring kernel reads them. */
size_t saki_score_topk_workspace_bytes(int B, int H_q, int index_heads, int Q, int N_valid,
                                       int r, int k, int sketch_dtype);

/*
 * saki_score_topk (GPU) -- Sec. 6: z_i = B_q^T q_i and b_i = q_i^T mu (float32;
 * z rounded to bf16 when sketch_dtype is bf16 or fp8), scores
 * s_ij = z_i . c_j + b_i with exact products accumulated in float32, and the top-k keys per (sequence, head, query).
 * Query row i sees keys j < N_valid, and with q_pos also only j <= q_pos[i]
 * (causal, inclusive).
 *
 *   index_heads  code sets per sequence in the index: H_q (one per query
 *              head, the paper's index) or H_kv (a GQA-shared index, built by
 *              saki_build_index with H_q = H_kv from SAKI_METHOD_SHARED
 *              factors); query head h reads code set h / (H_q / index_heads).
 *              With a shared index, decode-style calls (Q < 16) score all
 *              query heads of a group in one pass over its codes.
 *   index      device, built by saki_build_index with B, index_heads, N_cap, r, dtype
 *   q          device float [B, H_q, Q, d]
 *   q_pos      device int [Q] (shared by all sequences and heads), or NULL = no mask
 *   B_q        device float [H_q, d, r];  mu  device float [H_kv, d]
 *   top_idx    device int [B, H_q, Q, k] out
 *   top_score  device float [B, H_q, Q, k] out, or NULL
 *   ws         device workspace of ws_bytes >= saki_score_topk_workspace_bytes(...)
 */
int saki_score_topk(const void* index, int sketch_dtype, int B, int H_q, int H_kv,
                    int index_heads, int N_cap, int N_valid, int d, int r, const float* q,
                    const int* q_pos, int Q, const float* B_q, const float* mu,
                    int k, int* top_idx, float* top_score, void* ws,
                    size_t ws_bytes, void* stream);

/*
 * saki_score_topk_noalloc (GPU) -- for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, kernels and results as saki_score_topk,
 * without the workspace: the split-key partial lists, chunk gates, redo
 * flags and query sketches live in a static device array of saki_noalloc_scratch_bytes()
 * (32 MiB) that each GPU the library runs on holds until the process ends.
 * Nothing is allocated.  Returns SAKI_ERR_WORKSPACE when the call needs
 * more (saki_score_topk_workspace_bytes(...) > saki_noalloc_scratch_bytes()),
 * SAKI_ERR_HIP when the array's device address cannot be obtained.  Every
 * call on a GPU uses that GPU's one array: calls that overlap in time on the
 * same GPU (different streams, or host threads) race and must be serialised
 * by the caller.  The array keeps the last call's contents; each call writes
 * every entry it reads before reading it.
 */
int saki_score_topk_noalloc(const void* index, int sketch_dtype, int B, int H_q, int H_kv,
                            int index_heads, int N_cap, int N_valid, int d, int r,
                            const float* q, const int* q_pos, int Q, const float* B_q,
                            const float* mu, int k, int* top_idx, float* top_score,
                            void* stream);

/* Bytes of the static scratch array behind saki_score_topk_noalloc. */
size_t saki_noalloc_scratch_bytes(void);

/* Workspace for saki_recall with these sizes (bytes; 0 on bad arguments). */
size_t saki_recall_workspace_bytes(int B, int H_q, int H_kv, int Q, int N_valid, int d, int k);

/*
 * saki_recall (GPU) -- evaluation of Sec. 3: exact scores q_i . k_j in float64
 * (float32 inputs, so every product is exact), the exact top-k T_i per row
 * under the same candidate rule as saki_score_topk, and
 * hits_i = |S_i intersect T_i| with S_i = approx_idx row i (entries < 0 ignored).
 * Recall of a head is sum(hits) / (k * rows).
 *
 *   keys        device [B, H_kv, N_cap, d] (key_dtype);  q  device float [B, H_q, Q, d]
 *   approx_idx  device int [B, H_q, Q, k]
 *   hits        device int [B, H_q, Q] out
 *   exact_idx   device int [B, H_q, Q, k] out, or NULL
 */
int saki_recall(const void* keys, int key_dtype, const float* q, const int* q_pos,
                int B, int H_q, int H_kv, int N_cap, int N_valid, int Q, int d,
                int k, const int* approx_idx, int* hits, int* exact_idx,
                void* ws, size_t ws_bytes, void* stream);

/* Where saki_attend takes the selected keys from. */
enum {
  SAKI_KEYS_EXACT = 0,         /* the key cache (exact keys fetched for the winners) */
  SAKI_KEYS_RECONSTRUCTED = 1  /* mu + B_q c_j from the index codes (Sec. 6) */
};

/*
 * saki_attend (GPU) -- reading the index's winners (Sec. 1: the index
 * nominates candidates and only they are read; Sec. 3 and 6: codes are
 * pre-RoPE, the rotation is applied after reconstruction).  For every
 * (sequence, head, query) row, attention over the keys listed in top_idx,
 * in RoPE space:
 *   s_j = rope(q_i, pos_i) . rope(key_j, j) / sqrt(d),  p = softmax(s),
 *   out_i = sum_j p_j v_j,
 * where key_j is the cached key (SAKI_KEYS_EXACT) or its reconstruction
 * k_hat_j = mu + M_r (k_j - mu) = mu + B_q c_j from the index codes
 * (SAKI_KEYS_RECONSTRUCTED).  rope rotates the pairs (x_m, x_{m+d/2}),
 * m < d/2, by pos * rope_theta^(-2m/d); key j sits at position j, query i at
 * q_pos[i], or at N_valid - 1 when q_pos is NULL (a decode query attends as
 * the newest token).  Entries of top_idx < 0 are skipped; a row with none
 * writes zeros.  Scores and the softmax are float32; the rotation angles are
 * reduced in float64.
 *
 *   keys     device [B, H_kv, N_cap, d] key_dtype (read for SAKI_KEYS_EXACT, else may be NULL)
 *   values   device float [B, H_kv, N_cap, d]
 *   index    device index of saki_build_index (read for SAKI_KEYS_RECONSTRUCTED,
 *            else may be NULL), sketch_dtype and index_heads as for saki_score_topk
 *   q        device float [B, H_q, Q, d] (pre-RoPE);  q_pos device int [Q] or NULL
 *   B_q      device float [H_q, d, r];  mu device float [H_kv, d] (reconstruction)
 *   top_idx  device int [B, H_q, Q, k], k <= 64, entries < N_valid
 *   out      device float [B, H_q, Q, d]
 * d must be 128.  Errors: SAKI_ERR_ARG on bad sizes or pointers,
 * SAKI_ERR_UNSUPPORTED on unsupported d, r, k or dtypes.
 */
int saki_attend(const void* keys, int key_dtype, const float* values, const void* index,
                int sketch_dtype, int key_source, int B, int H_q, int H_kv, int index_heads,
                int N_cap, int N_valid, int d, int r, const float* q, const int* q_pos, int Q,
                const float* B_q, const float* mu, const int* top_idx, int k,
                float rope_theta, float* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SAKI_H */
