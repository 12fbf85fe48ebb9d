/*
 * crvq.h -- C ABI of libcrvq, the MI355X (gfx950) hot path of CRVQ,
 * "Channel-Relaxed Vector Quantization for Extreme Compression of LLMs"
 * (arXiv 2412.09282).
 *
 * Conventions shared by every call
 * --------------------------------
 * - Array arguments are DEVICE pointers owned by the caller.  The library
 *   never allocates, frees or retains them after the call returns.  Arrays of
 *   pointers (books, codes of several codebooks) are HOST arrays whose
 *   entries are device pointers.
 * - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *   Work is enqueued on it asynchronously; the call returns after enqueue.
 * - All arguments are validated on the host before anything is enqueued.  On
 *   a validation error nothing runs, outputs are untouched and a nonzero
 *   crvq_status is returned; crvq_last_error() gives the reason (thread-local
 *   text).  No exception crosses the ABI and the library never aborts.
 *   Launch failures return CRVQ_ERR_HIP.
 * - Device-resident indices (codes, perm, initial-codeword indices) cannot be
 *   checked on the host; every kernel bounds-checks them and treats an
 *   out-of-range entry as documented per call (it never reads out of bounds).
 * - Scratch memory comes from a caller-supplied `workspace` of at least the
 *   size the matching *_workspace_size() function returns (256-byte aligned).
 * - Layouts are row-major.  A codebook is K x d elements.  Codes are int32.
 * - A "vector set" is the paper's sub-vector partition (Sec. 3.1 Eq. 1): a
 *   matrix of n_rows rows is cut into vecs_per_row contiguous d-vectors per
 *   row; vector v = r * vecs_per_row + g starts at element r * ld + g * d of
 *   `X`.  The critical slab of a reordered matrix (its first n_crit columns,
 *   Sec. 4.3) is the vector set with vecs_per_row = n_crit / d, ld = N.
 * - Element types: CRVQ_F32 (float) and CRVQ_BF16 (bfloat16, stored as
 *   uint16 bit patterns).  Floating-point inputs must be finite.
 * - Results are deterministic: no floating-point atomics are used anywhere,
 *   so equal inputs give bitwise-equal outputs.
 */
#ifndef CRVQ_H
#define CRVQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CRVQ_OK = 0,
  CRVQ_ERR_INVALID = 1,     /* a NULL required pointer or an out-of-range size / option */
  CRVQ_ERR_UNSUPPORTED = 2, /* a valid request outside what the library implements */
  CRVQ_ERR_WORKSPACE = 3,   /* workspace missing or smaller than the *_workspace_size() result */
  CRVQ_ERR_HIP = 4          /* the HIP runtime reported an error while enqueueing */
} crvq_status;

/* CRVQ_F64 is accepted only where a call says so (the fp64 operands of the
 * refinement calls and the fp64 output of crvq_dequant / crvq_dequant_books). */
typedef enum { CRVQ_F32 = 0, CRVQ_BF16 = 1, CRVQ_F64 = 2 } crvq_dtype;
typedef enum { CRVQ_REDUCE_SUM = 0, CRVQ_REDUCE_MAX = 1 } crvq_reduce;

#define CRVQ_MAX_K 65536   /* codewords per codebook (e <= 16 bits) */
#define CRVQ_MAX_D 16      /* sub-vector length */
#define CRVQ_MAX_BEAM 16   /* residual beam width (each lane group keeps its top-B list in registers) */
#define CRVQ_MAX_BOOKS 8   /* basic + extended codebooks */

/* Library version (major * 10000 + minor * 100 + patch). */
int crvq_version(void);

/* Text describing the last error returned on the calling thread ("" if none). */
const char* crvq_last_error(void);

/* ---------------------------------------------------------------------------
 * crvq_channel_importance -- column (input-channel) reduction.
 *
 *   out[j] = s_j * R_{i < M} (A[i*lda + j] - B[i*ldb + j])^2,   j < N
 *
 * R = sum (CRVQ_REDUCE_SUM, accumulated in fp64) or max (CRVQ_REDUCE_MAX,
 * exact); B may be NULL (treated as 0); scale may be NULL (s_j = 1).
 * The paper's channel-importance metrics are modes of this one reduction:
 *  - Hessian diagonal h_j = [X X^T]_jj (Appendix A.2 Eq. 9): A = the
 *    calibration activations stored tokens x N, B = NULL, scale = NULL, SUM.
 *  - W-only importance I_j = max_i w_ij^2 (Sec. 4.1): A = W, MAX.
 *  - W-A importance (Sec. 4.1 Eq. 7 / Appendix A.2 Eq. 10): A = W,
 *    B = the prequantized W, MAX, scale = h/2 (Eq. 10) or 1/(2[H^-1]_jj) (Eq. 7).
 *  - Energy-weighted importance I_j = h_j * sum_i w_ij^2: A = W, SUM, scale = h.
 * A, B: M x N matrices of `dtype` with leading dimensions lda, ldb >= N.
 * scale: float[N] or NULL.  out: float[N] (fp32, rounded once from fp64).
 * workspace: crvq_importance_workspace_size(M, N) bytes.
 */
size_t crvq_importance_workspace_size(int64_t M, int64_t N);
crvq_status crvq_channel_importance(const void* A, int64_t lda, const void* B, int64_t ldb, int dtype,
                                    int64_t M, int64_t N, const float* scale, int reduce, float* out,
                                    void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * crvq_reorder -- channel reordering (Sec. 4.2, Alg. 1 ReorderChannels) and
 * its reverse (Sec. 4.3 / Fig. 3 right).
 *
 * If importance != NULL, first writes perm[N]: the channels in descending
 * importance, equal importance in ascending channel index, NaN last (a
 * stable descending sort).  Otherwise perm is an input and must hold a
 * permutation of 0..N-1.
 * Then forward (inverse == 0):  out[r*ld_out + k]       = in[r*ld_in + perm[k]]
 *      inverse (inverse != 0):  out[r*ld_out + perm[k]] = in[r*ld_in + k]
 * for r < M, k < N.  in and out are M x N of `dtype`, must not overlap.
 * in may be NULL (then only perm is computed; M is ignored).  An
 * out-of-range perm entry leaves the affected output elements unwritten.
 * workspace: crvq_reorder_workspace_size(N) bytes, needed when importance != NULL or
 * inverse != 0.  N <= 2^20.
 */
size_t crvq_reorder_workspace_size(int64_t N);
crvq_status crvq_reorder(const void* in, int64_t ld_in, void* out, int64_t ld_out, int dtype, int64_t M,
                         int64_t N, const float* importance, int32_t* perm, int inverse, void* workspace,
                         size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * crvq_assign -- nearest-codeword encoding (Sec. 3.1 Eq. 3-4; Alg. 1
 * VectorQuant):  codes[v] = argmin_k ||x_v - C_k||_2, v < n_rows*vecs_per_row.
 *
 * Exact: the chosen k minimises the fp64 squared distance
 * sum_t (x_vt - C_kt)^2 (t ascending); among equal distances the lowest k
 * wins.  dist[v] (optional) = that fp64 distance rounded to float.
 * X: vector set (see conventions) of x_dtype, d <= 16.
 * C: K x d codebook of c_dtype, 1 <= K <= 65536.
 * codes: int32[n]; dist: float[n] or NULL.
 * workspace: crvq_assign_workspace_size(n, d, K) bytes.
 */
size_t crvq_assign_workspace_size(int64_t n_vectors, int32_t d, int64_t K);
crvq_status crvq_assign(const void* X, int x_dtype, int64_t n_rows, int64_t vecs_per_row, int64_t ld,
                        int32_t d, const void* C, int c_dtype, int64_t K, int32_t* codes, float* dist,
                        void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * crvq_assign_noalloc -- crvq_assign for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same arguments and results without a workspace.  Its
 * scratch is a fixed array of CRVQ_NOALLOC_SCRATCH_BYTES inside the library's
 * device memory, one per GPU, held until the process ends; the call allocates
 * nothing.  A request whose crvq_assign_workspace_size(n, d, K) exceeds that
 * size returns CRVQ_ERR_UNSUPPORTED before anything is enqueued (128 MiB holds
 * about 2.5 million vectors against 65536 codewords, 4.8 million against 256).  Every call on a GPU
 * shares that GPU's array: calls that overlap on one GPU (on different
 * streams or from different threads) race and must be ordered by the caller;
 * calls on one stream are ordered already.  The array's contents left by one
 * call are never read by the next (every counter is reset by the call).
 */
#define CRVQ_NOALLOC_SCRATCH_BYTES (128LL << 20)
crvq_status crvq_assign_noalloc(const void* X, int x_dtype, int64_t n_rows, int64_t vecs_per_row, int64_t ld,
                                int32_t d, const void* C, int c_dtype, int64_t K, int32_t* codes, float* dist,
                                void* stream);

/* ---------------------------------------------------------------------------
 * crvq_assign_residual_beam -- joint code choice over additive codebooks by
 * beam search (Sec. 3.1 last paragraph; Sec. 4.3; Alg. 1 BeamSearchOptimize),
 * under the squared Euclidean error of the residual.
 *
 * books[0] is the basic codebook, books[1..n_books-1] the extended ones, in
 * the order they were fitted.  For each vector, starting from one empty
 * tuple with residual x: for book t, every kept tuple (rank p, residual r)
 * is extended by every codeword c of book t; a candidate's key is
 * (sum_j (r_j - c_j)^2 in fp64, p, codeword index), the `beam` smallest keys
 * survive in key order, and a survivor's residual is r - c (fp64).  The
 * answer is the rank-0 tuple after the last book.  beam = 1 is the greedy
 * additive fit of Alg. 1's extended-codebook loop.
 * X: vector set of x_dtype.  books: host array of n_books device pointers,
 * book t is Ks[t] x d of book_dtypes[t].  codes: host array of n_books
 * device pointers; the code of vector v = r * vecs_per_row + g for book t is
 * written to codes[t][r * ldc[t] + g] (ldc = NULL means ldc[t] = vecs_per_row;
 * otherwise ldc[t] >= vecs_per_row, so the basic codes of a critical slab can
 * land directly in the full matrix's code array).  err: float[n] (final
 * squared error, vector order) or NULL.
 * 1 <= beam <= 16, 1 <= n_books <= 8.
 * workspace: crvq_beam_workspace_size(n, d, n_books, Ks, beam) bytes.
 */
size_t crvq_beam_workspace_size(int64_t n_vectors, int32_t d, int32_t n_books, const int64_t* Ks, int32_t beam);
crvq_status crvq_assign_residual_beam(const void* X, int x_dtype, int64_t n_rows, int64_t vecs_per_row,
                                      int64_t ld, int32_t d, int32_t n_books, const void* const* books,
                                      const int32_t* book_dtypes, const int64_t* Ks, int32_t beam,
                                      int32_t* const* codes, const int64_t* ldc, float* err, void* workspace,
                                      size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * crvq_kmeans_update -- one Lloyd update of a K-means codebook (Sec. 3.1
 * Eq. 2; Alg. 1 KMeansCodebook):
 *
 *   C[k] := mean{ x_v : codes[v] == k }  (fp64 sums, rounded to c_dtype
 *   round-to-nearest-even); a codeword with no members is left unchanged.
 *
 * Atomic-free and deterministic: codes are stably counting-sorted, every
 * centroid is a fixed-order fp64 reduction over its segment.  Codes outside
 * [0, K) belong to no cluster.  counts: int32[K] member counts, or NULL.
 * workspace: crvq_kmeans_workspace_size(n, d, K) bytes.
 */
size_t crvq_kmeans_workspace_size(int64_t n_vectors, int32_t d, int64_t K);
crvq_status crvq_kmeans_update(const void* X, int x_dtype, int64_t n_rows, int64_t vecs_per_row, int64_t ld,
                               int32_t d, const int32_t* codes, int64_t K, void* C, int c_dtype,
                               int32_t* counts, void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * crvq_gather_vectors -- out[k] = x_{idx[k]} for k < count (the K-means
 * initial codewords drawn from the vector set, Alg. 1 KMeansCodebook).
 * idx: int64[count] device array; an index outside [0, n) yields a NaN row.
 * out: count x d of out_dtype (same as x_dtype, or F32 from BF16 widening).
 */
crvq_status crvq_gather_vectors(const void* X, int x_dtype, int64_t n_rows, int64_t vecs_per_row, int64_t ld,
                                int32_t d, const int64_t* idx, int64_t count, void* out, int out_dtype,
                                void* stream);

/* ---------------------------------------------------------------------------
 * crvq_dequant -- additive reconstruction, the ComputeError / Update steps of
 * Alg. 1, and the reverse reordering at inference (Sec. 4.3, Fig. 3 right).
 *
 * For an M x n_cols matrix in reordered channel order, vector (r, g), g <
 * n_cols/d, is rebuilt as
 *   R[r, g*d+t] = C_base[q_base[r*ldq_base+g]][t]
 *                 + sum_{e < n_ext, g < n_crit/d} C_ext[e][q_ext[e][r*ldq_ext+g]][t]
 * summed in fp64 in book order.  Then
 *   minuend != NULL (residual mode):  out[r*ld_out + c] = minuend[r*ld_min + c] - R[r, c]
 *   perm != NULL (reverse reorder):   out[r*ld_out + perm[c]] = R[r, c]
 *   otherwise:                        out[r*ld_out + c] = R[r, c]
 * each rounded once to out_dtype (CRVQ_F64 allowed when perm is NULL: the
 * residual of the refinement calls, minuend - R exact up to one fp64 rounding).
 * perm and minuend are mutually exclusive.
 * n_crit is a multiple of d, 0 <= n_crit <= n_cols.  A code outside its
 * codebook yields NaN for that vector.
 * workspace: crvq_dequant_workspace_size(n_cols) bytes (only used with perm).
 */
size_t crvq_dequant_workspace_size(int64_t n_cols);
crvq_status crvq_dequant(int64_t M, int64_t n_cols, int32_t d, int64_t n_crit, const int32_t* q_base,
                         int64_t ldq_base, const void* C_base, int base_dtype, int64_t K_base, int32_t n_ext,
                         const int32_t* const* q_ext, int64_t ldq_ext, const void* const* C_ext,
                         const int32_t* ext_dtypes, const int64_t* K_ext, const int32_t* perm,
                         const void* minuend, int minuend_dtype, int64_t ld_min, void* out, int out_dtype,
                         int64_t ld_out, void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * crvq_dequant_books -- crvq_dequant for a layout with n_base >= 1 basic
 * codebooks (the additive basic VQ with m > 1 books of Sec. 3.2 and Sec. 6.4,
 * e.g. m = 2 books on d = 16 vectors) followed by n_ext extended books:
 *   R[r, g*d+t] = sum_{b < n_base} C[b][q[b][r*ldq_base+g]][t]
 *                 + sum_{n_base <= b < n_base+n_ext, g < n_crit/d} C[b][q[b][r*ldq_ext+g]][t]
 * summed in fp64 in book order, then written exactly as by crvq_dequant
 * (residual mode with minuend, reverse reorder with perm, else plain), each
 * element rounded once.  q, C, dtypes, Ks: host arrays of n_base + n_ext
 * entries (device pointers for q and C).  n_base + n_ext <= 8.  crvq_dequant is
 * this call with n_base = 1.  A code outside its codebook yields NaN for
 * that vector.  workspace: crvq_dequant_workspace_size(n_cols) bytes (only
 * used with perm).
 */
crvq_status crvq_dequant_books(int64_t M, int64_t n_cols, int32_t d, int64_t n_crit, int32_t n_base, int32_t n_ext,
                               const int32_t* const* q, int64_t ldq_base, int64_t ldq_ext, const void* const* C,
                               const int32_t* dtypes, const int64_t* Ks, const int32_t* perm, const void* minuend,
                               int minuend_dtype, int64_t ld_min, void* out, int out_dtype, int64_t ld_out,
                               void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * crvq_bits_per_weight -- average storage per weight of a quantized layer
 * (Sec. 3.2 Eq. 6 and Appendix A.1 Eq. 8, counted for the exact layout):
 *
 *   bits = [ sum_{b < n_base} (rows*cols/d) * e_b
 *            + sum_{n_base <= b < n_base+n_ext} (rows*n_crit/d) * e_b
 *            + sum_b Ks[b] * d * codeword_bits + cols * perm_bits ] / (rows*cols)
 *
 * with e_b = ceil(log2 Ks[b]), the code width that indexes book b (0 for a
 * one-codeword book).  The paper stores codewords in FP16 (codeword_bits =
 * 16) and the channel permutation as 16-bit indices (perm_bits = 16, or 0 to
 * leave it out as Eq. 8 does).  With n_crit = lambda*cols this is Eq. 8 with
 * all m = n_base + n_ext codebooks counted in the codebook term; with
 * n_ext = 0 and perm_bits = 0 it is Eq. 6.
 * Host-only: Ks is a host array of n_base + n_ext entries, out a host double.
 * Needs rows, cols >= 1, d in [1, 16] dividing cols, n_crit a multiple of d in
 * [0, cols], n_base >= 1, n_ext >= 0, n_base + n_ext <= 8, Ks[b] in
 * [1, 65536], codeword_bits in [1, 64], perm_bits in [0, 64].
 */
crvq_status crvq_bits_per_weight(int64_t rows, int64_t cols, int32_t d, int64_t n_crit, int32_t n_base, int32_t n_ext,
                                 const int64_t* Ks, int32_t codeword_bits, int32_t perm_bits, double* out);

/* ===========================================================================
 * Loss-driven refinement (Alg. 1: QuantLoss, FineTuneCodebook,
 * BeamSearchOptimize at width 1).  A layer is taken in reordered channel order
 * (critical channels first).  With calibration activations X stored
 * tokens x N, H = X^T X is the paper's X X^T, R = W - W_hat, and
 *   QuantLoss = ||W X^T - W_hat X^T||_F^2 = sum_r R_r H R_r^T,
 *   d QuantLoss / d W_hat = -2 R H.
 * All refinement arithmetic is fp64; codebooks being tuned are fp32.
 * ------------------------------------------------------------------------- */

/* crvq_gram -- H = X^T X (Appendix A.2: the Hessian proxy X X^T of Eq. 9-10,
 * full matrix).  X: n_rows x n_cols of x_dtype (F32 or F64), row stride ld.
 * H: n_cols x n_cols fp64, row stride ldh >= n_cols.  Products are exact in
 * fp64 for fp32 input; sums are fused multiply-adds in row order. */
crvq_status crvq_gram(const void* X, int x_dtype, int64_t n_rows, int64_t n_cols, int64_t ld, double* H, int64_t ldh,
                      void* stream);

/* crvq_hessian_inverse_diagonal -- the denominator of the W-A channel
 * importance of Sec. 4.1 Eq. 7, [(X X^T)^-1]_jj, for every channel j:
 *
 *   hinv[j]  = [(H + delta I)^-1]_jj,   delta = damp * (sum_j H_jj) / N,
 *   scale[j] = float(1 / (2 hinv[j]))   (Eq. 7's factor, rounded once),
 *
 * so that crvq_channel_importance(W, B = the prequantized W, scale, MAX)
 * gives Eq. 7's I_j.  The damping (damp >= 0; 0.01 is the usual choice)
 * makes the proxy invertible when the calibration set has fewer tokens than
 * channels or a channel is never active.  H: N x N fp64, row stride ldh >= N,
 * symmetric; only its lower triangle (j <= i) is read.  hinv: double[N] and
 * scale: float[N], device memory, either may be NULL (not both).  Computed in
 * fp64 by a blocked Cholesky factorization A = L L^T with the inverse factor
 * T = L^-1 formed alongside ([A^-1]_jj = sum_i T_ij^2); deterministic.  If
 * the damped matrix is not positive definite (a pivot <= 0, NaN or infinite),
 * every hinv[j] and scale[j] is NaN: the status does not report it, since the
 * check runs on the device.  N <= 65536.
 * workspace: crvq_hessian_inverse_workspace_size(N) bytes (about 16 N^2).
 */
size_t crvq_hessian_inverse_workspace_size(int64_t N);
crvq_status crvq_hessian_inverse_diagonal(const double* H, int64_t ldh, int64_t N, double damp, double* hinv,
                                          float* scale, void* workspace, size_t ws_bytes, void* stream);

/* crvq_hessian_product -- G = R H[:, 0:n_out] (so -2 G is the gradient of
 * QuantLoss w.r.t. W_hat on those columns) and, when row_loss != NULL (needs
 * n_out == N), row_loss[r] = sum_j R[r][j] G[r][j], the QuantLoss of row r
 * (Alg. 1 QuantLoss).  When loss_total != NULL (needs row_loss), loss_total[0]
 * = sum_r row_loss[r], the layer's QuantLoss, summed on the device in a fixed
 * order (so a caller's loop guard needs no host-side reduction).
 * R: M x N fp64 (stride ldr), H: N x N fp64 (stride ldh), G: M x n_out fp64
 * (stride ldg >= n_out); loss_total: one fp64 device value.  Deterministic. */
crvq_status crvq_hessian_product(int64_t M, int64_t N, int64_t n_out, const double* R, int64_t ldr, const double* H,
                                 int64_t ldh, double* G, int64_t ldg, double* row_loss, double* loss_total,
                                 void* stream);

/* crvq_code_sums -- sums[k] = sum of the vectors x_v with codes[v] == k, in
 * fp64, and counts[k] their number (the per-codeword gradient of
 * FineTuneCodebook when X holds -2 R H, or plain cluster sums).  X: vector set
 * (see conventions) of CRVQ_F64 elements; codes: int32[n]; codes outside
 * [0, K) belong to no code.  sums: K x d fp64; counts: int32[K] or NULL.
 * 1 <= K <= 65536.  Deterministic: every code's members are added in vector
 * order per block, the blocks in block order (K > 1024: the vectors are first
 * grouped by the high byte of their code, and a code's members are added in
 * vector order per chunk of its group, the chunks in order).
 * workspace: crvq_code_sums_workspace_size(n, d, K) bytes. */
size_t crvq_code_sums_workspace_size(int64_t n_vectors, int32_t d, int64_t K);
crvq_status crvq_code_sums(const double* X, int64_t n_rows, int64_t vecs_per_row, int64_t ld, int32_t d,
                           const int32_t* codes, int64_t K, double* sums, int32_t* counts, void* workspace,
                           size_t ws_bytes, void* stream);

/* crvq_adam_step -- one Adam step (Kingma & Ba, with bias correction; the
 * paper fine-tunes codebooks with beta1 = 0.9, beta2 = 0.95) on n fp32
 * parameters C with gradient g = grad_scale * grad (fp64):
 *   m = b1 m + (1 - b1) g,  v = b2 v + (1 - b2) g^2,
 *   C = C - lr * (m / (1 - b1^step)) / (sqrt(v / (1 - b2^step)) + eps)
 * in fp64 (each operation rounded on its own), C rounded once to fp32.
 * m, v: fp64 state of n entries (zero before step 1).  step >= 1. */
crvq_status crvq_adam_step(float* C, const double* grad, double grad_scale, double* m, double* v, int64_t n,
                           int64_t step, double lr, double beta1, double beta2, double eps, void* stream);

/* crvq_adam_step_bf16 -- the same step for a bf16 codebook C (bit patterns)
 * tuned through an fp32 master copy (n floats, state like m and v): at step 1
 * the master is first set to C (exact); the master then moves as
 * crvq_adam_step moves an fp32 codebook, and C becomes the master rounded to
 * bf16, nearest-even (Alg. 1 FineTuneCodebook, as read for bf16 layers). */
crvq_status crvq_adam_step_bf16(uint16_t* C, float* master, const double* grad, double grad_scale, double* m,
                                double* v, int64_t n, int64_t step, double lr, double beta1, double beta2, double eps,
                                void* stream);

/* crvq_refine_codes -- BeamSearchOptimize of Alg. 1 at the paper's width 1,
 * under QuantLoss, for one codebook C (K x d, F32 or BF16) covering the
 * column groups 0 .. n_cols/d - 1 of an M x N layer (n_cols = N for a basic
 * book, n_crit for an extended one).  For every group in column order and
 * every row independently, the group's code becomes the k minimising QuantLoss
 * with all other codes fixed (lowest k among equal values); the residual
 * R (M x N fp64, stride ldr, in/out) and codes (int32, row stride ldq >=
 * n_cols/d, in/out) are updated as it goes.  H: N x N fp64.  The loss change
 * of candidate k in group g is evaluated as
 *   c_k^T H_gg c_k - 2 c_k . ((R H)_g + H_gg c_cur) (minus the same at c_cur),
 * with (R H) kept current as codes move: within a block of 64 columns by
 * delta^T H[g rows, block columns] per change, and for the later columns by one
 * product (the block's deltas) x H per block.  A code outside [0, K) leaves
 * that row's group unchanged.  1 <= K <= 65536: a codebook that fits a CU's
 * LDS (K d <= 8192) is searched from LDS by each workgroup's rows, group after
 * group; a larger one one group at a time over all rows, in codebook slices
 * merged per row (the same values and choices either way).
 * workspace: crvq_refine_workspace_size(M, N, n_cols) bytes. */
size_t crvq_refine_workspace_size(int64_t M, int64_t N, int64_t n_cols);
crvq_status crvq_refine_codes(int64_t M, int64_t N, int32_t d, int64_t n_cols, double* R, int64_t ldr, const double* H,
                              int64_t ldh, const void* C, int c_dtype, int64_t K, int32_t* codes, int64_t ldq,
                              void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * crvq_dequant_gemv -- matrix-vector product with a CRVQ-quantized layer, the
 * inference step the paper times (Sec. 4.3, Fig. 3 right; Table 7):
 *
 *   y = W_hat x,   W_hat[:, perm[k]] = R[:, k]   (W_hat = R when perm is NULL),
 *   R[r, 8g+t] = C_base[q_base[r*ldq_base+g]][t]
 *                + sum_{e < n_ext, g < n_crit/8} C_ext[e][q_ext[e][r*ldq_ext+g]][t]
 *
 * for an M x N layer stored as 8-bit codes (every book has K <= 256, d = 8),
 * x of N elements (x_dtype), y of M floats.  N must be a multiple of 64;
 * q_base 8-byte aligned with ldq_base a multiple of 8 and >= N/8; n_crit a
 * multiple of 8 in [0, N].  Products are formed in fp32 (codeword elements and
 * x widened exactly; per column group an 8-term fp32 dot product), partial sums
 * in fp32 over at most 1024 columns and in fp64 across them: |y - W_hat x| is
 * within a few times 2^-24 * sum_j |W_hat_rj x_j|.  A code outside its book or
 * a perm entry outside [0, N) makes y_r NaN.  M = 0 is a no-op.  Deterministic.
 * workspace: crvq_gemv_workspace_size(M, N, K_base) bytes.
 */
size_t crvq_gemv_workspace_size(int64_t M, int64_t N, int64_t K_base);
crvq_status crvq_dequant_gemv(int64_t M, int64_t N, int64_t n_crit, const uint8_t* q_base, int64_t ldq_base,
                              const void* C_base, int base_dtype, int64_t K_base, int32_t n_ext,
                              const uint8_t* const* q_ext, int64_t ldq_ext, const void* const* C_ext,
                              const int32_t* ext_dtypes, const int64_t* K_ext, const int32_t* perm, const void* x,
                              int x_dtype, float* y, void* workspace, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * crvq_workspace_size -- one entry for every call's workspace size: the value
 * the per-call *_workspace_size function above returns for the same shape.
 * op selects the call; each op reads only the arguments listed (others are
 * ignored and may be 0 / NULL):
 *   CRVQ_OP_IMPORTANCE  M, N                         (crvq_channel_importance)
 *   CRVQ_OP_REORDER     N                            (crvq_reorder)
 *   CRVQ_OP_ASSIGN      n_vectors, d, K              (crvq_assign)
 *   CRVQ_OP_BEAM        n_vectors, d, n_books, Ks, beam  (crvq_assign_residual_beam)
 *   CRVQ_OP_KMEANS      n_vectors, d, K              (crvq_kmeans_update)
 *   CRVQ_OP_DEQUANT     N = n_cols                   (crvq_dequant, crvq_dequant_books)
 *   CRVQ_OP_CODE_SUMS   n_vectors, d, K              (crvq_code_sums)
 *   CRVQ_OP_REFINE      M, N, n_cols                 (crvq_refine_codes)
 *   CRVQ_OP_GEMV        M, N, K = K_base             (crvq_dequant_gemv)
 *   CRVQ_OP_HINV        N                            (crvq_hessian_inverse_diagonal)
 * Returns 0 for an unknown op or a shape the call rejects (and for calls that
 * need no workspace at that shape).  Ks is a host array of n_books entries.
 */
typedef enum {
  CRVQ_OP_IMPORTANCE = 0,
  CRVQ_OP_REORDER = 1,
  CRVQ_OP_ASSIGN = 2,
  CRVQ_OP_BEAM = 3,
  CRVQ_OP_KMEANS = 4,
  CRVQ_OP_DEQUANT = 5,
  CRVQ_OP_CODE_SUMS = 6,
  CRVQ_OP_REFINE = 7,
  CRVQ_OP_GEMV = 8,
  CRVQ_OP_HINV = 9
} crvq_op;
size_t crvq_workspace_size(int op, int64_t n_vectors, int64_t K, int32_t beam, int32_t n_books, int32_t d,
                           const int64_t* Ks, int64_t M, int64_t N, int64_t n_cols);

/* ---------------------------------------------------------------------------
 * crvq_pack_codes_u8 -- 8-bit storage of codes (the e = 8 code width of Sec. 3.2
 * Eq. 6 / Appendix A.1): out[i] = codes[i] & 255 for i < n.  Codes produced
 * against a book of K <= 256 codewords lie in [0, K) and are stored exactly.
 */
crvq_status crvq_pack_codes_u8(const int32_t* codes, int64_t n, uint8_t* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CRVQ_H */
