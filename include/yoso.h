/*
 * yoso.h -- C ABI of the MI355X (gfx950) YOSO-attention library (libyoso.so).
 *
 * YOSO attention (You Only Sample (Almost) Once, arXiv 2111.09714) replaces the
 * softmax matrix by Bernoulli variables B_ij = [f(q_i) == f(k_j)] realised by
 * one locality-sensitive hash f per sample (Sec. 3.1, eq. yoso-formulation),
 * and averages m such samples.  With unit-length rows Q, K (Remark 1; the
 * experiments l2-normalise them, Sec. 4) and values V:
 *
 *   Y  = (1/m) sum_h B_h(Q,K) V                                   (Sec. 3.1-3.2)
 *   dV = (1/m) sum_h B_h^T dY                                     (eq. gradient-v)
 *   dQ = tau/(2m) sum_h [(dY V^T) .* B_h] K                      (eq. pseudo-gradient-q)
 *   dK = tau/(2m) sum_h [(dY V^T) .* B_h]^T Q                    (the symmetric form)
 *
 * Conventions shared by every call:
 *   - Every tensor pointer is a DEVICE pointer owned by the caller; the library
 *     allocates nothing and keeps no state between calls (beyond the opt-in
 *     timing pool below).
 *   - Tensors are dense row-major: x[bh][i][l] with bh = batch*heads flattened,
 *     i the row (token) and l < d the feature.  Hash codes are codes[bh][i][h]:
 *     the m codes of a row are contiguous.
 *   - All device pointers must be 16-byte aligned.
 *   - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL is the
 *     default stream).  Outputs are overwritten, never accumulated into.
 *   - Every argument check happens on the host before any HIP call, so a bad
 *     call returns an error without touching the device.  A HIP launch error is
 *     returned as YOSO_ERR_DEVICE; yoso_last_error() then holds its text.
 *   - Limits: d == 64; 1 <= tau <= 12; 1 <= m <= 64; m*tau <= 512;
 *     0 <= n <= 65536 per tensor; bh >= 0.  Zero-sized tensors are valid.
 *     tau stops at 12 because the tables live in LDS: one hash's 2^tau buckets
 *     for two feature dims take 2^tau x 8 bytes, 32 KiB at tau = 12, and the
 *     bucket sort keeps 2^tau counters and 64-bit lane masks per wave; with at
 *     most 65536 rows, tau > 12 would leave almost every bucket with 0 or 1 key.
 *   - Inputs must be finite.  The hash scales each row of x by a power of two
 *     before staging it through fp16 pairs, so rows may have any finite
 *     magnitude; R is staged unscaled, so |R| must stay below 65504 (entries
 *     below about 2^-3 keep their value to 2^-24 absolute).  The backward and
 *     YOSO-E scale every operand by a power of two before it is split into
 *     fp16 (hi, lo) pairs (per head and tensor, per row, or per 64-row tile),
 *     so V, dY, Q, K may have any magnitude between about 2^-40 and 2^40;
 *     values more than about 2^20 below the largest of their head (backward)
 *     or tile (YOSO-E) keep less than 22 significant bits.
 *   - Precision.  Y and dV are accumulated as exact fixed-point integers: each
 *     value of feature dim d is rounded to a multiple of 2^-k_d, where 2^k_d is
 *     the largest power of two keeping 2^k_d (1 + 2^-10) times a bound on every
 *     bucket sum of |value| of that dim below 2^30: the dim's sum of |value|
 *     over the n_src source rows, or, for fp32 outputs with n_src > 8192, the
 *     smaller of that sum and the largest bucket's row count times the dim's
 *     largest |value|; everything after that rounding is exact.  dQ and dK use fp32 accumulation of products formed
 *     from fp16 (hi, lo) pairs (about 22 significant bits; bf16 inputs are
 *     exact as the hi halves alone wherever they lie within 2^27 of their head's
 *     largest value); the contribution of each hash to a row is kept in 24-bit
 *     fixed point (one power-of-two exponent per row, exact to 2^-22 of that
 *     row's largest value; 16-bit, exact to 2^-15, for bf16 outputs, whose own
 *     rounding is 2^-9, four values of each row keeping 14 bits, 2^-13, beside
 *     the row's exponent), and the m contributions are summed in hash order in
 *     fp32.
 *   - Reproducibility.  Every accumulation order is fixed (integer tables, a
 *     stable bucket order, partial rows summed in hash order), so repeating a
 *     call on the same inputs gives bitwise identical outputs on any stream.
 */
#ifndef YOSO_H
#define YOSO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    YOSO_OK = 0,
    YOSO_ERR_NULL = 1,      /* a required pointer is NULL (and its tensor is not empty) */
    YOSO_ERR_SHAPE = 2,     /* bh < 0, n out of [0, 65536], d != 64, or bh*n too large */
    YOSO_ERR_TAU = 3,       /* tau, m or m*tau out of range */
    YOSO_ERR_DTYPE = 4,     /* unknown yoso_dtype */
    YOSO_ERR_ALIGN = 5,     /* a device pointer is not 16-byte aligned */
    YOSO_ERR_WORKSPACE = 6, /* workspace NULL or smaller than yoso_workspace_bytes() */
    YOSO_ERR_DEVICE = 7,    /* a HIP call failed; see yoso_last_error() */
    YOSO_ERR_OP = 8         /* unknown yoso_op */
} yoso_status;

/* Storage type of Q, K, V, dY and of the outputs Y, dQ, dK, dV.  Arithmetic is
 * fp32 (or exact integer) either way; bf16 outputs are rounded to nearest even
 * once at the end. */
typedef enum { YOSO_F32 = 0, YOSO_BF16 = 1 } yoso_dtype;

typedef enum {
    YOSO_OP_HASH = 0,
    YOSO_OP_FORWARD = 1,
    YOSO_OP_BACKWARD = 2,
    YOSO_OP_BACKWARD_STAR = 3
} yoso_op;

/*
 * Sign-random-projection hash (Sec. 3.2 overview; Fig. 2 caption: tau
 * concatenated hyperplane hashes, collision probability (1 - theta/pi)^tau).
 *
 *   codes[b][i][h] = sum_{t<tau} [ x[b][i] . R[:, h*tau + t] > 0 ] << t
 *
 * x      [bh][n][d]  rows to hash (fp32 or bf16 per dtype); Q and K are hashed
 *                    with the same R so that B_ij = [codes_q == codes_k].
 * R      [d][m*tau]  fp32 hyperplanes, column h*tau+t = hyperplane t of hash h.
 * codes  [bh][n][m]  uint16 output, low tau bits used (consumers read only the
 *                    low tau bits of the codes they are given).
 * The sign test is strict (a zero projection gives bit 0).  Bits whose
 * projection lies within about 2^-20 |x[b][i]| |R[:, c]| of zero (~1e-5 for a
 * unit row and Gaussian hyperplanes) may differ from an exact-arithmetic
 * evaluation; everywhere else the code is exact.
 */
yoso_status yoso_hash(const void *x, yoso_dtype dtype, int64_t bh, int64_t n, int32_t d,
                      const float *R, int32_t m, int32_t tau, uint16_t *codes, void *stream);

/*
 * Hyperplanes of the fast hash (Sec. 3.2, "Speed-up": the approximate random
 * projection of Andoni et al. 2015).  Rotation r = 0 .. ceil(m*tau/64) - 1 is the
 * pseudo-random rotation
 *
 *   M_r = (1/64) H D3 H D2 H D1,   H the 64 x 64 Walsh-Hadamard matrix (Sylvester
 *                                  order), D_i = diag(+-1) from signs[r][i-1],
 *
 * and column c = 64 r + l of R (c < m*tau) is row l of M_r:  R[j][c] = M_r[l][j].
 * yoso_hash(x, ..., R, m, tau, codes) with this R is the fast hash: bit t of hash
 * h is [ (M_r x)_l > 0 ] with h*tau + t = 64 r + l.  Expand once, then hash Q and
 * K with the same R.
 *
 * signs  [ceil(m*tau/64)][3] uint64 (device): bit l of signs[r][i] set means
 *        D_{i+1} of rotation r negates coordinate l.  The caller draws them
 *        (uniform random bits); they are the hash function.
 * R      [64][m*tau] fp32 (device), every entry written.  Each row of M_r has
 *        length 8 (= sqrt(64), the mean length of a Gaussian column); entries are
 *        multiples of 1/64 and come out exact.
 * d must be 64; m, tau as for yoso_hash.  One small kernel on `stream`.
 */
yoso_status yoso_fast_hyperplanes(const uint64_t *signs, int32_t d, int32_t m, int32_t tau, float *R,
                                  void *stream);

/*
 * The fast hash itself (Sec. 3.2, "Speed-up"; Andoni et al. 2015): the rotations
 * of yoso_fast_hyperplanes applied to each row by fast Walsh-Hadamard transforms,
 * O(m tau log2 d) additions per row instead of a dense projection.
 *
 *   codes[b][i][h] = sum_{t<tau} [ (H D3 H D2 H D1 x[b][i])_l > 0 ] << t,
 *                    rotation r and coordinate l given by h*tau + t = 64 r + l.
 *
 * x      [bh][n][d]  rows to hash (fp32 or bf16 per dtype), d = 64.
 * signs  [ceil(m*tau/64)][3] uint64 (device), as for yoso_fast_hyperplanes.
 * codes  [bh][n][m]  uint16 output, the same layout and sign convention as
 *                    yoso_hash (strict test; bit for bit equal to yoso_hash with
 *                    the R of yoso_fast_hyperplanes except for projections within
 *                    about 1e-6 |x| of zero).
 * Arithmetic is fp32 (each butterfly an exact +-1 fused multiply-add).
 */
yoso_status yoso_fast_hash(const void *x, yoso_dtype dtype, int64_t bh, int64_t n, int32_t d,
                           const uint64_t *signs, int32_t m, int32_t tau, uint16_t *codes, void *stream);

/*
 * Forward (Sec. 3.2 overview: per hash, a table of 2^tau buckets holding the sum
 * of V over the keys hashed to each bucket; each query reads the bucket of its
 * own code; Sec. 3.1: the m samples are averaged).
 *
 *   y[b][i] = (1/m) sum_h sum_{j : kcodes[b][j][h] == qcodes[b][i][h]} v[b][j]
 *
 * qcodes [bh][n_q][m], kcodes [bh][n_k][m]  from yoso_hash with the same R.
 * v      [bh][n_k][d],  y [bh][n_q][d]  (dtype).  Queries whose buckets are empty
 * get 0 (no renormalisation).
 * Many heads of short sequences (both sides at most 1024 rows, enough heads to
 * fill the GPU) take the same sum as y = (1/m) C v, C[i][j] the number of hashes
 * under which query i and key j collide, counted pair by pair from the codes; the
 * result differs from the tables' only in the rounding of the additions.
 * workspace: yoso_workspace_bytes(YOSO_OP_FORWARD, ...) bytes (0 for that form
 * and for every shape whose tables fit in one LDS pass; then workspace may be
 * NULL).
 */
yoso_status yoso_forward(const uint16_t *qcodes, const uint16_t *kcodes, const void *v,
                         yoso_dtype dtype, int64_t bh, int64_t n_q, int64_t n_k, int32_t d,
                         int32_t m, int32_t tau, void *y, void *workspace, size_t workspace_bytes,
                         void *stream);

/*
 * Backward of the forward above, reusing its codes (Sec. 3.3):
 *   dv = (1/m) sum_h B_h^T dy                          eq. (gradient-v), sampled form
 *   dq = tau/(2m) sum_h [(dy v^T) .* B_h] k           eq. (pseudo-gradient-q), sampled
 *   dk = tau/(2m) sum_h [(dy v^T) .* B_h]^T q         symmetric counterpart for K
 * with B_h(i,j) = [qcodes[b][i][h] == kcodes[b][j][h]].  dq, dk use the paper's
 * lower-bound surrogate (tau/2) p of the collision-probability derivative.
 *
 * q, dy, dq [bh][n_q][d];  k, v, dk, dv [bh][n_k][d]  (dtype).
 * workspace: yoso_workspace_bytes(YOSO_OP_BACKWARD, ...) bytes of scratch: the
 * per-hash bucket orders, the per-head maxima of |q|, |k|, |v|, |dy|, fp16
 * (hi, lo) copies of q, k, v, dy, and one 24-bit (bf16: 16-bit) fixed-point
 * partial row per (row, hash) for dq and dk, the codes transposed to [bh][m][n]
 * for the bucket sort, one exponent byte per row of dy and v: about
 * (3*m*d + 7*m + 8*d + 1) * (n_q + n_k) * bh bytes
 * (bf16: (2*m*d + 6*m + 8*d + 1) * (n_q + n_k) * bh).
 * A bucket with b_q queries and b_k keys whose sizes pass
 * yoso_backward_table_threshold() is summed in the table form of Sec. 3.3
 * restricted to that bucket (one d x d matrix per side and bucket, applied to the
 * bucket's rows); the others pair by pair.  Both give the same sums up to the
 * order of fp32 additions.
 */
yoso_status yoso_backward(const uint16_t *qcodes, const uint16_t *kcodes, const void *q,
                          const void *k, const void *v, const void *dy, yoso_dtype dtype,
                          int64_t bh, int64_t n_q, int64_t n_k, int32_t d, int32_t m, int32_t tau,
                          void *dq, void *dk, void *dv, void *workspace, size_t workspace_bytes,
                          void *stream);

/*
 * *YOSO (Sec. 3.3, eq. gradient-q; the *YOSO rows of Sec. 4): a sampled estimate
 * of the TRUE gradient of the expected attention for Q and K, on the same codes.
 * eq. gradient-q weighs the pair (i, j) by tau (1 - theta/pi)^(tau-1) /
 * (pi sqrt(1 - x^2)), x = q_i . k_j; (1 - theta/pi)^(tau-1) is the collision
 * probability of tau-1 hyperplane bits, so per hash
 *
 *   C_h(i, j) = #{ t < tau : codes of q_i, k_j agree on every bit except t }
 *             = tau [codes equal] + [codes differ in exactly one bit]
 *
 * has expectation tau (1 - theta/pi)^(tau-1), and
 *
 *   dq = (1/m) sum_h [(dy v^T) .* C_h ./ (pi sqrt(max(1 - (q k^T)^2, 1/64)))] k
 *   dk = (1/m) sum_h [(dy v^T) .* C_h ./ (pi sqrt(max(1 - (q k^T)^2, 1/64)))]^T q
 *   dv = (1/m) sum_h B_h^T dy                    (eq. gradient-v, as yoso_backward)
 *
 * is unbiased for eq. gradient-q wherever 1 - x^2 >= 1/64.  The true gradient
 * diverges as the alignment x approaches 1; the bound 1/64 caps the weight at
 * 8/pi (|x| > 0.99216).  x is the dot product of the rows as given, taken as
 * unit length (Remark 1).  Arguments, layouts and errors as for yoso_backward;
 * workspace: yoso_workspace_bytes(YOSO_OP_BACKWARD_STAR, ...) bytes, about
 * (3*m*tau*d + 9*m*tau + 8*d) * (n_q + n_k) * bh (the pairs of m*tau derived
 * (tau-1)-bit hashes, one 24-bit partial row per row and derived hash); m*tau is
 * also the limit on bh that yoso_backward puts on m.  Its pair pass does about
 * tau + 1 times the work of yoso_backward's (pairs one bit apart count too).
 */
yoso_status yoso_backward_star(const uint16_t *qcodes, const uint16_t *kcodes, const void *q, const void *k,
                               const void *v, const void *dy, yoso_dtype dtype, int64_t bh, int64_t n_q,
                               int64_t n_k, int32_t d, int32_t m, int32_t tau, void *dq, void *dk,
                               void *dv, void *workspace, size_t workspace_bytes, void *stream);

/*
 * yoso_backward without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation).  Same arguments, results and errors as yoso_backward;
 * its scratch is a fixed array inside the library, one per GPU, reserved when the
 * library is loaded and held until the process ends (its size:
 * yoso_backward_noalloc_limit(), 64 MiB; one head of 4096 queries and keys at
 * m = 32, tau = 8 needs about 56 MB).  Shapes whose backward needs more than
 * that return YOSO_ERR_WORKSPACE before anything is launched.  The call makes
 * no allocation; the first call on a device looks up that device's copy of the
 * array (the stream must belong to the current device, else YOSO_ERR_DEVICE).
 * Every call on one GPU uses the same array: calls that overlap in time on one
 * GPU (other streams, other threads) race and must be serialised by the caller.
 * Nothing in the array needs to start at zero (every byte read is first written
 * by the same call).
 */
yoso_status yoso_backward_noalloc(const uint16_t *qcodes, const uint16_t *kcodes, const void *q,
                                  const void *k, const void *v, const void *dy, yoso_dtype dtype,
                                  int64_t bh, int64_t n_q, int64_t n_k, int32_t d, int32_t m, int32_t tau,
                                  void *dq, void *dk, void *dv, void *stream);

/* Bytes of the fixed scratch array of yoso_backward_noalloc (per GPU). */
size_t yoso_backward_noalloc_limit(void);

/* T of yoso_backward's switch-over rule: a bucket takes the table form when
 * b_q * b_k > T * (b_q + b_k).  Informational (for work accounting by callers). */
int32_t yoso_backward_table_threshold(void);

/*
 * Row l2 normalisation: the output normalisation of N-YOSO (Sec. 3.1,
 * "Normalizing Attention", eq. normalized-yoso: N-YOSO(Q, K, V) = l2(B(Q, K) V))
 * and the normalisation of Q and K before hashing that the experiments use
 * (Sec. 4, opening paragraph; Remark 1 assumes unit-length rows).
 *
 *   y[r] = x[r] / ||x[r]||_2        (y[r] = 0 where x[r] is the zero row)
 *
 * x, y [rows][d] (dtype), any number of rows (bh*n for Q, K or Y); y may be x.
 * Arithmetic is fp32 (sum of squares, correctly rounded sqrt and division).
 * Errors as for the calls above (YOSO_ERR_SHAPE for d != 64 or rows < 0).
 */
yoso_status yoso_l2_normalize(const void *x, yoso_dtype dtype, int64_t rows, int32_t d, void *y,
                              void *stream);

/*
 * Backward of yoso_l2_normalize (the Jacobian of x -> x/||x|| applied to dy):
 *
 *   dx[r] = (dy[r] - y[r] (y[r] . dy[r])) / ||x[r]||,   y[r] = x[r] / ||x[r]||
 *   (dx[r] = 0 where x[r] is the zero row)
 *
 * x is the forward's INPUT (the norm and y are recomputed from it); dy, dx
 * [rows][d] (dtype).  dx may be dy; it must not be x.  Chaining it after
 * yoso_backward gives the gradients of the normalised-input, normalised-output
 * attention: dq = l2 backward(q, dq_hat), dk likewise, with yoso_backward run on
 * the normalised q, k and on dy_hat = l2 backward(y_raw, dy).
 */
yoso_status yoso_l2_normalize_backward(const void *x, const void *dy, yoso_dtype dtype, int64_t rows,
                                       int32_t d, void *dx, void *stream);

/*
 * YOSO-E: the exact expectation of the forward and of the sampled surrogate
 * backward over the hash functions, i.e. YOSO with infinitely many hashes (Sec. 4,
 * "YOSO-E"; the collision probability of eq. yoso-expectation and the Fig. 2
 * caption):
 *
 *   P[i][j] = (1 - arccos(q_i . k_j / (||q_i|| ||k_j||)) / pi)^tau
 *   y  = P v
 *   dv = P^T dy,  dq = (tau/2) [(dy v^T) .* P] k,  dk = (tau/2) [(dy v^T) .* P]^T q
 *
 * q, dy, y, dq [bh][n_q][d];  k, v, dk, dv [bh][n_k][d]  (dtype).  O(n_q n_k d)
 * work per head, no workspace.  Rows of q and k must be nonzero; |entries| of
 * q, k, v, dy below 4096.  Arithmetic: fp32 accumulation of products of fp16
 * (hi, lo) pairs (three products per step, about 22 significant bits) and an
 * fp32 arccos.
 */
yoso_status yoso_expectation_forward(const void *q, const void *k, const void *v, yoso_dtype dtype,
                                     int64_t bh, int64_t n_q, int64_t n_k, int32_t d, int32_t tau,
                                     void *y, void *stream);

yoso_status yoso_expectation_backward(const void *q, const void *k, const void *v, const void *dy,
                                      yoso_dtype dtype, int64_t bh, int64_t n_q, int64_t n_k, int32_t d,
                                      int32_t tau, void *dq, void *dk, void *dv, void *stream);

/* Bytes of device workspace that `op` (a yoso_op) needs for these arguments.
 * The arguments are validated exactly as the call itself validates them; on an
 * invalid argument the result is SIZE_MAX and yoso_last_error() says why. */
size_t yoso_workspace_bytes(int op, int64_t bh, int64_t n_q, int64_t n_k, int32_t d, int32_t m,
                            int32_t tau, yoso_dtype dtype);

/* Static description of a status code. */
const char *yoso_status_str(yoso_status status);

/* Detail of the last failing call on this thread ("" if none). */
const char *yoso_last_error(void);

/*
 * Kernel timing (a benchmarking aid, off by default).
 * yoso_timing_enable(capacity > 0) makes every later kernel launch of the
 * library record a pair of HIP events around itself on its launch stream, for
 * up to `capacity` launches per kernel name (events are created on a kernel's
 * first launch and live until the next yoso_timing_enable call; 0 disables and
 * frees them).  yoso_timing_reset() forgets the launches recorded so far.
 * yoso_timing_query() waits for the recorded events of `kernel` ("hash_kernel",
 * "fast_hash_kernel", "fast_hyperplanes_kernel", "table_kernel", "sort_kernel", "split_kernel", "pass_kernel", "reduce_kernel",
 * "zero_kernel", "l2norm_kernel", "l2norm_bwd_kernel", "expect_fwd_kernel",
 * "expect_bwd_kv_kernel", "expect_bwd_q_kernel")
 * and returns the summed duration and the launch count.
 * Not thread-safe with respect to concurrent launches on other threads' streams
 * beyond the pool bookkeeping, which is locked.
 */
yoso_status yoso_timing_enable(int32_t capacity);
yoso_status yoso_timing_reset(void);
yoso_status yoso_timing_query(const char *kernel, double *total_ms, int64_t *launches);

#ifdef __cplusplus
}
#endif

#endif /* YOSO_H */
