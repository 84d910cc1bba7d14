/*
 * mosaic.h -- C ABI of the MOSAIC hot path on AMD Instinct MI355X (gfx950).
 *
 * MOSAIC (arxiv 2607.29221) lets a trusted client outsource W X to an
 * untrusted accelerator by masking both operands over the ring Z_{2^32}
 * (protocol Pi_Sec-Approx-MatMul, Section 4.2) and recovering the product up
 * to a small error; a random Hadamard rotation (Section 5) keeps the
 * fixed-point error small. This library implements the data-parallel steps:
 * sampling of the mask material, the mask pass, the server's ring product,
 * unmasking, the rotation and fixed-point quantisation (also fused into one
 * client input pass), the client's products with the sparse LPN matrices,
 * and the comparison of Freivalds' integrity check.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Orientation. Matrices are row-major. Activations are tokens x features
 * (A is M x K, the transpose of the paper's X) and weights are
 * out-features x in-features (W is N x K, the paper's W). Products are
 * C = A B^T (M x N), the transpose of the paper's W X.
 *
 * Ring elements are uint32 holding residues mod 2^32; the signed value of a
 * result is the same 32 bits read as int32 (two's complement).
 *
 * Digit layout. The ring product consumes its operands as balanced base-256
 * digits: x = d_0 + 256 d_1 + 256^2 d_2 + 256^3 d_3 (mod 2^32), each d_t an
 * int8 in [-128, 127] (unique for every x). A rows x K ring matrix in digit
 * layout is an int8 array [rows][Kp/16][4][16] with Kp = 64 * ceil(K/64):
 * byte (i, g, t, b) at offset i * pitch + 64 g + 16 t + b is digit t of
 * element (i, 16 g + b); columns K .. Kp-1 hold zero digits. ``pitch`` is the
 * row pitch in bytes, a multiple of 64 and at least 4 * Kp. Blocks of
 * columns whose offsets are multiples of 64 can be placed side by side in
 * one wider digit matrix (this is how the protocol concatenates factors).
 *
 * Random streams. Mask material is drawn from Philox-4x32-10 (Salmon et al.,
 * SC'11). Stream (seed, stream, instance) has word t equal to word (t mod 4)
 * of Philox with key (seed mod 2^32, seed div 2^32) and counter
 * (b mod 2^32, b div 2^32, stream, instance), b = t div 4. A logical
 * rows x cols matrix visits its elements row-major, e = i * cols + j:
 *   UNIFORM  element e is word e (uniform over Z_{2^32});
 *   DGAUSS   element e is -B + #{k : word e >= T_k} with the thresholds of
 *            mosaic_dgauss_thresholds (discrete Gaussian of Section 4.1,
 *            truncated to [-B, B]);
 *   SPARSE   element e is word 2e+1 if the top s bits of word 2e are zero,
 *            else 0 (LPN noise of rate 2^-s, Section 3);
 *   WEIGHT   LPN noise with t entries per row (Example 4.1's
 *            parameterisation by the Hamming weight t): row i uses words
 *            2ti .. 2ti+2t-1. Starting from the identity permutation of the
 *            columns, step j (j = 0 .. t-1) swaps entries j and
 *            j + floor(u_j (cols - j) / 2^32), u_j = word 2ti + 2j; the column
 *            then at entry j holds word 2ti + 2j + 1 and every other
 *            column holds 0 (a partial Fisher-Yates shuffle: the t columns
 *            form a uniformly random subset up to the rounding of that
 *            product; a drawn value of 0 is kept, as for SPARSE);
 *   ZERO     element e is 0.
 *
 * Memory. Every pointer argument except ``mosaic_rng`` structs and the
 * threshold output of mosaic_dgauss_thresholds is a DEVICE pointer owned by
 * the caller. The library allocates nothing and keeps no state between
 * calls; calls are asynchronous on ``stream`` (a hipStream_t, NULL for the
 * default stream) and may be issued from several host threads.
 *
 * Empty matrices. A call whose output has no elements does nothing and
 * returns MOSAIC_OK; pointers of operands without elements may be NULL. A
 * product with K = 0 writes zeros.
 *
 * Errors. Arguments are validated before anything is launched; on error no
 * output is touched and a negative mosaic_status is returned. MOSAIC_ERR_HIP
 * means a launch failed; mosaic_last_error_message() describes the last
 * failure on the calling thread.
 */
#ifndef MOSAIC_H
#define MOSAIC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOSAIC_ABI_VERSION 3

typedef enum mosaic_status {
  MOSAIC_OK = 0,
  MOSAIC_ERR_INVALID_ARG = -1, /* null/misaligned pointer, bad size or pitch */
  MOSAIC_ERR_UNSUPPORTED = -2, /* valid but unsupported shape or option */
  MOSAIC_ERR_HIP = -3          /* a HIP launch failed */
} mosaic_status;

typedef enum mosaic_dist {
  MOSAIC_DIST_ZERO = 0,
  MOSAIC_DIST_UNIFORM = 1,
  MOSAIC_DIST_DGAUSS = 2,
  MOSAIC_DIST_SPARSE = 3,
  MOSAIC_DIST_WEIGHT = 4
} mosaic_dist;

typedef enum mosaic_dtype {
  MOSAIC_I8 = 0,  /* int8, sign-extended into the ring */
  MOSAIC_I16 = 1, /* int16, sign-extended */
  MOSAIC_I32 = 2, /* int32, two's complement */
  MOSAIC_U32 = 3  /* ring element */
} mosaic_dtype;

/* A random matrix drawn from a Philox stream (host struct, read at call
 * time). ``transposed`` != 0 writes logical element (j, i) of a cols x rows
 * matrix to output position (i, j): the same matrix stored transposed. */
typedef struct mosaic_rng {
  uint64_t seed;
  uint32_t stream;
  uint32_t instance;
  int32_t dist;             /* mosaic_dist */
  int32_t bound;            /* DGAUSS: support [-bound, bound], 0 <= bound <= 15 */
  double sigma;             /* DGAUSS: parameter sigma >= 0 */
  int32_t log2_inv_density; /* SPARSE: density 2^-s, 0 <= s <= 31 */
  int32_t transposed;
  int32_t row_weight;       /* WEIGHT: nonzeros per row t, 0 <= t <= cols */
} mosaic_rng;

/* ABI version (MOSAIC_ABI_VERSION of the built library). */
int32_t mosaic_abi_version(void);

/* Message for the last error on the calling thread ("" if none).
 * mosaic_last_error_string is the same function under a second name. */
const char* mosaic_last_error_message(void);
const char* mosaic_last_error_string(void);

/* Host-only. Discrete Gaussian thresholds T_0 .. T_{2B-1} (Section 4.1,
 * "Bounded protocol error": Pr[k] proportional to exp(-k^2 / (2 sigma^2)),
 * here restricted to [-B, B]): T_k = floor(2^32 F_k + 1/2), F_k the
 * probability of the values -B .. -B+k. ``out`` is a host array of 2B
 * entries. Touches no GPU. */
mosaic_status mosaic_dgauss_thresholds(double sigma, int32_t bound, uint64_t* out);

/* a1. Fill a rows x cols matrix from the stream ``rng`` (protocol box, Init W
 * step 1 and Init X step 1a: uniform L, M_i, N_i, R; discrete Gaussian E_w,
 * E_x; sparse S_i, T_i). Writes ring elements to ``out`` (leading dimension
 * ``ldo`` elements) and/or digits to ``out_dig`` (row pitch ``dig_pitch``
 * bytes); each output may be NULL but not both. WEIGHT streams need
 * transposed = 0, cols <= 8192 and 0 <= row_weight <= cols (else
 * MOSAIC_ERR_UNSUPPORTED / MOSAIC_ERR_INVALID_ARG). */
mosaic_status mosaic_sample(const mosaic_rng* rng, int64_t rows, int64_t cols,
                            uint32_t* out, int64_t ldo,
                            int8_t* out_dig, int64_t dig_pitch, void* stream);

/* a4. Mask (protocol box, online step 2: X' = X + U_x, here in the build's
 * orientation A' = A + U_a):
 *     out(i, j) = x(i, j) + u(i, j) + e(i, j)   (mod 2^32)
 * x: plaintext of type ``x_dtype`` at x[i * x_rs + j * x_cs] (element
 * strides; NULL means 0); u: ring matrix, leading dimension ``ldu`` (NULL
 * means 0); e: drawn from ``noise`` (NULL means 0), so the Init X error can be
 * generated in the same pass (any distribution but WEIGHT, whose rows are
 * drawn by mosaic_sample only). Outputs as in mosaic_sample. With x and
 * noise NULL this converts a ring matrix to digit layout. */
mosaic_status mosaic_mask(const void* x, int32_t x_dtype, int64_t x_rs, int64_t x_cs,
                          const uint32_t* u, int64_t ldu, const mosaic_rng* noise,
                          int64_t rows, int64_t cols,
                          uint32_t* out, int64_t ldo,
                          int8_t* out_dig, int64_t dig_pitch, void* stream);

/* a5. The untrusted accelerator's product (protocol box, online step 3,
 * Y' = W' X' and Q_i = (M_i ... M_1) X'; Section 6.1 emulation with 8-bit
 * limbs): C = A B^T over Z_{2^32}.
 * A: M x K digits (pitch a_pitch); B: N x K digits (pitch b_pitch);
 * C: M x N uint32, leading dimension ldc >= N. Stacking the rows of
 * M_i ... M_1 under W' in B returns [Y' | Q] from one call. Any K: inner
 * dimensions of 2^15 and more run as chunks whose partial products are
 * added into C (each chunk keeps the int32 shift-class sums exact). */
mosaic_status mosaic_masked_matmul(const int8_t* a_dig, int64_t a_pitch,
                                   const int8_t* b_dig, int64_t b_pitch,
                                   int64_t M, int64_t N, int64_t K,
                                   uint32_t* c, int64_t ldc, void* stream);

/* The same product with B given as ring words, for short A: C = A B^T over
 * Z_{2^32} (accumulate != 0: C += A B^T), A: M x K digits (a_pitch), B: N x K
 * uint32 with leading dimension ldb >= K, C: M x N (ldc >= N). This is the
 * client's side of the integrity check (Freivalds' test; Appendix
 * "Computational integrity", online step 4 of the Section 4.2 box): the
 * check vectors times the server's outputs [Y' | Q], which arrive as ring
 * words and are read once here instead of being converted to digits first.
 * Requirements: M <= 64, b 16-byte aligned and ldb a multiple of 4 (else
 * MOSAIC_ERR_UNSUPPORTED); A's digits past column K must be zero (the digit
 * layout's padding), because the words read past column K within a row are
 * whatever follows in memory. */
mosaic_status mosaic_masked_matmul_words(const int8_t* a_dig, int64_t a_pitch,
                                         const uint32_t* b, int64_t ldb,
                                         int64_t M, int64_t N, int64_t K,
                                         uint32_t* c, int64_t ldc, int32_t accumulate, void* stream);

/* a6. Unmask (protocol box, online step 5, in the build's orientation:
 * Y = Y' - K - Q_d L^T - sum_i Q_i S_{i+1}^T):
 *     y(i, j) = ym(i, j) - kc(i, j) - sum_{r < R} q(i, r) l(j, r)  (mod 2^32)
 * ym: M x N (ldy); kc: M x N (ldk, NULL means 0); q: M x R digits (q_pitch),
 * l: N x R digits (l_pitch) -- the factors concatenated along R; R may be 0
 * (then q and l are ignored). y: M x N int32 (ldo), the centred lift.
 * Optional dequantisation (Pi_Sec-Linear, online step 3, Section 5 box):
 * if y_f32 is not NULL it receives (float)y(i, j) * s_rows[i] * s_cols[j]
 * (ldf; products in that order, each rounded to fp32), plus bias[j] when
 * bias (N floats) is not NULL, added after the products in one more fp32
 * rounding; y may then be NULL. bias without y_f32 is
 * MOSAIC_ERR_INVALID_ARG. An output may coincide with ym or kc element for element (in
 * place, same leading dimension); otherwise outputs and inputs must not
 * overlap. Output memory may hold intermediate values while the call runs
 * (with at most 64 rows, an output that shares no memory with the inputs
 * accumulates the product before the final pass). */
mosaic_status mosaic_unmask(const uint32_t* ym, int64_t ldy,
                            const uint32_t* kc, int64_t ldk,
                            const int8_t* q_dig, int64_t q_pitch,
                            const int8_t* l_dig, int64_t l_pitch,
                            int64_t M, int64_t N, int64_t R,
                            int32_t* y, int64_t ldo,
                            const float* s_rows, const float* s_cols, const float* bias,
                            float* y_f32, int64_t ldf, void* stream);

/* mosaic_unmask with Q given as ring words, as the server returns it (the Q
 * columns of [Y' | Q]): q is M x R uint32 with leading dimension ldq >= R,
 * every other argument as in mosaic_unmask. Q's digit planes are formed as
 * the product reads it, so the client's pass that converts Q to digits is
 * not needed (one launch fewer per decode call). Requirements: M <= 16, q
 * 16-byte aligned and ldq a multiple of 4 (else MOSAIC_ERR_UNSUPPORTED);
 * l's digits past column R must be zero (the digit layout's padding),
 * because the words read past column R of a row of q are whatever follows
 * in memory. Results are bit-identical to mosaic_unmask with the digits of
 * the same Q. */
mosaic_status mosaic_unmask_words(const uint32_t* ym, int64_t ldy,
                                  const uint32_t* kc, int64_t ldk,
                                  const uint32_t* q, int64_t ldq,
                                  const int8_t* l_dig, int64_t l_pitch,
                                  int64_t M, int64_t N, int64_t R,
                                  int32_t* y, int64_t ldo,
                                  const float* s_rows, const float* s_cols, const float* bias,
                                  float* y_f32, int64_t ldf, void* stream);

/* Fused client input pass of Pi_Sec-Linear (Section 5 protocol box, online
 * step 1, then the mask of the Section 4.2 box, online step 2): for every row
 * of x (rows x n fp32, ldx), in one pass,
 *     y = forward rotation of mosaic_hadamard_rotate (block, signs),
 *     s = max_j |y_j| / qmax (1 for an all-zero row), q = round-half-even(y / s),
 *     A' = q + u + noise (mod 2^32), written as digits (out_dig, dig_pitch),
 * and scale[i] = s (scale is required; it also holds max |y| between the
 * call's two launches). The result is bit-identical to
 * mosaic_hadamard_rotate, mosaic_quantize_rows (int32 codes) and mosaic_mask
 * (x = the codes, u, noise) called in sequence. u (rows x n uint32, ldu) and
 * noise may be NULL. Requirements: block = 2^k with 10 <= k <= 14, n a
 * multiple of block, x and u 16-byte aligned with ldx, ldu multiples of 4,
 * noise not transposed; otherwise MOSAIC_ERR_UNSUPPORTED (the three calls
 * above remain available). */
mosaic_status mosaic_rotate_quantize_mask(const float* x, int64_t ldx, int64_t rows, int64_t n, int64_t block,
                                          const int8_t* signs, int32_t qmax, const uint32_t* u, int64_t ldu,
                                          const mosaic_rng* noise, int8_t* out_dig, int64_t dig_pitch,
                                          float* scale, void* stream);

/* Sparse LPN matrices in compressed-row form (Section 4.2 protocol box:
 * S_{i+1} and T_{i+1} are sparse, with noise rate 2^-s or with t nonzeros
 * per row as in Example 4.1; the client's products with them then cost
 * O(nonzeros) per output row, Section 4.2 cost analysis and Table
 * "lpn-tradeoff").
 *
 * The matrix is the rows x cols SPARSE or WEIGHT stream matrix of ``rng``
 * (rng->transposed 0; WEIGHT: cols <= 8192, row_weight <= 2048). Its
 * compressed rows are
 *   row_ptr[0 .. rows]     int64, row_ptr[0] = 0, row i owns
 *                          entries row_ptr[i] .. row_ptr[i+1]-1
 *                          (WEIGHT: row_ptr[i] = i t);
 *   col_idx[nnz], values[nnz]  column (int32) and ring value (uint32) of
 *                          each entry: SPARSE lists a row's nonzeros in
 *                          increasing column order, WEIGHT lists its t
 *                          entries in the order of the shuffle's steps (a
 *                          drawn value may be 0).
 * mosaic_sparse_csr_count writes row_ptr (rows + 1 entries); the caller
 * then sizes col_idx / values to at least row_ptr[rows] entries (reading it
 * back, or using the bound rows * cols) and calls mosaic_sparse_csr_fill. */
mosaic_status mosaic_sparse_csr_count(const mosaic_rng* rng, int64_t rows, int64_t cols, int64_t* row_ptr,
                                      void* stream);
mosaic_status mosaic_sparse_csr_fill(const mosaic_rng* rng, int64_t rows, int64_t cols, const int64_t* row_ptr,
                                     int32_t* col_idx, uint32_t* values, void* stream);

/* Products with a compressed-row sparse matrix P (rows of P given by
 * row_ptr / col_idx / values as above), over Z_{2^32}; ``subtract`` selects
 * c -= ... instead of c += ....
 *
 * mosaic_sparse_gather_rows: c(i, k) +-= sum_j P(i, j) d(j, k) for
 *   0 <= i < rows, 0 <= k < ncols: P is rows x r, d is a dense r x ncols
 *   uint32 matrix (ldd), c is rows x ncols (ldc). Used for T_{i+1} terms of
 *   U_x and K (Init X) and for S_{i+1} (M_i ... M_1) in U_w (Init W).
 * mosaic_sparse_gather_cols: c(m, n) +-= sum_j d(m, j) P(n, j) for
 *   0 <= m < M, 0 <= n < N: P is N x r, d is a dense M x r uint32 matrix
 *   (ldd), c is M x N (ldc). Used for the S_{i+1} Q_i terms of unmasking.
 *   When y_f32 is not NULL the finished c is also dequantised as in
 *   mosaic_unmask (Pi_Sec-Linear, online step 3): y_f32(m, n) =
 *   (float)c(m, n) * s_rows[m] * s_cols[n] (+ bias[n]), leading dimension
 *   ldf >= N; the last gather of a sparse unmasking then writes the
 *   floating-point output with no further pass. s_rows, s_cols, bias and
 *   ldf are ignored when y_f32 is NULL (bias without y_f32 is
 *   MOSAIC_ERR_INVALID_ARG).
 * c must not overlap d or the sparse arrays, y_f32 none of them. */
mosaic_status mosaic_sparse_gather_rows(int64_t rows, const int64_t* row_ptr, const int32_t* col_idx,
                                        const uint32_t* values, const uint32_t* d, int64_t ldd, int64_t ncols,
                                        uint32_t* c, int64_t ldc, int32_t subtract, void* stream);
/* mosaic_sparse_stream_gather_rows: as mosaic_sparse_gather_rows with P the
 *   rows x rcols SPARSE or WEIGHT stream matrix of ``rng`` itself (same
 *   validity rules as mosaic_sparse_csr_count): each row's nonzeros are
 *   drawn inside the call, so no compressed form is stored (T_{i+1} of
 *   Init X, drawn afresh for every call). */
mosaic_status mosaic_sparse_stream_gather_rows(const mosaic_rng* rng, int64_t rows, int64_t rcols, const uint32_t* d,
                                               int64_t ldd, int64_t ncols, uint32_t* c, int64_t ldc,
                                               int32_t subtract, void* stream);
mosaic_status mosaic_sparse_gather_cols(int64_t M, int64_t N, const int64_t* row_ptr, const int32_t* col_idx,
                                        const uint32_t* values, const uint32_t* d, int64_t ldd, uint32_t* c,
                                        int64_t ldc, int32_t subtract, const float* s_rows, const float* s_cols,
                                        const float* bias, float* y_f32, int64_t ldf, void* stream);

/* Integrity check (Freivalds' test; Appendix "Computational integrity" and
 * online step 4 of the Section 4.2 protocol box): the client compares two
 * short products that agree whenever the server's product was computed
 * honestly. This call counts the entries where two uint32 matrices differ:
 *     *count = #{(i, j) : a(i, j) != b(i, j)},  0 <= i < rows, 0 <= j < cols
 * a and b are device matrices with leading dimensions lda, ldb >= cols;
 * ``count`` is a device int64 written by the call (0 for an empty matrix):
 * a first launch clears it, a second adds the workgroups' partial counts to
 * it atomically, so two calls that share ``count`` on different streams
 * race. Fails with MOSAIC_ERR_INVALID_ARG for NULL pointers or leading
 * dimensions < cols. */
mosaic_status mosaic_count_mismatches(const uint32_t* a, int64_t lda, const uint32_t* b, int64_t ldb,
                                      int64_t rows, int64_t cols, int64_t* count, void* stream);

/* The whole integrity check of one call (online step 4 of the Section 4.2
 * protocol box; Appendix "Computational integrity"): with t check vectors,
 *     d = c^T A'^T - V [Y' | Q]^T   (t x M, over Z_{2^32}),
 *     *count = #{(j, i) : d(j, i) != 0},
 * where c^T (t x K, digit layout ct_dig / ct_pitch) is the client's key,
 * A' (M x K, a_dig / a_pitch) the masked activations the server received,
 * V = [a_W | a_Q] (t x NR, v_dig / v_pitch) the check vectors laid out like
 * the columns of [Y' | Q], and [Y' | Q] (M x NR uint32 ring words, leading
 * dimension ldyq) the server's output. count = 0 accepts the call; an
 * output the server changed by delta in column k is caught by the vectors
 * j with V(j, k) delta != 0. d (leading dimension ldd >= M) and count are
 * written by the call; d tells which tokens failed which vectors.
 * Constraints: 0 <= t <= 64; yq 16-byte aligned and ldyq a multiple of 4
 * (else MOSAIC_ERR_UNSUPPORTED), ldyq >= NR; digit pitches as for
 * mosaic_masked_matmul; row pitches at most 8 MiB. Columns of [Y' | Q]
 * past NR up to the next multiple of 64 are read (within each row's ldyq
 * words, and up to the 16-byte boundary past the last row's NR-th word)
 * and cancelled by V's zero padding digits. Four launches on the stream:
 * clear d and count, d += c^T A'^T, d -= V [Y' | Q]^T, count. */
mosaic_status mosaic_integrity_check(const int8_t* ct_dig, int64_t ct_pitch, const int8_t* a_dig, int64_t a_pitch,
                                     const int8_t* v_dig, int64_t v_pitch, const uint32_t* yq, int64_t ldyq,
                                     int64_t t, int64_t M, int64_t K, int64_t NR, uint32_t* d, int64_t ldd,
                                     int64_t* count, void* stream);

/* a1 (signs). Random sign vector of the rotation (Section 5: d drawn
 * uniformly from {+1, -1}^n): out[j] = +1 if bit 31 of word j of the stream
 * (rng->seed, rng->stream, rng->instance) is 0, else -1. ``out`` is a device
 * int8 array of n entries. rng->dist and rng->transposed are ignored. */
mosaic_status mosaic_sample_signs(const mosaic_rng* rng, int64_t n, int8_t* out, void* stream);

/* a7. Random Hadamard rotation (Section 5, R = H D, applied with Fino's fast
 * transform). Per row v of x (rows x n, leading dimension ldx):
 *     forward:  y = H_b (d * v) / sqrt(b)     inverse: y = d * (H_b v) / sqrt(b)
 * blockwise on consecutive blocks of length b = ``block`` (b a power of two,
 * 16 <= b <= 32768, n a multiple of b; b = n is the plain rotation). H_b is
 * the Sylvester-ordered Walsh-Hadamard matrix, H[i][j] = (-1)^popcount(i&j),
 * so the inverse undoes the forward rotation. ``signs`` is a device int8
 * vector of n entries +-1 (NULL means d = 1). y may equal x (in place, then
 * ldy == ldx); otherwise the two must not overlap. x, y 16-byte aligned,
 * ldx and ldy multiples of 4. fp32 throughout. */
mosaic_status mosaic_hadamard_rotate(const float* x, int64_t ldx, float* y, int64_t ldy,
                                     int64_t rows, int64_t n, int64_t block,
                                     const int8_t* signs, int32_t inverse, void* stream);

/* a7, for n = 28 b (e.g. 28672 = 28 x 1024): rotation by H_28 (x) H_b, which
 * mixes every entry of a row (Section 5's rotation for a length that is not
 * a power of two; the block-diagonal form above mixes only within blocks).
 * Entry i b + j of a row v is entry j of block i:
 *     forward:  y = (H_28 (x) H_b) (d * v) / sqrt(n)
 *     inverse:  y = d * ((H_28^T (x) H_b) v) / sqrt(n)   (undoes forward)
 * H_b is Sylvester-ordered as above; H_28 is Paley's first construction over
 * GF(27) = GF(3)[t]/(t^3 + 2t + 1): H = I + S, S = [[0, 1^T], [-1, Q]],
 * Q[i][k] = chi(e_i - e_k) with chi the quadratic character and e_i the
 * element whose coefficients of 1, t, t^2 are the base-3 digits of i
 * (H H^T = 28 I). b must be 256, 512 or 1024 (else MOSAIC_ERR_UNSUPPORTED).
 * signs: n entries +-1 or NULL. Pointers, alignment, leading dimensions and
 * in-place use as for mosaic_hadamard_rotate. fp32 throughout. */
mosaic_status mosaic_hadamard28_rotate(const float* x, int64_t ldx, float* y, int64_t ldy,
                                       int64_t rows, int64_t n,
                                       const int8_t* signs, int32_t inverse, void* stream);

/* a8. Per-row fixed-point quantisation (Pi_Sec-Linear, Init W step 2 and
 * online step 1): s_i = max_j |x(i, j)| / qmax (1 for an all-zero row),
 * q(i, j) = round-half-even(x(i, j) / s_i), both in fp32 arithmetic.
 * Writes q as int32 (ldq) and/or directly as digits (q_dig, q_pitch), and
 * the scales (rows floats). 1 <= qmax <= 2^24. */
mosaic_status mosaic_quantize_rows(const float* x, int64_t ldx, int64_t rows, int64_t n,
                                   int32_t qmax, int32_t* q, int64_t ldq,
                                   int8_t* q_dig, int64_t q_pitch,
                                   float* scale, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MOSAIC_H */
