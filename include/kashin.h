/*
 * kashin.h -- C ABI of the MI355X (gfx950) Kashin-DCT quantizer hot path.
 *
 * The method ("Structured Transforms for Low-Overhead Quantization of Language
 * Models"): every weight vector w of length N (one row of an M x N matrix, one
 * output channel) is decomposed by the Greedy Algorithm with Alternating Updates
 * (Alg. 2) into w = u + P vhat + r, where P z = IDCT(eps * DCT(z)) is the
 * orthonormal DCT-II conjugated by a Rademacher sign mask eps (Sec. 4.1), a
 * symmetric involution (App. C).  Each factor is then quantised to 2-bit codes
 * around four centres initialised in closed form at +-c1 +- c2 (Sec. 3.1) and
 * packed four codes per byte (App. C).
 *
 * Conventions shared by every entry point
 *   - Every function returns a status (KASHIN_OK or a negative KASHIN_E_*), never
 *     throws, and records a message readable with kashin_last_error() (thread-local).
 *   - All matrix pointers are DEVICE pointers owned by the caller.  The plan owns
 *     only its own tables.  Matrices are row-major; row i of a matrix with leading
 *     dimension ld starts at element i * ld.
 *   - Arguments are validated on the host before anything is launched; invalid
 *     arguments return KASHIN_E_INVALID / KASHIN_E_UNSUPPORTED_N and launch nothing.
 *   - Launches are asynchronous on `stream` (a hipStream_t; NULL is the null
 *     stream).  A failed launch returns KASHIN_E_HIP.  m == 0 is a no-op.
 *   - Outputs are undefined after an error.  A row containing NaN or Inf yields NaN
 *     factors, NaN centres and zero codes for that row only.
 *   - Rows are processed two at a time (rows 2p and 2p+1 share one complex FFT).
 *     Results are deterministic run to run; a row's last bits may depend on the
 *     row it is paired with.
 *   - Plans are immutable after creation and may be shared across host threads and
 *     streams.  No entry point other than kashin_plan (its tables) and kashin_optq_factor (its
 *     temporaries, freed before it returns) allocates device memory.
 */
#ifndef KASHIN_H_
#define KASHIN_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct kashin_plan_s* kashin_plan_t;

enum {
  KASHIN_OK = 0,
  KASHIN_E_INVALID = -1,       /* null pointer, bad size, ld < N, iters < 1, dead plan, ... */
  KASHIN_E_UNSUPPORTED_N = -2, /* vector length without a compiled kernel (see kashin_supported_n) */
  KASHIN_E_NOMEM = -3,         /* host or device allocation failed (kashin_plan only) */
  KASHIN_E_HIP = -4,           /* HIP runtime error (no device, launch failure, ...) */
};

/* Input element types of the weight rows (every computation is fp32): IEEE binary32, binary16,
 * and bfloat16 (the upper half of a binary32; widened exactly). */
enum { KASHIN_F32 = 0, KASHIN_F16 = 1, KASHIN_BF16 = 2 };

/* 1 if vectors of length n have a compiled kernel, else 0.  Host only, no device needed.
 * The supported lengths are exactly
 *     64, 96, 172, 256, 512, 768, 1024, 2048, 3072, 4096, 5120, 6144, 8192, 10000, 11008,
 *     13824, 14336, 16384
 * (the row widths of the OPT, Llama-2, Pythia and Mistral layers of Sec. 5, the N = 10^4 of the
 * convergence comparison of Sec. 4.1, and small lengths for tests).  Each has a transform shape
 * compiled for it (a mixed-radix FFT over radices 2, 3, 4, 5, 7, 8, 9, 12, 16 and 43);
 * other lengths, even ones whose factors are all available, return 0.  A row pair of length N
 * occupies 8N bytes of LDS, so no length above about 19800 can be added on gfx950 (160 KB). */
int kashin_supported_n(int32_t n);

/* The sign mask eps in {-1,+1}^n for `seed` (Sec. 4.1 T_E; Sec. 5 / App. C: one mask per
 * layer drawn once from a fixed seed): eps_j = -1 iff the top bit of the j-th output of
 * splitmix64 started at state `seed` is set.  Writes n int8 values to host memory `eps_host`.
 * Host only, no device needed. */
int kashin_signs(int32_t n, uint64_t seed, int8_t* eps_host);

/* Create a plan for vectors of length n, sign mask from `sign_seed`, and `iters` blocks of
 * Alg. 2 (each block = two u-steps and two vhat-steps).  Builds the FFT twiddle table and
 * the eps-folded frequency table on the current HIP device (the library's only lasting device
 * allocation; kashin_optq_factor's temporaries are freed before it returns).  Requires n even,
 * kashin_supported_n(n), iters >= 1. */
int kashin_plan(kashin_plan_t* out, int32_t n, uint64_t sign_seed, int32_t iters);

/* Free a plan.  The caller must have synchronised every stream that used it. */
int kashin_plan_destroy(kashin_plan_t plan);

/* Copy the plan's n signs (+1/-1) to host memory. */
int kashin_plan_signs(kashin_plan_t plan, int8_t* eps_host);

/* Plan properties (host). */
int kashin_plan_info(kashin_plan_t plan, int32_t* n, int32_t* iters, uint64_t* seed);

/* Alg. 2 on every row of w (m x n, leading dimension ldw >= n, dtype KASHIN_F32, KASHIN_F16 or
 * KASHIN_BF16; arithmetic is fp32).  Outputs, all fp32 row-major with leading dimension n:
 *   u, vhat   m x n  factors with w = u + P vhat + r                       (required)
 *   r         m x n  residual after the last block (costs one more P)      (nullable)
 *   cstep     m x 4  magnitudes c of the four steps of block 0: c1, c2 (u-steps) and
 *                    c3, c4 (vhat-steps), the closed-form centre inputs (Sec. 3.1) (nullable)
 *   bounds    m x 4  ||u||_inf, ||vhat||_inf and the coefficient sums sum(c_u), sum(c_v)
 *                    that bound them (App. F)                               (nullable) */
int kashin_decompose(kashin_plan_t plan, const void* w, int32_t dtype, int64_t m, int64_t ldw,
                     float* u, float* vhat, float* r, float* cstep, float* bounds, void* stream);

/* Four-peak 2-bit clustering of given factors (Sec. 3.1).  u, vhat: m x n fp32 (ld n);
 * cstep: m x 4 from kashin_decompose.  Centres start at +-c1 +- c2 (u) and +-c3 +- c4
 * (vhat), then `lloyd_iters` >= 0 plain 1-D k-means passes (an emptied cluster keeps its
 * centre; centres re-sorted after each pass).  code = number of centre midpoints strictly
 * below the value.  Outputs: codes_u, codes_v: m x ceil(n/4) bytes, code of element i in
 * bits 2(i&3) of byte i>>2; centers: m x 2 x 4 fp32 ascending ([row][u=0|vhat=1][4]). */
int kashin_cluster2bit(kashin_plan_t plan, const float* u, const float* vhat, const float* cstep,
                       int64_t m, int32_t lloyd_iters, uint8_t* codes_u, uint8_t* codes_v,
                       float* centers, void* stream);

/* Load-time reconstitution w_hat = u_q + P v_q from codes and centres (App. C).
 * w_hat: m x n fp32, leading dimension ldw >= n. */
int kashin_reconstruct(kashin_plan_t plan, const uint8_t* codes_u, const uint8_t* codes_v,
                       const float* centers, int64_t m, float* w_hat, int64_t ldw, void* stream);

/* One matrix of kashin_reconstruct_grouped: the arguments kashin_reconstruct takes for it. */
typedef struct {
  kashin_plan_t plan;       /* every item's plan has the same n and lives on the same device */
  const uint8_t* codes_u;   /* m x ceil(n/4) (device) */
  const uint8_t* codes_v;   /* m x ceil(n/4) (device) */
  const float* centers;     /* m x 2 x 4 (device) */
  int64_t m;                /* >= 0; an item with m == 0 is skipped */
  float* w_hat;             /* m rows of n fp32, leading dimension ldw >= n (device) */
  int64_t ldw;
} kashin_reconstruct_item;

/* kashin_reconstruct over several matrices of one vector length, in one launch per 16 matrices
 * (the load-time reconstitution of App. C for every matrix of a layer, each with its own plan).
 * The persistent grid is split between the matrices in proportion to their row pairs (at least
 * one workgroup each, at most one per pair); a workgroup loads its matrix's operator constants
 * once and walks that matrix's pairs, so small matrices do not each pay a launch with its partial
 * last wave.  Every matrix's w_hat equals kashin_reconstruct's bit for bit.
 * items: host array of `count` entries (count >= 0), read before the call returns; nothing is
 * allocated (the matrix table travels in the kernel arguments).  Output ranges must not overlap. */
int kashin_reconstruct_grouped(const kashin_reconstruct_item* items, int32_t count, void* stream);

/* The fused hot path: kashin_decompose followed by kashin_cluster2bit without writing the
 * factors: each row is read from HBM once and only codes and centres are written.
 * Same layouts as kashin_decompose (input) and kashin_cluster2bit (outputs). */
int kashin_quantize(kashin_plan_t plan, const void* w, int32_t dtype, int64_t m, int64_t ldw,
                    int32_t lloyd_iters, uint8_t* codes_u, uint8_t* codes_v, float* centers,
                    void* stream);

/* One matrix of kashin_quantize_grouped: the arguments kashin_quantize takes for it. */
typedef struct {
  kashin_plan_t plan; /* every item's plan has the same n and iters and lives on the same device */
  const void* w;      /* m rows of n, leading dimension ldw >= n (device) */
  int64_t m;          /* >= 0; an item with m == 0 is skipped */
  int64_t ldw;
  uint8_t* codes_u;   /* m x ceil(n/4) (device) */
  uint8_t* codes_v;   /* m x ceil(n/4) (device) */
  float* centers;     /* m x 2 x 4, ascending (device) */
} kashin_quantize_item;

/* kashin_quantize over several matrices of one vector length, in one launch per 16 matrices: the
 * quantisation of every matrix of a layer or a model (Sec. 5 applies the method to each weight
 * matrix, each with its own sign mask, hence its own plan).  The row pairs of all matrices share
 * one grid, so the chip stays full where a matrix alone would leave a partial last wave of
 * workgroups.  Every matrix's codes and centres equal those of kashin_quantize on it alone (or,
 * with rot_seed non-NULL, of kashin_quantize_rotated with seed *rot_seed), bit for bit.
 * items: host array of `count` entries (count >= 0), read before the call returns; the per-launch
 * matrix table travels in the kernel arguments (nothing is allocated).  All matrices share dtype,
 * lloyd_iters and the rotation.  Output ranges of different items must not overlap. */
int kashin_quantize_grouped(const kashin_quantize_item* items, int32_t count, int32_t dtype, int32_t lloyd_iters,
                            const uint64_t* rot_seed, void* stream);

/* y = P x row-wise for fp32 rows (m x n, ld n): the operator of Sec. 4.1 / Alg. 2 alone.
 * x and y may not alias. */
int kashin_apply_p(kashin_plan_t plan, const float* x, float* y, int64_t m, void* stream);

/* Step schedules of the greedy over the dictionary Q_N u P Q_N (Sec. 4.2 and App. B). */
enum {
  KASHIN_SCHED_ALTERNATING = 0, /* blocks u, u, vhat, vhat: Alg. 2 */
  KASHIN_SCHED_REVERSE = 1,     /* blocks vhat, vhat, u, u: the reverse order named in Sec. 4.2 */
  KASHIN_SCHED_ADAPTIVE = 2,    /* every step: the u-half when ||rho||_1 > ||P rho||_1, else the
                                   vhat-half, step ||.||_1 / N (greedy selection over the whole
                                   dictionary, which Alg. 2 replaces) */
  KASHIN_SCHED_ORIGINAL = 3     /* Alg. 1 (App. B): the same choice, the step the orthogonal
                                   projection onto the sign vector (||.||_1 / nnz); a row takes
                                   no further steps once ||rho||_2 < tol */
};

/* The decomposition w = u + P vhat + r with 4k atomic steps (k = the plan's iters) in the given
 * schedule; sign(0) = 0 as in Alg. 2.  Layouts as kashin_decompose (r nullable).  Every step
 * applies P once (both domains of the residual are kept), so a step costs twice the transforms
 * of the alternating schedule of kashin_decompose.  tol applies to KASHIN_SCHED_ORIGINAL only
 * (0: never stop early), in the units of w. */
int kashin_decompose_schedule(kashin_plan_t plan, int32_t schedule, float tol, const void* w, int32_t dtype,
                              int64_t m, int64_t ldw, float* u, float* vhat, float* r, void* stream);

/* Replay record of kashin_decompose_schedule for the listed rows (as kashin_trace):
 *   sign_trace    nrows x 4k x n int8, element order of w: sign taken in the stepped vector
 *   c_trace       nrows x 4k fp32: step size
 *   choice_trace  nrows x 4k int8: 0 u-step, 1 vhat-step, -1 stopped (KASHIN_SCHED_ORIGINAL)
 *   r2_trace      nrows x 4k fp32: ||rho||_2^2 after the step
 *   u, vhat       nrows x n fp32 factors (ld n). */
int kashin_trace_schedule(kashin_plan_t plan, int32_t schedule, float tol, const void* w, int32_t dtype, int64_t m,
                          int64_t ldw, const int64_t* rows, int64_t nrows, int8_t* sign_trace, float* c_trace,
                          int8_t* choice_trace, float* r2_trace, float* u, float* vhat, void* stream);

/* Incoherence pre-rotation of rows, the "+H" preprocessing of Sec. 5 (the paper names a
 * QuIP-style randomised Hadamard transform, with a Kronecker variant, applied to the weights
 * before the decomposition; it gives no construction, so this one is a reading):
 *   R = (H_{2^a} / sqrt(2^a) kron C_b) diag(s),   n = 2^a b, b odd,
 * H the Sylvester Hadamard matrix, C_b the orthonormal DCT-II of length b (C_1 = [1]), element
 * index i b + j for segment i and position j, s_i = -1 when the top bit of the i-th splitmix64
 * output of `seed` is set (the generator of kashin_signs).  R is orthogonal.
 * y = R x (inverse = 0) or y = R^T x (inverse = 1) for m rows.
 *   n       odd part b in {1, 3, 43}, n <= 16384 (else KASHIN_E_UNSUPPORTED_N)
 *   x       m rows, dtype KASHIN_F32, KASHIN_F16 or KASHIN_BF16, leading dimension ldx >= n (device)
 *   y       m fp32 rows, leading dimension ldy >= n (device); y == x is allowed (in place) for
 *           fp32 with ldy == ldx, any other overlap is KASHIN_E_INVALID
 * Plan-free: runs on the current device.  Quantising R w and reconstructing R^T w_hat
 * composes the rotation with the rest of the path. */
int kashin_rotate(int32_t n, uint64_t seed, int32_t inverse, const void* x, int32_t dtype, int64_t m,
                  int64_t ldx, float* y, int64_t ldy, void* stream);

/* The "+H" pipeline with the rotation fused: kashin_quantize of R w (R as kashin_rotate with
 * seed rot_seed; n = the plan's length), the rows rotated on the way in, so w is read once and the
 * rotated rows are never written.  Codes and centres are those of R w; results equal
 * kashin_rotate followed by kashin_quantize of its fp32 output bit for bit.  Plans whose length
 * kashin_rotate does not take (odd part other than 1, 3 or 43) return KASHIN_E_UNSUPPORTED_N; so
 * do kashin_reconstruct_rotated and kashin_quantize_grouped with a rotation seed. */
int kashin_quantize_rotated(kashin_plan_t plan, uint64_t rot_seed, const void* w, int32_t dtype, int64_t m,
                            int64_t ldw, int32_t lloyd_iters, uint8_t* codes_u, uint8_t* codes_v, float* centers,
                            void* stream);

/* Load-time reconstitution of a rotated quantisation: w_hat = R^T (u_q + P v_q), equal to
 * kashin_reconstruct followed by the inverse kashin_rotate bit for bit.  Layouts as
 * kashin_reconstruct. */
int kashin_reconstruct_rotated(kashin_plan_t plan, uint64_t rot_seed, const uint8_t* codes_u, const uint8_t* codes_v,
                               const float* centers, int64_t m, float* w_hat, int64_t ldw, void* stream);

/* Test hook: replay record of Alg. 2 for selected rows.  For each of the `nrows` row
 * indices in `rows` (device int64, each in [0, m)), the row is decomposed exactly as
 * kashin_decompose does (paired with the same neighbour) and the kernel writes
 *   sign_trace  nrows x 4k x n int8: sign (-1, 0, +1) taken at each atomic step, element
 *               order of w (steps 4t, 4t+1 are u-steps, 4t+2, 4t+3 vhat-steps)
 *   c_trace     nrows x 4k fp32: the step magnitudes c
 *   u, vhat     nrows x n fp32 factors (ld n). */
int kashin_trace(kashin_plan_t plan, const void* w, int32_t dtype, int64_t m, int64_t ldw,
                 const int64_t* rows, int64_t nrows, int8_t* sign_trace, float* c_trace,
                 float* u, float* vhat, void* stream);

/* Error-compensated quantisation (Sec. 5, Fig. 1: the columns of W quantised one after another, each
 * one's error carried into the columns not yet quantised, eq. optq_update with the 1 % damping of
 * the Sec. 5 remark).  W (d_out x d_in) is held transposed, w_t = W^T (d_in rows of n = d_out), so a
 * column of W is a row of w_t.
 *
 * kashin_optq_factor: from H (d x d fp32 row-major, leading dimension ldh >= d, symmetric; device),
 * the upper-triangular U with U^T U = (H + lambda I)^-1, lambda = damp * mean(diag H), and V = U^-1
 * (v nullable), both d x d float64 row-major (device, caller-owned).  Computed as the lower Cholesky
 * factor L of J (H + lambda I) J (J reverses the index order: then H + lambda I = V V^T with
 * V = J L J upper) and its triangular inverse, in float64 (rocSOLVER).  Unlike every other entry
 * point it allocates temporary device memory (d x d float64 and the solver's workspace) and frees it
 * before returning, and it synchronises `stream`.  KASHIN_E_INVALID if the damped Hessian is not
 * positive definite. */
int kashin_optq_factor(const float* h, int32_t d, int64_t ldh, double damp, double* u, double* v, void* stream);

/* Device workspace bytes kashin_optq_quantize needs for d_in rows of length n in chunks of `chunk`
 * (an error matrix, chunk x n fp32, and a factor block, chunk x d_in fp32); -1 for bad sizes
 * (d_in < 0, n < 1, chunk outside [1, 128]). */
int64_t kashin_optq_workspace_bytes(int64_t d_in, int32_t n, int32_t chunk);

/* Quantise rows 0 .. quantize_rows - 1 of w_t (d_in rows, fp32, leading dimension ldw >= n = the
 * plan's length; device) with error compensation, carrying their errors into every later row of
 * w_t, which is updated in place (quantize_rows = d_in: the whole matrix; a smaller count lets a
 * caller resume on the tail, with the factor's trailing block).  u, v: the output of
 * kashin_optq_factor for d = d_in, leading dimension ldu >= d_in (v may be NULL when exact = 1).
 * Outputs for the quantised rows (device): codes_u, codes_v rows x ceil(n/4), centers rows x 2 x 4 (as
 * kashin_quantize), q_t rows x n fp32 (ld n): the dequantised rows (as kashin_reconstruct).
 *   exact = 0: chunks of `chunk` rows (1 <= chunk <= 128) quantised together; after each chunk c,
 *              w_t[r] -= (U_cc^-1 U_cr)^T Delta with Delta = w_t[c] - q_t[c] for the later rows r;
 *              equal to eq. optq_update at chunk = 1.
 *   exact = 1: rows quantised one at a time; err_i = (w_t[i] - q_t[i]) / U_ii reaches the later rows
 *              j of its chunk at once (w_t[j] -= U_ij err_i) and the rows after the chunk in one
 *              product at the chunk's end (w_t[r] -= U_cr^T E): eq. optq_update row by row for any
 *              chunk size.
 * work: at least kashin_optq_workspace_bytes(d_in, n, chunk) bytes of device memory (its contents on
 * entry do not matter).  Allocates nothing; every launch is queued on `stream`. */
int kashin_optq_quantize(kashin_plan_t plan, float* w_t, int64_t d_in, int64_t ldw, const double* u, const double* v,
                         int64_t ldu, int64_t quantize_rows, int32_t chunk, int32_t exact, int32_t lloyd_iters,
                         uint8_t* codes_u, uint8_t* codes_v, float* centers, float* q_t, void* work,
                         int64_t work_bytes, void* stream);

/* kashin_optq_quantize for callers that cannot allocate (code under HIP graph capture, serving
 * loops, harnesses that forbid hipMalloc): the same computation with the workspace taken from a
 * static device array of the library instead of the `work` argument, so the caller passes only
 * inputs and outputs.  The array holds 16 MiB on each device (allocated with the library's code
 * object, held until the process ends); kashin_optq_workspace_bytes(d_in, n, chunk) must not exceed
 * it (chunk 128 with d_in + n <= 32768 fits), else KASHIN_E_INVALID.  Every call on a device uses
 * the same array: calls that overlap on one device race.  Results equal kashin_optq_quantize's. */
int kashin_optq_quantize_noalloc(kashin_plan_t plan, float* w_t, int64_t d_in, int64_t ldw, const double* u,
                                 const double* v, int64_t ldu, int64_t quantize_rows, int32_t chunk, int32_t exact,
                                 int32_t lloyd_iters, uint8_t* codes_u, uint8_t* codes_v, float* centers, float* q_t,
                                 void* stream);

/* Static text for a status code. */
const char* kashin_status_string(int status);

/* Message of the last failed call on this host thread ("" if none). */
const char* kashin_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* KASHIN_H_ */
