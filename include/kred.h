/*
 * kred: reductions over symbolic M x N kernel and distance matrices on one
 * AMD Instinct MI355X (gfx950).  C ABI.
 *
 * The library evaluates Eq. (2) of Charlier et al., "Kernel Operations on the
 * GPU, with Autodiff, without Memory Overflows" (arXiv:2004.11127, Sec. 2):
 *
 *     a_i = Reduction_{j = 0..N-1} F(p, x_i, y_j, b_j),   i = 0..M-1,
 *
 * for a fixed set of formulas F and the reductions Sec. 2 lists, without ever
 * storing the M x N matrix (Sec. 2: no N-by-M buffer in device memory; memory
 * stays linear in M + N).  The motivating case is Eq. (1), the Gaussian
 * kernel sum a_i = sum_j exp(-|x_i - y_j|^2 / (2 sigma^2)) b_j.  Indices are
 * 0-based (the paper counts i = 1..M, j = 1..N).
 *
 * Layout: every array is dense, contiguous, row-major fp32 (int32 for k-NN
 * indices) in device memory of the context's device: x is M x D, y is N x D,
 * b is N x E.  Pointers need 4-byte alignment.  The caller owns x, y, b and
 * out; the library never frees or keeps them past the call.
 *
 * Errors: every argument is checked on the host before anything is launched;
 * on any error nothing runs and out is untouched.  Launch failures return
 * KRED_ERR_HIP.  Faults inside a kernel surface at the caller's next
 * synchronisation.  The library never prints and never aborts.
 *
 * Concurrency: kred_run is asynchronous on `stream`.  A context owns scratch
 * memory (column-split partials and packed copies of y and b) that calls on it
 * reuse, so one context must not run on two streams at once; use one context
 * per stream.
 */
#ifndef KRED_H
#define KRED_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KRED_VERSION 1

/* Formulas F (Sec. 2 "symbolic formula"; Eq. (1) is KRED_F_GAUSS). */
typedef enum kred_formula {
  KRED_F_GAUSS = 0,       /* k = exp(-|x - y|^2 / (2 sigma^2)), F = k b            (Eq. (1)) */
  KRED_F_LAPLACE = 1,     /* k = exp(-|x - y| / sigma),         F = k b                      */
  KRED_F_SQDIST = 2,      /* d = |x - y|^2,                     F = d b (sum) or d (arg-K-min) */
  KRED_F_GAUSS_GRADX = 3, /* Eq. (1) and its gradient in x_i, fused (Sec. 2 "Backpropagation") */
  KRED_F_SINKHORN = 4     /* s = g_j - |x - y|^2 / eps, with g_j passed in b          */
} kred_formula;

/* Reductions over j (Sec. 2: .sum(), .logsumexp(), .min(), .max(), .argmin(),
 * .argKmin(K); arg-max and the K smallest values complete the set). */
typedef enum kred_reduction {
  KRED_R_SUM = 0,
  KRED_R_LSE = 1,
  KRED_R_ARGKMIN = 2,
  KRED_R_MIN = 3,
  KRED_R_MAX = 4,
  KRED_R_ARGMIN = 5,
  KRED_R_ARGMAX = 6,
  KRED_R_KMIN = 7
} kred_reduction;

typedef enum kred_status {
  KRED_OK = 0,
  KRED_ERR_INVALID_ARG = 1,  /* a null pointer, a size or parameter out of range */
  KRED_ERR_UNSUPPORTED = 2,  /* a (formula, reduction) pair the library does not provide */
  KRED_ERR_NOMEM = 3,        /* scratch allocation failed */
  KRED_ERR_HIP = 4,          /* a HIP runtime call or kernel launch failed */
  KRED_ERR_NO_DEVICE = 5,    /* no usable gfx950 device with that ordinal */
  KRED_ERR_SCRATCH = 6       /* kred_run_noalloc: the call needs more than its fixed scratch */
} kred_status;

/* flags */
#define KRED_FLAG_PROFILE 1u  /* time the main kernel of each call with HIP events (kred_profile_collect) */
#define KRED_FLAG_DIRECT 2u   /* D <= 4: always use the direct-form kernels, never the matrix-core exponent
                                 (used otherwise only below 2^28 pairs, or when the data's extent
                                 c R^2 exceeds the matrix-core form's accuracy limit: 2048 at D <= 3,
                                 128 at D = 4 for the sums and log-sum-exps, 2048 for the nearest
                                 distances; R is the half-diagonal of the joint bounding box of x and
                                 y, c = log2(e) / (2 sigma^2), log2(e) / eps, or 1).  Inside the limit
                                 the matrix-core exponent's error stays below the direct form's parity
                                 bar (1e-4 of sum_j |k_ij b_j|).  GAUSS_GRADX: the matrix-core path's
                                 gradient is within 1e-4 sum_j |k_ij b_j| / sigma per component; the
                                 direct form's within 1e-4 sum_j |k_ij b_j (y_jk - x_ik)| / sigma^2,
                                 which resolves components that nearly cancel (e.g. x a subset of y
                                 on data sparse against sigma).  D > 16 arg-K-min (and K-min,
                                 min / arg-min without b): always the fp32 matrix-core kernel, never
                                 the exact bf16 one */
#define KRED_FLAG_FAST 4u     /* D <= 4: use the matrix-core exponent whatever the problem size (the
                                 accuracy guard still falls back to the direct form).  D > 16
                                 sums (and LSE at 17 <= D <= 128): the split bf16 products whatever
                                 the size (same guard).  D > 16
                                 arg-K-min: consider the exact bf16 kernel whatever the size (it
                                 runs only when every coordinate is an integer with |v| <= 256 and
                                 D max|v|^2 <= 2^22, where bf16 products and fp32 sums are exact;
                                 otherwise the fp32 kernel runs; by default it is considered from
                                 2^28 pairs).  DIRECT wins */

/* Per-call parameters (the "parameters p" of Eq. (2)). */
typedef struct kred_params {
  float sigma;        /* kernel width for GAUSS, LAPLACE, GAUSS_GRADX; > 0, finite       */
  float eps;          /* temperature for SINKHORN; > 0, finite                            */
  int32_t K;          /* number of neighbours for ARGKMIN; 1 <= K <= min(N, 64)           */
  int32_t col_blocks; /* j split into this many blocks reduced in a second pass; 0 = auto */
  uint32_t flags;     /* KRED_FLAG_* */
} kred_params;

/* Limits */
#define KRED_MAX_D 256
#define KRED_MAX_E 64
#define KRED_MAX_K 64
#define KRED_MAX_COL_BLOCKS 256
/* Size of the fixed device scratch of kred_run_noalloc (32 MiB per GPU). */
#define KRED_NOALLOC_SCRATCH_BYTES (32u << 20)

typedef struct kred_ctx kred_ctx;

/*
 * Create a context on HIP device `device` (ordinal as seen by the process).
 * On success *ctx is set; release it with kred_destroy.  Allocates no device
 * memory until a call needs scratch.  Returns KRED_ERR_INVALID_ARG if ctx is
 * NULL, KRED_ERR_NO_DEVICE if the ordinal is invalid or not gfx950,
 * KRED_ERR_NOMEM if the host allocation fails.
 */
kred_status kred_create(kred_ctx** ctx, int device);

/* Free the context and its scratch memory (synchronises the device first).
 * NULL is accepted and ignored. */
kred_status kred_destroy(kred_ctx* ctx);

/*
 * Evaluate a_i = Reduction_j F(p, x_i, y_j, b_j) for i = 0..M-1 (Eq. (2)).
 *
 * Valid (formula, reduction) pairs and their operands:
 *   (GAUSS | LAPLACE | SQDIST, SUM):  b is N x E, out is fp32 M x E:
 *        out[i, e] = sum_j F(|x_i - y_j|^2) b[j, e].
 *   (GAUSS_GRADX, SUM), E = 1:  b is N x 1, out is fp32 M x (1 + D):
 *        out[i, 0]     = a_i = sum_j k_ij b_j                       (Eq. (1))
 *        out[i, 1 + k] = sum_j k_ij b_j (y_jk - x_ik) / sigma^2 = d a_i / d x_ik.
 *   (SINKHORN, LSE), E = 1:  b holds g (N x 1), out is fp32 M x 1:
 *        out[i] = log sum_j exp(g_j - |x_i - y_j|^2 / eps)   (natural log).
 *   (GAUSS | LAPLACE, LSE), E = 1:  the log-domain kernel sum with weights g
 *        in b: out[i] = log sum_j k_ij exp(g_j), i.e. log sum_j exp(g_j -
 *        |x_i - y_j|^2 / (2 sigma^2)) or log sum_j exp(g_j - |x_i - y_j| / sigma).
 *   (SQDIST, ARGKMIN):  b must be NULL and E is ignored (pass 0), out is int32
 *        M x K: the indices j of the K smallest |x_i - y_j|^2, ascending by
 *        (distance, index): equal distances keep the lower index first.
 *   (SQDIST, KMIN):  as ARGKMIN, but out is fp32 M x K: the K smallest
 *        squared distances themselves, in the same order.
 *   (GAUSS | LAPLACE | SQDIST, MIN | MAX | ARGMIN | ARGMAX) with b (N x E):
 *        per component e of F_ije = k(|x_i - y_j|^2) b_je (k as for SUM; k = d
 *        for SQDIST), the smallest / largest value over j (out fp32 M x E) or
 *        the lowest index j where it is reached (out int32 M x E).
 *   (SQDIST, MIN | MAX | ARGMIN | ARGMAX) with b = NULL:  F_ij = |x_i - y_j|^2,
 *        E ignored, out M x 1 (nearest / farthest distance or index).
 *   (SINKHORN, MIN | MAX | ARGMIN | ARGMAX), E = 1:  F_ij = g_j - |x_i - y_j|^2
 *        / eps with g in b, out M x 1 (the max is the hard limit of LSE).
 * Any other pair returns KRED_ERR_UNSUPPORTED.
 *
 * Ranges: 0 <= M, N <= 2^31 - 1; 1 <= D <= KRED_MAX_D; 1 <= E <= KRED_MAX_E
 * where b has E columns; p->col_blocks in [0, KRED_MAX_COL_BLOCKS].  D > 16
 * is supported by the sums, GAUSS_GRADX (as one Gaussian sum with the D + 1
 * signal columns [b, b (y - m)] for a centre m of y, then g = (A1 - (x - m)
 * A0) / sigma^2; scratch grows by about (M + 64 N)(D + 1) floats), every LSE,
 * ARGKMIN, KMIN, and every MIN / MAX / ARGMIN / ARGMAX (signal columns in
 * slices of 16), on the matrix cores in the expanded form |x'|^2 + |y'|^2 -
 * 2 <x', y'> of coordinates centred on m (the mean of y's first 256 rows) and
 * scaled by sqrt(c), c = log2(e) / (2 sigma^2), log2(e) / eps or 1.  Accuracy
 * guard (computed on the device, no host synchronisation): with L = c (max_i
 * |x_i - m|^2 + max_j |y_j - m|^2), the Gaussian and Sinkhorn forms use fp32
 * products (KRED_FLAG_DIRECT or below 2^28 pairs; error in the exponent below
 * (D + 10) 2^-24 L) or, for the sums and (at 17 <= D <= 128) the LSE, split
 * bf16 products (error below (D / 2 + 18) 2^-24 L; from 2^28 pairs, or with
 * KRED_FLAG_FAST) while that bound stays within 1.2e-4 in log2 units,
 * and the fp64 contraction beyond it; the Laplacian forms and the squared
 * distance's sums and extremes always use the fp64 contraction.  ARGKMIN /
 * KMIN rank in fp32 and re-rank the merged candidates by their direct-form
 * distance (KMIN values are the distances of the returned points).  Inputs
 * must be finite (NaN or Inf in x, y or b gives an undefined result).
 * Edge cases: M = 0 returns KRED_OK and touches nothing.  N = 0 writes zeros
 * (SUM), -infinity (LSE, MAX), +infinity (MIN) or -1 (ARGMIN, ARGMAX) and
 * reads no input (b may then be NULL; for SQDIST, a NULL b means one output
 * column); ARGKMIN and KMIN with N = 0 fail since they need K <= N.
 *
 * `stream` is a hipStream_t (NULL = the null stream of the context's device).
 * The call is asynchronous: it returns once the kernels are enqueued.
 * Scratch memory comes from the context and is grown with hipMalloc when a
 * call needs more than it holds; no M x N buffer is ever allocated (scratch
 * is O((M + N) (D + E)) plus O(M col_blocks (E + D + K))).
 */
kred_status kred_run(kred_ctx* ctx, kred_formula f, kred_reduction r, const kred_params* p,
                     int64_t M, int64_t N, int32_t D, int32_t E,
                     const float* x, const float* y, const float* b, void* out,
                     void* stream);

/*
 * kred_run for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, pairs, kernels and results as kred_run, but it calls no
 * hipMalloc, hipFree or other allocating routine: its device scratch (packed
 * copies of y and b, column-split partials, guards) comes from a fixed array
 * of KRED_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs
 * on until the process ends (its address is looked up in kred_create).
 *
 * Returns KRED_ERR_SCRATCH, before launching anything, when the call needs
 * more scratch than that (kred_scratch_bytes tells how much a call needs; for
 * example a 10^4 x 10^4 Gaussian sum needs about 3.4 MB, a 10^6-column D = 3
 * direct-form sum about 20 MB).  KRED_FLAG_PROFILE is refused
 * (KRED_ERR_INVALID_ARG): its events allocate.  Otherwise as kred_run.
 *
 * Every call on one GPU shares that GPU's array, whatever the context, and
 * the array keeps the last call's contents (the kernels initialise what they
 * read): calls that overlap in time on one GPU, on any streams or contexts,
 * race and give undefined results.  Serialise them (one stream, or events).
 */
kred_status kred_run_noalloc(kred_ctx* ctx, kred_formula f, kred_reduction r, const kred_params* p,
                             int64_t M, int64_t N, int32_t D, int32_t E,
                             const float* x, const float* y, const float* b, void* out,
                             void* stream);

/*
 * Block-sparse reduction (the cluster-wise block-sparsity patterns and the
 * block-sparse truncation rule of Sec. 3): kred_run restricted to a pattern
 * of (row cluster, column range) blocks.  Row cluster I = 0..nr-1 is the rows
 * [row_ranges[2I], row_ranges[2I+1]); its rows reduce over the columns of the
 * ranges [col_ranges[2q], col_ranges[2q+1]) for q in [col_ptr[I],
 * col_ptr[I+1]) only, as if F_ij were absent elsewhere.  Typical use: sort the
 * points by cluster, and list for each cluster of x the clusters of y whose
 * centroids are near enough (a truncation rule for a fast-decaying kernel).
 *
 * The three index arrays are int32 in device memory (row_ranges nr x 2,
 * col_ptr nr + 1, col_ranges col_ptr[nr] x 2), read by the kernels; the host
 * never dereferences them.  Row clusters must be disjoint; the column ranges
 * of a cluster should be sorted and disjoint for the arg-reductions' lowest-
 * index tie rule (otherwise ties resolve in list order).  Ranges are clamped
 * to [0, M) and [0, N); overlapping row clusters give an undefined result.
 * Rows in no cluster, and clusters without columns, hold the empty reduction
 * (as for N = 0; arg-K-min / K-min pad short lists with -1 / +infinity).
 *
 * Every pair kred_run accepts, on the same paths (direct form, the D <= 4
 * matrix-core exponent, and for 16 < D <= 256 the matrix-core kernels, which
 * start their column tiles 16-aligned and mask the columns outside a range).
 * col_blocks (0: automatic) splits each cluster's columns into that many
 * chunks, reduced by the second pass.  Arguments, layouts, errors and
 * asynchrony otherwise as kred_run; nr = 0 leaves every row empty.
 */
kred_status kred_run_ranges(kred_ctx* ctx, kred_formula f, kred_reduction r, const kred_params* p,
                            int64_t M, int64_t N, int32_t D, int32_t E,
                            const float* x, const float* y, const float* b, void* out,
                            int32_t nr, const int32_t* row_ranges, const int32_t* col_ptr,
                            const int32_t* col_ranges, void* stream);

/*
 * Block-sparse truncation pattern on the device (Sec. 3 cluster-wise
 * block-sparsity with the block-sparse truncation rule of Sec. 4), the arrays
 * kred_run_ranges takes, built without a pass through host memory:
 *   - a grid of cubic cells of side `cell` over the joint bounding box of x
 *     (M x D) and y (N x D): origin o = the coordinate-wise minimum, dims_d =
 *     floor((max_d - o_d) / cell) + 1; each point's cell k_d = min(floor((p_d -
 *     o_d) / cell), dims_d - 1), labelled k_0 dims_1 .. dims_{D-1} + .. + k_{D-1};
 *   - order_x (M) / order_y (N): the stable sort of each cloud by label
 *     (apply them to x, and to y and b, with kred_gather_rows; the result of
 *     kred_run_ranges on the sorted points comes back in row order with the
 *     inverse gather);
 *   - row_ranges (M x 2): cluster I of x is rows [row_ranges[2I],
 *     row_ranges[2I+1]) of the sorted x; entries from the cluster count up to
 *     M are the empty range [M, M), so nr = M is always a valid count;
 *   - col_ptr (M + 1) and col_ranges (col_cap x 2): for cluster I of x, the
 *     clusters of y whose cell centres o + (k + 1/2) cell lie within cutoff +
 *     cell sqrt(D) of its own centre, consecutive clusters merged into one
 *     range of the sorted y (col_ptr[I] = col_ptr[count] for the empty ones);
 *   - counts (4 int64): the clusters of x, the column ranges needed, the kept
 *     (i, j) pairs, and 1 when the column ranges exceed col_cap (the ranges
 *     past col_cap are then not written: call again with a larger col_cap).
 * Every step repeats in fp64 the arithmetic of clusters.truncation_pattern in
 * the Python package, so the arrays are identical to it.  1 <= M, N < 2^31 - 1,
 * 1 <= D <= 8, cell > 0 and cutoff >= 0 finite; every array is a device array
 * owned by the caller (col_ranges may be NULL when col_cap = 0).
 * Asynchronous on `stream`; counts is valid once it completes.  Uses the
 * context's scratch (about 40 bytes per point).
 */
kred_status kred_cluster_pattern(kred_ctx* ctx, int64_t M, int64_t N, int32_t D, const float* x,
                                 const float* y, double cell, double cutoff, int32_t* order_x,
                                 int32_t* order_y, int32_t* row_ranges, int32_t* col_ptr,
                                 int32_t* col_ranges, int64_t col_cap, int64_t* counts,
                                 void* stream);

/*
 * Row permutation of an n x width fp32 array on the device: dst[i] =
 * src[index[i]], or with inverse = 1 dst[index[i]] = src[i] (index a
 * permutation of 0 .. n-1, int32).  src and dst must not overlap.
 * Asynchronous on `stream`.
 */
kred_status kred_gather_rows(kred_ctx* ctx, int64_t n, int32_t width, const float* src,
                             const int32_t* index, float* dst, int32_t inverse, void* stream);

/* Host-only argument check of kred_run_ranges (the index arrays are only
 * checked for null and alignment). */
kred_status kred_validate_ranges(kred_formula f, kred_reduction r, const kred_params* p,
                                 int64_t M, int64_t N, int32_t D, int32_t E,
                                 const void* x, const void* y, const void* b, const void* out,
                                 int32_t nr, const void* row_ranges, const void* col_ptr,
                                 const void* col_ranges);

/*
 * Host-only argument check with the same rules kred_run applies (kred_run
 * calls it first).  Touches no device and dereferences no array pointer, so
 * it runs on machines without a GPU.  Returns KRED_OK or the error kred_run
 * would return.
 */
kred_status kred_validate(kred_formula f, kred_reduction r, const kred_params* p,
                          int64_t M, int64_t N, int32_t D, int32_t E,
                          const void* x, const void* y, const void* b, const void* out);

/*
 * Scratch bytes kred_run will need for this call (0 when none), or -1 when
 * the arguments are invalid.  Host-only.  For the MIN / MAX / ARGMIN / ARGMAX
 * reductions of SQDIST, E = 0 stands for a call without b.
 */
int64_t kred_scratch_bytes(kred_formula f, kred_reduction r, const kred_params* p,
                           int64_t M, int64_t N, int32_t D, int32_t E);

/*
 * Gradients of the Gaussian kernel sum (Sec. 2 "Backpropagation": the
 * derivative of a reduction of the form of Eq. (2) is again such a
 * reduction).  For a = K b with a_i = sum_j k_ij b_j, k_ij = exp(-|x_i - y_j|^2
 * / (2 sigma^2)), b N x E (Eq. (1) with E signal columns), and a cotangent e
 * (M x E, the gradient of a scalar loss with respect to a), this computes the
 * gradients of L = sum_i <e_i, a_i>:
 *   gx (M x D):  gx[i] = sum_j k_ij <e_i, b_j> (y_j - x_i) / sigma^2
 *   gy (N x D):  gy[j] = sum_i k_ij <e_i, b_j> (x_i - y_j) / sigma^2
 *   gb (N x E):  gb[j] = sum_i k_ij e_i
 * Each output pointer may be NULL, and that gradient is not computed.  gy is
 * the gx reduction with the roles of (x, e) and (y, b) exchanged, and gb the
 * Gaussian sum with x and y exchanged; all three run on the same kernels as
 * kred_run, one after the other on `stream`.  Outputs are fp32, dense,
 * row-major device arrays owned by the caller.
 *
 * Parameters: p->sigma (> 0, finite), p->col_blocks and p->flags as for
 * kred_run (KRED_FLAG_DIRECT / KRED_FLAG_FAST steer the path of every
 * reduction in the call; KRED_FLAG_PROFILE times each main kernel); p->eps
 * and p->K are ignored.  Ranges: 0 <= M, N <= 2^31 - 1, 1 <= D <= KRED_MAX_D,
 * 1 <= E <= KRED_MAX_E.  For D > 16, gx and gy run as one Gaussian sum with
 * the E (D + 1) signal columns [b_e, b_e (y - m)] (m a centre of y), 64
 * columns per matrix-core launch (on the split kernel at D <= 128 a last
 * single column is summed by the first launch), contracted with the
 * cotangent; scratch grows by about (M + 64 N) E (D + 1) floats.  With M = 0 or N = 0
 * the requested outputs are filled with zeros.  x, y and e are required, and
 * b too for gx or gy, whenever M, N > 0 and an output is requested.  Same
 * error and asynchrony rules as kred_run: on any argument error nothing runs.
 */
kred_status kred_gauss_backward(kred_ctx* ctx, const kred_params* p, int64_t M, int64_t N,
                                int32_t D, int32_t E, const float* x, const float* y,
                                const float* b, const float* e, float* gx, float* gy, float* gb,
                                void* stream);

/* Host-only argument check of kred_gauss_backward (no device, no dereference). */
kred_status kred_validate_backward(const kred_params* p, int64_t M, int64_t N, int32_t D,
                                   int32_t E, const void* x, const void* y, const void* b,
                                   const void* e, const void* gx, const void* gy,
                                   const void* gb);

/*
 * Gradients of the block-sparse Gaussian sum (Sec. 2 "Backpropagation" with
 * the cluster-wise block-sparsity of Sec. 3): a_i = sum_{j in S(i)} k_ij b_j,
 * S(i) the column ranges of row i's cluster as in kred_run_ranges, and the
 * gradients of L = sum_i <e_i, a_i> as in kred_gauss_backward restricted to
 * the kept pairs:
 *   gx[i] = sum_{j in S(i)} k_ij <e_i, b_j> (y_j - x_i) / sigma^2
 *   gy[j] = sum_{i : j in S(i)} k_ij <e_i, b_j> (x_i - y_j) / sigma^2
 *   gb[j] = sum_{i : j in S(i)} k_ij e_i
 * gx reduces over rows with the row-cluster pattern (nr, row_ranges,
 * col_ptr, col_ranges: exactly kred_run_ranges's arrays).  gy and gb reduce
 * over columns, so they take the same block set from the columns' side:
 * column cluster J = 0..nc-1 is the columns [col_clusters[2J],
 * col_clusters[2J+1]), and its columns sum over the rows of the ranges
 * [row_ranges_t[2q], row_ranges_t[2q+1]) for q in [row_ptr[J], row_ptr[J+1]).
 * The caller keeps the two patterns consistent (the same (i, j) pairs;
 * clusters.transpose_pattern in the Python package builds one from the
 * other); otherwise gy and gb are the gradients of another mask.  Columns
 * in no cluster get zero gy and gb, rows in no cluster zero gx.
 *
 * All index arrays are int32 device arrays with the rules of
 * kred_run_ranges (disjoint clusters, clamping to [0, M) and [0, N)); a
 * pattern's arrays may be NULL when its count is 0 or when the outputs it
 * serves are not requested.  Parameters, outputs, errors and asynchrony as
 * kred_gauss_backward (D and E limits, E-slices and col_blocks as there, the
 * column split applying to each cluster's ranges).
 */
kred_status kred_gauss_backward_ranges(kred_ctx* ctx, const kred_params* p, int64_t M, int64_t N,
                                       int32_t D, int32_t E, const float* x, const float* y,
                                       const float* b, const float* e, float* gx, float* gy,
                                       float* gb, int32_t nr, const int32_t* row_ranges,
                                       const int32_t* col_ptr, const int32_t* col_ranges,
                                       int32_t nc, const int32_t* col_clusters,
                                       const int32_t* row_ptr, const int32_t* row_ranges_t,
                                       void* stream);

/* Host-only argument check of kred_gauss_backward_ranges (the index arrays
 * are only checked for null and alignment). */
kred_status kred_validate_backward_ranges(const kred_params* p, int64_t M, int64_t N, int32_t D,
                                          int32_t E, const void* x, const void* y, const void* b,
                                          const void* e, const void* gx, const void* gy,
                                          const void* gb, int32_t nr, const void* row_ranges,
                                          const void* col_ptr, const void* col_ranges, int32_t nc,
                                          const void* col_clusters, const void* row_ptr,
                                          const void* row_ranges_t);

/*
 * With KRED_FLAG_PROFILE set on calls, the context records a HIP event pair
 * around the main reduction kernel of each call.  This waits for those
 * events, returns the number of timed launches in *count and their summed
 * duration in milliseconds in *total_ms, and forgets them.  Names the last
 * timed kernel family in *kernel (static string; may be NULL).  Where the
 * device picks the kernel (the small-D matrix-core path against the direct
 * form, the exact k-NN kernel against the fp32 one), the name is what the
 * device chose: for the small-D path over every profiled call since the last
 * collect, "fast_kernel+direct" when the choice differed between them.
 */
kred_status kred_profile_collect(kred_ctx* ctx, int32_t* count, double* total_ms,
                                 const char** kernel);

/* Static description of a status code. */
const char* kred_strerror(kred_status s);

/* KRED_VERSION of the built library. */
int32_t kred_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KRED_H */
