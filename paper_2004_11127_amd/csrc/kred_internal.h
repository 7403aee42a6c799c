// Internal declarations shared by the kred host runtime and its HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace kred {

// Formula codes used inside the kernels (same values as the public enum).
// Internal ones: F_VJP, the vector-Jacobian product of the Gaussian sum in x;
// F_LAPLACE_LSE, the log-sum-exp of g_j - |x_i - y_j| / sigma (the Gaussian's
// log-sum-exp, g_j - |x_i - y_j|^2 / (2 sigma^2), runs as F_SINKHORN).
enum : int {
  F_GAUSS = 0, F_LAPLACE = 1, F_SQDIST = 2, F_GRADX = 3, F_SINKHORN = 4, F_VJP = 5,
  F_LAPLACE_LSE = 6
};

constexpr int kThreads = 256;          // threads per workgroup for the direct-form kernels
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Small-D fast path (D <= 4): exponent on the bf16 matrix cores.  The
// prologue computes the joint bounding box of x and y on the device; the
// fast kernels run only when c R^2 <= the limit for D (R the half-diagonal of
// the box in prescaled units), otherwise the direct-form kernels do the work.
// Both are launched; each returns at once when the other one is selected.
// MIN: nearest distance / index; KNN: the K nearest (1 < K <= 16)
enum : int { FAST_SUM = 0, FAST_GRADX = 1, FAST_LSE = 2, FAST_MIN = 3, FAST_KNN = 4, FAST_SUMV = 5 };
// Largest c R^2 the matrix-core exponent takes.  The bound on its error in
// log2 units grows linearly with c R^2 (derived in k_small_mfma.hip): at
// D <= 3 eight products per coordinate fit the 32 K slots and the limit is
// 2048; at D = 4 only six fit, the two dropped ones dominate, and the limit
// is 128.  Both keep the worst-case bound below the 1e-4 parity bar.
// The nearest-neighbour forms use the expanded form only to rank candidates
// (their values are recomputed in the direct form) and take 2048 at every D.
constexpr float kFastLimit3 = 2048.0f;
constexpr float kFastLimit4 = 128.0f;
constexpr float kFastLimitNearest = 2048.0f;
inline float fast_limit(int D, bool nearest) {
  return nearest ? kFastLimitNearest : (D <= 3 ? kFastLimit3 : kFastLimit4);
}

struct FastGuard {
  int lo[4];   // order-preserving int encodings of the box corners
  int hi[4];
};

__device__ __forceinline__ int fenc(float f) {
  const int i = __float_as_int(f);
  return i >= 0 ? i : i ^ 0x7fffffff;
}
__device__ __forceinline__ float fdec(int i) { return __int_as_float(i >= 0 ? i : i ^ 0x7fffffff); }

constexpr int kFastMaxD = 4;   // coordinates the small-D matrix-core path takes

struct FastFrame {
  float m[kFastMaxD];   // centre of the box
  float U;              // largest prescaled half-width of the box over the coordinates
  bool ok;              // the expanded form meets the accuracy bound
};
// The decision (ok) is taken with this exact float arithmetic by the fast
// kernels and by the direct-form kernels alike, so exactly one of them runs.
__device__ __forceinline__ FastFrame fast_frame(const FastGuard* g, int D, float scale, float limit) {
  FastFrame f;
  float r2 = 0.0f, U = 0.0f;
  for (int d = 0; d < kFastMaxD; ++d) {
    if (d < D) {
      const float lo = fdec(g->lo[d]), hi = fdec(g->hi[d]);
      f.m[d] = 0.5f * (lo + hi);
      const float h = 0.5f * (hi - lo) * scale;
      r2 += h * h;
      U = fmaxf(U, h);
    } else {
      f.m[d] = 0.0f;
    }
  }
  f.U = U;
  f.ok = r2 <= limit;   // false for NaN
  return f;
}

// Prologue: copy y (and one E-slice of b) into a padded, prescaled,
// interleaved array ypk[j * S + s], S = DP + EP:
//   s <  D        : y[j, s] * yscale
//   D <= s < DP   : 0
//   DP <= s < DP+Ec: b[j, e0 + s - DP] * bscale      (Ec = min(EP, E - e0))
//   remaining     : 0
struct PackArgs {
  const float* y;
  const float* b;     // may be null (arg-K-min)
  float* ypk;
  int64_t N;
  int D, DP, E, EP, e0;
  float yscale, bscale;
  const FastGuard* guard;   // non-null: skip when the fast path is selected
  float fscale;             // prescale of the fast path (for its guard test)
  float flimit;             // the fast path's limit on c R^2 (for its guard test)
  int unit_b;               // b == null: the signal column is bscale (a constant 1 * sign)
};
hipError_t launch_pack(const PackArgs& a, hipStream_t s);

// Direct-form reduction over (i-rows, j-columns) for small D (<= 16).
struct DirectArgs {
  int formula;            // F_*
  int D, DP, E, EP, e0;   // E-slice [e0, e0 + min(EP, E - e0)) of b / out
  int64_t M, N;
  int C;                  // column blocks (block-sparse: column chunks); C == 1 writes the final output
  int64_t jpb;            // j per column block
  const float* x;         // M x D
  const float* ypk;       // N x (DP + EP), from the prologue
  float xscale;           // coordinate scale (1: the direct kernels work in input units)
  float kscale;           // pair scale: Gauss 2^(-kscale d), Laplace 2^(-kscale sqrt d), LSE g' - kscale d
  float gscale;           // gradient: out = -G * gscale; unused otherwise
  float fscale;           // prescale of the small-D fast path (for its guard test)
  float flimit;           // the fast path's limit on c R^2 (for its guard test)
  void* out;              // final output (C == 1)
  float* part;            // partials (C > 1), C x M x W
  int KP, K;              // arg-K-min list length (power of two) and K
  int rows;               // rows per thread of the sums (0: the kernel's default)
  const FastGuard* guard; // non-null: skip when the fast path is selected
  const float* xe;        // F_VJP: row cotangent e, M x E (this call reads its E-slice)
  int accumulate;         // F_VJP with C == 1: add to out instead of storing (E-slices after the first)
  int ext;                // min / max reductions: the kernel takes the min over j of sign * F
  float ext_sign;         // +1 (min) or -1 (max); folded into kscale and the packed b
  int arg;                // min / max: write the index (int32) instead of the value
  int kvalues;            // arg-K-min lists: write the distances (fp32) instead of the indices
  // Block-sparse reductions (nr > 0): row cluster I is rows [rr[2I], rr[2I+1]);
  // its reduction runs over the column ranges cr[2q], cr[2q+1]) for q in
  // [cp[I], cp[I+1]).  bstart[I] is the first workgroup of cluster I (a
  // prefix over clusters of their row-block counts, made on the device).
  int nr;
  const int* rr;
  const int* cp;
  const int* cr;
  const int* bstart;
};
hipError_t launch_direct(const DirectArgs& a, hipStream_t s);
// bstart[0..nr]: prefix sums of ceil(cluster rows / rows_per_block) (one workgroup).
hipError_t launch_range_blocks(const int* rr, int nr, int64_t M, int rows_per_block, int* bstart,
                               hipStream_t s);
// Workgroups a block-sparse launch needs at most (disjoint row ranges).
int64_t range_grid_bound(int nr, int64_t M, int rows_per_block);
int direct_rows_per_thread(int formula, int DP, int EP, int KP);
// Rows per thread for a direct-form call: the default, or 2 for a plain sum
// whose default grid would leave CUs idle (small M).
int direct_sum_rows(int formula, int DP, int EP, int KP, int ext, int64_t M, int64_t N,
                    int num_cus);
int direct_rows_for(const DirectArgs& a);   // rows per lane launch_direct uses for these args
int direct_pad_d(int D);      // DP for a given D, 0 if the direct path has none
int direct_pad_e(int E);      // EP for one E-slice
int knn_pad_k(int K);         // KP for a given K
int partial_width(int formula, int DP, int EP, int KP, int ext);  // W (floats per row per column block)

// Second pass: combine C column-block partials into the final output.
struct CombineArgs {
  int formula;
  int D, DP, E, EP, e0;
  int64_t M;
  int C;
  const float* part;
  void* out;
  float gscale;
  int KP, K;
  int accumulate;   // F_VJP: add to out instead of storing
  int ext;          // min / max partials: (sign * value, index) pairs
  float ext_sign;
  int arg;
  int kvalues;      // arg-K-min: write the distances instead of the indices
  // arg-K-min lists of the large-D kernels: the merged candidates get their
  // direct-form distance sum_d (x_d - y_d)^2 (x: M x rD, y: N x rD) and are
  // ranked again by it; null for the direct kernels' lists
  const float* rx;
  const float* ry;
  int rD;
};
hipError_t launch_combine(const CombineArgs& a, hipStream_t s);

// dst[i, k] = e[i] * src[i, 1 + k] for i < M, k < D (src is M x (1 + D)):
// the x-gradient of the fused value + gradient reduction times a scalar cotangent.
hipError_t launch_scale_rows(const float* src, int64_t M, int D, const float* e, float* dst,
                             hipStream_t s);

// Large-D path (matrix cores).  Prologue: Yop[j][d] = y[j][d] * yop_scale
// (zero for d >= D), ny[j] = nrm_sign * |y_j * coord_scale|^2 (pad_norm for
// the padding columns N <= j < N16), and the signal tiles bpk (16 * EB
// values of b per column, laid out as the B operand of the P . B product).
// Exactness guard of the bf16 arg-K-min kernel.  When every coordinate of x
// and y is an integer with |v| <= kExactMaxAbs and D max|v|^2 <= kExactMaxSum,
// every operand (v and -2 v) is exact in bf16 and every product, partial sum
// and norm is an integer below 2^24, exact in fp32: the bf16 matrix cores then
// give the same squared distances, and so the same ranking and ties, as exact
// arithmetic.  The prologue fills the guard on the device; the fp32 and bf16
// kernels are both launched and each returns at once unless it is selected.
struct ExactGuard {
  unsigned int maxabs;   // bit pattern of max |v| (non-negative floats order as unsigned ints)
  unsigned int nonint;   // non-zero once some coordinate is not an integer (NaN, inf included)
};
constexpr float kExactMaxAbs = 256.0f;
constexpr float kExactMaxSum = 4194304.0f;   // 2^22

__device__ __forceinline__ bool exact_ok(const ExactGuard* g, int D) {
  if (g == nullptr || g->nonint != 0u) return false;
  const float m = __uint_as_float(g->maxabs);
  return m <= kExactMaxAbs && (float)D * m * m <= kExactMaxSum;
}

// Accuracy guard of the large-D expanded form.  With m a centre of y and s =
// sqrt(c) in fp64, the kernels take X = fl32(s (x - m)) and Y = fl32(s (y - m))
// (formed in fp64, one rounding each), the norms nx = -|X|^2 and ny = -|Y|^2
// (+ g' for log-sum-exp) summed in fp64 and rounded once, and
//     T = fl(P + fl(nx + ny)),   P = sum_d 2 Y_d X_d
// accumulated on the matrix cores from zero.  With u = 2^-24 and L = c (max_i
// |x_i - m|^2 + max_j |y_j - m|^2), every pair has |x'|^2 + |y'|^2 <= L and
// sum_d |2 Y_d X_d| <= L, and the error in T = -c |x - y|^2 is at most
//   4 u L    the rounding of the coordinates (|X - Y|^2 against |x' - y'|^2),
//   2 u L    the two norms and their sum,
//   2 u L    the last addition (|T| <= 2 L),
// plus the contraction's own:
//   fp32 (v_mfma_f32_16x16x4_f32 adds its products to the accumulator one at
//   a time, each addition rounded; a product may round too): (D + 1) u L, in
//   all (D + 9) u L;
//   split bf16 (v_mfma_f32_16x16x32_bf16 adds each group of 8 products at
//   once: they are aligned to the largest, the bits below 2^-24 of it are
//   dropped, and the sum is rounded into the accumulator): per group at most
//   7 u max|p| + u |acc|.  The chain of the products hh, hm and mh (3 D / 8
//   groups, |acc| below 1.01 L) adds (3 D / 8 + 7) 1.01 u L, the chain of hl,
//   lh and mm (below 2^-15 of the products) and the dropped ml, lm and ll
//   below 1.1 u L, their sum u L: in all below (0.38 D + 17.2) u L.
// Each kernel runs while its bound, (D + 10) u L and (D / 2 + 18) u L with
// room for the higher-order terms, stays within the budget; beyond it the
// contraction runs in fp64 (mfma_kernel<..., F64>).  The exponentials of T
// keep their relative error ln 2 times it.  The Laplacian forms take
// sqrt(-T), which turns an absolute error e near d = 0 into sqrt(e), and the
// squared distance's sums have no lower bound on d against their normaliser:
// they always run in fp64 (limit < 0).
struct SpreadGuard {
  unsigned int maxx;   // bit pattern of max_i |x_i - m|^2 (non-negative floats order as unsigned)
  unsigned int maxy;   // max_j |y_j - m|^2
};
constexpr double kWideBudget = 1.2e-4;   // log2 units: ln 2 times it is below 1e-4
// the largest L each kernel takes
inline float wide_limit_f32(int D) { return (float)(kWideBudget * 16777216.0 / (D + 10.0)); }
inline float wide_limit_split(int D) { return (float)(kWideBudget * 16777216.0 / (0.5 * D + 18.0)); }
// true: the fp64 contraction does the work (also for a NaN spread)
__device__ __forceinline__ bool wide64(const SpreadGuard* g, float c, float limit) {
  if (g == nullptr) return false;
  const float L = c * (__uint_as_float(g->maxx) + __uint_as_float(g->maxy));
  return !(L <= limit);
}

struct MfmaPackArgs {
  const float* y;
  const float* b;
  int64_t N, N16;
  int D, DP, E, e0, Ec, EB;
  float yop_scale, coord_scale, nrm_sign, pad_norm;
  float* yop;
  float* ny;
  float* bpk;     // null for arg-K-min
  const ExactGuard* exact;   // arg-K-min with the exact path enabled, else null
  unsigned short* ybf;       // bf16 copy of yop (N16 x DP), written instead of yop when exact
  unsigned short* ysp;       // sums on the split path: yop as 3 bf16 planes (N16 x 3 x DP), written
                             // instead of yop
  int unit_b;                // min / max without b: a signal column of ones
  const float* goff;         // log-sum-exp: per-column offset g (N), added to ny times goff_scale
  float goff_scale;
  const float* yc;           // sums and log-sum-exp: a centre (D) subtracted from y, else null
  float* gpk;                // Laplacian log-sum-exp: g' = goff goff_scale per column (N16), else null
  // the fp64 contraction (when the guard selects it): yop and ny in fp64, in
  // the same buffers (sized for it)
  const SpreadGuard* spread;   // null: the fp32 kernels only (arg-K-min)
  float wide_c, wide_limit;
  double yop_scale64, coord_scale64;
  // the split kernel's Gaussian sum at DP <= 128 (unless the guard selects
  // fp64): b as three bf16 planes per 32-column pair in the P . B operand's K
  // order, written to bpk in place of the fp32 tiles (sized for both)
  int bpair;
};
hipError_t launch_mfma_pack(const MfmaPackArgs& a, hipStream_t s);

// A centre of y for the large-D kernels: m = the mean of its first min(N, 256)
// rows (D floats; zeros when N = 0).
hipError_t launch_centre(const float* y, int64_t N, int D, float* m, hipStream_t s);
// Fused Gaussian value + x-gradient for 16 < D <= 256 as one Gaussian sum with
// E (D + 1) signal columns [b_e, b_e (y - m)]: the signal columns [c0, c0 + Ec)
// (N x Ec), and from the sums T (column c in chunk c / 64, stored M x Ec_q at
// T + 64 M q) either the output M x (1 + D) (E = 1) or, for a cotangent e
// (M x E), the vector-Jacobian product M x D.
hipError_t launch_gradx_signal(const float* y, const float* b, int64_t N, int D, int E,
                               const float* m, int c0, int Ec, float* sig, hipStream_t s);
hipError_t launch_gradx_finish(const float* x, int64_t M, int D, const float* m, const float* T,
                               float gscale, float* out, hipStream_t s);
hipError_t launch_vjp_finish(const float* x, int64_t M, int D, int E, const float* m,
                             const float* T, const float* e, float gscale, float* out,
                             hipStream_t s);

struct MfmaArgs {
  int epi;        // 0 Gauss, 1 Laplace, 2 squared distance (sums), 3 arg-K-min, 4 log-sum-exp
                  // (Sinkhorn form), 5 log-sum-exp of the Laplacian, 6..9 min / max of
                  // F b (Gauss, Laplace, squared distance, Sinkhorn form)
  int D, DP, E, e0, EB;
  int64_t M, N16;
  int C;          // column blocks
  int64_t jpb;    // columns per block (multiple of the tile width)
  const float* x;
  float xscale;
  const float* yop;
  const float* ny;
  const float* bpk;
  void* out;      // final output (sums with C == 1)
  float* part;    // sums: C x M x 16 EB; arg-K-min: 4 C x M x 2 KP
  int KP, K;
  const ExactGuard* exact;     // arg-K-min: exact-path guard, or null (fp32 kernel only)
  const unsigned short* ybf;   // arg-K-min: bf16 column operand when exact
  const unsigned short* ysp;   // sums: the split column operand (split kernel), else null
  int64_t N;                   // columns (block-sparse ranges are clamped to it)
  float pad_ny;                // the padding columns' norm (masked columns of a tile)
  // block-sparse pattern (nr = 0: dense), as for the direct kernels; bstart is
  // the workgroup map for the kernels' rows per workgroup
  int nr;
  const int* rr;
  const int* cp;
  const int* cr;
  const int* bstart;
  const float* xc;   // sums and log-sum-exp: the centre (D) subtracted from x, as from y
  const float* gpk;  // Laplacian log-sum-exp: g' per column (N16; padding -infinity)
  float ext_sign;    // min / max (epi 6..9): +1 for min, -1 for max
  const SpreadGuard* spread;   // the guard choosing the fp32 or the fp64 contraction (null: fp32)
  float wide_c, wide_limit;    // c of the prescale, and the limit on L
  double xscale64;             // the row prescale in fp64 (fp64 contraction)
  // one more signal column summed on the vector ALU by the 32x32-tile split
  // sum with 64 columns: its fp32 values per column (N16 + 1 of them, zero
  // from N on), the output column (M floats) and its C x M partials; xskip:
  // the split kernel returns at once (that column was summed with the
  // previous launch; the fp64 contraction still runs when the guard picks it)
  const float* xb;
  float* xout;
  float* xpart;
  int xskip;
};
hipError_t launch_mfma(const MfmaArgs& a, hipStream_t s);
// The same reductions with the contraction in fp64 (runs only when the guard
// selects it; launched beside the fp32 or split kernel, which then return).
hipError_t launch_mfma64(const MfmaArgs& a, hipStream_t s);
int mfma64_rows_per_block(int DP);   // rows per workgroup of the fp64 variant (its bstart map)
// Zero the guard, then fold max |x_i - m|^2 and max |y_j - m|^2 into it.
hipError_t launch_spread(const float* x, int64_t M, const float* y, int64_t N, int D,
                         const float* m, SpreadGuard* g, hipStream_t s);
// counts[0] += 1 when the guard selects the fp64 contraction, counts[1] += 1 (profiling)
hipError_t launch_wide_record(const SpreadGuard* g, float c, float limit, int* counts,
                              hipStream_t s);
// Exact-path prologue: reset the guard, then fold every coordinate of x and y into it.
hipError_t launch_exact_check(const float* x, int64_t M, const float* y, int64_t N, int D,
                              ExactGuard* g, hipStream_t s);
// The bf16 arg-K-min kernel (runs only when the guard allows it); same partial layout as the
// fp32 kernel for the same C and jpb.
hipError_t launch_knn_bf16(const MfmaArgs& a, hipStream_t s);
// Sums with the contraction on the bf16 matrix cores, fp32-accurate (3-way split, 6 products).
hipError_t launch_mfma_split(const MfmaArgs& a, hipStream_t s);
int mfma_pad_d(int D);               // DP for D > 16 (0 if D > 256)
int mfma_tile_cols(int DP);          // columns per LDS tile
int mfma_knn_pad_k(int K);           // list length of the matrix-core arg-K-min kernels
int mfma_rows_per_block(int DP, int KP);
int mfma_split_rows_per_block(int DP, int epi);   // rows per workgroup of the split kernels
// the padded widths at which the log-sum-exp takes the split kernel (32x32 tiles)
inline bool split_lse_dp(int DP) { return DP == 32 || DP == 64 || DP == 128; }
int64_t mfma_row_groups(const MfmaArgs& a, int rows);   // row-block slots of the grid

struct FastPackArgs {
  int epi, D;
  int64_t N, N16;
  const float* y;
  const float* b;     // b (sums, gradient) or g (log-sum-exp)
  float scale;        // prescale sqrt(c) (the guard's decision uses this float)
  double scale64;     // the same prescale in fp64 (the operands are formed in fp64)
  float limit;        // largest c R^2 the fast path takes for this call
  const FastGuard* guard;
  uint4* apk;         // N16 x 4 uint4: 32 bf16 A-operand slots per column
  float4* ex;         // gradient: (b, b v0, b v1, b v2) per column; FAST_SUMV: b's E <= 4 columns
  float* eb;          // sum: b per column
  int E;              // FAST_SUMV: signal columns of b (2..4)
};
hipError_t launch_fast_prologue(const FastPackArgs& a, const float* x, int64_t M, hipStream_t s);

struct FastArgs {
  int epi, D, DP;
  int64_t M, N, N16;
  int C;
  int64_t jpb;        // multiple of 256
  const float* x;
  float scale, gscale;
  double scale64;     // the prescale in fp64 (row operands are formed in fp64)
  float limit;        // largest c R^2 the fast path takes for this call
  const FastGuard* guard;
  const uint4* apk;
  const float4* ex;
  const float* eb;
  void* out;
  float* part;
  int kvalues;        // FAST_MIN, FAST_KNN: write the distances (else the indices)
  int K, KP;          // FAST_KNN: K, and the list length of the output / partial layout
  const float* y;     // FAST_MIN, FAST_KNN: the points (N x D), for the exact final distances
  int E, EP;          // FAST_SUMV: signal columns, and the partial width of the sums' combine
  // block-sparse pattern (nr > 0), as in DirectArgs; bstart counts row
  // blocks of fast_rows_per_block rows
  int nr;
  const int* rr;
  const int* cp;
  const int* cr;
  const int* bstart;
};
hipError_t launch_fast(const FastArgs& a, hipStream_t s);
// counts[0] += 1 when the guard selects the fast path for (D, scale, limit),
// counts[1] += 1 always: which kernel did the work, for the profile.
hipError_t launch_fast_record(const FastGuard* g, int D, float scale, float limit, int* counts,
                              hipStream_t s);
int fast_rows_per_block(int epi, int K);

// Fill out with a constant (N = 0 cases); a kernel, not a memset, so that
// callers may capture it in a graph.
// Latency-bound Gaussian sums (D <= 4, E <= 4, below 2^28 pairs) in one
// launch: rows in blocks of kSumRows, columns in C blocks of jpb <=
// kSumCols read straight into LDS, the pair term on the matrix cores within
// each workgroup's own accuracy bound (else the direct form), and the last
// workgroup of a row block to arrive adding the C partials.
constexpr int kSumRows = 128;
constexpr int kSumCols = 1024;
constexpr int kSumMaxRowBlocks = 16384;   // counters: 64 KB
struct SmallArgs {
  const float* x;
  const float* y;
  const float* b;
  float* out;       // M x E
  float* part;      // C > 1: C x M x E partial sums
  int* count;       // C > 1: one counter per row block, zero between calls
  int64_t M, N;
  int D, E, C, jpb;
  double c64, s64;  // c = log2(e) / (2 sigma^2) and sqrt(c)
  float limit;      // the largest L the matrix-core form takes
};
hipError_t launch_small(const SmallArgs& a, hipStream_t s);

// Block-sparse truncation pattern on the device (k_cluster.hip): grid
// clusters of x and y, their stable sort by label, cluster ranges, and per
// cluster of x the runs of clusters of y within reach.
constexpr int kClusterMaxD = 8;
struct ClusterGrid {
  double origin[kClusterMaxD];
  int64_t dims[kClusterMaxD];
};
struct TruncArgs {
  const uint64_t* ux;        // distinct labels of x (ascending)
  const uint64_t* uy;        // ... of y
  const int32_t* rx;         // cluster ranges of x (2 per cluster)
  const int32_t* ry;         // ... of y
  const int32_t* nx;         // cluster counts (device)
  const int32_t* ny;
  int64_t cap_x;             // clusters of x provided for (M)
  int D;
  double cell, reach2;
  const ClusterGrid* g;
  int32_t* runs;             // per cluster of x: its column ranges (pass 1)
  const int32_t* col_ptr;    // exclusive scan of runs (pass 2)
  int32_t* col_ranges;
  int64_t cap_c;             // column ranges provided for
  unsigned long long* pairs; // kept (i, j) pairs
};
struct ClusterCall {
  const float* x;
  const float* y;
  int64_t M, N;
  int D;
  double cell, reach2;
  int32_t* order_x;
  int32_t* order_y;
  int32_t* row_ranges;   // M x 2 (clusters beyond the count: empty)
  int32_t* col_ptr;      // M + 1
  int32_t* col_ranges;   // col_cap x 2
  int64_t col_cap;
  int64_t* counts;       // 4: clusters of x, column ranges, pairs, overflow
};
size_t cluster_scratch_bytes(int64_t M, int64_t N);
hipError_t build_cluster_pattern(const ClusterCall& c, void* scratch, size_t bytes, hipStream_t s);
// dst[i] = src[index[i]] (inverse: dst[index[i]] = src[i]), rows of `width` floats
hipError_t launch_gather_rows(const float* src, const int32_t* index, int64_t n, int width,
                              int inverse, float* dst, hipStream_t s);

hipError_t launch_fill(float* out, int64_t count, float value, hipStream_t s);
hipError_t launch_fill2(float* out, int64_t count, float v0, float v1, hipStream_t s);

}  // namespace kred
