// Small-D (D <= 4) reductions with the exponent on the bf16 matrix cores.
//
// The direct form of the pair term costs about 6 VALU instructions per pair
// before the exp.  Here the whole exponent T_ij = -c |x_i - y_j|^2 (log2
// units) comes from one v_mfma_f32_16x16x32_bf16 per 16 x 16 block of
// (column j, row i) pairs, which runs alongside the VALU/exp work, so the VALU
// is left with the exp and the reduction itself.
//
// Operands.  With u = sqrt(c) (x - m) and v = sqrt(c) (y - m) for the centre m
// of the joint bounding box of x and y (formed in fp64 from the fp32 inputs),
//     T = 2 <u, v> - |u|^2 - |v|^2.
// U is the largest prescaled half-width of the box, L = c R^2 its squared
// prescaled half-diagonal, and qu the power of two with U <= 255 qu < 2 U.
// Each coordinate is split into three bf16 parts on a common grid:
//     u = uh + um + ul,  uh = qu k (|k| <= 256, exact in bf16),
// um and ul the bf16 roundings of what is left (|u - (uh + um + ul)| <= 2^-19 qu);
// V = 2 v the same way with the grid 2 qu.  Every leading product Vh uh is
// then a multiple of q = 2 qu^2 no larger than 2^16 q.  The row norm |u~|^2 and
// the column norm w = -|v~|^2 (+ g' = g log2(e) for the log-sum-exp) of the
// represented coordinates are computed in fp64; their leading parts are
// rounded to multiples of max(q, their bf16 spacing), so they too are exact
// in bf16 and multiples of q.
//
// K slots (A: column side, B: row side).  Group 0 (slots 0..7) holds every
// term of size O(L), all multiples of q, so their sum is exact whatever order
// or width the matrix core adds them in (partial sums stay below 2^20 q):
//     slot d < D: (Vh_d, uh_d);  slot 4: (w_h, 1);  slot 5: (1, -h) with h the
//     leading part of |u~|^2 (+h, rounded up, for the nearest distances).
// From slot 8 on, per coordinate d, the products (Vh,um), (Vm,uh), (Vh,ul),
// (Vl,uh), (Vm,um), (Vm,ul), (Vl,um) (D <= 3: seven per coordinate, slots
// 8 + 7d ..; D = 4: the first five, slots 8 + 5d ..), then the column norm's
// three trailing parts with B = 1 (slots 29..31; D = 4: 28..30).  The row
// norm's remainder r = |u~|^2 - h stays out of the product: the matrix core
// returns T' = T~ + r, and the epilogue scales the row's sums by 2^-r (the
// log-sum-exp subtracts r).  The nearest-neighbour forms need no correction:
// with h rounded up, T' = |u~ - v~|^2 + (h - |u~|^2) ranks like the distance.
//
// Error of T' - r against -c |x - y|^2 in log2 units, for a pair with
// t = c |x - y|^2, every rounding at its largest:
//   representation of u and v   sqrt(D t) U 2^-24
//   dropped products            D <= 3: (Vl, ul), below D L 2^-33;
//                               D = 4: also (Vm, ul) and (Vl, um), below L 2^-21
//   norms                       column: 4 parts, below 2^-35 |w|; row: exact
//   fp32 accumulation           group 0 is exact; groups 1..3 hold terms of
//                               total size M1 <= sqrt(D) L / 64 + L / 256, so
//                               the 7 roundings inside group 1 are below
//                               2^-24 M1 each, and the 3 that add the groups
//                               below 2^-24 (t + L / 256 + 2 M1) each.
// At D <= 3 and L = 2048 the sum is below 1.2e-4 for every t <= 126, so a
// term's relative error (ln 2 times that) stays below 8e-5; at D = 4 and
// L = 128 below 7.5e-5 (the dropped products dominate).  Typical errors are
// about 40 times smaller (2e-6 at L = 2000 on uniform data).  kFastLimit3 and
// kFastLimit4 keep inputs there: the prologue computes the box on the device
// and the kernels fall back to the direct form beyond the limit (no host
// synchronisation).
//
// The nearest-neighbour variants (FAST_MIN, FAST_KNN) flip every sign, so the
// matrix core returns the squared distance (plus the row constant h - |u~|^2)
// with c = 1: minimum and arg-minimum then need no exp at all.  They rank by
// it and recompute the final candidates' distances in the direct form.
//
// Lane layout of v_mfma_f32_16x16x32_bf16 (lane l = 16 g + li): A: lane
// supplies A[li][8g .. 8g+7]; B: lane supplies B[8g .. 8g+7][li]; D: lane holds
// D[4g + r][li].  With A = columns and B = rows, lane l gets T for row li and
// columns 4g + r of the block.
#include "kred_internal.h"

#include <climits>

namespace kred {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int TJF = 256;             // columns per LDS tile
constexpr float kRescaleF = 32.0f;   // log-sum-exp rescale threshold (log2 units)
constexpr double kLog2eD = 1.4426950408889634;

// Products beyond (h, h) per coordinate as (column part, row part), 0 = h,
// 1 = m, 2 = l: D <= 3 takes all seven, D = 4 the first five.
constexpr int kProdA[7] = {0, 1, 0, 2, 1, 1, 2};
constexpr int kProdB[7] = {1, 0, 2, 0, 1, 2, 1};
template <bool D4>
struct Slots {
  static constexpr int per = D4 ? 5 : 7;      // products beyond (h, h) per coordinate
  static constexpr int tail = D4 ? 28 : 29;   // the column norm's three trailing parts
};
constexpr int kSlotW = 4;   // leading part of the column norm (B = 1)
constexpr int kSlotH = 5;   // leading part of the row norm (A = 1)

// The grid of the leading parts: the power of two qu with U (1 + 2^-10) <= 255 qu
// (the margin covers the fp32 rounding of the box), so |u| / qu <= 256.
__device__ __forceinline__ double fast_quantum(float U) {
  int e;
  (void)frexp((double)U * (1.0 + 1.0 / 1024.0) / 255.0, &e);
  return ldexp(1.0, e);
}

__device__ __forceinline__ __bf16 to_bf16(double v) { return (__bf16)(float)v; }
__device__ __forceinline__ double of_bf16(__bf16 v) { return (double)(float)v; }

// v = h + m + l: h = q rint(v / q) (|v| <= 256 q, exact in bf16), m and l the
// bf16 roundings of what is left.  Returns h + m + l (exact in fp64).
__device__ __forceinline__ double split_fixed(double v, double q, __bf16& h, __bf16& m, __bf16& l) {
  const double hv = q * rint(v / q);
  h = to_bf16(hv);
  double r = v - hv;
  m = to_bf16(r);
  r -= of_bf16(m);
  l = to_bf16(r);
  return hv + of_bf16(m) + of_bf16(l);
}

// Leading part of a norm: the nearest multiple of max(q, the bf16 spacing at
// w) (up: the next one at or above w), exact in bf16 and a multiple of q.
__device__ __forceinline__ double norm_head(double w, double q, bool up) {
  int e;
  (void)frexp(w, &e);   // |w| in [2^(e-1), 2^e)
  const double Q = w == 0.0 ? q : fmax(q, ldexp(1.0, e - 8));
  return Q * (up ? ceil(w / Q) : rint(w / Q));
}

__global__ void guard_init_kernel(FastGuard* g) {
  const int t = threadIdx.x;
  if (t < 4) {
    g->lo[t] = fenc(__builtin_inff());
    g->hi[t] = fenc(-__builtin_inff());
  }
}

// Joint bounding box of x (M x D) and y (N x D): per-block reduction (wave
// shuffles, then LDS), then one atomic per block and coordinate.
__global__ __launch_bounds__(256) void bounds_kernel(const float* __restrict__ x, int64_t M,
                                                     const float* __restrict__ y, int64_t N, int D,
                                                     FastGuard* g) {
  __shared__ float red[2][kFastMaxD][4];
  float lo[kFastMaxD], hi[kFastMaxD];
#pragma unroll
  for (int d = 0; d < kFastMaxD; ++d) {
    lo[d] = __builtin_inff();
    hi[d] = -__builtin_inff();
  }
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < M + N; t += stride) {
    const float* p = t < M ? x + t * D : y + (t - M) * D;
    for (int d = 0; d < D; ++d) {
      lo[d] = fminf(lo[d], p[d]);
      hi[d] = fmaxf(hi[d], p[d]);
    }
  }
  const int wave = threadIdx.x >> 6;
  for (int d = 0; d < kFastMaxD; ++d) {
    float a = lo[d], b = hi[d];
    for (int o = 32; o > 0; o >>= 1) {
      a = fminf(a, __shfl_xor(a, o));
      b = fmaxf(b, __shfl_xor(b, o));
    }
    if ((threadIdx.x & 63) == 0) {
      red[0][d][wave] = a;
      red[1][d][wave] = b;
    }
  }
  __syncthreads();
  if (threadIdx.x < D) {
    const int d = threadIdx.x;
    const float a = fminf(fminf(red[0][d][0], red[0][d][1]), fminf(red[0][d][2], red[0][d][3]));
    const float b = fmaxf(fmaxf(red[1][d][0], red[1][d][1]), fmaxf(red[1][d][2], red[1][d][3]));
    atomicMin(&g->lo[d], fenc(a));
    atomicMax(&g->hi[d], fenc(b));
  }
}

// Column side of one column j < N: its 32 A slots, and the represented
// prescaled coordinates v~ (for the gradient's extras).  g2: g' of the
// log-sum-exp (else 0).
template <bool D4>
__device__ __forceinline__ void pack_column(const FastPackArgs& a, const FastFrame& fr, double qu,
                                            int64_t j, bool nearest, double g2, __bf16 (&s)[32],
                                            float (&vt)[kFastMaxD]) {
  using S = Slots<D4>;
  double nv = 0.0;
#pragma unroll
  for (int d = 0; d < kFastMaxD; ++d) {
    if (D4 || d < a.D) {
      const double v = ((double)a.y[j * a.D + d] - (double)fr.m[d]) * a.scale64;
      __bf16 p[3];
      // V = 2 v for the sums, -2 v for the nearest distances (T = +|u - v|^2)
      const double V = split_fixed((nearest ? -2.0 : 2.0) * v, 2.0 * qu, p[0], p[1], p[2]);
      nv = fma(0.5 * V, 0.5 * V, nv);
      vt[d] = (float)(nearest ? -0.5 * V : 0.5 * V);
      s[d] = p[0];
#pragma unroll
      for (int i = 0; i < S::per; ++i) s[8 + S::per * d + i] = p[kProdA[i]];
    }
  }
  const double w = (nearest ? nv : -nv) + g2;
  const double h = norm_head(w, 2.0 * qu * qu, false);
  s[kSlotW] = to_bf16(h);
  s[kSlotH] = (__bf16)1.0f;
  double r = w - h;
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    s[S::tail + k] = to_bf16(r);
    r -= of_bf16(s[S::tail + k]);
  }
}

// Column-side packing: A row (32 bf16) and per-column extras.
//   sum:   eb = b                   gradx: ex = (b, b v~0, b v~1, b v~2)
//   sumv:  ex = b's E <= 4 columns  lse:   g' = g log2(e) joins the column norm
// Padding columns (N <= j < N16) get zero A rows and zero extras.
__global__ __launch_bounds__(256) void fast_pack_kernel(FastPackArgs a) {
  const FastFrame fr = fast_frame(a.guard, a.D, a.scale, a.limit);
  if (!fr.ok) return;
  const double qu = fast_quantum(fr.U);
  const bool nearest = a.epi == FAST_MIN || a.epi == FAST_KNN;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < a.N16; j += stride) {
    __bf16 s[32];
#pragma unroll
    for (int k = 0; k < 32; ++k) s[k] = (__bf16)0.0f;
    float4 ex = {0.f, 0.f, 0.f, 0.f};
    if (j < a.N) {
      float vt[kFastMaxD] = {0.f, 0.f, 0.f, 0.f};
      const float bj = (nearest || a.epi == FAST_SUMV) ? 0.0f : a.b[j];   // MIN, KNN read no b
      const double g2 = a.epi == FAST_LSE ? (double)bj * kLog2eD : 0.0;
      if (a.D == 4) pack_column<true>(a, fr, qu, j, nearest, g2, s, vt);
      else pack_column<false>(a, fr, qu, j, nearest, g2, s, vt);
      if (a.epi == FAST_SUMV) {
        float bv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) bv[e] = e < a.E ? a.b[j * a.E + e] : 0.0f;
        ex = float4{bv[0], bv[1], bv[2], bv[3]};
      } else if (a.epi == FAST_GRADX) {
        ex = float4{bj, bj * vt[0], bj * vt[1], bj * vt[2]};
      } else if (a.epi == FAST_SUM) {
        ex.x = bj;
      }
    }
    uint4 w[4];
    __builtin_memcpy(w, s, 64);
#pragma unroll
    for (int q = 0; q < 4; ++q) a.apk[j * 4 + q] = w[q];
    if (a.epi == FAST_GRADX || a.epi == FAST_SUMV) a.ex[j] = ex;
    else if (a.epi == FAST_SUM) a.eb[j] = ex.x;
  }
}

// Row side of one row: its 32 B slots from the centred, prescaled coordinates
// u (fp64), the represented coordinates u~ (fp32, for the gradient), and the
// row norm's remainder r = |u~|^2 - h left out of the product.
template <bool D4>
__device__ __forceinline__ double row_slots(const double (&u)[kFastMaxD], int D, double qu,
                                            bool nearest, __bf16 (&s)[32], float (&ut)[kFastMaxD]) {
  using S = Slots<D4>;
#pragma unroll
  for (int k = 0; k < 32; ++k) s[k] = (__bf16)0.0f;
  double nu = 0.0;
#pragma unroll
  for (int d = 0; d < kFastMaxD; ++d) {
    ut[d] = 0.0f;
    if (D4 || d < D) {
      __bf16 p[3];
      const double ud = split_fixed(u[d], qu, p[0], p[1], p[2]);
      nu = fma(ud, ud, nu);
      ut[d] = (float)ud;
      s[d] = p[0];
#pragma unroll
      for (int i = 0; i < S::per; ++i) s[8 + S::per * d + i] = p[kProdB[i]];
    }
  }
  const double h = norm_head(nu, 2.0 * qu * qu, nearest);
  s[kSlotW] = (__bf16)1.0f;
  s[kSlotH] = to_bf16(nearest ? h : -h);
#pragma unroll
  for (int k = 0; k < 3; ++k) s[S::tail + k] = (__bf16)1.0f;
  return nu - h;
}

// Row-side B operand: this lane's 8 K slots (8g .. 8g+7) for its row, and the
// row norm's remainder (see row_slots).
__device__ __forceinline__ bf16x8 row_operand(const double (&u)[kFastMaxD], int D, int g, double qu,
                                               bool nearest, double* rem, float (&ut)[kFastMaxD]) {
  __bf16 s[32];
  *rem = D == 4 ? row_slots<true>(u, D, qu, nearest, s, ut) : row_slots<false>(u, D, qu, nearest, s, ut);
  bf16x8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = s[8 * g + e];
  return o;
}

// Insert (d, j) into the ascending list (dk, jk): entries arrive in column
// order, so equal distances keep the earlier entry first.  Entry p becomes
// dk[p-1], d or itself: the median of (dk[p-1], d, dk[p]) for a sorted list.
template <int KL>
__device__ __forceinline__ void list_insert(float (&dk)[KL], int (&jk)[KL], float d, int j) {
  bool lt[KL];
#pragma unroll
  for (int p = 0; p < KL; ++p) lt[p] = d < dk[p];
#pragma unroll
  for (int p = KL - 1; p > 0; --p) {
    dk[p] = __builtin_amdgcn_fmed3f(dk[p - 1], d, dk[p]);
    jk[p] = lt[p - 1] ? jk[p - 1] : (lt[p] ? j : jk[p]);
  }
  dk[0] = lt[0] ? d : dk[0];
  jk[0] = lt[0] ? j : jk[0];
}

// The same, ordered by (distance, index): for merging lists of different lanes.
template <int KL>
__device__ __forceinline__ void list_insert_lex(float (&dk)[KL], int (&jk)[KL], float d, int j) {
  bool lt[KL];
#pragma unroll
  for (int p = 0; p < KL; ++p) lt[p] = d < dk[p] || (d == dk[p] && j < jk[p]);
#pragma unroll
  for (int p = KL - 1; p > 0; --p) {
    dk[p] = lt[p - 1] ? dk[p - 1] : (lt[p] ? d : dk[p]);
    jk[p] = lt[p - 1] ? jk[p - 1] : (lt[p] ? j : jk[p]);
  }
  dk[0] = lt[0] ? d : dk[0];
  jk[0] = lt[0] ? j : jk[0];
}

// EPI: FAST_SUM (Gauss, E = 1), FAST_GRADX, FAST_LSE, FAST_MIN, FAST_KNN, and
// FAST_SUMV (Gauss, 2 <= E <= 4: the gradient's four accumulators on b's columns).

// KV (FAST_MIN): write the distance (else the index).  KL (FAST_KNN): the
// length of each lane's sorted list.
//
// Waves per SIMD: the log-sum-exp form and the K-lists up to K = 12 are
// compiled for 4.  Their natural allocations (131 to 142 VGPRs) would give 3;
// held to 128 they spill 12 to 52 bytes per lane, and the fourth wave pays
// (1e6 x 1e6, D = 3: Sinkhorn log-sum-exp 117.9 -> 113.8 ms, 4 nearest
// 78.4 -> 63.6 ms, 12 nearest 117.8 -> 109.3 ms).  For the gradient the same
// hold spills 92 bytes and loses (154 -> 167 ms), and for 16 nearest it
// loses too (127 -> 188 ms), so the other forms keep the compiler's choice.
constexpr int fast_waves(int EPI, int KL) {
  return (EPI == FAST_LSE || (EPI == FAST_KNN && KL <= 12)) ? 4 : 1;
}

template <int EPI, int RB, bool KV = false, int KL = 1>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(fast_waves(EPI, KL))))
void fast_kernel(FastArgs a) {
  constexpr bool kLse = EPI == FAST_LSE;
  constexpr bool kKnn = EPI == FAST_KNN;
  constexpr bool kMin = EPI == FAST_MIN;
  __shared__ uint4 As[2][TJF * 4];
  constexpr bool kVec = EPI == FAST_GRADX || EPI == FAST_SUMV;
  __shared__ float4 Xs[2][kVec ? TJF : 1];   // (b, b v) or b's columns, per column
  __shared__ float4 Bq[2][EPI == FAST_SUM ? TJF / 4 : 1];  // b per column, 4 to a float4
  // per row of the workgroup: the row norm's remainder (sums, log-sum-exp)
  // and the represented coordinates (gradient), from the set-up to the end
  constexpr bool kRem = !kMin && !kKnn;
  __shared__ float Rs[kRem ? 64 * RB : 1];
  __shared__ float Us[EPI == FAST_GRADX ? 3 : 1][EPI == FAST_GRADX ? 64 * RB : 1];

  const FastFrame fr = fast_frame(a.guard, a.D, a.scale, a.limit);
  if (!fr.ok) return;
  const double qu = fast_quantum(fr.U);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, li = lane & 15, g = lane >> 4;
  const int c = blockIdx.x % a.C;
  const int64_t rbk = blockIdx.x / a.C;
  // Dense: row block rbk and column block c.  Block-sparse: a row block of
  // row cluster I and chunk c of its column ranges (the chunk's window
  // [w0, w1) counts columns in the ranges' concatenated order).
  int64_t row0 = rbk * (64 * RB), row_end = a.M;
  int64_t w0 = (int64_t)c * a.jpb, w1 = min(a.N16, w0 + a.jpb);
  const int* cr = nullptr;
  int nrange = 0;
  if (a.nr > 0) {
    const int blk = (int)rbk;
    if (blk >= a.bstart[a.nr]) return;   // a spare workgroup of the grid bound
    int lo = 0, hi = a.nr - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (a.bstart[mid] <= blk) lo = mid;
      else hi = mid - 1;
    }
    const int64_t r0 = min(max((int64_t)a.rr[2 * lo], (int64_t)0), a.M);
    row_end = min(max((int64_t)a.rr[2 * lo + 1], r0), a.M);
    row0 = r0 + (int64_t)(blk - a.bstart[lo]) * (64 * RB);
    cr = a.cr + 2 * (int64_t)a.cp[lo];
    nrange = a.cp[lo + 1] - a.cp[lo];
    int64_t L = 0;
    for (int q = 0; q < nrange; ++q) {
      const int64_t js = min(max((int64_t)cr[2 * q], (int64_t)0), a.N);
      L += min(max((int64_t)cr[2 * q + 1], js), a.N) - js;
    }
    w0 = L * c / a.C;
    w1 = L * (c + 1) / a.C;
  }
  const int64_t i0 = row0 + wave * (16 * RB);

  // The row's centred, prescaled coordinates in fp64, its B operand, and the
  // row norm's remainder r left out of the product (row_slots); the epilogue
  // forms them again rather than keeping them live through the column loop.
  auto row_coords = [&](int64_t row, double (&u)[kFastMaxD]) __attribute__((always_inline)) {
#pragma unroll
    for (int d = 0; d < kFastMaxD; ++d)
      u[d] = (row < row_end && d < a.D) ? ((double)a.x[row * a.D + d] - (double)fr.m[d]) * a.scale64 : 0.0;
  };
  bf16x8 xb[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    double u[kFastMaxD], rem;
    float ut[kFastMaxD];
    row_coords(i0 + 16 * rb + li, u);
    xb[rb] = row_operand(u, a.D, g, qu, kMin || kKnn, &rem, ut);
    const int rs = wave * (16 * RB) + 16 * rb + li;
    if constexpr (kRem) {
      if (g == 0) Rs[rs] = (float)rem;
    }
    if constexpr (EPI == FAST_GRADX) {
      if (g == 0) {
#pragma unroll
        for (int d = 0; d < 3; ++d) Us[d][rs] = ut[d];
      }
    }
    // one row block at a time: interleaved, the fp64 set-up of all four would
    // set the kernel's register count
    __builtin_amdgcn_sched_barrier(0);
  }
  // per lane: sums over its columns (4 g + r of every block) for row li;
  // MIN: the smallest distance (as its int bits, exact order for d >= 0) and its column
  // MIN: per lane its smallest expanded-form distance (int bits) and the tile
  // [btile, bend) where it last improved; that tile's columns of the lane get
  // their direct-form distance at the end (see exact_d)
  int best[RB], btile[RB], bend[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    best[rb] = INT_MAX;
    btile[rb] = INT_MAX;
    bend[rb] = 0;
  }
  // KNN: per lane and row block a sorted list of (distance, column) over the
  // lane's columns, and the row's shared filter (see refresh_filter)
  float dk[RB][KL];
  int jk[RB][KL];
  int thi[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    thi[rb] = __float_as_int(__builtin_inff());
#pragma unroll
    for (int p = 0; p < KL; ++p) {
      dk[rb][p] = __builtin_inff();
      jk[rb][p] = INT_MAX;
    }
  }
  // Any value with at least KL of the row's candidates at or below it bounds
  // the row's K-th nearest here (K <= KL): the smaller of the 4 lane groups'
  // smallest KL-th value and their largest ceil(KL/4)-th value.  Ties pass.
  // The test runs on the bit patterns as signed integers: for values >= 0
  // that is the float order, and a negative value (a tiny distance that
  // rounding pushed below zero) reads as smaller than every non-negative one;
  // a negative bound is raised to +0, so the test only ever passes more
  // columns than the float test would.
  auto refresh_filter = [&]() {
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      float v = dk[rb][KL - 1];
      v = fminf(v, __shfl_xor(v, 16));
      v = fminf(v, __shfl_xor(v, 32));
      float u = dk[rb][(KL + 3) / 4 - 1];
      u = fmaxf(u, __shfl_xor(u, 16));
      u = fmaxf(u, __shfl_xor(u, 32));
      thi[rb] = max(__float_as_int(fminf(v, u)), 0);
    }
  };
  float acc[RB][4], tot[RB][4], mref[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[rb][q] = tot[rb][q] = 0.0f;
    mref[rb] = -__builtin_inff();
  }

  uint4 sa[4];
  float4 sx;
  float sb;
  int64_t j1 = 0;   // end of the column range being streamed (columns beyond it read as zero)
  auto fetch = [&](int64_t jt) {
    const int ncol = (int)min((int64_t)TJF, j1 - jt);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int f = tid + q * 256;
      sa[q] = (f / 4 < ncol) ? a.apk[jt * 4 + f] : uint4{0u, 0u, 0u, 0u};
    }
    if constexpr (kVec) sx = (tid < ncol) ? a.ex[jt + tid] : float4{0.f, 0.f, 0.f, 0.f};
    if constexpr (EPI == FAST_SUM) sb = (tid < ncol) ? a.eb[jt + tid] : 0.0f;
  };
  auto put = [&](int buf) {
#pragma unroll
    for (int q = 0; q < 4; ++q) As[buf][tid + q * 256] = sa[q];
    if constexpr (kVec) Xs[buf][tid] = sx;
    if constexpr (EPI == FAST_SUM) reinterpret_cast<float*>(&Bq[buf][0])[tid] = sb;
  };
  auto a_operand = [&](int buf, int blk) {
    const uint4 av = As[buf][(blk * 16 + li) * 4 + g];
    bf16x8 am;
    __builtin_memcpy(&am, &av, 16);
    return am;
  };
  // Stream the columns [j0, j1) in tiles.  Columns past j1 load as zero rows,
  // which add nothing to the sums; the log-sum-exp masks them explicitly.
  // (always inlined: it is called from two sites, and an outlined copy would
  // keep the per-lane lists and sums in scratch memory)
  auto run_columns = [&](int64_t j0, int64_t jend) __attribute__((always_inline)) {
    j1 = jend;
    const int64_t jlim = min(j1, a.N);
    const int64_t ntiles = (j1 - j0 + TJF - 1) / TJF;
    if (ntiles > 0) {
      fetch(j0);
      put(0);
    }
    __syncthreads();
    for (int64_t t = 0; t < ntiles; ++t) {
      const int64_t jt = j0 + t * TJF;
      const int buf = (int)(t & 1);
      const int nblk = (int)((min((int64_t)TJF, j1 - jt) + 15) / 16);
      if (t + 1 < ntiles) fetch(jt + TJF);
      if constexpr (kKnn) {
        refresh_filter();
        // the lane's 4 distances of each row block.  Full blocks first, then
        // the range's last block if columns past its end (zero A rows) must
        // read as +infinity.  All products and filter tests come before the
        // first branch.
        const bool ragged = jt + 16 * nblk > jlim;
        const int nfull = ragged ? nblk - 1 : nblk;
        auto knn_block = [&](int blk, bool masked) __attribute__((always_inline)) {
          const bf16x8 am = a_operand(buf, blk);
          const int64_t jb = jt + blk * 16 + 4 * g;
          float dd[RB][4];
          bool any[RB];
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            const f4 T = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, xb[rb], f4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
#pragma unroll
            for (int r = 0; r < 4; ++r) dd[rb][r] = (!masked || jb + r < jlim) ? T[r] : __builtin_inff();
          }
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            const int m = min(min(__float_as_int(dd[rb][0]), __float_as_int(dd[rb][1])),
                              min(__float_as_int(dd[rb][2]), __float_as_int(dd[rb][3])));
            any[rb] = m <= thi[rb];
          }
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            if (__builtin_expect(any[rb], 0)) {
#pragma unroll
              for (int r = 0; r < 4; ++r)
                if (dd[rb][r] < dk[rb][KL - 1]) list_insert<KL>(dk[rb], jk[rb], dd[rb][r], (int)(jb + r));
            }
          }
        };
        for (int blk = 0; blk < nfull; ++blk) knn_block(blk, false);
        if (ragged) knn_block(nblk - 1, true);
      } else if constexpr (kMin) {
        // d for the lane's columns 4g + r of each block.  Full blocks first,
        // then the range's last block if columns past its end (zero A rows,
        // d = 0) must be masked; each MFMA is followed by straight-line
        // reads of its result, with no branch in between.
        const bool ragged = jt + 16 * nblk > jlim;
        const int nfull = ragged ? nblk - 1 : nblk;
        int before[RB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) before[rb] = best[rb];
        auto take = [&](int rb, int64_t jb, const int (&d)[4]) {
          best[rb] = min(best[rb], min(min(min(d[0], d[1]), d[2]), d[3]));
        };
        for (int blk = 0; blk < nfull; ++blk) {
          const bf16x8 am = a_operand(buf, blk);
          const int64_t jb = jt + blk * 16 + 4 * g;
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            const f4 T = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, xb[rb], f4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
            const int d[4] = {__float_as_int(T[0]), __float_as_int(T[1]), __float_as_int(T[2]),
                              __float_as_int(T[3])};
            take(rb, jb, d);
          }
        }
        if (ragged) {
          const int blk = nblk - 1;
          const bf16x8 am = a_operand(buf, blk);
          const int64_t jb = jt + blk * 16 + 4 * g;
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            const f4 T = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, xb[rb], f4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
            const int d[4] = {jb + 0 < jlim ? __float_as_int(T[0]) : INT_MAX,
                              jb + 1 < jlim ? __float_as_int(T[1]) : INT_MAX,
                              jb + 2 < jlim ? __float_as_int(T[2]) : INT_MAX,
                              jb + 3 < jlim ? __float_as_int(T[3]) : INT_MAX};
            take(rb, jb, d);
          }
        }
        // a strictly smaller value in this tile: remember the tile (the
        // earliest such tile keeps ties)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          const bool lt = best[rb] < before[rb];
          btile[rb] = lt ? (int)jt : btile[rb];
          bend[rb] = lt ? (int)min(jt + TJF, jlim) : bend[rb];
        }
      } else if constexpr (!kLse) {
        // Padding columns have zero extras, so they add nothing: no masking.
        for (int blk = 0; blk < nblk; ++blk) {
          const bf16x8 am = a_operand(buf, blk);
          float4 xv[4];
          float4 bq;
          if constexpr (EPI == FAST_SUM) {
            bq = Bq[buf][blk * 4 + g];   // b of columns 4g .. 4g+3 of the block
          } else {
#pragma unroll
            for (int r = 0; r < 4; ++r) xv[r] = Xs[buf][blk * 16 + 4 * g + r];
          }
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            const f4 T = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, xb[rb], f4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
            if constexpr (EPI == FAST_SUM) {
              acc[rb][0] = __builtin_fmaf(__builtin_amdgcn_exp2f(T[0]), bq.x, acc[rb][0]);
              acc[rb][1] = __builtin_fmaf(__builtin_amdgcn_exp2f(T[1]), bq.y, acc[rb][1]);
              acc[rb][2] = __builtin_fmaf(__builtin_amdgcn_exp2f(T[2]), bq.z, acc[rb][2]);
              acc[rb][3] = __builtin_fmaf(__builtin_amdgcn_exp2f(T[3]), bq.w, acc[rb][3]);
            } else {
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const float k = __builtin_amdgcn_exp2f(T[r]);
                acc[rb][0] = __builtin_fmaf(k, xv[r].x, acc[rb][0]);
                acc[rb][1] = __builtin_fmaf(k, xv[r].y, acc[rb][1]);
                acc[rb][2] = __builtin_fmaf(k, xv[r].z, acc[rb][2]);
                acc[rb][3] = __builtin_fmaf(k, xv[r].w, acc[rb][3]);
              }
            }
          }
        }
      } else {
        // Fast path: the running reference enters the matrix product as its C
        // operand, so the MFMA returns u = T - m directly; a running maximum of u
        // over the tile tells afterwards whether any term needed a rescale.
        const bool ragged = jt + 16 * nblk > jlim;   // columns past the range must be masked
        // The maximum is taken over the bit patterns as signed integers: that
        // orders non-negative floats correctly and puts every negative one
        // below them, which is all the test against the threshold needs (and
        // it avoids the NaN quieting a float max would add per operand).
        int run[RB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) run[rb] = INT_MIN;
        if (!ragged) {
          f4 negm[RB];
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) negm[rb] = f4{-mref[rb], -mref[rb], -mref[rb], -mref[rb]};
          for (int blk = 0; blk < nblk; ++blk) {
            const bf16x8 am = a_operand(buf, blk);
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
              const f4 u = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, xb[rb], negm[rb], 0, 0, 0);
              run[rb] = max(max(run[rb], __float_as_int(u[0])), __float_as_int(u[1]));
              run[rb] = max(max(run[rb], __float_as_int(u[2])), __float_as_int(u[3]));
              acc[rb][0] += (__builtin_amdgcn_exp2f(u[0]) + __builtin_amdgcn_exp2f(u[1])) +
                            (__builtin_amdgcn_exp2f(u[2]) + __builtin_amdgcn_exp2f(u[3]));
            }
          }
        }
        bool need[RB], redo = false;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          need[rb] = ragged || run[rb] > __float_as_int(kRescaleF);
          redo |= need[rb];
        }
        if (__any(redo)) {
          // Rare (a new running maximum, the first tile, or padding columns): the
          // whole wave recomputes the tile; lanes that need it redo their sums
          // term by term with rescaling and masking.
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            if (need[rb]) acc[rb][0] = 0.0f;
          for (int blk = 0; blk < nblk; ++blk) {
            const bf16x8 am = a_operand(buf, blk);
            const int64_t jb = jt + blk * 16 + 4 * g;
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
              const f4 T = __builtin_amdgcn_mfma_f32_16x16x32_bf16(am, xb[rb], f4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
              if (!need[rb]) continue;
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                if (jb + r >= jlim) continue;
                float d = T[r] - mref[rb];
                if (d > kRescaleF) {
                  const float f = __builtin_amdgcn_exp2f(-d);
                  acc[rb][0] *= f;
                  tot[rb][0] *= f;
                  mref[rb] = T[r];
                  d = 0.0f;
                }
                acc[rb][0] += __builtin_amdgcn_exp2f(d);
              }
            }
          }
        }
      }
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          tot[rb][q] += acc[rb][q];
          acc[rb][q] = 0.0f;
        }
      if (t + 1 < ntiles) put((int)((t + 1) & 1));
      __syncthreads();
    }
  };
  if (nrange == 0) {
    if (a.nr == 0) run_columns(w0, w1);
  } else {
    int64_t off = 0;
    for (int q = 0; q < nrange && off < w1; ++q) {
      const int64_t js = min(max((int64_t)cr[2 * q], (int64_t)0), a.N);
      const int64_t len = min(max((int64_t)cr[2 * q + 1], js), a.N) - js;
      const int64_t a0 = max(w0 - off, (int64_t)0), a1 = min(w1 - off, len);
      off += len;
      if (a1 > a0) run_columns(js + a0, js + a1);
    }
  }

  // The expanded form's distance carries an absolute error of about 2^-24 R^2
  // (R the box's half-diagonal), large against a close neighbour's distance;
  // it only ranks.  The final candidates get their distance in the direct
  // form, sum_d (x_d - y_d)^2, which is accurate relative to itself (and
  // exact on integer coordinates), and are ranked again by it.
  auto load_row = [&](int64_t row, bool live_row, float (&xr)[kFastMaxD]) __attribute__((always_inline)) {
#pragma unroll
    for (int d = 0; d < kFastMaxD; ++d) xr[d] = (live_row && d < a.D) ? a.x[row * a.D + d] : 0.0f;
  };
  auto exact_d = [&](const float (&xr)[kFastMaxD], int j) __attribute__((always_inline)) {
    float s = 0.0f;
#pragma unroll
    for (int d = 0; d < kFastMaxD; ++d)
      if (d < a.D) {
        const float t = xr[d] - a.y[(int64_t)j * a.D + d];
        s = __builtin_fmaf(t, t, s);
      }
    return s;
  };

  // KNN: lane group 0 gathers the four groups' candidates (4 KL per row, each
  // group's own KL nearest by the expanded form) and keeps the K nearest by
  // the direct-form distance, ordered by (distance, index) so that ties keep
  // the lower index; every lane takes part in the shuffles.  The lists come
  // in by reference, so that every index is a compile-time constant (a
  // runtime row-block index would put them in scratch memory).
  auto knn_out = [&](const float (&dl)[KL], const int (&jl)[KL], int64_t row, bool live_row)
      __attribute__((always_inline)) {
    (void)dl;
    float xr[kFastMaxD];
    load_row(row, live_row, xr);
    float md[16];
    int mj[16];
#pragma unroll
    for (int p = 0; p < 16; ++p) {
      md[p] = __builtin_inff();
      mj[p] = INT_MAX;
    }
#pragma unroll
    for (int src = 0; src <= 48; src += 16) {
#pragma unroll
      for (int p = 0; p < KL; ++p) {
        const int j2 = src == 0 ? jl[p] : __shfl(jl[p], li + src);
        if (g == 0 && live_row && j2 != INT_MAX) list_insert_lex<16>(md, mj, exact_d(xr, j2), j2);
      }
    }
    if (g == 0 && live_row) {
      if (a.C == 1) {
#pragma unroll
        for (int p = 0; p < 16; ++p) {
          if (p >= a.K) break;
          if (a.kvalues) static_cast<float*>(a.out)[row * a.K + p] = mj[p] == INT_MAX ? __builtin_inff() : fmaxf(md[p], 0.0f);
          else static_cast<int*>(a.out)[row * a.K + p] = mj[p] == INT_MAX ? -1 : mj[p];
        }
      } else {
        float* q = a.part + ((int64_t)c * a.M + row) * (2 * a.KP);   // the direct kernel's list layout
#pragma unroll
        for (int p = 0; p < 16; ++p) {
          if (p >= a.KP) break;
          q[2 * p] = md[p];
          q[2 * p + 1] = __int_as_float(mj[p]);
        }
      }
    }
  };

  // KNN (two row blocks): the merge unrolled by hand, so that the lists are
  // indexed by constants only
  if constexpr (kKnn) {
    static_assert(RB == 2 || RB == 4, "the K-nearest epilogue runs 2 or 4 row blocks per wave");
    knn_out(dk[0], jk[0], i0 + li, i0 + li < row_end);
    knn_out(dk[1], jk[1], i0 + 16 + li, i0 + 16 + li < row_end);
    if constexpr (RB == 4) {
      knn_out(dk[RB > 2 ? 2 : 0], jk[RB > 2 ? 2 : 0], i0 + 32 + li, i0 + 32 + li < row_end);
      knn_out(dk[RB > 3 ? 3 : 0], jk[RB > 3 ? 3 : 0], i0 + 48 + li, i0 + 48 + li < row_end);
    }
  }

  // merge the four lane groups of each row (lanes li, li+16, li+32, li+48)
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int64_t row = i0 + 16 * rb + li;
    const bool live_row = row < row_end;
    if constexpr (kKnn) {
      // (written out below, outside this loop)
    } else if constexpr (kMin) {
      // smallest (distance, index) over the four lane groups; ties keep the
      // lower index.  With indices, each group's candidate gets its
      // direct-form distance first (see exact_d).
      int v = INT_MAX, j = INT_MAX;
      if (live_row && btile[rb] != INT_MAX) {
        float xr[kFastMaxD];
        load_row(row, true, xr);
        // the lane's columns 4 g + r of each block of that tile, in column order
        for (int jb = btile[rb] + 4 * g; jb < bend[rb]; jb += 16) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int jr = jb + r;
            if (jr >= bend[rb]) break;
            const int vr = __float_as_int(exact_d(xr, jr));   // >= 0: int order is float order
            if (vr < v) {
              v = vr;
              j = jr;
            }
          }
        }
      }
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const int v2 = __shfl_xor(v, o), j2 = __shfl_xor(j, o);
        if (v2 < v || (v2 == v && j2 < j)) {
          v = v2;
          j = j2;
        }
      }
      if (g == 0 && live_row) {
        // a tiny negative distance from rounding reads as 0
        const float dv = v == INT_MAX ? __builtin_inff() : fmaxf(__int_as_float(v), 0.0f);
        if (a.C == 1) {
          if constexpr (KV) static_cast<float*>(a.out)[row] = dv;
          else static_cast<int*>(a.out)[row] = j == INT_MAX ? -1 : j;
        } else {
          float* p = a.part + ((int64_t)c * a.M + row) * 2;   // one (distance, index) list entry
          p[0] = dv;
          p[1] = __int_as_float(j);
        }
      }
    } else if constexpr (EPI == FAST_LSE) {
      float m = mref[rb], s = tot[rb][0];
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const float m2 = __shfl_xor(m, o), s2 = __shfl_xor(s, o);
        const float mx = fmaxf(m, m2);
        s = (m == -__builtin_inff() ? 0.0f : s * __builtin_amdgcn_exp2f(m - mx)) +
            (m2 == -__builtin_inff() ? 0.0f : s2 * __builtin_amdgcn_exp2f(m2 - mx));
        m = mx;
      }
      if (g == 0 && live_row) {
        // the matrix core returned T + r for the row norm's remainder r
        const float rem = Rs[wave * (16 * RB) + 16 * rb + li];
        if (a.C == 1) {
          static_cast<float*>(a.out)[row] = (m + __builtin_amdgcn_logf(s) - rem) * kLn2;
        } else {
          float* p = a.part + ((int64_t)c * a.M + row) * 2;
          p[0] = m - rem;
          p[1] = s;
        }
      }
    } else {
      float v[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v[q] = tot[rb][q];
        v[q] += __shfl_xor(v[q], 16);
        v[q] += __shfl_xor(v[q], 32);
      }
      if (g == 0 && live_row) {
        // the matrix core returned T + r for the row norm's remainder r
        const int rs = wave * (16 * RB) + 16 * rb + li;
        const float f = __builtin_amdgcn_exp2f(-Rs[rs]);   // 2^-r
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] *= f;
        if constexpr (EPI == FAST_SUM) {
          const float sum = (v[0] + v[1]) + (v[2] + v[3]);
          if (a.C == 1) static_cast<float*>(a.out)[row] = sum;
          else a.part[(int64_t)c * a.M + row] = sum;
        } else if constexpr (EPI == FAST_SUMV) {
          // the sums' layout: out M x E, partials C x M x EP
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (e >= a.E) break;
            if (a.C == 1) static_cast<float*>(a.out)[row * a.E + e] = v[e];
            else a.part[((int64_t)c * a.M + row) * a.EP + e] = v[e];
          }
        } else {
          // G_d = sum_j k b (u_d - v_jd) = u_d a - H_d in prescaled units; divided
          // by the prescale it is sum_j k b (x_d - y_jd), as the direct kernel sums
          const float inv = (float)(1.0 / a.scale64);
          const float G[3] = {(Us[0][rs] * v[0] - v[1]) * inv, (Us[1][rs] * v[0] - v[2]) * inv,
                              (Us[2][rs] * v[0] - v[3]) * inv};
          if (a.C == 1) {
            float* o = static_cast<float*>(a.out) + row * (1 + a.D);
            o[0] = v[0];
#pragma unroll
            for (int d = 0; d < 3; ++d)
              if (d < a.D) o[1 + d] = -G[d] * a.gscale;
          } else {
            float* p = a.part + ((int64_t)c * a.M + row) * (1 + a.DP);
            p[0] = v[0];
#pragma unroll
            for (int d = 0; d < 3; ++d)
              if (d < a.DP) p[1 + d] = G[d];
          }
        }
      }
    }
  }
}

}  // namespace

// Rows per workgroup: four row blocks per wave, except the K-nearest lists
// beyond 4 entries, which run two (measured at 1e6 x 1e6, D = 3: four row
// blocks gain at K = 4, 123 -> 112 ms, and lose at K = 10, 132 -> 165 ms).
int fast_rows_per_block(int epi, int K) { return (epi == FAST_KNN && K > 4) ? 64 * 2 : 64 * 4; }

hipError_t launch_fast_prologue(const FastPackArgs& a, const float* x, int64_t M, hipStream_t s) {
  FastGuard* g = const_cast<FastGuard*>(a.guard);   // the prologue fills the guard
  hipLaunchKernelGGL(guard_init_kernel, dim3(1), dim3(64), 0, s, g);
  const int64_t items = M + a.N;
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((items + 255) / 256, 512));
  hipLaunchKernelGGL(bounds_kernel, dim3((unsigned)blocks), dim3(256), 0, s, x, M, a.y, a.N, a.D, g);
  if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
  const int64_t pb = std::max<int64_t>(1, std::min<int64_t>((a.N16 + 255) / 256, 8192));
  hipLaunchKernelGGL(fast_pack_kernel, dim3((unsigned)pb), dim3(256), 0, s, a);
  return hipGetLastError();
}

namespace {
__global__ void fast_record_kernel(const FastGuard* g, int D, float scale, float limit, int* counts) {
  if (threadIdx.x == 0) {
    if (fast_frame(g, D, scale, limit).ok) atomicAdd(&counts[0], 1);
    atomicAdd(&counts[1], 1);
  }
}
}  // namespace

hipError_t launch_fast_record(const FastGuard* g, int D, float scale, float limit, int* counts,
                              hipStream_t s) {
  hipLaunchKernelGGL(fast_record_kernel, dim3(1), dim3(64), 0, s, g, D, scale, limit, counts);
  return hipGetLastError();
}

hipError_t launch_fast(const FastArgs& a, hipStream_t s) {
  const int rows = fast_rows_per_block(a.epi, a.K);
  const int64_t rb = a.nr > 0 ? range_grid_bound(a.nr, a.M, rows) : (a.M + rows - 1) / rows;
  const dim3 grid((unsigned)(rb * a.C));
  switch (a.epi) {
    case FAST_SUM: hipLaunchKernelGGL((fast_kernel<FAST_SUM, 4>), grid, dim3(256), 0, s, a); break;
    case FAST_GRADX: hipLaunchKernelGGL((fast_kernel<FAST_GRADX, 4>), grid, dim3(256), 0, s, a); break;
    case FAST_SUMV: hipLaunchKernelGGL((fast_kernel<FAST_SUMV, 4>), grid, dim3(256), 0, s, a); break;
    case FAST_LSE: hipLaunchKernelGGL((fast_kernel<FAST_LSE, 4>), grid, dim3(256), 0, s, a); break;
    case FAST_MIN:
      if (a.kvalues) hipLaunchKernelGGL((fast_kernel<FAST_MIN, 4, true>), grid, dim3(256), 0, s, a);
      else hipLaunchKernelGGL((fast_kernel<FAST_MIN, 4, false>), grid, dim3(256), 0, s, a);
      break;
    case FAST_KNN:
      // row blocks per wave as fast_rows_per_block: the lists hold 2 KL registers each
      if (a.K <= 4) hipLaunchKernelGGL((fast_kernel<FAST_KNN, 4, false, 4>), grid, dim3(256), 0, s, a);
      else if (a.K <= 8) hipLaunchKernelGGL((fast_kernel<FAST_KNN, 2, false, 8>), grid, dim3(256), 0, s, a);
      else if (a.K <= 10) hipLaunchKernelGGL((fast_kernel<FAST_KNN, 2, false, 10>), grid, dim3(256), 0, s, a);
      else if (a.K <= 12) hipLaunchKernelGGL((fast_kernel<FAST_KNN, 2, false, 12>), grid, dim3(256), 0, s, a);
      else if (a.K <= 16) hipLaunchKernelGGL((fast_kernel<FAST_KNN, 2, false, 16>), grid, dim3(256), 0, s, a);
      else return hipErrorInvalidValue;
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace kred
