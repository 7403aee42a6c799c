// The fp32 matrix-core reduction kernel (16 < D <= 256) and the helpers the
// large-D kernels share: work items, masked loads, k-NN lists.  Included by
// k_mfma.hip (fp32 contraction, with the split bf16 and exact k-NN kernels)
// and k_mfma64.hip (the fp64-contraction variant, beyond the fp32 kernels'
// accuracy guard); each translation unit instantiates its own variants.
//
// Large-D reductions (16 < D <= 256) on the fp32 matrix cores of gfx950.
//
// For large D the pair term is dominated by the inner product <x_i, y_j>, a
// genuine dense contraction.  Each wave owns RB blocks of 16 rows x_i and
// streams the workgroup's column block through double-buffered LDS tiles.
// Per 16 x 16 (column, row) block it computes, with v_mfma_f32_16x16x4_f32,
//
//     T[j][i] = sum_d Yop[j][d] X[i][d] + (ny_j + nx_i)
//
// where the prologue has packed Yop = 2 y' and ny = -|y'|^2 (sums) or
// Yop = -2 y and ny = |y|^2 (arg-K-min), so that T = -|x' - y'|^2 in the
// expanded form |x|^2 + |y|^2 - 2 <x, y> (prescaled coordinates, log2 units).
//   * sums:  p = 2^T (Gauss), 2^-sqrt(-T) (Laplace) or -T (squared distance);
//     the 16 x 16 tile p is already laid out as the A operand of the next
//     v_mfma_f32_16x16x4_f32, so a = P . B accumulates on the matrix cores
//     with no data movement;
//   * arg-K-min: T = |y|^2 - 2 <x, y> ranks the columns of a row exactly like
//     |x - y|^2; each lane keeps a sorted K-list of T over the columns it
//     sees, adds the row norm |x|^2 to its values once at the end (so the
//     second pass can return squared distances), and the second pass merges
//     the lists.  Keeping |x|^2 out of the loop also keeps it out of the
//     register budget: one more live value per row block pushed the kernel
//     past 168 VGPRs, from 3 to 2 waves per SIMD, and cost 12%.
//
// MFMA 16x16x4 f32 operand layout (lane l = 16 g + li, g = l / 16):
//   A (16 x 4):  lane l supplies A[li][g];   B (4 x 16): lane l supplies B[g][li];
//   D (16 x 16): lane l holds D[4 g + r][li] in register r = 0..3.
// With A = Y rows (m = column j) and B = X rows (n = row i), the result lane
// l holds T[j = 4 g + r][i = li], i.e. P[i = li][j = 4 g + r]: exactly the A
// operand of the P . B product when its k index is j = 4 g + r.
// The contraction index d is split by lane group: chunk q of lane group g
// covers d = g Q + q, so each lane reads Q contiguous floats of a row.
#pragma once

#include "kred_internal.h"

#include <climits>

namespace kred {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f4 mfma4(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

constexpr int tile_cols(int DP) {
  // LDS budget per buffer: about 4608 floats of y rows (padded stride DP + 4)
  return (4608 / (DP + 4)) >= 64 ? 64 : ((4608 / (DP + 4)) >= 32 ? 32 : 16);
}
// fp64 y rows: the same bytes per buffer (at least one 16-column block)
constexpr int tile_cols64(int DP) {
  return (2304 / (DP + 2)) >= 64 ? 64 : ((2304 / (DP + 2)) >= 32 ? 32 : 16);
}

typedef double d4 __attribute__((ext_vector_type(4)));

// Lane layout of v_mfma_f64_16x16x4_f64 (lane l = 16 g + li, measured on
// gfx950 with in-bounds probes): A from lane l is A[li][g], B from lane l is
// B[g][li], like the fp32 product, but D in lane l register r is D[g + 4 r][li]
// (the fp32 product: D[4 g + r][li]).  Lane li supplying the y row of column
// perm64(li) = 4 (li % 4) + li / 4 as its A row puts T of column 4 g + r in
// register r, the fp32 layout, so the epilogues are shared.
__device__ __forceinline__ int perm64(int li) { return 4 * (li & 3) + (li >> 2); }

template <bool F64> struct ctype { typedef float type; };
template <> struct ctype<true> { typedef double type; };
__device__ __forceinline__ float cfma(float a, float b, float c) { return __builtin_fmaf(a, b, c); }
__device__ __forceinline__ double cfma(double a, double b, double c) { return __builtin_fma(a, b, c); }

// fp64 norms of the 2 columns col, col + 1 (16-byte aligned), those outside
// [lo, hi) replaced by pad (see masked_ny)
__device__ __forceinline__ float4 masked_ny64(const double* __restrict__ ny, double pad, int64_t col,
                                              int64_t lo, int64_t hi) {
  double v[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) v[u] = (col + u >= lo && col + u < hi) ? ny[col + u] : pad;
  const double2 d2 = {v[0], v[1]};
  return __builtin_bit_cast(float4, d2);
}


// Insert (d, j) into the ascending list (dk, jk) of KP entries; equal
// distances keep the earlier entry first (columns arrive in index order).
// Entry p becomes dk[p-1] (d moves in above it), d (it lands here) or stays:
// that is the median of (dk[p-1], d, dk[p]) for a sorted list, one v_med3;
// the indices follow the same two comparisons, each made once.
template <int KP>
__device__ __forceinline__ void list_insert(float (&dk)[KP], int (&jk)[KP], float d, int j) {
  bool lt[KP];
#pragma unroll
  for (int p = 0; p < KP; ++p) lt[p] = d < dk[p];
#pragma unroll
  for (int p = KP - 1; p > 0; --p) {
    dk[p] = __builtin_amdgcn_fmed3f(dk[p - 1], d, dk[p]);
    jk[p] = lt[p - 1] ? jk[p - 1] : (lt[p] ? j : jk[p]);
  }
  dk[0] = lt[0] ? d : dk[0];
  jk[0] = lt[0] ? j : jk[0];
}

// The exact kernel's lists hold (d, j) as one fp64 key d 2^28 + j: d is an
// integer with |d| < 2^24 and 0 <= j < 2^28, so the key is exact and orders
// as (d, j).  Insertion runs from the top down, in place: entry p becomes
// min(old p, max(old p-1, key)), two fp64 operations and no comparison.
constexpr double kKeyScale = 268435456.0;   // 2^28
constexpr double kKeyInv = 1.0 / 268435456.0;

template <int KP>
__device__ __forceinline__ void key_insert(double (&kk)[KP], double key) {
#pragma unroll
  for (int p = KP - 1; p > 0; --p) kk[p] = __builtin_fmin(kk[p], __builtin_fmax(kk[p - 1], key));
  kk[0] = __builtin_fmin(kk[0], key);
}

// the distance part of a key (+infinity stays +infinity)
__device__ __forceinline__ float key_d(double key) { return (float)__builtin_floor(key * kKeyInv); }

// ------------------------------------------------------------ work items
// A workgroup's work: dense, a (row block, column block) pair; block-sparse,
// a row block inside row cluster I and chunk c of I's columns, the chunk
// being an equal share of the columns of I's ranges in their concatenated
// order (clamped to [0, N)).  Both are walked as segments [a0, a1) of
// consecutive columns, in tiles that start 16-aligned (a0 rounded down); the
// tile's columns outside the segment get b = 0 and the padding norm, which
// remove them (sums: the norm -infinity gives 2^-inf = 0, and the squared
// distance's finite value meets b = 0; arg-K-min: +infinity never enters a
// list).
struct MItem {
  int c;                    // column block (dense) or chunk (block-sparse)
  int64_t row0, row_end;    // the workgroup's first row and the end of its rows
  int64_t w0, w1;           // dense: the columns; block-sparse: the chunk's window
  const int* cr;            // block-sparse: the cluster's ranges
  int nrange;               // 0: dense
  bool live;                // false: a spare workgroup of a block-sparse grid
};

__device__ __forceinline__ void mcol_range(const MfmaArgs& a, const int* cr, int q, int64_t& js,
                                           int64_t& je) {
  js = min(max((int64_t)cr[2 * q], (int64_t)0), a.N);
  je = min(max((int64_t)cr[2 * q + 1], js), a.N);
}

template <bool SP>
__device__ __forceinline__ MItem mitem(const MfmaArgs& a, int rows) {
  MItem it;
  it.cr = nullptr;
  it.nrange = 0;
  it.live = true;
  it.c = blockIdx.x % a.C;
  if (!SP) {
    it.row0 = (int64_t)(blockIdx.x / a.C) * rows;
    it.row_end = a.M;
    it.w0 = (int64_t)it.c * a.jpb;
    it.w1 = min(a.N16, it.w0 + a.jpb);
    return it;
  }
  const int blk = (int)(blockIdx.x / a.C);
  if (blk >= a.bstart[a.nr]) {
    it.live = false;
    it.row0 = it.row_end = it.w0 = it.w1 = 0;
    return it;
  }
  int lo = 0, hi = a.nr - 1;   // last cluster I with bstart[I] <= blk
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.bstart[mid] <= blk) lo = mid;
    else hi = mid - 1;
  }
  const int64_t r0 = min(max((int64_t)a.rr[2 * lo], (int64_t)0), a.M);
  const int64_t r1 = min(max((int64_t)a.rr[2 * lo + 1], r0), a.M);
  it.row0 = r0 + (int64_t)(blk - a.bstart[lo]) * rows;
  it.row_end = r1;
  it.cr = a.cr + 2 * (int64_t)a.cp[lo];
  it.nrange = a.cp[lo + 1] - a.cp[lo];
  int64_t L = 0;
  for (int q = 0; q < it.nrange; ++q) {
    int64_t js, je;
    mcol_range(a, it.cr, q, js, je);
    L += je - js;
  }
  it.w0 = L * it.c / a.C;
  it.w1 = L * (it.c + 1) / a.C;
  return it;
}

// Calls seg(a0, a1) for each segment of the item's columns (workgroup-uniform).
template <class Seg>
__device__ __forceinline__ void for_segments(const MfmaArgs& a, const MItem& it, Seg&& seg) {
  if (it.nrange == 0) {
    if (it.w0 < it.w1) seg(it.w0, it.w1);
    return;
  }
  int64_t off = 0;
  for (int q = 0; q < it.nrange && off < it.w1; ++q) {
    int64_t js, je;
    mcol_range(a, it.cr, q, js, je);
    const int64_t s0 = max(js, js + (it.w0 - off)), s1 = min(je, js + (it.w1 - off));
    if (s0 < s1) seg(s0, s1);
    off += je - js;
  }
}

// ny of the 4 columns col .. col + 3 (16-byte aligned), those outside [lo, hi)
// replaced by the padding norm pad (a value, so that the compiler selects
// values, not the addresses of two loads).
__device__ __forceinline__ float4 masked_ny(const float* __restrict__ ny, float pad, int64_t col,
                                            int64_t lo, int64_t hi) {
  if (col >= lo && col + 4 <= hi) return *reinterpret_cast<const float4*>(ny + col);
  float v[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    v[u] = pad;
    if (col + u >= lo && col + u < hi) v[u] = ny[col + u];
  }
  return float4{v[0], v[1], v[2], v[3]};
}

// A float4 of packed b holding columns col .. col + 3 (one signal column),
// those outside [lo, hi) zeroed; p is its address.
__device__ __forceinline__ float4 masked_b(const float4* p, int64_t col, int64_t lo, int64_t hi) {
  if (col >= lo && col + 4 <= hi) return *p;
  if (col + 4 <= lo || col >= hi) return float4{0.f, 0.f, 0.f, 0.f};
  const float4 v = *p;
  return float4{(col >= lo && col < hi) ? v.x : 0.f, (col + 1 >= lo && col + 1 < hi) ? v.y : 0.f,
                (col + 2 >= lo && col + 2 < hi) ? v.z : 0.f, (col + 3 >= lo && col + 3 < hi) ? v.w : 0.f};
}

// Column of the first of the 4 packed-b floats at float offset t4 of a tile
// starting at column jt (layout: 16-column blocks, 4-column groups, W signal columns).
__device__ __forceinline__ int64_t bpk_col(int64_t jt, int t4, int W) {
  return jt + (int64_t)(t4 / (16 * W)) * 16 + ((t4 % (16 * W)) / (4 * W)) * 4;
}

// EPI: 0 Gauss, 1 Laplace, 2 squared distance (sums), 3 arg-K-min, 4 log-sum-exp
// of s_ij = g_j - |x_i - y_j|^2 / eps (log2 units: the column norms carry g_j),
// 5 log-sum-exp of s_ij = g_j - |x_i - y_j| / sigma (g_j from its own array),
// 6..9 min / max of F_ij b_je per signal column e (F: 6 Gauss, 7 Laplace, 8
// squared distance, 9 the Sinkhorn form s_ij, with b = 1), lowest index on ties.
// SP: block-sparse (a pattern of row clusters and column ranges) or dense.
//
// F64: the contraction and the norms in fp64 (v_mfma_f64_16x16x4_f64), T
// rounded to fp32 once for the epilogues; the variant the accuracy guard picks
// when the fp32 expanded form's error bound exceeds the budget (SpreadGuard).
template <int Q, int RB, int EPI, int EB, int KP, bool SP, bool F64 = false>
__global__ __launch_bounds__(256) void mfma_kernel(MfmaArgs a) {
  static_assert(!(F64 && EPI == 3), "the k-NN lists rank in fp32 (their values are re-ranked exactly)");
  typedef typename ctype<F64>::type CT;
  constexpr int DP = 4 * Q;
  constexpr int EPU = F64 ? 2 : 4;   // elements per 16-byte unit
  constexpr int LDY = DP + EPU;      // padded row stride in elements
  constexpr int TJ = F64 ? tile_cols64(DP) : tile_cols(DP);
  constexpr int NU = TJ * (int)sizeof(CT) / 16;   // 16-byte units of norms per tile
  constexpr bool SUM = EPI < 3;
  constexpr bool LSE = EPI == 4 || EPI == 5;
  constexpr bool EXT = EPI >= 6;
  constexpr bool BSIG = SUM || EXT;   // packed b tiles in LDS
  constexpr bool LAPG = EPI == 5;   // per-column g' staged like the norms
  constexpr int W = 16 * EB;                       // signal columns per row in a tile
  constexpr int YF4 = TJ * DP / EPU;               // 16-byte units of y per tile
  constexpr int YL = (YF4 + 255) / 256;            // per thread
  constexpr int BF4 = BSIG ? TJ * W / 4 : 0;       // float4s of b per tile
  constexpr int BL = BSIG ? (BF4 + 255) / 256 : 0;
  constexpr int KL = EPI == 3 ? KP : 1;

  __shared__ float4 ys[2][TJ * LDY / EPU];
  __shared__ float4 ns[2][NU];
  __shared__ float4 bs[2][BSIG ? TJ * W / 4 : 1];
  __shared__ float4 gsh[2][LAPG ? TJ / 4 : 1];

  if constexpr (EPI == 3) {
    if (exact_ok(a.exact, a.D)) return;   // the bf16 kernel does the work
  } else {
    if (wide64(a.spread, a.wide_c, a.wide_limit) != F64) return;   // the other precision does
  }
  const MItem it = mitem<SP>(a, 64 * RB);
  if (!it.live) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int li = lane & 15, g = lane >> 4;
  const int c = it.c;
  const int64_t rend = it.row_end;
  const float pad_ny = a.pad_ny;
  const int64_t i0 = it.row0 + wave * (16 * RB);

  // rows: lane supplies X[i = li][d = g Q + q] of each of its RB row blocks.
  // The centred forms in fp32 take X = fl32(s (x - m)) formed in fp64 and
  // nx = -fl32(|X|^2) summed in fp64 (the accuracy guard's arithmetic)
  constexpr bool PREP64 = !F64 && EPI != 3;
  CT xr[RB][Q];
  CT nx[RB];
  const CT xs = F64 ? (CT)a.xscale64 : (CT)a.xscale;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int64_t row = i0 + 16 * rb + li;
    const bool ok = row < rend;
    CT part = 0;
    double part64 = 0.0;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int d = g * Q + q;
      CT v;
      if constexpr (PREP64) {
        v = (ok && d < a.D)
                ? (CT)(((double)a.x[row * a.D + d] - (double)(a.xc != nullptr ? a.xc[d] : 0.0f)) *
                       a.xscale64)
                : (CT)0;
        part64 = __builtin_fma((double)v, (double)v, part64);
      } else {
        v = (ok && d < a.D) ? ((CT)a.x[row * a.D + d] - (CT)(a.xc != nullptr ? a.xc[d] : 0.0f)) * xs
                            : (CT)0;
        part = cfma(v, v, part);
      }
      xr[rb][q] = v;
    }
    if constexpr (PREP64) {
      part64 += __shfl_xor(part64, 16);
      part64 += __shfl_xor(part64, 32);
      part = (CT)part64;
    } else {
      part += __shfl_xor(part, 16);
      part += __shfl_xor(part, 32);
    }
    nx[rb] = -part;   // sums and log-sum-exp; arg-K-min recomputes it after the loop
  }
  // log-sum-exp: per lane a running reference (log2 units; a finite floor, so
  // that differences never meet -inf - -inf), the sum of the current tile and
  // the total, both relative to it
  float lm[RB], lp[RB], ls[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    lm[rb] = -3.0e38f;
    lp[rb] = ls[rb] = 0.0f;
  }
  // extremes: per row block and signal column the smallest key sign * F b so
  // far over the lane's columns, and its column (-1: none)
  constexpr int XW = EXT ? W : 1;
  float xbest[RB][XW];
  int xidx[RB][XW];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int e = 0; e < XW; ++e) {
      xbest[rb][e] = __builtin_inff();
      xidx[rb][e] = -1;
    }

  f4 oacc[RB][EB], tot[RB][EB];
  float dk[RB][KL];
  int jk[RB][KL];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
    for (int eb = 0; eb < EB; ++eb) oacc[rb][eb] = tot[rb][eb] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int p = 0; p < KL; ++p) {
      dk[rb][p] = __builtin_inff();
      jk[rb][p] = INT_MAX;
    }
  }

  float4 ystage[YL];
  float4 bstage[BL > 0 ? BL : 1];
  float4 nstage, gstage;
  // the tile at column jt (16-aligned), its columns outside [lo, hi) masked
  auto fetch = [&](int64_t jt, int64_t lo, int64_t hi) {
    // y of masked columns is loaded as is (inside the padded array): their
    // padding norm and zero b already remove them
    const int ncol = (int)min((int64_t)TJ, ((hi + 15) & ~(int64_t)15) - jt);
    // (fp64: yop and ny hold doubles, in the same buffers)
    const float4* ysrc = reinterpret_cast<const float4*>(a.yop) + jt * DP / EPU;
#pragma unroll
    for (int k = 0; k < YL; ++k) {
      const int f = tid + k * 256;
      ystage[k] = (f < YF4 && f < ncol * (DP / EPU)) ? ysrc[f] : float4{0.f, 0.f, 0.f, 0.f};
    }
    if constexpr (F64) {
      if (tid < NU) {
        const double* ny64 = reinterpret_cast<const double*>(a.ny);
        if constexpr (SP) nstage = masked_ny64(ny64, (double)pad_ny, jt + 2 * tid, lo, hi);
        else nstage = (tid * 2 < ncol) ? reinterpret_cast<const float4*>(ny64 + jt)[tid]
                                       : float4{0.f, 0.f, 0.f, 0.f};
      }
    }
    if (tid < TJ / 4) {
      if constexpr (!F64) {
        if constexpr (SP) nstage = masked_ny(a.ny, pad_ny, jt + 4 * tid, lo, hi);
        else nstage = (tid * 4 < ncol) ? reinterpret_cast<const float4*>(a.ny + jt)[tid]
                                       : float4{0.f, 0.f, 0.f, 0.f};
      }
      if constexpr (LAPG) {
        const float ninf = -__builtin_inff();
        if constexpr (SP) gstage = masked_ny(a.gpk, ninf, jt + 4 * tid, lo, hi);
        else gstage = (tid * 4 < ncol) ? reinterpret_cast<const float4*>(a.gpk + jt)[tid]
                                       : float4{ninf, ninf, ninf, ninf};
      }
    }
    if constexpr (BSIG) {
      const float4* bsrc = reinterpret_cast<const float4*>(a.bpk + jt * W);
#pragma unroll
      for (int k = 0; k < BL; ++k) {
        const int f = tid + k * 256;
        if constexpr (SP)
          bstage[k] = f < BF4 ? masked_b(bsrc + f, bpk_col(jt, 4 * f, W), lo, hi)
                              : float4{0.f, 0.f, 0.f, 0.f};
        else
          bstage[k] = (f < BF4 && f < ncol * W / 4) ? bsrc[f] : float4{0.f, 0.f, 0.f, 0.f};
      }
    }
  };
  auto put = [&](int buf) {
#pragma unroll
    for (int k = 0; k < YL; ++k) {
      const int f = tid + k * 256;
      if (f < YF4) {
        const int row = f / (DP / EPU), cq = f % (DP / EPU);
        ys[buf][row * (LDY / EPU) + cq] = ystage[k];
      }
    }
    if (tid < NU) ns[buf][tid] = nstage;
    if constexpr (LAPG) {
      if (tid < TJ / 4) gsh[buf][tid] = gstage;
    }
    if constexpr (BSIG) {
#pragma unroll
      for (int k = 0; k < BL; ++k) {
        const int f = tid + k * 256;
        if (f < BF4) bs[buf][f] = bstage[k];
      }
    }
  };

  auto segment = [&](int64_t a0, int64_t a1) {
  const int64_t base = a0 & ~(int64_t)15;
  const int64_t ntiles = (a1 - base + TJ - 1) / TJ;
  fetch(base, a0, a1);
  put(0);
  __syncthreads();
  for (int64_t t = 0; t < ntiles; ++t) {
    const int64_t jt = base + t * TJ;
    const int buf = (int)(t & 1);
    const int nblk = (int)((min((int64_t)TJ, a1 - jt) + 15) / 16);
    if (t + 1 < ntiles) fetch(jt + TJ, a0, a1);
    for (int blk = 0; blk < nblk; ++blk) {
      CT yo[Q];
      // fp64: this lane supplies the y row of column perm64(li) (see perm64)
      const int yl = F64 ? perm64(li) : li;
      const float4* yrow = &ys[buf][(blk * 16 + yl) * (LDY / EPU) + g * (Q / EPU)];
#pragma unroll
      for (int qq = 0; qq < Q / EPU; ++qq) {
        const float4 v = yrow[qq];
        if constexpr (F64) {
          const double2 dv = __builtin_bit_cast(double2, v);
          yo[2 * qq + 0] = dv.x;
          yo[2 * qq + 1] = dv.y;
        } else {
          yo[4 * qq + 0] = v.x;
          yo[4 * qq + 1] = v.y;
          yo[4 * qq + 2] = v.z;
          yo[4 * qq + 3] = v.w;
        }
      }
      // the norms of the lane's columns 4 g .. 4 g + 3
      CT nyv[4];
      if constexpr (F64) {
        const double2 n0 = __builtin_bit_cast(double2, ns[buf][blk * 8 + 2 * g]);
        const double2 n1 = __builtin_bit_cast(double2, ns[buf][blk * 8 + 2 * g + 1]);
        nyv[0] = n0.x; nyv[1] = n0.y; nyv[2] = n1.x; nyv[3] = n1.y;
      } else {
        const float4 n = ns[buf][blk * 4 + g];
        nyv[0] = n.x; nyv[1] = n.y; nyv[2] = n.z; nyv[3] = n.w;
      }
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        f4 acc;
        if constexpr (F64) {
          d4 accd = {nx[rb] + nyv[0], nx[rb] + nyv[1], nx[rb] + nyv[2], nx[rb] + nyv[3]};
#pragma unroll
          for (int q = 0; q < Q; ++q)
            accd = __builtin_amdgcn_mfma_f64_16x16x4f64(yo[q], xr[rb][q], accd, 0, 0, 0);
          acc = f4{(float)accd[0], (float)accd[1], (float)accd[2], (float)accd[3]};
        } else if constexpr (EPI == 3) {
          acc = f4{nyv[0], nyv[1], nyv[2], nyv[3]};
#pragma unroll
          for (int q = 0; q < Q; ++q) acc = mfma4(yo[q], xr[rb][q], acc);
        } else {
          // T = fl(P + fl(nx + ny)) with P accumulated from zero: the norms
          // never enter the chain of roundings
          acc = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int q = 0; q < Q; ++q) acc = mfma4(yo[q], xr[rb][q], acc);
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[r] += nx[rb] + nyv[r];
        }
        if constexpr (SUM) {
          f4 p;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            if constexpr (EPI == 0) p[r] = __builtin_amdgcn_exp2f(acc[r]);
            else if constexpr (EPI == 1) p[r] = __builtin_amdgcn_exp2f(-__builtin_amdgcn_sqrtf(fmaxf(-acc[r], 0.0f)));
            else p[r] = fmaxf(-acc[r], 0.0f);
          }
#pragma unroll
          for (int eb = 0; eb < EB; ++eb) {
            // lane needs b[j = blk*16 + 4g + r][e = 16 eb + li] for r = 0..3
            const float* bl = reinterpret_cast<const float*>(&bs[buf][0]) +
                              blk * 16 * W + g * 4 * W + (16 * eb + li) * 4;
            const float4 bv = *reinterpret_cast<const float4*>(bl);
            oacc[rb][eb] = mfma4(p[0], bv.x, oacc[rb][eb]);
            oacc[rb][eb] = mfma4(p[1], bv.y, oacc[rb][eb]);
            oacc[rb][eb] = mfma4(p[2], bv.z, oacc[rb][eb]);
            oacc[rb][eb] = mfma4(p[3], bv.w, oacc[rb][eb]);
          }
        } else if constexpr (EXT) {
          // F of the lane's 4 columns, then for every signal column e the
          // key sign * F b; columns outside [a0, min(a1, N)) never win.
          // Columns arrive in index order, so a strict test keeps the lowest
          // index on ties.
          const int64_t jb = jt + blk * 16 + 4 * g;
          const int64_t jend = min(a1, a.N);
          float fv[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            if constexpr (EPI == 6) fv[r] = __builtin_amdgcn_exp2f(acc[r]);
            else if constexpr (EPI == 7) fv[r] = __builtin_amdgcn_exp2f(-__builtin_amdgcn_sqrtf(fmaxf(-acc[r], 0.0f)));
            else if constexpr (EPI == 8) fv[r] = fmaxf(-acc[r], 0.0f);
            else fv[r] = acc[r] * kLn2;
            fv[r] = (jb + r >= a0 && jb + r < jend) ? fv[r] * a.ext_sign : __builtin_nanf("");
          }
#pragma unroll
          for (int e = 0; e < W; ++e) {
            // b of the lane's 4 columns for signal column e
            const float4 bv = *reinterpret_cast<const float4*>(
                reinterpret_cast<const float*>(&bs[buf][0]) + blk * 16 * W + g * 4 * W + e * 4);
            const float bb[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float key = fv[r] * bb[r];   // NaN (an excluded column) never compares less
              const bool lt = key < xbest[rb][e];
              xbest[rb][e] = lt ? key : xbest[rb][e];
              xidx[rb][e] = lt ? (int)(jb + r) : xidx[rb][e];
            }
          }
        } else if constexpr (LSE) {
          // s of the lane's 4 columns (padding columns: -inf); the reference
          // moves up to the largest s seen, rescaling both sums
          if constexpr (LAPG) {
            // acc = -(log2(e) / sigma)^2 d: s = g' - sqrt(-acc)
            const float4 gv = gsh[buf][blk * 4 + g];
            acc[0] = gv.x - __builtin_amdgcn_sqrtf(fmaxf(-acc[0], 0.0f));
            acc[1] = gv.y - __builtin_amdgcn_sqrtf(fmaxf(-acc[1], 0.0f));
            acc[2] = gv.z - __builtin_amdgcn_sqrtf(fmaxf(-acc[2], 0.0f));
            acc[3] = gv.w - __builtin_amdgcn_sqrtf(fmaxf(-acc[3], 0.0f));
          }
          const float mb = fmaxf(fmaxf(acc[0], acc[1]), fmaxf(acc[2], acc[3]));
          const float nm = fmaxf(lm[rb], mb);
          const float sc = __builtin_amdgcn_exp2f(lm[rb] - nm);
          lp[rb] = lp[rb] * sc + ((__builtin_amdgcn_exp2f(acc[0] - nm) + __builtin_amdgcn_exp2f(acc[1] - nm)) +
                                  (__builtin_amdgcn_exp2f(acc[2] - nm) + __builtin_amdgcn_exp2f(acc[3] - nm)));
          ls[rb] *= sc;
          lm[rb] = nm;
        } else {
          const float kth = dk[rb][KL - 1];
          const bool any = acc[0] < kth || acc[1] < kth || acc[2] < kth || acc[3] < kth;
          if (__builtin_expect(any, 0)) {
            const int jb = (int)(jt + blk * 16 + 4 * g);
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (acc[r] < dk[rb][KL - 1]) list_insert<KL>(dk[rb], jk[rb], acc[r], jb + r);
          }
        }
      }
    }
    if constexpr (SUM) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int eb = 0; eb < EB; ++eb) {
          tot[rb][eb] += oacc[rb][eb];
          oacc[rb][eb] = f4{0.f, 0.f, 0.f, 0.f};
        }
    }
    if constexpr (LSE) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        ls[rb] += lp[rb];
        lp[rb] = 0.0f;
      }
    }
    // buffer (t+1)&1 was last read in iteration t-1, which ended with a barrier
    if (t + 1 < ntiles) put((int)((t + 1) & 1));
    __syncthreads();
  }
  };
  if constexpr (SP) for_segments(a, it, segment);
  else if (it.w0 < it.w1) segment(it.w0, it.w1);

  if constexpr (SUM) {
    // D layout of the P . B product: lane holds out[i = 4 g + r][e = 16 eb + li]
    const int Ec = min(W, a.E - a.e0);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int eb = 0; eb < EB; ++eb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t row = i0 + 16 * rb + 4 * g + r;
          const int e = 16 * eb + li;
          if (row >= rend) continue;
          if (a.C == 1) {
            if (e < Ec) static_cast<float*>(a.out)[row * a.E + a.e0 + e] = tot[rb][eb][r];
          } else {
            a.part[((int64_t)c * a.M + row) * W + e] = tot[rb][eb][r];
          }
        }
  } else if constexpr (EXT) {
    // one (key, index) pair per (column block, lane group, row, signal column):
    // the second pass merges the 4 C partials of a row
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const int64_t row = i0 + 16 * rb + li;
      if (row >= rend) continue;
      float* q = a.part + (((int64_t)c * 4 + g) * a.M + row) * (2 * W);
#pragma unroll
      for (int e = 0; e < W; ++e) {
        q[2 * e] = xbest[rb][e];
        q[2 * e + 1] = __int_as_float(xidx[rb][e]);
      }
    }
  } else if constexpr (LSE) {
    // merge the row's four lane groups: (m, s) + (m', s') relative to max(m, m')
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      float m = lm[rb], t = ls[rb];
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const float m2 = __shfl_xor(m, o), t2 = __shfl_xor(t, o);
        const float nm = fmaxf(m, m2);
        t = t * __builtin_amdgcn_exp2f(m - nm) + t2 * __builtin_amdgcn_exp2f(m2 - nm);
        m = nm;
      }
      const int64_t row = i0 + 16 * rb + li;
      if (g != 0 || row >= rend) continue;
      if (a.C == 1) {
        // an empty row (t = 0) gives -infinity
        static_cast<float*>(a.out)[row] = (m + __builtin_amdgcn_logf(t)) * kLn2;
      } else {
        float* pp = a.part + ((int64_t)c * a.M + row) * 2;   // the (m, s) pair the combine merges
        pp[0] = t > 0.0f ? m : -__builtin_inff();
        pp[1] = t;
      }
    }
  } else {
    // one partial list per (column block, lane group); the second pass merges them
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      // the row norm, summed in the same order as before the loop
      float part = 0.0f;
#pragma unroll
      for (int q = 0; q < Q; ++q) part = __builtin_fmaf(xr[rb][q], xr[rb][q], part);
      part += __shfl_xor(part, 16);
      part += __shfl_xor(part, 32);
      const int64_t row = i0 + 16 * rb + li;
      if (row >= rend) continue;
      float* q = a.part + (((int64_t)c * 4 + g) * a.M + row) * (2 * KL);
#pragma unroll
      for (int p = 0; p < KL; ++p) {
        q[2 * p] = dk[rb][p] + part;
        q[2 * p + 1] = __int_as_float(jk[rb][p]);
      }
    }
  }
}

}  // namespace
}  // namespace kred
