// Direct-form reduction kernels for small D (D <= 16) on gfx950.
//
// The reduction of Eq. (2) (Sec. 2) over a symbolic M x N matrix that is
// never stored.  Each lane owns R rows x_i held in VGPRs.  The workgroup
// streams its column block of packed (y_j, b_j) rows through a double-
// buffered LDS tile: coalesced global loads of tile t+1 are in flight while
// the pair loop runs on tile t, and every lane reads y_j with one broadcast
// LDS load into VGPRs.  Keeping every pair-loop operand in VGPRs matters on
// gfx950: an FP32 VALU instruction whose sources are all VGPRs issues in about
// half the cycles of one that takes a scalar (SGPR) operand.
//
// The pair term uses the direct form |x - y|^2 = sum_k (x_k - y_k)^2 in the
// input coordinates, which keeps full fp32 accuracy where x is close to y
// (where the Gaussian is large) whatever the scale of the data; the kernel
// value is then one multiply and one v_exp_f32, 2^(-kscale d) with kscale =
// log2(e) / (2 sigma^2).  (Prescaling the coordinates by sqrt(kscale) would
// save the multiply but loses absolute precision in x - y when |x| sqrt(kscale)
// is large.)  Sums are two-level (a per-tile
// partial folded into the running total once per tile), which keeps fp32
// rounding growth near u (sqrt(T) + sqrt(N / T)) instead of u N.
#include "kred.h"
#include "kred_internal.h"

#include <cfloat>
#include <climits>

namespace kred {
namespace {

constexpr float kRescale = 32.0f;   // log-sum-exp: rescale once a term exceeds 2^32 x reference

__device__ __forceinline__ float fast_exp2(float v) { return __builtin_amdgcn_exp2f(v); }
__device__ __forceinline__ float fast_sqrt(float v) { return __builtin_amdgcn_sqrtf(v); }
__device__ __forceinline__ float fast_log2(float v) { return __builtin_amdgcn_logf(v); }

// ------------------------------------------------------------------ prologue
__global__ __launch_bounds__(256) void pack_kernel(PackArgs a) {
  if (a.guard != nullptr && fast_frame(a.guard, a.D, a.fscale, a.flimit).ok) return;
  const int S = a.DP + a.EP;
  const int64_t total = a.N * S;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t j = t / S;
    const int s = (int)(t - j * S);
    float v = 0.0f;
    if (s < a.D) {
      v = a.y[j * a.D + s] * a.yscale;
    } else if (s >= a.DP) {
      const int e = a.e0 + s - a.DP;
      if (a.b != nullptr && e < a.E) v = a.b[j * a.E + e] * a.bscale;
      else if (a.unit_b && s == a.DP) v = a.bscale;
    }
    a.ypk[t] = v;
  }
}

// Alternating two-value fill: (v0, v1, v0, v1, ...), the empty value of
// (value, index) or (max, sum) partials.
__global__ __launch_bounds__(256) void fill2_kernel(float* out, int64_t count, float v0, float v1) {
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < count;
       t += (int64_t)gridDim.x * blockDim.x)
    out[t] = (t & 1) ? v1 : v0;
}

__global__ __launch_bounds__(256) void fill_kernel(float* out, int64_t count, float value) {
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < count;
       t += (int64_t)gridDim.x * blockDim.x)
    out[t] = value;
}

// ------------------------------------------------------ LDS tile streaming
// Packed rows have S floats; in LDS each row is padded to SP (a multiple of
// 4) so that one row is read with SP/4 aligned 16-byte broadcast loads.
template <int S>
struct Tile {
  static constexpr int SP = (S + 3) / 4 * 4;
  static constexpr int TJ = SP <= 4 ? 256 : (SP <= 8 ? 128 : 64);   // rows per tile
  static constexpr int LOADS = (TJ * S + kThreads - 1) / kThreads;   // floats per thread per tile
  static constexpr int U = SP <= 8 ? 4 : 2;                          // j unroll
};

// Walk columns [j0, j1) of ypk through LDS; call pair(yv, j) for each column
// (yv: the SP floats of row j, in VGPRs), skipping the first `skip` columns,
// and tile_end() after each tile.  All threads of the block must call this.
template <int S, typename PairFn, typename TileEndFn>
__device__ __forceinline__ void stream_columns(const float* __restrict__ ypk, int64_t j0,
                                               int64_t j1, int skip, float4* lds, PairFn&& pair,
                                               TileEndFn&& tile_end) {
  using T = Tile<S>;
  constexpr int SP = T::SP, TJ = T::TJ, U = T::U;
  constexpr int ROW4 = SP / 4;
  const int tid = threadIdx.x;
  float* ldsf = reinterpret_cast<float*>(lds);
  const int64_t ntiles = (j1 - j0 + TJ - 1) / TJ;
  float stage[T::LOADS];

  auto fetch = [&](int64_t t) {
    const int64_t jt = j0 + t * TJ;
    const int nf = (int)(min((int64_t)TJ, j1 - jt)) * S;
    const float* src = ypk + jt * S;
#pragma unroll
    for (int q = 0; q < T::LOADS; ++q) {
      const int i = tid + q * kThreads;
      stage[q] = (i < nf) ? src[i] : 0.0f;
    }
  };
  auto put = [&](int64_t t) {
    float* dst = ldsf + (t & 1) * (TJ * SP);
#pragma unroll
    for (int q = 0; q < T::LOADS; ++q) {
      const int i = tid + q * kThreads;
      if (i < TJ * S) dst[(i / S) * SP + (i % S)] = stage[q];
    }
  };

  if (ntiles <= 0) return;
  fetch(0);
  put(0);
  __syncthreads();
  for (int64_t t = 0; t < ntiles; ++t) {
    const int64_t jt = j0 + t * TJ;
    const int n = (int)min((int64_t)TJ, j1 - jt);
    if (t + 1 < ntiles) fetch(t + 1);
    const float4* buf = lds + (t & 1) * (TJ * ROW4);
    int jj = (t == 0) ? skip : 0;
    // One y row in registers at a time: the scheduler then keeps the R
    // independent pair chains of that row in flight instead of holding
    // several rows and serialising each chain under the VGPR cap.
    for (; jj + U <= n; jj += U) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float yv[SP];
#pragma unroll
        for (int q = 0; q < ROW4; ++q) {
          const float4 v = buf[(jj + u) * ROW4 + q];
          yv[4 * q + 0] = v.x;
          yv[4 * q + 1] = v.y;
          yv[4 * q + 2] = v.z;
          yv[4 * q + 3] = v.w;
        }
        pair(yv, jt + jj + u);
      }
    }
    for (; jj < n; ++jj) {
      float yv[SP];
#pragma unroll
      for (int q = 0; q < ROW4; ++q) {
        const float4 v = buf[jj * ROW4 + q];
        yv[4 * q + 0] = v.x;
        yv[4 * q + 1] = v.y;
        yv[4 * q + 2] = v.z;
        yv[4 * q + 3] = v.w;
      }
      pair(yv, jt + jj);
    }
    tile_end();
    if (t + 1 < ntiles) put(t + 1);
    __syncthreads();
  }
}

// -------------------------------------------------------- common row set-up
// Work item of a block.
//   Dense: row block rb and column block c (consecutive blocks take
//   consecutive column blocks, so with C a multiple of 8 each XCD streams its
//   own share of the columns through its L2).
//   Block-sparse: one row block inside row cluster I; its reduction runs over
//   I's list of column ranges (ranges are clamped to [0, N), rows to [0, M)).
// Row r of a lane is row0 + r * 256 + threadIdx.x (rows of one r are
// contiguous across the block, so loads and stores coalesce), valid below
// row_end.  Indices are recomputed where needed instead of being held in
// registers: the pair loop runs at its best issue rate only with enough
// waves resident per SIMD.
struct Item {
  int c;                    // column block (dense) or column chunk (block-sparse)
  int64_t row0, row_end;
  int64_t j0, j1;           // dense: the column block; block-sparse: the chunk's window
  int nrange;               // block-sparse: number of column ranges (0: dense)
  const int* cr;            // block-sparse: this cluster's column ranges
  bool live;                // false: a spare workgroup of a block-sparse grid
};

// Column range q of a block-sparse cluster, clamped to [0, N).
__device__ __forceinline__ void col_range(const DirectArgs& a, const int* cr, int q, int64_t& js,
                                          int64_t& je) {
  js = min(max((int64_t)cr[2 * q], (int64_t)0), a.N);
  je = min(max((int64_t)cr[2 * q + 1], js), a.N);
}

template <int R>
__device__ __forceinline__ Item item_of(const DirectArgs& a) {
  Item it;
  it.nrange = 0;
  it.cr = nullptr;
  it.live = true;
  it.c = blockIdx.x % a.C;
  if (a.nr == 0) {
    const int64_t rb = blockIdx.x / a.C;
    it.row0 = rb * (int64_t)(kThreads * R);
    it.row_end = a.M;
    it.j0 = (int64_t)it.c * a.jpb;
    it.j1 = min(a.N, it.j0 + a.jpb);
    return it;
  }
  const int blk = (int)(blockIdx.x / a.C);
  if (blk >= a.bstart[a.nr]) {
    it.live = false;
    it.row0 = it.row_end = 0;
    it.j0 = it.j1 = 0;
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
  it.row0 = r0 + (int64_t)(blk - a.bstart[lo]) * (kThreads * R);
  it.row_end = r1;
  it.cr = a.cr + 2 * (int64_t)a.cp[lo];
  it.nrange = a.cp[lo + 1] - a.cp[lo];
  // chunk c of C takes an equal share of the cluster's columns, counted in
  // the concatenated order of its ranges
  int64_t L = 0;
  for (int q = 0; q < it.nrange; ++q) {
    int64_t js, je;
    col_range(a, it.cr, q, js, je);
    L += je - js;
  }
  it.j0 = L * it.c / a.C;
  it.j1 = L * (it.c + 1) / a.C;
  return it;
}

__device__ __forceinline__ int64_t row_at(const Item& it, int r, int lane_id) {
  return it.row0 + (int64_t)r * kThreads + lane_id;
}

// threadIdx.x behind an empty asm: the compiler cannot prove it equal to the
// value used before the pair loop, so it recomputes row indices after the
// loop instead of keeping R 64-bit row values alive (and spilled) across it.
__device__ __forceinline__ int opaque_tid() {
  int t = threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}

template <int DP, int R>
__device__ __forceinline__ void load_rows(const DirectArgs& a, const Item& it,
                                          float (&xr)[R][DP]) {
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int64_t row = row_at(it, r, threadIdx.x);
    const bool ok = row < it.row_end;
#pragma unroll
    for (int k = 0; k < DP; ++k)
      xr[r][k] = (ok && k < a.D) ? a.x[row * a.D + k] * a.xscale : 0.0f;
  }
}

template <int DP>
__device__ __forceinline__ float sq_dist(const float (&xr)[DP], const float* yv) {
  float t = xr[0] - yv[0];
  float d = t * t;
#pragma unroll
  for (int k = 1; k < DP; ++k) {
    t = xr[k] - yv[k];
    d = __builtin_fmaf(t, t, d);
  }
  return d;
}

// The item's columns through stream_columns: the column block, or, in list
// order, the parts of the column ranges that fall in the chunk's window
// (`skip` applies to the first column streamed).  Block-uniform, as
// stream_columns requires.
template <int S, typename PairFn, typename TileEndFn>
__device__ __forceinline__ void stream_item(const DirectArgs& a, const Item& it, int skip,
                                            float4* lds, PairFn&& pair, TileEndFn&& tile_end) {
  if (it.nrange == 0) {
    stream_columns<S>(a.ypk, it.j0, it.j1, skip, lds, pair, tile_end);
    return;
  }
  int64_t off = 0;   // window coordinate of the range's first column
  for (int q = 0; q < it.nrange && off < it.j1; ++q) {
    int64_t js, je;
    col_range(a, it.cr, q, js, je);
    const int64_t len = je - js;
    const int64_t a0 = max(it.j0 - off, (int64_t)0), a1 = min(it.j1 - off, len);
    off += len;
    if (a1 <= a0) continue;
    stream_columns<S>(a.ypk, js + a0, js + a1, skip, lds, pair, tile_end);
    skip = 0;
  }
}

// First column of the item (-1 when it has none).
__device__ __forceinline__ int64_t first_column(const DirectArgs& a, const Item& it) {
  if (it.nrange == 0) return it.j0 < it.j1 ? it.j0 : -1;
  int64_t off = 0;
  for (int q = 0; q < it.nrange && off < it.j1; ++q) {
    int64_t js, je;
    col_range(a, it.cr, q, js, je);
    const int64_t len = je - js;
    const int64_t a0 = max(it.j0 - off, (int64_t)0), a1 = min(it.j1 - off, len);
    off += len;
    if (a1 > a0) return js + a0;
  }
  return -1;
}

// ------------------------------------------------------- sum-type formulas
// F = k(d) b_j with k = 2^(-ks d) (Gauss), 2^(-ks sqrt(d)) (Laplace) or d
// (squared distance).
template <int F>
__device__ __forceinline__ float kernel_of(float d, float ks) {
  if constexpr (F == F_GAUSS) return fast_exp2(-(ks * d));
  else if constexpr (F == F_LAPLACE) return fast_exp2(-(ks * fast_sqrt(d)));
  else return d;
}

template <int F, int DP, int EP, int R>
__global__ __launch_bounds__(kThreads) void sum_kernel(DirectArgs a) {
  constexpr int S = DP + EP;
  __shared__ float4 lds[2 * Tile<S>::TJ * Tile<S>::SP / 4];
  if (a.guard != nullptr && fast_frame(a.guard, a.D, a.fscale, a.flimit).ok) return;
  const Item it = item_of<R>(a);
  if (!it.live) return;
  float xr[R][DP];
  load_rows<DP, R>(a, it, xr);
  float tot[R][EP], part[R][EP];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int e = 0; e < EP; ++e) tot[r][e] = part[r][e] = 0.0f;
  const float ks = a.kscale;

  stream_item<S>(
      a, it, 0, lds,
      [&](const float* yv, int64_t) {
        // distances of all R rows first (R independent chains interleave),
        // then the kernel values and accumulations
        float d[R];
#pragma unroll
        for (int r = 0; r < R; ++r) d[r] = sq_dist<DP>(xr[r], yv);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const float k = kernel_of<F>(d[r], ks);
#pragma unroll
          for (int e = 0; e < EP; ++e) part[r][e] = __builtin_fmaf(k, yv[DP + e], part[r][e]);
        }
        // keep each column's LDS read next to its own pair work: hoisting all
        // the unrolled reads first costs the registers the R chains need
        __builtin_amdgcn_sched_barrier(0);
      },
      [&]() {
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
          for (int e = 0; e < EP; ++e) {
            tot[r][e] += part[r][e];
            part[r][e] = 0.0f;
          }
      });

  const int Ec = min(EP, a.E - a.e0);
  const int tid_out = opaque_tid();
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int64_t row = row_at(it, r, tid_out);
    if (row >= it.row_end) continue;
    if (a.C == 1) {
      float* o = static_cast<float*>(a.out) + row * a.E + a.e0;
#pragma unroll
      for (int e = 0; e < EP; ++e)
        if (e < Ec) o[e] = tot[r][e];
    } else {
      float* p = a.part + ((int64_t)it.c * a.M + row) * EP;
#pragma unroll
      for (int e = 0; e < EP; ++e) p[e] = tot[r][e];
    }
  }
}

// ------------------------------------------- Gaussian sum + x-gradient
// w = 2^(-ks d) b_j,  a += w,  G_k += w (x_k - y_k);  gradient = -G * gscale.
template <int DP, int R>
__global__ __launch_bounds__(kThreads) void gradx_kernel(DirectArgs a) {
  constexpr int S = DP + 1;
  constexpr int W = DP + 1;
  __shared__ float4 lds[2 * Tile<S>::TJ * Tile<S>::SP / 4];
  if (a.guard != nullptr && fast_frame(a.guard, a.D, a.fscale, a.flimit).ok) return;
  const Item it = item_of<R>(a);
  if (!it.live) return;
  float xr[R][DP];
  load_rows<DP, R>(a, it, xr);
  float tot[R][W], part[R][W];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int w = 0; w < W; ++w) tot[r][w] = part[r][w] = 0.0f;

  stream_item<S>(
      a, it, 0, lds,
      [&](const float* yv, int64_t) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
          float t[DP];
          float d = 0.0f;
#pragma unroll
          for (int k = 0; k < DP; ++k) {
            t[k] = xr[r][k] - yv[k];
            d = (k == 0) ? t[0] * t[0] : __builtin_fmaf(t[k], t[k], d);
          }
          const float w = fast_exp2(-(a.kscale * d)) * yv[DP];
          part[r][0] += w;
#pragma unroll
          for (int k = 0; k < DP; ++k) part[r][1 + k] = __builtin_fmaf(w, t[k], part[r][1 + k]);
        }
      },
      [&]() {
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
          for (int w = 0; w < W; ++w) {
            tot[r][w] += part[r][w];
            part[r][w] = 0.0f;
          }
      });

  const int tid_out = opaque_tid();
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int64_t row = row_at(it, r, tid_out);
    if (row >= it.row_end) continue;
    if (a.C == 1) {
      float* o = static_cast<float*>(a.out) + row * (1 + a.D);
      o[0] = tot[r][0];
#pragma unroll
      for (int k = 0; k < DP; ++k)
        if (k < a.D) o[1 + k] = -tot[r][1 + k] * a.gscale;
    } else {
      float* p = a.part + ((int64_t)it.c * a.M + row) * W;
#pragma unroll
      for (int w = 0; w < W; ++w) p[w] = tot[r][w];
    }
  }
}

// ------------------------- Gaussian sum: vector-Jacobian product in x
// For a cotangent e_i of a_i = sum_j k_ij b_j (E signal columns):
// w = 2^(-ks d) <e_i, b_j>,  G_k += w (x_k - y_k);  the x-gradient of
// L = sum_i <e_i, a_i> is -G * gscale.  Rows hold x_i and this E-slice of
// e_i; columns hold (y_j, the same E-slice of b_j), packed as for the sums.
// The product is linear in <e_i, b_j>, so E-slices after the first add to
// the output.
template <int DP, int EP, int R>
__global__ __launch_bounds__(kThreads) void vjp_kernel(DirectArgs a) {
  constexpr int S = DP + EP;
  __shared__ float4 lds[2 * Tile<S>::TJ * Tile<S>::SP / 4];
  const Item it = item_of<R>(a);
  if (!it.live) return;
  float xr[R][DP];
  load_rows<DP, R>(a, it, xr);
  float er[R][EP];
  const int Ec = min(EP, a.E - a.e0);
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int64_t row = row_at(it, r, threadIdx.x);
    const bool ok = row < it.row_end;
#pragma unroll
    for (int e = 0; e < EP; ++e) er[r][e] = (ok && e < Ec) ? a.xe[row * a.E + a.e0 + e] : 0.0f;
  }
  float tot[R][DP], part[R][DP];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int k = 0; k < DP; ++k) tot[r][k] = part[r][k] = 0.0f;

  stream_item<S>(
      a, it, 0, lds,
      [&](const float* yv, int64_t) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
          float t[DP];
          float d = 0.0f;
#pragma unroll
          for (int k = 0; k < DP; ++k) {
            t[k] = xr[r][k] - yv[k];
            d = (k == 0) ? t[0] * t[0] : __builtin_fmaf(t[k], t[k], d);
          }
          float dot = er[r][0] * yv[DP];
#pragma unroll
          for (int e = 1; e < EP; ++e) dot = __builtin_fmaf(er[r][e], yv[DP + e], dot);
          const float w = fast_exp2(-(a.kscale * d)) * dot;
#pragma unroll
          for (int k = 0; k < DP; ++k) part[r][k] = __builtin_fmaf(w, t[k], part[r][k]);
        }
      },
      [&]() {
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
          for (int k = 0; k < DP; ++k) {
            tot[r][k] += part[r][k];
            part[r][k] = 0.0f;
          }
      });

  const int tid_out = opaque_tid();
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int64_t row = row_at(it, r, tid_out);
    if (row >= it.row_end) continue;
    if (a.C == 1) {
      float* o = static_cast<float*>(a.out) + row * a.D;
#pragma unroll
      for (int k = 0; k < DP; ++k)
        if (k < a.D) {
          const float v = -tot[r][k] * a.gscale;
          o[k] = a.accumulate ? o[k] + v : v;
        }
    } else {
      float* p = a.part + ((int64_t)it.c * a.M + row) * DP;
#pragma unroll
      for (int k = 0; k < DP; ++k) p[k] = tot[r][k];
    }
  }
}

__global__ __launch_bounds__(256) void scale_rows_kernel(const float* __restrict__ src, int64_t M,
                                                         int D, const float* __restrict__ e,
                                                         float* __restrict__ dst) {
  const int64_t total = M * D;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = t / D;
    const int k = (int)(t - i * D);
    dst[t] = e[i] * src[i * (1 + D) + 1 + k];
  }
}

// ------------------------------------------------ Sinkhorn log-sum-exp
// In log2 units: s_ij = g'_j - ks d_ij with g' = g log2(e), ks = log2(e) / eps
// (LAP: s_ij = g'_j - ks sqrt(d_ij), ks = log2(e) / sigma).
// Running reference m_i (<= max_j s_ij + kRescale): terms are 2^(s - m);
// when a term would exceed 2^kRescale the sums are rescaled and m moves up.
template <int DP, bool LAP>
__device__ __forceinline__ float lse_dist(const float (&xr)[DP], const float* yv) {
  const float d = sq_dist<DP>(xr, yv);
  if constexpr (LAP) return fast_sqrt(d);
  else return d;
}

template <int DP, int R, bool LAP>
__global__ __launch_bounds__(kThreads) void lse_kernel(DirectArgs a) {
  constexpr int S = DP + 1;
  __shared__ float4 lds[2 * Tile<S>::TJ * Tile<S>::SP / 4];
  if (a.guard != nullptr && fast_frame(a.guard, a.D, a.fscale, a.flimit).ok) return;
  const Item it = item_of<R>(a);
  if (!it.live) return;
  float xr[R][DP];
  load_rows<DP, R>(a, it, xr);
  float m[R], tot[R], part[R];
  const int64_t jf = first_column(a, it);
  if (jf >= 0) {
    // the item's first column sets the reference: its term is 2^0 = 1
    const float* y0 = a.ypk + jf * S;
    float yv[S];
#pragma unroll
    for (int s = 0; s < S; ++s) yv[s] = y0[s];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      m[r] = __builtin_fmaf(-a.kscale, lse_dist<DP, LAP>(xr[r], yv), yv[DP]);
      tot[r] = 0.0f;
      part[r] = 1.0f;
    }
  } else {
    // no columns: the empty sum, log 0 = -infinity
#pragma unroll
    for (int r = 0; r < R; ++r) {
      m[r] = -__builtin_inff();
      tot[r] = part[r] = 0.0f;
    }
  }

  stream_item<S>(
      a, it, 1, lds,
      [&](const float* yv, int64_t) {
        float uu[R];
        bool big = false;
#pragma unroll
        for (int r = 0; r < R; ++r) {
          const float u = __builtin_fmaf(-a.kscale, lse_dist<DP, LAP>(xr[r], yv), yv[DP] - m[r]);
          uu[r] = u;
          big |= (u > kRescale);
        }
        __builtin_amdgcn_sched_barrier(0);
        if (__builtin_expect(big, 0)) {
#pragma unroll
          for (int r = 0; r < R; ++r)
            if (uu[r] > kRescale) {
              const float f = fast_exp2(-uu[r]);
              part[r] *= f;
              tot[r] *= f;
              m[r] += uu[r];
              uu[r] = 0.0f;
            }
        }
#pragma unroll
        for (int r = 0; r < R; ++r) part[r] += fast_exp2(uu[r]);
      },
      [&]() {
#pragma unroll
        for (int r = 0; r < R; ++r) {
          tot[r] += part[r];
          part[r] = 0.0f;
        }
      });
#pragma unroll
  for (int r = 0; r < R; ++r) tot[r] += part[r];

  const int tid_out = opaque_tid();
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int64_t row = row_at(it, r, tid_out);
    if (row >= it.row_end) continue;
    if (a.C == 1) {
      static_cast<float*>(a.out)[row] = (m[r] + fast_log2(tot[r])) * kLn2;
    } else {
      float* p = a.part + ((int64_t)it.c * a.M + row) * 2;
      p[0] = m[r];
      p[1] = tot[r];
    }
  }
}

// ------------------------------------------------- min / max / arg-min / arg-max
// Minimum over j of f = sign * F_ije with the lowest index on ties (the max
// of F is the min of -F; the sign is folded into the packed b and kscale):
//   Gauss / Laplace / squared distance: f = kernel(d) * (sign b_je)
//   log-sum-exp formula:                f = (sign g_j) - (sign / eps) d
// Columns are visited in increasing j and the compare is strict, so a later
// equal value never replaces an earlier one.  Partials are (f, j) pairs.
template <int F, int DP, int EP, int R>
__global__ __launch_bounds__(kThreads) void extreme_kernel(DirectArgs a) {
  constexpr int S = DP + EP;
  __shared__ float4 lds[2 * Tile<S>::TJ * Tile<S>::SP / 4];
  const Item it = item_of<R>(a);
  if (!it.live) return;
  float xr[R][DP];
  load_rows<DP, R>(a, it, xr);
  float best[R][EP];
  int bj[R][EP];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int e = 0; e < EP; ++e) {
      best[r][e] = __builtin_inff();
      bj[r][e] = -1;
    }
  const float ks = a.kscale;

  stream_item<S>(
      a, it, 0, lds,
      [&](const float* yv, int64_t j) {
        float d[R];
#pragma unroll
        for (int r = 0; r < R; ++r) d[r] = sq_dist<DP>(xr[r], yv);
#pragma unroll
        for (int r = 0; r < R; ++r) {
          if constexpr (F == F_SINKHORN) {
            const float f = __builtin_fmaf(-ks, d[r], yv[DP]);
            if (f < best[r][0]) {
              best[r][0] = f;
              bj[r][0] = (int)j;
            }
          } else {
            const float k = kernel_of<F>(d[r], ks);
#pragma unroll
            for (int e = 0; e < EP; ++e) {
              const float f = k * yv[DP + e];
              if (f < best[r][e]) {
                best[r][e] = f;
                bj[r][e] = (int)j;
              }
            }
          }
        }
      },
      [&]() {});

  const int Ec = min(EP, a.E - a.e0);
  const int tid_out = opaque_tid();
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int64_t row = row_at(it, r, tid_out);
    if (row >= it.row_end) continue;
    if (a.C == 1) {
#pragma unroll
      for (int e = 0; e < EP; ++e)
        if (e < Ec) {
          if (a.arg) static_cast<int*>(a.out)[row * a.E + a.e0 + e] = bj[r][e];
          else static_cast<float*>(a.out)[row * a.E + a.e0 + e] = a.ext_sign * best[r][e];
        }
    } else {
      float* p = a.part + ((int64_t)it.c * a.M + row) * (2 * EP);
#pragma unroll
      for (int e = 0; e < EP; ++e) {
        p[2 * e] = best[r][e];
        p[2 * e + 1] = __int_as_float(bj[r][e]);
      }
    }
  }
}

// ------------------------------------------------------------ arg-K-min
// Per row a sorted register list of the KP smallest (d, j) seen; columns are
// visited in increasing j, so a later equal distance never displaces an
// earlier one: the strict compare d < list gives the (distance, index) order.
template <int KP>
__device__ __forceinline__ void knn_insert(float (&dk)[KP], int (&jk)[KP], float d, int j) {
#pragma unroll
  for (int p = KP - 1; p > 0; --p) {
    const bool shift = d < dk[p - 1];
    const bool here = !shift && d < dk[p];
    dk[p] = shift ? dk[p - 1] : (here ? d : dk[p]);
    jk[p] = shift ? jk[p - 1] : (here ? j : jk[p]);
  }
  if (d < dk[0]) {
    dk[0] = d;
    jk[0] = j;
  }
}

template <int DP, int KP, int R>
__global__ __launch_bounds__(kThreads) void knn_kernel(DirectArgs a) {
  constexpr int S = DP + 1;   // the prologue pads one zero signal column
  __shared__ float4 lds[2 * Tile<S>::TJ * Tile<S>::SP / 4];
  if (a.guard != nullptr && fast_frame(a.guard, a.D, a.fscale, a.flimit).ok) return;   // K = 1 on the fast path
  const Item it = item_of<R>(a);
  if (!it.live) return;
  float xr[R][DP];
  load_rows<DP, R>(a, it, xr);
  float dk[R][KP];
  int jk[R][KP];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int p = 0; p < KP; ++p) {
      dk[r][p] = __builtin_inff();
      jk[r][p] = INT_MAX;
    }

  stream_item<S>(
      a, it, 0, lds,
      [&](const float* yv, int64_t j) {
        float d[R];
        bool any = false;
#pragma unroll
        for (int r = 0; r < R; ++r) {
          d[r] = sq_dist<DP>(xr[r], yv);
          any |= d[r] < dk[r][KP - 1];
        }
        if (__builtin_expect(any, 0)) {
#pragma unroll
          for (int r = 0; r < R; ++r)
            if (d[r] < dk[r][KP - 1]) knn_insert<KP>(dk[r], jk[r], d[r], (int)j);
        }
      },
      [&]() {});

  const int tid_out = opaque_tid();
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int64_t row = row_at(it, r, tid_out);
    if (row >= it.row_end) continue;
    if (a.C == 1) {
      if (a.kvalues) {
        float* o = static_cast<float*>(a.out) + row * a.K;
#pragma unroll
        for (int p = 0; p < KP; ++p)
          if (p < a.K) o[p] = dk[r][p];
      } else {
        int* o = static_cast<int*>(a.out) + row * a.K;
#pragma unroll
        for (int p = 0; p < KP; ++p)
          if (p < a.K) o[p] = jk[r][p] == INT_MAX ? -1 : jk[r][p];
      }
    } else {
      float* q = a.part + ((int64_t)it.c * a.M + row) * (2 * KP);
#pragma unroll
      for (int p = 0; p < KP; ++p) {
        q[2 * p] = dk[r][p];
        q[2 * p + 1] = __int_as_float(jk[r][p]);
      }
    }
  }
}

// ------------------------------------------------------------- dispatch
// Rows per lane: as many as fit a budget of VGPRs of per-row state.  Wide
// signals (16 columns) get a larger budget: each column's LDS read then
// serves at least two rows, which outweighs the lower occupancy.
constexpr int kStateBudget = 48;
constexpr int kWideStateBudget = 96;

constexpr int pow2_floor(int v) { return v >= 8 ? 8 : v >= 4 ? 4 : v >= 2 ? 2 : 1; }

constexpr int rows_for(int formula, int DP, int EP, int KP) {
  const int state = formula == F_GRADX      ? DP + 2 * (DP + 1)
                    : formula == F_VJP      ? DP + EP + 2 * DP
                    : (formula == F_SINKHORN || formula == F_LAPLACE_LSE) ? DP + 3
                    : KP > 0                ? DP + 2 * KP
                                            : DP + 2 * EP;
  const int budget = (EP >= 16 && KP == 0) ? kWideStateBudget : kStateBudget;
  return pow2_floor(budget / state > 0 ? budget / state : 1);
}

// The sums come in two row counts: the default, and 2 rows per thread for
// small M, where the default's few row blocks would leave CUs idle.
constexpr int kSmallRows = 2;

template <int F, int DP, int EP>
void launch_sum_f(const DirectArgs& a, dim3 grid, hipStream_t s) {
  constexpr int R = rows_for(F, DP, EP, 0);
  if (R > kSmallRows && a.rows == kSmallRows)
    hipLaunchKernelGGL((sum_kernel<F, DP, EP, (R > kSmallRows ? kSmallRows : R)>), grid,
                       dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL((sum_kernel<F, DP, EP, R>), grid, dim3(kThreads), 0, s, a);
}

template <int DP, int EP>
hipError_t launch_sum_e(const DirectArgs& a, dim3 grid, hipStream_t s) {
  switch (a.formula) {
    case F_GAUSS:
      launch_sum_f<F_GAUSS, DP, EP>(a, grid, s);
      break;
    case F_LAPLACE:
      launch_sum_f<F_LAPLACE, DP, EP>(a, grid, s);
      break;
    case F_SQDIST:
      launch_sum_f<F_SQDIST, DP, EP>(a, grid, s);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int DP, int EP>
hipError_t launch_ext_e(const DirectArgs& a, dim3 grid, hipStream_t s) {
  constexpr int R = rows_for(F_SQDIST, DP, EP, 0);   // same per-row state as the sums
  switch (a.formula) {
    case F_GAUSS:
      hipLaunchKernelGGL((extreme_kernel<F_GAUSS, DP, EP, R>), grid, dim3(kThreads), 0, s, a);
      break;
    case F_LAPLACE:
      hipLaunchKernelGGL((extreme_kernel<F_LAPLACE, DP, EP, R>), grid, dim3(kThreads), 0, s, a);
      break;
    case F_SQDIST:
      hipLaunchKernelGGL((extreme_kernel<F_SQDIST, DP, EP, R>), grid, dim3(kThreads), 0, s, a);
      break;
    case F_SINKHORN:
      if constexpr (EP == 1) {
        hipLaunchKernelGGL((extreme_kernel<F_SINKHORN, DP, 1, R>), grid, dim3(kThreads), 0, s, a);
        break;
      }
      return hipErrorInvalidValue;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int DP>
hipError_t launch_dp(const DirectArgs& a, dim3 grid, hipStream_t s) {
  if (a.ext) {
    switch (a.EP) {
      case 1: return launch_ext_e<DP, 1>(a, grid, s);
      case 4: return launch_ext_e<DP, 4>(a, grid, s);
      case 16: return launch_ext_e<DP, 16>(a, grid, s);
      default: return hipErrorInvalidValue;
    }
  }
  if (a.KP > 0) {
    switch (a.KP) {
#define KRED_KNN(KPV)                                                                           \
  case KPV:                                                                                    \
    hipLaunchKernelGGL((knn_kernel<DP, KPV, rows_for(F_SQDIST, DP, 1, KPV)>), grid,           \
                       dim3(kThreads), 0, s, a);                                               \
    return hipGetLastError();
      KRED_KNN(1) KRED_KNN(4) KRED_KNN(16) KRED_KNN(64)
#undef KRED_KNN
      default:
        return hipErrorInvalidValue;
    }
  }
  switch (a.formula) {
    case F_GRADX:
      hipLaunchKernelGGL((gradx_kernel<DP, rows_for(F_GRADX, DP, 1, 0)>), grid, dim3(kThreads),
                         0, s, a);
      return hipGetLastError();
    case F_SINKHORN:
      hipLaunchKernelGGL((lse_kernel<DP, rows_for(F_SINKHORN, DP, 1, 0), false>), grid,
                         dim3(kThreads), 0, s, a);
      return hipGetLastError();
    case F_LAPLACE_LSE:
      hipLaunchKernelGGL((lse_kernel<DP, rows_for(F_LAPLACE_LSE, DP, 1, 0), true>), grid,
                         dim3(kThreads), 0, s, a);
      return hipGetLastError();
    case F_VJP:
      switch (a.EP) {
#define KRED_VJP(EPV)                                                                           \
  case EPV:                                                                                    \
    hipLaunchKernelGGL((vjp_kernel<DP, EPV, rows_for(F_VJP, DP, EPV, 0)>), grid, dim3(kThreads), \
                       0, s, a);                                                               \
    return hipGetLastError();
        KRED_VJP(1) KRED_VJP(4) KRED_VJP(16)
#undef KRED_VJP
        default:
          return hipErrorInvalidValue;
      }
    default:
      switch (a.EP) {
        case 1: return launch_sum_e<DP, 1>(a, grid, s);
        case 4: return launch_sum_e<DP, 4>(a, grid, s);
        case 16: return launch_sum_e<DP, 16>(a, grid, s);
        default: return hipErrorInvalidValue;
      }
  }
}

}  // namespace

int direct_pad_d(int D) {
  if (D >= 1 && D <= 4) return D;
  if (D <= 8) return 8;
  if (D <= 16) return 16;
  return 0;
}

int direct_pad_e(int E) { return E <= 1 ? 1 : (E <= 4 ? 4 : 16); }

int knn_pad_k(int K) { return K <= 1 ? 1 : (K <= 4 ? 4 : (K <= 16 ? 16 : 64)); }

int direct_rows_per_thread(int formula, int DP, int EP, int KP) {
  return rows_for(formula, DP, EP, KP);
}

int direct_sum_rows(int formula, int DP, int EP, int KP, int ext, int64_t M, int64_t N,
                    int num_cus) {
  const int R = ext ? rows_for(F_SQDIST, DP, EP, 0) : rows_for(formula, DP, EP, KP);
  const bool sum = !ext && KP == 0 &&
                   (formula == F_GAUSS || formula == F_LAPLACE || formula == F_SQDIST);
  if (!sum || R <= kSmallRows) return R;
  // the default grid's work items at the largest useful column split
  const int64_t rb = (M + (int64_t)kThreads * R - 1) / ((int64_t)kThreads * R);
  const int64_t cmax = std::max<int64_t>(1, std::min<int64_t>(KRED_MAX_COL_BLOCKS, N / 128));
  return rb * cmax < 4 * (int64_t)num_cus ? kSmallRows : R;
}

int partial_width(int formula, int DP, int EP, int KP, int ext) {
  if (KP > 0) return 2 * KP;
  if (ext) return 2 * EP;
  if (formula == F_GRADX) return DP + 1;
  if (formula == F_VJP) return DP;
  if (formula == F_SINKHORN || formula == F_LAPLACE_LSE) return 2;
  return EP;
}

hipError_t launch_pack(const PackArgs& a, hipStream_t s) {
  const int64_t total = a.N * (a.DP + a.EP);
  if (total == 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(pack_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_scale_rows(const float* src, int64_t M, int D, const float* e, float* dst,
                             hipStream_t s) {
  const int64_t total = M * D;
  if (total == 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(scale_rows_kernel, dim3((unsigned)blocks), dim3(256), 0, s, src, M, D, e, dst);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void range_blocks_kernel(const int* __restrict__ rr, int nr,
                                                           int64_t M, int rpb,
                                                           int* __restrict__ bstart) {
  // one workgroup: each thread counts a contiguous chunk of clusters, the 256
  // chunk totals are scanned in LDS, then each thread writes its prefixes
  __shared__ int tot[256];
  const int t = threadIdx.x;
  const int chunk = (nr + 255) / 256;
  const int c0 = min(nr, t * chunk), c1 = min(nr, c0 + chunk);
  auto blocks = [&](int I) {
    const int64_t r0 = min(max((int64_t)rr[2 * I], (int64_t)0), M);
    const int64_t r1 = min(max((int64_t)rr[2 * I + 1], r0), M);
    return (int)((r1 - r0 + rpb - 1) / rpb);
  };
  int sum = 0;
  for (int I = c0; I < c1; ++I) sum += blocks(I);
  tot[t] = sum;
  __syncthreads();
  for (int o = 1; o < 256; o <<= 1) {
    const int v = t >= o ? tot[t - o] : 0;
    __syncthreads();
    tot[t] += v;
    __syncthreads();
  }
  int run = t > 0 ? tot[t - 1] : 0;
  for (int I = c0; I < c1; ++I) {
    bstart[I] = run;
    run += blocks(I);
  }
  if (t == 255) bstart[nr] = tot[255];
}

hipError_t launch_range_blocks(const int* rr, int nr, int64_t M, int rows_per_block, int* bstart,
                               hipStream_t s) {
  hipLaunchKernelGGL(range_blocks_kernel, dim3(1), dim3(256), 0, s, rr, nr, M, rows_per_block,
                     bstart);
  return hipGetLastError();
}

int64_t range_grid_bound(int nr, int64_t M, int rows_per_block) {
  return (int64_t)nr + (M + rows_per_block - 1) / rows_per_block;
}

hipError_t launch_fill2(float* out, int64_t count, float v0, float v1, hipStream_t s) {
  if (count == 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((count + 255) / 256, 8192);
  hipLaunchKernelGGL(fill2_kernel, dim3((unsigned)blocks), dim3(256), 0, s, out, count, v0, v1);
  return hipGetLastError();
}

hipError_t launch_fill(float* out, int64_t count, float value, hipStream_t s) {
  if (count == 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((count + 255) / 256, 8192);
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(256), 0, s, out, count, value);
  return hipGetLastError();
}

int direct_rows_for(const DirectArgs& a) {
  const int R = a.ext ? direct_rows_per_thread(F_SQDIST, a.DP, a.EP, 0)
                      : direct_rows_per_thread(a.formula, a.DP, a.EP, a.KP);
  return (a.rows == kSmallRows && R > kSmallRows) ? kSmallRows : R;
}

hipError_t launch_direct(const DirectArgs& a, hipStream_t s) {
  const int R = direct_rows_for(a);
  const int64_t rb = (a.M + (int64_t)kThreads * R - 1) / ((int64_t)kThreads * R);
  const dim3 grid((unsigned)((a.nr > 0 ? range_grid_bound(a.nr, a.M, kThreads * R) : rb) * a.C));
  switch (a.DP) {
    case 1: return launch_dp<1>(a, grid, s);
    case 2: return launch_dp<2>(a, grid, s);
    case 3: return launch_dp<3>(a, grid, s);
    case 4: return launch_dp<4>(a, grid, s);
    case 8: return launch_dp<8>(a, grid, s);
    case 16: return launch_dp<16>(a, grid, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace kred
