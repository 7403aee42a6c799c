// Latency-bound Gaussian sums in one launch: a_i = sum_j exp(-|x_i - y_j|^2 /
// (2 sigma^2)) b_j (Eq. (1)) for D <= 4 coordinates and E <= 4 signal columns
// on problems below 2^28 pairs, where the pack pass, the separate combine and
// their launches cost as much as the pairs themselves.
//
// A workgroup owns 128 rows (4 waves x 2 blocks of 16) and a block of at most
// 1024 columns, which it reads straight from y and b into LDS: there is no
// prologue pass.  The pair term comes from the matrix cores in the expanded
// form on coordinates centred on the midpoint m of the workgroup's column
// bounding box and scaled by s = sqrt(c), c = log2(e) / (2 sigma^2), with X,
// Y and the norms nx = -|X|^2, ny = -|Y|^2 formed in fp64 and rounded once.
// For D <= 3 one v_mfma_f32_16x16x4_f32 returns T itself: A holds (2 Y, ny)
// and B (X, 1), the accumulator starts at nx, and the instruction adds its
// four products in order (each addition rounded): four roundings of partial
// sums below 2 L, the products' below u L, the coordinates' 4 u L and the
// norms' 2 u L bound the error in T by 15 u L, u = 2^-24, L = c (max_i |x_i -
// m|^2 + max_j |y_j - m|^2) over the workgroup's rows and columns.  For D = 4,
// T = fl(2 P + fl(nx + ny)) with P = sum_k Y_k X_k from zero, the large-D
// kernels' (D + 10) u L.  Each workgroup computes its own L; above the budget it takes T
// in the direct form -sum_k (X_k - Y_k)^2 on the same coordinates instead, so
// no pass over the whole data precedes the sums.  The result's lane layout,
// T[column 4 g + r][row li] in lane 16 g + li, is shared by both forms; p =
// 2^T is multiplied by b on the VALU.
//
// With C > 1 column blocks, each workgroup writes its partial sums and the
// last one of its row block to arrive (a device-scope counter per row block)
// adds the C partials in block order, writes the output and resets the
// counter to zero for the next call.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "kred_internal.h"

namespace kred {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

template <int D, int E>
__global__ __launch_bounds__(256) void small_sum_kernel(SmallArgs a) {
  constexpr int RB = kSumRows / 64;   // 16-row blocks per wave
  static_assert(RB >= 1 && kSumRows == 64 * RB, "four waves of 16 RB rows");
  // D <= 3: the column norm rides in the fourth K slot and the row norm in
  // the accumulator, so the matrix cores return T itself
  constexpr bool FOLD = D <= 3;
  __shared__ float ys[4][kSumCols];   // Y by coordinate (coordinates >= D zero)
  __shared__ float nys[D <= 3 ? 1 : kSumCols];   // D = 4 only
  __shared__ float bsh[E][kSumCols];
  __shared__ float bbox[4][8];          // per wave: D lows, then D highs
  __shared__ double spread[4][2];       // per wave: max |x - m|^2, max |y - m|^2
  __shared__ int last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int li = lane & 15, g = lane >> 4;
  const int rbk = blockIdx.x / a.C, cb = blockIdx.x - rbk * a.C;
  const int64_t j0 = (int64_t)cb * a.jpb;
  const int ncol = (int)min((int64_t)a.jpb, a.N - j0);   // at least 1 (host plan)
  const int ncol16 = (ncol + 15) & ~15;
  const int64_t i0 = (int64_t)rbk * kSumRows;

  // every global load of the prologue is issued at once, from in-range
  // addresses (indices clamped to the last column and row; the values of
  // clamped ones are replaced below): the thread's (at most four) columns of
  // y and b, and the lane's rows of x
  constexpr int JT = kSumCols / 256;
  float yv[JT][D], bv[JT][E], xv[RB][D];
#pragma unroll
  for (int q = 0; q < JT; ++q) {
    const int64_t j = j0 + min(tid + 256 * q, ncol - 1);
#pragma unroll
    for (int k = 0; k < D; ++k) yv[q][k] = a.y[j * D + k];
#pragma unroll
    for (int e = 0; e < E; ++e) bv[q][e] = a.b[j * E + e];
  }
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int64_t i = min(i0 + 16 * RB * wave + 16 * rb + li, a.M - 1);
#pragma unroll
    for (int k = 0; k < D; ++k) xv[rb][k] = a.x[i * D + k];
  }

  // the centre: midpoint of the bounding box of the workgroup's columns
  float lo[D], hi[D];
#pragma unroll
  for (int k = 0; k < D; ++k) {
    lo[k] = __builtin_inff();
    hi[k] = -__builtin_inff();
  }
#pragma unroll
  for (int q = 0; q < JT; ++q)
    if (tid + 256 * q < ncol) {
#pragma unroll
      for (int k = 0; k < D; ++k) {
        lo[k] = fminf(lo[k], yv[q][k]);
        hi[k] = fmaxf(hi[k], yv[q][k]);
      }
    }
#pragma unroll
  for (int k = 0; k < D; ++k)
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      lo[k] = fminf(lo[k], __shfl_xor(lo[k], o));
      hi[k] = fmaxf(hi[k], __shfl_xor(hi[k], o));
    }
  if (lane == 0) {
#pragma unroll
    for (int k = 0; k < D; ++k) {
      bbox[wave][k] = lo[k];
      bbox[wave][4 + k] = hi[k];
    }
  }
  __syncthreads();
  float m[D];
#pragma unroll
  for (int k = 0; k < D; ++k) {
    const float l = fminf(fminf(bbox[0][k], bbox[1][k]), fminf(bbox[2][k], bbox[3][k]));
    const float h = fmaxf(fmaxf(bbox[0][4 + k], bbox[1][4 + k]), fmaxf(bbox[2][4 + k], bbox[3][4 + k]));
    m[k] = 0.5f * l + 0.5f * h;
  }

  // the column block: Y = fl32(s (y - m)) and ny = -fl32(|Y|^2) from fp64,
  // b; padding columns get Y = 0, ny = -infinity (p = 0) and b = 0
  double sy = 0.0;
#pragma unroll
  for (int q = 0; q < JT; ++q) {
    const int jj = tid + 256 * q;
    if (jj < ncol16) {
      const bool ok = jj < ncol;
      double n2 = 0.0, d2 = 0.0;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        float v = 0.0f;
        if (k < D && ok) {
          const double d = (double)yv[q][k] - (double)m[k];
          d2 = __builtin_fma(d, d, d2);
          v = (float)(d * a.s64);
          n2 = __builtin_fma((double)v, (double)v, n2);
        }
        if (!FOLD || k < 3) ys[k][jj] = FOLD ? 2.0f * v : v;
      }
      const float nyj = ok ? (float)(-n2) : -__builtin_inff();
      if (FOLD) ys[3][jj] = nyj;
      else nys[jj] = nyj;
      sy = fmax(sy, d2);
#pragma unroll
      for (int e = 0; e < E; ++e) bsh[e][jj] = ok ? bv[q][e] : 0.0f;
    }
  }

  // the rows: X of the lane's row li in each 16-row block (all four lane
  // groups hold it; group g supplies coordinate g to the matrix cores)
  float xk[RB][4], nx[RB], xb[RB];
  double sx = 0.0;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const bool ok = i0 + 16 * RB * wave + 16 * rb + li < a.M;
    double n2 = 0.0, d2 = 0.0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      float v = 0.0f;
      if (k < D && ok) {
        const double d = (double)xv[rb][k] - (double)m[k];
        d2 = __builtin_fma(d, d, d2);
        v = (float)(d * a.s64);
        n2 = __builtin_fma((double)v, (double)v, n2);
      }
      xk[rb][k] = v;
    }
    nx[rb] = -(float)n2;
    xb[rb] = g == 0 ? xk[rb][0] : g == 1 ? xk[rb][1] : g == 2 ? xk[rb][2] : (FOLD ? 1.0f : xk[rb][3]);
    if (FOLD) {
#pragma unroll
      for (int k = 0; k < 4; ++k) xk[rb][k] *= 2.0f;   // the direct form on 2 X and 2 Y
    }
    sx = fmax(sx, d2);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    sx = fmax(sx, __shfl_xor(sx, o));
    sy = fmax(sy, __shfl_xor(sy, o));
  }
  if (lane == 0) {
    spread[wave][0] = sx;
    spread[wave][1] = sy;
  }
  __syncthreads();   // also publishes the column block
  sx = fmax(fmax(spread[0][0], spread[1][0]), fmax(spread[2][0], spread[3][0]));
  sy = fmax(fmax(spread[0][1], spread[1][1]), fmax(spread[2][1], spread[3][1]));
  // workgroup-uniform: the expanded form on the matrix cores within the bound
  const bool mc = a.c64 * (sx + sy) * (1.0 + 1.0 / 1048576.0) <= (double)a.limit;

  // p = 2^T times b into the lane's sums, one per column position r of the
  // lane's four (columns 4 g + r of each block): four independent chains
  float acc[RB][E][4];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int e = 0; e < E; ++e)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[rb][e][r] = 0.0f;
  // NB 16-column blocks from column jb: all LDS reads first, then the pair
  // terms of every block, then the exponentials and products (NB = 4 in the
  // loop, 1 for the tail): independent work for the in-order issue of a wave
  auto step = [&](int jb, auto nbc) {
    constexpr int NB = decltype(nbc)::value;
    float4 nv[NB], bq[NB][E];
    f4 T[NB][RB];
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      if (!FOLD) nv[u] = *reinterpret_cast<const float4*>(&nys[jb + 16 * u + 4 * g]);
#pragma unroll
      for (int e = 0; e < E; ++e)
        bq[u][e] = *reinterpret_cast<const float4*>(&bsh[e][jb + 16 * u + 4 * g]);
    }
    if (mc) {
      float ya[NB];
#pragma unroll
      for (int u = 0; u < NB; ++u) ya[u] = ys[g][jb + 16 * u + li];   // A[j = li][k = g]
#pragma unroll
      for (int u = 0; u < NB; ++u)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          if (FOLD) {
            // nx + 2 Y_0 X_0 + 2 Y_1 X_1 + 2 Y_2 X_2 + ny, summed in that order
            T[u][rb] = __builtin_amdgcn_mfma_f32_16x16x4f32(ya[u], xb[rb],
                                                            f4{nx[rb], nx[rb], nx[rb], nx[rb]}, 0, 0, 0);
          } else {
            const f4 P = __builtin_amdgcn_mfma_f32_16x16x4f32(ya[u], xb[rb], f4{0.f, 0.f, 0.f, 0.f},
                                                              0, 0, 0);
            T[u][rb][0] = __builtin_fmaf(2.0f, P[0], nx[rb] + nv[u].x);
            T[u][rb][1] = __builtin_fmaf(2.0f, P[1], nx[rb] + nv[u].y);
            T[u][rb][2] = __builtin_fmaf(2.0f, P[2], nx[rb] + nv[u].z);
            T[u][rb][3] = __builtin_fmaf(2.0f, P[3], nx[rb] + nv[u].w);
          }
        }
    } else {
      float4 yq[NB][D];
#pragma unroll
      for (int u = 0; u < NB; ++u)
#pragma unroll
        for (int k = 0; k < D; ++k)
          yq[u][k] = *reinterpret_cast<const float4*>(&ys[k][jb + 16 * u + 4 * g]);
#pragma unroll
      for (int u = 0; u < NB; ++u)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          float t[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int k = 0; k < D; ++k) {
            const float d0 = xk[rb][k] - yq[u][k].x, d1 = xk[rb][k] - yq[u][k].y;
            const float d2 = xk[rb][k] - yq[u][k].z, d3 = xk[rb][k] - yq[u][k].w;
            t[0] = __builtin_fmaf(d0, d0, t[0]);
            t[1] = __builtin_fmaf(d1, d1, t[1]);
            t[2] = __builtin_fmaf(d2, d2, t[2]);
            t[3] = __builtin_fmaf(d3, d3, t[3]);
          }
          // (FOLD: the coordinates are doubled, 4 times the squared distance)
          constexpr float sc = FOLD ? -0.25f : -1.0f;
          T[u][rb] = f4{sc * t[0], sc * t[1], sc * t[2], sc * t[3]};
        }
    }
#pragma unroll
    for (int u = 0; u < NB; ++u)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        float p[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) p[r] = __builtin_amdgcn_exp2f(T[u][rb][r]);
#pragma unroll
        for (int e = 0; e < E; ++e) {
          acc[rb][e][0] = __builtin_fmaf(p[0], bq[u][e].x, acc[rb][e][0]);
          acc[rb][e][1] = __builtin_fmaf(p[1], bq[u][e].y, acc[rb][e][1]);
          acc[rb][e][2] = __builtin_fmaf(p[2], bq[u][e].z, acc[rb][e][2]);
          acc[rb][e][3] = __builtin_fmaf(p[3], bq[u][e].w, acc[rb][e][3]);
        }
      }
  };
  int jb = 0;
  for (; jb + 64 <= ncol16; jb += 64) step(jb, std::integral_constant<int, 4>{});
  for (; jb < ncol16; jb += 16) step(jb, std::integral_constant<int, 1>{});

  // the four lane groups hold different columns of the same row li
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int e = 0; e < E; ++e) {
      float v = (acc[rb][e][0] + acc[rb][e][1]) + (acc[rb][e][2] + acc[rb][e][3]);
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      const int64_t i = i0 + 16 * RB * wave + 16 * rb + li;
      if (g == 0 && i < a.M) {
        if (a.C == 1) a.out[i * E + e] = v;
        else __hip_atomic_store(&a.part[((int64_t)cb * a.M + i) * E + e], v, __ATOMIC_RELAXED,
                                __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  if (a.C == 1) return;

  // The last workgroup of the row block to arrive adds the C partials.  The
  // partials are device-scope atomic stores and loads (coherent across the
  // XCDs' caches by themselves), so the hand-over needs no cache write-back:
  // every wave waits for its stores to complete (s_waitcnt vmcnt(0)) before
  // the barrier after which the count goes up, and the last workgroup loads
  // them only after it has seen the count reach C - 1.
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (tid == 0)
    last = __hip_atomic_fetch_add(&a.count[rbk], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
           a.C - 1;
  __syncthreads();
  if (!last) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  const int rows = (int)min((int64_t)kSumRows, a.M - i0);
  for (int t = tid; t < rows * E; t += 256) {
    const int64_t i = i0 + t / E;
    const int e = t - (t / E) * E;
    const float* src = a.part + i * E + e;
    const int64_t stride = a.M * E;
    // eight loads in flight at a time, added in block order
    float s = 0.0f;
    for (int c0 = 0; c0 < a.C; c0 += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        v[u] = c0 + u < a.C ? __hip_atomic_load(src + (int64_t)(c0 + u) * stride, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT)
                            : 0.0f;
#pragma unroll
      for (int u = 0; u < 8; ++u) s += v[u];
    }
    a.out[i * E + e] = s;
  }
  if (tid == 0) __hip_atomic_store(&a.count[rbk], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int D>
hipError_t launch_small_d(const SmallArgs& a, dim3 grid, hipStream_t s) {
  switch (a.E) {
    case 1: hipLaunchKernelGGL((small_sum_kernel<D, 1>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((small_sum_kernel<D, 2>), grid, dim3(256), 0, s, a); break;
    case 3: hipLaunchKernelGGL((small_sum_kernel<D, 3>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((small_sum_kernel<D, 4>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_small(const SmallArgs& a, hipStream_t s) {
  const int64_t nrb = (a.M + kSumRows - 1) / kSumRows;
  const dim3 grid((unsigned)(nrb * a.C));
  switch (a.D) {
    case 1: return launch_small_d<1>(a, grid, s);
    case 2: return launch_small_d<2>(a, grid, s);
    case 3: return launch_small_d<3>(a, grid, s);
    case 4: return launch_small_d<4>(a, grid, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace kred
