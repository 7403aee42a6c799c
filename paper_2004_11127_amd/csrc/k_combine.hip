// Second pass over column-block partials (when the j range was split into C
// blocks to give a small-M problem enough workgroups).  Each partial is the
// reduction of Eq. (2) over one block of columns; this pass applies the same
// reduction across blocks in a fixed order (so results are reproducible run
// to run; the sums interleave four lanes per element, see combine_sum_kernel):
//   sum:          a = sum_c a_c  (also the x-gradient sums of the Gaussian
//                 vector-Jacobian product, scaled by -1/sigma^2)
//   log-sum-exp:  (m, s) = (max_c m_c, sum_c s_c 2^(m_c - m)),  a = (m + log2 s) ln 2
//   arg-K-min:    merge the C sorted (distance, index) lists, keep the K first.
// The second pass reads C x M x W floats once; it is HBM-bound.
#include "kred_internal.h"

#include <climits>

namespace kred {
namespace {

// Four lanes per output element: lane q of a group sums the blocks c = q,
// q + 4, q + 8, ... in increasing order (four loads in flight), and the group
// then adds its four sums as (s0 + s1) + (s2 + s3).  The order is fixed, so
// results repeat run to run; the group's lanes share t and leave the loop
// together, so the shuffles see the whole group.
__global__ __launch_bounds__(256) void combine_sum_kernel(CombineArgs a) {
  const int Ec = min(a.EP, a.E - a.e0);
  const int64_t total = a.M * Ec;
  const int q = threadIdx.x & 3;
  const int64_t st = a.M * a.EP;   // floats between consecutive blocks
  for (int64_t t = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 2; t < total;
       t += ((int64_t)gridDim.x * blockDim.x) >> 2) {
    const int64_t row = t / Ec;
    const int e = (int)(t - row * Ec);
    const float* p = a.part + row * a.EP + e;
    float s = 0.0f;
    int c = q;
    for (; c + 12 < a.C; c += 16) {
      const float v0 = p[c * st], v1 = p[(c + 4) * st], v2 = p[(c + 8) * st], v3 = p[(c + 12) * st];
      s += v0;
      s += v1;
      s += v2;
      s += v3;
    }
    for (; c < a.C; c += 4) s += p[c * st];
    s += __shfl_xor(s, 1);
    s += __shfl_xor(s, 2);
    if (q == 0) static_cast<float*>(a.out)[row * a.E + a.e0 + e] = s;
  }
}

__global__ __launch_bounds__(256) void combine_gradx_kernel(CombineArgs a) {
  const int W = a.DP + 1;
  const int64_t total = a.M * (1 + a.D);
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = t / (1 + a.D);
    const int w = (int)(t - row * (1 + a.D));
    float s = 0.0f;
    for (int c = 0; c < a.C; ++c) s += a.part[((int64_t)c * a.M + row) * W + w];
    static_cast<float*>(a.out)[t] = (w == 0) ? s : -s * a.gscale;
  }
}

// vector-Jacobian product in x: partials are the DP sums G_k; out = -G * gscale
__global__ __launch_bounds__(256) void combine_vjp_kernel(CombineArgs a) {
  const int64_t total = a.M * a.D;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = t / a.D;
    const int k = (int)(t - row * a.D);
    float s = 0.0f;
    for (int c = 0; c < a.C; ++c) s += a.part[((int64_t)c * a.M + row) * a.DP + k];
    float* o = static_cast<float*>(a.out) + t;
    const float v = -s * a.gscale;
    *o = a.accumulate ? *o + v : v;
  }
}

__global__ __launch_bounds__(256) void combine_lse_kernel(CombineArgs a) {
  for (int64_t row = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; row < a.M;
       row += (int64_t)gridDim.x * blockDim.x) {
    float m = -__builtin_inff();
    for (int c = 0; c < a.C; ++c) m = fmaxf(m, a.part[((int64_t)c * a.M + row) * 2]);
    float s = 0.0f;
    for (int c = 0; c < a.C; ++c) {
      const float* p = a.part + ((int64_t)c * a.M + row) * 2;
      if (p[0] == -__builtin_inff()) continue;   // an empty block (its sum is 0)
      s += p[1] * __builtin_amdgcn_exp2f(p[0] - m);
    }
    static_cast<float*>(a.out)[row] = (m + __builtin_amdgcn_logf(s)) * kLn2;
  }
}

// (d, j) strictly before (d2, j2) in (distance, index) order.
__device__ __forceinline__ bool before(float d, int j, float d2, int j2) {
  return d < d2 || (d == d2 && j < j2);
}

template <int KP>
__global__ __launch_bounds__(256) void combine_knn_kernel(CombineArgs a) {
  for (int64_t row = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; row < a.M;
       row += (int64_t)gridDim.x * blockDim.x) {
    float dk[KP];
    int jk[KP];
#pragma unroll
    for (int p = 0; p < KP; ++p) {
      dk[p] = __builtin_inff();
      jk[p] = INT_MAX;
    }
    for (int c = 0; c < a.C; ++c) {
      const float* q = a.part + ((int64_t)c * a.M + row) * (2 * KP);
      for (int i = 0; i < KP; ++i) {
        const float d = q[2 * i];
        const int j = __float_as_int(q[2 * i + 1]);
        if (!before(d, j, dk[KP - 1], jk[KP - 1])) break;   // each list is sorted
#pragma unroll
        for (int p = KP - 1; p > 0; --p) {
          const bool shift = before(d, j, dk[p - 1], jk[p - 1]);
          const bool here = !shift && before(d, j, dk[p], jk[p]);
          dk[p] = shift ? dk[p - 1] : (here ? d : dk[p]);
          jk[p] = shift ? jk[p - 1] : (here ? j : jk[p]);
        }
        if (before(d, j, dk[0], jk[0])) {
          dk[0] = d;
          jk[0] = j;
        }
      }
    }
    if (a.rx != nullptr) {
      // large-D lists rank by the expanded form, whose error is absolute (about
      // 2^-24 (|x|^2 + |y|^2) per term): the merged candidates get their
      // direct-form distance, accurate relative to itself (exact on integer
      // data), and are ordered again by (distance, index)
      const float* xr = a.rx + row * a.rD;
#pragma unroll
      for (int p = 0; p < KP; ++p) {
        if (jk[p] == INT_MAX) continue;
        const float* yr = a.ry + (int64_t)jk[p] * a.rD;
        float s = 0.0f;
        for (int d = 0; d < a.rD; ++d) {
          const float t = xr[d] - yr[d];
          s = __builtin_fmaf(t, t, s);
        }
        dk[p] = s;
      }
      // insertion sort by (distance, index); the unfilled entries (+inf, INT_MAX) stay last
      for (int p = 1; p < KP; ++p)
        for (int q = p; q > 0 && before(dk[q], jk[q], dk[q - 1], jk[q - 1]); --q) {
          const float td = dk[q]; dk[q] = dk[q - 1]; dk[q - 1] = td;
          const int tj = jk[q]; jk[q] = jk[q - 1]; jk[q - 1] = tj;
        }
    }
    if (a.kvalues) {
      // the expanded form can round a zero distance to a tiny negative value
      float* o = static_cast<float*>(a.out) + row * a.K;
#pragma unroll
      for (int p = 0; p < KP; ++p)
        if (p < a.K) o[p] = fmaxf(dk[p], 0.0f);
    } else {
      int* o = static_cast<int*>(a.out) + row * a.K;
#pragma unroll
      for (int p = 0; p < KP; ++p)
        if (p < a.K) o[p] = jk[p] == INT_MAX ? -1 : jk[p];   // short (block-sparse) lists
    }
  }
}

// min / max: partials are (sign * value, index) pairs; keep the smallest in
// (value, index) order, so equal values keep the lowest index.
__global__ __launch_bounds__(256) void combine_extreme_kernel(CombineArgs a) {
  const int Ec = min(a.EP, a.E - a.e0);
  const int64_t total = a.M * Ec;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = t / Ec;
    const int e = (int)(t - row * Ec);
    float v = __builtin_inff();
    int j = -1;
    for (int c = 0; c < a.C; ++c) {
      const float* p = a.part + ((int64_t)c * a.M + row) * (2 * a.EP) + 2 * e;
      const int pj = __float_as_int(p[1]);
      if (pj >= 0 && (j < 0 || p[0] < v || (p[0] == v && pj < j))) {
        v = p[0];
        j = pj;
      }
    }
    const int64_t o = row * a.E + a.e0 + e;
    if (a.arg) static_cast<int*>(a.out)[o] = j;
    else static_cast<float*>(a.out)[o] = a.ext_sign * v;
  }
}

unsigned grid_for(int64_t items) {
  const int64_t b = (items + 255) / 256;
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>(b, 16384));
}

}  // namespace

hipError_t launch_combine(const CombineArgs& a, hipStream_t s) {
  if (a.M == 0) return hipSuccess;
  if (a.ext) {
    hipLaunchKernelGGL(combine_extreme_kernel, dim3(grid_for(a.M * a.EP)), dim3(256), 0, s, a);
    return hipGetLastError();
  }
  if (a.KP > 0) {
    const dim3 g(grid_for(a.M));
    switch (a.KP) {
      case 1: hipLaunchKernelGGL(combine_knn_kernel<1>, g, dim3(256), 0, s, a); break;
      case 4: hipLaunchKernelGGL(combine_knn_kernel<4>, g, dim3(256), 0, s, a); break;
      case 8: hipLaunchKernelGGL(combine_knn_kernel<8>, g, dim3(256), 0, s, a); break;
      case 10: hipLaunchKernelGGL(combine_knn_kernel<10>, g, dim3(256), 0, s, a); break;
      case 12: hipLaunchKernelGGL(combine_knn_kernel<12>, g, dim3(256), 0, s, a); break;
      case 16: hipLaunchKernelGGL(combine_knn_kernel<16>, g, dim3(256), 0, s, a); break;
      case 64: hipLaunchKernelGGL(combine_knn_kernel<64>, g, dim3(256), 0, s, a); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  switch (a.formula) {
    case F_GRADX:
      hipLaunchKernelGGL(combine_gradx_kernel, dim3(grid_for(a.M * (1 + a.D))), dim3(256), 0, s, a);
      break;
    case F_SINKHORN:
    case F_LAPLACE_LSE:
      hipLaunchKernelGGL(combine_lse_kernel, dim3(grid_for(a.M)), dim3(256), 0, s, a);
      break;
    case F_VJP:
      hipLaunchKernelGGL(combine_vjp_kernel, dim3(grid_for(a.M * a.D)), dim3(256), 0, s, a);
      break;
    default:
      hipLaunchKernelGGL(combine_sum_kernel, dim3(grid_for(4 * a.M * a.EP)), dim3(256), 0, s, a);
      break;
  }
  return hipGetLastError();
}

}  // namespace kred
