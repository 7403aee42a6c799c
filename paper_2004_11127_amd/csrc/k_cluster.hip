// Block-sparse truncation pattern built on the device: the cluster-wise
// block-sparsity of Sec. 3 with the block-sparse truncation rule of Sec. 4
// (clusters of x interact only with the clusters of y close enough to matter).
//
//   1. the joint bounding box of x and y (fp64): origin o = the coordinate-wise
//      minimum, dims_d = floor((max_d - o_d) / cell) + 1 cells per axis;
//   2. a cell label per point, k_d = min(floor((p_d - o_d) / cell), dims_d - 1),
//      key = the mixed-radix number of (k_0, .., k_{D-1});
//   3. a stable sort of each cloud by label (the permutation that makes every
//      cluster a contiguous range), its distinct labels and their ranges;
//   4. for each cluster of x, the clusters of y whose cell centres o + (k +
//      1/2) cell lie within cutoff + cell sqrt(D) of its own centre, as
//      column ranges, runs of consecutive kept clusters merged into one.
//
// Every step repeats the host construction's arithmetic in the same order
// and precision (fp64, each operation rounded on its own: this file is
// compiled without contraction into fused multiply-adds), so the arrays are
// bit-identical to it.  The sort and the run-length encoding are
// rocPRIM's device primitives; the rest are the kernels below.
#include <hip/hip_runtime.h>

#include <rocprim/device/device_radix_sort.hpp>
#include <rocprim/device/device_run_length_encode.hpp>
#include <rocprim/device/device_scan.hpp>

#include <algorithm>
#include <cstdint>

#include "kred_internal.h"

namespace kred {
namespace {

constexpr int kBoxBlocks = 256;

// per block, the coordinate-wise minimum and maximum of the rows of x and y
// it visits: part[(blk * 2 + 0) * D + d] = min, part[(blk * 2 + 1) * D + d] = max
__global__ __launch_bounds__(256) void box_partial_kernel(const float* __restrict__ x, int64_t M,
                                                          const float* __restrict__ y, int64_t N,
                                                          int D, double* __restrict__ part) {
  __shared__ double red[2][kClusterMaxD][256];
  double lo[kClusterMaxD], hi[kClusterMaxD];
#pragma unroll
  for (int d = 0; d < kClusterMaxD; ++d) {
    lo[d] = __builtin_inf();
    hi[d] = -__builtin_inf();
  }
  for (int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; r < M + N;
       r += (int64_t)gridDim.x * blockDim.x) {
    const float* p = r < M ? x + r * D : y + (r - M) * D;
#pragma unroll
    for (int d = 0; d < kClusterMaxD; ++d)
      if (d < D) {
        const double v = (double)p[d];
        lo[d] = fmin(lo[d], v);
        hi[d] = fmax(hi[d], v);
      }
  }
#pragma unroll
  for (int d = 0; d < kClusterMaxD; ++d) {
    red[0][d][threadIdx.x] = lo[d];
    red[1][d][threadIdx.x] = hi[d];
  }
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) {
#pragma unroll
      for (int d = 0; d < kClusterMaxD; ++d) {
        red[0][d][threadIdx.x] = fmin(red[0][d][threadIdx.x], red[0][d][threadIdx.x + s]);
        red[1][d][threadIdx.x] = fmax(red[1][d][threadIdx.x], red[1][d][threadIdx.x + s]);
      }
    }
    __syncthreads();
  }
  if ((int)threadIdx.x < D) {
    part[(blockIdx.x * 2 + 0) * D + threadIdx.x] = red[0][threadIdx.x][0];
    part[(blockIdx.x * 2 + 1) * D + threadIdx.x] = red[1][threadIdx.x][0];
  }
}

// the grid: origin and cells per axis
__global__ void box_final_kernel(const double* __restrict__ part, int nparts, int D, double cell,
                                 ClusterGrid* __restrict__ g) {
  const int d = threadIdx.x;
  if (d >= D) return;
  double lo = __builtin_inf(), hi = -__builtin_inf();
  for (int b = 0; b < nparts; ++b) {
    lo = fmin(lo, part[(b * 2 + 0) * D + d]);
    hi = fmax(hi, part[(b * 2 + 1) * D + d]);
  }
  g->origin[d] = lo;
  g->dims[d] = (int64_t)__builtin_floor(__ddiv_rn(__dsub_rn(hi, lo), cell)) + 1;
}

// the cell label of every point (mixed radix, dimension 0 most significant),
// and the identity permutation the sort carries along
__global__ __launch_bounds__(256) void label_kernel(const float* __restrict__ p, int64_t n, int D,
                                                    double cell, const ClusterGrid* __restrict__ g,
                                                    uint64_t* __restrict__ key,
                                                    int32_t* __restrict__ idx) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    uint64_t k = 0;
    for (int d = 0; d < D; ++d) {
      const double t = __builtin_floor(__ddiv_rn(__dsub_rn((double)p[i * D + d], g->origin[d]), cell));
      const int64_t kd = min((int64_t)t, g->dims[d] - 1);
      k = k * (uint64_t)g->dims[d] + (uint64_t)kd;   // two's complement, as the host's int64
    }
    key[i] = k;
    idx[i] = (int32_t)i;
  }
}

// cluster c = [start_c, start_c + count_c) of the sorted order, as int32 pairs
// (clusters from the count up to cap: the empty range [cap, cap), so that a
// caller may pass cap as the number of clusters without reading the count)
__global__ __launch_bounds__(256) void ranges_kernel(const int32_t* __restrict__ start,
                                                     const int32_t* __restrict__ count,
                                                     const int32_t* __restrict__ nclusters,
                                                     int64_t cap, int32_t* __restrict__ ranges) {
  const int64_t nc = *nclusters;
  for (int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; c < cap;
       c += (int64_t)gridDim.x * blockDim.x) {
    ranges[2 * c] = c < nc ? start[c] : (int32_t)cap;
    ranges[2 * c + 1] = c < nc ? start[c] + count[c] : (int32_t)cap;
  }
}

__global__ void zero_i32_kernel(int32_t* v) {
  if (threadIdx.x == 0) *v = 0;
}

// the centre of the cell with label key, coordinate d: o_d + (k_d + 1/2) cell
__device__ __forceinline__ double centre(uint64_t key, int d, int D, double cell,
                                         const ClusterGrid* g) {
  uint64_t rest = key;
  int64_t kd = 0;
  for (int e = D - 1; e >= d; --e) {
    const uint64_t n = (uint64_t)g->dims[e];
    kd = (int64_t)(rest % n);
    rest /= n;
  }
  return __dadd_rn(g->origin[d], __dmul_rn(__dadd_rn((double)kd, 0.5), cell));
}

__device__ __forceinline__ bool kept(const TruncArgs& a, const double* cx, int k) {
  double s = 0.0;
  for (int d = 0; d < a.D; ++d) {
    const double t = __dsub_rn(centre(a.uy[k], d, a.D, a.cell, a.g), cx[d]);
    s = __dadd_rn(s, __dmul_rn(t, t));
  }
  return s <= a.reach2;
}

// Pass 1 (WRITE false): per cluster of x, the number of column runs and the
// kept pairs.  Pass 2 (WRITE true): the runs themselves from col_ptr[i].  One
// workgroup per cluster of x at a time, the clusters of y in chunks of 256
// threads: a run starts at a kept cluster whose predecessor is not kept and
// ends at a kept cluster whose successor is not kept.  Clusters of x beyond
// the count (up to cap_x) get no runs.
template <bool WRITE>
__global__ __launch_bounds__(256) void truncate_kernel(TruncArgs a) {
  __shared__ int flag[258];   // kept flags of clusters k0 - 1 .. k0 + 256
  __shared__ int wsum[4];
  __shared__ unsigned long long wpairs[4];
  const int nx = *a.nx, ny = *a.ny;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int64_t i = blockIdx.x; i < a.cap_x; i += gridDim.x) {
    if (i >= nx) {
      if (!WRITE && tid == 0) a.runs[i] = 0;
      continue;
    }
    double cx[kClusterMaxD];
    for (int d = 0; d < a.D; ++d) cx[d] = centre(a.ux[i], d, a.D, a.cell, a.g);
    const int64_t rows = (int64_t)a.rx[2 * i + 1] - a.rx[2 * i];
    int64_t total = WRITE ? a.col_ptr[i] : 0;   // runs before this chunk
    unsigned long long cols = 0;                // kept columns, this thread
    int prev = 0;                               // kept flag of cluster k0 - 1
    for (int k0 = 0; k0 < ny; k0 += 256) {
      const int k = k0 + tid;
      const int keep = (k < ny && kept(a, cx, k)) ? 1 : 0;
      if (keep) cols += (unsigned long long)(a.ry[2 * k + 1] - a.ry[2 * k]);
      flag[tid + 1] = keep;
      if (tid == 0) flag[0] = prev;
      if (tid == 255) flag[257] = (k + 1 < ny && kept(a, cx, k + 1)) ? 1 : 0;
      __syncthreads();
      const int start = (keep && !flag[tid]) ? 1 : 0;
      const bool last = keep && !flag[tid + 2];
      const unsigned long long bal = __ballot(start);
      const int before_w = __popcll(bal & ((1ull << lane) - 1ull));
      if (lane == 0) wsum[wave] = __popcll(bal);
      __syncthreads();
      int before = before_w;
      for (int w = 0; w < wave; ++w) before += wsum[w];
      if (WRITE) {
        // this cluster's run: the last start at or before it
        const int64_t q = total + before + start - 1;
        if (start && q < a.cap_c) a.col_ranges[2 * q] = a.ry[2 * k];
        if (last && q >= 0 && q < a.cap_c) a.col_ranges[2 * q + 1] = a.ry[2 * k + 1];
      }
      total += wsum[0] + wsum[1] + wsum[2] + wsum[3];
      prev = flag[256];
      __syncthreads();
    }
    if (!WRITE) {
      for (int o = 32; o > 0; o >>= 1) cols += __shfl_xor(cols, o);
      if (lane == 0) wpairs[wave] = cols;
      __syncthreads();
      if (tid == 0) {
        a.runs[i] = (int32_t)total;
        atomicAdd(a.pairs, (unsigned long long)rows *
                               (wpairs[0] + wpairs[1] + wpairs[2] + wpairs[3]));
      }
      __syncthreads();
    }
  }
}

// counts[0] = clusters of x, counts[1] = column ranges, counts[2] = kept
// pairs, counts[3] = 1 when the column ranges exceed their capacity
__global__ void counts_kernel(const int32_t* nx, const int32_t* col_ptr,
                              const unsigned long long* pairs, int64_t cap_c, int64_t* counts) {
  if (threadIdx.x == 0) {
    const int64_t nnz = col_ptr[*nx];
    counts[0] = *nx;
    counts[1] = nnz;
    counts[2] = (int64_t)*pairs;
    counts[3] = nnz > cap_c ? 1 : 0;
  }
}

__global__ void zero_kernel(unsigned long long* v) {
  if (threadIdx.x == 0) *v = 0ull;
}

__global__ __launch_bounds__(256) void gather_kernel(const float* __restrict__ src,
                                                     const int32_t* __restrict__ index, int64_t n,
                                                     int width, int inverse, float* __restrict__ dst) {
  const int64_t total = n * width;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = t / width;
    const int c = (int)(t - i * width);
    const int64_t j = index[i];
    if (inverse) dst[j * width + c] = src[i * width + c];
    else dst[i * width + c] = src[j * width + c];
  }
}

unsigned int grid_for(int64_t n) {
  return (unsigned int)std::max<int64_t>(1, std::min<int64_t>((n + 255) / 256, 4096));
}

template <class T>
size_t align_bytes(size_t n) {
  return (n * sizeof(T) + 255) / 256 * 256;
}

// the sort, run-length encoding and scans: the largest temporary storage
size_t prim_bytes(int64_t M, int64_t N) {
  size_t need = 0, b = 0;
  const int64_t n = std::max(M, N);
  uint64_t* k = nullptr;
  int32_t* v = nullptr;
  int32_t* c = nullptr;
  (void)rocprim::radix_sort_pairs(nullptr, b, k, k, v, v, n);
  need = std::max(need, b);
  (void)rocprim::run_length_encode(nullptr, b, k, n, k, c, c);
  need = std::max(need, b);
  (void)rocprim::exclusive_scan(nullptr, b, c, c, 0, n + 1, rocprim::plus<int32_t>());
  need = std::max(need, b);
  return need;
}

}  // namespace

size_t cluster_scratch_bytes(int64_t M, int64_t N) {
  const int64_t n = std::max(M, N);
  return align_bytes<double>((size_t)kBoxBlocks * 2 * kClusterMaxD) + align_bytes<ClusterGrid>(1) +
         4 * align_bytes<uint64_t>((size_t)n) +   // keys, sorted keys, labels of x and of y
         4 * align_bytes<int32_t>((size_t)n + 1) +   // counts, starts, identity, runs
         align_bytes<int32_t>(2 * (size_t)N) +      // ranges of y
         2 * align_bytes<int32_t>(1) + align_bytes<unsigned long long>(1) + prim_bytes(M, N) + 256;
}

hipError_t build_cluster_pattern(const ClusterCall& c, void* scratch, size_t bytes, hipStream_t s) {
  const int64_t n = std::max(c.M, c.N);
  char* p = static_cast<char*>(scratch);
  auto take = [&](size_t b) {
    char* q = p;
    p += b;
    return q;
  };
  double* box = reinterpret_cast<double*>(take(align_bytes<double>((size_t)kBoxBlocks * 2 * kClusterMaxD)));
  ClusterGrid* g = reinterpret_cast<ClusterGrid*>(take(align_bytes<ClusterGrid>(1)));
  uint64_t* key = reinterpret_cast<uint64_t*>(take(align_bytes<uint64_t>((size_t)n)));
  uint64_t* skey = reinterpret_cast<uint64_t*>(take(align_bytes<uint64_t>((size_t)n)));
  uint64_t* ux = reinterpret_cast<uint64_t*>(take(align_bytes<uint64_t>((size_t)n)));
  uint64_t* uy = reinterpret_cast<uint64_t*>(take(align_bytes<uint64_t>((size_t)n)));
  int32_t* cnt = reinterpret_cast<int32_t*>(take(align_bytes<int32_t>((size_t)n + 1)));
  int32_t* start = reinterpret_cast<int32_t*>(take(align_bytes<int32_t>((size_t)n + 1)));
  int32_t* iota = reinterpret_cast<int32_t*>(take(align_bytes<int32_t>((size_t)n + 1)));
  int32_t* runs = reinterpret_cast<int32_t*>(take(align_bytes<int32_t>((size_t)n + 1)));
  int32_t* ry = reinterpret_cast<int32_t*>(take(align_bytes<int32_t>(2 * (size_t)c.N)));
  int32_t* nx = reinterpret_cast<int32_t*>(take(align_bytes<int32_t>(1)));
  int32_t* ny = reinterpret_cast<int32_t*>(take(align_bytes<int32_t>(1)));
  unsigned long long* pairs = reinterpret_cast<unsigned long long*>(take(align_bytes<unsigned long long>(1)));
  void* tmp = p;
  size_t tmp_bytes = bytes - (size_t)(p - static_cast<char*>(scratch));
  hipError_t e;

  hipLaunchKernelGGL(box_partial_kernel, dim3(kBoxBlocks), dim3(256), 0, s, c.x, c.M, c.y, c.N, c.D, box);
  hipLaunchKernelGGL(box_final_kernel, dim3(1), dim3(64), 0, s, box, kBoxBlocks, c.D, c.cell, g);
  if ((e = hipGetLastError()) != hipSuccess) return e;

  // each cloud: labels, the stable sort (the permutation is the output
  // order), its distinct labels with their counts, and the ranges
  for (int side = 0; side < 2; ++side) {
    const float* pts = side == 0 ? c.x : c.y;
    const int64_t m = side == 0 ? c.M : c.N;
    int32_t* order = side == 0 ? c.order_x : c.order_y;
    uint64_t* uniq = side == 0 ? ux : uy;
    int32_t* nclus = side == 0 ? nx : ny;
    int32_t* ranges = side == 0 ? c.row_ranges : ry;
    hipLaunchKernelGGL(label_kernel, dim3(grid_for(m)), dim3(256), 0, s, pts, m, c.D, c.cell, g, key, iota);
    // counts past the number of clusters stay zero for the scan
    if ((e = launch_fill(reinterpret_cast<float*>(cnt), m, 0.0f, s)) != hipSuccess) return e;
    size_t b = tmp_bytes;
    if ((e = rocprim::radix_sort_pairs(tmp, b, key, skey, iota, order, m, 0, 64, s)) != hipSuccess) return e;
    b = tmp_bytes;
    if ((e = rocprim::run_length_encode(tmp, b, skey, m, uniq, cnt, nclus, s)) != hipSuccess) return e;
    b = tmp_bytes;
    if ((e = rocprim::exclusive_scan(tmp, b, cnt, start, 0, m, rocprim::plus<int32_t>(), s)) != hipSuccess)
      return e;
    hipLaunchKernelGGL(ranges_kernel, dim3(grid_for(m)), dim3(256), 0, s, start, cnt, nclus,
                       side == 0 ? c.M : c.N, ranges);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }

  TruncArgs ta{};
  ta.ux = ux;
  ta.uy = uy;
  ta.rx = c.row_ranges;
  ta.ry = ry;
  ta.nx = nx;
  ta.ny = ny;
  ta.cap_x = c.M;
  ta.D = c.D;
  ta.cell = c.cell;
  ta.reach2 = c.reach2;
  ta.g = g;
  ta.runs = runs;
  ta.col_ptr = c.col_ptr;
  ta.col_ranges = c.col_ranges;
  ta.cap_c = c.col_cap;
  ta.pairs = pairs;
  const unsigned int tg = (unsigned int)std::min<int64_t>(c.M, 2048);
  hipLaunchKernelGGL(zero_kernel, dim3(1), dim3(64), 0, s, pairs);
  hipLaunchKernelGGL(truncate_kernel<false>, dim3(tg), dim3(256), 0, s, ta);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // col_ptr[i] = runs before cluster i, for i = 0 .. M (runs[M] = 0)
  hipLaunchKernelGGL(zero_i32_kernel, dim3(1), dim3(64), 0, s, runs + c.M);
  size_t b = tmp_bytes;
  if ((e = rocprim::exclusive_scan(tmp, b, runs, c.col_ptr, 0, c.M + 1, rocprim::plus<int32_t>(), s)) !=
      hipSuccess)
    return e;
  hipLaunchKernelGGL(truncate_kernel<true>, dim3(tg), dim3(256), 0, s, ta);
  hipLaunchKernelGGL(counts_kernel, dim3(1), dim3(64), 0, s, nx, c.col_ptr, pairs, c.col_cap, c.counts);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const float* src, const int32_t* index, int64_t n, int width,
                              int inverse, float* dst, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(gather_kernel, dim3(grid_for(n * width)), dim3(256), 0, s, src, index, n, width,
                     inverse, dst);
  return hipGetLastError();
}

}  // namespace kred
