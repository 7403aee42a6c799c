// Internal declarations shared by the kred host runtime and its HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace kred {

// Formula codes used inside the kernels (same values as the public enum).
enum : int { F_GAUSS = 0, F_LAPLACE = 1, F_SQDIST = 2, F_GRADX = 3, F_SINKHORN = 4 };

constexpr int kThreads = 256;          // threads per workgroup for the direct-form kernels
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

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
};
hipError_t launch_pack(const PackArgs& a, hipStream_t s);

// Direct-form reduction over (i-rows, j-columns) for small D (<= 16).
struct DirectArgs {
  int formula;            // F_*
  int D, DP, E, EP, e0;   // E-slice [e0, e0 + min(EP, E - e0)) of b / out
  int64_t M, N;
  int C;                  // column blocks; C == 1 writes the final output
  int64_t jpb;            // j per column block
  const float* x;         // M x D
  const float* ypk;       // N x (DP + EP), from the prologue
  float xscale;           // same scale as yscale of the prologue
  float gscale;           // gradient: out = -G * gscale; unused otherwise
  void* out;              // final output (C == 1)
  float* part;            // partials (C > 1), C x M x W
  int KP, K;              // arg-K-min list length (power of two) and K
};
hipError_t launch_direct(const DirectArgs& a, hipStream_t s);
int direct_rows_per_thread(int formula, int DP, int EP, int KP);
int direct_pad_d(int D);      // DP for a given D, 0 if the direct path has none
int direct_pad_e(int E);      // EP for one E-slice
int knn_pad_k(int K);         // KP for a given K
int partial_width(int formula, int DP, int EP, int KP);  // W (floats per row per column block)

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
};
hipError_t launch_combine(const CombineArgs& a, hipStream_t s);

// Fill out with a constant (N = 0 cases); a kernel, not a memset, so that
// callers may capture it in a graph.
hipError_t launch_fill(float* out, int64_t count, float value, hipStream_t s);

}  // namespace kred
