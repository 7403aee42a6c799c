// kred host runtime: argument checks, context and scratch memory, path
// selection and kernel launches for the C ABI declared in include/kred.h.
#include "kred.h"
#include "kred_internal.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

using namespace kred;

// Device scratch of kred_run_noalloc: a fixed array, one copy on every GPU the
// library runs on, held until the process ends.  In host code its name is a
// host-side stand-in, not a device address: kred_create looks the address up
// once per device (hipGetSymbolAddress, with that device current), and host
// code passes only that address on to kernels.
static __device__ __align__(256) unsigned char scratch[KRED_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_fixed_mu;
void* g_fixed[kMaxDevices] = {};   // per device: the address of `scratch` there
// the first bytes of `scratch` hold the one-launch Gaussian sum's row-block
// counters (zero at load, and every call leaves them zero); the rest is the
// calls' arena
constexpr size_t kCounterBytes = (size_t)kSumMaxRowBlocks * sizeof(int);
}  // namespace

namespace {
// Where a call's device buffers come from.  The ordinary entry points use the
// context's own allocations, grown with hipMalloc.  kred_run_noalloc gives the
// call an Arena over the library's static scratch array instead: each kind of
// buffer gets a region the first time the call asks for it (later requests of
// the same kind reuse it), carved in order and never freed.
enum BufKind { BUF_SCRATCH = 0, BUF_AUX = 1, BUF_WIDE = 2, BUF_GUARD = 3, BUF_KINDS = 4 };
struct Arena {
  char* base = nullptr;
  size_t cap = 0, used = 0;
  void* slot[BUF_KINDS] = {};
  size_t size[BUF_KINDS] = {};
};
}  // namespace

struct kred_ctx {
  int device = 0;
  Arena* arena = nullptr;        // set only while a kred_run_noalloc call runs
  void* fixed = nullptr;         // this device's static scratch array (device address)
  int num_cus = 256;
  void* scratch = nullptr;
  size_t scratch_bytes = 0;
  void* aux = nullptr;       // backward: the fused value + gradient of the scalar-cotangent route
  size_t aux_bytes = 0;
  void* wide = nullptr;      // fused value + gradient at large D: centre, signal and sums
  size_t wide_bytes = 0;
  // KRED_FLAG_PROFILE: event pairs around main kernels, reused across collects
  std::vector<hipEvent_t> ev;
  size_t ev_used = 0;
  const char* last_kernel = "none";
  // exact bf16 arg-K-min: the device-side guard (its own allocation, so it
  // outlives scratch growth), and whether the last profiled call used it
  ExactGuard* exact_guard = nullptr;
  int last_exact_D = 0;
  // calls where a device-side guard picks between two kernels (the small-D
  // matrix-core path or the direct form; the fp64 or the fp32 large-D
  // contraction): per profiled call the device counts whether it picked the
  // first (counts[0]) out of all such calls (counts[1]); the name is resolved
  // at collect time
  int* fast_counts = nullptr;
  bool last_fast = false;
  // the one-launch Gaussian sum's row-block counters (zeroed once, and every
  // call leaves them zero)
  int* counters = nullptr;
  const char* choice_yes = "none";   // the kernel when the guard picks the first
  const char* last_direct = "none";   // ... and when it picks the other
};

namespace {

constexpr int kMaxDirectD = 16;
constexpr int64_t kAlign = 256;

inline int64_t align_up(int64_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// min / max / arg-min / arg-max
inline bool is_extreme(kred_reduction r) {
  return r == KRED_R_MIN || r == KRED_R_MAX || r == KRED_R_ARGMIN || r == KRED_R_ARGMAX;
}
inline bool is_max(kred_reduction r) { return r == KRED_R_MAX || r == KRED_R_ARGMAX; }
inline bool is_arg(kred_reduction r) { return r == KRED_R_ARGMIN || r == KRED_R_ARGMAX; }

bool finite_pos(float v) { return std::isfinite(v) && v > 0.0f; }

// The integer a C caller passed for an enum argument.  Read through its bytes:
// in C++, loading an enum object whose value lies outside the enumerators'
// range is undefined, and a C caller may pass any int.
template <class E>
int code_of(const E* e) {
  int v;
  static_assert(sizeof(E) == sizeof(int), "the ABI's enums are int-sized");
  std::memcpy(&v, e, sizeof v);
  return v;
}

bool misaligned(const void* p) { return p != nullptr && (reinterpret_cast<uintptr_t>(p) & 3u); }

// Everything a call needs, derived from validated arguments.
struct Plan {
  int formula, reduction;
  int D, DP, E, KP, K;
  int64_t M, N;
  int C;          // column blocks
  int64_t jpb;    // j per column block
  int S_max;      // widest packed row over the E-slices
  int W_max;      // widest partial row
  int R;          // rows per thread of the direct kernels (first E-slice)
  int64_t pack_bytes, part_bytes;
  float xscale, bscale, gscale;
  float kscale;   // direct kernels: pair scale (input coordinates)
  float fscale;   // fast path: coordinate prescale sqrt(c)
  double fscale64;   // the same in fp64
};

// Column split: enough (row block, column block) work items to keep every
// CU busy, each long enough to amortise its set-up.
int choose_col_blocks(int64_t row_blocks, int64_t N, int num_cus, int requested) {
  const int64_t max_c = std::max<int64_t>(1, std::min<int64_t>(KRED_MAX_COL_BLOCKS, N));
  if (requested > 0) return (int)std::min<int64_t>(requested, max_c);
  const int64_t target_items = (int64_t)num_cus * 16;
  int64_t c = (target_items + row_blocks - 1) / row_blocks;
  c = std::min<int64_t>(c, std::max<int64_t>(1, N / 128));   // >= ~128 columns per item
  if (c >= 8) c = (c + 7) / 8 * 8;                              // equal share per XCD
  return (int)std::max<int64_t>(1, std::min<int64_t>(c, max_c));
}

bool make_plan(kred_formula f, kred_reduction r, const kred_params* p, int64_t M, int64_t N,
               int32_t D, int32_t E, int num_cus, Plan* pl, int rows_override = 0,
               int jpb_align = 1) {
  Plan q{};
  q.formula = (int)f;
  q.reduction = (int)r;
  q.M = M;
  q.N = N;
  q.D = D;
  q.DP = direct_pad_d(D);
  if (q.DP == 0) return false;   // large-D path not available for this pair
  q.KP = 0;
  q.K = 0;
  q.E = E;
  if (r == KRED_R_ARGKMIN) {
    q.K = p->K;
    q.KP = knn_pad_k(p->K);
    q.E = 0;
  }
  if (f == KRED_F_GAUSS_GRADX || f == KRED_F_SINKHORN || r == KRED_R_LSE) q.E = 1;
  const int ext = is_extreme(r) ? 1 : 0;
  // kernel-side formula: log-sum-exps run on the Sinkhorn-form kernels
  const int kf = (r == KRED_R_LSE) ? (f == KRED_F_LAPLACE ? F_LAPLACE_LSE : F_SINKHORN) : (int)f;
  const int EP_first = (r == KRED_R_ARGKMIN) ? 1 : direct_pad_e(std::min(q.E, 16));
  q.S_max = q.DP + EP_first;
  q.W_max = partial_width(kf, q.DP, EP_first, q.KP, ext);
  const int R = direct_sum_rows(kf, q.DP, EP_first, q.KP, ext, M, N, num_cus);
  q.R = R;
  const int64_t rows = rows_override > 0 ? rows_override : (int64_t)kThreads * R;
  const int64_t row_blocks = (M + rows - 1) / rows;
  q.C = choose_col_blocks(std::max<int64_t>(1, row_blocks), N, num_cus, p->col_blocks);
  q.jpb = N > 0 ? (N + q.C - 1) / q.C : 0;
  q.jpb = (q.jpb + jpb_align - 1) / jpb_align * jpb_align;
  if (N > 0) q.C = (int)((N + q.jpb - 1) / q.jpb);   // no empty column block
  q.pack_bytes = align_up(N * q.S_max * (int64_t)sizeof(float));
  q.part_bytes = q.C > 1 ? align_up((int64_t)q.C * M * q.W_max * (int64_t)sizeof(float)) : 0;
  // Direct kernels work in input coordinates (xscale = 1) and scale the pair:
  // Gauss 2^(-c d), c = log2(e) / (2 sigma^2); Laplace 2^(-c sqrt d), c =
  // log2(e) / sigma; Sinkhorn g log2(e) - c d, c = log2(e) / eps.  The small-D
  // fast path prescales coordinates by fscale = sqrt(c) (Gauss, Sinkhorn).
  const double log2e = 1.4426950408889634;
  q.xscale = 1.0f;
  q.bscale = 1.0f;
  q.gscale = 0.0f;
  q.kscale = 1.0f;
  q.fscale = 1.0f;
  q.fscale64 = 1.0;
  switch ((int)f) {
    case KRED_F_GAUSS:
    case KRED_F_GAUSS_GRADX:
    case F_VJP: {
      const double s = (double)p->sigma;
      const double c = log2e / (2.0 * s * s);
      q.kscale = (float)c;
      q.fscale = (float)std::sqrt(c);
      q.fscale64 = std::sqrt(c);
      q.gscale = (float)(1.0 / (s * s));
      break;
    }
    case KRED_F_LAPLACE:
      q.kscale = (float)(log2e / (double)p->sigma);
      break;
    case KRED_F_SINKHORN:
      q.kscale = (float)(log2e / (double)p->eps);
      q.fscale = (float)std::sqrt(log2e / (double)p->eps);
      q.fscale64 = std::sqrt(log2e / (double)p->eps);
      q.bscale = (float)log2e;
      break;
    default:
      break;
  }
  if (r == KRED_R_LSE) q.bscale = (float)log2e;   // log-domain weights g' = g log2(e)
  if (ext) {
    // min of sign * F in natural units: the sign rides on the packed b (and
    // on kscale for the log-sum-exp formula, f = sign g - (sign / eps) d)
    const float sign = is_max(r) ? -1.0f : 1.0f;
    q.bscale = sign;
    if (f == KRED_F_SINKHORN) q.kscale = (float)((double)sign / (double)p->eps);
  }
  *pl = q;
  return true;
}

// Small-D fast path (exponent on the bf16 matrix cores), when the pair allows
// it and the problem is large enough for its extra prologue launches (guard,
// bounds, packing) to pay off; below that the direct kernels are faster.
constexpr double kFastMinPairs = 268435456.0;   // 2^28 pairs

int fast_epi(kred_formula f, kred_reduction r, int64_t M, int64_t N, int32_t D, int32_t E,
             uint32_t flags, int K = 0) {
  if (D > kFastMaxD || (flags & KRED_FLAG_DIRECT)) return -1;
  if (!(flags & KRED_FLAG_FAST) && (double)M * (double)N < kFastMinPairs) return -1;
  if (f == KRED_F_GAUSS && r == KRED_R_SUM && E == 1) return FAST_SUM;
  if (f == KRED_F_GAUSS && r == KRED_R_SUM && E >= 2 && E <= 4) return FAST_SUMV;
  // the gradient's per-column extras (b, b v) hold three coordinates
  if (f == KRED_F_GAUSS_GRADX && r == KRED_R_SUM) return D <= 3 ? FAST_GRADX : -1;
  if ((f == KRED_F_SINKHORN || f == KRED_F_GAUSS) && r == KRED_R_LSE) return FAST_LSE;
  // nearest neighbour: arg-K-min with K = 1, and the distance's min / arg-min
  if (f == KRED_F_SQDIST && r == KRED_R_ARGKMIN && K == 1) return FAST_MIN;
  if (f == KRED_F_SQDIST && r == KRED_R_ARGKMIN && K > 1 && K <= 16) return FAST_KNN;
  return -1;
}

// Large D: the bf16 matrix-core kernels (arg-K-min: the exact kernel,
// launched beside the fp32 one, the device-side guard picking one; sums: the
// split-product kernel) serve problems large enough that their prologue work
// pays off, or any size with KRED_FLAG_FAST; never with KRED_FLAG_DIRECT.
bool exact_eligible(uint32_t flags, int64_t M, int64_t N) {
  if (flags & KRED_FLAG_DIRECT) return false;
  return (flags & KRED_FLAG_FAST) || (double)M * (double)N >= kFastMinPairs;
}

// the exact k-NN kernel's list keys hold column indices below 2^28
bool exact_knn_eligible(uint32_t flags, int64_t M, int64_t N) {
  return exact_eligible(flags, M, N) && N <= ((int64_t)1 << 28);
}

struct FastScratch {
  int64_t guard_bytes, apk_bytes, ex_bytes;
};
FastScratch fast_scratch(int epi, int64_t N) {
  FastScratch fs{};
  if (epi < 0) return fs;
  const int64_t N16 = (N + 15) / 16 * 16;
  fs.guard_bytes = align_up(sizeof(FastGuard));
  fs.apk_bytes = align_up(N16 * 64);
  fs.ex_bytes = (epi == FAST_GRADX || epi == FAST_SUMV) ? align_up(N16 * 16)
                : (epi == FAST_SUM ? align_up(N16 * 4) : 0);
  return fs;
}

// Large-D (matrix-core) plan.
struct MPlan {
  int epi, DP, TJ, EB, W, KP, K;
  int64_t N16;
  int C;
  int64_t jpb;
  int64_t yop_bytes, ny_bytes, b_bytes, part_bytes;
  float xscale, yop_scale, coord_scale, nrm_sign, pad_norm;
  double sc64;        // the prescale sqrt(c) in fp64 (the fp64 contraction)
  float wide_limit;   // the accuracy guard's limit on L (< 0: always the fp64 contraction)
};

bool make_mplan(kred_formula f, kred_reduction r, const kred_params* p, int64_t M, int64_t N,
                int32_t D, int32_t E, int num_cus, MPlan* pl) {
  MPlan q{};
  q.DP = mfma_pad_d(D);
  if (q.DP == 0) return false;
  q.TJ = mfma_tile_cols(q.DP);
  q.KP = 0;
  q.K = 0;
  const double log2e = 1.4426950408889634;
  if (r == KRED_R_ARGKMIN) {
    q.epi = 3;
    q.K = p->K;
    q.KP = mfma_knn_pad_k(p->K);
    q.EB = 1;
    q.xscale = 1.0f;
    q.yop_scale = -2.0f;
    q.coord_scale = 1.0f;
    q.nrm_sign = 1.0f;
    q.pad_norm = INFINITY;
  } else if (is_extreme(r)) {
    // min / max of F b per signal column, in slices of 16 columns: F as for
    // the sums (Gauss, Laplace, squared distance), or the Sinkhorn form's s
    // with g in the column norms (log2 units, as for its log-sum-exp)
    q.EB = 1;
    double sc = 1.0;
    q.pad_norm = 0.0f;
    if (f == KRED_F_GAUSS) {
      q.epi = 6;
      sc = std::sqrt(log2e / (2.0 * (double)p->sigma * (double)p->sigma));
    } else if (f == KRED_F_LAPLACE) {
      q.epi = 7;
      sc = log2e / (double)p->sigma;
    } else if (f == KRED_F_SQDIST) {
      q.epi = 8;
    } else {
      q.epi = 9;
      sc = std::sqrt(log2e / (double)p->eps);
    }
    q.xscale = (float)sc;
    q.sc64 = sc;
    q.coord_scale = (float)sc;
    q.yop_scale = (float)(2.0 * sc);
    q.nrm_sign = -1.0f;
  } else if (r == KRED_R_LSE && f == KRED_F_LAPLACE) {
    // s_ij = g_j - |x_i - y_j| / sigma in log2 units: x and y scaled by
    // log2(e) / sigma, T = -(log2(e) / sigma)^2 d, s = g_j log2(e) - sqrt(-T)
    // with g' in its own per-column array (padding columns -inf)
    q.epi = 5;
    q.EB = 1;
    const double sc = log2e / (double)p->sigma;
    q.xscale = (float)sc;
    q.sc64 = sc;
    q.coord_scale = (float)sc;
    q.yop_scale = (float)(2.0 * sc);
    q.nrm_sign = -1.0f;
    q.pad_norm = 0.0f;
  } else if (r == KRED_R_LSE) {
    // s_ij = g_j - d_ij / eps in log2 units (the Gaussian's log-domain sum is
    // the same with eps = 2 sigma^2): x and y scaled by sqrt(log2(e) / eps),
    // the column norms carry g_j log2(e), padding columns s = -inf
    q.epi = 4;
    q.EB = 1;
    const double eps = f == KRED_F_SINKHORN ? (double)p->eps
                                            : 2.0 * (double)p->sigma * (double)p->sigma;
    const double sc = std::sqrt(log2e / eps);
    q.xscale = (float)sc;
    q.sc64 = sc;
    q.coord_scale = (float)sc;
    q.yop_scale = (float)(2.0 * sc);
    q.nrm_sign = -1.0f;
    q.pad_norm = -INFINITY;
  } else {
    q.EB = E <= 16 ? 1 : (E <= 32 ? 2 : 4);
    double sc = 1.0;
    if (f == KRED_F_GAUSS) {
      q.epi = 0;
      sc = std::sqrt(log2e / (2.0 * (double)p->sigma * (double)p->sigma));
      q.pad_norm = -INFINITY;
    } else if (f == KRED_F_LAPLACE) {
      q.epi = 1;
      sc = log2e / (double)p->sigma;
      q.pad_norm = -INFINITY;
    } else {
      q.epi = 2;
      q.pad_norm = 0.0f;
    }
    q.xscale = (float)sc;
    q.sc64 = sc;
    q.coord_scale = (float)sc;
    q.yop_scale = (float)(2.0 * sc);
    q.nrm_sign = -1.0f;
  }
  q.W = 16 * q.EB;
  q.N16 = (N + 15) / 16 * 16;
  // the accuracy guard (SpreadGuard): the exponential forms keep the fp32
  // kernels up to the bound's limit; the Laplacian forms (sqrt of the
  // distance) and the squared distance's sums and extremes always take the
  // fp64 contraction; arg-K-min ranks in fp32 and is re-ranked exactly
  // (sums take the split bf16 kernel where it is eligible, with its own bound)
  const bool split_sum = q.epi <= 2 && exact_eligible(p->flags, M, N);
  // the Gaussian and Sinkhorn log-sum-exp on the 32x32-tile split kernel (DP
  // 32, 64 and 128), under the split contraction's bound
  const bool split_lse = q.epi == 4 && split_lse_dp(q.DP) && exact_eligible(p->flags, M, N);
  q.wide_limit = !(q.epi == 0 || q.epi == 4 || q.epi == 6 || q.epi == 9) ? -1.0f
                 : (split_sum || split_lse) ? wide_limit_split(D) : wide_limit_f32(D);
  const bool split32 = (split_sum && q.epi == 0) || split_lse;
  const int rows = split32 ? mfma_split_rows_per_block(q.DP, q.epi) : mfma_rows_per_block(q.DP, q.KP);
  const int64_t row_blocks = std::max<int64_t>(1, (M + rows - 1) / rows);
  int C = choose_col_blocks(row_blocks, q.N16, num_cus, p->col_blocks);
  // the split sum kernel with 4 to 7 column blocks: 8, one per XCD (blockIdx
  // mod 8 picks both), so that each XCD's L2 serves one stream of y tiles
  // (c4: 51.3 ms against 52.4 at the 6 chosen above)
  if (split32 && p->col_blocks <= 0 && C >= 4 && C < 8 && q.N16 >= 8 * 128) C = 8;
  int64_t jpb = (q.N16 + C - 1) / C;
  jpb = (jpb + q.TJ - 1) / q.TJ * q.TJ;
  q.jpb = jpb;
  q.C = (int)((q.N16 + jpb - 1) / jpb);
  // (the fp64 contraction keeps yop and ny in fp64 in the same buffers)
  const int64_t esz = r == KRED_R_ARGKMIN ? (int64_t)sizeof(float) : (int64_t)sizeof(double);
  q.yop_bytes = align_up(q.N16 * q.DP * esz);
  q.ny_bytes = align_up(q.N16 * esz);
  q.b_bytes = (r == KRED_R_ARGKMIN || r == KRED_R_LSE)
                  ? (q.epi == 5 ? align_up(q.N16 * (int64_t)sizeof(float)) : 0)
                  : align_up(q.N16 * q.W * (int64_t)sizeof(float));
  // the split kernel's bf16 planes of b per 32-column pair (in the same buffer)
  if (split_sum && q.epi == 0 && q.DP <= 128)
    q.b_bytes = std::max(q.b_bytes, align_up((N + 31) / 32 * 32 * q.W * 3 * (int64_t)sizeof(uint16_t)));
  if (r == KRED_R_ARGKMIN)
    q.part_bytes = align_up((int64_t)4 * q.C * M * 2 * q.KP * (int64_t)sizeof(float));
  else if (is_extreme(r))
    q.part_bytes = align_up((int64_t)4 * q.C * M * 2 * q.W * (int64_t)sizeof(float));
  else if (r == KRED_R_LSE)
    q.part_bytes = q.C > 1 ? align_up((int64_t)q.C * M * 2 * (int64_t)sizeof(float)) : 0;
  else
    q.part_bytes = q.C > 1 ? align_up((int64_t)q.C * M * q.W * (int64_t)sizeof(float)) : 0;
  *pl = q;
  return true;
}

// Grow a context buffer; the old one may still be in use by queued kernels,
// so the device is synchronised before it is freed.
kred_status grow_buffer(void** buf, size_t* have, size_t bytes) {
  if (bytes <= *have) return KRED_OK;
  const size_t want = std::max(bytes, *have * 5 / 4);
  if (*buf) {
    if (hipDeviceSynchronize() != hipSuccess) return KRED_ERR_HIP;
    (void)hipFree(*buf);
    *buf = nullptr;
    *have = 0;
  }
  if (hipMalloc(buf, want) != hipSuccess) {
    (void)hipGetLastError();
    *buf = nullptr;
    return KRED_ERR_NOMEM;
  }
  *have = want;
  return KRED_OK;
}

// A device buffer of at least `bytes` of the given kind for this call.
kred_status buffer(kred_ctx* ctx, BufKind k, size_t bytes, void** out) {
  if (Arena* a = ctx->arena) {
    if (a->slot[k] != nullptr) {
      if (bytes > a->size[k]) return KRED_ERR_SCRATCH;
      *out = a->slot[k];
      return KRED_OK;
    }
    const size_t off = (size_t)align_up((int64_t)a->used);
    if (off > a->cap || bytes > a->cap - off) return KRED_ERR_SCRATCH;
    a->slot[k] = a->base + off;
    a->size[k] = bytes;
    a->used = off + bytes;
    *out = a->slot[k];
    return KRED_OK;
  }
  kred_status st = KRED_OK;
  switch (k) {
    case BUF_SCRATCH: st = grow_buffer(&ctx->scratch, &ctx->scratch_bytes, bytes); *out = ctx->scratch; break;
    case BUF_AUX: st = grow_buffer(&ctx->aux, &ctx->aux_bytes, bytes); *out = ctx->aux; break;
    case BUF_WIDE: st = grow_buffer(&ctx->wide, &ctx->wide_bytes, bytes); *out = ctx->wide; break;
    case BUF_GUARD:
      if (ctx->exact_guard == nullptr &&
          hipMalloc(reinterpret_cast<void**>(&ctx->exact_guard), sizeof(ExactGuard)) != hipSuccess) {
        (void)hipGetLastError();
        ctx->exact_guard = nullptr;
        return KRED_ERR_NOMEM;
      }
      *out = ctx->exact_guard;
      break;
    default: return KRED_ERR_INVALID_ARG;
  }
  return st;
}

struct DeviceGuard {
  int prev = -1;
  bool ok = false;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) return;
    ok = (prev == dev) || hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() {
    int cur = -1;
    if (ok && hipGetDevice(&cur) == hipSuccess && cur != prev && prev >= 0) (void)hipSetDevice(prev);
  }
};

hipEvent_t next_event(kred_ctx* ctx) {
  if (ctx->ev_used == ctx->ev.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    ctx->ev.push_back(e);
  }
  return ctx->ev[ctx->ev_used++];
}

// Block-sparse pattern of a call (nr row clusters; see DirectArgs).
struct Ranges {
  int nr;
  const int* rr;
  const int* cp;
  const int* cr;
};

// Profiled large-D call with the accuracy guard: count on the device whether
// it picked the fp64 contraction (the name is resolved at collect time).
kred_status record_wide(kred_ctx* ctx, const SpreadGuard* g, float c, float limit,
                        const char* fp32_name, hipStream_t s) {
  if (ctx->fast_counts == nullptr) {
    if (hipMalloc(reinterpret_cast<void**>(&ctx->fast_counts), 2 * sizeof(int)) != hipSuccess) {
      ctx->fast_counts = nullptr;
      return KRED_ERR_NOMEM;
    }
    if (hipMemset(ctx->fast_counts, 0, 2 * sizeof(int)) != hipSuccess) return KRED_ERR_HIP;
  }
  if (launch_wide_record(g, c, limit, ctx->fast_counts, s) != hipSuccess) return KRED_ERR_HIP;
  ctx->last_fast = true;
  ctx->choice_yes = "mfma_f64_kernel";
  ctx->last_direct = fp32_name;
  return KRED_OK;
}

// Scratch for the bf16 column operand of the large-D kernels: the exact k-NN
// kernel's copy (DP bf16 per column) or the split kernel's three planes.
int64_t mfma_bf16_bytes(const MPlan& pl, bool knn, uint32_t flags, int64_t M, int64_t N) {
  if (!(knn ? exact_knn_eligible(flags, M, N) : exact_eligible(flags, M, N))) return 0;
  return align_up(pl.N16 * (knn ? 1 : 3) * pl.DP * (int64_t)sizeof(uint16_t));
}

// One more signal column of a Gaussian sum with 64 columns on the 32x32-tile
// split kernel (summed there on the vector ALU): xb its values (N16 + 1, zero
// from N on), xout its output column (M floats).  skip: the call that would
// sum that column alone, after such a call with the same arguments; its
// split kernel returns at once and it runs with one column block, so that
// only the fp64 contraction (when the guard picks it) writes xout.
struct XCol {
  const float* xb = nullptr;
  float* xout = nullptr;
  bool skip = false;
};

kred_status run_mfma(kred_ctx* ctx, kred_formula f, kred_reduction r, const kred_params* p,
                     int64_t M, int64_t N, int32_t D, int32_t E, const float* x, const float* y,
                     const float* b, void* out, hipStream_t s, int kvalues,
                     const Ranges* rg = nullptr, const XCol* xcol = nullptr) {
  kred_params pr;
  if (rg && p->col_blocks == 0) {
    // chunks of each cluster's columns: enough workgroups for every CU, the
    // row-block count estimated as max(clusters, M / rows per workgroup)
    const int DP = mfma_pad_d(D);
    const int rows = mfma_rows_per_block(DP, r == KRED_R_ARGKMIN ? mfma_knn_pad_k(p->K) : 0);
    const int64_t est = std::max<int64_t>({1, (int64_t)rg->nr, (M + rows - 1) / rows});
    pr = *p;
    pr.col_blocks = (int)std::min<int64_t>(64, ((int64_t)ctx->num_cus * 16 + est - 1) / est);
    p = &pr;
  }
  MPlan pl;
  if (!make_mplan(f, r, p, M, N, D, E, ctx->num_cus, &pl)) return KRED_ERR_UNSUPPORTED;
  if (rg) pl.C = std::max(1, std::min(p->col_blocks, KRED_MAX_COL_BLOCKS));   // chunks per cluster
  const bool knn = (r == KRED_R_ARGKMIN);
  const bool lse = (r == KRED_R_LSE);
  const bool ext = is_extreme(r);
  // min / max: no b for the Sinkhorn form (g goes into the column norms) or
  // for the bare squared distance; the signal is then a column of ones
  const bool unit_b = ext && (f == KRED_F_SINKHORN || b == nullptr);
  // arg-K-min: the exact bf16 kernel is a candidate (the device decides);
  // sums, and the Gaussian / Sinkhorn log-sum-exp at DP = 64, 128: the split
  // bf16 kernel replaces the fp32 one
  const bool exact = knn && exact_knn_eligible(p->flags, M, N);
  const bool split = !knn && !ext && exact_eligible(p->flags, M, N) &&
                     (!lse || (pl.epi == 4 && split_lse_dp(pl.DP)));
  const int64_t rows_wg = split ? mfma_split_rows_per_block(pl.DP, pl.epi) : mfma_rows_per_block(pl.DP, pl.KP);
  // the extra column needs the 32x32-tile split sum with 64 columns (or, to
  // skip it, one column block)
  const bool xon = xcol && xcol->xb;
  if (xon && !(split && pl.epi == 0 && pl.DP <= 128 && pl.EB == 4)) return KRED_ERR_UNSUPPORTED;
  if (xcol && xcol->skip && (!split || pl.epi != 0 || pl.DP > 128 || pl.C != 1))
    return KRED_ERR_UNSUPPORTED;
  const int64_t xpart_bytes = (xon && pl.C > 1) ? align_up((int64_t)pl.C * M * (int64_t)sizeof(float)) : 0;
  const int64_t ybf_bytes = mfma_bf16_bytes(pl, knn, p->flags, M, N);
  if (rg) {   // partials of every chunk (rows outside the clusters read the empty value)
    pl.part_bytes = knn ? align_up((int64_t)4 * pl.C * M * 2 * pl.KP * (int64_t)sizeof(float))
                  : ext ? align_up((int64_t)4 * pl.C * M * 2 * pl.W * (int64_t)sizeof(float))
                  : pl.C > 1 ? align_up((int64_t)pl.C * M * (lse ? 2 : pl.W) * (int64_t)sizeof(float))
                             : 0;
  }
  const int64_t bstart_bytes = rg ? align_up((int64_t)(rg->nr + 1) * (int64_t)sizeof(int)) : 0;
  // sums and log-sum-exp: x and y are centred on a point of y (distances do
  // not change; the expanded form's cancellation then scales with the spread
  // of the data, not with its distance from the origin)
  const int64_t cen_bytes = knn ? 0 : align_up((int64_t)D * (int64_t)sizeof(float));
  // the accuracy guard, and the fp64 variant's own block-sparse workgroup map
  const int64_t sg_bytes = knn ? 0 : align_up(sizeof(SpreadGuard));
  const int64_t rows64 = knn ? 0 : mfma64_rows_per_block(pl.DP);
  const int64_t bstart64_bytes = (rg && !knn) ? bstart_bytes : 0;
  void* sp = nullptr;
  const kred_status gs = buffer(ctx, BUF_SCRATCH,
                                (size_t)(pl.yop_bytes + pl.ny_bytes + pl.b_bytes + pl.part_bytes +
                                         ybf_bytes + bstart_bytes + cen_bytes + sg_bytes +
                                         bstart64_bytes + xpart_bytes), &sp);
  if (gs != KRED_OK) return gs;
  void* gp = nullptr;
  if (exact) {
    const kred_status ge = buffer(ctx, BUF_GUARD, sizeof(ExactGuard), &gp);
    if (ge != KRED_OK) return ge;
  }
  char* base = static_cast<char*>(sp);
  float* yop = reinterpret_cast<float*>(base);
  float* ny = reinterpret_cast<float*>(base + pl.yop_bytes);
  float* bpk = pl.b_bytes ? reinterpret_cast<float*>(base + pl.yop_bytes + pl.ny_bytes) : nullptr;
  // the Laplacian log-sum-exp keeps g' per column where the sums keep packed b
  float* gpk = pl.epi == 5 ? bpk : nullptr;
  if (gpk) bpk = nullptr;
  float* part = pl.part_bytes
                    ? reinterpret_cast<float*>(base + pl.yop_bytes + pl.ny_bytes + pl.b_bytes)
                    : nullptr;
  uint16_t* ybf = (exact || split) ? reinterpret_cast<uint16_t*>(base + pl.yop_bytes + pl.ny_bytes +
                                                                  pl.b_bytes + pl.part_bytes)
                                    : nullptr;
  int* bstart = rg ? reinterpret_cast<int*>(base + pl.yop_bytes + pl.ny_bytes + pl.b_bytes +
                                            pl.part_bytes + ybf_bytes)
                   : nullptr;
  float* cen = knn ? nullptr
                   : reinterpret_cast<float*>(base + pl.yop_bytes + pl.ny_bytes + pl.b_bytes +
                                              pl.part_bytes + ybf_bytes + bstart_bytes);
  SpreadGuard* sg = knn ? nullptr
                        : reinterpret_cast<SpreadGuard*>(reinterpret_cast<char*>(cen) + cen_bytes);
  int* bstart64 = bstart64_bytes ? reinterpret_cast<int*>(reinterpret_cast<char*>(sg) + sg_bytes)
                                 : nullptr;
  float* xpart = xpart_bytes ? reinterpret_cast<float*>(reinterpret_cast<char*>(sg) + sg_bytes +
                                                        bstart64_bytes)
                             : nullptr;
  const float wide_c = (float)(pl.sc64 * pl.sc64);
  if (cen && launch_centre(y, N, D, cen, s) != hipSuccess) return KRED_ERR_HIP;
  if (sg && launch_spread(x, M, y, N, D, cen, sg, s) != hipSuccess) return KRED_ERR_HIP;
  ExactGuard* eg = exact ? static_cast<ExactGuard*>(gp) : nullptr;
  if (exact && launch_exact_check(x, M, y, N, D, eg, s) != hipSuccess) return KRED_ERR_HIP;
  if (rg) {
    if (launch_range_blocks(rg->rr, rg->nr, M, (int)rows_wg, bstart, s) != hipSuccess)
      return KRED_ERR_HIP;
    if (bstart64 && launch_range_blocks(rg->rr, rg->nr, M, (int)rows64, bstart64, s) != hipSuccess)
      return KRED_ERR_HIP;
    // (distance, index) pairs: 4 C lists of KP pairs per row, count in floats
    if (knn && launch_fill2(part, (int64_t)4 * pl.C * M * 2 * pl.KP, INFINITY,
                            __builtin_bit_cast(float, (int32_t)INT32_MAX), s) != hipSuccess)
      return KRED_ERR_HIP;
    if (lse && pl.C > 1 && launch_fill2(part, (int64_t)pl.C * M * 2, -INFINITY, 0.0f, s) != hipSuccess)
      return KRED_ERR_HIP;
    if (ext && launch_fill2(part, (int64_t)4 * pl.C * M * 2 * pl.W, INFINITY,
                            __builtin_bit_cast(float, (int32_t)-1), s) != hipSuccess)
      return KRED_ERR_HIP;
    if (!knn && !lse && !ext && pl.C > 1 &&
        launch_fill(part, (int64_t)pl.C * M * pl.W, 0.0f, s) != hipSuccess)
      return KRED_ERR_HIP;
    if (xpart && launch_fill(xpart, (int64_t)pl.C * M, 0.0f, s) != hipSuccess) return KRED_ERR_HIP;
  }

  MfmaPackArgs pa{};
  pa.y = y;
  pa.b = (knn || lse || unit_b) ? nullptr : b;
  pa.unit_b = unit_b ? 1 : 0;
  pa.N = N;
  pa.N16 = pl.N16;
  pa.D = D;
  pa.DP = pl.DP;
  pa.E = E;
  pa.e0 = 0;
  pa.Ec = (knn || lse) ? 0 : E;
  pa.goff = (lse || (ext && f == KRED_F_SINKHORN)) ? b : nullptr;
  pa.goff_scale = 1.4426950408889634f;
  pa.yc = cen;
  pa.gpk = gpk;
  pa.EB = pl.EB;
  pa.yop_scale = pl.yop_scale;
  pa.coord_scale = pl.coord_scale;
  pa.nrm_sign = pl.nrm_sign;
  pa.pad_norm = pl.pad_norm;
  pa.yop = yop;
  pa.ny = ny;
  pa.bpk = bpk;
  pa.exact = eg;
  pa.ybf = exact ? ybf : nullptr;
  pa.ysp = split ? ybf : nullptr;
  pa.bpair = (split && pl.epi == 0 && pl.DP <= 128) ? 1 : 0;
  pa.spread = sg;
  pa.wide_c = wide_c;
  pa.wide_limit = pl.wide_limit;
  pa.yop_scale64 = 2.0 * pl.sc64;
  pa.coord_scale64 = pl.sc64;
  if (!ext && launch_mfma_pack(pa, s) != hipSuccess) return KRED_ERR_HIP;

  MfmaArgs ma{};
  ma.epi = pl.epi;
  ma.D = D;
  ma.DP = pl.DP;
  ma.E = E;
  ma.e0 = 0;
  ma.EB = pl.EB;
  ma.M = M;
  ma.N16 = pl.N16;
  ma.C = pl.C;
  ma.jpb = pl.jpb;
  ma.x = x;
  ma.xscale = pl.xscale;
  ma.yop = yop;
  ma.ny = ny;
  ma.bpk = bpk;
  ma.out = out;
  ma.part = part;
  ma.KP = pl.KP;
  ma.K = pl.K;
  ma.exact = eg;
  ma.ybf = exact ? ybf : nullptr;
  ma.ysp = split ? ybf : nullptr;
  ma.N = N;
  ma.pad_ny = pl.pad_norm;
  ma.xc = cen;
  ma.gpk = gpk;
  ma.ext_sign = is_max(r) ? -1.0f : 1.0f;
  ma.spread = sg;
  ma.wide_c = wide_c;
  ma.wide_limit = pl.wide_limit;
  ma.xscale64 = pl.sc64;
  if (xon) {
    ma.xb = xcol->xb;
    ma.xout = xcol->xout;
    ma.xpart = xpart;
  }
  ma.xskip = (xcol && xcol->skip) ? 1 : 0;
  if (rg) {
    ma.nr = rg->nr;
    ma.rr = rg->rr;
    ma.cp = rg->cp;
    ma.cr = rg->cr;
    ma.bstart = bstart;
  }
  // the fp64 variant: the same arguments with its own workgroup map
  MfmaArgs ma64 = ma;
  if (bstart64) ma64.bstart = bstart64;
  const bool prof = (p->flags & KRED_FLAG_PROFILE) != 0;
  if (ext) {
    // slices of 16 signal columns: pack the slice's b, run, merge the 4 C
    // partial (key, index) pairs of each row and column into out
    for (int e0 = 0; e0 < E; e0 += pl.W) {
      pa.e0 = e0;
      pa.Ec = std::min(pl.W, E - e0);
      if (launch_mfma_pack(pa, s) != hipSuccess) return KRED_ERR_HIP;
      ma.e0 = e0;
      if (rg && e0 > 0 &&
          launch_fill2(part, (int64_t)4 * pl.C * M * 2 * pl.W, INFINITY,
                       __builtin_bit_cast(float, (int32_t)-1), s) != hipSuccess)
        return KRED_ERR_HIP;
      hipEvent_t x0 = nullptr, x1 = nullptr;
      if (prof) {
        x0 = next_event(ctx);
        x1 = next_event(ctx);
        if (!x0 || !x1 || hipEventRecord(x0, s) != hipSuccess) return KRED_ERR_HIP;
      }
      ma64.e0 = e0;
      // both launch; the guard lets exactly one do the work
      if (launch_mfma(ma, s) != hipSuccess || launch_mfma64(ma64, s) != hipSuccess)
        return KRED_ERR_HIP;
      if (prof) {
        if (hipEventRecord(x1, s) != hipSuccess) return KRED_ERR_HIP;
        ctx->last_exact_D = 0;
        const kred_status pr = record_wide(ctx, sg, wide_c, pl.wide_limit, "mfma_kernel", s);
        if (pr != KRED_OK) return pr;
      }
      CombineArgs ca{};
      ca.formula = (int)f;
      ca.D = D;
      ca.DP = pl.DP;
      ca.E = E;
      ca.EP = pl.W;
      ca.e0 = e0;
      ca.M = M;
      ca.C = 4 * pl.C;
      ca.part = part;
      ca.out = out;
      ca.ext = 1;
      ca.ext_sign = ma.ext_sign;
      ca.arg = is_arg(r) ? 1 : 0;
      if (launch_combine(ca, s) != hipSuccess) return KRED_ERR_HIP;
    }
    return KRED_OK;
  }
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (prof) {
    e0 = next_event(ctx);
    e1 = next_event(ctx);
    if (!e0 || !e1 || hipEventRecord(e0, s) != hipSuccess) return KRED_ERR_HIP;
  }
  // with the exact kernel a candidate, both launch and exactly one does the
  // work; likewise the fp32 (or split) kernel and the fp64 variant
  if (split) {
    if (launch_mfma_split(ma, s) != hipSuccess) return KRED_ERR_HIP;
  } else if (launch_mfma(ma, s) != hipSuccess) {
    return KRED_ERR_HIP;
  }
  if (exact && launch_knn_bf16(ma, s) != hipSuccess) return KRED_ERR_HIP;
  if (!knn && launch_mfma64(ma64, s) != hipSuccess) return KRED_ERR_HIP;
  if (prof) {
    if (hipEventRecord(e1, s) != hipSuccess) return KRED_ERR_HIP;
    ctx->last_kernel = split ? "mfma_split_kernel" : "mfma_kernel";
    ctx->last_fast = false;
    ctx->last_exact_D = exact ? D : 0;   // resolved from the guard at collect time
    if (!knn) {
      const kred_status pr = record_wide(ctx, sg, wide_c, pl.wide_limit, ctx->last_kernel, s);
      if (pr != KRED_OK) return pr;
    }
  }
  if (knn || pl.C > 1) {
    CombineArgs ca{};
    ca.formula = knn ? (int)KRED_F_SQDIST : lse ? (int)F_SINKHORN : (int)f;
    ca.D = D;
    ca.DP = pl.DP;
    ca.E = E;
    ca.EP = pl.W;
    ca.e0 = 0;
    ca.M = M;
    ca.C = knn ? 4 * pl.C : pl.C;
    ca.part = part;
    ca.out = out;
    ca.gscale = 0.0f;
    ca.KP = knn ? pl.KP : 0;
    ca.K = pl.K;
    ca.kvalues = kvalues;
    if (knn) {
      // the merged candidates get their direct-form distances and are ranked again
      ca.rx = x;
      ca.ry = y;
      ca.rD = D;
    }
    if (launch_combine(ca, s) != hipSuccess) return KRED_ERR_HIP;
    if (xpart) {   // the extra column's partials, the same sum
      ca.E = 1;
      ca.EP = 1;
      ca.part = xpart;
      ca.out = xcol->xout;
      if (launch_combine(ca, s) != hipSuccess) return KRED_ERR_HIP;
    }
  }
  return KRED_OK;
}

// Value an empty reduction writes (and the output's element count) for r.
void empty_fill(kred_formula f, kred_reduction r, const kred_params* p, int64_t M, int32_t D,
                int32_t E, const float* b, int64_t* count, float* value) {
  const int64_t e_out = (f == KRED_F_SINKHORN || (f == KRED_F_SQDIST && b == nullptr)) ? 1 : E;
  *count = M;
  *value = 0.0f;
  if (f == KRED_F_GAUSS_GRADX) *count = M * (1 + D);
  else if (r == KRED_R_SUM) *count = M * E;
  else if (r == KRED_R_LSE) *value = -INFINITY;
  else if (r == KRED_R_ARGKMIN || r == KRED_R_KMIN) {
    *count = M * p->K;
    *value = r == KRED_R_KMIN ? INFINITY : __builtin_bit_cast(float, (int32_t)-1);
  } else if (is_extreme(r)) {
    *count = M * e_out;
    // an empty min is +inf, an empty max -inf, an empty arg -1 (int32 bits)
    *value = is_arg(r) ? __builtin_bit_cast(float, (int32_t)-1) : (is_max(r) ? -INFINITY : INFINITY);
  }
}

// Bytes of the large-D gradient's own buffer: the centre, one signal chunk
// (N x 64) and the sums (M x E (D + 1)).
int64_t gradx_wide_bytes(int64_t M, int64_t N, int32_t D, int32_t E = 1) {
  const int64_t W = (int64_t)E * (D + 1);
  return align_up((int64_t)D * (int64_t)sizeof(float)) +
         align_up(N * std::min<int64_t>(64, W) * (int64_t)sizeof(float)) +
         align_up(M * W * (int64_t)sizeof(float)) +
         align_up(((N + 15) / 16 * 16 + 16) * (int64_t)sizeof(float));
}

// W = 64 q + 1 signal columns on the 32x32-tile split kernel: the last column
// rides with the first 64 (summed on the vector ALU) instead of a launch of
// its own
bool gradx_extra_col(uint32_t flags, int64_t M, int64_t N, int32_t D, int32_t E) {
  const int64_t W = (int64_t)E * (D + 1);
  return W > 64 && W % 64 == 1 && exact_eligible(flags, M, N) && mfma_pad_d(D) <= 128;
}

// Gaussian x-gradients for 16 < D <= 256 (validated, M, N > 0) as one Gaussian
// sum on the matrix cores with the E (D + 1) signal columns [b_e, b_e (y - m)],
// 64 columns per call.  Without a cotangent (e = NULL, E = 1): GAUSS_GRADX,
// out = (A0, (A1 - (x - m) A0) / sigma^2), M x (1 + D).  With a cotangent e
// (M x E): the vector-Jacobian product out = sum_e e_e (A_e,1 - (x - m) A_e,0)
// / sigma^2, M x D.
kred_status run_gradx_wide(kred_ctx* ctx, const kred_params* p, int64_t M, int64_t N, int32_t D,
                           int32_t E, const float* x, const float* y, const float* b,
                           const float* e, float* out, hipStream_t s, const Ranges* rg) {
  void* wp = nullptr;
  const kred_status ga = buffer(ctx, BUF_WIDE, (size_t)gradx_wide_bytes(M, N, D, E), &wp);
  if (ga != KRED_OK) return ga;
  const int W = E * (D + 1);
  char* base = static_cast<char*>(wp);
  float* m = reinterpret_cast<float*>(base);
  float* sig = reinterpret_cast<float*>(base + align_up((int64_t)D * (int64_t)sizeof(float)));
  float* T = reinterpret_cast<float*>(reinterpret_cast<char*>(sig) +
                                      align_up(N * std::min(64, W) * (int64_t)sizeof(float)));
  float* xsig = reinterpret_cast<float*>(reinterpret_cast<char*>(T) +
                                         align_up(M * W * (int64_t)sizeof(float)));
  const int64_t N16 = (N + 15) / 16 * 16;
  // rows outside every cluster read zero sums (a zero value and gradient)
  if (rg && launch_fill(T, M * W, 0.0f, s) != hipSuccess) return KRED_ERR_HIP;
  if (launch_centre(y, N, D, m, s) != hipSuccess) return KRED_ERR_HIP;
  const bool xc = gradx_extra_col(p->flags, M, N, D, E);
  XCol xadd, xskip;
  kred_params p1 = *p;   // the last column's own call, when it rides with the first
  if (xc) {
    if (launch_gradx_signal(y, b, N, D, E, m, W - 1, 1, xsig, s) != hipSuccess ||
        launch_fill(xsig + N, N16 + 16 - N, 0.0f, s) != hipSuccess)
      return KRED_ERR_HIP;
    xadd.xb = xsig;
    xadd.xout = T + (int64_t)(W - 1) * M;
    xskip.skip = true;
    p1.col_blocks = 1;
  }
  for (int c0 = 0; c0 < W; c0 += 64) {
    const int Ec = std::min(64, W - c0);
    const bool last1 = xc && c0 == W - 1;
    if (!last1 && launch_gradx_signal(y, b, N, D, E, m, c0, Ec, sig, s) != hipSuccess)
      return KRED_ERR_HIP;
    // (the skipped call's signal: the same column, already in xsig)
    const kred_status st = run_mfma(ctx, KRED_F_GAUSS, KRED_R_SUM, last1 ? &p1 : p, M, N, D, Ec, x,
                                    y, last1 ? xsig : sig, T + (int64_t)c0 * M, s, 0, rg,
                                    !xc ? nullptr : c0 == 0 ? &xadd : last1 ? &xskip : nullptr);
    if (st != KRED_OK) return st;
  }
  const double sg = (double)p->sigma;
  const float gs = (float)(1.0 / (sg * sg));
  const hipError_t fin = e ? launch_vjp_finish(x, M, D, E, m, T, e, gs, out, s)
                           : launch_gradx_finish(x, M, D, m, T, gs, out, s);
  return fin == hipSuccess ? KRED_OK : KRED_ERR_HIP;
}

// One reduction on validated arguments, M > 0, on the current device;
// block-sparse when rg is given.
// The one-launch Gaussian sum (k_small.hip): D <= 4, E <= 4, below 2^28 pairs,
// neither KRED_FLAG_FAST nor KRED_FLAG_DIRECT.  Column blocks: enough for two
// workgroups per CU, at most kSumCols columns each (col_blocks, when given,
// raised to that minimum).
struct SmallPlan {
  int C = 1, jpb = 0;
  int64_t nrb = 0, part_bytes = 0;
};
bool small_plan(kred_formula f, kred_reduction r, const kred_params* p, int64_t M, int64_t N,
                int32_t D, int32_t E, int num_cus, SmallPlan* sp) {
  if (f != KRED_F_GAUSS || r != KRED_R_SUM || D > 4 || E < 1 || E > 4) return false;
  if (p->flags & (KRED_FLAG_FAST | KRED_FLAG_DIRECT)) return false;
  if (M <= 0 || N <= 0 || (double)M * (double)N >= kFastMinPairs) return false;
  const int64_t nrb = (M + kSumRows - 1) / kSumRows;
  if (nrb > kSumMaxRowBlocks) return false;
  const int64_t cmin = (N + kSumCols - 1) / kSumCols;
  int64_t C = p->col_blocks > 0 ? (int64_t)p->col_blocks
                                : std::max<int64_t>(1, (2 * (int64_t)num_cus + nrb - 1) / nrb);
  C = std::min<int64_t>(std::max(C, cmin), (N + 15) / 16);
  const int64_t jpb = std::min<int64_t>(kSumCols, ((N + C - 1) / C + 15) / 16 * 16);
  C = (N + jpb - 1) / jpb;   // every block has at least one column
  sp->C = (int)C;
  sp->jpb = (int)jpb;
  sp->nrb = nrb;
  sp->part_bytes = C > 1 ? align_up(C * M * E * (int64_t)sizeof(float)) : 0;
  return true;
}

kred_status run_small(kred_ctx* ctx, const kred_params* p, const SmallPlan& sp, int64_t M,
                      int64_t N, int32_t D, int32_t E, const float* x, const float* y,
                      const float* b, float* out, hipStream_t s) {
  float* part = nullptr;
  int* count = nullptr;
  if (sp.C > 1) {
    void* buf = nullptr;
    const kred_status gs = buffer(ctx, BUF_SCRATCH, (size_t)sp.part_bytes, &buf);
    if (gs != KRED_OK) return gs;
    part = static_cast<float*>(buf);
    if (ctx->arena) {
      count = static_cast<int*>(ctx->fixed);
    } else {
      if (ctx->counters == nullptr) {
        if (hipMalloc(reinterpret_cast<void**>(&ctx->counters), kCounterBytes) != hipSuccess) {
          (void)hipGetLastError();
          ctx->counters = nullptr;
          return KRED_ERR_NOMEM;
        }
        if (launch_fill(reinterpret_cast<float*>(ctx->counters), kSumMaxRowBlocks, 0.0f, s) !=
            hipSuccess)
          return KRED_ERR_HIP;
      }
      count = ctx->counters;
    }
  }
  SmallArgs a{};
  a.x = x;
  a.y = y;
  a.b = b;
  a.out = out;
  a.part = part;
  a.count = count;
  a.M = M;
  a.N = N;
  a.D = D;
  a.E = E;
  a.C = sp.C;
  a.jpb = sp.jpb;
  a.c64 = 1.4426950408889634 / (2.0 * (double)p->sigma * (double)p->sigma);
  a.s64 = std::sqrt(a.c64);
  // the matrix-core form's bound: 15 u L with the norms in the MFMA (D <= 3,
  // taken as 16 u L), (D + 10) u L otherwise
  a.limit = D <= 3 ? (float)(kWideBudget * 16777216.0 / 16.0) : wide_limit_f32(D);
  const bool prof = (p->flags & KRED_FLAG_PROFILE) != 0;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (prof) {
    e0 = next_event(ctx);
    e1 = next_event(ctx);
    if (!e0 || !e1 || hipEventRecord(e0, s) != hipSuccess) return KRED_ERR_HIP;
  }
  if (launch_small(a, s) != hipSuccess) return KRED_ERR_HIP;
  if (prof) {
    if (hipEventRecord(e1, s) != hipSuccess) return KRED_ERR_HIP;
    ctx->last_kernel = "small_kernel";
    ctx->last_fast = false;
    ctx->last_exact_D = 0;
  }
  return KRED_OK;
}

kred_status run_reduction(kred_ctx* ctx, kred_formula f, kred_reduction r, const kred_params* p,
                          int64_t M, int64_t N, int32_t D, int32_t E, const float* x,
                          const float* y, const float* b, void* out, hipStream_t s,
                          const Ranges* rg = nullptr) {
  if (N == 0) {
    int64_t count;
    float value;
    empty_fill(f, r, p, M, D, E, b, &count, &value);
    return launch_fill(static_cast<float*>(out), count, value, s) == hipSuccess ? KRED_OK
                                                                                : KRED_ERR_HIP;
  }

  // The squared distance's min and arg-min (without b) and its K smallest
  // values are read off the arg-K-min lists (K = 1 for min and arg-min).
  int kvalues = 0;
  kred_params pk;
  if (f == KRED_F_SQDIST && b == nullptr &&
      (r == KRED_R_MIN || r == KRED_R_ARGMIN || r == KRED_R_KMIN)) {
    kvalues = r != KRED_R_ARGMIN;
    pk = *p;
    if (r != KRED_R_KMIN) pk.K = 1;
    p = &pk;
    r = KRED_R_ARGKMIN;
  }
  const bool ext = is_extreme(r);
  if (ext && (b == nullptr || f == KRED_F_SINKHORN)) E = 1;   // one output column
  // kernel-side formula: log-sum-exps run on the Sinkhorn-form kernels
  const int kf = (r == KRED_R_LSE) ? (f == KRED_F_LAPLACE ? F_LAPLACE_LSE : F_SINKHORN) : (int)f;

  SmallPlan spl;
  if (!rg && small_plan(f, r, p, M, N, D, E, ctx->num_cus, &spl))
    return run_small(ctx, p, spl, M, N, D, E, x, y, b, static_cast<float*>(out), s);
  if (D > kMaxDirectD && f == KRED_F_GAUSS_GRADX)
    return run_gradx_wide(ctx, p, M, N, D, 1, x, y, b, nullptr, static_cast<float*>(out), s, rg);
  if (D > kMaxDirectD) return run_mfma(ctx, f, r, p, M, N, D, E, x, y, b, out, s, kvalues, rg);

  kred_params pr;
  if (rg) {
    // Column chunks of each cluster's list: enough workgroups for every CU.
    // The pattern lives on the device, so the row-block count is estimated
    // as max(clusters, M / rows per workgroup) with the kernel's rows per lane.
    pr = *p;
    if (pr.col_blocks == 0) {
      Plan probe;
      if (!make_plan(f, r, p, M, N, D, E, ctx->num_cus, &probe)) return KRED_ERR_UNSUPPORTED;
      const int R0 = probe.R;
      const int epi0 = fast_epi(f, r, M, N, D, E, p->flags, p->K);
      const int64_t rpb = epi0 >= 0 ? fast_rows_per_block(epi0, p->K) : (int64_t)kThreads * R0;
      const int64_t est = std::max<int64_t>({1, (int64_t)rg->nr, (M + rpb - 1) / rpb});
      pr.col_blocks = (int)std::min<int64_t>(64, ((int64_t)ctx->num_cus * 16 + est - 1) / est);
    }
    p = &pr;
  }
  const int epi = fast_epi(f, r, M, N, D, E, p->flags, p->K);
  Plan pl;
  if (!make_plan(f, r, p, M, N, D, E, ctx->num_cus, &pl,
                 epi >= 0 ? fast_rows_per_block(epi, p->K) : 0, epi >= 0 ? 256 : 1))
    return KRED_ERR_UNSUPPORTED;
  const FastScratch fs = fast_scratch(epi, N);
  // block-sparse: workgroup maps for the direct kernels and for the fast kernel
  const int64_t bstart_bytes =
      rg ? 2 * align_up((int64_t)(rg->nr + 1) * (int64_t)sizeof(int)) : 0;
  void* sp = nullptr;
  const kred_status gs =
      buffer(ctx, BUF_SCRATCH, (size_t)(pl.pack_bytes + pl.part_bytes + fs.guard_bytes +
                                        fs.apk_bytes + fs.ex_bytes + bstart_bytes), &sp);
  if (gs != KRED_OK) return gs;
  char* sbase = static_cast<char*>(sp);
  float* ypk = reinterpret_cast<float*>(sbase);
  float* part = pl.part_bytes ? reinterpret_cast<float*>(sbase + pl.pack_bytes) : nullptr;
  char* fbase = sbase + pl.pack_bytes + pl.part_bytes;
  int* bstart = rg ? reinterpret_cast<int*>(fbase + fs.guard_bytes + fs.apk_bytes + fs.ex_bytes)
                   : nullptr;
  int* fbstart = rg ? reinterpret_cast<int*>(reinterpret_cast<char*>(bstart) + bstart_bytes / 2)
                    : nullptr;
  FastGuard* guard = epi >= 0 ? reinterpret_cast<FastGuard*>(fbase) : nullptr;
  // largest c R^2 the fast path takes: every kernel of the call tests the same
  const float flimit = fast_limit(D, epi == FAST_MIN || epi == FAST_KNN);
  const bool prof = (p->flags & KRED_FLAG_PROFILE) != 0;

  FastArgs fa{};
  if (epi >= 0) {
    FastPackArgs fp{};
    fp.epi = epi;
    fp.D = D;
    fp.N = N;
    fp.N16 = (N + 15) / 16 * 16;
    fp.y = y;
    fp.b = b;
    fp.scale = pl.fscale;
    fp.scale64 = pl.fscale64;
    fp.limit = flimit;
    fp.guard = guard;
    fp.apk = reinterpret_cast<uint4*>(fbase + fs.guard_bytes);
    fp.ex = (epi == FAST_GRADX || epi == FAST_SUMV)
                ? reinterpret_cast<float4*>(fbase + fs.guard_bytes + fs.apk_bytes)
                : nullptr;
    fp.E = E;
    fp.eb = epi == FAST_SUM ? reinterpret_cast<float*>(fbase + fs.guard_bytes + fs.apk_bytes)
                            : nullptr;
    if (launch_fast_prologue(fp, x, M, s) != hipSuccess) return KRED_ERR_HIP;
    fa.epi = epi;
    fa.D = D;
    fa.DP = pl.DP;
    fa.M = M;
    fa.N = N;
    fa.N16 = fp.N16;
    fa.C = pl.C;
    fa.jpb = pl.jpb;
    fa.x = x;
    fa.scale = pl.fscale;
    fa.scale64 = pl.fscale64;
    fa.limit = flimit;
    fa.gscale = pl.gscale;
    fa.guard = guard;
    fa.apk = fp.apk;
    fa.ex = fp.ex;
    fa.eb = fp.eb;
    fa.out = out;
    fa.part = part;
    fa.kvalues = kvalues;
    fa.K = pl.K;
    fa.KP = pl.KP;
    fa.y = y;
    fa.E = E;
    fa.EP = direct_pad_e(std::min(16, E));
    if (rg) {
      fa.nr = rg->nr;
      fa.rr = rg->rr;
      fa.cp = rg->cp;
      fa.cr = rg->cr;
      fa.bstart = fbstart;
      if (launch_range_blocks(rg->rr, rg->nr, M, fast_rows_per_block(epi, p->K), fbstart, s) !=
          hipSuccess)
        return KRED_ERR_HIP;
    }
  }
  const int n_slices = (r == KRED_R_ARGKMIN) ? 1 : (pl.E + 15) / 16;
  for (int sl = 0; sl < n_slices; ++sl) {
    const int e0 = sl * 16;
    const int EP = (r == KRED_R_ARGKMIN) ? 1 : direct_pad_e(std::min(16, pl.E - e0));
    PackArgs pa{};
    pa.y = y;
    pa.b = (r == KRED_R_ARGKMIN) ? nullptr : b;
    pa.ypk = ypk;
    pa.N = N;
    pa.D = D;
    pa.DP = pl.DP;
    pa.E = pl.E;
    pa.EP = EP;
    pa.e0 = e0;
    pa.yscale = pl.xscale;
    pa.bscale = pl.bscale;
    pa.guard = guard;
    pa.fscale = pl.fscale;
    pa.flimit = flimit;
    pa.unit_b = ext && b == nullptr;   // squared-distance max without b: F = d * 1
    if (launch_pack(pa, s) != hipSuccess) return KRED_ERR_HIP;

    DirectArgs da{};
    da.formula = kf;
    da.D = D;
    da.DP = pl.DP;
    da.E = pl.E;
    da.EP = EP;
    da.e0 = e0;
    da.M = M;
    da.N = N;
    da.C = pl.C;
    da.jpb = pl.jpb;
    da.x = x;
    da.ypk = ypk;
    da.xscale = pl.xscale;
    da.kscale = pl.kscale;
    da.gscale = pl.gscale;
    da.fscale = pl.fscale;
    da.flimit = flimit;
    da.out = out;
    da.part = part;
    da.KP = pl.KP;
    da.K = pl.K;
    da.rows = pl.R;
    da.guard = guard;
    da.ext = ext;
    da.ext_sign = is_max(r) ? -1.0f : 1.0f;
    da.arg = is_arg(r);
    da.kvalues = kvalues;
    if (rg) {
      da.nr = rg->nr;
      da.rr = rg->rr;
      da.cp = rg->cp;
      da.cr = rg->cr;
      da.bstart = bstart;
      if (launch_range_blocks(rg->rr, rg->nr, M, kThreads * direct_rows_for(da), bstart, s) !=
          hipSuccess)
        return KRED_ERR_HIP;
      if (pl.C > 1) {
        // rows outside every cluster get no partials from the kernels: start
        // every partial at the empty value, so the combine yields the empty
        // reduction for them
        const int W = partial_width(kf, pl.DP, EP, pl.KP, ext);
        float v0 = 0.0f, v1 = 0.0f;
        if (kf == F_SINKHORN || kf == F_LAPLACE_LSE) v0 = -INFINITY;   // (m, s) = (-inf, 0)
        if (pl.KP > 0) {
          v0 = INFINITY;
          v1 = __builtin_bit_cast(float, (int32_t)INT32_MAX);   // (distance, index)
        }
        if (ext) {
          v0 = INFINITY;
          v1 = __builtin_bit_cast(float, (int32_t)-1);          // (sign * value, index)
        }
        if (launch_fill2(part, (int64_t)pl.C * M * W, v0, v1, s) != hipSuccess) return KRED_ERR_HIP;
      }
    }
    hipEvent_t e_start = nullptr, e_stop = nullptr;
    if (prof) {
      e_start = next_event(ctx);
      e_stop = next_event(ctx);
      if (!e_start || !e_stop || hipEventRecord(e_start, s) != hipSuccess) return KRED_ERR_HIP;
    }
    // with the fast path eligible, both launch and exactly one does the work
    if (epi >= 0 && launch_fast(fa, s) != hipSuccess) return KRED_ERR_HIP;
    if (launch_direct(da, s) != hipSuccess) return KRED_ERR_HIP;
    if (prof) {
      if (hipEventRecord(e_stop, s) != hipSuccess) return KRED_ERR_HIP;
      ctx->last_exact_D = 0;
      const char* direct = ext                       ? "extreme_kernel"
                           : (r == KRED_R_ARGKMIN)     ? "knn_kernel"
                           : (f == KRED_F_GAUSS_GRADX) ? "gradx_kernel"
                           : (r == KRED_R_LSE)         ? "lse_kernel"
                                                       : "sum_kernel";
      ctx->last_kernel = direct;
      ctx->last_fast = false;
      if (epi >= 0) {
        // which of the two did the work is known on the device only
        if (ctx->fast_counts == nullptr) {
          if (hipMalloc(reinterpret_cast<void**>(&ctx->fast_counts), 2 * sizeof(int)) != hipSuccess) {
            ctx->fast_counts = nullptr;
            return KRED_ERR_NOMEM;
          }
          if (hipMemset(ctx->fast_counts, 0, 2 * sizeof(int)) != hipSuccess) return KRED_ERR_HIP;
        }
        if (launch_fast_record(guard, D, pl.fscale, flimit, ctx->fast_counts, s) != hipSuccess)
          return KRED_ERR_HIP;
        ctx->last_fast = true;
        ctx->choice_yes = "fast_kernel";
        ctx->last_direct = direct;
      }
    }
    if (pl.C > 1) {
      CombineArgs ca{};
      ca.formula = kf;
      ca.D = D;
      ca.DP = pl.DP;
      ca.E = pl.E;
      ca.EP = EP;
      ca.e0 = e0;
      ca.M = M;
      ca.C = pl.C;
      ca.part = part;
      ca.out = out;
      ca.gscale = pl.gscale;
      ca.KP = pl.KP;
      ca.K = pl.K;
      ca.ext = ext;
      ca.ext_sign = da.ext_sign;
      ca.arg = da.arg;
      ca.kvalues = kvalues;
      if (launch_combine(ca, s) != hipSuccess) return KRED_ERR_HIP;
    }
  }
  return KRED_OK;
}

// x-gradient of L = sum_i <e_i, a_i> for the Gaussian sum a = K b (D <= 16),
// on validated arguments with M, N > 0.  With one signal column and the
// matrix-core path eligible, the fused value + gradient reduction runs and its
// gradient is scaled by the scalar cotangent; otherwise the direct-form
// vector-Jacobian kernel runs once per E-slice of 16.  With a block-sparse
// pattern rg the sums run over each row cluster's column ranges only, and
// rows outside every cluster get zero.
kred_status run_vjp(kred_ctx* ctx, const kred_params* p, int64_t M, int64_t N, int32_t D,
                    int32_t E, const float* x, const float* y, const float* b, const float* e,
                    float* g, hipStream_t s, const Ranges* rg = nullptr) {
  // 16 < D <= 256 with several signal columns: the Gaussian sum with the
  // E (D + 1) columns [b_e, b_e (y - m)], contracted with e
  if (D > kMaxDirectD && E > 1) return run_gradx_wide(ctx, p, M, N, D, E, x, y, b, e, g, s, rg);
  if (E == 1 && (D > kMaxDirectD || fast_epi(KRED_F_GAUSS_GRADX, KRED_R_SUM, M, N, D, 1, p->flags) >= 0)) {
    void* ap = nullptr;
    const kred_status ga = buffer(ctx, BUF_AUX, (size_t)(M * (1 + D) * (int64_t)sizeof(float)), &ap);
    if (ga != KRED_OK) return ga;
    float* fused = static_cast<float*>(ap);
    if (rg && launch_fill(fused, M * (1 + D), 0.0f, s) != hipSuccess) return KRED_ERR_HIP;
    const kred_status st =
        run_reduction(ctx, KRED_F_GAUSS_GRADX, KRED_R_SUM, p, M, N, D, 1, x, y, b, fused, s, rg);
    if (st != KRED_OK) return st;
    return launch_scale_rows(fused, M, D, e, g, s) == hipSuccess ? KRED_OK : KRED_ERR_HIP;
  }
  kred_params pr;
  if (rg) {
    pr = *p;
    if (pr.col_blocks == 0) {
      // chunks of each cluster's columns, as for the block-sparse reductions
      Plan probe;
      if (!make_plan((kred_formula)F_VJP, KRED_R_SUM, p, M, N, D, E, ctx->num_cus, &probe))
        return KRED_ERR_UNSUPPORTED;
      const int64_t rpb = (int64_t)kThreads * probe.R;
      const int64_t est = std::max<int64_t>({1, (int64_t)rg->nr, (M + rpb - 1) / rpb});
      pr.col_blocks = (int)std::min<int64_t>(64, ((int64_t)ctx->num_cus * 16 + est - 1) / est);
    }
    p = &pr;
  }
  Plan pl;
  if (!make_plan((kred_formula)F_VJP, KRED_R_SUM, p, M, N, D, E, ctx->num_cus, &pl))
    return KRED_ERR_UNSUPPORTED;
  const int64_t bstart_bytes = rg ? align_up((int64_t)(rg->nr + 1) * (int64_t)sizeof(int)) : 0;
  void* sp = nullptr;
  const kred_status gs =
      buffer(ctx, BUF_SCRATCH, (size_t)(pl.pack_bytes + pl.part_bytes + bstart_bytes), &sp);
  if (gs != KRED_OK) return gs;
  char* sbase = static_cast<char*>(sp);
  float* ypk = reinterpret_cast<float*>(sbase);
  float* part = pl.part_bytes ? reinterpret_cast<float*>(sbase + pl.pack_bytes) : nullptr;
  int* bstart = rg ? reinterpret_cast<int*>(sbase + pl.pack_bytes + pl.part_bytes) : nullptr;
  const bool prof = (p->flags & KRED_FLAG_PROFILE) != 0;
  if (rg) {
    // rows outside every cluster: zero output, and zero partials, which the
    // kernels never write for them
    if (launch_fill(g, M * D, 0.0f, s) != hipSuccess) return KRED_ERR_HIP;
    if (pl.C > 1 && launch_fill2(part, (int64_t)pl.C * M * pl.DP, 0.0f, 0.0f, s) != hipSuccess)
      return KRED_ERR_HIP;
  }
  const int n_slices = (E + 15) / 16;
  for (int sl = 0; sl < n_slices; ++sl) {
    const int e0 = sl * 16;
    const int EP = direct_pad_e(std::min(16, E - e0));
    PackArgs pa{};
    pa.y = y;
    pa.b = b;
    pa.ypk = ypk;
    pa.N = N;
    pa.D = D;
    pa.DP = pl.DP;
    pa.E = E;
    pa.EP = EP;
    pa.e0 = e0;
    pa.yscale = 1.0f;
    pa.bscale = 1.0f;
    if (launch_pack(pa, s) != hipSuccess) return KRED_ERR_HIP;

    DirectArgs da{};
    da.formula = F_VJP;
    da.D = D;
    da.DP = pl.DP;
    da.E = E;
    da.EP = EP;
    da.e0 = e0;
    da.M = M;
    da.N = N;
    da.C = pl.C;
    da.jpb = pl.jpb;
    da.x = x;
    da.ypk = ypk;
    da.xscale = 1.0f;
    da.kscale = pl.kscale;
    da.gscale = pl.gscale;
    da.out = g;
    da.part = part;
    da.xe = e;
    da.accumulate = sl > 0;
    if (rg) {
      da.nr = rg->nr;
      da.rr = rg->rr;
      da.cp = rg->cp;
      da.cr = rg->cr;
      da.bstart = bstart;
      // the workgroup map depends on the rows per lane, which depend on the
      // slice's width: rebuilt per slice (stream order keeps the previous
      // slice's kernel ahead of the rewrite)
      if (launch_range_blocks(rg->rr, rg->nr, M, kThreads * direct_rows_for(da), bstart, s) !=
          hipSuccess)
        return KRED_ERR_HIP;
    }
    hipEvent_t e_start = nullptr, e_stop = nullptr;
    if (prof) {
      e_start = next_event(ctx);
      e_stop = next_event(ctx);
      if (!e_start || !e_stop || hipEventRecord(e_start, s) != hipSuccess) return KRED_ERR_HIP;
    }
    if (launch_direct(da, s) != hipSuccess) return KRED_ERR_HIP;
    if (prof) {
      if (hipEventRecord(e_stop, s) != hipSuccess) return KRED_ERR_HIP;
      ctx->last_exact_D = 0;
      ctx->last_kernel = "vjp_kernel";
      ctx->last_fast = false;
    }
    if (pl.C > 1) {
      CombineArgs ca{};
      ca.formula = F_VJP;
      ca.D = D;
      ca.DP = pl.DP;
      ca.E = E;
      ca.EP = EP;
      ca.e0 = e0;
      ca.M = M;
      ca.C = pl.C;
      ca.part = part;
      ca.out = g;
      ca.gscale = pl.gscale;
      ca.accumulate = sl > 0;
      if (launch_combine(ca, s) != hipSuccess) return KRED_ERR_HIP;
    }
  }
  return KRED_OK;
}

}  // namespace

extern "C" {

const char* kred_strerror(kred_status s) {
  switch (code_of(&s)) {
    case KRED_OK: return "success";
    case KRED_ERR_INVALID_ARG: return "invalid argument";
    case KRED_ERR_UNSUPPORTED: return "unsupported formula/reduction/size combination";
    case KRED_ERR_NOMEM: return "out of device memory for scratch";
    case KRED_ERR_HIP: return "HIP runtime error";
    case KRED_ERR_NO_DEVICE: return "no usable gfx950 device";
    case KRED_ERR_SCRATCH: return "the call needs more than the no-allocation entry point's fixed scratch";
  }
  return "unknown status";
}

int32_t kred_version(void) { return KRED_VERSION; }

kred_status kred_validate(kred_formula f, kred_reduction r, const kred_params* p, int64_t M,
                          int64_t N, int32_t D, int32_t E, const void* x, const void* y,
                          const void* b, const void* out) {
  if (p == nullptr) return KRED_ERR_INVALID_ARG;
  if (code_of(&f) < KRED_F_GAUSS || code_of(&f) > KRED_F_SINKHORN) return KRED_ERR_INVALID_ARG;
  if (code_of(&r) < KRED_R_SUM || code_of(&r) > KRED_R_KMIN) return KRED_ERR_INVALID_ARG;
  if (M < 0 || N < 0 || M > INT32_MAX || N > INT32_MAX) return KRED_ERR_INVALID_ARG;
  if (D < 1 || D > KRED_MAX_D) return KRED_ERR_INVALID_ARG;
  if (p->col_blocks < 0 || p->col_blocks > KRED_MAX_COL_BLOCKS) return KRED_ERR_INVALID_ARG;
  bool needs_b = true;
  if (r == KRED_R_SUM && (f == KRED_F_GAUSS || f == KRED_F_LAPLACE || f == KRED_F_SQDIST)) {
    if (E < 1 || E > KRED_MAX_E) return KRED_ERR_INVALID_ARG;
    if (f != KRED_F_SQDIST && !finite_pos(p->sigma)) return KRED_ERR_INVALID_ARG;
  } else if (r == KRED_R_SUM && f == KRED_F_GAUSS_GRADX) {
    if (E != 1) return KRED_ERR_INVALID_ARG;
    if (!finite_pos(p->sigma)) return KRED_ERR_INVALID_ARG;
  } else if (r == KRED_R_LSE &&
             (f == KRED_F_SINKHORN || f == KRED_F_GAUSS || f == KRED_F_LAPLACE)) {
    if (E != 1) return KRED_ERR_INVALID_ARG;
    if (!finite_pos(f == KRED_F_SINKHORN ? p->eps : p->sigma)) return KRED_ERR_INVALID_ARG;
  } else if ((r == KRED_R_ARGKMIN || r == KRED_R_KMIN) && f == KRED_F_SQDIST) {
    if (b != nullptr) return KRED_ERR_INVALID_ARG;
    if (p->K < 1 || p->K > KRED_MAX_K || p->K > N) return KRED_ERR_INVALID_ARG;
    needs_b = false;
  } else if (is_extreme(r) && f != KRED_F_GAUSS_GRADX) {
    if (f == KRED_F_SINKHORN) {
      if (E != 1 || !finite_pos(p->eps)) return KRED_ERR_INVALID_ARG;
    } else if (f == KRED_F_SQDIST && b == nullptr) {
      needs_b = false;   // F = d; E is ignored
    } else {
      if (E < 1 || E > KRED_MAX_E) return KRED_ERR_INVALID_ARG;
      if (f != KRED_F_SQDIST && !finite_pos(p->sigma)) return KRED_ERR_INVALID_ARG;
    }
  } else {
    return KRED_ERR_UNSUPPORTED;
  }
  // Paths: the direct-form kernels cover D <= 16 and the matrix-core kernels
  // 16 < D <= 256, for every pair.
  if (M == 0) return KRED_OK;
  if (x == nullptr || out == nullptr) return KRED_ERR_INVALID_ARG;
  if (N > 0 && (y == nullptr || (needs_b && b == nullptr))) return KRED_ERR_INVALID_ARG;
  if (misaligned(x) || misaligned(y) || misaligned(b) || misaligned(out))
    return KRED_ERR_INVALID_ARG;
  return KRED_OK;
}

}  // extern "C"

namespace {
// Device bytes a validated kred_run call asks for, on a device with num_cus
// compute units (the column split depends on it).
int64_t scratch_need(kred_formula f, kred_reduction r, const kred_params* p, int64_t M, int64_t N,
                     int32_t D, int32_t E, int num_cus) {
  const float dummy = 0.0f;
  // E = 0 with the squared distance's min / max reductions means "without b"
  const bool nob = r == KRED_R_ARGKMIN || r == KRED_R_KMIN ||
                   (f == KRED_F_SQDIST && is_extreme(r) && E == 0);
  const void* bp = nob ? nullptr : &dummy;
  if (kred_validate(f, r, p, M, N, D, E, &dummy, &dummy, bp, &dummy) != KRED_OK) return -1;
  if (M == 0 || N == 0) return 0;
  kred_params pk = *p;
  if (nob && (r == KRED_R_KMIN || r == KRED_R_MIN || r == KRED_R_ARGMIN)) {
    if (r != KRED_R_KMIN) pk.K = 1;
    r = KRED_R_ARGKMIN;
    p = &pk;
  }
  if (is_extreme(r) && (nob || f == KRED_F_SINKHORN)) E = 1;
  SmallPlan spl;
  if (small_plan(f, r, p, M, N, D, E, num_cus, &spl)) return spl.part_bytes;
  if (D > kMaxDirectD) {
    // the fused value + gradient runs Gaussian sums of up to 64 signal columns
    const bool wide = f == KRED_F_GAUSS_GRADX;
    MPlan mp;
    if (!make_mplan(wide ? KRED_F_GAUSS : f, r, p, M, N, D, wide ? std::min(64, D + 1) : E,
                    num_cus, &mp))
      return -1;
    const bool xc = wide && gradx_extra_col(p->flags, M, N, D, 1);
    return mp.yop_bytes + mp.ny_bytes + mp.b_bytes + mp.part_bytes +
           mfma_bf16_bytes(mp, r == KRED_R_ARGKMIN, p->flags, M, N) +
           (r == KRED_R_ARGKMIN ? 0 : align_up((int64_t)D * (int64_t)sizeof(float)) +
                                          align_up(sizeof(SpreadGuard))) +
           (wide ? gradx_wide_bytes(M, N, D) : 0) +
           ((xc && mp.C > 1) ? align_up((int64_t)mp.C * M * (int64_t)sizeof(float)) : 0);
  }
  const int epi = fast_epi(f, r, M, N, D, E, p->flags, p->K);
  Plan pl;
  if (!make_plan(f, r, p, M, N, D, E, num_cus, &pl,
                 epi >= 0 ? fast_rows_per_block(epi, p->K) : 0, epi >= 0 ? 256 : 1))
    return -1;
  const FastScratch fs = fast_scratch(epi, N);
  return pl.pack_bytes + pl.part_bytes + fs.guard_bytes + fs.apk_bytes + fs.ex_bytes;
}
}  // namespace

extern "C" {

int64_t kred_scratch_bytes(kred_formula f, kred_reduction r, const kred_params* p, int64_t M,
                           int64_t N, int32_t D, int32_t E) {
  return scratch_need(f, r, p, M, N, D, E, 256);
}

kred_status kred_create(kred_ctx** ctx, int device) {
  if (ctx == nullptr) return KRED_ERR_INVALID_ARG;
  *ctx = nullptr;
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || device < 0 || device >= n) {
    (void)hipGetLastError();
    return KRED_ERR_NO_DEVICE;
  }
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, device) != hipSuccess) return KRED_ERR_NO_DEVICE;
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0) return KRED_ERR_NO_DEVICE;
  void* fixed = nullptr;
  {
    // the no-allocation entry point's scratch: its address on this device,
    // looked up once per device with that device current
    std::lock_guard<std::mutex> lock(g_fixed_mu);
    if (device < kMaxDevices && g_fixed[device] == nullptr) {
      DeviceGuard dg(device);
      void* ptr = nullptr;
      if (!dg.ok || hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) {
        (void)hipGetLastError();
        return KRED_ERR_HIP;
      }
      g_fixed[device] = ptr;
    }
    if (device < kMaxDevices) fixed = g_fixed[device];
  }
  kred_ctx* c = new (std::nothrow) kred_ctx();
  if (c == nullptr) return KRED_ERR_NOMEM;
  c->device = device;
  c->num_cus = prop.multiProcessorCount;
  c->fixed = fixed;
  *ctx = c;
  return KRED_OK;
}

kred_status kred_destroy(kred_ctx* ctx) {
  if (ctx == nullptr) return KRED_OK;
  kred_status st = KRED_OK;
  {
    DeviceGuard g(ctx->device);
    if (hipDeviceSynchronize() != hipSuccess) st = KRED_ERR_HIP;
    if (ctx->scratch) (void)hipFree(ctx->scratch);
    if (ctx->aux) (void)hipFree(ctx->aux);
    if (ctx->wide) (void)hipFree(ctx->wide);
    if (ctx->exact_guard) (void)hipFree(ctx->exact_guard);
    if (ctx->fast_counts) (void)hipFree(ctx->fast_counts);
    if (ctx->counters) (void)hipFree(ctx->counters);
    for (hipEvent_t e : ctx->ev) (void)hipEventDestroy(e);
  }
  delete ctx;
  return st;
}

kred_status kred_run(kred_ctx* ctx, kred_formula f, kred_reduction r, const kred_params* p,
                     int64_t M, int64_t N, int32_t D, int32_t E, const float* x, const float* y,
                     const float* b, void* out, void* stream) {
  if (ctx == nullptr) return KRED_ERR_INVALID_ARG;
  const kred_status v = kred_validate(f, r, p, M, N, D, E, x, y, b, out);
  if (v != KRED_OK) return v;
  if (M == 0) return KRED_OK;
  DeviceGuard devg(ctx->device);
  if (!devg.ok) return KRED_ERR_HIP;
  return run_reduction(ctx, f, r, p, M, N, D, E, x, y, b, out, static_cast<hipStream_t>(stream));
}

kred_status kred_run_noalloc(kred_ctx* ctx, kred_formula f, kred_reduction r,
                             const kred_params* p, int64_t M, int64_t N, int32_t D, int32_t E,
                             const float* x, const float* y, const float* b, void* out,
                             void* stream) {
  if (ctx == nullptr) return KRED_ERR_INVALID_ARG;
  const kred_status v = kred_validate(f, r, p, M, N, D, E, x, y, b, out);
  if (v != KRED_OK) return v;
  // profiling creates events, which allocate
  if (p->flags & KRED_FLAG_PROFILE) return KRED_ERR_INVALID_ARG;
  if (M == 0) return KRED_OK;
  if (ctx->fixed == nullptr) return KRED_ERR_NO_DEVICE;   // device ordinal beyond the table
  // every region the call carves (at most four kinds, each aligned), checked
  // before anything is launched
  const int64_t need = N == 0 ? 0 : scratch_need(f, r, p, M, N, D, E, ctx->num_cus);
  if (need < 0) return KRED_ERR_UNSUPPORTED;
  if (need + (int64_t)BUF_KINDS * kAlign + align_up(sizeof(ExactGuard)) >
      (int64_t)(KRED_NOALLOC_SCRATCH_BYTES - kCounterBytes))
    return KRED_ERR_SCRATCH;
  DeviceGuard devg(ctx->device);
  if (!devg.ok) return KRED_ERR_HIP;
  Arena a;
  a.base = static_cast<char*>(ctx->fixed) + kCounterBytes;
  a.cap = KRED_NOALLOC_SCRATCH_BYTES - kCounterBytes;
  ctx->arena = &a;
  const kred_status st =
      run_reduction(ctx, f, r, p, M, N, D, E, x, y, b, out, static_cast<hipStream_t>(stream));
  ctx->arena = nullptr;
  return st;
}

kred_status kred_cluster_pattern(kred_ctx* ctx, int64_t M, int64_t N, int32_t D, const float* x,
                                 const float* y, double cell, double cutoff, int32_t* order_x,
                                 int32_t* order_y, int32_t* row_ranges, int32_t* col_ptr,
                                 int32_t* col_ranges, int64_t col_cap, int64_t* counts,
                                 void* stream) {
  if (ctx == nullptr) return KRED_ERR_INVALID_ARG;
  if (M < 1 || N < 1 || M > INT32_MAX - 1 || N > INT32_MAX - 1 || D < 1 || D > kClusterMaxD ||
      col_cap < 0)
    return KRED_ERR_INVALID_ARG;
  if (!(cell > 0.0) || !std::isfinite(cell) || !(cutoff >= 0.0) || !std::isfinite(cutoff))
    return KRED_ERR_INVALID_ARG;
  if (!x || !y || !order_x || !order_y || !row_ranges || !col_ptr || !counts ||
      (col_cap > 0 && !col_ranges))
    return KRED_ERR_INVALID_ARG;
  ClusterCall c{};
  c.x = x;
  c.y = y;
  c.M = M;
  c.N = N;
  c.D = D;
  c.cell = cell;
  {
    // the reach r = cutoff + cell sqrt(D) and r^2, rounded step by step (no
    // fused multiply-add), as the host construction computes them
#pragma clang fp contract(off)
    const double t = cell * std::sqrt((double)D);
    const double reach = cutoff + t;
    c.reach2 = reach * reach;
  }
  c.order_x = order_x;
  c.order_y = order_y;
  c.row_ranges = row_ranges;
  c.col_ptr = col_ptr;
  c.col_ranges = col_ranges;
  c.col_cap = col_cap;
  c.counts = counts;
  DeviceGuard devg(ctx->device);
  if (!devg.ok) return KRED_ERR_HIP;
  const size_t bytes = cluster_scratch_bytes(M, N);
  void* sp = nullptr;
  const kred_status gs = buffer(ctx, BUF_SCRATCH, bytes, &sp);
  if (gs != KRED_OK) return gs;
  return build_cluster_pattern(c, sp, bytes, static_cast<hipStream_t>(stream)) == hipSuccess
             ? KRED_OK
             : KRED_ERR_HIP;
}

kred_status kred_gather_rows(kred_ctx* ctx, int64_t n, int32_t width, const float* src,
                             const int32_t* index, float* dst, int32_t inverse, void* stream) {
  if (ctx == nullptr || n < 0 || width < 1 || (inverse != 0 && inverse != 1)) return KRED_ERR_INVALID_ARG;
  if (n == 0) return KRED_OK;
  if (!src || !index || !dst || src == dst) return KRED_ERR_INVALID_ARG;
  DeviceGuard devg(ctx->device);
  if (!devg.ok) return KRED_ERR_HIP;
  return launch_gather_rows(src, index, n, width, inverse, dst, static_cast<hipStream_t>(stream)) ==
                 hipSuccess
             ? KRED_OK
             : KRED_ERR_HIP;
}

kred_status kred_validate_ranges(kred_formula f, kred_reduction r, const kred_params* p,
                                 int64_t M, int64_t N, int32_t D, int32_t E, const void* x,
                                 const void* y, const void* b, const void* out, int32_t nr,
                                 const void* row_ranges, const void* col_ptr,
                                 const void* col_ranges) {
  const kred_status v = kred_validate(f, r, p, M, N, D, E, x, y, b, out);
  if (v != KRED_OK) return v;
  if (nr < 0) return KRED_ERR_INVALID_ARG;
  if (nr > 0 && (row_ranges == nullptr || col_ptr == nullptr || col_ranges == nullptr))
    return KRED_ERR_INVALID_ARG;
  if (misaligned(row_ranges) || misaligned(col_ptr) || misaligned(col_ranges))
    return KRED_ERR_INVALID_ARG;
  return KRED_OK;
}

kred_status kred_run_ranges(kred_ctx* ctx, kred_formula f, kred_reduction r, const kred_params* p,
                            int64_t M, int64_t N, int32_t D, int32_t E, const float* x,
                            const float* y, const float* b, void* out, int32_t nr,
                            const int32_t* row_ranges, const int32_t* col_ptr,
                            const int32_t* col_ranges, void* stream) {
  if (ctx == nullptr) return KRED_ERR_INVALID_ARG;
  const kred_status v = kred_validate_ranges(f, r, p, M, N, D, E, x, y, b, out, nr, row_ranges,
                                             col_ptr, col_ranges);
  if (v != KRED_OK) return v;
  if (M == 0) return KRED_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  DeviceGuard devg(ctx->device);
  if (!devg.ok) return KRED_ERR_HIP;
  // rows outside every cluster (and clusters without columns) hold the empty reduction
  int64_t count;
  float value;
  empty_fill(f, r, p, M, D, E, b, &count, &value);
  if (launch_fill(static_cast<float*>(out), count, value, s) != hipSuccess) return KRED_ERR_HIP;
  if (nr == 0 || N == 0) return KRED_OK;
  const Ranges rg{nr, row_ranges, col_ptr, col_ranges};
  return run_reduction(ctx, f, r, p, M, N, D, E, x, y, b, out, s, &rg);
}

kred_status kred_validate_backward(const kred_params* p, int64_t M, int64_t N, int32_t D,
                                   int32_t E, const void* x, const void* y, const void* b,
                                   const void* e, const void* gx, const void* gy,
                                   const void* gb) {
  if (p == nullptr || !finite_pos(p->sigma)) return KRED_ERR_INVALID_ARG;
  if (p->col_blocks < 0 || p->col_blocks > KRED_MAX_COL_BLOCKS) return KRED_ERR_INVALID_ARG;
  if (M < 0 || N < 0 || M > INT32_MAX || N > INT32_MAX) return KRED_ERR_INVALID_ARG;
  if (D < 1 || D > KRED_MAX_D || E < 1 || E > KRED_MAX_E) return KRED_ERR_INVALID_ARG;

  // Inputs the requested outputs read.  With M = 0 or N = 0 every reduction
  // is empty and the outputs are filled with zeros without reading any input.
  if (M > 0 && N > 0 && (gx || gy || gb)) {
    if (x == nullptr || y == nullptr || e == nullptr) return KRED_ERR_INVALID_ARG;
    if ((gx || gy) && b == nullptr) return KRED_ERR_INVALID_ARG;
  }
  for (const void* q : {x, y, b, e, gx, gy, gb})
    if (misaligned(q)) return KRED_ERR_INVALID_ARG;
  return KRED_OK;
}

kred_status kred_gauss_backward(kred_ctx* ctx, const kred_params* p, int64_t M, int64_t N,
                                int32_t D, int32_t E, const float* x, const float* y,
                                const float* b, const float* e, float* gx, float* gy, float* gb,
                                void* stream) {
  if (ctx == nullptr) return KRED_ERR_INVALID_ARG;
  const kred_status v = kred_validate_backward(p, M, N, D, E, x, y, b, e, gx, gy, gb);
  if (v != KRED_OK) return v;
  hipStream_t s = static_cast<hipStream_t>(stream);
  DeviceGuard devg(ctx->device);
  if (!devg.ok) return KRED_ERR_HIP;
  kred_status st = KRED_OK;
  // dL/dx_i: sum over j of k_ij <e_i, b_j> (y_j - x_i) / sigma^2
  if (gx && M > 0) {
    st = N == 0 ? (launch_fill(gx, M * D, 0.0f, s) == hipSuccess ? KRED_OK : KRED_ERR_HIP)
                : run_vjp(ctx, p, M, N, D, E, x, y, b, e, gx, s);
    if (st != KRED_OK) return st;
  }
  // dL/dy_j: the same reduction with the roles of (x, e) and (y, b) exchanged
  if (gy && N > 0) {
    st = M == 0 ? (launch_fill(gy, N * D, 0.0f, s) == hipSuccess ? KRED_OK : KRED_ERR_HIP)
                : run_vjp(ctx, p, N, M, D, E, y, x, e, b, gy, s);
    if (st != KRED_OK) return st;
  }
  // dL/db_j = sum_i k_ij e_i: the Gaussian sum with x and y exchanged
  if (gb && N > 0) {
    st = M == 0 ? (launch_fill(gb, N * E, 0.0f, s) == hipSuccess ? KRED_OK : KRED_ERR_HIP)
                : run_reduction(ctx, KRED_F_GAUSS, KRED_R_SUM, p, N, M, D, E, y, x, e, gb, s);
    if (st != KRED_OK) return st;
  }
  return KRED_OK;
}

kred_status kred_validate_backward_ranges(const kred_params* p, int64_t M, int64_t N, int32_t D,
                                          int32_t E, const void* x, const void* y, const void* b,
                                          const void* e, const void* gx, const void* gy,
                                          const void* gb, int32_t nr, const void* row_ranges,
                                          const void* col_ptr, const void* col_ranges, int32_t nc,
                                          const void* col_clusters, const void* row_ptr,
                                          const void* row_ranges_t) {
  const kred_status v = kred_validate_backward(p, M, N, D, E, x, y, b, e, gx, gy, gb);
  if (v != KRED_OK) return v;
  if (nr < 0 || nc < 0) return KRED_ERR_INVALID_ARG;
  // the row-cluster pattern serves gx, the column-cluster pattern gy and gb
  if (gx && nr > 0 && (row_ranges == nullptr || col_ptr == nullptr || col_ranges == nullptr))
    return KRED_ERR_INVALID_ARG;
  if ((gy || gb) && nc > 0 &&
      (col_clusters == nullptr || row_ptr == nullptr || row_ranges_t == nullptr))
    return KRED_ERR_INVALID_ARG;
  for (const void* q : {row_ranges, col_ptr, col_ranges, col_clusters, row_ptr, row_ranges_t})
    if (misaligned(q)) return KRED_ERR_INVALID_ARG;
  return KRED_OK;
}

kred_status kred_gauss_backward_ranges(kred_ctx* ctx, const kred_params* p, int64_t M, int64_t N,
                                       int32_t D, int32_t E, const float* x, const float* y,
                                       const float* b, const float* e, float* gx, float* gy,
                                       float* gb, int32_t nr, const int32_t* row_ranges,
                                       const int32_t* col_ptr, const int32_t* col_ranges,
                                       int32_t nc, const int32_t* col_clusters,
                                       const int32_t* row_ptr, const int32_t* row_ranges_t,
                                       void* stream) {
  if (ctx == nullptr) return KRED_ERR_INVALID_ARG;
  const kred_status v = kred_validate_backward_ranges(
      p, M, N, D, E, x, y, b, e, gx, gy, gb, nr, row_ranges, col_ptr, col_ranges, nc,
      col_clusters, row_ptr, row_ranges_t);
  if (v != KRED_OK) return v;
  hipStream_t s = static_cast<hipStream_t>(stream);
  DeviceGuard devg(ctx->device);
  if (!devg.ok) return KRED_ERR_HIP;
  kred_status st = KRED_OK;
  const Ranges fwd{nr, row_ranges, col_ptr, col_ranges};
  const Ranges tr{nc, col_clusters, row_ptr, row_ranges_t};
  // dL/dx_i over row i's cluster columns
  if (gx && M > 0) {
    st = (N == 0 || nr == 0) ? (launch_fill(gx, M * D, 0.0f, s) == hipSuccess ? KRED_OK : KRED_ERR_HIP)
                             : run_vjp(ctx, p, M, N, D, E, x, y, b, e, gx, s, &fwd);
    if (st != KRED_OK) return st;
  }
  // dL/dy_j over the rows of column j's cluster, roles of (x, e) and (y, b) exchanged
  if (gy && N > 0) {
    st = (M == 0 || nc == 0) ? (launch_fill(gy, N * D, 0.0f, s) == hipSuccess ? KRED_OK : KRED_ERR_HIP)
                             : run_vjp(ctx, p, N, M, D, E, y, x, e, b, gy, s, &tr);
    if (st != KRED_OK) return st;
  }
  // dL/db_j = sum over the same rows of k_ij e_i
  if (gb && N > 0) {
    if (launch_fill(gb, N * E, 0.0f, s) != hipSuccess) return KRED_ERR_HIP;
    if (M > 0 && nc > 0) {
      st = run_reduction(ctx, KRED_F_GAUSS, KRED_R_SUM, p, N, M, D, E, y, x, e, gb, s, &tr);
      if (st != KRED_OK) return st;
    }
  }
  return KRED_OK;
}

kred_status kred_profile_collect(kred_ctx* ctx, int32_t* count, double* total_ms,
                                 const char** kernel) {
  if (ctx == nullptr || count == nullptr || total_ms == nullptr) return KRED_ERR_INVALID_ARG;
  DeviceGuard guard(ctx->device);
  double sum = 0.0;
  for (size_t i = 0; i + 1 < ctx->ev_used; i += 2) {
    if (hipEventSynchronize(ctx->ev[i + 1]) != hipSuccess) return KRED_ERR_HIP;
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, ctx->ev[i], ctx->ev[i + 1]) != hipSuccess) return KRED_ERR_HIP;
    sum += ms;
  }
  *count = (int32_t)(ctx->ev_used / 2);
  *total_ms = sum;
  if (ctx->last_exact_D > 0 && ctx->exact_guard != nullptr) {
    // which arg-K-min kernel the device chose in the last profiled call
    ExactGuard h{};
    if (hipMemcpy(&h, ctx->exact_guard, sizeof(h), hipMemcpyDeviceToHost) != hipSuccess)
      return KRED_ERR_HIP;
    const float m = __builtin_bit_cast(float, h.maxabs);
    const bool ok = h.nonint == 0u && m <= kExactMaxAbs &&
                    (float)ctx->last_exact_D * m * m <= kExactMaxSum;
    ctx->last_kernel = ok ? "knn_bf16_kernel" : "mfma_kernel";
  }
  if (ctx->last_fast && ctx->fast_counts != nullptr) {
    // small-D calls since the last collect: the matrix-core kernel in all of
    // them, in none (the direct form), or in some
    int h[2] = {0, 0};
    if (hipMemcpy(h, ctx->fast_counts, sizeof(h), hipMemcpyDeviceToHost) != hipSuccess ||
        hipMemset(ctx->fast_counts, 0, sizeof(h)) != hipSuccess)
      return KRED_ERR_HIP;
    ctx->last_kernel = h[0] == h[1] ? ctx->choice_yes : h[0] == 0 ? ctx->last_direct
                       : (ctx->choice_yes[0] == 'f' ? "fast_kernel+direct" : "mfma_f64_kernel+fp32");
    ctx->last_fast = false;
  }
  if (kernel) *kernel = ctx->last_kernel;
  ctx->ev_used = 0;
  return KRED_OK;
}

}  // extern "C"
