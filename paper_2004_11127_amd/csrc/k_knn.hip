// Exact arg-K-min on the bf16 matrix cores (Sec. 2 reductions: the K
// nearest columns of every row under the squared distance), for data the
// guard in k_mfma.hip has shown to be exact there: integer coordinates with
// |v| <= 256 and D max|v|^2 <= 2^22, so every product and partial sum below is
// an exact integer in fp32.
//
// This file is compiled with IEEE mode off (-fno-honor-nans
// -mno-amdgpu-ieee): its values are integers and +-infinity, never NaN, and
// without IEEE mode the fp64 minimum and maximum take their operands as they
// are, without a quieting step in front of each.
#include "k_mfma_kernel.h"

#include <climits>

namespace kred {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// T[j][i] = ny_j + sum_d (-2 y_jd) x_id with one v_mfma_f32_16x16x32_bf16 per
// 32 coordinates of a 16 x 16 block.  bf16 16x16x32 operand layout (lane
// l = 16 g + li): A (16 x 32): lane l supplies A[li][8 g .. 8 g + 7]; B
// (32 x 16): lane l supplies B[8 g .. 8 g + 7][li]; D: lane l holds
// D[4 g + r][li].  With A = Y rows and B = X rows, lane l sees columns
// j = 4 g + r of row i = li: the sixteen columns of a block lie in the row's
// four lanes g = 0..3.
//
// One list per row, spread over those four lanes.  Keys are d 2^28 + j in
// fp64 (d = T, an integer with |d| < 2^24, so the key is exact and orders as
// (d, j)).  The row holds 4P slots, P = ceil(KP / 4) per lane, each lane's P
// ascending; 4P - KP of them are fixed at -infinity, so the KP others are the
// row's K nearest so far and their largest key (the maximum over the four
// lanes' last slots) is the row's current bound.  Slots not yet filled hold
// distinct keys above every real one.  Every lane of the row keeps the
// distance part of the bound as its filter: a column passes when its T is at
// or below it (a tie may still win on its index).  A block with a passing
// column anywhere in a row block sends the wave through the merge, which
// repeats, for all rows at once: m = the row's smallest pending key (a
// minimum over its four lanes); if m is below the bound, the lane holding
// the bound drops it and inserts m in its own slots (key_insert), and the
// bound is taken again.  The keys decide every comparison, so each list ends
// as the exact K smallest (d, j) of the row's columns, whatever the order of
// arrival.  The partial layout is the fp32 kernel's: lane group g writes its
// slots, ascending and without the fixed ones, as list g of the row.
constexpr int knn_slots(int KP) { return (KP + 3) / 4; }
// rows per workgroup: the fp32 kernel's, so both share one grid and one
// block-sparse workgroup map
constexpr int knn_rows(int NCH, int KP) { return (NCH >= 8 || KP == 64) ? 64 : 128; }
// row blocks of 16 per wave (their x operand, two blocks of products and two
// of column operands in flight fit the registers of 2 waves per SIMD)
constexpr int knn_rb(int NCH, int KP) { return knn_slots(KP) >= 8 ? 1 : (NCH >= 8 ? 2 : 4); }
constexpr int knn_waves(int NCH, int KP) { return knn_rows(NCH, KP) / (16 * knn_rb(NCH, KP)); }
constexpr int knn_threads(int NCH, int KP) { return 64 * knn_waves(NCH, KP); }
// the lists live in LDS (fp64 keys, RB P per lane): only the merge reads them
constexpr int knn_list_bytes(int NCH, int KP) {
  return 8 * knn_rb(NCH, KP) * knn_slots(KP) * knn_threads(NCH, KP);
}
// tile width: two buffers of TJ columns, their norms and the lists in a
// workgroup's share of the LDS at 8 waves per CU (20 KB per wave), in whole
// direct loads per lane
constexpr bool knn_tile_fits(int NCH, int KP, int TJ) {
  return 4 * TJ * 32 * NCH + 8 * TJ + knn_list_bytes(NCH, KP) <= 20480 * knn_waves(NCH, KP) &&
         (TJ * 4 * NCH) % knn_threads(NCH, KP) == 0;
}
constexpr int knn_tile_cols(int NCH, int KP) {
  return knn_tile_fits(NCH, KP, 128) ? 128 : knn_tile_fits(NCH, KP, 64) ? 64
       : knn_tile_fits(NCH, KP, 32) ? 32 : 16;
}
// uint4 q of tile column cl sits at cl PU + (q ^ knn_swz(cl)).  The sixteen
// columns a wave reads at one q fall on distinct 16-byte bank groups, or two
// to a group at PU = 8; the XOR stays inside q's group of four for PU <= 8,
// so the chunks of one column keep fixed distances.  It depends on cl mod 16
// only (a block's lane li reads column 16 blk + li).
template <int PU>
__device__ __forceinline__ int knn_swz(int cl) {
  return PU == 4 ? ((cl >> 2) & 3) : PU == 8 ? ((cl >> 1) & 3) : (cl & 15);
}

// Trades among the four 16-lane groups of a wave (g = lane / 16) on the gfx950
// swap instructions: permlane16_swap(v, v) yields the values of groups
// (0, 0, 2, 2) and (1, 1, 3, 3) in groups 0..3, permlane32_swap(v, v) those
// of (0, 1, 0, 1) and (2, 3, 2, 3).  Every lane of the wave must be active.
struct DwordPair {
  unsigned int lo, hi;
};
__device__ __forceinline__ void swap16(double x, double& e, double& o) {
  const DwordPair u = __builtin_bit_cast(DwordPair, x);
  const auto a = __builtin_amdgcn_permlane16_swap(u.lo, u.lo, false, false);
  const auto b = __builtin_amdgcn_permlane16_swap(u.hi, u.hi, false, false);
  e = __builtin_bit_cast(double, DwordPair{a[0], b[0]});
  o = __builtin_bit_cast(double, DwordPair{a[1], b[1]});
}
__device__ __forceinline__ void swap32(double x, double& e, double& o) {
  const DwordPair u = __builtin_bit_cast(DwordPair, x);
  const auto a = __builtin_amdgcn_permlane32_swap(u.lo, u.lo, false, false);
  const auto b = __builtin_amdgcn_permlane32_swap(u.hi, u.hi, false, false);
  e = __builtin_bit_cast(double, DwordPair{a[0], b[0]});
  o = __builtin_bit_cast(double, DwordPair{a[1], b[1]});
}
// the minimum / maximum over the four groups, in every group
__device__ __forceinline__ double group_min(double x) {
  double e, o;
  swap16(x, e, o);
  swap32(__builtin_fmin(e, o), e, o);
  return __builtin_fmin(e, o);
}
__device__ __forceinline__ double group_max(double x) {
  double e, o;
  swap16(x, e, o);
  swap32(__builtin_fmax(e, o), e, o);
  return __builtin_fmax(e, o);
}

// keys of unfilled slots: distinct, above every real key (|key| < 2^53) and
// exact in fp64 (multiples of 2^9 above 2^60); their distance part passes
// every real column
__device__ __forceinline__ double knn_unfilled(int slot) { return 1152921504606846976.0 + 512.0 * slot; }
constexpr float kKnnOpen = 4294967296.0f;   // 2^32: the filter while slots are unfilled

template <int NCH, int KP, bool SP>
__global__ __launch_bounds__(knn_threads(NCH, KP)) __attribute__((amdgpu_waves_per_eu(2)))
void knn_bf16_kernel(MfmaArgs a) {
  if (!exact_ok(a.exact, a.D)) return;   // the fp32 kernel does the work
  constexpr int DP = 32 * NCH;
  constexpr int PU = DP / 8;                 // uint4 per column
  constexpr int RB = knn_rb(NCH, KP);
  constexpr int ROWS = knn_rows(NCH, KP);
  constexpr int WAVES = knn_waves(NCH, KP);
  constexpr int NT = 64 * WAVES;
  constexpr int TJ = knn_tile_cols(NCH, KP);
  constexpr int TU = TJ * PU;                // uint4 of y per tile
  constexpr int YI = TU / NT;                // direct loads per lane and tile
  static_assert(WAVES * 16 * RB == ROWS && TU % NT == 0 && YI >= 1, "whole direct loads");
  constexpr int P = knn_slots(KP);
  constexpr int NFIX = 4 * P - KP;           // slots fixed at -infinity: the first ones in lane order

  // two tile buffers as distinct arrays: the direct loads into one are then
  // known not to touch the other, and reading the current tile waits for none
  __shared__ uint4 ys0[TU], ys1[TU];
  __shared__ float4 ns0[TJ / 4], ns1[TJ / 4];
  // slot p of row block rb of thread tid: kls[rb P + p][tid]
  __shared__ double kls[RB * P][NT];

  const MItem it = mitem<SP>(a, ROWS);
  if (!it.live) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int li = lane & 15, g = lane >> 4;
  const int c = it.c;
  const int64_t rend = it.row_end;
  const float pad_ny = a.pad_ny;
  const int64_t i0 = it.row0 + wave * (16 * RB);

  bf16x8 xb[RB][NCH];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int64_t row = i0 + 16 * rb + li;
    const bool ok = row < rend;
    const float* xr = a.x + (ok ? row : rend - 1) * a.D;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int d = 32 * ch + 8 * g + t;
        const float keep = (ok && d < a.D) ? 1.0f : 0.0f;   // the data are finite
        xb[rb][ch][t] = (__bf16)(xr[d < a.D ? d : a.D - 1] * keep);
      }
  }

  // per row block the lane's P slots of its row (in LDS) and the distance
  // part of the row's bound (the filter)
  float thr[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    thr[rb] = kKnnOpen;
#pragma unroll
    for (int p = 0; p < P; ++p)
      kls[rb * P + p][tid] = g * P + p < NFIX ? -__builtin_inf() : knn_unfilled(g * P + p);
  }

  // the lane's uint4 of chunk 4 ch + g in a block's column li (for PU <= 8
  // the chunks of a column keep their distances: one base, fixed offsets)
  int loff[NCH];
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch)
    loff[ch] = PU <= 8 ? li * PU + (g ^ knn_swz<PU>(li)) + 4 * ch
                       : li * PU + ((4 * ch + g) ^ knn_swz<PU>(li));

  float4 nstage;   // block-sparse: the masked norms of the next tile
  // the tile at column jt (16-aligned) into (yd, nd), its columns outside
  // [lo, hi) masked: y straight into LDS (global_load_lds_dwordx4: lane l of a
  // wave writes 16 B at the window's base + 16 l, so each lane loads the uint4
  // that belongs at its position), and the norms too when dense; the masked
  // norms of a block-sparse tile go through registers (put)
  auto fetch = [&](uint4 (&yd)[TU], float4 (&nd)[TJ / 4], int64_t jt, int64_t lo, int64_t hi) {
    // y of masked columns is loaded as is (inside the padded array): their
    // padding norm (+infinity) keeps them out of every list; columns past the
    // loaded blocks keep stale values, never used
    const int ncol = (int)min((int64_t)TJ, ((hi + 15) & ~(int64_t)15) - jt);
    const uint4* ysrc = reinterpret_cast<const uint4*>(a.ybf + jt * DP);
#pragma unroll
    for (int k = 0; k < YI; ++k) {
      const int s0 = 64 * (WAVES * k + wave);   // the wave's window of the tile
      // window position s0 + lane holds uint4 q ^ knn_swz(cc) of column cc;
      // for PU <= 8 the swizzle of the window's columns is g, so that is
      // uint4 s0 + (lane ^ g) of the tile
      const int cc = (s0 + lane) / PU;
      const int src = PU <= 8 ? s0 + (lane ^ g)
                              : cc * PU + (((s0 + lane) % PU) ^ knn_swz<PU>(cc));
      if (cc < ncol)
        __builtin_amdgcn_global_load_lds(static_cast<const void*>(ysrc + src),
                                         (__attribute__((address_space(3))) void*)(&yd[s0]),
                                         16, 0, 0);
    }
    if (tid < TJ / 4) {
      if constexpr (SP) {
        nstage = masked_ny(a.ny, pad_ny, jt + 4 * tid, lo, hi);
      } else if (tid * 4 < ncol) {
        __builtin_amdgcn_global_load_lds(
            static_cast<const void*>(reinterpret_cast<const float4*>(a.ny + jt) + tid),
            (__attribute__((address_space(3))) void*)(&nd[0]), 16, 0, 0);
      }
    }
  };
  auto put = [&](float4 (&nd)[TJ / 4]) {
    if constexpr (SP)
      if (tid < TJ / 4) nd[tid] = nstage;
  };

  // merges the passing columns of one row block's block (all lanes active)
  // merges the passing columns of row block rb's block (all lanes active);
  // the lane's slots come from LDS and go back there
  auto merge = [&](int rb, float& tr, const f4& v, const double (&jd)[4])
                   __attribute__((always_inline)) {
    double kr[P];
#pragma unroll
    for (int p = 0; p < P; ++p) kr[p] = kls[rb * P + p][tid];
    double cand[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) cand[r] = __builtin_fma((double)v[r], kKeyScale, jd[r]);
    double bd = group_max(kr[P - 1]);
    for (;;) {
      const double mine = __builtin_fmin(__builtin_fmin(cand[0], cand[1]),
                                         __builtin_fmin(cand[2], cand[3]));
      if (__builtin_amdgcn_ballot_w64(mine < bd) == 0) break;
      const double m = group_min(mine);
      if (m < bd && kr[P - 1] == bd) key_insert<P>(kr, m);
#pragma unroll
      for (int r = 0; r < 4; ++r) cand[r] = cand[r] == m ? __builtin_inf() : cand[r];
      bd = group_max(kr[P - 1]);
    }
#pragma unroll
    for (int p = 0; p < P; ++p) kls[rb * P + p][tid] = kr[p];
    tr = key_d(bd);
  };

  // one tile from (yc, nc), the next one's loads into (yn, nn) when `more`
  auto tile = [&](const uint4 (&yc)[TU], const float4 (&nc)[TJ / 4], uint4 (&yn)[TU],
                  float4 (&nn)[TJ / 4], int64_t jt, bool more, int64_t a0, int64_t a1)
                  __attribute__((always_inline)) {
    const int nblk = (int)((min((int64_t)TJ, a1 - jt) + 15) / 16);
    // yn was last read by the tile before this one, which ended with a barrier
    if (more) fetch(yn, nn, jt + TJ, a0, a1);
    // the tile's blocks unrolled into a pipeline: the operands of block b + 2
    // are read from LDS and the products of block b + 1 formed while block b
    // is filtered, so one wave's stream alternates matrix-core and vector
    // work.  Blocks past the tile's end (a partial tile) compute on stale LDS
    // and are never filtered.
    constexpr int NB = TJ / 16;
    bf16x8 ya[NB][NCH];
    float4 nyv[NB];
    f4 acc[NB][RB];
    auto read = [&](int b) __attribute__((always_inline)) {
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch)
        ya[b][ch] = __builtin_bit_cast(bf16x8, yc[b * 16 * PU + loff[ch]]);
      nyv[b] = nc[b * 4 + g];
    };
    auto products = [&](int b) __attribute__((always_inline)) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) acc[b][rb] = f4{nyv[b].x, nyv[b].y, nyv[b].z, nyv[b].w};
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          acc[b][rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ya[b][ch], xb[rb][ch], acc[b][rb], 0, 0, 0);
    };
    read(0);
    if (NB > 1) read(1);
    products(0);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (b + 2 < NB) read(b + 2);
      if (b + 1 < NB) products(b + 1);
      bool hit[RB];
      bool any = false;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const float lo = __builtin_elementwise_minimum(
            __builtin_elementwise_minimum(acc[b][rb][0], acc[b][rb][1]),
            __builtin_elementwise_minimum(acc[b][rb][2], acc[b][rb][3]));
        hit[rb] = lo <= thr[rb];
        any = any || hit[rb];
      }
      if (__builtin_expect(__builtin_amdgcn_ballot_w64(any && b < nblk) != 0, 0)) {
        const int jb = (int)(jt + b * 16 + 4 * g);
        double jd[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) jd[r] = (double)(jb + r);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          if (__builtin_amdgcn_ballot_w64(hit[rb]) != 0) merge(rb, thr[rb], acc[b][rb], jd);
      }
    }
    if (more) put(nn);
    __builtin_amdgcn_s_waitcnt(0);   // this wave's direct loads have landed
    __syncthreads();
  };

  auto segment = [&](int64_t a0, int64_t a1) {
    const int64_t base = a0 & ~(int64_t)15;
    const int64_t ntiles = (a1 - base + TJ - 1) / TJ;
    // the previous segment's last tile was read before its final barrier
    fetch(ys0, ns0, base, a0, a1);
    put(ns0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    for (int64_t t = 0; t < ntiles; t += 2) {
      tile(ys0, ns0, ys1, ns1, base + t * TJ, t + 1 < ntiles, a0, a1);
      if (t + 1 < ntiles) tile(ys1, ns1, ys0, ns0, base + (t + 1) * TJ, t + 2 < ntiles, a0, a1);
    }
  };
  if constexpr (SP) for_segments(a, it, segment);
  else if (it.w0 < it.w1) segment(it.w0, it.w1);

#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    // the row norm (exact: integers below 2^24), from x again rather than
    // kept in registers through the loop
    const int64_t row = i0 + 16 * rb + li;
    const bool ok = row < rend;
    float part = 0.0f;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int d = 32 * ch + 8 * g + t;
        const float v = (ok && d < a.D) ? a.x[row * a.D + d] : 0.0f;
        part = __builtin_fmaf(v, v, part);
      }
    part += __shfl_xor(part, 16);
    part += __shfl_xor(part, 32);
    if (!ok) continue;
    float* q = a.part + (((int64_t)c * 4 + g) * a.M + row) * (2 * KP);
    // the lane's slots past its fixed ones, then empty entries
#pragma unroll
    for (int gg = 0; gg < 4; ++gg) {
      if (g != gg) continue;
      const int nfix = gg * P >= NFIX ? 0 : (NFIX - gg * P < P ? NFIX - gg * P : P);
#pragma unroll
      for (int p = 0; p < KP; ++p) {
        const double key = p + nfix < P ? kls[rb * P + (p + nfix < P ? p + nfix : 0)][tid]
                                        : __builtin_inf();
        const bool empty = !(key < 1152921504606846976.0);   // unfilled, or past the slots
        const double d = __builtin_floor(key * kKeyInv);
        q[2 * p] = empty ? __builtin_inff() : (float)d + part;
        q[2 * p + 1] = __int_as_float(empty ? INT_MAX : (int)(key - d * kKeyScale));
      }
    }
  }
}

template <int NCH, bool SP>
hipError_t launch_knn_bf16_n(const MfmaArgs& a, dim3 grid, hipStream_t s) {
  switch (a.KP) {
#define KRED_KNN_BF16(KPV)                                                                     \
  case KPV:                                                                                     \
    hipLaunchKernelGGL((knn_bf16_kernel<NCH, KPV, SP>), grid, dim3(knn_threads(NCH, KPV)), 0, \
                       s, a);                                                                   \
    break;
    KRED_KNN_BF16(1) KRED_KNN_BF16(4) KRED_KNN_BF16(8) KRED_KNN_BF16(10) KRED_KNN_BF16(12)
    KRED_KNN_BF16(16) KRED_KNN_BF16(64)
#undef KRED_KNN_BF16
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_knn_bf16(const MfmaArgs& a, hipStream_t s) {
  const int rows = mfma_rows_per_block(a.DP, a.KP);
  if (rows != knn_rows(a.DP / 32, a.KP)) return hipErrorInvalidValue;   // one grid for both kernels
  const dim3 grid((unsigned)(mfma_row_groups(a, rows) * a.C));
  switch (a.DP) {
    case 32: return a.nr > 0 ? launch_knn_bf16_n<1, true>(a, grid, s) : launch_knn_bf16_n<1, false>(a, grid, s);
    case 64: return a.nr > 0 ? launch_knn_bf16_n<2, true>(a, grid, s) : launch_knn_bf16_n<2, false>(a, grid, s);
    case 128: return a.nr > 0 ? launch_knn_bf16_n<4, true>(a, grid, s) : launch_knn_bf16_n<4, false>(a, grid, s);
    case 256: return a.nr > 0 ? launch_knn_bf16_n<8, true>(a, grid, s) : launch_knn_bf16_n<8, false>(a, grid, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace kred
