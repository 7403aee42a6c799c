// Large-D (16 < D <= 256) prologue, the exactness guard of the bf16 arg-K-min
// kernel (the kernel is in k_knn.hip), the split-bf16 sum kernel, the centre
// and the large-D gradient kernels, and the launchers of the fp32 matrix-core
// kernel (its template is in k_mfma_kernel.h).
#include "k_mfma_kernel.h"

#include <climits>

namespace kred {
namespace {


// v = h + m + l exactly, each part a bf16 (round to nearest): h keeps the top
// 8 significant bits, the remainder v - h is exact in fp32 with at most 16,
// m keeps 8 of those and l the last 8.
__device__ __forceinline__ void split3(float v, __bf16& h, __bf16& m, __bf16& l) {
  h = (__bf16)v;
  const float r = v - (float)h;
  m = (__bf16)r;
  l = (__bf16)(r - (float)m);
}

// ------------------------------------------------------------------ prologue
// Coalesced: consecutive threads handle consecutive d of one column.
__global__ __launch_bounds__(256) void mfma_pack_kernel(MfmaPackArgs a) {
  const bool ex = exact_ok(a.exact, a.D);   // arg-K-min on the exact bf16 path
  const bool w64 = wide64(a.spread, a.wide_c, a.wide_limit);   // the fp64 contraction
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t total = a.N16 * a.DP;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total; t += stride) {
    const int64_t j = t / a.DP;
    const int d = (int)(t - j * a.DP);
    if (w64) {
      // in fp64: y - m exact, one rounding of the product
      const double v = (j < a.N && d < a.D)
                           ? (double)a.y[j * a.D + d] - (double)(a.yc != nullptr ? a.yc[d] : 0.0f)
                           : 0.0;
      reinterpret_cast<double*>(a.yop)[t] = v * a.yop_scale64;
      continue;
    }
    const float v =
        (j < a.N && d < a.D) ? a.y[j * a.D + d] - (a.yc != nullptr ? a.yc[d] : 0.0f) : 0.0f;
    // the centred forms (those with a guard): 2 Y = fl32(2 s (y - m)) formed in
    // fp64, one rounding (2 Y: the column norms use Y = fl32(s (y - m)))
    const float w = a.spread == nullptr ? v * a.yop_scale
                  : (j < a.N && d < a.D)
                      ? (float)(((double)a.y[j * a.D + d] - (double)(a.yc != nullptr ? a.yc[d] : 0.0f)) *
                                a.yop_scale64)
                      : 0.0f;
    if (ex) {
      a.ybf[t] = __builtin_bit_cast(unsigned short, (__bf16)(v * a.yop_scale));
    } else if (a.ysp != nullptr) {
      __bf16 h, m, l;
      split3(w, h, m, l);
      unsigned short* q = a.ysp + j * 3 * a.DP + d;   // planes h, m, l of column j
      q[0] = __builtin_bit_cast(unsigned short, h);
      q[a.DP] = __builtin_bit_cast(unsigned short, m);
      q[2 * a.DP] = __builtin_bit_cast(unsigned short, l);
    } else {
      a.yop[t] = w;
    }
  }
  // Laplacian log-sum-exp: g' = g log2(e) per column, -infinity for padding
  if (a.gpk != nullptr) {
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < a.N16; j += stride)
      a.gpk[j] = j < a.N ? a.goff[j] * a.goff_scale : -__builtin_inff();
  }
  if (a.bpk != nullptr && a.bpair && !w64) {
    // bf16 planes h, m, l of b per 32-column pair: plane p, signal column e
    // and K index k at pair 96 W + p 32 W + e 32 + k, where k = 8 g + 4 h + r
    // holds column 16 h + 4 g + r of the pair (the P . B operand's K order)
    const int W = 16 * a.EB;
    const int64_t total_b = (a.N + 31) / 32 * 32 * W;
    unsigned short* bp = reinterpret_cast<unsigned short*>(a.bpk);
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total_b; t += stride) {
      const int k = (int)(t & 31);
      const int64_t pe = t >> 5;          // pair W + e
      const int64_t pair = pe / W;
      const int e = (int)(pe - pair * W);
      const int64_t j = pair * 32 + 16 * ((k >> 2) & 1) + 4 * (k >> 3) + (k & 3);
      const float v = (j < a.N && e < a.Ec) ? (a.unit_b ? 1.0f : a.b[j * a.E + a.e0 + e]) : 0.0f;
      __bf16 h, m, l;
      split3(v, h, m, l);
      const int64_t o = pair * 96 * W + (int64_t)e * 32 + k;
      bp[o] = __builtin_bit_cast(unsigned short, h);
      bp[o + 32 * W] = __builtin_bit_cast(unsigned short, m);
      bp[o + 64 * W] = __builtin_bit_cast(unsigned short, l);
    }
  } else if (a.bpk != nullptr) {
    // signal tiles: b[j][e0 + e] stored at (j/16)*16W + ((j%16)/4)*4W + e*4 + j%4, W = 16*EB
    // (unit_b: ones in place of b)
    const int W = 16 * a.EB;
    const int64_t total_b = a.N16 * W;
    for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total_b; t += stride) {
      const int64_t j = t / W;
      const int e = (int)(t - j * W);
      const float v = (j < a.N && e < a.Ec) ? (a.unit_b ? 1.0f : a.b[j * a.E + a.e0 + e]) : 0.0f;
      const int64_t blk = j / 16;
      const int jr = (int)(j % 16);
      a.bpk[blk * 16 * W + (jr / 4) * 4 * W + e * 4 + (jr % 4)] = v;
    }
  }
}

// Column norms: one wave per column at a time, lanes stride over d (coalesced),
// reduced across the wave: the squares of the represented coordinates summed in
// fp64 and rounded once (centred forms), or an fp32 sum (arg-K-min).
__global__ __launch_bounds__(256) void mfma_norm_kernel(MfmaPackArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int64_t waves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  if (wide64(a.spread, a.wide_c, a.wide_limit)) {
    // the fp64 contraction: the norms (with g') in fp64
    double* ny64 = reinterpret_cast<double*>(a.ny);
    for (int64_t j = wave; j < a.N16; j += waves) {
      double s = 0.0;
      if (j < a.N)
        for (int d = lane; d < a.D; d += 64) {
          const double v = ((double)a.y[j * a.D + d] - (double)(a.yc != nullptr ? a.yc[d] : 0.0f)) *
                           a.coord_scale64;
          s = __builtin_fma(v, v, s);
        }
      for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
      if (lane == 0)
        ny64[j] = j < a.N ? (double)a.nrm_sign * s + ((a.goff != nullptr && a.gpk == nullptr)
                                                          ? (double)a.goff[j] * (double)a.goff_scale : 0.0)
                          : (double)a.pad_norm;
    }
    return;
  }
  if (a.spread != nullptr) {
    // the centred forms: ny = fl32(-|Y|^2 (+ g')) with Y = fl32(s (y - m)) the
    // coordinates the contraction uses, the sum in fp64 and one rounding; the
    // split kernel also reads 16 padding norms after the N16 columns (the
    // source of its masked columns' norms; the buffer is sized for fp64)
    const int64_t nend = a.N16 + (a.ysp != nullptr ? 16 : 0);
    for (int64_t j = wave; j < nend; j += waves) {
      double s = 0.0;
      if (j < a.N)
        for (int d = lane; d < a.D; d += 64) {
          const double v = (double)(float)(((double)a.y[j * a.D + d] -
                                             (double)(a.yc != nullptr ? a.yc[d] : 0.0f)) *
                                            a.coord_scale64);
          s = __builtin_fma(v, v, s);
        }
      for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
      if (lane == 0)
        a.ny[j] = j < a.N ? (float)((double)a.nrm_sign * s +
                                    ((a.goff != nullptr && a.gpk == nullptr)
                                         ? (double)a.goff[j] * (double)a.goff_scale : 0.0))
                          : a.pad_norm;
    }
    return;
  }
  for (int64_t j = wave; j < a.N16; j += waves) {
    float s = 0.0f;
    if (j < a.N)
      for (int d = lane; d < a.D; d += 64) {
        const float v = (a.y[j * a.D + d] - (a.yc != nullptr ? a.yc[d] : 0.0f)) * a.coord_scale;
        s = __builtin_fmaf(v, v, s);
      }
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    if (lane == 0)
      a.ny[j] = j < a.N ? a.nrm_sign * s + ((a.goff != nullptr && a.gpk == nullptr)
                                                ? a.goff[j] * a.goff_scale : 0.0f)
                        : a.pad_norm;
  }
}




// ------------------------------------------------------- exact bf16 arg-K-min
// Guard: the largest |v| and whether every v is an integer, over x and y.
__global__ void exact_init_kernel(ExactGuard* g) {
  if (threadIdx.x == 0) {
    g->maxabs = 0u;
    g->nonint = 0u;
  }
}

__global__ __launch_bounds__(256) void exact_check_kernel(const float* __restrict__ x, int64_t nx,
                                                          const float* __restrict__ y, int64_t ny,
                                                          ExactGuard* g) {
  unsigned int m = 0u, bad = 0u;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < nx + ny; t += stride) {
    const float v = t < nx ? x[t] : y[t - nx];
    m = max(m, __float_as_uint(fabsf(v)));   // NaN and inf exceed every limit
    bad |= (v != rintf(v)) ? 1u : 0u;        // true for NaN
  }
  for (int o = 32; o > 0; o >>= 1) {
    m = max(m, (unsigned int)__shfl_xor((int)m, o));
    bad |= (unsigned int)__shfl_xor((int)bad, o);
  }
  if ((threadIdx.x & 63) == 0) {
    if (m != 0u) atomicMax(&g->maxabs, m);
    if (bad != 0u) atomicOr(&g->nonint, 1u);
  }
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));

// ------------------------------------------------ sums, split bf16 products
// The Gaussian sum of mfma_kernel with the inner product on the bf16 matrix
// cores: every coordinate is split exactly into three bf16 parts (v = h + m +
// l, 24 significant bits), and per 32 coordinates six v_mfma_f32_16x16x32_bf16
// accumulate the partial products hh, hm, mh, hl, lh and mm, each exact in
// fp32.  The dropped ml, lm and ll terms are below 2^-24 |x||y|, so the result
// carries fp32 accuracy at six bf16 products per coordinate instead of one fp32
// product (a sixth of the matrix-core time per flop for the fp32 form, at 16x
// the rate).  Column operand: three bf16 planes per column (prologue); row
// operand: the planes of x in registers.
//
// With 32-column tiles or wider (DP <= 128) the P . B product runs on the bf16
// matrix cores too, two 16-column blocks at a time: the lane's four p values
// of each block (P[i = li][j = 4 g + r], the exponent's own D layout) are the 8
// K values k = 8 g + 4 h + r of one v_mfma_f32_16x16x32_bf16, split into three
// bf16 parts like the coordinates, and the signal is stored by the prologue as
// three bf16 planes in the matching K order (mfma_pack_kernel), so six products
// per 32 columns replace eight v_mfma_f32_16x16x4_f32 (48 matrix-core cycles
// per 16 columns instead of 128).  Wider D keeps the fp32 P . B.
// DP = 32, 64 and 128 take mfma_split_kernel below (32 x 32 tiles); this
// kernel serves DP = 256.
constexpr int split_tile_cols(int DP) { return DP <= 64 ? 64 : (DP <= 128 ? 32 : 16); }

template <int NCH, int RB, int EB, bool SP>
__global__ __launch_bounds__(256) void mfma_split16_kernel(MfmaArgs a) {
  constexpr int DP = 32 * NCH;
  constexpr int TJ = split_tile_cols(DP);
  constexpr bool PAIR = TJ % 32 == 0;          // P . B on the bf16 matrix cores
  constexpr int PU = DP / 8;                  // uint4 per plane of a column
  constexpr int TU = TJ * 3 * PU;             // uint4 of y planes per tile
  static_assert(TU % 256 == 0, "whole direct loads per tile");
  constexpr int YI = TU / 256;                // direct loads per wave and tile
  constexpr int W = 16 * EB;
  // signal: fp32 float4s (16-column tiles), or bf16 planes of 32-column pairs,
  // 3 W rows of 32 values (four uint4) per pair, 5 uint4 per row in LDS
  constexpr int BF4 = PAIR ? TJ / 32 * 12 * W : TJ * W / 4;
  constexpr int BL = (BF4 + 255) / 256;

  // y planes as in HBM (3 PU uint4 per column), uint4 q of column c at
  // position q ^ (c & (PU - 1)) within its plane: the 16 columns a wave reads
  // at once fall on distinct bank groups
  __shared__ uint4 ys[2][TU];
  __shared__ float4 ns[2][TJ / 4];
  __shared__ float4 bs[2][PAIR ? 1 : TJ * W / 4];
  __shared__ uint4 bq[2][PAIR ? TJ / 32 * 15 * W : 1];

  if (wide64(a.spread, a.wide_c, a.wide_limit)) return;   // the fp64 contraction does the work
  const MItem it = mitem<SP>(a, 64 * RB);
  if (!it.live) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int li = lane & 15, g = lane >> 4;
  const int c = it.c;
  const int64_t rend = it.row_end;
  const float pad_ny = a.pad_ny;
  const int64_t i0 = it.row0 + wave * (16 * RB);

  // planes of x[i = li][32 ch + 8 g + t]; X = fl32(s (x - m)) formed in fp64
  // and nx = -fl32(|X|^2) summed in fp64 (the accuracy guard's arithmetic)
  bf16x8 xh[RB][NCH], xm[RB][NCH], xl[RB][NCH];
  float nx[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int64_t row = i0 + 16 * rb + li;
    const bool ok = row < rend;
    double part = 0.0;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int d = 32 * ch + 8 * g + t;
        const float v =
            (ok && d < a.D) ? (float)(((double)a.x[row * a.D + d] -
                                       (double)(a.xc != nullptr ? a.xc[d] : 0.0f)) * a.xscale64)
                            : 0.0f;
        __bf16 h, m, l;
        split3(v, h, m, l);
        xh[rb][ch][t] = h;
        xm[rb][ch][t] = m;
        xl[rb][ch][t] = l;
        part = __builtin_fma((double)v, (double)v, part);
      }
    part += __shfl_xor(part, 16);
    part += __shfl_xor(part, 32);
    nx[rb] = -(float)part;
  }

  f4 oacc[RB][EB], tot[RB][EB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int eb = 0; eb < EB; ++eb) oacc[rb][eb] = tot[rb][eb] = f4{0.f, 0.f, 0.f, 0.f};

  float4 bstage[BL];
  float4 nstage;
  // the tile at column jt (16-aligned; 32-aligned with PAIR) into buffer
  // nbuf, its columns outside [lo, hi) masked: the y planes straight into LDS
  // (global_load_lds_dwordx4: lane l of a wave writes 16 B at the window's
  // base + 16 l; each lane loads the uint4 that belongs at its position),
  // norms and signal through registers (put)
  auto fetch = [&](int nbuf, int64_t jt, int64_t lo, int64_t hi) {
    // y of masked columns is loaded as is (inside the padded array): their
    // padding norm (-infinity) makes p exactly 0, which removes them; columns
    // past the loaded blocks keep stale values, never used
    const int ncol = (int)min((int64_t)TJ, ((hi + 15) & ~(int64_t)15) - jt);
    const uint4* ysrc = reinterpret_cast<const uint4*>(a.ysp + jt * 3 * DP);
#pragma unroll
    for (int k = 0; k < YI; ++k) {
      const int s0 = 64 * (4 * k + wave);   // the wave's window of the tile
      const int sl = s0 + lane;
      const int cc = sl / (3 * PU), qq = sl - cc * 3 * PU;
      if (cc < ncol)
        __builtin_amdgcn_global_load_lds(
            static_cast<const void*>(ysrc + cc * 3 * PU + (qq ^ (cc & (PU - 1)))),
            (__attribute__((address_space(3))) void*)(&ys[nbuf][s0]), 16, 0, 0);
    }
    if (tid < TJ / 4) {
      if constexpr (SP) nstage = masked_ny(a.ny, pad_ny, jt + 4 * tid, lo, hi);
      else nstage = (tid * 4 < ncol) ? reinterpret_cast<const float4*>(a.ny + jt)[tid]
                                     : float4{0.f, 0.f, 0.f, 0.f};
    }
    if constexpr (PAIR) {
      // whole pairs from the prologue's array (sized for 32-column pairs)
      const float4* bsrc = reinterpret_cast<const float4*>(a.bpk) + (jt / 32) * (12 * W);
#pragma unroll
      for (int k = 0; k < BL; ++k) {
        const int f = tid + k * 256;
        bstage[k] = (f < BF4 && (f / (12 * W)) * 32 < ncol) ? bsrc[f] : float4{0.f, 0.f, 0.f, 0.f};
      }
    } else {
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
    if (tid < TJ / 4) ns[buf][tid] = nstage;
#pragma unroll
    for (int k = 0; k < BL; ++k) {
      const int f = tid + k * 256;
      if (f < BF4) {
        if constexpr (PAIR) {
          // (pair q, row plane W + e, quarter kc) -> row q 3W + plane W + e of 5 uint4
          const int q = f / (12 * W), rem = f - q * 12 * W;
          bq[buf][(q * 3 * W + (rem >> 2)) * 5 + (rem & 3)] = __builtin_bit_cast(uint4, bstage[k]);
        } else {
          bs[buf][f] = bstage[k];
        }
      }
    }
  };

  // T of block blk for every row block: two chains per row block, both from
  // zero (four independent matrix-core chains per wave): acc the products hh,
  // hm and mh, acc2 the small ones, mm, hl and lh (below 2^-15 of the
  // products), so that only 3 of the 6 instructions per chunk round at the
  // scale of the sum; then T = fl(fl(acc + acc2) + fl(nx + ny))
  auto exponent = [&](int buf, int blk, f4 (&acc)[RB]) {
    const float4 nyv = ns[buf][blk * 4 + g];
    f4 acc2[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) acc[rb] = acc2[rb] = f4{0.f, 0.f, 0.f, 0.f};
    const int cl = blk * 16 + li;
    const uint4* col = &ys[buf][cl * 3 * PU];
    const int sw = cl & (PU - 1);
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      const int q = (4 * ch + g) ^ sw;
      const bf16x8 yh = __builtin_bit_cast(bf16x8, col[q]);
      const bf16x8 ym = __builtin_bit_cast(bf16x8, col[PU + q]);
      const bf16x8 yl = __builtin_bit_cast(bf16x8, col[2 * PU + q]);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        acc2[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ym, xm[rb][ch], acc2[rb], 0, 0, 0);
        acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ym, xh[rb][ch], acc[rb], 0, 0, 0);
        acc2[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(yl, xh[rb][ch], acc2[rb], 0, 0, 0);
        acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(yh, xm[rb][ch], acc[rb], 0, 0, 0);
        acc2[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(yh, xl[rb][ch], acc2[rb], 0, 0, 0);
        acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(yh, xh[rb][ch], acc[rb], 0, 0, 0);
      }
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      acc[rb] += acc2[rb];
      acc[rb] += f4{nx[rb] + nyv.x, nx[rb] + nyv.y, nx[rb] + nyv.z, nx[rb] + nyv.w};
    }
  };

  auto segment = [&](int64_t a0, int64_t a1) {
  const int64_t base = a0 & ~(int64_t)(PAIR ? 31 : 15);
  const int64_t ntiles = (a1 - base + TJ - 1) / TJ;
  // the previous segment's last tile was read before its final barrier
  fetch(0, base, a0, a1);
  put(0);
  __builtin_amdgcn_s_waitcnt(0);   // this wave's direct loads have landed
  __syncthreads();
  for (int64_t t = 0; t < ntiles; ++t) {
    const int64_t jt = base + t * TJ;
    const int buf = (int)(t & 1);
    const int nblk = (int)((min((int64_t)TJ, a1 - jt) + 15) / 16);
    // buffer (t+1)&1 was last read in iteration t-1, which ended with a barrier
    if (t + 1 < ntiles) fetch(buf ^ 1, jt + TJ, a0, a1);
    if constexpr (PAIR) {
      for (int bp = 0; bp < (nblk + 1) / 2; ++bp) {
        // A planes of the pair: K values 8 g + 4 h + r = p of block 2 bp + h,
        // column 4 g + r; a block beyond the tile's columns (odd nblk) has p = 0
        bf16x8 ph[RB], pm[RB], pl[RB];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          f4 acc[RB];
          exponent(buf, 2 * bp + h, acc);
          const bool live = 2 * bp + h < nblk;
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float pv = live ? __builtin_amdgcn_exp2f(acc[rb][r]) : 0.0f;
              __bf16 hh, mm, ll;
              split3(pv, hh, mm, ll);
              ph[rb][4 * h + r] = hh;
              pm[rb][4 * h + r] = mm;
              pl[rb][4 * h + r] = ll;
            }
        }
#pragma unroll
        for (int eb = 0; eb < EB; ++eb) {
          // B planes: b[j(k)][e = 16 eb + li] for k = 8 g .. 8 g + 7
          const uint4* brow = &bq[buf][(bp * 3 * W + 16 * eb + li) * 5 + g];
          const bf16x8 bh = __builtin_bit_cast(bf16x8, brow[0]);
          const bf16x8 bm = __builtin_bit_cast(bf16x8, brow[5 * W]);
          const bf16x8 bl = __builtin_bit_cast(bf16x8, brow[10 * W]);
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            // smallest partial products first
            f4 o = oacc[rb][eb];
            o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pm[rb], bm, o, 0, 0, 0);
            o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pl[rb], bh, o, 0, 0, 0);
            o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph[rb], bl, o, 0, 0, 0);
            o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pm[rb], bh, o, 0, 0, 0);
            o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph[rb], bm, o, 0, 0, 0);
            oacc[rb][eb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph[rb], bh, o, 0, 0, 0);
          }
        }
        // issue order: the first block's products alone, then the second's
        // with the first block's exponentials and splits between them (the
        // VALU work of one block hidden under the other's matrix-core work;
        // 3-6% on the D = 128 sums)
        for (int q = 0; q < 6 * NCH * RB; ++q) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        for (int q = 0; q < 6 * NCH * RB; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
        }
      }
    } else {
      for (int blk = 0; blk < nblk; ++blk) {
        f4 acc[RB];
        exponent(buf, blk, acc);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          f4 p;
#pragma unroll
          for (int r = 0; r < 4; ++r) p[r] = __builtin_amdgcn_exp2f(acc[rb][r]);
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
        }
      }
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int eb = 0; eb < EB; ++eb) {
        tot[rb][eb] += oacc[rb][eb];
        oacc[rb][eb] = f4{0.f, 0.f, 0.f, 0.f};
      }
    if (t + 1 < ntiles) put(buf ^ 1);
    __builtin_amdgcn_s_waitcnt(0);   // this wave's direct loads have landed
    __syncthreads();
  }
  };
  if constexpr (SP) for_segments(a, it, segment);
  else if (it.w0 < it.w1) segment(it.w0, it.w1);

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
}

template <int NCH, bool SP>
hipError_t launch_split_n(const MfmaArgs& a, dim3 grid, hipStream_t s) {
  constexpr int RB = NCH >= 8 ? 1 : 2;   // the row count of the fp32 kernel's grid
  // the Gaussian sum only: the Laplacian and squared-distance sums always take
  // the fp64 contraction, launched beside this one
  if (a.epi != 0) return hipSuccess;
  switch (a.EB) {
    case 1: hipLaunchKernelGGL((mfma_split16_kernel<NCH, RB, 1, SP>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((mfma_split16_kernel<NCH, RB, 2, SP>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((mfma_split16_kernel<NCH, RB, 4, SP>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// ---------------------- sums and log-sum-exp, split bf16 products, 32x32 tiles
// The same split sum for DP = 32, 64 and 128 (and the Gaussian / Sinkhorn
// log-sum-exp, EPI 4: a running maximum and rescaled sum per lane instead of
// P . B) with the exponent on v_mfma_f32_32x32x16_bf16: one wave owns 32 rows, and each 32-column tile is
// one 32 x 32 block of T, six instructions per 16 coordinates (hh, hm, mh into
// one chain, mm, hl, lh into the other, both from zero).  The instruction adds
// its products in groups of 8 exactly as the 16x16x32 form does (in-bounds
// probes: one group's 2^24 + 1 + 1 is exact, two groups give 2^24, the same
// roundings of 1 +- 2^-24 (1 + 2^-7)), so the split form's error bound is
// unchanged; its matrix-core rate is the higher one (two chains per wave come
// near the dense bf16 peak where the 16x16x32 form needs many more).
// Lane l = 32 h + i supplies column i of the tile's y and row i of x, each at
// coordinates 16 ch + 8 h .. + 7, and holds T[i][j] for the 16 columns
// j = 8 q + 4 h + r (q, r < 4).  P . B stays on v_mfma_f32_16x16x32_bf16 (E is
// 16 per block, a 32-wide B would be half empty): the lane's p values of
// q = 0, 2 (U) and q = 1, 3 (V) pass through one permlane32 and one permlane16
// swap, which leaves in every lane group g of 16 lanes the 8 K values
// k = 8 g + t (column 16 (t / 4) + 4 g + t % 4, the prologue's b order) of
// rows 0-15 (first register) and rows 16-31 (second).
// Workgroups of 8 waves (256 rows, two waves per SIMD) halve the y traffic
// per row against 4-wave ones; the log-sum-exp at DP = 64 (158 VGPRs) runs
// 4-wave workgroups, three waves per SIMD, instead, and so does DP = 32
// (a tile there is six wave loads).  Every part of a tile
// (y planes, norms, b planes) goes from memory straight into LDS, two tiles
// ahead, into four sets of buffers
// that are distinct arrays indexed statically (the loop is unrolled by 4):
// the compiler then sees that no read aliases an outstanding direct load and
// waits for none; the waits are explicit (the newest tile's loads stay in
// flight) and the barrier orders LDS only.  With 16 signal columns the
// exponent's products of tile t are issued together with the vector work of
// tile t - 1 (norms, 2^T, swaps, splits) and its P . B, so that neither unit
// waits for the other inside a wave.

// v0, v1 -> packed bf16 pairs h, m, l with v = h + m + l exactly (each part
// rounded to nearest; the remainders are exact in fp32)
__device__ __forceinline__ void split3x2(float v0, float v1, unsigned& h, unsigned& m, unsigned& l) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  typedef float f2 __attribute__((ext_vector_type(2)));
  h = __builtin_bit_cast(unsigned, __builtin_convertvector((f2{v0, v1}), bf16x2));
  const float r0 = v0 - __builtin_bit_cast(float, h << 16);
  const float r1 = v1 - __builtin_bit_cast(float, h & 0xffff0000u);
  m = __builtin_bit_cast(unsigned, __builtin_convertvector((f2{r0, r1}), bf16x2));
  const float s0 = r0 - __builtin_bit_cast(float, m << 16);
  const float s1 = r1 - __builtin_bit_cast(float, m & 0xffff0000u);
  l = __builtin_bit_cast(unsigned, __builtin_convertvector((f2{s0, s1}), bf16x2));
}

// the fewest direct loads one of nwv waves makes per tile: y windows
// round-robin, b windows round-robin, and the norms by the last wave
constexpr int split32_min_loads(int yw, int bo, int nwv) {
  int best = 1 << 30;
  for (int w = 0; w < nwv; ++w) {
    int n = 0;
    for (int o = w; o < yw; o += nwv) ++n;
    for (int o = w; o < bo; o += nwv) ++n;
    if (w == nwv - 1) ++n;
    best = n < best ? n : best;
  }
  return best;
}

template <int NC, int EB, int EPI, int NWV, bool SP, bool XC = false>
__global__ __launch_bounds__(64 * NWV) __attribute__((amdgpu_waves_per_eu(NWV == 4 ? 3 : 2, NWV == 4 ? 3 : 2)))
void mfma_split_kernel(MfmaArgs a) {
  // NWV waves per workgroup, 32 rows each
  constexpr int DP = 16 * NC;
  constexpr int TJ = 32;
  constexpr int PU = DP / 8;                  // uint4 per plane of a column
  constexpr int TU = TJ * 3 * PU;             // uint4 of y planes per tile
  static_assert(TU % 64 == 0, "whole wave loads per tile");
  constexpr int YI = (TU / 64 + NWV - 1) / NWV;   // direct loads per wave and tile (at most)
  constexpr int YMIN = (TU / 64) / NWV;           // ... made by every wave
  static_assert(YMIN >= 1 && YI <= 3, "tile shape");
  constexpr bool LSE = EPI == 4;              // log-sum-exp (E = 1, no b planes)
  constexpr int W = 16 * EB;
  constexpr int BQ = LSE ? 1 : 15 * W;        // uint4 of a slot's b planes
  constexpr int BO = LSE ? 0 : (BQ + 63) / 64;   // wave loads of a slot's b planes
  constexpr int BI = (BO + NWV - 1) / NWV;
  // direct loads per wave and tile, the fewest over the waves (y, b, norms)
  constexpr int VKEEP = split32_min_loads(TU / 64, BO, NWV);
  static_assert(VKEEP >= 1 && VKEEP <= 15, "wait count");
  // XC: one more signal column (fp32, a.xb) summed per lane on the vector ALU;
  // its tile of 32 values sits after the norms in the same buffer
  static_assert(!XC || (!LSE && EB == 4 && NWV >= 2), "extra column with 64 signal columns");
  constexpr int NQ = XC ? TJ / 2 : TJ / 4;   // float4 of a slot's norms (and extra column)

  // four buffers of a tile: y planes as in HBM, uint4 q of column c at
  // position q ^ (c & (PU - 1)) within its plane (16 consecutive columns on
  // distinct bank groups), the norms, and the b planes (rows of 5 uint4);
  // distinct arrays, indexed statically, so that the compiler knows that the
  // direct loads into one buffer never alias the reads of another
  __shared__ uint4 ys0[TU], ys1[TU], ys2[TU], ys3[TU];
  __shared__ float4 ns0[NQ], ns1[NQ], ns2[NQ], ns3[NQ];
  __shared__ uint4 bq0[BQ], bq1[BQ], bq2[BQ], bq3[BQ];

  if (a.xskip) return;   // (summed with the previous launch)
  if (wide64(a.spread, a.wide_c, a.wide_limit)) return;   // the fp64 contraction does the work
  const MItem it = mitem<SP>(a, 32 * NWV);
  if (!it.live) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int li = lane & 15, g = lane >> 4;    // P . B lanes
  const int i32 = lane & 31, h = lane >> 5;   // exponent lanes
  const int c = it.c;
  const int64_t rend = it.row_end;
  const int64_t i0 = it.row0 + wave * 32;

  // planes of x[i32][16 ch + 8 h + t]; X = fl32(s (x - m)) formed in fp64 and
  // nx = -fl32(|X|^2) summed in fp64
  bf16x8 xh[NC], xm[NC], xl[NC];
  float nx;
  {
    const int64_t row = i0 + i32;
    const bool ok = row < rend;
    double part = 0.0;
#pragma unroll
    for (int ch = 0; ch < NC; ++ch)
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int d = 16 * ch + 8 * h + t;
        const float v =
            (ok && d < a.D) ? (float)(((double)a.x[row * a.D + d] -
                                       (double)(a.xc != nullptr ? a.xc[d] : 0.0f)) * a.xscale64)
                            : 0.0f;
        __bf16 vh, vm, vl;
        split3(v, vh, vm, vl);
        xh[ch][t] = vh;
        xm[ch][t] = vm;
        xl[ch][t] = vl;
        part = __builtin_fma((double)v, (double)v, part);
      }
    part += __shfl_xor(part, 32);
    nx = -(float)part;
  }

  f4 tot[2][EB];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int eb = 0; eb < EB; ++eb) tot[u][eb] = f4{0.f, 0.f, 0.f, 0.f};

  // source of the uint4 this lane loads into slot k of a whole tile
  int yoff[YI];
#pragma unroll
  for (int k = 0; k < YI; ++k) {
    const int sl = 64 * (NWV * k + wave) + lane;
    const int cc = sl / (3 * PU), qq = sl - cc * 3 * PU;
    yoff[k] = cc * 3 * PU + (qq ^ (cc & (PU - 1)));
  }

  // the tile at column jt (32-aligned) into buffers yd, nd, bd, every
  // part straight from memory into LDS (lane l of a wave writes the 4 or 16
  // bytes at the window's base + l times that; each lane loads what belongs
  // at its position): the norms (a column outside [lo, hi) or past the
  // loaded 16-column blocks reads a padding norm), the b planes (the row
  // padding slots read any b), and the y planes (a column past the loaded
  // blocks reads a copy of the last loaded one: finite, removed by its norm)
  // (with XC the per-lane load offsets pass through an empty asm statement
  // each tile, so that the compiler recomputes their 64-bit addresses instead
  // of keeping them across the loop: at DP = 128, 64 signal columns, that
  // spilled them, 79.4 ms per launch against 74.4 without)
  auto fetch = [&](uint4 (&yd)[TU], float4 (&nd)[NQ], uint4 (&bd)[BQ], int64_t jt, int64_t lo,
                   int64_t hi) __attribute__((always_inline)) {
    const int ncol = (int)min((int64_t)TJ, ((hi + 15) & ~(int64_t)15) - jt);
    if (wave == NWV - 1 && lane < TJ) {
      int ln = lane;
      if constexpr (XC) asm volatile("" : "+v"(ln));
      const int64_t col = jt + ln;
      const bool live = SP ? (col >= lo && col < hi) : (lane < ncol);
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(a.ny + (live ? col : a.N16)),
                                       (__attribute__((address_space(3))) void*)(&nd[0]), 4, 0, 0);
    }
    if constexpr (XC) {
      // the extra column's values (a masked column reads the zero at N16)
      if (wave == NWV - 2 && lane < TJ) {
        int ln = lane;
        asm volatile("" : "+v"(ln));
        const int64_t col = jt + ln;
        const bool live = SP ? (col >= lo && col < hi) : (lane < ncol);
        __builtin_amdgcn_global_load_lds(static_cast<const void*>(a.xb + (live ? col : a.N16)),
                                         (__attribute__((address_space(3))) void*)(&nd[TJ / 4]), 4, 0, 0);
      }
    }
    const uint4* bsrc = LSE ? nullptr : reinterpret_cast<const uint4*>(a.bpk) + (jt / 32) * (12 * W);
#pragma unroll
    for (int k = 0; k < BI; ++k) {
      const int o = NWV * k + wave;   // the wave's window of the slot
      if (o >= BO) break;             // wave-uniform
      const int sl = 64 * o + lane, row = sl / 5, kc = sl - row * 5;
      int bo = row * 4 + (kc < 4 ? kc : 0);
      if constexpr (XC) asm volatile("" : "+v"(bo));
      if (sl < 15 * W)
        __builtin_amdgcn_global_load_lds(static_cast<const void*>(bsrc + bo),
                                         (__attribute__((address_space(3))) void*)(&bd[64 * o]), 16, 0, 0);
    }
    const uint4* ysrc = reinterpret_cast<const uint4*>(a.ysp + jt * 3 * DP);
#pragma unroll
    for (int k = 0; k < YI; ++k) {
      const int s0 = 64 * (NWV * k + wave);
      if (k >= YMIN && s0 >= TU) break;   // wave-uniform
      int src = yoff[k];
      if constexpr (XC) asm volatile("" : "+v"(src));
      if (ncol < TJ) {
        const int sl = s0 + lane;
        const int cc = sl / (3 * PU), qq = sl - cc * 3 * PU;
        src = min(cc, ncol - 1) * 3 * PU + (qq ^ (cc & (PU - 1)));
      }
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(ysrc + src),
                                       (__attribute__((address_space(3))) void*)(&yd[s0]), 16, 0, 0);
    }
  };
  // vector-memory waits: the newest tile's direct loads (at least VKEEP per
  // wave, issued last) may stay in flight, or none
  auto wait_vm_keep = [&]() { __builtin_amdgcn_s_waitcnt((VKEEP & 15) | (0x7 << 4) | (0xf << 8)); };
  auto wait_vm_all = [&]() { __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xf << 8)); };
  // workgroup barrier ordering LDS only (vector-memory waits are explicit)
  auto barrier = [&]() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
  };

  // the tile's T less the norms: acc (hh, hm, mh) and acc2 (mm, hl, lh)
  auto exponent = [&](const uint4 (&yc)[TU], f16v& acc, f16v& acc2) __attribute__((always_inline)) {
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = acc2[r] = 0.0f;
    const uint4* col = &yc[i32 * 3 * PU];
    const int sw = i32 & (PU - 1);
#pragma unroll
    for (int ch = 0; ch < NC; ++ch) {
      const int q = (2 * ch + h) ^ sw;
      const bf16x8 yh = __builtin_bit_cast(bf16x8, col[q]);
      const bf16x8 ym = __builtin_bit_cast(bf16x8, col[PU + q]);
      const bf16x8 yl = __builtin_bit_cast(bf16x8, col[2 * PU + q]);
      acc2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ym, xm[ch], acc2, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ym, xh[ch], acc, 0, 0, 0);
      acc2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(yl, xh[ch], acc2, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(yh, xm[ch], acc, 0, 0, 0);
      acc2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(yh, xl[ch], acc2, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(yh, xh[ch], acc, 0, 0, 0);
    }
  };

  // p = 2^T of a tile from its fl(acc + acc2) and its norms nd, and p . b
  // (b planes bd) into tot
  // log-sum-exp: per lane the running maximum lm of its row's s (= T, log2
  // units) and the sum ls of 2^(s - lm), rescaled when lm moves (as the fp32
  // kernel; lm starts finite, so an empty start never forms inf - inf)
  float lm = -3.0e38f, ls = 0.0f;
  float xacc = 0.0f;   // the extra column: this lane's share of its row's sum
  auto finish = [&](const float4 (&nd)[NQ], const uint4 (&bd)[BQ], const f16v& ap)
                    __attribute__((always_inline)) {
    if constexpr (LSE) {
      float sv[16];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 nyv = nd[2 * q + h];
        sv[4 * q + 0] = ap[4 * q + 0] + (nx + nyv.x);
        sv[4 * q + 1] = ap[4 * q + 1] + (nx + nyv.y);
        sv[4 * q + 2] = ap[4 * q + 2] + (nx + nyv.z);
        sv[4 * q + 3] = ap[4 * q + 3] + (nx + nyv.w);
      }
      float mb = sv[0];
#pragma unroll
      for (int r = 1; r < 16; ++r) mb = fmaxf(mb, sv[r]);
      const float nm = fmaxf(lm, mb);
      float e[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) e[r] = __builtin_amdgcn_exp2f(sv[r] - nm);
#pragma unroll
      for (int w = 8; w >= 1; w >>= 1)
#pragma unroll
        for (int r = 0; r < w; ++r) e[r] += e[r + w];
      ls = ls * __builtin_amdgcn_exp2f(lm - nm) + e[0];
      lm = nm;
      return;
    }
    // T = fl(fl(acc + acc2) + fl(nx + ny)), p = 2^T; column 8 q + 4 h + r
    float p[16];
    float xq[4];   // XC: p times the extra column over each group of 4 columns
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 nyv = nd[2 * q + h];
      p[4 * q + 0] = __builtin_amdgcn_exp2f(ap[4 * q + 0] + (nx + nyv.x));
      p[4 * q + 1] = __builtin_amdgcn_exp2f(ap[4 * q + 1] + (nx + nyv.y));
      p[4 * q + 2] = __builtin_amdgcn_exp2f(ap[4 * q + 2] + (nx + nyv.z));
      p[4 * q + 3] = __builtin_amdgcn_exp2f(ap[4 * q + 3] + (nx + nyv.w));
      if constexpr (XC) {
        const float4 xv = nd[TJ / 4 + 2 * q + h];
        xq[q] = __builtin_fmaf(p[4 * q + 3], xv.w,
                               __builtin_fmaf(p[4 * q + 2], xv.z,
                                              __builtin_fmaf(p[4 * q + 1], xv.y, p[4 * q + 0] * xv.x)));
      }
    }
    // the tile's 16 columns into the running sum once (one rounding per tile,
    // as P . B)
    if constexpr (XC) xacc += (xq[0] + xq[1]) + (xq[2] + xq[3]);
    // U = q 0, 2 and V = q 1, 3 -> rows 0-15 (u = 0) and 16-31 (u = 1)
    float pr[2][8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const int ru = t < 4 ? t : t + 4, rv = ru + 4;
      const auto s1 = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, p[ru]),
                                                       __builtin_bit_cast(unsigned, p[rv]), false, false);
      const auto s2 = __builtin_amdgcn_permlane16_swap(s1[0], s1[1], false, false);
      pr[0][t] = __builtin_bit_cast(float, (unsigned)s2[0]);
      pr[1][t] = __builtin_bit_cast(float, (unsigned)s2[1]);
    }
    bf16x8 ph[2], pm[2], pl[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      unsigned hw[4], mw[4], lw[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) split3x2(pr[u][2 * k], pr[u][2 * k + 1], hw[k], mw[k], lw[k]);
      ph[u] = __builtin_bit_cast(bf16x8, uint4{hw[0], hw[1], hw[2], hw[3]});
      pm[u] = __builtin_bit_cast(bf16x8, uint4{mw[0], mw[1], mw[2], mw[3]});
      pl[u] = __builtin_bit_cast(bf16x8, uint4{lw[0], lw[1], lw[2], lw[3]});
    }
#pragma unroll
    for (int eb = 0; eb < EB; ++eb) {
      // B planes: b[j(k)][e = 16 eb + li] for k = 8 g .. 8 g + 7
      const uint4* brow = &bd[(16 * eb + li) * 5 + g];
      const bf16x8 bh = __builtin_bit_cast(bf16x8, brow[0]);
      const bf16x8 bm = __builtin_bit_cast(bf16x8, brow[5 * W]);
      const bf16x8 bl = __builtin_bit_cast(bf16x8, brow[10 * W]);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        // smallest partial products first, from zero; then into the total
        f4 o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pm[u], bm, f4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
        o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pl[u], bh, o, 0, 0, 0);
        o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph[u], bl, o, 0, 0, 0);
        o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pm[u], bh, o, 0, 0, 0);
        o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph[u], bm, o, 0, 0, 0);
        o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph[u], bh, o, 0, 0, 0);
        tot[u][eb] += o;
      }
    }
  };

  // Pipeline per tile t (buffers t % 4): at its start tile t has landed and
  // tile t + 1 may be in flight; it prefetches tile t + 2 (into the buffers
  // tile t - 2 used), forms tile t's products and finishes tile t - 1 (its
  // buffers stay untouched until tile t + 3's prefetch; without PIPE, tile t),
  // and waits for tile t + 1.  Each segment ends with a barrier, as the next one starts over at
  // buffers 0.
  // (with 32 or 64 signal columns the registers do not hold two tiles: each tile is
  // finished right after its products)
  constexpr bool PIPE = EB == 1;
  f16v accp;   // fl(acc + acc2) of the pending tile
  auto step = [&](int t, int ntiles, int64_t base, int64_t a0, int64_t a1, const uint4 (&yc)[TU],
                  const float4 (&nc)[NQ], const uint4 (&bc)[BQ], const float4 (&nf)[NQ],
                  const uint4 (&bf)[BQ], uint4 (&yn)[TU], float4 (&nn)[NQ],
                  uint4 (&bn)[BQ]) __attribute__((always_inline)) {
    const bool more = t + 2 < ntiles;
    if (more) fetch(yn, nn, bn, base + (int64_t)(t + 2) * TJ, a0, a1);
    f16v acc, acc2;
    exponent(yc, acc, acc2);
    if constexpr (PIPE) {
      if (t > 0) finish(nf, bf, accp);
      accp = acc + acc2;
    } else {
      finish(nc, bc, acc + acc2);
    }
    if (more) wait_vm_keep();   // tile t + 1 has landed
    else wait_vm_all();
    barrier();
  };
  auto segment = [&](int64_t a0, int64_t a1) {
    const int64_t base = a0 & ~(int64_t)31;
    const int ntiles = (int)((a1 - base + TJ - 1) / TJ);
    fetch(ys0, ns0, bq0, base, a0, a1);
    if (ntiles > 1) {
      fetch(ys1, ns1, bq1, base + TJ, a0, a1);
      wait_vm_keep();   // tile 0 has landed
    } else {
      wait_vm_all();
    }
    barrier();
    step(0, ntiles, base, a0, a1, ys0, ns0, bq0, ns3, bq3, ys2, ns2, bq2);   // (no tile -1)
    for (int t = 1; t < ntiles; t += 4) {
      step(t, ntiles, base, a0, a1, ys1, ns1, bq1, ns0, bq0, ys3, ns3, bq3);
      if (t + 1 < ntiles) step(t + 1, ntiles, base, a0, a1, ys2, ns2, bq2, ns1, bq1, ys0, ns0, bq0);
      if (t + 2 < ntiles) step(t + 2, ntiles, base, a0, a1, ys3, ns3, bq3, ns2, bq2, ys1, ns1, bq1);
      if (t + 3 < ntiles) step(t + 3, ntiles, base, a0, a1, ys0, ns0, bq0, ns3, bq3, ys2, ns2, bq2);
    }
    if constexpr (PIPE) {
      switch ((ntiles - 1) & 3) {
        case 0: finish(ns0, bq0, accp); break;
        case 1: finish(ns1, bq1, accp); break;
        case 2: finish(ns2, bq2, accp); break;
        default: finish(ns3, bq3, accp); break;
      }
    }
    barrier();
  };
  if constexpr (SP) for_segments(a, it, segment);
  else if (it.w0 < it.w1) segment(it.w0, it.w1);

  if constexpr (LSE) {
    // merge the row's two lanes (h = 0, 1): (m, s) + (m', s') relative to max(m, m')
    const float m2 = __shfl_xor(lm, 32), s2 = __shfl_xor(ls, 32);
    const float nm = fmaxf(lm, m2);
    const float t = ls * __builtin_amdgcn_exp2f(lm - nm) + s2 * __builtin_amdgcn_exp2f(m2 - nm);
    const int64_t row = i0 + i32;
    if (h == 0 && row < rend) {
      if (a.C == 1) {
        // an empty row (t = 0) gives -infinity
        static_cast<float*>(a.out)[row] = (nm + __builtin_amdgcn_logf(t)) * kLn2;
      } else {
        float* pp = a.part + ((int64_t)c * a.M + row) * 2;   // the (m, s) pair the combine merges
        pp[0] = t > 0.0f ? nm : -__builtin_inff();
        pp[1] = t;
      }
    }
    return;
  }
  if constexpr (XC) {
    // the row's two lanes (h = 0, 1) hold halves of its extra-column sum
    const float xs = xacc + __shfl_xor(xacc, 32);
    const int64_t row = i0 + i32;
    if (h == 0 && row < rend) {
      if (a.C == 1) a.xout[row] = xs;
      else a.xpart[(int64_t)c * a.M + row] = xs;
    }
  }
  // lane holds out[i = 16 u + 4 g + r][e = 16 eb + li]
  const int Ec = min(W, a.E - a.e0);
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int eb = 0; eb < EB; ++eb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = i0 + 16 * u + 4 * g + r;
        const int e = 16 * eb + li;
        if (row >= rend) continue;
        if (a.C == 1) {
          if (e < Ec) static_cast<float*>(a.out)[row * a.E + a.e0 + e] = tot[u][eb][r];
        } else {
          a.part[((int64_t)c * a.M + row) * W + e] = tot[u][eb][r];
        }
      }
}

// waves per workgroup of mfma_split_kernel: 8 (two per SIMD); the
// log-sum-exp at DP = 64 holds 158 VGPRs and runs three per SIMD in
// workgroups of 4 (lse_d64: 4.5% faster than with 8), and DP = 32 takes
// workgroups of 4 as well (the whole tile is six wave loads)
constexpr int split32_waves(int NC, int EPI) { return (NC <= 2 || (EPI == 4 && NC <= 4)) ? 4 : 8; }

template <int NC, bool SP>
hipError_t launch_split32_n(const MfmaArgs& a, dim3 grid, hipStream_t s) {
  if (a.epi == 4) {   // the Gaussian and Sinkhorn log-sum-exp
    constexpr int NW = split32_waves(NC, 4);
    hipLaunchKernelGGL((mfma_split_kernel<NC, 1, 4, NW, SP>), grid, dim3(64 * NW), 0, s, a);
    return hipGetLastError();
  }
  if (a.epi != 0) return hipSuccess;   // as launch_split_n
  constexpr int NW = split32_waves(NC, 0);
  switch (a.EB) {
    case 1: hipLaunchKernelGGL((mfma_split_kernel<NC, 1, 0, NW, SP>), grid, dim3(64 * NW), 0, s, a); break;
    case 2: hipLaunchKernelGGL((mfma_split_kernel<NC, 2, 0, NW, SP>), grid, dim3(64 * NW), 0, s, a); break;
    case 4:
      if (a.xb) hipLaunchKernelGGL((mfma_split_kernel<NC, 4, 0, NW, SP, true>), grid, dim3(64 * NW), 0, s, a);
      else hipLaunchKernelGGL((mfma_split_kernel<NC, 4, 0, NW, SP>), grid, dim3(64 * NW), 0, s, a);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}


template <int Q>
constexpr int rows_blocks() { return Q >= 64 ? 1 : 2; }

template <int Q, int EPI, bool SP>
hipError_t launch_sum_q(const MfmaArgs& a, dim3 grid, hipStream_t s) {
  constexpr int RB = rows_blocks<Q>();
  switch (a.EB) {
    case 1: hipLaunchKernelGGL((mfma_kernel<Q, RB, EPI, 1, 1, SP>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((mfma_kernel<Q, RB, EPI, 2, 1, SP>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((mfma_kernel<Q, RB, EPI, 4, 1, SP>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int Q, bool SP>
hipError_t launch_q(const MfmaArgs& a, dim3 grid, hipStream_t s) {
  constexpr int RB = rows_blocks<Q>();
  switch (a.epi) {
    case 0: return launch_sum_q<Q, 0, SP>(a, grid, s);
    case 1: return launch_sum_q<Q, 1, SP>(a, grid, s);
    case 2: return launch_sum_q<Q, 2, SP>(a, grid, s);
    case 4:
      hipLaunchKernelGGL((mfma_kernel<Q, RB, 4, 1, 1, SP>), grid, dim3(256), 0, s, a);
      return hipGetLastError();
    case 5:
      hipLaunchKernelGGL((mfma_kernel<Q, RB, 5, 1, 1, SP>), grid, dim3(256), 0, s, a);
      return hipGetLastError();
#define KRED_EXT_F32(EPV)                                                                      \
  case EPV:                                                                                    \
    hipLaunchKernelGGL((mfma_kernel<Q, RB, EPV, 1, 1, SP>), grid, dim3(256), 0, s, a);        \
    return hipGetLastError();
    KRED_EXT_F32(6) KRED_EXT_F32(7) KRED_EXT_F32(8) KRED_EXT_F32(9)
#undef KRED_EXT_F32
    case 3:
      switch (a.KP) {
#define KRED_KNN_F32(KPV, RBV)                                                                 \
  case KPV:                                                                                     \
    hipLaunchKernelGGL((mfma_kernel<Q, RBV, 3, 1, KPV, SP>), grid, dim3(256), 0, s, a);        \
    break;
        KRED_KNN_F32(1, RB) KRED_KNN_F32(4, RB) KRED_KNN_F32(8, RB) KRED_KNN_F32(10, RB)
        KRED_KNN_F32(12, RB) KRED_KNN_F32(16, RB) KRED_KNN_F32(64, 1)
#undef KRED_KNN_F32
        default: return hipErrorInvalidValue;
      }
      return hipGetLastError();
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace

int mfma_pad_d(int D) { return D <= 32 ? 32 : (D <= 64 ? 64 : (D <= 128 ? 128 : (D <= 256 ? 256 : 0))); }

int mfma_tile_cols(int DP) { return tile_cols(DP); }

int64_t mfma_row_groups(const MfmaArgs& a, int rows) {
  return a.nr > 0 ? range_grid_bound(a.nr, a.M, rows) : (a.M + rows - 1) / rows;
}

int mfma_knn_pad_k(int K) {
  return K <= 1 ? 1 : K <= 4 ? 4 : K <= 8 ? 8 : K <= 10 ? 10 : K <= 12 ? 12 : K <= 16 ? 16 : 64;
}

int mfma_rows_per_block(int DP, int KP) {
  const int Q = DP / 4;
  return 64 * ((Q >= 64 || KP == 64) ? 1 : 2);
}

int mfma_split_rows_per_block(int DP, int epi) {
  if (DP == 32 || DP == 64 || DP == 128) return 32 * (epi == 4 ? split32_waves(DP / 16, 4) : split32_waves(DP / 16, 0));
  return mfma_rows_per_block(DP, 0);
}

// ------------------------------------------ centre; fused gradient, large D
// Distances do not change when x and y move by the same point m; taking m
// inside the data (the mean of up to the first 256 rows of y) keeps the
// expanded form's cancellation, |x|^2 + |y|^2 - 2 <x, y>, at the scale of the
// data's spread rather than its distance from the origin.
// The Gaussian sum's x-gradient g_i = sum_j k_ij b_j (y_j - x_i) / sigma^2
// (the derivative of Eq. (1)) is, for any point m, (A1_i - (x_i - m) A0_i) /
// sigma^2 with A0 = K b and A1 = K [b (y - m)]: one Gaussian sum with D + 1
// signal columns; with the same m, |y - m| stays of the order of |y - x| and
// the subtraction loses little.

namespace {

__global__ __launch_bounds__(256) void centre_kernel(const float* __restrict__ y, int64_t N,
                                                           int D, float* __restrict__ m) {
  const int d = threadIdx.x;
  if (d >= D) return;
  const int n = (int)min(N, (int64_t)256);
  // 16 independent sums, so 16 loads are in flight per step
  float s[16];
#pragma unroll
  for (int u = 0; u < 16; ++u) s[u] = 0.0f;
  int j = 0;
  for (; j + 16 <= n; j += 16) {
#pragma unroll
    for (int u = 0; u < 16; ++u) s[u] += y[(int64_t)(j + u) * D + d];
  }
  for (; j < n; ++j) s[0] += y[(int64_t)j * D + d];
#pragma unroll
  for (int w = 8; w > 0; w >>= 1)
#pragma unroll
    for (int u = 0; u < w; ++u) s[u] += s[u + w];
  m[d] = n > 0 ? s[0] / (float)n : 0.0f;
}

// The guard's spread: max |x_i - m|^2 and max |y_j - m|^2, one wave per row
// (lanes stride over d), folded in with atomicMax on the bit patterns (the
// values are non-negative).  Each is rounded up by 2^-20 relative, so the
// fp32 sum is an upper bound.
__global__ void spread_init_kernel(SpreadGuard* g) {
  if (threadIdx.x == 0) {
    g->maxx = 0u;
    g->maxy = 0u;
  }
}
__global__ __launch_bounds__(256) void spread_kernel(const float* __restrict__ x, int64_t M,
                                                     const float* __restrict__ y, int64_t N, int D,
                                                     const float* __restrict__ m, SpreadGuard* g) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
  const int64_t waves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  float bx = 0.0f, by = 0.0f;
  for (int64_t r = wave; r < M + N; r += waves) {
    const float* p = r < M ? x + r * D : y + (r - M) * D;
    // in fp64 (the differences exact), rounded up by a margin far above the
    // roundings of the sum and of L = c (maxx + maxy) in fp32
    double s = 0.0;
    for (int d = lane; d < D; d += 64) {
      const double v = (double)p[d] - (double)m[d];
      s = __builtin_fma(v, v, s);
    }
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    const float sf = (float)(s * (1.0 + 1.0 / 1048576.0));
    if (r < M) bx = fmaxf(bx, sf);
    else by = fmaxf(by, sf);
  }
  if (lane == 0) {
    atomicMax(&g->maxx, __float_as_uint(bx));
    atomicMax(&g->maxy, __float_as_uint(by));
  }
}
__global__ void wide_record_kernel(const SpreadGuard* g, float c, float limit, int* counts) {
  if (threadIdx.x == 0) {
    if (wide64(g, c, limit)) atomicAdd(&counts[0], 1);
    atomicAdd(&counts[1], 1);
  }
}

// columns [c0, c0 + Ec) of the signal [b_e, b_e (y - m)] for e = 0..E-1
// (column e (D + 1) + k): N x Ec, row-major
__global__ __launch_bounds__(256) void gradx_signal_kernel(const float* __restrict__ y,
                                                           const float* __restrict__ b, int64_t N,
                                                           int D, int E, const float* __restrict__ m,
                                                           int c0, int Ec, float* __restrict__ sig) {
  const int64_t total = N * Ec;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t j = t / Ec;
    const int c = c0 + (int)(t - j * Ec);
    const int e = c / (D + 1), k = c - e * (D + 1);
    const float be = b[j * E + e];
    sig[t] = k == 0 ? be : be * (y[j * D + k - 1] - m[k - 1]);
  }
}

// column c of the sums T (M x W in chunks of 64 columns, chunk q stored M x Ec_q
// at T + 64 M q)
__device__ __forceinline__ float wide_at(const float* __restrict__ T, int64_t M, int W, int64_t i,
                                         int c) {
  const int q = c / 64, last = (W - 1) / 64;
  const int ec = q == last ? W - 64 * last : 64;
  return T[64 * M * q + i * ec + (c - 64 * q)];
}

// the vector-Jacobian product: out[i, d] = gscale sum_e e_ie (A_e,1+d - (x_id - m_d) A_e,0)
__global__ __launch_bounds__(256) void vjp_finish_kernel(const float* __restrict__ x, int64_t M,
                                                         int D, int E, const float* __restrict__ m,
                                                         const float* __restrict__ T,
                                                         const float* __restrict__ e,
                                                         float gscale, float* __restrict__ out) {
  const int W = E * (D + 1);
  const int64_t total = M * D;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = t / D;
    const int d = (int)(t - i * D);
    const float xd = x[i * D + d] - m[d];
    float acc = 0.0f;
    for (int f = 0; f < E; ++f) {
      const int c = f * (D + 1);
      acc = __builtin_fmaf(e[i * E + f], wide_at(T, M, W, i, c + 1 + d) - xd * wide_at(T, M, W, i, c), acc);
    }
    out[t] = acc * gscale;
  }
}

// out[i] = (A0, (A1 - (x_i - m) A0) gscale); column c of A sits in chunk c / 64
// (M x Ec_q at T + 64 M q)
__global__ __launch_bounds__(256) void gradx_finish_kernel(const float* __restrict__ x, int64_t M,
                                                           int D, const float* __restrict__ m,
                                                           const float* __restrict__ T,
                                                           float gscale, float* __restrict__ out) {
  const int W = D + 1;
  const int64_t total = M * W;
  const int last = (W - 1) / 64;
  const int Elast = W - 64 * last;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = t / W;
    const int c = (int)(t - i * W);
    const int q = c / 64;
    const int ec = q == last ? Elast : 64;
    const float a = T[64 * M * q + i * ec + (c - 64 * q)];
    if (c == 0) {
      out[t] = a;
    } else {
      const float a0 = T[i * (last == 0 ? Elast : 64)];
      out[t] = (a - (x[i * D + c - 1] - m[c - 1]) * a0) * gscale;
    }
  }
}

int64_t grid_of(int64_t items) {
  return std::max<int64_t>(1, std::min<int64_t>((items + 255) / 256, 8192));
}

}  // namespace

hipError_t launch_centre(const float* y, int64_t N, int D, float* m, hipStream_t s) {
  hipLaunchKernelGGL(centre_kernel, dim3(1), dim3(256), 0, s, y, N, D, m);
  return hipGetLastError();
}

hipError_t launch_spread(const float* x, int64_t M, const float* y, int64_t N, int D,
                         const float* m, SpreadGuard* g, hipStream_t s) {
  hipLaunchKernelGGL(spread_init_kernel, dim3(1), dim3(64), 0, s, g);
  if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
  if (M + N == 0) return hipSuccess;
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((M + N + 3) / 4, 2048));
  hipLaunchKernelGGL(spread_kernel, dim3((unsigned)blocks), dim3(256), 0, s, x, M, y, N, D, m, g);
  return hipGetLastError();
}

hipError_t launch_wide_record(const SpreadGuard* g, float c, float limit, int* counts,
                              hipStream_t s) {
  hipLaunchKernelGGL(wide_record_kernel, dim3(1), dim3(64), 0, s, g, c, limit, counts);
  return hipGetLastError();
}

hipError_t launch_gradx_signal(const float* y, const float* b, int64_t N, int D, int E,
                               const float* m, int c0, int Ec, float* sig, hipStream_t s) {
  if (N == 0) return hipSuccess;
  hipLaunchKernelGGL(gradx_signal_kernel, dim3((unsigned)grid_of(N * Ec)), dim3(256), 0, s, y, b,
                     N, D, E, m, c0, Ec, sig);
  return hipGetLastError();
}

hipError_t launch_vjp_finish(const float* x, int64_t M, int D, int E, const float* m,
                             const float* T, const float* e, float gscale, float* out,
                             hipStream_t s) {
  if (M == 0) return hipSuccess;
  hipLaunchKernelGGL(vjp_finish_kernel, dim3((unsigned)grid_of(M * D)), dim3(256), 0, s, x, M, D,
                     E, m, T, e, gscale, out);
  return hipGetLastError();
}

hipError_t launch_gradx_finish(const float* x, int64_t M, int D, const float* m, const float* T,
                               float gscale, float* out, hipStream_t s) {
  if (M == 0) return hipSuccess;
  hipLaunchKernelGGL(gradx_finish_kernel, dim3((unsigned)grid_of(M * (D + 1))), dim3(256), 0, s,
                     x, M, D, m, T, gscale, out);
  return hipGetLastError();
}

hipError_t launch_mfma_pack(const MfmaPackArgs& a, hipStream_t s) {
  if (a.N16 == 0) return hipSuccess;
  const int64_t items = a.N16 * std::max(a.DP, 16 * a.EB);
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((items + 255) / 256, 8192));
  hipLaunchKernelGGL(mfma_pack_kernel, dim3((unsigned)blocks), dim3(256), 0, s, a);
  if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
  const int64_t nb = std::max<int64_t>(1, std::min<int64_t>((a.N16 + 3) / 4, 4096));
  hipLaunchKernelGGL(mfma_norm_kernel, dim3((unsigned)nb), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_exact_check(const float* x, int64_t M, const float* y, int64_t N, int D,
                              ExactGuard* g, hipStream_t s) {
  hipLaunchKernelGGL(exact_init_kernel, dim3(1), dim3(64), 0, s, g);
  if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
  const int64_t total = (M + N) * (int64_t)D;
  if (total == 0) return hipSuccess;
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((total + 255) / 256, 4096));
  hipLaunchKernelGGL(exact_check_kernel, dim3((unsigned)blocks), dim3(256), 0, s, x, M * D, y,
                     N * D, g);
  return hipGetLastError();
}

hipError_t launch_mfma_split(const MfmaArgs& a, hipStream_t s) {
  const int rows = mfma_split_rows_per_block(a.DP, a.epi);
  const dim3 grid((unsigned)(mfma_row_groups(a, rows) * a.C));
  switch (a.DP) {
    case 32: return a.nr > 0 ? launch_split32_n<2, true>(a, grid, s) : launch_split32_n<2, false>(a, grid, s);
    case 64: return a.nr > 0 ? launch_split32_n<4, true>(a, grid, s) : launch_split32_n<4, false>(a, grid, s);
    case 128: return a.nr > 0 ? launch_split32_n<8, true>(a, grid, s) : launch_split32_n<8, false>(a, grid, s);
    case 256: return a.nr > 0 ? launch_split_n<8, true>(a, grid, s) : launch_split_n<8, false>(a, grid, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_mfma(const MfmaArgs& a, hipStream_t s) {
  const int rows = mfma_rows_per_block(a.DP, a.KP);
  const dim3 grid((unsigned)(mfma_row_groups(a, rows) * a.C));
  switch (a.DP) {
    case 32: return a.nr > 0 ? launch_q<8, true>(a, grid, s) : launch_q<8, false>(a, grid, s);
    case 64: return a.nr > 0 ? launch_q<16, true>(a, grid, s) : launch_q<16, false>(a, grid, s);
    case 128: return a.nr > 0 ? launch_q<32, true>(a, grid, s) : launch_q<32, false>(a, grid, s);
    case 256: return a.nr > 0 ? launch_q<64, true>(a, grid, s) : launch_q<64, false>(a, grid, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace kred
