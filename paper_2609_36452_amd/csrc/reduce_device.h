// Device pieces of the cross-tile reductions (k_reduce_score, k_lazy_reduce):
// the fixed-order merge of a row's vocabulary-tile states and the
// resolution of exact argmax ties after a projection whose tiles sum a
// row's products in different orders.
#pragma once

#include "rpd_device.h"

namespace rpd {
namespace {

// ------------------------------------------------------ exact argmax ties --
//
// The streaming projection takes each vocabulary tile's k-chunks in its own
// rotated order, and the MFMA tile with a single row tile one order per XCD
// (both against HBM channel crowding), so two equal W_U rows in different
// tiles can round to different fp32 logits, and the cross-tile
// merge alone would then not give the lowest index of an exact tie. After
// the merge, every tile whose best row has a lower index than the winner y
// and a maximum below it by at most the accumulation-rounding bound
// 4 (d+1) 2^-24 |scale| sum_k |W_U[y,k] x_k| is a candidate: its row and y
// are evaluated again in float64, in one fixed order that is the same for
// every row (so equal rows give equal values), and the largest wins, the
// lowest index among equals. The bound needs y's row; it is read only when
// some lower-index tile lies within 0.25 (|m| + 1) of the maximum m (a
// sharp row never does). Exact as long as the rounding bound stays within
// that window, i.e. |scale| sum|W_U[y] x| <= 256 (|m| + 1) at d = 4096 (a
// ratio of about 8 for random rows at that size).
struct TieArgs {
  const uint16_t* w_u;   // NULL: the plan sums every row in the same order (nothing to resolve)
  int d;
  float scale;
};

// float64 dot product and sum of |products| of bf16 rows w and x (d % 8 ==
// 0, 16-byte aligned) by one wave, always in the same order: lane l sums the
// 8-element pieces l, l+64, ... in turn, then a fixed xor butterfly (each
// step adds two equal-shaped partial sums, and addition commutes, so every
// lane ends with the same value). Products of bf16 values are exact in
// float64. A lane issues the loads of eight pieces before it uses any (a
// single memory round trip at d <= 4096; one per piece in turn cost the
// call 5-6 us whenever a row was checked).
__device__ __forceinline__ void canon_dot_bf16(const uint16_t* __restrict__ w, const uint16_t* __restrict__ x,
                                               int d, int lane, double& z, double& a) {
  double zs = 0.0, as = 0.0;
  for (int p0 = lane; 8 * p0 < d; p0 += 64 * 8) {
    u32x4 wv[8], xv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int pc = p0 + 64 * u;
      wv[u] = u32x4{0u, 0u, 0u, 0u};
      xv[u] = u32x4{0u, 0u, 0u, 0u};
      if (8 * pc < d) {
        wv[u] = *reinterpret_cast<const u32x4*>(w + 8 * pc);
        xv[u] = *reinterpret_cast<const u32x4*>(x + 8 * pc);
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (8 * (p0 + 64 * u) >= d) break;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double p0_ = (double)__uint_as_float(wv[u][e] << 16) * (double)__uint_as_float(xv[u][e] << 16);
        const double p1_ =
            (double)__uint_as_float(wv[u][e] & 0xffff0000u) * (double)__uint_as_float(xv[u][e] & 0xffff0000u);
        zs += p0_;
        as += fabs(p0_);
        zs += p1_;
        as += fabs(p1_);
      }
    }
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    zs += __shfl_xor(zs, m);
    as += __shfl_xor(as, m);
  }
  z = zs;
  a = as;
}

__device__ __forceinline__ bool tie_candidate(const Soft& q, const Soft& s, float win) {
  return q.S > 0.f && q.idx < s.idx && q.m < s.m && q.m >= s.m - win;
}

// The tie resolution a reduction needs after a projection run with plan pl:
// needed where vocabulary tiles take their full 64-wide chunks in rotated
// orders (two or more of them).
inline TieArgs tie_args(const Launch& a, const ProjPlan& pl) {
  // the streaming kernels, and the MFMA tiles with a single row tile
  const bool big = pl.variant == PROJ_BF16_BIG || pl.variant == PROJ_BF16_BIG192 || pl.variant == PROJ_BF16_BIG128;
  const bool rotated = (pl.variant == PROJ_BF16_S32 || pl.variant == PROJ_BF16_S64 || (big && pl.nrt == 1)) &&
                       a.d / 64 >= 2;
  return TieArgs{rotated ? static_cast<const uint16_t*>(a.w_u) : nullptr, a.d, a.logit_scale};
}

// Fixed-order merge of one row's nvt vocabulary-tile states by one wave:
// lane folds tiles lane, lane+64, ... in tile order (loads batched eight at
// a time: one round trip for up to 512 tiles), then an xor butterfly
// combines the lanes. Every lane returns the row's state; keep[u] receives
// the lane's state of tile lane + 64u (u < 8; empty past nvt).
__device__ __forceinline__ Soft wave_merge_row(const float4* __restrict__ src, int nvt, int lane,
                                               float4 (&keep)[8]) {
  const float4 empty = soft_pack(soft_empty());
  Soft s = soft_empty();
  for (int t0 = lane; t0 < nvt; t0 += 64 * 8) {
    float4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = (t0 + 64 * u < nvt) ? src[t0 + 64 * u] : empty;
    if (t0 == lane) {
#pragma unroll
      for (int u = 0; u < 8; ++u) keep[u] = v[u];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) s = soft_merge(s, soft_unpack(v[u]));
  }
  if (nvt <= lane) {
#pragma unroll
    for (int u = 0; u < 8; ++u) keep[u] = empty;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) s = soft_merge(s, soft_shfl_xor(s, m));
  return s;
}

// The argmax of a merged row state s with its exact ties resolved (see
// above). src: the row's nvt tile states; keep: as wave_merge_row left it;
// x: the row's hidden state (after any normalization). Called by the whole
// wave.
__device__ __forceinline__ int resolve_tie(const Soft& s, const float4 (&keep)[8], const float4* __restrict__ src,
                                           int nvt, const TieArgs& ta, const uint16_t* __restrict__ x, int lane) {
  const int y = s.idx;
  if (!ta.w_u || y == INT_MAX || !(fabsf(s.m) <= 3.0e38f)) return y;
  const float wide = 0.25f * (fabsf(s.m) + 1.0f);
  bool near = false;
#pragma unroll
  for (int u = 0; u < 8; ++u) near |= tie_candidate(soft_unpack(keep[u]), s, wide);
  for (int t = 512 + lane; t < nvt; t += 64) near |= tie_candidate(soft_unpack(src[t]), s, wide);
  if (!__any(near)) return y;
  double zb, ay;
  canon_dot_bf16(ta.w_u + (long long)y * ta.d, x, ta.d, lane, zb, ay);
  const float win = (float)(4.0 * (ta.d + 1) * 0x1p-24 * ay * fabs((double)ta.scale));
  int best = y;
  // every candidate of a batch of 64 tiles (one per lane), in tile order
  auto batch = [&](const Soft& q) {
    unsigned long long bal = __ballot(tie_candidate(q, s, win));
    while (bal) {
      const int from = __ffsll((long long)bal) - 1;
      bal &= bal - 1ull;
      const int v = __shfl(q.idx, from);
      double zv, av;
      canon_dot_bf16(ta.w_u + (long long)v * ta.d, x, ta.d, lane, zv, av);
      if (zv > zb || (zv == zb && v < best)) {
        zb = zv;
        best = v;
      }
    }
  };
#pragma unroll
  for (int u = 0; u < 8; ++u) batch(soft_unpack(keep[u]));
  for (int t0 = 512; t0 < nvt; t0 += 64) batch(t0 + lane < nvt ? soft_unpack(src[t0 + lane]) : soft_empty());
  return best;
}

}  // namespace
}  // namespace rpd
