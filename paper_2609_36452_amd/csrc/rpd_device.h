// Device-side pieces shared by the gfx950 kernels of the RPD commit step:
// vector types, output flag bits, the softmax state that the projection
// kernels produce and the reduction merges, and the XCD-aware job mapping.
//
// Pipeline of one call (all on the caller's stream):
//   k_compact       masked positions of the canvas -> compacted list
//                   (only masked positions are projected, Appendix A.6)
//   k_proj_bf16*    logit-lens projection z = W_U x for every (masked
//                   position, layer) row on the bf16 matrix cores, with the
//                   softmax statistics folded in per vocabulary tile, so the
//                   V-wide logits never reach memory (Section 2.2 readout;
//                   Eq. 1 entropy); one variant per range of row counts
//   k_proj_f32      the same on the vector ALU for fp32 inputs
//   k_reduce_score  merge of the per-tile statistics -> argmax, top
//                   probability and entropy per layer; persistence (Eq. 2),
//                   drop (Eq. 3), stability (Eq. 4) and candidacy (Eq. 5)
//   k_commit        per sequence: budgeted cumulative-entropy commitment and
//                   progress fallback (Section 3.2) as prefix scans
//
// The softmax statistics of a set of logits {z_v} are kept as
//   m = max z, idx = lowest v with z_v = m, S = sum e^{z-m}, T = sum e^{z-m}(z-m)
// from which top probability = 1/S and entropy = ln S - T/S. Two such states
// over disjoint vocabulary ranges merge exactly (up to rounding) by rescaling
// to the larger maximum; merges happen in a fixed order, so results are
// bitwise reproducible run to run.
#pragma once

#include <climits>
#include <cmath>

#include "rpd_launch.h"

namespace rpd {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr unsigned kFlagCandidate = 1u, kFlagHigh = 2u, kFlagStable = 4u, kFlagCommitted = 8u,
                   kFlagFallback = 16u;

// ------------------------------------------------------------ soft state --

struct Soft {
  float m;
  int idx;
  float S;
  float T;
};

__device__ __forceinline__ Soft soft_empty() {
  Soft s;
  s.m = -INFINITY;
  s.idx = INT_MAX;
  s.S = 0.f;
  s.T = 0.f;
  return s;
}

// S == 0 only for a state that has seen no vocabulary entry (a state with
// one or more entries has S >= 1, or NaN). Merging with an empty state
// returns the other one unchanged; the general formula is evaluated anyway
// and the empty cases are chosen by selects, so that lanes holding states
// of different kinds never branch.
__device__ __forceinline__ Soft soft_merge(const Soft a, const Soft b) {
  const float M = fmaxf(a.m, b.m);
  const float da = a.m - M, db = b.m - M;
  const float ea = __expf(da), eb = __expf(db);
  Soft r;
  r.m = M;
  r.S = a.S * ea + b.S * eb;
  r.T = (a.T + da * a.S) * ea + (b.T + db * b.S) * eb;
  r.idx = (a.m > b.m) ? a.idx : ((b.m > a.m) ? b.idx : min(a.idx, b.idx));
  const bool a_empty = a.S == 0.f, b_empty = b.S == 0.f;
  r.m = b_empty ? a.m : (a_empty ? b.m : r.m);
  r.idx = b_empty ? a.idx : (a_empty ? b.idx : r.idx);
  r.S = b_empty ? a.S : (a_empty ? b.S : r.S);
  r.T = b_empty ? a.T : (a_empty ? b.T : r.T);
  return r;
}

__device__ __forceinline__ Soft soft_shfl_xor(const Soft s, int mask) {
  Soft o;
  o.m = __shfl_xor(s.m, mask);
  o.idx = __shfl_xor(s.idx, mask);
  o.S = __shfl_xor(s.S, mask);
  o.T = __shfl_xor(s.T, mask);
  return o;
}

__device__ __forceinline__ float4 soft_pack(const Soft s) {
  return make_float4(s.m, __int_as_float(s.idx), s.S, s.T);
}

__device__ __forceinline__ Soft soft_unpack(const float4 v) {
  Soft s;
  s.m = v.x;
  s.idx = __float_as_int(v.y);
  s.S = v.z;
  s.T = v.w;
  return s;
}

// Statistics of N logits held by one lane, vocabulary indices increasing;
// entries with valid == false add nothing. NaN logits never win the max and
// turn S and T into NaN. Written with selects instead of branches (an
// invalid entry adds an exact 0 to S and T), since the validity differs
// from lane to lane and the branches cost more than the arithmetic.
template <int N>
__device__ __forceinline__ Soft soft_from_values(const float (&z)[N], const int (&v)[N], const bool (&ok)[N]) {
  float m = -INFINITY;
  int idx = INT_MAX;
#pragma unroll
  for (int e = 0; e < N; ++e) {
    const bool take = ok[e] && z[e] > m;
    m = take ? z[e] : m;
    idx = take ? v[e] : idx;
  }
  float S = 0.f, T = 0.f;
#pragma unroll
  for (int e = 0; e < N; ++e) {
    const float dz = ok[e] ? z[e] - m : 0.f;
    const float ex = ok[e] ? __expf(dz) : 0.f;
    S += ex;
    T = fmaf(ex, dz, T);
  }
  Soft s;
  s.m = m;
  s.idx = idx;
  s.S = S;
  s.T = T;
  return s;
}

// Map a workgroup to (row tile, vocab tile). Consecutive workgroup ids are
// dispatched round-robin over the 8 XCDs, so id % 8 selects the XCD and the
// jobs of one XCD are laid out so that its concurrently running workgroups
// share operands in that XCD's L2: with many row tiles each XCD owns a block
// of row tiles and sweeps the vocabulary for groups of up to 8 of them (all
// tiles of one vocabulary range and one group run together); with few row
// tiles each XCD owns a contiguous range of vocabulary tiles.
__device__ __forceinline__ bool map_job(int bid, int nvt, int nrt, int split_rows, int& rt, int& vt) {
  const int xcd = bid & 7, local = bid >> 3;
  if (split_rows) {
    const int lo = (int)((long long)xcd * nrt / 8), hi = (int)((long long)(xcd + 1) * nrt / 8);
    const int nr = hi - lo;
    if (nr <= 0 || local >= nr * nvt) return false;
    // the XCD's row tiles in groups of at most kRowGroup: a group's hidden rows stay cached while the
    // vocabulary streams past once per group (with more row tiles than that, sweeping the vocabulary
    // for all of them at once would re-read their hidden rows from HBM for every vocabulary tile)
    constexpr int kRowGroup = 8;
    const int g0 = local / (kRowGroup * nvt) * kRowGroup;
    const int gsz = min(kRowGroup, nr - g0);
    const int rem = local - g0 * nvt;
    vt = rem / gsz;
    rt = lo + g0 + (rem - vt * gsz);
  } else {
    const int lo = (int)((long long)xcd * nvt / 8), hi = (int)((long long)(xcd + 1) * nvt / 8);
    const int nv = hi - lo;
    if (nv <= 0 || local >= nv * nrt) return false;
    const int q = local / nrt;
    vt = lo + q;
    rt = local - q * nrt;
  }
  return true;
}

}  // namespace
}  // namespace rpd
