// gfx950 (CDNA4) kernels of the RPD commit step.
//
// Pipeline of one call (all on the caller's stream):
//   k_compact       masked positions of the canvas -> compacted list
//                   (only masked positions are projected, Appendix A.6)
//   k_proj_bf16     logit-lens projection z = W_U x for every (masked
//                   position, layer) row on the bf16 matrix cores, with the
//                   softmax statistics folded in per vocabulary tile, so the
//                   V-wide logits never reach memory (Section 2.2 readout;
//                   Eq. 1 entropy)
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
// one or more entries has S >= 1, or NaN).
__device__ __forceinline__ Soft soft_merge(const Soft a, const Soft b) {
  if (b.S == 0.f) return a;
  if (a.S == 0.f) return b;
  const float M = fmaxf(a.m, b.m);
  const float da = a.m - M, db = b.m - M;
  const float ea = __expf(da), eb = __expf(db);
  Soft r;
  r.m = M;
  r.S = a.S * ea + b.S * eb;
  r.T = (a.T + da * a.S) * ea + (b.T + db * b.S) * eb;
  r.idx = (a.m > b.m) ? a.idx : ((b.m > a.m) ? b.idx : min(a.idx, b.idx));
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
// entries with valid == false are skipped. NaN logits never win the max and
// turn S and T into NaN.
template <int N>
__device__ __forceinline__ Soft soft_from_values(const float (&z)[N], const int (&v)[N], const bool (&ok)[N]) {
  Soft s = soft_empty();
#pragma unroll
  for (int e = 0; e < N; ++e)
    if (ok[e] && z[e] > s.m) {
      s.m = z[e];
      s.idx = v[e];
    }
  float S = 0.f, T = 0.f;
#pragma unroll
  for (int e = 0; e < N; ++e)
    if (ok[e]) {
      const float dz = z[e] - s.m;
      const float ex = __expf(dz);
      S += ex;
      T = fmaf(ex, dz, T);
    }
  s.S = S;
  s.T = T;
  return s;
}

// ------------------------------------------------------------ K0 compact --

__global__ __launch_bounds__(1024) void k_compact(const uint8_t* __restrict__ mask, int BL, int cap,
                                                   int32_t* __restrict__ rows, int32_t* __restrict__ n_out,
                                                   int32_t* __restrict__ dev_status,
                                                   int32_t* __restrict__ user_status) {
  __shared__ int wsum[16];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int carry = 0;
  for (int base = 0; base < BL; base += blockDim.x) {
    const int i = base + threadIdx.x;
    const int f = (i < BL && mask[i] != 0) ? 1 : 0;
    const unsigned long long bal = __ballot(f);
    const int before = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) wsum[wid] = __popcll(bal);
    __syncthreads();
    int off = 0, tot = 0;
    for (int w = 0; w < nw; ++w) {
      const int c = wsum[w];
      off += (w < wid) ? c : 0;
      tot += c;
    }
    const int pos = carry + off + before;
    if (f && pos < cap) rows[pos] = i;
    carry += tot;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    int st = 0, n = carry;
    if (n > cap) {
      st |= 1;
      n = cap;
    }
    *n_out = n;
    *dev_status = st;
    if (user_status) *user_status = st;
  }
}

// ----------------------------------------------------- K1 projection bf16 --

// Map a workgroup to (row tile, vocab tile). Consecutive workgroup ids are
// dispatched round-robin over the 8 XCDs, so id % 8 selects the XCD and the
// jobs of one XCD are laid out so that its concurrently running workgroups
// share operands in that XCD's L2: with many row tiles each XCD owns a block
// of row tiles and sweeps the vocabulary (all its tiles of one vocabulary
// range run together); with few row tiles each XCD owns a contiguous range of
// vocabulary tiles.
__device__ __forceinline__ bool map_job(int bid, int nvt, int nrt, int split_rows, int& rt, int& vt) {
  const int xcd = bid & 7, local = bid >> 3;
  if (split_rows) {
    const int lo = (int)((long long)xcd * nrt / 8), hi = (int)((long long)(xcd + 1) * nrt / 8);
    const int nr = hi - lo;
    if (nr <= 0 || local >= nr * nvt) return false;
    vt = local / nr;
    rt = lo + (local - vt * nr);
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

// hidden-state chunk c (TR rows x KC elements) -> registers. GUARD: the
// chunk may cross d (zero fill past it); otherwise every load is in bounds.
template <int TR, int KC, int NT, int XPT, bool GUARD>
__device__ __forceinline__ void load_x_chunk(u32x4 (&xr)[XPT], const uint16_t* __restrict__ hidden,
                                             const long long* xoff, int c, int tid, int d) {
  constexpr int XP = TR * (KC / 8);
#pragma unroll
  for (int j = 0; j < XPT; ++j) {
    const int q = tid + j * NT;
    if (XP % NT == 0 || q < XP) {
      const int row = q / (KC / 8), c8 = q - row * (KC / 8);
      const int k = c * KC + c8 * 8;
      const u32x4* src = reinterpret_cast<const u32x4*>(hidden + xoff[row] + k);
      if (GUARD)
        xr[j] = k < d ? *src : u32x4{0u, 0u, 0u, 0u};
      else
        xr[j] = *src;
    }
  }
}

template <int TR, int KC, int KCP, int NT, int XPT>
__device__ __forceinline__ void store_x_chunk(uint16_t (*xsb)[KCP], const u32x4 (&xr)[XPT], int tid) {
  constexpr int XP = TR * (KC / 8);
#pragma unroll
  for (int j = 0; j < XPT; ++j) {
    const int q = tid + j * NT;
    if (XP % NT == 0 || q < XP) {
      const int row = q / (KC / 8), c8 = q - row * (KC / 8);
      *reinterpret_cast<u32x4*>(&xsb[row][c8 * 8]) = xr[j];
    }
  }
}

// this lane's W_U operand for chunk c: KS 32-wide k-steps x MV 16-row blocks
template <int MV, int KS, bool GUARD, bool NTA>
__device__ __forceinline__ void load_a_chunk(u32x4 (&dst)[KS][MV], const uint16_t* __restrict__ w_u,
                                             const long long (&aoff)[MV], int c, int kl, int d) {
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int k = (c * KS + s) * 32;
#pragma unroll
    for (int mv = 0; mv < MV; ++mv) {
      const u32x4* src = reinterpret_cast<const u32x4*>(w_u + aoff[mv] + k);
      if (GUARD)
        dst[s][mv] = k + kl < d ? *src : u32x4{0u, 0u, 0u, 0u};
      else if (NTA)
        dst[s][mv] = __builtin_nontemporal_load(src);
      else
        dst[s][mv] = *src;
    }
  }
}

// MFMAs of one staged chunk. The B fragments (hidden rows, from LDS) of
// k-step s+1 are read while the MFMAs of step s run, so the LDS latency is
// hidden even with one wave per SIMD.
template <int MV, int NB, int KS, int KCP>
__device__ __forceinline__ void mfma_chunk(f32x4 (&acc)[MV][NB], const u32x4 (&a)[KS][MV],
                                           const uint16_t (*xsb)[KCP], int lane, int kl) {
  u32x4 bq[2][NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
    bq[0][nb] = *reinterpret_cast<const u32x4*>(&xsb[nb * 16 + (lane & 15)][kl]);
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    if (s + 1 < KS) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        bq[(s + 1) & 1][nb] = *reinterpret_cast<const u32x4*>(&xsb[nb * 16 + (lane & 15)][(s + 1) * 32 + kl]);
    }
    // keep the prefetch of step s+1 ahead of the MFMAs of step s
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const bf16x8 bv = __builtin_bit_cast(bf16x8, bq[s & 1][nb]);
#pragma unroll
      for (int mv = 0; mv < MV; ++mv)
        acc[mv][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a[s][mv]), bv, acc[mv][nb],
                                                               0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Workgroup tile: TR = 16*NB projected rows x up to 16*MV*NW vocabulary rows,
// over the full hidden dimension. Each wave owns 16*MV consecutive W_U rows;
// its W_U operand goes straight from memory into registers (every W_U element
// is used by exactly one wave) with one 64-element chunk of prefetch, while
// the TR rows of hidden states, shared by all waves, are staged through a
// double-buffered LDS tile. v_mfma_f32_16x16x32_bf16 computes 16 vocab x 16
// rows; W_U is the A operand, so accumulator lane l holds, for row (l & 15)
// of its 16-row block, the logits of vocabulary entries 4*(l >> 4) + 0..3.
// The epilogue turns each lane's logits into a softmax state, merges the four
// lanes of a row and then the waves, and writes one 16-byte partial state per
// (row, vocab tile).
template <int NW, int MV, int NB, int KC, int NSTG, bool NTA>
__global__ __launch_bounds__(NW * 64) void k_proj_bf16(
    const uint16_t* __restrict__ hidden, const uint16_t* __restrict__ w_u, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ n_ptr, float4* __restrict__ partials, int K, int B, int L, int d, int V,
    int nvt, int nrt, int split_rows) {
  constexpr int TR = 16 * NB;
  static_assert(KC % 32 == 0, "a chunk is a whole number of MFMA k-steps");
  constexpr int KS = KC / 32;      // MFMA k-steps per chunk
  constexpr int KCP = KC + 8;      // padded LDS row length (elements)
  constexpr int NT = NW * 64;
  constexpr int XP = TR * (KC / 8);           // 16-byte pieces per hidden chunk
  constexpr int XPT = (XP + NT - 1) / NT;     // pieces per thread

  static_assert(NSTG >= 2, "at least double buffering");
  __shared__ __attribute__((aligned(16))) uint16_t xs[NSTG][TR][KCP];
  __shared__ long long xoff[TR];
  __shared__ float4 red[NW][TR];

  int rt, vt;
  if (!map_job(blockIdx.x, nvt, nrt, split_rows, rt, vt)) return;
  const int R = *n_ptr * K;
  const int r0 = rt * TR;
  if (r0 >= R) return;
  const int vb = (int)((long long)vt * V / nvt);
  const int ve = (int)((long long)(vt + 1) * V / nvt);

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;

  for (int t = tid; t < TR; t += NT) {
    const int r = r0 + t < R ? r0 + t : r0;   // padding rows re-read a real row; discarded at the end
    const int p = r / K, l = r - p * K;
    const int pos = rows[p];
    const int b = pos / L, i = pos - b * L;
    xoff[t] = (((long long)l * B + b) * L + i) * (long long)d;
  }
  __syncthreads();

  const int vw = vb + wid * 16 * MV;
  const int kl = (lane >> 4) * 8;  // this lane's k offset inside a 32-wide k-step
  long long aoff[MV];               // element offset of this lane's W_U row, per 16-row block
#pragma unroll
  for (int mv = 0; mv < MV; ++mv) aoff[mv] = (long long)min(vw + mv * 16 + (lane & 15), ve - 1) * d + kl;

  f32x4 acc[MV][NB];
#pragma unroll
  for (int mv = 0; mv < MV; ++mv)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mv][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // NSTG-stage ring: while chunk c is multiplied, the W_U and hidden loads
  // of chunks c+1 .. c+NSTG-1 are in flight. Buffer indices are compile-time
  // (the loop is unrolled by NSTG) and the body has no branches, so the
  // compiler's waits cover exactly the chunk being consumed.
  u32x4 A[NSTG][KS][MV];
  u32x4 xr[NSTG][XPT];
  const int nchf = d / KC;   // full chunks

#define RPD_LOAD_CHUNK(buf, chunk)                                                  \
  do {                                                                              \
    load_x_chunk<TR, KC, NT, XPT, false>(xr[buf], hidden, xoff, (chunk), tid, d);   \
    load_a_chunk<MV, KS, false, NTA>(A[buf], w_u, aoff, (chunk), kl, d);            \
  } while (0)

  if (nchf > 0) {
#pragma unroll
    for (int j = 0; j < NSTG - 1; ++j) RPD_LOAD_CHUNK(j, min(j, nchf - 1));
    store_x_chunk<TR, KC, KCP, NT, XPT>(xs[0], xr[0], tid);
    __syncthreads();
    const int nmain = (nchf / NSTG) * NSTG;
    for (int c0 = 0; c0 < nmain; c0 += NSTG) {
#pragma unroll
      for (int j = 0; j < NSTG; ++j) {
        // chunks past the end re-load the last chunk (never multiplied)
        RPD_LOAD_CHUNK((j + NSTG - 1) % NSTG, min(c0 + j + NSTG - 1, nchf - 1));
        __builtin_amdgcn_sched_barrier(0);
        mfma_chunk<MV, NB, KS, KCP>(acc, A[j], xs[j], lane, kl);
        store_x_chunk<TR, KC, KCP, NT, XPT>(xs[(j + 1) % NSTG], xr[(j + 1) % NSTG], tid);
        __syncthreads();
      }
    }
    // fewer than NSTG chunks remain; the ring already holds them in order
    const int rem = nchf - nmain;
#pragma unroll
    for (int j = 0; j < NSTG - 1; ++j) {
      if (j < rem) {
        mfma_chunk<MV, NB, KS, KCP>(acc, A[j], xs[j], lane, kl);
        if (j + 1 < rem) store_x_chunk<TR, KC, KCP, NT, XPT>(xs[j + 1], xr[j + 1], tid);
        __syncthreads();
      }
    }
  }
#undef RPD_LOAD_CHUNK
  if (d % KC != 0) {   // partial last chunk, zero-filled past d
    load_x_chunk<TR, KC, NT, XPT, true>(xr[0], hidden, xoff, nchf, tid, d);
    load_a_chunk<MV, KS, true, false>(A[0], w_u, aoff, nchf, kl, d);
    store_x_chunk<TR, KC, KCP, NT, XPT>(xs[0], xr[0], tid);
    __syncthreads();
    mfma_chunk<MV, NB, KS, KCP>(acc, A[0], xs[0], lane, kl);
  }

  // epilogue: softmax state per projected row
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float z[MV * 4];
    int vi[MV * 4];
    bool ok[MV * 4];
#pragma unroll
    for (int mv = 0; mv < MV; ++mv)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int v = vw + mv * 16 + (lane >> 4) * 4 + e;
        z[mv * 4 + e] = acc[mv][nb][e];
        vi[mv * 4 + e] = v;
        ok[mv * 4 + e] = v < ve;
      }
    Soft st = soft_from_values(z, vi, ok);
    st = soft_merge(st, soft_shfl_xor(st, 16));
    st = soft_merge(st, soft_shfl_xor(st, 32));
    if (lane < 16) red[wid][nb * 16 + lane] = soft_pack(st);
  }
  __syncthreads();
  for (int t = tid; t < TR; t += NT) {
    const int r = r0 + t;
    if (r < R) {
      Soft s = soft_unpack(red[0][t]);
#pragma unroll
      for (int w = 1; w < NW; ++w) s = soft_merge(s, soft_unpack(red[w][t]));
      partials[(long long)r * nvt + vt] = soft_pack(s);
    }
  }
}

// ------------------------------------------- K1 projection bf16, 32x32 --

// Large row counts (compute-bound): v_mfma_f32_32x32x16_bf16, which keeps the
// matrix pipe busy from a single wave per SIMD (the 16x16 form cannot).
// Workgroup tile: TR = 32*NB projected rows x 32*MV*NW vocabulary rows. As in
// k_proj_bf16, each wave owns its W_U rows (A operand, straight to
// registers: lane l holds row l & 31, k elements 8*(l >> 5) .. +8 of each
// 16-wide k-step) and the hidden rows go through an NSTG-stage LDS ring.
// Accumulator register q of lane l holds vocabulary row
// 8*(q >> 2) + 4*(l >> 5) + (q & 3) of its 32-row block and projected row
// l & 31.
template <int MV, int KS, bool GUARD>
__device__ __forceinline__ void load_a_chunk32(u32x4 (&dst)[KS][MV], const uint16_t* __restrict__ w_u,
                                               const long long (&aoff)[MV], int c, int kl, int d) {
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int k = (c * KS + s) * 16;
#pragma unroll
    for (int mv = 0; mv < MV; ++mv) {
      const u32x4* src = reinterpret_cast<const u32x4*>(w_u + aoff[mv] + k);
      if (GUARD)
        dst[s][mv] = k + kl < d ? *src : u32x4{0u, 0u, 0u, 0u};
      else
        dst[s][mv] = *src;
    }
  }
}

template <int MV, int NB, int KS, int KCP>
__device__ __forceinline__ void mfma_chunk32(f32x16 (&acc)[MV][NB], const u32x4 (&a)[KS][MV],
                                             const uint16_t (*xsb)[KCP], int lane, int kl) {
  u32x4 bq[2][NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
    bq[0][nb] = *reinterpret_cast<const u32x4*>(&xsb[nb * 32 + (lane & 31)][kl]);
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    if (s + 1 < KS) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        bq[(s + 1) & 1][nb] = *reinterpret_cast<const u32x4*>(&xsb[nb * 32 + (lane & 31)][(s + 1) * 16 + kl]);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const bf16x8 bv = __builtin_bit_cast(bf16x8, bq[s & 1][nb]);
#pragma unroll
      for (int mv = 0; mv < MV; ++mv)
        acc[mv][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[s][mv]), bv, acc[mv][nb],
                                                               0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <int NW, int MV, int NB, int KC, int NSTG, int MAP = 0>
__global__ __launch_bounds__(NW * 64) void k_proj_bf16_m32(
    const uint16_t* __restrict__ hidden, const uint16_t* __restrict__ w_u, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ n_ptr, float4* __restrict__ partials, int K, int B, int L, int d, int V,
    int nvt, int nrt, int split_rows) {
  constexpr int TR = 32 * NB;
  static_assert(KC % 16 == 0 && NSTG >= 2, "chunk of whole k-steps, at least double buffering");
  constexpr int KS = KC / 16;
  constexpr int KCP = KC + 8;
  constexpr int NT = NW * 64;
  constexpr int XP = TR * (KC / 8);
  constexpr int XPT = (XP + NT - 1) / NT;

  __shared__ __attribute__((aligned(16))) uint16_t xs[NSTG][TR][KCP];
  __shared__ long long xoff[TR];
  __shared__ float4 red[NW][TR];

  int rt, vt;
  if (MAP == 0) {
    if (!map_job(blockIdx.x, nvt, nrt, split_rows, rt, vt)) return;
  } else {
    const int bid = blockIdx.x;
    if (bid >= nvt * nrt) return;
    if (MAP == 1) { rt = bid / nvt; vt = bid - rt * nvt; }      // row tiles outer
    else { vt = bid / nrt; rt = bid - vt * nrt; }               // vocabulary tiles outer
  }
  const int R = *n_ptr * K;
  const int r0 = rt * TR;
  if (r0 >= R) return;
  const int vb = (int)((long long)vt * V / nvt);
  const int ve = (int)((long long)(vt + 1) * V / nvt);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;

  for (int t = tid; t < TR; t += NT) {
    const int r = r0 + t < R ? r0 + t : r0;   // padding rows re-read a real row; discarded at the end
    const int p = r / K, l = r - p * K;
    const int pos = rows[p];
    const int b = pos / L, i = pos - b * L;
    xoff[t] = (((long long)l * B + b) * L + i) * (long long)d;
  }
  __syncthreads();

  const int vw = vb + wid * 32 * MV;
  const int kl = (lane >> 5) * 8;
  long long aoff[MV];
#pragma unroll
  for (int mv = 0; mv < MV; ++mv) aoff[mv] = (long long)min(vw + mv * 32 + (lane & 31), ve - 1) * d + kl;

  f32x16 acc[MV][NB];
#pragma unroll
  for (int mv = 0; mv < MV; ++mv)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[mv][nb][q] = 0.f;

  u32x4 A[NSTG][KS][MV];
  u32x4 xr[NSTG][XPT];
  const int nchf = d / KC;

#define RPD_LOAD_CHUNK32(buf, chunk)                                                \
  do {                                                                              \
    load_x_chunk<TR, KC, NT, XPT, false>(xr[buf], hidden, xoff, (chunk), tid, d);   \
    load_a_chunk32<MV, KS, false>(A[buf], w_u, aoff, (chunk), kl, d);               \
  } while (0)

  if (nchf > 0) {
#pragma unroll
    for (int j = 0; j < NSTG - 1; ++j) RPD_LOAD_CHUNK32(j, min(j, nchf - 1));
    store_x_chunk<TR, KC, KCP, NT, XPT>(xs[0], xr[0], tid);
    __syncthreads();
    const int nmain = (nchf / NSTG) * NSTG;
    for (int c0 = 0; c0 < nmain; c0 += NSTG) {
#pragma unroll
      for (int j = 0; j < NSTG; ++j) {
        RPD_LOAD_CHUNK32((j + NSTG - 1) % NSTG, min(c0 + j + NSTG - 1, nchf - 1));
        __builtin_amdgcn_sched_barrier(0);
        mfma_chunk32<MV, NB, KS, KCP>(acc, A[j], xs[j], lane, kl);
        store_x_chunk<TR, KC, KCP, NT, XPT>(xs[(j + 1) % NSTG], xr[(j + 1) % NSTG], tid);
        __syncthreads();
      }
    }
    const int rem = nchf - nmain;
#pragma unroll
    for (int j = 0; j < NSTG - 1; ++j) {
      if (j < rem) {
        mfma_chunk32<MV, NB, KS, KCP>(acc, A[j], xs[j], lane, kl);
        if (j + 1 < rem) store_x_chunk<TR, KC, KCP, NT, XPT>(xs[j + 1], xr[j + 1], tid);
        __syncthreads();
      }
    }
  }
#undef RPD_LOAD_CHUNK32
  if (d % KC != 0) {
    load_x_chunk<TR, KC, NT, XPT, true>(xr[0], hidden, xoff, nchf, tid, d);
    load_a_chunk32<MV, KS, true>(A[0], w_u, aoff, nchf, kl, d);
    store_x_chunk<TR, KC, KCP, NT, XPT>(xs[0], xr[0], tid);
    __syncthreads();
    mfma_chunk32<MV, NB, KS, KCP>(acc, A[0], xs[0], lane, kl);
  }

#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float z[MV * 16];
    int vi[MV * 16];
    bool ok[MV * 16];
#pragma unroll
    for (int mv = 0; mv < MV; ++mv)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int v = vw + mv * 32 + (q >> 2) * 8 + (lane >> 5) * 4 + (q & 3);
        z[mv * 16 + q] = acc[mv][nb][q];
        vi[mv * 16 + q] = v;
        ok[mv * 16 + q] = v < ve;
      }
    Soft st = soft_from_values(z, vi, ok);
    st = soft_merge(st, soft_shfl_xor(st, 32));
    if (lane < 32) red[wid][nb * 32 + lane] = soft_pack(st);
  }
  __syncthreads();
  for (int t = tid; t < TR; t += NT) {
    const int r = r0 + t;
    if (r < R) {
      Soft sres = soft_unpack(red[0][t]);
#pragma unroll
      for (int w = 1; w < NW; ++w) sres = soft_merge(sres, soft_unpack(red[w][t]));
      partials[(long long)r * nvt + vt] = soft_pack(sres);
    }
  }
}

// -------------------------------- K1 projection bf16, 256 x 256 tiles --

// Compute-bound row counts: a GEMM tile of 256 vocabulary rows x 256
// projected rows with both operands staged in LDS by direct global->LDS
// loads (global_load_lds_dwordx4: each lane's 16 bytes land at the wave's
// LDS base + 16 * lane), so no registers hold loads in flight and three
// 32-wide k-chunks can be in flight per workgroup in a four-stage ring. A
// load instruction covers 16 rows x 64 bytes; the 16-byte pieces of row r
// are stored XOR-swizzled by (r >> 2) & 3 (chosen through which global
// piece each lane fetches), which makes the MFMA fragment reads free of
// bank conflicts. Four waves in a 2 x 2 layout each compute 128 x 128 with
// v_mfma_f32_32x32x16_bf16 (256 accumulators per lane, one wave per SIMD).
namespace big {
constexpr int TV = 256, TR = 256, KC = 32, NSTG = 4;
constexpr int LOADS = 8;   // direct loads per wave per chunk: 4 for W_U rows, 4 for hidden rows

// One direct global->LDS load of 16 bytes per lane (lane l writes LDS bytes
// [lds + 16 l, +16)). Issued through inline asm so that the compiler's
// wait-count insertion does not treat it as an LDS store that every later
// LDS read must wait for; the kernel orders these loads with explicit
// vmcnt waits and barriers instead. No compiler-visible vector-memory load
// may be in flight where those explicit waits are relied on.
__device__ __forceinline__ void dma16(const uint16_t* gptr, const void* lds) {
  const uint32_t lds_addr =
      __builtin_amdgcn_readfirstlane((uint32_t)(size_t)(__attribute__((address_space(3))) const void*)lds);
  asm volatile(
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, off"
      :
      : "v"(gptr), "s"(lds_addr)
      : "memory", "m0");
}

__device__ __forceinline__ void vmcnt_wait_loads(int outstanding_chunks) {
  // s_waitcnt vmcnt(outstanding_chunks * LOADS); expcnt and lgkmcnt left unconstrained
  switch (outstanding_chunks) {
    case 0: __builtin_amdgcn_s_waitcnt(0x0F70 | 0); break;
    case 1: __builtin_amdgcn_s_waitcnt(0x0F70 | LOADS); break;
    case 2: __builtin_amdgcn_s_waitcnt((0x0F70 | ((2 * LOADS) & 15)) | (((2 * LOADS) >> 4) << 14)); break;
    default: __builtin_amdgcn_s_waitcnt(0); break;
  }
}
}  // namespace big

__global__ __launch_bounds__(256) void k_proj_bf16_big(
    const uint16_t* __restrict__ hidden, const uint16_t* __restrict__ w_u, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ n_ptr, float4* __restrict__ partials, int K, int B, int L, int d, int V,
    int nvt, int nrt, int split_rows) {
  using namespace big;
  static_assert(NSTG == 4 && 2 * LOADS < 64, "wait counts below assume three chunks in flight");
  // one LDS object per ring stage: the compiler then knows that reads of the
  // stage being multiplied do not alias the direct loads filling another
  // stage, and does not wait for those loads before the reads
  __shared__ __attribute__((aligned(16))) uint16_t sa0[TV][KC], sa1[TV][KC], sa2[TV][KC], sa3[TV][KC];
  __shared__ __attribute__((aligned(16))) uint16_t sb0[TR][KC], sb1[TR][KC], sb2[TR][KC], sb3[TR][KC];
  __shared__ float4 red[2][TR];
#define RPD_SA(S) ((S) == 0 ? sa0 : (S) == 1 ? sa1 : (S) == 2 ? sa2 : sa3)
#define RPD_SB(S) ((S) == 0 ? sb0 : (S) == 1 ? sb1 : (S) == 2 ? sb2 : sb3)

  int rt, vt;
  if (!map_job(blockIdx.x, nvt, nrt, split_rows, rt, vt)) return;
  const int R = *n_ptr * K;
  const int r0 = rt * TR;
  if (r0 >= R) return;
  const int vb = (int)((long long)vt * V / nvt);
  const int ve = (int)((long long)(vt + 1) * V / nvt);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wv = wid & 1, wr = wid >> 1;

  // direct-load sources: instruction j of this wave covers tile rows
  // 64*wid + 16*j .. +16; lane l fills LDS piece (l & 3) of row (l >> 2) with
  // the global piece (l & 3) ^ swizzle(row)
  long long ga[4], gb[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int tr = 64 * wid + 16 * j + (lane >> 2);
    const int piece = (lane & 3) ^ ((tr >> 2) & 3);
    ga[j] = (long long)min(vb + tr, ve - 1) * d + piece * 8;
    const int r = r0 + tr < R ? r0 + tr : r0;   // padding rows re-read a real row; discarded at the end
    const int p = r / K, l = r - p * K;
    const int pos = rows[p];
    const int b = pos / L, i = pos - b * L;
    gb[j] = (((long long)l * B + b) * L + i) * (long long)d + piece * 8;
  }
  // fragment reads: lane reads row base + (lane & 31), logical piece 2s + (lane >> 5)
  const int swl = ((lane & 31) >> 2) & 3;
  const int fcol0 = 8 * ((0 + (lane >> 5)) ^ swl), fcol1 = 8 * ((2 + (lane >> 5)) ^ swl);

  f32x16 acc[4][4];
#pragma unroll
  for (int mv = 0; mv < 4; ++mv)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[mv][nb][q] = 0.f;

#define RPD_BIG_ISSUE(chunk, stage)                                                                      \
  do {                                                                                                   \
    _Pragma("unroll") for (int u_ = 0; u_ < 4; ++u_) {                                                  \
      dma16(w_u + ga[u_] + (chunk) * KC, &RPD_SA(stage)[64 * wid + 16 * u_][0]);                       \
      dma16(hidden + gb[u_] + (chunk) * KC, &RPD_SB(stage)[64 * wid + 16 * u_][0]);                    \
    }                                                                                                    \
  } while (0)
#define RPD_BIG_COMPUTE(stage)                                                                            \
  do {                                                                                                   \
    const uint16_t(*pa_)[KC] = RPD_SA(stage);                                                            \
    const uint16_t(*pb_)[KC] = RPD_SB(stage);                                                            \
    _Pragma("unroll") for (int s_ = 0; s_ < 2; ++s_) {                                                  \
      const int fc_ = s_ ? fcol1 : fcol0;                                                                \
      u32x4 fa_[4], fb_[4];                                                                              \
      _Pragma("unroll") for (int m = 0; m < 4; ++m) {                                                   \
        fa_[m] = *reinterpret_cast<const u32x4*>(&pa_[128 * wv + 32 * m + (lane & 31)][fc_]);           \
        fb_[m] = *reinterpret_cast<const u32x4*>(&pb_[128 * wr + 32 * m + (lane & 31)][fc_]);           \
      }                                                                                                  \
      _Pragma("unroll") for (int mv = 0; mv < 4; ++mv)                                                  \
      _Pragma("unroll") for (int nb = 0; nb < 4; ++nb)                                                  \
        acc[mv][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa_[mv]),       \
                                                               __builtin_bit_cast(bf16x8, fb_[nb]),       \
                                                               acc[mv][nb], 0, 0, 0);                    \
    }                                                                                                    \
  } while (0)

  const int nchf = d / KC;
  if (nchf > 0) {
#pragma unroll
    for (int j = 0; j < NSTG - 1; ++j) RPD_BIG_ISSUE(min(j, nchf - 1), j);
    vmcnt_wait_loads(NSTG - 2);
    __syncthreads();
    // unrolled by NSTG so that every stage is a compile-time choice; a stage
    // refilled in a trip was consumed in the previous one (all waves passed
    // the barrier since); chunks past the end repeat the last one
    const int nmain = (nchf / NSTG) * NSTG;
    for (int c0 = 0; c0 < nmain; c0 += NSTG) {
#pragma unroll
      for (int j = 0; j < NSTG; ++j) {
        RPD_BIG_ISSUE(min(c0 + j + NSTG - 1, nchf - 1), (j + NSTG - 1) % NSTG);
        RPD_BIG_COMPUTE(j);
        vmcnt_wait_loads(NSTG - 2);   // chunk c+1 has landed (this wave's share)
        __syncthreads();              // ... and every wave's share
      }
    }
    const int rem = nchf - nmain;   // < NSTG chunks left, already in stages 0 .. rem-1
#pragma unroll
    for (int j = 0; j < NSTG - 1; ++j)
      if (j < rem) {
        RPD_BIG_COMPUTE(j);
        vmcnt_wait_loads(0);
        __syncthreads();
      }
    vmcnt_wait_loads(0);
    __syncthreads();
  }
  if (d % KC != 0) {   // partial last chunk through registers, zero-filled past d
    const int k0 = nchf * KC;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int tr = 64 * wid + 16 * j + (lane >> 2);
      const int piece = (lane & 3) ^ ((tr >> 2) & 3);
      const bool in = k0 + piece * 8 < d;
      const u32x4 va = in ? *reinterpret_cast<const u32x4*>(w_u + ga[j] + k0) : u32x4{0u, 0u, 0u, 0u};
      const u32x4 vbv = in ? *reinterpret_cast<const u32x4*>(hidden + gb[j] + k0) : u32x4{0u, 0u, 0u, 0u};
      *reinterpret_cast<u32x4*>(&sa0[tr][(lane & 3) * 8]) = va;
      *reinterpret_cast<u32x4*>(&sb0[tr][(lane & 3) * 8]) = vbv;
    }
    __syncthreads();
    RPD_BIG_COMPUTE(0);
  }
#undef RPD_BIG_ISSUE
#undef RPD_BIG_COMPUTE
#undef RPD_SA
#undef RPD_SB

  // epilogue: lane holds projected row 128*wr + 32*nb + (lane & 31) against
  // vocabulary rows 128*wv + 32*mv + 8*(q >> 2) + 4*(lane >> 5) + (q & 3)
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) {
    Soft sst = soft_empty();
#pragma unroll
    for (int mv = 0; mv < 4; ++mv) {
      float z[16];
      int vi[16];
      bool ok[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int v = vb + 128 * wv + 32 * mv + (q >> 2) * 8 + (lane >> 5) * 4 + (q & 3);
        z[q] = acc[mv][nb][q];
        vi[q] = v;
        ok[q] = v < ve;
      }
      sst = soft_merge(sst, soft_from_values(z, vi, ok));
    }
    sst = soft_merge(sst, soft_shfl_xor(sst, 32));
    if (lane < 32) red[wv][128 * wr + 32 * nb + lane] = soft_pack(sst);
  }
  __syncthreads();
  {
    const int r = r0 + tid;   // one projected row per thread (TR == 256 threads)
    if (r < R) {
      const Soft sres = soft_merge(soft_unpack(red[0][tid]), soft_unpack(red[1][tid]));
      partials[(long long)r * nvt + vt] = soft_pack(sres);
    }
  }
}

// Small row counts (TR = 16*NB >= all projected rows): no LDS staging and no
// barrier in the main loop. Each wave owns 16*MV consecutive W_U rows of the
// workgroup's vocabulary range and streams them through a DEPTH-deep register
// pipeline with non-temporal loads (W_U is read exactly once per call); the
// hidden rows, at most 16*NB of them, are read by every wave straight from L2
// in the MFMA B-operand layout. Rows past the last projected row read row 0
// again and are discarded in the epilogue.
template <int NW, int MV, int NB, int DEPTH>
__global__ __launch_bounds__(NW * 64) void k_proj_bf16_stream(
    const uint16_t* __restrict__ hidden, const uint16_t* __restrict__ w_u, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ n_ptr, float4* __restrict__ partials, int K, int B, int L, int d, int V, int nvt) {
  constexpr int TR = 16 * NB;
  constexpr int NS = DEPTH + 1;
  __shared__ float4 red[NW][TR];

  const int R = *n_ptr * K;
  if (R <= 0) return;
  // workgroup ids are dispatched round-robin over the XCDs: give each XCD a
  // contiguous range of vocabulary tiles
  const int vt = (int)(((long long)(blockIdx.x & 7) * nvt) / 8) + (blockIdx.x >> 3);
  if (vt >= (int)(((long long)((blockIdx.x & 7) + 1) * nvt) / 8)) return;
  const int vb = (int)((long long)vt * V / nvt);
  const int ve = (int)((long long)(vt + 1) * V / nvt);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int vw = vb + wid * 16 * MV;
  const int kl = (lane >> 4) * 8;

  long long aoff[MV];
#pragma unroll
  for (int mv = 0; mv < MV; ++mv) aoff[mv] = (long long)min(vw + mv * 16 + (lane & 15), ve - 1) * d + kl;
  long long boff[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    int r = nb * 16 + (lane & 15);
    r = r < R ? r : 0;
    const int p = r / K, l = r - p * K;
    const int pos = rows[p];
    const int b = pos / L, i = pos - b * L;
    boff[nb] = (((long long)l * B + b) * L + i) * (long long)d + kl;
  }

  f32x4 acc[MV][NB];
#pragma unroll
  for (int mv = 0; mv < MV; ++mv)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mv][nb] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 A[NS][MV], X[NS][NB];
  const u32x4 z4 = {0u, 0u, 0u, 0u};

  // full 32-wide k-steps: every lane in bounds, loads are unconditional
#define RPD_LOAD_STEP(buf, step)                                                                  \
  do {                                                                                            \
    const int k_ = (step) * 32;                                                                   \
    _Pragma("unroll") for (int mv = 0; mv < MV; ++mv) A[buf][mv] =                               \
        __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(w_u + aoff[mv] + k_));          \
    _Pragma("unroll") for (int nb = 0; nb < NB; ++nb) X[buf][nb] =                               \
        *reinterpret_cast<const u32x4*>(hidden + boff[nb] + k_);                                  \
  } while (0)
#define RPD_MFMA_STEP(buf)                                                                        \
  do {                                                                                            \
    _Pragma("unroll") for (int nb = 0; nb < NB; ++nb)                                            \
    _Pragma("unroll") for (int mv = 0; mv < MV; ++mv)                                            \
      acc[mv][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, A[buf][mv]), \
                                                             __builtin_bit_cast(bf16x8, X[buf][nb]), \
                                                             acc[mv][nb], 0, 0, 0);               \
  } while (0)

  const int nkf = d / 32;
  if (nkf > 0) {
#pragma unroll
    for (int j = 0; j < DEPTH; ++j) RPD_LOAD_STEP(j, min(j, nkf - 1));
    const int nmain = (nkf / NS) * NS;
    for (int s0 = 0; s0 < nmain; s0 += NS) {
#pragma unroll
      for (int j = 0; j < NS; ++j) {
        // steps past the end re-load the last step (discarded); the
        // scheduling barrier keeps these loads ahead of this step's MFMAs
        RPD_LOAD_STEP((j + DEPTH) % NS, min(s0 + j + DEPTH, nkf - 1));
        __builtin_amdgcn_sched_barrier(0);
        RPD_MFMA_STEP(j);
      }
    }
    // the remaining (< NS) steps were loaded by the last group into buffers 0..
    const int rem = nkf - nmain;
#pragma unroll
    for (int j = 0; j < NS - 1; ++j)
      if (j < rem) RPD_MFMA_STEP(j);
  }
  if (d % 32 != 0) {   // partial last k-step (d is a multiple of 8)
    const int k_ = nkf * 32;
    const bool in_ = k_ + kl < d;
#pragma unroll
    for (int mv = 0; mv < MV; ++mv)
      A[0][mv] = in_ ? *reinterpret_cast<const u32x4*>(w_u + aoff[mv] + k_) : z4;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) X[0][nb] = in_ ? *reinterpret_cast<const u32x4*>(hidden + boff[nb] + k_) : z4;
    RPD_MFMA_STEP(0);
  }
#undef RPD_MFMA_STEP
#undef RPD_LOAD_STEP

#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float z[MV * 4];
    int vi[MV * 4];
    bool ok[MV * 4];
#pragma unroll
    for (int mv = 0; mv < MV; ++mv)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int v = vw + mv * 16 + (lane >> 4) * 4 + e;
        z[mv * 4 + e] = acc[mv][nb][e];
        vi[mv * 4 + e] = v;
        ok[mv * 4 + e] = v < ve;
      }
    Soft st = soft_from_values(z, vi, ok);
    st = soft_merge(st, soft_shfl_xor(st, 16));
    st = soft_merge(st, soft_shfl_xor(st, 32));
    if (lane < 16) red[wid][nb * 16 + lane] = soft_pack(st);
  }
  __syncthreads();
  for (int t = tid; t < TR; t += NW * 64) {
    if (t < R) {
      Soft sres = soft_unpack(red[0][t]);
#pragma unroll
      for (int w = 1; w < NW; ++w) sres = soft_merge(sres, soft_unpack(red[w][t]));
      partials[(long long)t * nvt + vt] = soft_pack(sres);
    }
  }
}

// ------------------------------------------------------ K1 projection f32 --

// fp32 inputs: 64 vocabulary rows (one per lane) x 16 projected rows (four
// per wave) per workgroup, fp32 FMA on the vector ALU through LDS tiles.
__global__ __launch_bounds__(256) void k_proj_f32(const float* __restrict__ hidden, const float* __restrict__ w_u,
                                                  const int32_t* __restrict__ rows,
                                                  const int32_t* __restrict__ n_ptr, float4* __restrict__ partials,
                                                  int K, int B, int L, int d, int V, int nvt) {
  __shared__ float ws[64][33];
  __shared__ float xsm[16][33];
  __shared__ long long xoff[16];
  const int vt = blockIdx.x % nvt, rt = blockIdx.x / nvt;
  const int R = *n_ptr * K;
  const int r0 = rt * 16;
  if (r0 >= R) return;
  const int vb = (int)((long long)vt * V / nvt);
  const int ve = (int)((long long)(vt + 1) * V / nvt);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  if (tid < 16) {
    const int r = r0 + tid;
    long long off = -1;
    if (r < R) {
      const int p = r / K, l = r - p * K;
      const int pos = rows[p];
      const int b = pos / L, i = pos - b * L;
      off = (((long long)l * B + b) * L + i) * (long long)d;
    }
    xoff[tid] = off;
  }
  __syncthreads();
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < d; k0 += 32) {
    for (int q = tid; q < 64 * 32; q += 256) {
      const int row = q >> 5, kk = q & 31;
      const int v = vb + row;
      ws[row][kk] = (v < ve && k0 + kk < d) ? w_u[(long long)v * d + k0 + kk] : 0.f;
    }
    for (int q = tid; q < 16 * 32; q += 256) {
      const int row = q >> 5, kk = q & 31;
      const long long off = xoff[row];
      xsm[row][kk] = (off >= 0 && k0 + kk < d) ? hidden[off + k0 + kk] : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < 32; ++kk) {
      const float wv = ws[lane][kk];
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[j] = fmaf(wv, xsm[wid * 4 + j][kk], acc[j]);
    }
    __syncthreads();
  }
  const int v = vb + lane;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float z[1] = {acc[j]};
    int vi[1] = {v};
    bool ok[1] = {v < ve};
    Soft st = soft_from_values(z, vi, ok);
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) st = soft_merge(st, soft_shfl_xor(st, m));
    const int r = r0 + wid * 4 + j;
    if (lane == 0 && r < R) partials[(long long)r * nvt + vt] = soft_pack(st);
  }
}

// ------------------------------------------------------ scoring (Eq. 2-5) --

__device__ __forceinline__ float stability_score(int k_i, float r_i, int k_max, float w) {
  return fmaf(-w, r_i, (float)min(k_i, k_max));
}

__device__ __forceinline__ unsigned route_flags(float c, float s, float theta_h, float theta_c, float theta_s) {
  const bool high = c >= theta_h;
  const bool stab = (c >= theta_c) && (c < theta_h) && (s >= theta_s);
  return (high || stab ? kFlagCandidate : 0u) | (high ? kFlagHigh : 0u) | (stab ? kFlagStable : 0u);
}

struct ScoreArgs {
  int K, B, L;
  float theta_h, theta_c, theta_s, w;
  int k_max;
  int32_t* token;
  float* entropy;
  float* confidence;
  int32_t* persistence;
  float* drop;
  float* stability;
  uint8_t* flags;
  int32_t* layer_argmax;
  float* layer_conf;
  float* layer_entropy;
};

// One workgroup of four waves per masked position. Wave w merges the
// vocab-tile states of layers w, w+4, ...: each lane folds tiles lane,
// lane+64, ... in tile order (loads batched four at a time), then a fixed
// xor butterfly combines the lanes. Wave 0 then evaluates persistence, drop
// and stability with one lane per layer.
constexpr int kReduceWaves = 4;

__global__ __launch_bounds__(64 * kReduceWaves) void k_reduce_score(const float4* __restrict__ partials,
                                                                     const int32_t* __restrict__ rows,
                                                                     const int32_t* __restrict__ n_ptr, int nvt,
                                                                     ScoreArgs a) {
  __shared__ int ly[64];
  __shared__ float lc[64], lh[64];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int p = blockIdx.x;
  if (p >= *n_ptr) return;
  const int pos = rows[p];
  const int b = pos / a.L, i = pos - b * a.L;
  const float4 empty = soft_pack(soft_empty());
  for (int l = wid; l < a.K; l += kReduceWaves) {
    const float4* src = partials + ((long long)p * a.K + l) * nvt;
    Soft s = soft_empty();
    for (int t0 = lane; t0 < nvt; t0 += 64 * 4) {
      float4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = (t0 + 64 * u < nvt) ? src[t0 + 64 * u] : empty;
#pragma unroll
      for (int u = 0; u < 4; ++u) s = soft_merge(s, soft_unpack(v[u]));
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) s = soft_merge(s, soft_shfl_xor(s, m));
    if (lane == 0) {
      const float h = fmaxf(logf(s.S) - s.T / s.S, 0.0f);
      ly[l] = (s.idx == INT_MAX) ? -1 : s.idx;
      lc[l] = 1.0f / s.S;
      lh[l] = (s.S != s.S) ? s.S : h;   // keep NaN visible
    }
  }
  __syncthreads();
  if (wid != 0) return;
  const int my_y = lane < a.K ? ly[lane] : -1;
  const float my_c = lane < a.K ? lc[lane] : 0.f;
  const float my_h = lane < a.K ? lh[lane] : 0.f;
  const int yK = ly[a.K - 1];
  const float cK = lc[a.K - 1];
  const float hK = lh[a.K - 1];
  // Eq. 2: agreement suffix ending at the final layer
  const unsigned long long dis = __ballot(lane < a.K && my_y != yK);
  const int last_dis = dis ? 63 - __clzll(dis) : -1;
  const int k_i = a.K - 1 - last_dis;
  // Eq. 3: inside the suffix the final token is each layer's argmax, so its
  // probability there is that layer's top probability
  float pk = (lane >= a.K - k_i && lane < a.K) ? my_c : -INFINITY;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) pk = fmaxf(pk, __shfl_xor(pk, m));
  const float r_i = pk - cK;
  const float s_i = stability_score(k_i, r_i, a.k_max, a.w);
  const unsigned fl = route_flags(cK, s_i, a.theta_h, a.theta_c, a.theta_s);
  const long long o = (long long)b * a.L + i;
  if (lane == 0) {
    a.token[o] = yK;
    a.entropy[o] = hK;
    a.confidence[o] = cK;
    a.persistence[o] = k_i;
    a.drop[o] = r_i;
    a.stability[o] = s_i;
    a.flags[o] = (uint8_t)fl;
  }
  if (a.layer_argmax && lane < a.K) {
    const long long ol = ((long long)lane * a.B + b) * a.L + i;
    a.layer_argmax[ol] = my_y;
    a.layer_conf[ol] = my_c;
    a.layer_entropy[ol] = my_h;
  }
}

// Scoring from caller-supplied per-layer statistics, one thread per canvas
// position (same formulas as k_reduce_score, evaluated sequentially).
__global__ __launch_bounds__(256) void k_gate_score(const uint8_t* __restrict__ mask,
                                                     const int32_t* __restrict__ l_y,
                                                     const float* __restrict__ l_c,
                                                     const float* __restrict__ l_h, ScoreArgs a) {
  const long long BL = (long long)a.B * a.L;
  const long long o = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (o >= BL || mask[o] == 0) return;
  const int yK = l_y[(long long)(a.K - 1) * BL + o];
  const float cK = l_c[(long long)(a.K - 1) * BL + o];
  const float hK = l_h[(long long)(a.K - 1) * BL + o];
  int k_i = 1;
  float pk = cK;
  for (int l = a.K - 2; l >= 0; --l) {
    if (l_y[(long long)l * BL + o] != yK) break;
    ++k_i;
    pk = fmaxf(pk, l_c[(long long)l * BL + o]);
  }
  const float r_i = pk - cK;
  const float s_i = stability_score(k_i, r_i, a.k_max, a.w);
  a.token[o] = yK;
  a.entropy[o] = hK;
  a.confidence[o] = cK;
  a.persistence[o] = k_i;
  a.drop[o] = r_i;
  a.stability[o] = s_i;
  a.flags[o] = (uint8_t)route_flags(cK, s_i, a.theta_h, a.theta_c, a.theta_s);
}

// --------------------------------------------------- commitment (Sec. 3.2) --

constexpr int kCommitThreads = 1024;

// exclusive prefix sum over the workgroup in thread order (fixed tree order);
// `total` receives the sum of all values
template <typename T>
__device__ __forceinline__ T block_exclusive_scan(T v, T* sh, T& total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  T x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const T y = __shfl_up(x, o);
    if (lane >= o) x = x + y;
  }
  if (lane == 63) sh[wid] = x;
  __syncthreads();
  if (wid == 0) {
    T s = (lane < nw) ? sh[lane] : T(0);
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const T y = __shfl_up(s, o);
      if (lane >= o) s = s + y;
    }
    if (lane < nw) sh[32 + lane] = s;   // inclusive over waves
  }
  __syncthreads();
  const T wave_before = (wid == 0) ? T(0) : sh[32 + wid - 1];
  total = sh[32 + nw - 1];
  const T res = wave_before + x - v;
  __syncthreads();
  return res;
}

struct CommitArgs {
  int B, L;
  float beta;
  int window;
  uint8_t* commit;
  int32_t* token;
  float* entropy;
  float* confidence;
  int32_t* persistence;
  float* drop;
  float* stability;
  uint8_t* flags;
  float* upstream_entropy;
  int32_t* n_commit;
};

// One workgroup per sequence. N_i = entropy summed over earlier masked
// non-candidates; a candidate is committed iff N_i <= beta, which is exactly
// the left-to-right construction of the paper (every earlier candidate of an
// accepted position is accepted, so the positions left out before it are the
// non-candidates; a rejected candidate's sum only grows). E_i (reported) is
// the entropy over earlier masked positions not committed. Without any
// commit, the most confident of the first `window` masked positions is
// committed (lowest index on ties; NaN confidences never win).
__global__ __launch_bounds__(kCommitThreads) void k_commit(const uint8_t* __restrict__ mask, CommitArgs a) {
  __shared__ float shf[64];
  __shared__ int shi[64];
  __shared__ float red_c[16];
  __shared__ int red_i[16];
  const int b = blockIdx.x;
  const long long base = (long long)b * a.L;
  float carryN = 0.f, carryE = 0.f;
  int carryM = 0, ncommit = 0;
  float best_c = -INFINITY;
  int best_i = INT_MAX;
  for (int c0 = 0; c0 < a.L; c0 += blockDim.x) {
    const int i = c0 + threadIdx.x;
    const bool in = i < a.L;
    const bool masked = in && mask[base + i] != 0;
    const unsigned fl = masked ? a.flags[base + i] : 0u;
    const bool cand = (fl & kFlagCandidate) != 0;
    const float H = masked ? a.entropy[base + i] : 0.f;
    float totN, totE;
    int totM;
    const float N_i = carryN + block_exclusive_scan<float>((masked && !cand) ? H : 0.f, shf, totN);
    const bool com = masked && cand && (N_i <= a.beta);
    const float E_i = carryE + block_exclusive_scan<float>((masked && !com) ? H : 0.f, shf, totE);
    const int rank = carryM + block_exclusive_scan<int>(masked ? 1 : 0, shi, totM);
    int ncom_chunk;
    (void)block_exclusive_scan<int>(com ? 1 : 0, shi, ncom_chunk);
    if (in) {
      const long long o = base + i;
      if (masked) {
        a.commit[o] = com ? 1 : 0;
        a.flags[o] = (uint8_t)(fl | (com ? kFlagCommitted : 0u));
        a.upstream_entropy[o] = E_i;
        if (rank < a.window) {
          float cv = a.confidence[o];
          cv = (cv != cv) ? -INFINITY : cv;
          if (cv > best_c || (cv == best_c && i < best_i)) {
            best_c = cv;
            best_i = i;
          }
        }
      } else {
        a.commit[o] = 0;
        a.token[o] = -1;
        a.entropy[o] = 0.f;
        a.confidence[o] = 0.f;
        a.persistence[o] = 0;
        a.drop[o] = 0.f;
        a.stability[o] = 0.f;
        a.flags[o] = 0;
        a.upstream_entropy[o] = 0.f;
      }
    }
    carryN += totN;
    carryE += totE;
    carryM += totM;
    ncommit += ncom_chunk;
  }
  if (ncommit == 0 && carryM > 0) {
    // workgroup argmax of (confidence, -index) over the window
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const float oc = __shfl_xor(best_c, m);
      const int oi = __shfl_xor(best_i, m);
      if (oc > best_c || (oc == best_c && oi < best_i)) {
        best_c = oc;
        best_i = oi;
      }
    }
    if (lane == 0) {
      red_c[wid] = best_c;
      red_i[wid] = best_i;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      float bc = red_c[0];
      int bi = red_i[0];
      for (int w = 1; w < nw; ++w)
        if (red_c[w] > bc || (red_c[w] == bc && red_i[w] < bi)) {
          bc = red_c[w];
          bi = red_i[w];
        }
      if (bi != INT_MAX) {   // the window always holds a masked position here
        const long long o = base + bi;
        a.commit[o] = 1;
        a.flags[o] = (uint8_t)(a.flags[o] | kFlagCommitted | kFlagFallback);
        ncommit = 1;
      }
    }
  }
  if (threadIdx.x == 0) a.n_commit[b] = ncommit;
}

ScoreArgs score_args(const Launch& a) {
  ScoreArgs s;
  s.K = a.K;
  s.B = a.B;
  s.L = a.L;
  s.theta_h = a.theta_h;
  s.theta_c = a.theta_c;
  s.theta_s = a.theta_s;
  s.w = a.w;
  s.k_max = a.k_max;
  s.token = a.token;
  s.entropy = a.entropy;
  s.confidence = a.confidence;
  s.persistence = a.persistence;
  s.drop = a.drop;
  s.stability = a.stability;
  s.flags = a.flags;
  s.layer_argmax = a.layer_argmax;
  s.layer_conf = a.layer_conf;
  s.layer_entropy = a.layer_entropy;
  return s;
}

CommitArgs commit_args(const Launch& a) {
  CommitArgs c;
  c.B = a.B;
  c.L = a.L;
  c.beta = a.beta;
  c.window = a.window;
  c.commit = a.commit;
  c.token = a.token;
  c.entropy = a.entropy;
  c.confidence = a.confidence;
  c.persistence = a.persistence;
  c.drop = a.drop;
  c.stability = a.stability;
  c.flags = a.flags;
  c.upstream_entropy = a.upstream_entropy;
  c.n_commit = a.n_commit;
  return c;
}

template <int NW, int MV, int NB, int KC, int NSTG, bool NTA>
void launch_proj_bf16(const Launch& a, hipStream_t s) {
  const ProjPlan& p = a.plan;
  hipLaunchKernelGGL((k_proj_bf16<NW, MV, NB, KC, NSTG, NTA>), dim3(p.grid), dim3(NW * 64), 0, s,
                     static_cast<const uint16_t*>(a.hidden), static_cast<const uint16_t*>(a.w_u), a.rows,
                     a.n_masked, a.partials, a.K, a.B, a.L, a.d, a.V, p.nvt, p.nrt, p.split_rows);
}

}  // namespace

// ------------------------------------------------------------------ host --

ProjPlan plan_projection(int dtype, long long rows_cap, int V) {
  ProjPlan p{};
  if (rows_cap < 1) rows_cap = 1;
  if (dtype == 1) {   // fp32
    p.variant = PROJ_F32;
    p.rows_per_tile = 16;
    p.vocab_cap = 64;
    p.nvt = (V + 63) / 64;
    p.nrt = (int)((rows_cap + 15) / 16);
    p.split_rows = 0;
    p.per_xcd = 0;
    p.grid = p.nvt * p.nrt;
    return p;
  }
  if (rows_cap <= 64) {
    p.variant = rows_cap <= 32 ? PROJ_BF16_R32 : PROJ_BF16_R64;
    p.rows_per_tile = rows_cap <= 32 ? 32 : 64;
    p.vocab_cap = 8 * 64;
    // every CU streams an equal share of W_U: a multiple of 256 tiles
    int nvt = (V + p.vocab_cap - 1) / p.vocab_cap;
    nvt = ((nvt + 255) / 256) * 256;
    p.nvt = nvt < V ? nvt : V;
  } else if (rows_cap <= 192) {
    p.variant = PROJ_BF16_M32;
    p.rows_per_tile = 128;
    p.vocab_cap = 8 * 64;
    p.nvt = (V + p.vocab_cap - 1) / p.vocab_cap;
  } else {
    p.variant = PROJ_BF16_BIG;
    p.rows_per_tile = big::TR;
    p.vocab_cap = big::TV;
    p.nvt = (V + p.vocab_cap - 1) / p.vocab_cap;
  }
  p.nrt = (int)((rows_cap + p.rows_per_tile - 1) / p.rows_per_tile);
  p.split_rows = p.nrt >= 8 ? 1 : 0;
  p.per_xcd = p.split_rows ? ((p.nrt + 7) / 8) * p.nvt : ((p.nvt + 7) / 8) * p.nrt;
  p.grid = 8 * p.per_xcd;
  return p;
}

hipError_t launch_compact(const Launch& a, hipStream_t s) {
  hipLaunchKernelGGL(k_compact, dim3(1), dim3(1024), 0, s, a.mask, a.B * a.L, a.max_masked, a.rows, a.n_masked,
                     a.dev_status, a.user_status);
  return hipGetLastError();
}

hipError_t launch_projection(const Launch& a, hipStream_t s) {
  if (a.max_masked <= 0) return hipSuccess;
  switch (a.plan.variant) {
    case PROJ_BF16_R32: launch_proj_bf16<8, 4, 2, 64, 3, false>(a, s); break;
    case PROJ_BF16_R64: launch_proj_bf16<8, 4, 4, 64, 3, false>(a, s); break;
    case PROJ_BF16_M32:
      hipLaunchKernelGGL((k_proj_bf16_m32<8, 2, 4, 64, 2>), dim3(a.plan.grid), dim3(512), 0, s,
                         static_cast<const uint16_t*>(a.hidden), static_cast<const uint16_t*>(a.w_u), a.rows,
                         a.n_masked, a.partials, a.K, a.B, a.L, a.d, a.V, a.plan.nvt, a.plan.nrt, a.plan.split_rows);
      break;
    case PROJ_BF16_BIG:
      hipLaunchKernelGGL(k_proj_bf16_big, dim3(a.plan.grid), dim3(256), 0, s, static_cast<const uint16_t*>(a.hidden),
                         static_cast<const uint16_t*>(a.w_u), a.rows, a.n_masked, a.partials, a.K, a.B, a.L, a.d, a.V,
                         a.plan.nvt, a.plan.nrt, a.plan.split_rows);
      break;
    case PROJ_F32:
      hipLaunchKernelGGL(k_proj_f32, dim3(a.plan.grid), dim3(256), 0, s, static_cast<const float*>(a.hidden),
                         static_cast<const float*>(a.w_u), a.rows, a.n_masked, a.partials, a.K, a.B, a.L, a.d, a.V,
                         a.plan.nvt);
      break;
  }
  return hipGetLastError();
}

hipError_t launch_reduce_score(const Launch& a, hipStream_t s) {
  if (a.max_masked <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_reduce_score, dim3(a.max_masked), dim3(64 * kReduceWaves), 0, s, a.partials, a.rows,
                     a.n_masked, a.plan.nvt, score_args(a));
  return hipGetLastError();
}

int commit_threads(int L) {
  const int t = ((L + 63) / 64) * 64;
  return t < kCommitThreads ? t : kCommitThreads;
}

hipError_t launch_commit(const Launch& a, hipStream_t s) {
  hipLaunchKernelGGL(k_commit, dim3(a.B), dim3(commit_threads(a.L)), 0, s, a.mask, commit_args(a));
  return hipGetLastError();
}

hipError_t launch_gate_commit(const Launch& a, const int32_t* l_y, const float* l_c, const float* l_h,
                              hipStream_t s) {
  const long long BL = (long long)a.B * a.L;
  hipLaunchKernelGGL(k_gate_score, dim3((unsigned)((BL + 255) / 256)), dim3(256), 0, s, a.mask, l_y, l_c, l_h,
                     score_args(a));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_commit, dim3(a.B), dim3(commit_threads(a.L)), 0, s, a.mask, commit_args(a));
  return hipGetLastError();
}

}  // namespace rpd
