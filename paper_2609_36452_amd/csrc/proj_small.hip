// K1 projection, bf16, small row counts (up to 64 projected rows): the
// HBM-bound regime, where streaming W_U once per call sets the time.
#include "proj_stage.h"

namespace rpd {
namespace {

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

template <int NW, int MV, int NB, int KC, int NSTG, bool NTA>
void launch_proj_bf16(const Launch& a, hipStream_t s) {
  const ProjPlan& p = a.plan;
  hipLaunchKernelGGL((k_proj_bf16<NW, MV, NB, KC, NSTG, NTA>), dim3(p.grid), dim3(NW * 64), 0, s,
                     static_cast<const uint16_t*>(a.hidden), static_cast<const uint16_t*>(a.w_u), a.rows,
                     a.n_masked, a.partials, a.K, a.B, a.L, a.d, a.V, p.nvt, p.nrt, p.split_rows);
}

}  // namespace

hipError_t launch_proj_small(const Launch& a, hipStream_t s) {
  if (a.plan.variant == PROJ_BF16_R32)
    launch_proj_bf16<8, 4, 2, 64, 3, false>(a, s);
  else
    launch_proj_bf16<8, 4, 4, 64, 3, false>(a, s);
  return hipGetLastError();
}

}  // namespace rpd
