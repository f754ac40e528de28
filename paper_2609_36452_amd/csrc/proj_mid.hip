// K1 projection, bf16, mid row counts (65 to 192 projected rows).
#include "proj_stage.h"

namespace rpd {
namespace {

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

}  // namespace

hipError_t launch_proj_mid(const Launch& a, hipStream_t s) {
  hipLaunchKernelGGL((k_proj_bf16_m32<8, 2, 4, 64, 2>), dim3(a.plan.grid), dim3(512), 0, s,
                     static_cast<const uint16_t*>(a.hidden), static_cast<const uint16_t*>(a.w_u), a.rows,
                     a.n_masked, a.partials, a.K, a.B, a.L, a.d, a.V, a.plan.nvt, a.plan.nrt, a.plan.split_rows);
  return hipGetLastError();
}

}  // namespace rpd
