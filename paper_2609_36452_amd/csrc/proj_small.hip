// K1 projection, bf16, small row counts (up to 64 projected rows): the
// HBM-bound regime, where streaming W_U once per call sets the time.
// k_proj_bf16_stream serves up to 32 rows, k_proj_bf16 33 to 64.
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


// At most 32 projected rows: every wave streams its own W_U rows, with no
// barrier until the epilogue. Wave w of the workgroup owns 32*MV
// consecutive W_U rows. They are read in full 128-byte lines (a load
// instruction covers 8 rows x 8 lanes x 16 B, non-temporal: W_U is read
// exactly once per call), D = 2 chunks of 64 k-elements ahead in registers,
// and written to a two-stage LDS ring private to the wave, with the eight
// 16-byte pieces of row r stored XOR-swizzled by (r >> 1) & 7 so that the
// MFMA fragment reads are conflict-free. Private stages need no barrier:
// one wave's LDS accesses complete in order. The hidden rows (at most 32,
// shared by every workgroup, resident in L2) are read by each wave straight
// into the B-operand layout of v_mfma_f32_32x32x16_bf16: lane l holds row
// l & 31, k-elements 8*(l >> 5) .. +8 of each 16-wide k-step. Accumulator
// register q of lane l holds vocabulary row 32*mv + 8*(q >> 2) + 4*(l >> 5)
// + (q & 3) of the wave's block and projected row l & 31.
//
// Full-line, non-temporal, row-private streaming measured 168 us at the
// LLaDA-8B shape (77% of 8 TB/s) against 187 us for k_proj_bf16's 16-row x
// 64-byte register layout.
template <int NW, int MV>
__global__ __launch_bounds__(NW * 64) void k_proj_bf16_stream(
    const uint16_t* __restrict__ hidden, const uint16_t* __restrict__ w_u, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ n_ptr, float4* __restrict__ partials, int K, int B, int L, int d, int V,
    int nvt, int nrt, int split_rows) {
  constexpr int TR = 32, WR = 32 * MV, KC = 64, NLD = WR / 8, D = 2;
  __shared__ __attribute__((aligned(16))) uint16_t wl[NW][2][WR][KC];
  __shared__ float4 red[NW][TR];

  int rt, vt;
  if (!map_job(blockIdx.x, nvt, nrt, split_rows, rt, vt)) return;
  const int R = *n_ptr * K;
  const int r0 = rt * TR;
  if (r0 >= R) return;
  const int vb = (int)((long long)vt * V / nvt);
  const int ve = (int)((long long)(vt + 1) * V / nvt);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int vw = vb + wid * WR;

  // W_U: load u covers wave rows 8u + (lane >> 3); lane fetches the global
  // piece that belongs at LDS piece (lane & 7) of that row
  long long wa[NLD];
#pragma unroll
  for (int u = 0; u < NLD; ++u) {
    const int row = 8 * u + (lane >> 3);
    wa[u] = (long long)min(vw + row, ve - 1) * d + (((lane & 7) ^ ((row >> 1) & 7)) * 8);
  }
  const int srow = lane >> 3, spc = (lane & 7) * 8;
  // hidden: this lane's projected row (rows past the last re-read row r0; discarded at the end)
  long long xo;
  {
    const int r = r0 + (lane & 31) < R ? r0 + (lane & 31) : r0;
    const int p = r / K, l = r - p * K;
    const int pos = rows[p];
    const int b = pos / L, i = pos - b * L;
    xo = (((long long)l * B + b) * L + i) * (long long)d + 8 * (lane >> 5);
  }
  const int fr = lane & 31, fsw = (fr >> 1) & 7, fhi = lane >> 5;

  f32x16 acc[MV];
#pragma unroll
  for (int mv = 0; mv < MV; ++mv)
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[mv][q] = 0.f;
  u32x4 ld[D][NLD];
  u32x4 xb[D][4];
  const int nchf = d / KC;

#define RPD_SLOAD(slot, chunk)                                                                          \
  do {                                                                                                  \
    const long long k0_ = (long long)(chunk) * KC;                                                      \
    _Pragma("unroll") for (int u_ = 0; u_ < NLD; ++u_)                                                 \
      ld[slot][u_] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(w_u + wa[u_] + k0_));    \
    _Pragma("unroll") for (int s_ = 0; s_ < 4; ++s_)                                                   \
      xb[slot][s_] = *reinterpret_cast<const u32x4*>(hidden + xo + k0_ + 16 * s_);                      \
  } while (0)
  // chunk c: registers of slot SL -> LDS stage ST, refill SL with chunk
  // c + D (chunks past the end repeat the last one, never multiplied), then
  // the four k-steps of chunk c
#define RPD_SCHUNK(c, SL, ST)                                                                           \
  do {                                                                                                  \
    _Pragma("unroll") for (int u_ = 0; u_ < NLD; ++u_)                                                 \
      *reinterpret_cast<u32x4*>(&wl[wid][ST][8 * u_ + srow][spc]) = ld[SL][u_];                        \
    u32x4 xc_[4];                                                                                       \
    _Pragma("unroll") for (int s_ = 0; s_ < 4; ++s_) xc_[s_] = xb[SL][s_];                             \
    RPD_SLOAD(SL, min((c) + D, nchf - 1));                                                              \
    _Pragma("unroll") for (int s_ = 0; s_ < 4; ++s_) {                                                 \
      const int pc_ = 8 * ((2 * s_ + fhi) ^ fsw);                                                       \
      u32x4 fa_[MV];                                                                                    \
      _Pragma("unroll") for (int mv_ = 0; mv_ < MV; ++mv_)                                             \
        fa_[mv_] = *reinterpret_cast<const u32x4*>(&wl[wid][ST][32 * mv_ + fr][pc_]);                  \
      _Pragma("unroll") for (int mv_ = 0; mv_ < MV; ++mv_)                                             \
        acc[mv_] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa_[mv_]),        \
                                                            __builtin_bit_cast(bf16x8, xc_[s_]), acc[mv_], \
                                                            0, 0, 0);                                   \
    }                                                                                                   \
  } while (0)

  if (nchf > 0) {
    RPD_SLOAD(0, 0);
    RPD_SLOAD(1, min(1, nchf - 1));
    int c = 0;
    for (; c + 2 <= nchf; c += 2) {
      RPD_SCHUNK(c, 0, 0);
      RPD_SCHUNK(c + 1, 1, 1);
    }
    if (c < nchf) RPD_SCHUNK(c, 0, 0);
  }
#undef RPD_SCHUNK
#undef RPD_SLOAD
  if (d % KC != 0) {   // partial last chunk, zero-filled past d (d % 8 == 0: a piece is all in or all out)
    const long long k0 = (long long)nchf * KC;
#pragma unroll
    for (int u = 0; u < NLD; ++u) {
      const int row = 8 * u + srow;
      const int piece = (lane & 7) ^ ((row >> 1) & 7);
      *reinterpret_cast<u32x4*>(&wl[wid][0][row][spc]) =
          k0 + piece * 8 < d ? *reinterpret_cast<const u32x4*>(w_u + wa[u] + k0) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const long long k = k0 + 16 * s + 8 * fhi;
      const u32x4 xv = k < d ? *reinterpret_cast<const u32x4*>(hidden + xo + k0 + 16 * s) : u32x4{0u, 0u, 0u, 0u};
      const int pc = 8 * ((2 * s + fhi) ^ fsw);
      u32x4 fa[MV];
#pragma unroll
      for (int mv = 0; mv < MV; ++mv) fa[mv] = *reinterpret_cast<const u32x4*>(&wl[wid][0][32 * mv + fr][pc]);
#pragma unroll
      for (int mv = 0; mv < MV; ++mv)
        acc[mv] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa[mv]),
                                                          __builtin_bit_cast(bf16x8, xv), acc[mv], 0, 0, 0);
    }
  }

  // epilogue: softmax state of the wave's vocabulary rows per projected row,
  // then a fixed-order merge over the waves
  {
    Soft sst = soft_empty();
#pragma unroll
    for (int mv = 0; mv < MV; ++mv) {
      float z[16];
      int vi[16];
      bool ok[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int v = vw + 32 * mv + (q >> 2) * 8 + (lane >> 5) * 4 + (q & 3);
        z[q] = acc[mv][q];
        vi[q] = v;
        ok[q] = v < ve;
      }
      sst = soft_merge(sst, soft_from_values(z, vi, ok));
    }
    sst = soft_merge(sst, soft_shfl_xor(sst, 32));
    if (lane < 32) red[wid][lane] = soft_pack(sst);
  }
  __syncthreads();
  for (int t = tid; t < TR; t += NW * 64) {
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
  const ProjPlan& p = a.plan;
  if (p.variant == PROJ_BF16_R32)
    hipLaunchKernelGGL((k_proj_bf16_stream<kStreamWaves, kStreamBlocks>), dim3(p.grid), dim3(kStreamWaves * 64), 0,
                       s, static_cast<const uint16_t*>(a.hidden), static_cast<const uint16_t*>(a.w_u), a.rows,
                       a.n_masked, a.partials, a.K, a.B, a.L, a.d, a.V, p.nvt, p.nrt, p.split_rows);
  else
    launch_proj_bf16<8, 4, 4, 64, 3, false>(a, s);
  return hipGetLastError();
}

}  // namespace rpd
