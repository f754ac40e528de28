// K1 projection, bf16, large row counts (more than 256 projected rows): the
// MFMA-bound regime.
#include "rpd_device.h"

namespace rpd {
namespace {

// A GEMM tile of 256 vocabulary rows x 256 projected rows over the full
// hidden dimension, four waves in a 2 x 2 layout, each computing 128 x 128
// with v_mfma_f32_32x32x16_bf16 (256 fp32 accumulators per lane in AGPRs,
// one wave per SIMD).
//
// Operands move global -> registers -> LDS -> MFMA fragments. A 32-wide
// k-chunk of both operands (256 rows x 64 bytes each) is loaded into
// registers three chunks ahead (16 B per lane, a wave instruction covering 16
// rows x 64 bytes), written to one of two LDS stages, and read back as MFMA
// fragments. With one wave per SIMD nothing else hides the load latency:
// three chunks in flight instead of two measured 4-5% faster from 512 rows up
// (the register slots rotate with period 3 against the stages' period 2, so
// the loop is unrolled six times to keep every slot index static). Within a tile row the four 16-byte pieces are stored XOR-
// swizzled by (row >> 2) & 3 (chosen through which global piece each lane
// fetches), so the fragment reads are free of bank conflicts.
//
// Plain loads into registers rather than direct global->LDS loads: with one
// wave per SIMD, direct loads sustain about 17 B/clk per CU, below the
// 32 B/clk this tile needs at full MFMA rate, and being opaque to the
// compiler's scheduler they cannot be spread between MFMAs; register loads
// sustain about 26 B/clk and interleave.
//
// Per chunk c (stage c & 1), the instruction stream is fixed with scheduling
// groups so that one memory instruction issues between consecutive MFMAs:
//   first half:  MFMAs of k-step (c,0), interleaved with the fragment reads
//                of (c,1), the LDS writes of chunk c+1 and the global loads
//                of chunk c+4;
//   barrier:     publishes chunk c+1 and frees stage c & 1;
//   second half: MFMAs of (c,1), interleaved with the fragment reads of
//                (c+1,0).
namespace big {
constexpr int TV = kBigTileVocab, TR = kBigTileRows, KC = 32;
constexpr int D = 3;   // chunks in flight in registers
}  // namespace big

__global__ __launch_bounds__(256) void k_proj_bf16_big(
    const uint16_t* __restrict__ hidden, const uint16_t* __restrict__ w_u, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ n_ptr, float4* __restrict__ partials, int K, int B, int L, int d, int V,
    int nvt, int nrt, int split_rows, const uint16_t* __restrict__ xrows, const long long* __restrict__ rowoff,
    float scale) {
  using namespace big;
  static_assert(TV == 256 && TR == 256 && D == 3, "wave layout and register ring below assume these");
  __shared__ __attribute__((aligned(16))) uint16_t sa0[TV][KC], sa1[TV][KC];
  __shared__ __attribute__((aligned(16))) uint16_t sb0[TR][KC], sb1[TR][KC];
  __shared__ float4 red[2][TR];
#define RPD_SA(S) ((S) == 0 ? sa0 : sa1)
#define RPD_SB(S) ((S) == 0 ? sb0 : sb1)

  int rt, vt;
  if (!map_job(blockIdx.x, nvt, nrt, split_rows, rt, vt)) return;
  const int R = rowoff ? *n_ptr : *n_ptr * K;   // an explicit row list counts rows, not positions
  const int r0 = rt * TR;
  if (r0 >= R) return;
  const int vb = (int)((long long)vt * V / nvt);
  const int ve = (int)((long long)(vt + 1) * V / nvt);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wv = wid & 1, wr = wid >> 1;

  // load sources: instruction u of this wave covers tile rows
  // 64*wid + 16*u .. +16; lane l holds LDS piece (l & 3) of row (l >> 2),
  // fetched from the global piece (l & 3) ^ swizzle(row)
  long long ga[4], gb[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int tr = 64 * wid + 16 * u + (lane >> 2);
    const int piece = (lane & 3) ^ ((tr >> 2) & 3);
    ga[u] = (long long)min(vb + tr, ve - 1) * d + piece * 8;
    const int r = r0 + tr < R ? r0 + tr : r0;   // padding rows re-read a real row; discarded at the end
    if (xrows) {   // normalized rows, already in projected-row order
      gb[u] = (long long)r * d + piece * 8;
    } else if (rowoff) {   // an explicit row list
      gb[u] = rowoff[r] + piece * 8;
    } else {
      const int p = r / K, l = r - p * K;
      const int pos = rows[p];
      const int b = pos / L, i = pos - b * L;
      gb[u] = (((long long)l * B + b) * L + i) * (long long)d + piece * 8;
    }
  }
  const uint16_t* __restrict__ xsrc = xrows ? xrows : hidden;
  const int srow = lane >> 2, scol = (lane & 3) * 8;
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
  u32x4 ld[D][8];
  u32x4 fa0[4], fb0[4], fa1[4], fb1[4];

#define RPD_LOAD(slot, chunk)                                                                             \
  do {                                                                                                    \
    const long long k0_ = (long long)(chunk) * KC;                                                        \
    _Pragma("unroll") for (int u_ = 0; u_ < 4; ++u_) {                                                   \
      ld[slot][u_] = *reinterpret_cast<const u32x4*>(w_u + ga[u_] + k0_);                                 \
      ld[slot][4 + u_] = *reinterpret_cast<const u32x4*>(xsrc + gb[u_] + k0_);                            \
    }                                                                                                     \
  } while (0)
#define RPD_STORE(slot, stage)                                                                            \
  do {                                                                                                    \
    _Pragma("unroll") for (int u_ = 0; u_ < 4; ++u_) {                                                   \
      *reinterpret_cast<u32x4*>(&RPD_SA(stage)[64 * wid + 16 * u_ + srow][scol]) = ld[slot][u_];         \
      *reinterpret_cast<u32x4*>(&RPD_SB(stage)[64 * wid + 16 * u_ + srow][scol]) = ld[slot][4 + u_];     \
    }                                                                                                     \
  } while (0)
#define RPD_FRAGS(FA, FB, stage, kstep)                                                                   \
  do {                                                                                                    \
    const int fc_ = (kstep) ? fcol1 : fcol0;                                                              \
    _Pragma("unroll") for (int m_ = 0; m_ < 4; ++m_) {                                                   \
      FA[m_] = *reinterpret_cast<const u32x4*>(&RPD_SA(stage)[128 * wv + 32 * m_ + (lane & 31)][fc_]);   \
      FB[m_] = *reinterpret_cast<const u32x4*>(&RPD_SB(stage)[128 * wr + 32 * m_ + (lane & 31)][fc_]);   \
    }                                                                                                     \
  } while (0)
#define RPD_MMA(FA, FB)                                                                                   \
  do {                                                                                                    \
    _Pragma("unroll") for (int mv_ = 0; mv_ < 4; ++mv_)                                                  \
    _Pragma("unroll") for (int nb_ = 0; nb_ < 4; ++nb_)                                                  \
      acc[mv_][nb_] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, FA[mv_]),        \
                                                               __builtin_bit_cast(bf16x8, FB[nb_]),        \
                                                               acc[mv_][nb_], 0, 0, 0);                   \
  } while (0)
  // one chunk c, held in stage ST; its successor goes to stage ST^1 from
  // register slot SL, which is then refilled with chunk c+1+D. Chunks past
  // the end repeat the last one (loaded and staged, never multiplied).
#define RPD_CHUNK(c, ST, SL)                                                                              \
  do {                                                                                                    \
    __builtin_amdgcn_sched_barrier(0);                                                                    \
    RPD_FRAGS(fa1, fb1, ST, 1);                                                                           \
    RPD_STORE(SL, (ST) ^ 1);                                                                              \
    RPD_LOAD(SL, min((c) + 1 + D, nchf - 1));                                                             \
    RPD_MMA(fa0, fb0);                                                                                    \
    _Pragma("unroll") for (int g_ = 0; g_ < 8; ++g_) {                                                   \
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0); /* MFMA */                                       \
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0); /* LDS read */                                   \
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0); /* MFMA */                                       \
      __builtin_amdgcn_sched_group_barrier(0x200, 1, 0); /* LDS write */                                  \
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0); /* global load */                                \
    }                                                                                                     \
    __builtin_amdgcn_sched_barrier(0);                                                                    \
    __syncthreads();                                                                                      \
    __builtin_amdgcn_sched_barrier(0);                                                                    \
    RPD_FRAGS(fa0, fb0, (ST) ^ 1, 0);                                                                     \
    RPD_MMA(fa1, fb1);                                                                                    \
    _Pragma("unroll") for (int g_ = 0; g_ < 8; ++g_) {                                                   \
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                                                  \
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);                                                  \
    }                                                                                                     \
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);                                                    \
    __builtin_amdgcn_sched_barrier(0);                                                                    \
  } while (0)

  const int nchf = d / KC;
  if (nchf > 0) {
#pragma unroll
    for (int j = 0; j < D; ++j) RPD_LOAD(j, min(j, nchf - 1));
    RPD_STORE(0, 0);
    RPD_LOAD(0, min(D, nchf - 1));
    __syncthreads();
    RPD_FRAGS(fa0, fb0, 0, 0);
    // chunk c: stage c & 1, register slot (c + 1) % 3
    int c = 0;
    for (; c + 6 <= nchf; c += 6) {
      RPD_CHUNK(c, 0, 1);
      RPD_CHUNK(c + 1, 1, 2);
      RPD_CHUNK(c + 2, 0, 0);
      RPD_CHUNK(c + 3, 1, 1);
      RPD_CHUNK(c + 4, 0, 2);
      RPD_CHUNK(c + 5, 1, 0);
    }
    if (c < nchf) RPD_CHUNK(c, 0, 1);
    if (c + 1 < nchf) RPD_CHUNK(c + 1, 1, 2);
    if (c + 2 < nchf) RPD_CHUNK(c + 2, 0, 0);
    if (c + 3 < nchf) RPD_CHUNK(c + 3, 1, 1);
    if (c + 4 < nchf) RPD_CHUNK(c + 4, 0, 2);
  }
  if (d % KC != 0) {   // partial last chunk, zero-filled past d (d % 8 == 0: a piece is all in or all out)
    __syncthreads();   // every wave is done with both stages
    const long long k0 = (long long)nchf * KC;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int tr = 64 * wid + 16 * u + srow;
      const int piece = (lane & 3) ^ ((tr >> 2) & 3);
      const bool in = k0 + piece * 8 < d;
      const u32x4 va = in ? *reinterpret_cast<const u32x4*>(w_u + ga[u] + k0) : u32x4{0u, 0u, 0u, 0u};
      const u32x4 vh = in ? *reinterpret_cast<const u32x4*>(xsrc + gb[u] + k0) : u32x4{0u, 0u, 0u, 0u};
      *reinterpret_cast<u32x4*>(&sa0[tr][scol]) = va;
      *reinterpret_cast<u32x4*>(&sb0[tr][scol]) = vh;
    }
    __syncthreads();
    RPD_FRAGS(fa0, fb0, 0, 0);
    RPD_MMA(fa0, fb0);
    RPD_FRAGS(fa1, fb1, 0, 1);
    RPD_MMA(fa1, fb1);
  }
#undef RPD_CHUNK
#undef RPD_MMA
#undef RPD_FRAGS
#undef RPD_STORE
#undef RPD_LOAD
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
        z[q] = acc[mv][nb][q] * scale;
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

}  // namespace

hipError_t launch_proj_big(const Launch& a, hipStream_t s) {
  hipLaunchKernelGGL(k_proj_bf16_big, dim3(a.plan.grid), dim3(256), 0, s, static_cast<const uint16_t*>(a.hidden),
                     static_cast<const uint16_t*>(a.w_u), a.rows, a.n_masked, a.partials, a.K, a.B, a.L, a.d, a.V,
                     a.plan.nvt, a.plan.nrt, a.plan.split_rows, static_cast<const uint16_t*>(a.xrows), a.rowoff,
                     a.logit_scale);
  return hipGetLastError();
}

}  // namespace rpd
