// K1 projection, bf16, large row counts (more than 192 projected rows): the
// MFMA-bound regime.
#include "rpd_device.h"

namespace rpd {
namespace {

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
constexpr int TV = kBigTileVocab, TR = kBigTileRows, KC = 32, NSTG = 4;
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

}  // namespace

hipError_t launch_proj_big(const Launch& a, hipStream_t s) {
  hipLaunchKernelGGL(k_proj_bf16_big, dim3(a.plan.grid), dim3(256), 0, s, static_cast<const uint16_t*>(a.hidden),
                     static_cast<const uint16_t*>(a.w_u), a.rows, a.n_masked, a.partials, a.K, a.B, a.L, a.d, a.V,
                     a.plan.nvt, a.plan.nrt, a.plan.split_rows);
  return hipGetLastError();
}

}  // namespace rpd
