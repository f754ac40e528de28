// K1 projection, bf16, up to 64 projected rows: the regime where streaming
// W_U once per call from HBM sets the time (the ridge of MI355X is about
// 315 rows; from 65 rows on the MFMA tile of proj_big.hip is faster).
#include "rpd_device.h"

namespace rpd {
namespace {

// The masked-position compaction (K0) folded into the projection's
// prologue, for small canvases: every workgroup scans the mask itself (while
// its first W_U loads are in flight) and keeps the first `need` positions;
// workgroup 0 also publishes the list, the count and the status for the
// kernels that follow, exactly as k_compact does.
struct CompactArgs {
  const uint8_t* mask;
  int BL, cap;
  int32_t* rows;
  int32_t* n;
  int32_t* dev_status;
  int32_t* user_status;
};

template <int NW>
__device__ int compact_in_workgroup(const CompactArgs& ca, int* s_pos, int need, int* s_wave) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const bool publish = blockIdx.x == 0;
  int carry = 0;
  for (int base = 0; base < ca.BL; base += NW * 64) {
    const int i = base + threadIdx.x;
    const bool f = i < ca.BL && ca.mask[i] != 0;
    const unsigned long long bal = __ballot(f);
    const int before = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) s_wave[wid] = __popcll(bal);
    __syncthreads();
    int off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const int c = s_wave[w];
      off += (w < wid) ? c : 0;
      tot += c;
    }
    const int rank = carry + off + before;
    if (f && rank < need) s_pos[rank] = i;
    if (f && publish && rank < ca.cap) ca.rows[rank] = i;
    carry += tot;
    __syncthreads();
  }
  const int n = carry < ca.cap ? carry : ca.cap;
  if (publish && threadIdx.x == 0) {
    const int st = carry > ca.cap ? 1 : 0;
    *ca.n = n;
    *ca.dev_status = st;
    if (ca.user_status) *ca.user_status = st;
  }
  return n;
}

// A workgroup of NW waves owns 32*MV*NW consecutive W_U rows (one
// vocabulary tile) and all TR = 32*NB projected rows, over the full hidden
// dimension, in 64-wide k-chunks.
//
// W_U: wave w owns 32*MV rows of the tile. They are read in full 128-byte
// lines (a load instruction covers 8 rows x 8 lanes x 16 B; non-temporal,
// since W_U is read exactly once per call), two chunks ahead in registers,
// and written to a one-chunk LDS buffer private to the wave, with the eight
// 16-byte pieces of row r stored XOR-swizzled by (r >> 1) & 7 so that the
// MFMA fragment reads are free of bank conflicts. A private buffer needs
// neither a second stage nor a barrier: one wave's LDS accesses complete in
// program order.
//
// Chunk order: workgroup tile vt takes the full chunks starting at
// (7 * vt) mod (d / 64) and wrapping around. In plain order every workgroup
// reads the same 128-byte column of rows 8 KB apart at the same time, so the
// low 13 address bits of all requests in flight match and they crowd onto
// a few HBM channels: a read probe of that order reached 5.7-5.9 TB/s where
// linear reads reach 7.0, and rotated starts 6.9 (the spread between boxes
// came mostly from this).
//
// Hidden rows: the TR rows of chunk c are loaded cooperatively by all
// threads (same line layout and swizzle) into one of two workgroup-shared
// LDS stages; one barrier per chunk publishes it, and the stage is refilled
// two chunks later, after every wave has passed the next barrier.
//
// v_mfma_f32_32x32x16_bf16 with W_U as A: lane l holds row l & 31 of a
// 32-row block and k-elements 8*(l >> 5) .. +8 of each 16-wide k-step (the
// same for the hidden rows as B). Accumulator register q of lane l holds
// vocabulary row 32*mv + 8*(q >> 2) + 4*(l >> 5) + (q & 3) of the wave's
// block and projected row 32*nb + (l & 31).
//
// Measured at the LLaDA-8B shape (d = 4096, V = 126464; projection alone,
// median of 60 calls on one GPU): 156 us at 32 rows (83% of 8 TB/s), 162-164
// us at 48-64. An 8-wave form for 65..128 rows (256 vocabulary rows x 128
// projected rows, one workgroup per CU) took 196-210 us at 68-128 rows, 7-12%
// slower than the 256 x 128 MFMA tile, and is no longer built.
//
// FC: the workgroup compacts the mask itself (compact_in_workgroup).
//
// Occupancy: the 4-wave forms run two workgroups per CU, which doubles the
// W_U bytes in flight per CU (what the streaming rate depends on). The
// 64-row form needs the launch bound's second argument for that (left to
// itself the compiler took 185 VGPRs + 80 AGPRs, one workgroup per CU):
// 4% faster at 64 rows.
template <int NW, int MV, int NB, bool FC>
__global__ __launch_bounds__(NW * 64, (NW == 4 && NB >= 2) ? 2 : 1) void k_proj_bf16_stream(
    const uint16_t* __restrict__ hidden, const uint16_t* __restrict__ w_u, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ n_ptr, float4* __restrict__ partials, int K, int B, int L, int d, int V,
    int nvt, int nrt, int split_rows, CompactArgs ca, const uint16_t* __restrict__ xrows,
    const long long* __restrict__ rowoff, float scale) {
  constexpr int TR = 32 * NB, WR = 32 * MV, KC = 64, NT = NW * 64;
  constexpr int NLD = WR / 8;          // W_U load instructions per wave per chunk
  constexpr int XLD = TR * 8 / NT;     // hidden-row pieces per thread per chunk
  constexpr int D = 2;                 // chunks in flight in registers
  static_assert(TR * 8 % NT == 0, "the hidden-row pieces of a chunk divide evenly over the threads");
  __shared__ __attribute__((aligned(16))) uint16_t wl[NW][WR][KC];
  __shared__ __attribute__((aligned(16))) uint16_t xl[2][TR][KC];
  __shared__ float4 red[NW][TR];
  __shared__ int s_pos[FC ? TR : 1];
  __shared__ int s_wave[NW];

  int rt = 0, vt = 0;
  const bool has_job = map_job(blockIdx.x, nvt, nrt, split_rows, rt, vt);
  if (!has_job && !(FC && blockIdx.x == 0)) return;   // workgroup 0 always publishes the compaction
  const int vb = (int)((long long)vt * V / nvt);
  const int ve = (int)((long long)(vt + 1) * V / nvt);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int vw = vb + wid * WR;

  // W_U: load u covers wave rows 8u + (lane >> 3); the lane fetches the
  // global piece that belongs at LDS piece (lane & 7) of that row. Rows past
  // the tile re-read its last row (never used).
  long long wa[NLD];
  int wpiece[NLD];
#pragma unroll
  for (int u = 0; u < NLD; ++u) {
    const int row = 8 * u + (lane >> 3);
    wpiece[u] = (lane & 7) ^ ((row >> 1) & 7);
    wa[u] = (long long)min(vw + row, ve - 1) * d + wpiece[u] * 8;
  }
  const int srow = lane >> 3, spc = (lane & 7) * 8;
  u32x4 ld[D][NLD];
  u32x4 xr[D][XLD];
  const int nchf = d / KC;
  // full chunks are taken in the order rot, rot+1, .., nchf-1, 0, .., rot-1
  const int rot = nchf > 0 ? (int)((7ll * vt) % nchf) : 0;
#define RPD_PCHUNK(c) ((c) + rot >= nchf ? (c) + rot - nchf : (c) + rot)
  // An explicit row list (a lazy pass) often has no rows at all, so its count
  // is read first (an empty launch then reads nothing: 1 us instead of 5).
  // Otherwise the W_U loads of the first two chunks go out before anything
  // waits.
  int R = 0;
  if (!FC && rowoff) {
    R = *n_ptr;
    if (rt * TR >= R) return;
  }
  if (has_job && nchf > 0) {
#pragma unroll
    for (int j = 0; j < D; ++j)
#pragma unroll
      for (int u = 0; u < NLD; ++u)
        ld[j][u] = __builtin_nontemporal_load(
            reinterpret_cast<const u32x4*>(w_u + wa[u] + (long long)RPD_PCHUNK(min(j, nchf - 1)) * KC));
  }
  if (FC) {
    // one row tile (r0 = 0): rows 0 .. TR-1 need positions 0 .. TR-1 at most
    R = compact_in_workgroup<NW>(ca, s_pos, TR, s_wave) * K;
    if (!has_job) return;
  } else if (!rowoff) {
    R = *n_ptr * K;   // an explicit row list (above) counts rows, not positions
  }
  const int r0 = rt * TR;
  if (r0 >= R) return;
  // hidden rows: piece q = tid + NT*u is row q >> 3, LDS piece q & 7. Rows
  // past the last projected row re-read row r0 (their results are dropped).
  long long xa[XLD];
  int xrow[XLD], xpiece[XLD];
#pragma unroll
  for (int u = 0; u < XLD; ++u) {
    const int q = tid + NT * u;
    const int row = q >> 3;
    xrow[u] = row;
    xpiece[u] = (q & 7) ^ ((row >> 1) & 7);
    const int r = r0 + row < R ? r0 + row : r0;
    if (xrows) {   // normalized rows, already in projected-row (or list) order
      xa[u] = (long long)r * d + xpiece[u] * 8;
    } else if (rowoff) {   // an explicit row list
      xa[u] = rowoff[r] + xpiece[u] * 8;
    } else {
      const int p = r / K, l = r - p * K;
      const int pos = FC ? s_pos[p] : rows[p];
      const int b = pos / L, i = pos - b * L;
      xa[u] = (((long long)l * B + b) * L + i) * (long long)d + xpiece[u] * 8;
    }
  }
  const uint16_t* __restrict__ xsrc = xrows ? xrows : hidden;
  const int xpc = (tid & 7) * 8;       // LDS piece of this thread's hidden-row loads
  // fragments: row base + (lane & 31), logical piece 2s + (lane >> 5)
  const int fr = lane & 31, fsw = (fr >> 1) & 7, fhi = lane >> 5;

  f32x16 acc[MV][NB];
#pragma unroll
  for (int mv = 0; mv < MV; ++mv)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[mv][nb][q] = 0.f;
#define RPD_XLOAD(slot, chunk)                                                                           \
  do {                                                                                                   \
    const long long k0_ = (long long)RPD_PCHUNK(chunk) * KC;                                             \
    _Pragma("unroll") for (int u_ = 0; u_ < XLD; ++u_)                                                  \
      xr[slot][u_] = *reinterpret_cast<const u32x4*>(xsrc + xa[u_] + k0_);                               \
  } while (0)
#define RPD_SLOAD(slot, chunk)                                                                           \
  do {                                                                                                   \
    const long long k0_ = (long long)RPD_PCHUNK(chunk) * KC;                                             \
    _Pragma("unroll") for (int u_ = 0; u_ < NLD; ++u_)                                                  \
      ld[slot][u_] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(w_u + wa[u_] + k0_));     \
    RPD_XLOAD(slot, chunk);                                                                              \
  } while (0)
  // the MFMAs of one staged chunk (W_U in the wave's buffer, hidden rows in stage XS)
#define RPD_SMMA(XS)                                                                                     \
  do {                                                                                                   \
    _Pragma("unroll") for (int s_ = 0; s_ < 4; ++s_) {                                                  \
      const int pc_ = 8 * ((2 * s_ + fhi) ^ fsw);                                                        \
      u32x4 fa_[MV], fb_[NB];                                                                            \
      _Pragma("unroll") for (int mv_ = 0; mv_ < MV; ++mv_)                                              \
        fa_[mv_] = *reinterpret_cast<const u32x4*>(&wl[wid][32 * mv_ + fr][pc_]);                       \
      _Pragma("unroll") for (int nb_ = 0; nb_ < NB; ++nb_)                                              \
        fb_[nb_] = *reinterpret_cast<const u32x4*>(&xl[XS][32 * nb_ + fr][pc_]);                        \
      _Pragma("unroll") for (int mv_ = 0; mv_ < MV; ++mv_)                                              \
      _Pragma("unroll") for (int nb_ = 0; nb_ < NB; ++nb_)                                              \
        acc[mv_][nb_] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa_[mv_]),    \
                                                                 __builtin_bit_cast(bf16x8, fb_[nb_]),    \
                                                                 acc[mv_][nb_], 0, 0, 0);                \
    }                                                                                                    \
  } while (0)
  // chunk c: register slot SL -> LDS (W_U buffer, hidden stage XS), refill
  // SL with chunk c + D (chunks past the end repeat the last one, never
  // multiplied), publish, multiply
#define RPD_SCHUNK(c, SL, XS)                                                                            \
  do {                                                                                                   \
    _Pragma("unroll") for (int u_ = 0; u_ < NLD; ++u_)                                                  \
      *reinterpret_cast<u32x4*>(&wl[wid][8 * u_ + srow][spc]) = ld[SL][u_];                             \
    _Pragma("unroll") for (int u_ = 0; u_ < XLD; ++u_)                                                  \
      *reinterpret_cast<u32x4*>(&xl[XS][xrow[u_]][xpc]) = xr[SL][u_];                                    \
    RPD_SLOAD(SL, min((c) + D, nchf - 1));                                                               \
    __syncthreads();                                                                                     \
    RPD_SMMA(XS);                                                                                        \
  } while (0)

  if (nchf > 0) {
    RPD_XLOAD(0, 0);
    RPD_XLOAD(1, min(1, nchf - 1));
    int c = 0;
    for (; c + 2 <= nchf; c += 2) {
      RPD_SCHUNK(c, 0, 0);
      RPD_SCHUNK(c + 1, 1, 1);
    }
    if (c < nchf) RPD_SCHUNK(c, 0, 0);
  }
  if (d % KC != 0) {   // partial last chunk, zero-filled past d (d % 8 == 0: a piece is all in or all out)
    const long long k0 = (long long)nchf * KC;
    const int XS = nchf & 1;   // the stage not read by the last full chunk
#pragma unroll
    for (int u = 0; u < NLD; ++u)
      *reinterpret_cast<u32x4*>(&wl[wid][8 * u + srow][spc]) =
          k0 + wpiece[u] * 8 < d ? *reinterpret_cast<const u32x4*>(w_u + wa[u] + k0) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int u = 0; u < XLD; ++u)
      *reinterpret_cast<u32x4*>(&xl[XS][xrow[u]][xpc]) =
          k0 + xpiece[u] * 8 < d ? *reinterpret_cast<const u32x4*>(xsrc + xa[u] + k0) : u32x4{0u, 0u, 0u, 0u};
    __syncthreads();
    if (XS == 0)
      RPD_SMMA(0);
    else
      RPD_SMMA(1);
  }
#undef RPD_SCHUNK
#undef RPD_SMMA
#undef RPD_PCHUNK
#undef RPD_SLOAD
#undef RPD_XLOAD

  // epilogue: softmax state of the wave's vocabulary rows per projected row,
  // then a fixed-order merge over the waves
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    Soft sst = soft_empty();
#pragma unroll
    for (int mv = 0; mv < MV; ++mv) {
      float z[16];
      int vi[16];
      bool ok[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int v = vw + 32 * mv + (q >> 2) * 8 + (lane >> 5) * 4 + (q & 3);
        z[q] = acc[mv][nb][q] * scale;
        vi[q] = v;
        ok[q] = v < ve;
      }
      sst = soft_merge(sst, soft_from_values(z, vi, ok));
    }
    sst = soft_merge(sst, soft_shfl_xor(sst, 32));
    if (lane < 32) red[wid][32 * nb + lane] = soft_pack(sst);
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

template <int NW, int MV, int NB>
void launch_stream(const Launch& a, hipStream_t s) {
  static_assert(32 * MV * NW == kStreamTileVocab, "every streaming variant covers the same vocabulary tile");
  const ProjPlan& p = a.plan;
  const CompactArgs ca{a.mask, a.B * a.L, a.max_masked, a.rows, a.n_masked, a.dev_status, a.user_status};
  if (a.fused_compact)
    hipLaunchKernelGGL((k_proj_bf16_stream<NW, MV, NB, true>), dim3(p.grid), dim3(NW * 64), 0, s,
                       static_cast<const uint16_t*>(a.hidden), static_cast<const uint16_t*>(a.w_u), a.rows,
                       a.n_masked, a.partials, a.K, a.B, a.L, a.d, a.V, p.nvt, p.nrt, p.split_rows, ca,
                       static_cast<const uint16_t*>(a.xrows), a.rowoff, a.logit_scale);
  else
    hipLaunchKernelGGL((k_proj_bf16_stream<NW, MV, NB, false>), dim3(p.grid), dim3(NW * 64), 0, s,
                       static_cast<const uint16_t*>(a.hidden), static_cast<const uint16_t*>(a.w_u), a.rows,
                       a.n_masked, a.partials, a.K, a.B, a.L, a.d, a.V, p.nvt, p.nrt, p.split_rows, ca,
                       static_cast<const uint16_t*>(a.xrows), a.rowoff, a.logit_scale);
}

}  // namespace

bool compact_fused(const Launch& a) {
  const ProjVariant v = a.plan.variant;
  const bool streaming = v == PROJ_BF16_S32 || v == PROJ_BF16_S64;
  return streaming && a.plan.nrt == 1 && a.max_masked > 0 && (long long)a.B * a.L <= kFusedCompactMax &&
         !a.xrows && !a.rowoff;   // the normalization and explicit row lists need the compaction first
}

hipError_t launch_proj_stream(const Launch& a, hipStream_t s) {
  switch (a.plan.variant) {
    case PROJ_BF16_S32: launch_stream<4, 2, 1>(a, s); break;
    case PROJ_BF16_S64: launch_stream<4, 2, 2>(a, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace rpd
