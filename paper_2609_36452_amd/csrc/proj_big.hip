// K1 projection, bf16, more than 64 projected rows: the MFMA-bound regime
// (and the approach to it).
#include "rpd_device.h"

namespace rpd {
namespace {

// A GEMM tile of 256 vocabulary rows x TR projected rows (TR = 256, 192 or
// 128) over the full hidden dimension, four waves in a 2 x 2 layout, each
// computing 128 x TR/2 with v_mfma_f32_32x32x16_bf16 (up to 256 fp32
// accumulators per lane in AGPRs, one wave per SIMD). 65..128 rows take one
// 128-row tile per vocabulary tile (7-12% faster there than streaming W_U
// through registers); above, the plan takes whichever of 192 and 256 rows
// pads the projected rows less (192 rows measured 18% faster at 576 rows,
// where 256-row tiles do a third more MFMA work).
//
// Operands go from global memory straight into LDS (each load instruction
// deposits 64 lanes x 16 B = 8 rows x 128 B of one operand at the LDS address
// in M0), in 64-wide k-chunks, and are read back as MFMA fragments. Both come
// through buffer loads (a resource at W_U's tile or at the row source, fixed
// 32-bit lane offsets, the chunk's offset in a scalar register: no per-load
// 64-bit address arithmetic); a row source of 2^31 bytes or more takes
// global_load_lds from 64-bit lane addresses instead (HB = false). No register
// staging and no LDS store instructions: with them, the LDS instruction queue
// saturated (counters showed its data FIFO full for 1.2e7 cycles per call at
// 1024 rows). The eight 16-byte pieces of row r sit XOR-swizzled by
// (r >> 1) & 7 (each lane fetches the global piece that belongs at its LDS
// slot), which keeps the fragment reads free of bank conflicts.
//
// Stages: three for W_U (32 KB each) and two for the hidden rows (TR x 128 B
// each): 160, 144 and 128 KB of LDS at TR = 256, 192 and 128 (the epilogue's
// reduction array reuses W_U stage 0). A W_U chunk is first fetched from HBM
// by whichever of the workgroups sharing it gets there first, while hidden
// rows mostly come from L2 or the MALL, so W_U is loaded one chunk further
// ahead than the hidden rows.
//
// Chunk c (W_U stage c % 3, hidden stage c % 2) is multiplied in four
// k-steps of 4 * TR/64 MFMAs per wave, each reading the next step's
// fragments. After the
// third step every wave waits until only its newest 8 loads (W_U of chunk
// c+2) may be outstanding, so chunk c+1 has landed, and for its fragment
// reads; one barrier then publishes chunk c+1 and frees chunk c's stages
// for the hidden rows of chunk c+2 and W_U of chunk c+3. Those loads are
// spread over the next four k-steps (see RPD_CHUNK). The barrier is a plain
// s_barrier: the waits before it are exactly the ones this schedule needs,
// where a fenced barrier would also drain the loads still in flight.
//
// Measured, in steps, against loads staged through registers in 32-wide
// chunks two ahead: three chunks in flight 4-5% faster; direct loads, 64-wide
// chunks, two stages each: another 4-6%; a third W_U stage: another 3-7%;
// the loads spread over the k-steps instead of all in the fourth: 12% fewer
// cycles in the main loop, 3.5% less time (the chip then runs at its power
// limit and lowers the clock); the epilogue without validity selects on full
// tiles: 38% fewer epilogue cycles; buffer loads for W_U, then for the hidden
// rows: 4% and 6% fewer main-loop cycles (9.5 ms at 12288 rows on one GPU);
// the epilogue's sums in base-2 units from one fma per logit and 3-input
// maxima: 0.2-1.6% less time from 192 to 12288 rows (interleaved A/B), the
// 256-row form's spills down from 19 VGPRs to 3; the maxima on
// NaN-propagating v_maximum3_f32 (fmaxf made the compiler canonicalize every
// accumulator first): another 0.1-1.1%. The same tile on 16x16x32 MFMAs
// (fragments of 16 rows x 32 k) measured 2-4% slower at 128-576 rows, and
// its 256-row form spilled 338-538 VGPRs. Per tile at 12288 rows
// (shader clock read at the phase boundaries): 9.5k cycles until the first
// chunk has landed, 136.4k in the main loop (131k of MFMA issue), 15.4k in
// the epilogue, 2k between tiles; the clock, read against the fixed 100 MHz
// counter, was 1.61 GHz there and 1.2-1.55 GHz at 256-1024 rows in the same
// run, so the chip's power limit, not the schedule, sets most of the time.
// A persistent form (one workgroup per CU looping over its tiles, the next
// tile's W_U chunks loaded during the epilogue) spilled 110-140 VGPRs per
// tile at 256 rows and measured 9-15% slower; rebuilt without spills at 128
// and 192 rows, it was still 0-2% slower there and 6-10% slower from 256
// rows up: workgroups walking fixed strides of jobs drift apart, where the
// dispatcher's window of consecutive jobs keeps the L2 sharing intact.
namespace big {
constexpr int TV = kBigTileVocab, KC = 64;
}  // namespace big

// s_waitcnt immediate: vmcnt <= n, lgkmcnt == 0, expcnt unconstrained
constexpr unsigned vm_lgkm_wait(int n) { return (unsigned)((n & 15) | ((n >> 4) << 14) | (7 << 4)); }

// NT: W_U loads non-temporal, for a single row tile (no other workgroup reads
// the same W_U chunk: 11% faster at 256 rows; with several row tiles sharing
// chunks through L2 it was 3% slower). HB: the hidden rows through buffer
// loads as well, with 32-bit byte offsets (the row source spans less than
// 2^31 bytes; 6% fewer main-loop cycles), else global_load_lds from 64-bit
// lane addresses.
template <int TR, bool NT, bool HB>
__global__ __launch_bounds__(256) void k_proj_bf16_big(
    const uint16_t* __restrict__ hidden, const uint16_t* __restrict__ w_u, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ n_ptr, float4* __restrict__ partials, int K, int B, int L, int d, int V,
    int nvt, int nrt, int split_rows, const uint16_t* __restrict__ xrows, const long long* __restrict__ rowoff,
    float scale) {
  using namespace big;
  static_assert(TV == 256 && (TR == 256 || TR == 192 || TR == 128), "wave layout below assumes 256 x TR");
  constexpr int NB = TR / 64;   // 32-row fragment blocks of the hidden rows per wave
  constexpr int BL = TR / 32;   // hidden-row load instructions per wave per chunk
  __shared__ __attribute__((aligned(1024))) uint16_t sa0[TV][KC], sa1[TV][KC], sa2[TV][KC];
  __shared__ __attribute__((aligned(1024))) uint16_t sb0[TR][KC], sb1[TR][KC];
  float4 (*red)[TR] = reinterpret_cast<float4 (*)[TR]>(&sa0[0][0]);   // used after the loop only
#define RPD_SA(X) ((X) == 0 ? sa0 : (X) == 1 ? sa1 : sa2)
#define RPD_SB(X) ((X) == 0 ? sb0 : sb1)

  int rt, vt;
  if (!map_job(blockIdx.x, nvt, nrt, split_rows, rt, vt)) return;
  const int R = rowoff ? *n_ptr : *n_ptr * K;   // an explicit row list counts rows, not positions
  const int r0 = rt * TR;
  if (r0 >= R) return;
  const int vb = (int)((long long)vt * V / nvt);
  const int ve = (int)((long long)(vt + 1) * V / nvt);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wv = wid & 1, wr = wid >> 1;

  // load sources: W_U instruction u of this wave covers tile rows 64*wid + 8*u
  // .. +8, hidden-row instruction u rows (TR/4)*wid + 8*u .. +8; lane l lands
  // at LDS piece (l & 7) of row (l >> 3) and fetches the global piece
  // (l & 7) ^ swizzle(row). Rows past the tile re-read its last vocabulary
  // row, rows past the last projected row re-read row r0 (both discarded at
  // the end).
  int pa[8];   // byte offsets of this lane's pieces from the tile's first W_U row (< 256 * d * 2)
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(w_u + (long long)vb * d), (short)0, (ve - vb) * d * 2, 0x00020000);
  // hidden-row sources: byte offsets from xsrc (HB) or addresses. Sized 8
  // (>= BL): an array sized by the template parameter, passed to the buffer
  // load builtin, made clang drop the kernel's host stub without a diagnostic.
  int pbo[8];
  const uint16_t* pb[8];
  const uint16_t* __restrict__ xsrc = xrows ? xrows : hidden;
  const __amdgpu_buffer_rsrc_t hrs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(xsrc), (short)0, 0x7fffffff, 0x00020000);
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int tr = 64 * wid + 8 * u + (lane >> 3);
    const int piece = (lane & 7) ^ ((tr >> 1) & 7);
    pa[u] = ((min(vb + tr, ve - 1) - vb) * d + piece * 8) * 2;
  }
#pragma unroll
  for (int u = 0; u < BL; ++u) {
    const int tr = (TR / 4) * wid + 8 * u + (lane >> 3);
    const int piece = (lane & 7) ^ ((tr >> 1) & 7);
    const int r = r0 + tr < R ? r0 + tr : r0;
    long long ob;
    if (xrows) {   // normalized rows, already in projected-row order
      ob = (long long)r * d + piece * 8;
    } else if (rowoff) {   // an explicit row list
      ob = rowoff[r] + piece * 8;
    } else {
      const int p = r / K, l = r - p * K;
      const int pos = rows[p];
      const int b = pos / L, i = pos - b * L;
      ob = (((long long)l * B + b) * L + i) * (long long)d + piece * 8;
    }
    pb[u] = xsrc + ob;
    pbo[u] = (int)(ob * 2);
  }
  // fragment reads: lane reads row base + (lane & 31), logical piece 2s + (lane >> 5)
  const int fr = lane & 31, fsw = (fr >> 1) & 7, fhi = lane >> 5;

  f32x16 acc[4][NB];
#pragma unroll
  for (int mv = 0; mv < 4; ++mv)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[mv][nb][q] = 0.f;
  u32x4 fa0[4], fb0[NB], fa1[4], fb1[NB];

#define RPD_ALOAD(XA, chunk) RPD_ALOAD_R(XA, chunk, 0, 8)
#define RPD_BLOAD(XB, chunk) RPD_BLOAD_R(XB, chunk, 0, BL)
#define RPD_ALOAD_R(XA, chunk, U0, U1)                                                                    \
  do {                                                                                                    \
    const long long k0_ = (long long)RPD_PCHUNK(chunk) * KC;                                              \
    _Pragma("unroll") for (int u_ = (U0); u_ < (U1); ++u_)                                               \
      __builtin_amdgcn_raw_ptr_buffer_load_lds(wrs,                                                        \
          (__attribute__((address_space(3))) void*)&RPD_SA(XA)[64 * wid + 8 * u_][0], 16, pa[u_],           \
          (int)(2 * k0_), 0, NT ? 2 : 0);                                                                  \
  } while (0)
#define RPD_BLOAD_R(XB, chunk, U0, U1)                                                                    \
  do {                                                                                                    \
    const long long k0_ = (long long)RPD_PCHUNK(chunk) * KC;                                              \
    _Pragma("unroll") for (int u_ = (U0); u_ < (U1); ++u_)                                               \
      if constexpr (HB)                                                                                   \
        __builtin_amdgcn_raw_ptr_buffer_load_lds(hrs,                                                      \
            (__attribute__((address_space(3))) void*)&RPD_SB(XB)[(TR / 4) * wid + 8 * u_][0], 16, pbo[u_],  \
            (int)(2 * k0_), 0, 0);                                                                         \
      else                                                                                                \
        __builtin_amdgcn_global_load_lds((const void*)(pb[u_] + k0_),                                     \
            (__attribute__((address_space(3))) void*)&RPD_SB(XB)[(TR / 4) * wid + 8 * u_][0], 16, 0, 0); \
  } while (0)
#define RPD_FRAGS(FA, FB, XA, XB, kstep)                                                                  \
  do {                                                                                                    \
    const int fc_ = 8 * ((2 * (kstep) + fhi) ^ fsw);                                                      \
    _Pragma("unroll") for (int m_ = 0; m_ < 4; ++m_)                                                     \
      FA[m_] = *reinterpret_cast<const u32x4*>(&RPD_SA(XA)[128 * wv + 32 * m_ + fr][fc_]);               \
    _Pragma("unroll") for (int m_ = 0; m_ < NB; ++m_)                                                    \
      FB[m_] = *reinterpret_cast<const u32x4*>(&RPD_SB(XB)[(TR / 2) * wr + 32 * m_ + fr][fc_]);          \
  } while (0)
#define RPD_MMA(FA, FB)                                                                                   \
  do {                                                                                                    \
    _Pragma("unroll") for (int mv_ = 0; mv_ < 4; ++mv_)                                                  \
    _Pragma("unroll") for (int nb_ = 0; nb_ < NB; ++nb_)                                                 \
      acc[mv_][nb_] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, FA[mv_]),        \
                                                               __builtin_bit_cast(bf16x8, FB[nb_]),        \
                                                               acc[mv_][nb_], 0, 0, 0);                   \
  } while (0)
  // the 4*NB MFMAs of a k-step with the 4 + NB fragment reads of the next one between the first of them
  // and NL global->LDS loads spread evenly over the step
#define RPD_MIX(NL)                                                                                       \
  do {                                                                                                    \
    _Pragma("unroll") for (int g_ = 0; g_ < 4 * NB; ++g_) {                                              \
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0); /* MFMA */                                       \
      if (g_ < 4 + NB) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0); /* LDS read */                  \
      if ((g_ * (NL)) % (4 * NB) < (NL)) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0); /* load */     \
    }                                                                                                     \
  } while (0)
  // Chunk c in A stage XA = c % 3 and B stage XB = c % 2 (fragments of its first k-step already in
  // fa0/fb0); XAP = (c + 2) % 3 and XB ^ 1 are chunk c-1's stages, freed at the previous barrier, and
  // XAN = (c + 1) % 3. A barrier frees a chunk's stages for the hidden rows of the chunk two ahead and
  // W_U of the chunk three ahead; those 8 + BL loads per wave are spread over four k-steps (the address
  // unit takes about 16 cycles per load instruction, and 64 of them in one k-step of 512 MFMA cycles
  // stalled the MFMAs): the first half of the hidden rows after the barrier, the second half in the
  // next chunk's first k-step, W_U in its second and third. So at a barrier the newest 8 loads (W_U of
  // chunk c+2) may still be in flight, and every earlier one (chunk c+1) has landed. Chunk 0 (FIRST)
  // issues no deferred loads: the prologue loaded chunks 1 and 2 whole.
#define RPD_CHUNK(c, XA, XB, XAN, XAP, FIRST)                                                             \
  do {                                                                                                    \
    __builtin_amdgcn_sched_barrier(0);                                                                    \
    RPD_FRAGS(fa1, fb1, XA, XB, 1);                                                                       \
    RPD_MMA(fa0, fb0);                                                                                    \
    if (!(FIRST)) RPD_BLOAD_R((XB) ^ 1, min((c) + 1, nchf - 1), BL / 2, BL);                              \
    RPD_MIX((FIRST) ? 0 : BL - BL / 2);                                                                   \
    __builtin_amdgcn_sched_barrier(0);                                                                    \
    RPD_FRAGS(fa0, fb0, XA, XB, 2);                                                                       \
    RPD_MMA(fa1, fb1);                                                                                    \
    if (!(FIRST)) RPD_ALOAD_R(XAP, min((c) + 2, nchf - 1), 0, 4);                                         \
    RPD_MIX((FIRST) ? 0 : 4);                                                                             \
    __builtin_amdgcn_sched_barrier(0);                                                                    \
    RPD_FRAGS(fa1, fb1, XA, XB, 3);                                                                       \
    RPD_MMA(fa0, fb0);                                                                                    \
    if (!(FIRST)) RPD_ALOAD_R(XAP, min((c) + 2, nchf - 1), 4, 8);                                         \
    RPD_MIX((FIRST) ? 0 : 4);                                                                             \
    __builtin_amdgcn_sched_barrier(0);                                                                    \
    __builtin_amdgcn_s_waitcnt(vm_lgkm_wait(8)); /* chunk c+1 landed (A of c+2 may be in flight) */      \
    __builtin_amdgcn_s_barrier();                                                                         \
    __builtin_amdgcn_sched_barrier(0);                                                                    \
    RPD_FRAGS(fa0, fb0, XAN, (XB) ^ 1, 0);                                                                \
    RPD_BLOAD_R(XB, min((c) + 2, nchf - 1), 0, BL / 2);                                                   \
    RPD_MMA(fa1, fb1);                                                                                    \
    RPD_MIX(BL / 2);                                                                                      \
    __builtin_amdgcn_sched_barrier(0);                                                                    \
  } while (0)

  // Chunks past the end repeat the last one (loaded, never multiplied). With a
  // single row tile (NT) the workgroups of XCD x (workgroup id mod 8) take
  // the full chunks in the order r, r+1, .., nchf-1, 0, .., r-1 with
  // r = x*nchf/8: the requests in flight on the eight XCDs then read eight
  // different columns of W_U (in plain order they all read one column and
  // crowd onto a few HBM channels on some boxes: 226 against 176 us at 104
  // rows, 253 against 203 at 192), while the workgroups of one XCD still
  // read the same hidden-row chunk at a time through its L2 (a rotation by
  // vocabulary tile cost 2-8% at 104-256 rows on boxes without the
  // crowding). Equal rows within a tile are summed in one order and tie
  // exactly; across tiles the reduction settles a near-tie in float64
  // (reduce_device.h). With several row tiles the plain order stays: the
  // workgroups of one row tile share its hidden rows through L2 only while
  // they read the same chunk (rotated, 7-8% slower from 1024 rows up).
  const int nchf = d / KC;
  const int rot = NT && nchf > 0 ? (int)(((long long)(blockIdx.x & 7) * nchf) / 8) : 0;
#define RPD_PCHUNK(c) ((c) + rot >= nchf ? (c) + rot - nchf : (c) + rot)
  if (nchf > 0) {
    RPD_ALOAD(0, 0);
    RPD_BLOAD(0, 0);
    RPD_ALOAD(1, min(1, nchf - 1));
    RPD_BLOAD(1, min(1, nchf - 1));
    RPD_ALOAD(2, min(2, nchf - 1));
    __builtin_amdgcn_s_waitcnt(vm_lgkm_wait(16 + BL));   // chunk 0 landed (A1, B1, A2 in flight)
    __builtin_amdgcn_s_barrier();
    RPD_FRAGS(fa0, fb0, 0, 0, 0);
    RPD_CHUNK(0, 0, 0, 1, 2, 1);
    int c = 1;
    for (; c + 6 <= nchf; c += 6) {   // chunk c + j in stages ((c + j) % 3, (c + j) % 2), c = 1 mod 6
      RPD_CHUNK(c, 1, 1, 2, 0, 0);
      RPD_CHUNK(c + 1, 2, 0, 0, 1, 0);
      RPD_CHUNK(c + 2, 0, 1, 1, 2, 0);
      RPD_CHUNK(c + 3, 1, 0, 2, 0, 0);
      RPD_CHUNK(c + 4, 2, 1, 0, 1, 0);
      RPD_CHUNK(c + 5, 0, 0, 1, 2, 0);
    }
    if (c < nchf) RPD_CHUNK(c, 1, 1, 2, 0, 0);
    if (c + 1 < nchf) RPD_CHUNK(c + 1, 2, 0, 0, 1, 0);
    if (c + 2 < nchf) RPD_CHUNK(c + 2, 0, 1, 1, 2, 0);
    if (c + 3 < nchf) RPD_CHUNK(c + 3, 1, 0, 2, 0, 0);
    if (c + 4 < nchf) RPD_CHUNK(c + 4, 2, 1, 0, 1, 0);
    __builtin_amdgcn_s_waitcnt(vm_lgkm_wait(0));    // no load outstanding past the loop
    __syncthreads();
  }
  if (d % KC != 0) {   // partial last chunk, zero-filled past d (d % 8 == 0: a piece is all in or all out)
    const long long k0 = (long long)nchf * KC;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int tr = 64 * wid + 8 * u + (lane >> 3);
      const int piece = (lane & 7) ^ ((tr >> 1) & 7);
      const bool in = k0 + piece * 8 < d;
      const u32x4 va = in ? *reinterpret_cast<const u32x4*>(reinterpret_cast<const char*>(w_u + (long long)vb * d) + 2 * k0 + pa[u])
                          : u32x4{0u, 0u, 0u, 0u};
      *reinterpret_cast<u32x4*>(&sa0[tr][(lane & 7) * 8]) = va;
    }
#pragma unroll
    for (int u = 0; u < BL; ++u) {
      const int tr = (TR / 4) * wid + 8 * u + (lane >> 3);
      const int piece = (lane & 7) ^ ((tr >> 1) & 7);
      const bool in = k0 + piece * 8 < d;
      const u32x4 vh = in ? *reinterpret_cast<const u32x4*>(pb[u] + k0) : u32x4{0u, 0u, 0u, 0u};
      *reinterpret_cast<u32x4*>(&sb0[tr][(lane & 7) * 8]) = vh;
    }
    __syncthreads();
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
      RPD_FRAGS(fa0, fb0, 0, 0, s4);
      RPD_MMA(fa0, fb0);
    }
  }
#undef RPD_CHUNK
#undef RPD_MIX
#undef RPD_MMA
#undef RPD_FRAGS
#undef RPD_ALOAD
#undef RPD_BLOAD
#undef RPD_ALOAD_R
#undef RPD_PCHUNK
#undef RPD_BLOAD_R
#undef RPD_SA
#undef RPD_SB

  __syncthreads();   // red aliases A stage 0
  // epilogue: lane holds projected row (TR/2)*wr + 32*nb + (lane & 31) against
  // vocabulary rows 128*wv + 32*mv + 8*(q >> 2) + 4*(lane >> 5) + (q & 3)
  if (ve - vb == TV) {
    // A full vocabulary tile: no entry to exclude. Each projected row's 64
    // raw accumulators in this lane take one max pass (3-input maxima that
    // propagate NaN and need no canonicalized inputs); the
    // scale is positive, so the lowest slot holding the raw maximum is the
    // argmax of the scaled logits (slots increase with the vocabulary
    // index). The sums are taken in base-2 units: t = (z - m) log2(e) in one
    // fma from the raw accumulator, e^(z-m) = 2^t, and T = ln(2) sum 2^t t.
    const float s2 = scale * 1.44269504088896340736f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      float mraw = acc[0][nb][0];
#pragma unroll
      for (int mv = 0; mv < 4; ++mv)
#pragma unroll
        for (int q = (mv == 0 ? 1 : 0); q < 16; q += 2) {
          if (q + 1 < 16)
            mraw = __builtin_elementwise_maximum(
                mraw, __builtin_elementwise_maximum(acc[mv][nb][q], acc[mv][nb][q + 1]));
          else
            mraw = __builtin_elementwise_maximum(mraw, acc[mv][nb][q]);
        }
      const float m2 = mraw * s2;
      int slot = 64;
      float Sp[4], Tp[4];
#pragma unroll
      for (int mv = 3; mv >= 0; --mv) {
        Sp[mv] = 0.f;
        Tp[mv] = 0.f;
#pragma unroll
        for (int q = 15; q >= 0; --q) {
          const float a = acc[mv][nb][q];
          slot = a == mraw ? 16 * mv + q : slot;
          const float t = __builtin_fmaf(a, s2, -m2);
          const float ex = __builtin_amdgcn_exp2f(t);
          Sp[mv] += ex;
          Tp[mv] = __builtin_fmaf(ex, t, Tp[mv]);
        }
      }
      Soft sst;
      sst.m = mraw * scale;
      sst.S = (Sp[0] + Sp[1]) + (Sp[2] + Sp[3]);
      sst.T = ((Tp[0] + Tp[1]) + (Tp[2] + Tp[3])) * 0.69314718055994530942f;
      sst.idx = (slot == 64 || mraw == -INFINITY)
                    ? INT_MAX
                    : vb + 128 * wv + 32 * (slot >> 4) + 8 * ((slot >> 2) & 3) + 4 * (lane >> 5) + (slot & 3);
      sst = soft_merge(sst, soft_shfl_xor(sst, 32));
      if (lane < 32) red[wv][(TR / 2) * wr + 32 * nb + lane] = soft_pack(sst);
    }
  } else {   // a ragged last tile: entries past ve are excluded
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
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
      if (lane < 32) red[wv][(TR / 2) * wr + 32 * nb + lane] = soft_pack(sst);
    }
  }
  __syncthreads();
  if (tid < TR) {   // one projected row per thread
    const int r = r0 + tid;
    if (r < R) {
      const Soft sres = soft_merge(soft_unpack(red[0][tid]), soft_unpack(red[1][tid]));
      partials[(long long)r * nvt + vt] = soft_pack(sres);
    }
  }
}

}  // namespace

hipError_t launch_proj_big(const Launch& a, hipStream_t s) {
  const bool nt = a.plan.nrt == 1;
  // the hidden rows, and the normalized rows (at most K * B * L of them), span less than 2^31 bytes
  const bool hb = (long long)a.K * a.B * a.L * a.d * 2 < (1ll << 31);
  decltype(&k_proj_bf16_big<256, false, false>) kernel;
  if (a.plan.rows_per_tile == 128)
    kernel = nt ? (hb ? k_proj_bf16_big<128, true, true> : k_proj_bf16_big<128, true, false>)
                : (hb ? k_proj_bf16_big<128, false, true> : k_proj_bf16_big<128, false, false>);
  else if (a.plan.rows_per_tile == 192)
    kernel = nt ? (hb ? k_proj_bf16_big<192, true, true> : k_proj_bf16_big<192, true, false>)
                : (hb ? k_proj_bf16_big<192, false, true> : k_proj_bf16_big<192, false, false>);
  else
    kernel = nt ? (hb ? k_proj_bf16_big<256, true, true> : k_proj_bf16_big<256, true, false>)
                : (hb ? k_proj_bf16_big<256, false, true> : k_proj_bf16_big<256, false, false>);
  hipLaunchKernelGGL(kernel, dim3(a.plan.grid), dim3(256), 0, s, static_cast<const uint16_t*>(a.hidden),
                     static_cast<const uint16_t*>(a.w_u), a.rows, a.n_masked, a.partials, a.K, a.B, a.L, a.d, a.V,
                     a.plan.nvt, a.plan.nrt, a.plan.split_rows, static_cast<const uint16_t*>(a.xrows), a.rowoff,
                     a.logit_scale);
  return hipGetLastError();
}

}  // namespace rpd
