// Register -> LDS staging of the gathered hidden-state rows, shared by the
// register-streaming projection kernels (proj_small.hip, proj_mid.hip).
#pragma once

#include "rpd_device.h"

namespace rpd {
namespace {

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

}  // namespace
}  // namespace rpd
