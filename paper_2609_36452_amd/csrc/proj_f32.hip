// K1 projection for fp32 inputs (vector ALU).
#include "rpd_device.h"

namespace rpd {
namespace {

// fp32 inputs: 64 vocabulary rows (one per lane) x 16 projected rows (four
// per wave) per workgroup, fp32 FMA on the vector ALU through LDS tiles.
__global__ __launch_bounds__(256) void k_proj_f32(const float* __restrict__ hidden, const float* __restrict__ w_u,
                                                  const int32_t* __restrict__ rows,
                                                  const int32_t* __restrict__ n_ptr, float4* __restrict__ partials,
                                                  int K, int B, int L, int d, int V, int nvt,
                                                  const float* __restrict__ xrows,
                                                  const long long* __restrict__ rowoff, float scale) {
  __shared__ float ws[64][33];
  __shared__ float xsm[16][33];
  __shared__ long long xoff[16];
  const int vt = blockIdx.x % nvt, rt = blockIdx.x / nvt;
  const int R = rowoff ? *n_ptr : *n_ptr * K;   // an explicit row list counts rows, not positions
  const int r0 = rt * 16;
  if (r0 >= R) return;
  const int vb = (int)((long long)vt * V / nvt);
  const int ve = (int)((long long)(vt + 1) * V / nvt);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  if (tid < 16) {
    const int r = r0 + tid;
    long long off = -1;
    if (r < R) {
      if (xrows) {   // normalized rows, already in projected-row order
        off = (long long)r * d;
      } else if (rowoff) {   // an explicit row list
        off = rowoff[r];
      } else {
        const int p = r / K, l = r - p * K;
        const int pos = rows[p];
        const int b = pos / L, i = pos - b * L;
        off = (((long long)l * B + b) * L + i) * (long long)d;
      }
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
      xsm[row][kk] = (off >= 0 && k0 + kk < d) ? (xrows ? xrows : hidden)[off + k0 + kk] : 0.f;
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
    float z[1] = {acc[j] * scale};
    int vi[1] = {v};
    bool ok[1] = {v < ve};
    Soft st = soft_from_values(z, vi, ok);
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) st = soft_merge(st, soft_shfl_xor(st, m));
    const int r = r0 + wid * 4 + j;
    if (lane == 0 && r < R) partials[(long long)r * nvt + vt] = soft_pack(st);
  }
}

}  // namespace

hipError_t launch_proj_f32(const Launch& a, hipStream_t s) {
  hipLaunchKernelGGL(k_proj_f32, dim3(a.plan.grid), dim3(256), 0, s, static_cast<const float*>(a.hidden),
                     static_cast<const float*>(a.w_u), a.rows, a.n_masked, a.partials, a.K, a.B, a.L, a.d, a.V,
                     a.plan.nvt, static_cast<const float*>(a.xrows), a.rowoff, a.logit_scale);
  return hipGetLastError();
}

}  // namespace rpd
