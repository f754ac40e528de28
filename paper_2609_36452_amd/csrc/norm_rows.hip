// The model's final normalization applied to the projected rows before the
// output head (Appendix A.2 "Intermediate-layer readout", A.6 "Layerwise
// projection"): RMS normalization g * x / sqrt(mean(x^2) + eps) of every
// (masked position, layer) row, in the compacted row order, written to the
// workspace; the projection then reads these rows instead of gathering from
// the hidden states. The final layer's native state is copied unchanged
// unless norm_final is set.
//
// The sum of squares, the scale and the product are evaluated in float64
// (each x^2 of a bf16 value is exact there), and the result is rounded once
// to the input type, round to nearest with ties to even, so the normalized
// rows the output head sees are reproducible to the last bit.
#include "rpd_device.h"

namespace rpd {
namespace {

__device__ __forceinline__ double load_f64(const uint16_t* p, long long k) {
  return (double)__uint_as_float((uint32_t)p[k] << 16);
}
__device__ __forceinline__ double load_f64(const float* p, long long k) { return (double)p[k]; }

// float64 -> bfloat16 bits, round to nearest, ties to even, in one step
// (8 significant bits; below 2^-126 the bfloat16 grid is 2^-133)
__device__ __forceinline__ uint16_t f64_to_bf16(double v) {
  const unsigned long long u = (unsigned long long)__double_as_longlong(v);
  const uint16_t sign = (uint16_t)((u >> 63) << 15);
  const int e = (int)((u >> 52) & 0x7FF);
  const unsigned long long m = u & ((1ull << 52) - 1);
  if (e == 0x7FF) return (uint16_t)(sign | 0x7F80 | (m ? 0x40 : 0));   // inf, NaN
  int be = e - 1023 + 127;
  if (be <= 0) {   // bfloat16 subnormal (or zero): a multiple of 2^-133
    const double q = rint(fabs(v) * 0x1p133);                        // ties to even
    return (uint16_t)(sign | (uint16_t)q);                           // q == 128 is the smallest normal
  }
  unsigned long long keep = m >> 45;
  const unsigned long long rem = m & ((1ull << 45) - 1), half = 1ull << 44;
  if (rem > half || (rem == half && (keep & 1))) ++keep;
  if (keep == 128) {
    keep = 0;
    ++be;
  }
  if (be >= 255) return (uint16_t)(sign | 0x7F80);
  return (uint16_t)(sign | (be << 7) | keep);
}
__device__ __forceinline__ void store_f64(uint16_t* p, long long k, double v) { p[k] = f64_to_bf16(v); }
__device__ __forceinline__ void store_f64(float* p, long long k, double v) { p[k] = (float)v; }

constexpr int kNormThreads = 256;

// one workgroup per projected row r = p*K + l (r < n*K)
// With an explicit row list (rowoff, a lazy pass over layer pass_layer),
// row r < *n_ptr is hidden + rowoff[r]; otherwise rows are gathered for
// r < *n_ptr * K.
template <typename T>
__global__ __launch_bounds__(kNormThreads) void k_norm_rows(const T* __restrict__ hidden, const T* __restrict__ g,
                                                           const int32_t* __restrict__ rows,
                                                           const int32_t* __restrict__ n_ptr, T* __restrict__ xrows,
                                                           int K, int B, int L, int d, float eps, int norm_final,
                                                           const long long* __restrict__ rowoff, int pass_layer) {
  __shared__ double s_ss[kNormThreads / 64];
  const int r = blockIdx.x;
  int l;
  const T* src;
  if (rowoff) {
    if (r >= *n_ptr) return;
    l = pass_layer;
    src = hidden + rowoff[r];
  } else {
    if (r >= *n_ptr * K) return;
    const int p = r / K;
    l = r - p * K;
    const int pos = rows[p];
    const int b = pos / L, i = pos - b * L;
    src = hidden + (((long long)l * B + b) * L + i) * (long long)d;
  }
  T* dst = xrows + (long long)r * d;
  if (l == K - 1 && !norm_final) {
    for (int k = threadIdx.x; k < d; k += kNormThreads) dst[k] = src[k];
    return;
  }
  double ss = 0.0;
  for (int k = threadIdx.x; k < d; k += kNormThreads) {
    const double x = load_f64(src, k);
    ss += x * x;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m);
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  if (lane == 0) s_ss[wid] = ss;
  __syncthreads();
  ss = 0.0;
#pragma unroll
  for (int w = 0; w < kNormThreads / 64; ++w) ss += s_ss[w];
  const double den = sqrt(ss / (double)d + (double)eps);
  for (int k = threadIdx.x; k < d; k += kNormThreads) store_f64(dst, k, load_f64(g, k) * load_f64(src, k) / den);
}

}  // namespace

hipError_t launch_norm_rows(const Launch& a, hipStream_t s) {
  if (a.max_masked <= 0) return hipSuccess;
  // an explicit row list holds max_masked rows
  const dim3 grid((unsigned)(a.rowoff ? (long long)a.max_masked : (long long)a.K * a.max_masked));
  const int K = a.K;
  if (a.plan.variant == PROJ_F32)
    hipLaunchKernelGGL(k_norm_rows<float>, grid, dim3(kNormThreads), 0, s, static_cast<const float*>(a.hidden),
                       static_cast<const float*>(a.norm_weight), a.rows, a.n_masked, static_cast<float*>(a.xrows),
                       K, a.B, a.L, a.d, a.norm_eps, a.norm_final, a.rowoff, a.pass_layer);
  else
    hipLaunchKernelGGL(k_norm_rows<uint16_t>, grid, dim3(kNormThreads), 0, s,
                       static_cast<const uint16_t*>(a.hidden), static_cast<const uint16_t*>(a.norm_weight), a.rows,
                       a.n_masked, static_cast<uint16_t*>(a.xrows), K, a.B, a.L, a.d, a.norm_eps, a.norm_final,
                       a.rowoff, a.pass_layer);
  return hipGetLastError();
}

}  // namespace rpd
