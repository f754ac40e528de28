// Lazy layerwise projection (Appendix A.6 "Layerwise projection"): a
// position's intermediate layers are projected from the final one down, and
// no further than its first disagreeing layer, where its agreement suffix
// (Eq. 2) is known.
//
// The host drives one pass per layer, from the final layer down:
//   pass 0      the final layer of every masked position;
//   pass t > 0  layer K-1-t of the positions still "alive": those that walk
//               (every position with a finite final confidence with
//               RPD_PARAM_LAZY_ALL, the procedure as the paper states it;
//               otherwise only those in the band theta_c <= c < theta_h, the
//               only ones whose candidacy the stability test decides, Eq. 5,
//               a further saving that leaves every decision unchanged) and
//               whose layers K-t .. K-1 all agreed with the final token.
// Each pass is the ordinary projection over an explicit list of rows (a
// table of element offsets into the hidden states, or normalized rows),
// followed by k_lazy_reduce (merge the tile states, update each position's
// suffix length and peak probability) and k_lazy_next (list the positions
// still alive with the row offsets of the next layer, and their count; the
// host plans the next pass for a bound on it or reads it back). k_lazy_score then
// evaluates Eq. 2-5 from the per-position state, with persistence exact for
// every position that walked; elsewhere stability is not evaluated
// (persistence -1, drop and stability NaN). The commitment follows as usual.
#include "reduce_device.h"

namespace rpd {
namespace {

// one wave per row j < m of the pass (layer l): statistics of the row (with
// exact argmax ties resolved after a streaming projection, whose tiles sum
// in different orders: bit c of tie_cls for size class c), then the update
// of its position's state
__global__ __launch_bounds__(64) void k_lazy_reduce(const float4* __restrict__ partials, int nvt0, int nvt1,
                                                    int nvt2, int t0, int t1, TieArgs ta, int tie_cls,
                                                    const uint16_t* __restrict__ hidden,
                                                    const uint16_t* __restrict__ xrows, int d,
                                                    const int32_t* __restrict__ m_ptr, LazyState st, int l, int K,
                                                    int B, int L, const int32_t* __restrict__ rows, float theta_c,
                                                    float theta_h, int walk_all, int32_t* __restrict__ layer_argmax,
                                                    float* __restrict__ layer_conf, float* __restrict__ layer_entropy) {
  const int j = blockIdx.x, lane = threadIdx.x;
  // the row's position is loaded with the count (j < m_cap stays inside act),
  // and the position's state with the tile states (unused in the final-layer
  // pass): two memory round trips before the update instead of four. A
  // workgroup beyond the count (most of them in the passes of the size
  // classes the count is not in) exits before reading anything else.
  const int m = *m_ptr;
  const int p = st.act[j];
  if (j >= m) return;
  // the partials follow the plan of the size class the count is in (<= t0,
  // <= t1, above; one plan when the pass was launched once)
  const int cls = m <= t0 ? 0 : (m <= t1 ? 1 : 2);
  const int nvt = cls == 0 ? nvt0 : (cls == 1 ? nvt1 : nvt2);
  const int y_prev = st.y[p], k_prev = st.k[p];
  const float pmax_prev = st.pmax[p];
  const int pos = layer_argmax ? rows[p] : 0;
  const float4* src = partials + (long long)j * nvt;
  float4 keep[8];
  Soft s = wave_merge_row(src, nvt, lane, keep);
  if ((tie_cls >> cls) & 1) {
    const uint16_t* x = xrows ? xrows + (long long)j * d : hidden + st.rowoff[j];
    s.idx = resolve_tie(s, keep, src, nvt, ta, x, lane);
  }
  if (lane != 0) return;
  const int y = (s.idx == INT_MAX) ? -1 : s.idx;
  const float c = 1.0f / s.S;
  const float h = (s.S != s.S) ? s.S : fmaxf(logf(s.S) - s.T / s.S, 0.0f);
  if (l == K - 1) {
    st.y[p] = y;
    st.c[p] = c;
    st.h[p] = h;
    st.k[p] = 1;
    st.pmax[p] = c;
    // NaN fails both tests
    st.alive[p] = (K > 1 && (walk_all ? c == c : (c >= theta_c && c < theta_h))) ? 1 : 0;
  } else if (y == y_prev) {
    st.k[p] = k_prev + 1;
    st.pmax[p] = fmaxf(pmax_prev, c);
    st.alive[p] = l > 0 ? 1 : 0;
  } else {
    st.alive[p] = 0;
  }
  st.depth[p] = K - l;
  if (layer_argmax) {
    const int b = pos / L, i = pos - b * L;
    const long long ol = ((long long)l * B + b) * L + i;
    layer_argmax[ol] = y;
    layer_conf[ol] = c;
    layer_entropy[ol] = h;
  }
}

// one workgroup: the positions still alive, in order, with the element
// offsets of their layer-l rows; the count goes to *m_out and, as the count
// of the one size class (<= t0, <= t1, above) it falls in, to tier[0..2]
// (the others get 0). The final-layer pass, every masked position, is
// listed by the compaction.
constexpr int kLazyNextThreads = 1024;
__global__ __launch_bounds__(kLazyNextThreads) void k_lazy_next(const int32_t* __restrict__ n_ptr, LazyState st,
                                                                const int32_t* __restrict__ rows, int cap, int l,
                                                                int B, int L, int d,
                                                                int32_t* __restrict__ m_out, int32_t* __restrict__ tier,
                                                                int t0, int t1) {
  __shared__ int wsum[kLazyNextThreads / 64];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  // the first chunk's state and row are loaded with the count (p < cap stays
  // inside both buffers; entries at or beyond the count are not used)
  const bool in0 = (int)threadIdx.x < cap;
  const int alive0 = in0 ? st.alive[threadIdx.x] : 0;
  const int row0 = in0 ? rows[threadIdx.x] : 0;
  const int n = *n_ptr;
  int carry = 0;
  for (int base = 0; base < n; base += blockDim.x) {
    const int p = base + threadIdx.x;
    const int alive = base == 0 ? alive0 : (p < n ? st.alive[p] : 0);
    const bool f = p < n && alive != 0;
    const unsigned long long bal = __ballot(f);
    const int before = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) wsum[wid] = __popcll(bal);
    __syncthreads();
    int off = 0, tot = 0;
    for (int w = 0; w < nw; ++w) {
      const int c = wsum[w];
      off += (w < wid) ? c : 0;
      tot += c;
    }
    if (f) {
      const int j = carry + off + before;
      const int pos = base == 0 ? row0 : rows[p];
      const int b = pos / L, i = pos - b * L;
      st.act[j] = p;
      st.rowoff[j] = (((long long)l * B + b) * L + i) * (long long)d;
    }
    carry += tot;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    *m_out = carry;
    tier[0] = carry <= t0 ? carry : 0;
    tier[1] = carry > t0 && carry <= t1 ? carry : 0;
    tier[2] = carry > t1 ? carry : 0;
  }
}

// Eq. 2-5 from the per-position state, one thread per masked position
__global__ __launch_bounds__(256) void k_lazy_score(const int32_t* __restrict__ n_ptr, LazyState st,
                                                    const int32_t* __restrict__ rows, LazyScoreArgs a) {
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= *n_ptr) return;
  const int pos = rows[p];
  const int b = pos / a.L, i = pos - b * a.L;
  const long long o = (long long)b * a.L + i;
  const float c = st.c[p];
  const bool band = c >= a.theta_c && c < a.theta_h;
  const bool walked = a.walk_all ? c == c : band;
  const bool high = c >= a.theta_h;
  float r = NAN, s = NAN;
  int k = -1;
  bool stab = false;
  if (walked) {
    k = st.k[p];
    r = st.pmax[p] - c;
    s = fmaf(-a.w, r, (float)min(k, a.k_max));
    stab = band && s >= a.theta_s;
  }
  a.token[o] = st.y[p];
  a.entropy[o] = st.h[p];
  a.confidence[o] = c;
  a.persistence[o] = k;
  a.drop[o] = r;
  a.stability[o] = s;
  a.flags[o] = (uint8_t)((high || stab ? kFlagCandidate : 0u) | (high ? kFlagHigh : 0u) | (stab ? kFlagStable : 0u));
  if (a.layer_argmax)   // layers never projected
    for (int l = 0; l < a.K - st.depth[p]; ++l) {
      const long long ol = ((long long)l * a.B + b) * a.L + i;
      a.layer_argmax[ol] = -1;
      a.layer_conf[ol] = NAN;
      a.layer_entropy[ol] = NAN;
    }
}

}  // namespace

hipError_t launch_lazy_next(const Launch& a, int l, hipStream_t s) {
  hipLaunchKernelGGL(k_lazy_next, dim3(1), dim3(kLazyNextThreads), 0, s, a.n_masked, a.lazy, a.rows, a.max_masked, l,
                     a.B, a.L, a.d, a.lazy.m, a.lazy.tier, kStreamMaxRows, kBigTileRowsMid);
  return hipGetLastError();
}

hipError_t launch_lazy_reduce(const Launch& a, int l, int m_cap, const ProjPlan* class_plans, hipStream_t s) {
  if (m_cap <= 0) return hipSuccess;
  const ProjPlan* pl[3] = {&a.plan, &a.plan, &a.plan};
  if (class_plans)
    for (int c = 0; c < 3; ++c) pl[c] = class_plans + c;
  int tie_cls = 0;
  for (int c = 0; c < 3; ++c) tie_cls |= tie_args(a, *pl[c]).w_u ? 1 << c : 0;
  const TieArgs ta{static_cast<const uint16_t*>(a.w_u), a.d, a.logit_scale};
  hipLaunchKernelGGL(k_lazy_reduce, dim3(m_cap), dim3(64), 0, s, a.partials, pl[0]->nvt, pl[1]->nvt, pl[2]->nvt,
                     kStreamMaxRows, kBigTileRowsMid, ta, tie_cls, static_cast<const uint16_t*>(a.hidden),
                     static_cast<const uint16_t*>(a.xrows), a.d, a.n_masked, a.lazy, l, a.K,
                     a.B, a.L, a.rows, a.theta_c, a.theta_h, a.lazy_all ? 1 : 0, a.layer_argmax, a.layer_conf,
                     a.layer_entropy);
  return hipGetLastError();
}

hipError_t launch_lazy_score(const Launch& a, hipStream_t s) {
  if (a.max_masked <= 0) return hipSuccess;
  LazyScoreArgs sa{a.K,          a.B,          a.L,         a.theta_h,     a.theta_c,    a.theta_s,
                   a.w,          a.k_max,      a.lazy_all ? 1 : 0,        a.token,      a.entropy,
                   a.confidence, a.persistence, a.drop,     a.stability,   a.flags,      a.layer_argmax,
                   a.layer_conf, a.layer_entropy};
  hipLaunchKernelGGL(k_lazy_score, dim3((unsigned)((a.max_masked + 255) / 256)), dim3(256), 0, s, a.n_masked,
                     a.lazy, a.rows, sa);
  return hipGetLastError();
}

}  // namespace rpd
