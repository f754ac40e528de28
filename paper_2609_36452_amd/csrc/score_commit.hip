// K0 masked-position compaction, K2 cross-tile reduction with the
// layerwise stability test (Eq. 2-5), K3 budgeted commitment with the
// progress fallback (Section 3.2), and their launchers.
#include <algorithm>

#include "reduce_device.h"

namespace rpd {
namespace {

// ------------------------------------------------------------ K0 compact --

// With lazy projection the compaction also lists the first pass (the final
// layer of every masked position, in order): act, the rows' element offsets,
// the count and its size class (<= t0, <= t1, above) as k_lazy_next writes
// them for the later passes.
struct FirstPassList {
  int32_t* act;          // NULL: no listing
  long long* rowoff;
  int32_t* m;
  int32_t* tier;
  long long layer_off;   // (K-1) * B * L: the final layer's first row
  int d, t0, t1;
};

__global__ __launch_bounds__(1024) void k_compact(const uint8_t* __restrict__ mask, int BL, int cap,
                                                   int32_t* __restrict__ rows, int32_t* __restrict__ n_out,
                                                   int32_t* __restrict__ dev_status,
                                                   int32_t* __restrict__ user_status, FirstPassList fp) {
  __shared__ int wsum[16];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int carry = 0;
  for (int base = 0; base < BL; base += blockDim.x) {
    const int i = base + threadIdx.x;
    const int f = (i < BL && mask[i] != 0) ? 1 : 0;
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
    const int pos = carry + off + before;
    if (f && pos < cap) {
      rows[pos] = i;
      if (fp.act) {
        fp.act[pos] = pos;
        fp.rowoff[pos] = (fp.layer_off + i) * fp.d;
      }
    }
    carry += tot;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    int st = 0, n = carry;
    if (n > cap) {
      st |= 1;
      n = cap;
    }
    *n_out = n;
    *dev_status = st;
    if (user_status) *user_status = st;
    if (fp.act) {
      *fp.m = n;
      fp.tier[0] = n <= fp.t0 ? n : 0;
      fp.tier[1] = n > fp.t0 && n <= fp.t1 ? n : 0;
      fp.tier[2] = n > fp.t1 ? n : 0;
    }
  }
}

// ------------------------------------------------------ scoring (Eq. 2-5) --

__device__ __forceinline__ float stability_score(int k_i, float r_i, int k_max, float w) {
  return fmaf(-w, r_i, (float)min(k_i, k_max));
}

__device__ __forceinline__ unsigned route_flags(float c, float s, float theta_h, float theta_c, float theta_s) {
  const bool high = c >= theta_h;
  const bool stab = (c >= theta_c) && (c < theta_h) && (s >= theta_s);
  return (high || stab ? kFlagCandidate : 0u) | (high ? kFlagHigh : 0u) | (stab ? kFlagStable : 0u);
}

struct ScoreArgs {
  int K, B, L;
  float theta_h, theta_c, theta_s, w;
  int k_max;
  int32_t* token;
  float* entropy;
  float* confidence;
  int32_t* persistence;
  float* drop;
  float* stability;
  uint8_t* flags;
  int32_t* layer_argmax;
  float* layer_conf;
  float* layer_entropy;
};

// One workgroup of four waves per masked position. Wave w merges the
// vocab-tile states of layers w, w+4, ...: each lane folds tiles lane,
// lane+64, ... in tile order (loads batched four at a time), then a fixed
// xor butterfly combines the lanes. Wave 0 then evaluates persistence, drop
// and stability with one lane per layer.
constexpr int kReduceWaves = 4;

// argmax (-1 if none), top probability 1/S and entropy ln S - T/S (Eq. 1) of
// a merged state; NaN stays visible in the entropy
__device__ __forceinline__ void state_stats(const Soft& s, int& y, float& c, float& h) {
  const float e = fmaxf(logf(s.S) - s.T / s.S, 0.0f);
  y = (s.idx == INT_MAX) ? -1 : s.idx;
  c = 1.0f / s.S;
  h = (s.S != s.S) ? s.S : e;
}


// Eq. 2-5 for one position from its per-layer argmax / top probability /
// entropy (layer l at offset l * stride), evaluated sequentially from the
// final layer down the agreement suffix. Inside the suffix the final token is
// each layer's argmax, so its probability there is that layer's top
// probability (Eq. 3). Same results as the wave-parallel form in
// k_reduce_score (the maximum is exact in any order).
struct Scored {
  int y, k;
  float c, h, r, s;
  unsigned flags;
};
template <typename TY, typename TF>
__device__ __forceinline__ Scored score_layers(const TY* y, const TF* c, const TF* h, long long stride,
                                              const ScoreArgs& a) {
  Scored o;
  o.y = y[(long long)(a.K - 1) * stride];
  o.c = c[(long long)(a.K - 1) * stride];
  o.h = h[(long long)(a.K - 1) * stride];
  int k_i = 1;
  float pk = o.c;
  for (int l = a.K - 2; l >= 0; --l) {
    if (y[(long long)l * stride] != o.y) break;
    ++k_i;
    pk = fmaxf(pk, c[(long long)l * stride]);
  }
  o.k = k_i;
  o.r = pk - o.c;
  o.s = stability_score(k_i, o.r, a.k_max, a.w);
  o.flags = route_flags(o.c, o.s, a.theta_h, a.theta_c, a.theta_s);
  return o;
}

__device__ __forceinline__ void write_scored(const ScoreArgs& a, long long o, const Scored& sc) {
  a.token[o] = sc.y;
  a.entropy[o] = sc.h;
  a.confidence[o] = sc.c;
  a.persistence[o] = sc.k;
  a.drop[o] = sc.r;
  a.stability[o] = sc.s;
  a.flags[o] = (uint8_t)sc.flags;
}

// Scoring from caller-supplied per-layer statistics, one thread per canvas
// position (same formulas as k_reduce_score, evaluated sequentially).
__global__ __launch_bounds__(256) void k_gate_score(const uint8_t* __restrict__ mask,
                                                     const int32_t* __restrict__ l_y,
                                                     const float* __restrict__ l_c,
                                                     const float* __restrict__ l_h, ScoreArgs a) {
  const long long BL = (long long)a.B * a.L;
  const long long o = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (o >= BL || mask[o] == 0) return;
  const Scored sc = score_layers(l_y + o, l_c + o, l_h + o, BL, a);
  write_scored(a, o, sc);
}

// --------------------------------------------------- commitment (Sec. 3.2) --

constexpr int kCommitThreads = 1024;

// two exclusive prefix sums over the workgroup in thread order (a fixed
// tree order: wave scans, then a scan of the wave totals); va / vb are
// replaced by their prefixes, tota / totb receive the sums
template <typename TA, typename TB>
__device__ __forceinline__ void block_exclusive_scan2(TA& va, TB& vb, TA* sha, TB* shb, TA& tota, TB& totb) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
  TA xa = va;
  TB xb = vb;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const TA ya = __shfl_up(xa, o);
    const TB yb = __shfl_up(xb, o);
    if (lane >= o) {
      xa = xa + ya;
      xb = xb + yb;
    }
  }
  if (lane == 63) {
    sha[wid] = xa;
    shb[wid] = xb;
  }
  __syncthreads();
  if (wid == 0) {
    TA sa = (lane < nw) ? sha[lane] : TA(0);
    TB sb = (lane < nw) ? shb[lane] : TB(0);
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const TA ya = __shfl_up(sa, o);
      const TB yb = __shfl_up(sb, o);
      if (lane >= o) {
        sa = sa + ya;
        sb = sb + yb;
      }
    }
    if (lane < nw) {
      sha[32 + lane] = sa;
      shb[32 + lane] = sb;
    }
  }
  __syncthreads();
  const TA wa = (wid == 0) ? TA(0) : sha[32 + wid - 1];
  const TB wb = (wid == 0) ? TB(0) : shb[32 + wid - 1];
  tota = sha[32 + nw - 1];
  totb = shb[32 + nw - 1];
  va = wa + xa - va;
  vb = wb + xb - vb;
  __syncthreads();
}

struct CommitArgs {
  int B, L;
  float beta;
  int window;
  int block;   // 0: full RPD; > 0: RPD-block with blocks of this many positions
  uint8_t* commit;
  int32_t* token;
  float* entropy;
  float* confidence;
  int32_t* persistence;
  float* drop;
  float* stability;
  uint8_t* flags;
  float* upstream_entropy;
  int32_t* n_commit;
};

// Where the commitment reads a masked position's scoring results (the
// output arrays, written by the scoring).
struct GlobalScores {
  const uint8_t* flags;
  const float* entropy;
  const float* confidence;
  __device__ unsigned flag(long long o) const { return flags[o]; }
  __device__ float ent(long long o) const { return entropy[o]; }
  __device__ float conf(long long o) const { return confidence[o]; }
};

// The commitment of sequence b by the whole workgroup. N_i = entropy summed
// over earlier masked non-candidates; a candidate is committed iff
// N_i <= beta, which is exactly the left-to-right construction of the paper
// (every earlier candidate of an accepted position is accepted, so the
// positions left out before it are the non-candidates; a rejected
// candidate's sum only grows). E_i (reported) is the entropy over earlier
// masked positions not committed. Without any commit, the most confident of
// the first `window` masked positions is committed (lowest index on ties;
// NaN confidences never win). Unmasked positions receive the sentinels.
template <class Scores>
__device__ __forceinline__ void commit_sequence(const uint8_t* __restrict__ mask, const CommitArgs& a, int b,
                                                const Scores& sc) {
  __shared__ float shf[64], shf2[64];
  __shared__ int shi[64], shi2[64];
  __shared__ float red_c[16];
  __shared__ int red_i[16];
  const long long base = (long long)b * a.L;
  // RPD-block: the active block is the run of a.block positions holding the
  // first masked position of the sequence
  int blo = 0, bhi = 0;
  if (a.block > 0) {
    int first = INT_MAX;
    for (int c0 = 0; c0 < a.L && first == INT_MAX; c0 += blockDim.x) {
      const int i = c0 + threadIdx.x;
      int f = (i < a.L && mask[base + i] != 0) ? i : INT_MAX;
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) f = min(f, __shfl_xor(f, m));
      if ((threadIdx.x & 63) == 0) shi[threadIdx.x >> 6] = f;
      __syncthreads();
      for (int w = 0; w < (int)(blockDim.x >> 6); ++w) first = min(first, shi[w]);
      __syncthreads();
    }
    if (first != INT_MAX) {
      blo = first / a.block * a.block;
      bhi = blo + a.block;
    }
  }
  float carryN = 0.f, carryE = 0.f;
  int carryM = 0, ncommit = 0;
  float best_c = -INFINITY;
  int best_i = INT_MAX;
  for (int c0 = 0; c0 < a.L; c0 += blockDim.x) {
    const int i = c0 + threadIdx.x;
    const bool in = i < a.L;
    const long long o = base + i;
    // loads issued together (entries of unmasked positions are read and ignored)
    const bool masked = in && mask[o] != 0;
    const unsigned fl_in = in ? sc.flag(o) : 0u;
    const float H_in = in ? sc.ent(o) : 0.f;
    const float c_in = in ? sc.conf(o) : 0.f;
    const unsigned fl = masked ? fl_in : 0u;
    const bool cand = (fl & kFlagCandidate) != 0;
    const float H = masked ? H_in : 0.f;
    // masked rank and N_i in one pass, then E_i and the commit count
    int rank = masked ? 1 : 0, totM;
    float N_i = (masked && !cand) ? H : 0.f, totN;
    block_exclusive_scan2<int, float>(rank, N_i, shi, shf, totM, totN);
    rank += carryM;
    N_i += carryN;
    const bool in_block = i >= blo && i < bhi;
    const bool com = masked && cand && (a.block > 0 ? in_block : (N_i <= a.beta));
    float E_i = (masked && !com) ? H : 0.f, totE;
    int ncom_before = com ? 1 : 0, ncom_chunk;
    block_exclusive_scan2<float, int>(E_i, ncom_before, shf2, shi2, totE, ncom_chunk);
    E_i += carryE;
    if (in) {
      if (masked) {
        a.commit[o] = com ? 1 : 0;
        a.flags[o] = (uint8_t)(fl | (com ? kFlagCommitted : 0u));
        a.upstream_entropy[o] = E_i;
        if (a.block > 0 ? in_block : (rank < a.window)) {
          const float cv = (c_in != c_in) ? -INFINITY : c_in;
          if (cv > best_c || (cv == best_c && i < best_i)) {
            best_c = cv;
            best_i = i;
          }
        }
      } else {
        a.commit[o] = 0;
        a.token[o] = -1;
        a.entropy[o] = 0.f;
        a.confidence[o] = 0.f;
        a.persistence[o] = 0;
        a.drop[o] = 0.f;
        a.stability[o] = 0.f;
        a.flags[o] = 0;
        a.upstream_entropy[o] = 0.f;
      }
    }
    carryN += totN;
    carryE += totE;
    carryM += totM;
    ncommit += ncom_chunk;
  }
  if (ncommit == 0 && carryM > 0) {
    // workgroup argmax of (confidence, -index) over the window
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const float oc = __shfl_xor(best_c, m);
      const int oi = __shfl_xor(best_i, m);
      if (oc > best_c || (oc == best_c && oi < best_i)) {
        best_c = oc;
        best_i = oi;
      }
    }
    if (lane == 0) {
      red_c[wid] = best_c;
      red_i[wid] = best_i;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      float bc = red_c[0];
      int bi = red_i[0];
      for (int w = 1; w < nw; ++w)
        if (red_c[w] > bc || (red_c[w] == bc && red_i[w] < bi)) {
          bc = red_c[w];
          bi = red_i[w];
        }
      if (bi != INT_MAX) {   // the window (or the active block) always holds a masked position here
        const long long o = base + bi;
        a.commit[o] = 1;
        a.flags[o] = (uint8_t)(a.flags[o] | kFlagCommitted | kFlagFallback);
        ncommit = 1;
      }
    }
  }
  if (threadIdx.x == 0) a.n_commit[b] = ncommit;
}

// K3 alone: one workgroup per sequence, scoring results from the outputs
__global__ __launch_bounds__(kCommitThreads) void k_commit(const uint8_t* __restrict__ mask, CommitArgs a) {
  commit_sequence(mask, a, blockIdx.x, GlobalScores{a.flags, a.entropy, a.confidence});
}

// K2: one workgroup of four waves per masked position. Wave w merges the
// vocab-tile states of layers w, w+4, ... (wave_merge_row) and, after a
// projection whose tiles sum in different orders, resolves exact argmax
// ties (resolve_tie; ta.w_u NULL otherwise); wave 0 then evaluates
// persistence, drop and stability with one lane per layer. The
// commitment (K3) follows as its own launch: handing it to the last
// workgroup to finish instead needs a device-scope release and acquire in
// every workgroup (an L2 write-back and invalidate each), which measured
// slower than the launch.
__global__ __launch_bounds__(64 * kReduceWaves) void k_reduce_score(const float4* __restrict__ partials,
                                                                     const int32_t* __restrict__ rows,
                                                                     const int32_t* __restrict__ n_ptr, int nvt,
                                                                     ScoreArgs a, TieArgs ta,
                                                                     const uint16_t* __restrict__ hidden,
                                                                     const uint16_t* __restrict__ xrows, int d) {
  __shared__ int ly[64];
  __shared__ float lc[64], lh[64];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int p = blockIdx.x;
  // The count, the row and the partials are loaded together: workgroup p <
  // max_masked reads inside the rows and partials buffers (sized for
  // max_masked positions) whatever the count, and a workgroup beyond the
  // count drops what it read.
  const int n = *n_ptr;
  {
    const int pos = rows[p];
    const int b = pos / a.L, i = pos - b * a.L;
    for (int l = wid; l < a.K; l += kReduceWaves) {
      const float4* src = partials + ((long long)p * a.K + l) * nvt;
      float4 keep[8];
      Soft s = wave_merge_row(src, nvt, lane, keep);
      if (ta.w_u && p < n) {   // rows past the count are not valid (and never read)
        const uint16_t* x = xrows ? xrows + ((long long)p * a.K + l) * d
                                  : hidden + (((long long)l * a.B + b) * a.L + i) * (long long)d;
        s.idx = resolve_tie(s, keep, src, nvt, ta, x, lane);
      }
      if (lane == 0) state_stats(s, ly[l], lc[l], lh[l]);
    }
    if (p >= n) return;
    __syncthreads();
    if (wid == 0) {
      const int my_y = lane < a.K ? ly[lane] : -1;
      const float my_c = lane < a.K ? lc[lane] : 0.f;
      const float my_h = lane < a.K ? lh[lane] : 0.f;
      const int yK = ly[a.K - 1];
      const float cK = lc[a.K - 1];
      const float hK = lh[a.K - 1];
      // Eq. 2: agreement suffix ending at the final layer
      const unsigned long long dis = __ballot(lane < a.K && my_y != yK);
      const int last_dis = dis ? 63 - __clzll(dis) : -1;
      const int k_i = a.K - 1 - last_dis;
      // Eq. 3: inside the suffix the final token is each layer's argmax, so
      // its probability there is that layer's top probability
      float pk = (lane >= a.K - k_i && lane < a.K) ? my_c : -INFINITY;
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) pk = fmaxf(pk, __shfl_xor(pk, m));
      const float r_i = pk - cK;
      const float s_i = stability_score(k_i, r_i, a.k_max, a.w);
      const unsigned fl = route_flags(cK, s_i, a.theta_h, a.theta_c, a.theta_s);
      const long long o = (long long)b * a.L + i;
      if (lane == 0) {
        a.token[o] = yK;
        a.entropy[o] = hK;
        a.confidence[o] = cK;
        a.persistence[o] = k_i;
        a.drop[o] = r_i;
        a.stability[o] = s_i;
        a.flags[o] = (uint8_t)fl;
      }
      if (a.layer_argmax && lane < a.K) {
        const long long ol = ((long long)lane * a.B + b) * a.L + i;
        a.layer_argmax[ol] = my_y;
        a.layer_conf[ol] = my_c;
        a.layer_entropy[ol] = my_h;
      }
    }
  }
}

// End of an iteration (Section 3.2): committed positions take their token in
// the canvas and leave the mask. With `progress`, one workgroup does the
// whole canvas and records the masked positions left: progress[0] counts the
// calls, progress[1 + t] holds call t's remainder (while t < progress_len),
// and `step` (optional) receives the call index at each committed position.
// Without it the canvas is covered grid-stride.
constexpr int kApplyThreads = 1024;
__global__ __launch_bounds__(kApplyThreads) void k_apply_commit(long long BL, uint8_t* __restrict__ mask,
                                                                int32_t* __restrict__ canvas,
                                                                const uint8_t* __restrict__ commit,
                                                                const int32_t* __restrict__ token,
                                                                int32_t* __restrict__ progress, int progress_len,
                                                                int32_t* __restrict__ step) {
  __shared__ int wsum[kApplyThreads / 64];
  const int t = progress ? progress[0] : 0;
  int left = 0;
  for (long long o = blockIdx.x * (long long)blockDim.x + threadIdx.x; o < BL; o += (long long)gridDim.x * blockDim.x) {
    if (mask[o] != 0) {
      if (commit[o] != 0) {
        canvas[o] = token[o];
        mask[o] = 0;
        if (step) step[o] = t;
      } else {
        ++left;
      }
    }
  }
  if (!progress) return;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) left += __shfl_xor(left, m);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = left;
  __syncthreads();   // also orders every thread's read of progress[0] before its update
  if (threadIdx.x == 0) {
    int tot = 0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) tot += wsum[w];
    if (t < progress_len) progress[1 + t] = tot;
    progress[0] = t + 1;
  }
}

ScoreArgs score_args(const Launch& a) {
  ScoreArgs s;
  s.K = a.K;
  s.B = a.B;
  s.L = a.L;
  s.theta_h = a.theta_h;
  s.theta_c = a.theta_c;
  s.theta_s = a.theta_s;
  s.w = a.w;
  s.k_max = a.k_max;
  s.token = a.token;
  s.entropy = a.entropy;
  s.confidence = a.confidence;
  s.persistence = a.persistence;
  s.drop = a.drop;
  s.stability = a.stability;
  s.flags = a.flags;
  s.layer_argmax = a.layer_argmax;
  s.layer_conf = a.layer_conf;
  s.layer_entropy = a.layer_entropy;
  return s;
}

CommitArgs commit_args(const Launch& a) {
  CommitArgs c;
  c.B = a.B;
  c.L = a.L;
  c.beta = a.beta;
  c.window = a.window;
  c.block = a.block;
  c.commit = a.commit;
  c.token = a.token;
  c.entropy = a.entropy;
  c.confidence = a.confidence;
  c.persistence = a.persistence;
  c.drop = a.drop;
  c.stability = a.stability;
  c.flags = a.flags;
  c.upstream_entropy = a.upstream_entropy;
  c.n_commit = a.n_commit;
  return c;
}

}  // namespace

hipError_t launch_compact(const Launch& a, bool lazy_list, hipStream_t s) {
  FirstPassList fp{};
  if (lazy_list)
    fp = FirstPassList{a.lazy.act, a.lazy.rowoff, a.lazy.m, a.lazy.tier, (long long)(a.K - 1) * a.B * a.L, a.d,
                       kStreamMaxRows, kBigTileRowsMid};
  hipLaunchKernelGGL(k_compact, dim3(1), dim3(1024), 0, s, a.mask, a.B * a.L, a.max_masked, a.rows, a.n_masked,
                     a.dev_status, a.user_status, fp);
  return hipGetLastError();
}

hipError_t launch_reduce_score(const Launch& a, hipStream_t s) {
  if (a.max_masked <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_reduce_score, dim3(a.max_masked), dim3(64 * kReduceWaves), 0, s, a.partials, a.rows,
                     a.n_masked, a.plan.nvt, score_args(a), tie_args(a, a.plan), static_cast<const uint16_t*>(a.hidden),
                     static_cast<const uint16_t*>(a.xrows), a.d);
  return hipGetLastError();
}

int commit_threads(int L) {
  const int t = ((L + 63) / 64) * 64;
  return t < kCommitThreads ? t : kCommitThreads;
}

hipError_t launch_commit(const Launch& a, hipStream_t s) {
  hipLaunchKernelGGL(k_commit, dim3(a.B), dim3(commit_threads(a.L)), 0, s, a.mask, commit_args(a));
  return hipGetLastError();
}

hipError_t launch_apply_commit(long long BL, uint8_t* mask, int32_t* canvas, const uint8_t* commit,
                               const int32_t* token, int32_t* progress, int progress_len, int32_t* step,
                               hipStream_t s) {
  const unsigned grid = progress ? 1u : (unsigned)std::min<long long>((BL + kApplyThreads - 1) / kApplyThreads, 1024);
  hipLaunchKernelGGL(k_apply_commit, dim3(grid), dim3(kApplyThreads), 0, s, BL, mask, canvas, commit, token, progress,
                     progress_len, step);
  return hipGetLastError();
}

hipError_t launch_gate_commit(const Launch& a, const int32_t* l_y, const float* l_c, const float* l_h,
                              hipStream_t s) {
  const long long BL = (long long)a.B * a.L;
  hipLaunchKernelGGL(k_gate_score, dim3((unsigned)((BL + 255) / 256)), dim3(256), 0, s, a.mask, l_y, l_c, l_h,
                     score_args(a));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_commit, dim3(a.B), dim3(commit_threads(a.L)), 0, s, a.mask, commit_args(a));
  return hipGetLastError();
}

}  // namespace rpd
