// C ABI of the RPD commit step: argument validation, workspace layout,
// launch planning and error reporting. Kernels live in proj_*.hip and
// score_commit.hip; the projection plan in proj_plan.cpp.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "rpd.h"
#include "rpd_launch.h"

namespace {

thread_local char g_err[512] = "";

rpd_status fail(rpd_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return s;
}

constexpr size_t kHeaderBytes = 256;   // n_masked (0), device status (4), lazy pass rows (12), by size class (16)
constexpr long long kMaxBL = 1LL << 24;
constexpr int kMaxK = 64;
// hidden sizes up to 2^20: the MFMA tile's 32-bit byte offsets within its
// 256 W_U rows (256 * d * 2) stay below 2^31
constexpr int kMaxD = 1 << 20;

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

bool shape_ok(const rpd_problem* p) {
  return p->K >= 1 && p->K <= kMaxK && p->B >= 1 && p->L >= 1 && (long long)p->B * p->L <= kMaxBL && p->d >= 1 &&
         p->d <= kMaxD && p->V >= 1 && p->V < 0x7fffffff;
}

long long masked_cap(const rpd_problem* p) {
  const long long BL = (long long)p->B * p->L;
  return (p->max_masked < 0 || p->max_masked > BL) ? BL : p->max_masked;
}

size_t partial_bytes(const rpd::ProjPlan& pl, long long rows) { return (size_t)rows * pl.nvt * 16; }

size_t elem_bytes(const rpd_problem* p) { return p->dtype == RPD_DTYPE_BF16 ? 2 : 4; }

// per-position state of the lazy projection: act (4 B), rowoff (8 B) and
// seven 4-byte arrays per position
size_t lazy_bytes(long long cap) { return align256((size_t)cap * 8) + 8 * align256((size_t)cap * 4); }

// the normalized, compacted rows [K * cap][d] (only with a normalization)
size_t norm_bytes(const rpd_problem* p, long long cap) {
  return p->norm_weight ? align256((size_t)((long long)p->K * cap) * (size_t)p->d * elem_bytes(p)) : 0;
}

// Bytes for the plan chosen at `cap` masked positions. Any smaller row count
// may be planned as well (the exact count read back when max_masked < 0, or
// a lazy pass over fewer rows), so every variant boundary below it is
// covered too.
size_t workspace_bytes_for(const rpd_problem* p, long long cap) {
  const long long rows = (long long)p->K * cap;
  size_t part = partial_bytes(rpd::plan_projection(p->dtype, rows, p->V), rows);
  for (long long r : {32LL, 33LL, 64LL, 65LL, 128LL, 129LL, 192LL, 193LL, 256LL, 257LL}) {
    const long long rr = r < rows ? r : rows;
    const size_t b = partial_bytes(rpd::plan_projection(p->dtype, rr, p->V), rr);
    if (b > part) part = b;
  }
  return kHeaderBytes + align256((size_t)((long long)p->B * p->L) * 4) + align256(part) + lazy_bytes(cap) +
         norm_bytes(p, cap);
}

rpd_status check_params(const rpd_params* q) {
  if (!q) return fail(RPD_ERR_NULL_POINTER, "params is NULL");
  const float f[] = {q->theta_h, q->theta_c, q->theta_s, q->w};
  for (float v : f)
    if (!std::isfinite(v)) return fail(RPD_ERR_BAD_PARAM, "theta_h, theta_c, theta_s and w must be finite");
  if (!(q->theta_c >= 0.f && q->theta_c <= q->theta_h))
    return fail(RPD_ERR_BAD_PARAM, "need 0 <= theta_c <= theta_h (got %g, %g)", q->theta_c, q->theta_h);
  if (q->w < 0.f) return fail(RPD_ERR_BAD_PARAM, "w must be >= 0 (got %g)", q->w);
  if (q->k_max < 1) return fail(RPD_ERR_BAD_PARAM, "k_max must be >= 1 (got %d)", q->k_max);
  if (std::isnan(q->beta) || q->beta < 0.f) return fail(RPD_ERR_BAD_PARAM, "beta must be >= 0 (got %g)", q->beta);
  if (q->window < 1) return fail(RPD_ERR_BAD_PARAM, "window must be >= 1 (got %d)", q->window);
  if (q->flags & ~(uint32_t)(RPD_PARAM_LAZY | RPD_PARAM_LAZY_ALL))
    return fail(RPD_ERR_BAD_PARAM, "flags holds unknown bits (0x%x); RPD_PARAM_LAZY and RPD_PARAM_LAZY_ALL are defined",
                q->flags);
  if ((q->flags & RPD_PARAM_LAZY_ALL) && !(q->flags & RPD_PARAM_LAZY))
    return fail(RPD_ERR_BAD_PARAM, "RPD_PARAM_LAZY_ALL needs RPD_PARAM_LAZY");
  if (q->block < 0) return fail(RPD_ERR_BAD_PARAM, "block must be >= 0 (got %d)", q->block);
  if (!std::isfinite(q->logit_scale) || q->logit_scale < 0.f)
    return fail(RPD_ERR_BAD_PARAM, "logit_scale must be finite and > 0, or 0 for 1 (got %g)", q->logit_scale);
  return RPD_OK;
}

rpd_status check_outputs(const rpd_outputs* o) {
  if (!o) return fail(RPD_ERR_NULL_POINTER, "outputs is NULL");
  if (!o->commit || !o->token || !o->entropy || !o->confidence || !o->persistence || !o->drop || !o->stability ||
      !o->flags || !o->upstream_entropy || !o->n_commit)
    return fail(RPD_ERR_NULL_POINTER, "a required output pointer is NULL");
  const int nl = (o->layer_argmax != nullptr) + (o->layer_conf != nullptr) + (o->layer_entropy != nullptr);
  if (nl != 0 && nl != 3)
    return fail(RPD_ERR_NULL_POINTER, "layer_argmax, layer_conf and layer_entropy must be all set or all NULL");
  return RPD_OK;
}

void fill_common(rpd::Launch& a, const rpd_params* q, const rpd_outputs* o) {
  a.theta_h = q->theta_h;
  a.theta_c = q->theta_c;
  a.theta_s = q->theta_s;
  a.w = q->w;
  a.beta = q->beta;
  a.k_max = q->k_max;
  a.window = q->window;
  a.block = q->block;
  a.logit_scale = q->logit_scale == 0.f ? 1.f : q->logit_scale;
  a.lazy_all = (q->flags & RPD_PARAM_LAZY_ALL) != 0;
  a.commit = o->commit;
  a.token = o->token;
  a.entropy = o->entropy;
  a.confidence = o->confidence;
  a.persistence = o->persistence;
  a.drop = o->drop;
  a.stability = o->stability;
  a.flags = o->flags;
  a.upstream_entropy = o->upstream_entropy;
  a.n_commit = o->n_commit;
  a.layer_argmax = o->layer_argmax;
  a.layer_conf = o->layer_conf;
  a.layer_entropy = o->layer_entropy;
  a.user_status = o->status;
}

// Lazy layerwise projection: one projection pass per layer from the final
// one down over the positions still walking their agreement suffix (rows
// listed by k_lazy_next); how a pass is planned for a count that only the
// device knows is described in the loop.
template <class Mark>
hipError_t run_lazy(rpd::Launch& a, int dtype, hipStream_t s, Mark& mark) {
  hipError_t e = mark(1);
  if (e != hipSuccess) return e;
  if (a.max_masked > 0) {
    int m_host = a.max_masked;   // pass 0, listed by the compaction: every masked position (<= max_masked)
    // A pass runs the plan for its row count, which only the device knows.
    // While the bound on it is at most kLazyGateRows the host reads nothing
    // back: the pass is launched once per size class the count may fall in
    // (<= 64 rows: streaming; <= 128; up to the bound), each taking its
    // count from the device as that class's count, 0 unless it is the
    // class, so all but one exit at once. Above the bound the count is read
    // back (one stream synchronisation) and the pass planned for it. A
    // single pass planned for the bound would run an MFMA tile whatever the
    // count (lazy call at 256 positions: 838 -> 1010 us), and above 256 rows
    // its few row tiles would land on a few XCDs.
    // a pass over `cap` rows whose count is at `count`
    auto pass_launch = [&](int l, int32_t* count, int cap) {
      rpd::Launch ap = a;
      ap.n_masked = count;
      ap.max_masked = cap;
      ap.rowoff = a.lazy.rowoff;
      ap.pass_layer = l;
      ap.fused_compact = false;
      ap.plan = rpd::plan_projection(dtype, cap, a.V);
      return ap;
    };
    for (int t = 0; t < a.K; ++t) {
      const int l = a.K - 1 - t;
      bool known = t == 0;
      if (t > 0 && m_host > rpd::kLazyGateRows) {
        int32_t m = 0;
        if ((e = hipMemcpyAsync(&m, a.lazy.m, sizeof m, hipMemcpyDeviceToHost, s)) != hipSuccess) return e;
        if ((e = hipStreamSynchronize(s)) != hipSuccess) return e;
        if (m <= 0) break;
        m_host = m;
        known = true;
      }
      // the pass's rows are normalized once and reduced once; in between one
      // projection, or one per size class, of which only the count's class
      // writes the partials (the reduction takes that class's layout)
      const rpd::Launch whole = pass_launch(l, a.lazy.m, m_host);
      if (whole.xrows && (e = rpd::launch_norm_rows(whole, s)) != hipSuccess) return e;
      if (known || m_host <= rpd::kStreamMaxRows) {
        if ((e = rpd::launch_projection(whole, s)) != hipSuccess) return e;
        if ((e = rpd::launch_lazy_reduce(whole, l, m_host, nullptr, s)) != hipSuccess) return e;
      } else {
        const int caps[3] = {rpd::kStreamMaxRows, std::min(m_host, rpd::kBigTileRowsMid), m_host};
        const int ncls = m_host > rpd::kBigTileRowsMid ? 3 : 2;
        rpd::ProjPlan plans[3];
        for (int c = 0; c < 3; ++c) {
          const rpd::Launch ap = pass_launch(l, a.lazy.tier + c, caps[c]);
          plans[c] = ap.plan;
          if (c < ncls && (e = rpd::launch_projection(ap, s)) != hipSuccess) return e;
        }
        if ((e = rpd::launch_lazy_reduce(whole, l, m_host, plans, s)) != hipSuccess) return e;
      }
      if (l > 0 && (e = rpd::launch_lazy_next(a, l - 1, s)) != hipSuccess) return e;
    }
  }
  if ((e = mark(2)) != hipSuccess) return e;
  if ((e = rpd::launch_lazy_score(a, s)) != hipSuccess) return e;
  if ((e = mark(3)) != hipSuccess) return e;
  if ((e = rpd::launch_commit(a, s)) != hipSuccess) return e;
  return mark(4);
}

}  // namespace

// The workspace of rpd_score_commit_noalloc: one static device array per
// GPU, for callers that cannot allocate. In host code `scratch` names a
// host-side stand-in, not device memory: only the address that
// hipGetSymbolAddress returns for the current device is ever used.
static __device__ __align__(256) unsigned char scratch[RPD_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};   // device address of `scratch` per device (looked up once)

// the current device's address of `scratch`, looked up on its first use with that device current
hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!ptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" {

size_t rpd_workspace_size(const rpd_problem* p) {
  if (!p || !shape_ok(p) || (p->dtype != RPD_DTYPE_BF16 && p->dtype != RPD_DTYPE_F32)) return 0;
  return workspace_bytes_for(p, masked_cap(p));
}

int32_t rpd_projection_variant(const rpd_problem* p) {
  if (!p || !shape_ok(p) || (p->dtype != RPD_DTYPE_BF16 && p->dtype != RPD_DTYPE_F32)) return -1;
  return (int32_t)rpd::plan_projection(p->dtype, (long long)p->K * masked_cap(p), p->V).variant;
}

static rpd_status score_commit_impl(const rpd_problem* p, const rpd_params* q, const rpd_outputs* o,
                                    void* workspace, size_t workspace_bytes, void* stream, void* const* events,
                                    int32_t n_events) {
  g_err[0] = '\0';
  if (!p) return fail(RPD_ERR_NULL_POINTER, "problem is NULL");
  if (!p->hidden || !p->w_u || !p->mask) return fail(RPD_ERR_NULL_POINTER, "hidden, w_u and mask are required");
  if (!shape_ok(p))
    return fail(RPD_ERR_BAD_SHAPE, "need 1<=K<=%d, B,L>=1, B*L<=2^24, 1<=d<=2^20, 1<=V<2^31-1 (got K=%d B=%d L=%d d=%d V=%d)",
                kMaxK, p->K, p->B, p->L, p->d, p->V);
  if (p->dtype != RPD_DTYPE_BF16 && p->dtype != RPD_DTYPE_F32)
    return fail(RPD_ERR_UNSUPPORTED, "dtype %d is not supported", p->dtype);
  if (p->dtype == RPD_DTYPE_BF16) {
    if (p->d % 8 != 0) return fail(RPD_ERR_UNSUPPORTED, "bf16 needs d %% 8 == 0 (got d=%d)", p->d);
    if (((uintptr_t)p->hidden | (uintptr_t)p->w_u) & 15)
      return fail(RPD_ERR_UNSUPPORTED, "bf16 hidden and w_u must be 16-byte aligned");
  } else if (((uintptr_t)p->hidden | (uintptr_t)p->w_u) & 3) {
    return fail(RPD_ERR_UNSUPPORTED, "fp32 hidden and w_u must be 4-byte aligned");
  }
  if (p->norm_weight) {
    if (((uintptr_t)p->norm_weight) & (p->dtype == RPD_DTYPE_BF16 ? 15 : 3))
      return fail(RPD_ERR_UNSUPPORTED, "norm_weight must be aligned like hidden");
    if (!std::isfinite(p->norm_eps) || p->norm_eps < 0.f)
      return fail(RPD_ERR_BAD_PARAM, "norm_eps must be finite and >= 0 (got %g)", p->norm_eps);
    if (p->norm_final != 0 && p->norm_final != 1)
      return fail(RPD_ERR_BAD_PARAM, "norm_final must be 0 or 1 (got %d)", p->norm_final);
  }
  rpd_status st = check_params(q);
  if (st != RPD_OK) return st;
  st = check_outputs(o);
  if (st != RPD_OK) return st;
  if (n_events < 0 || n_events > 5 || (n_events > 0 && !events))
    return fail(RPD_ERR_BAD_PARAM, "need 0 <= n_events <= 5 and a non-NULL events array");

  const long long cap = masked_cap(p);
  const size_t need = workspace_bytes_for(p, cap);
  if (!workspace) return fail(RPD_ERR_NULL_POINTER, "workspace is NULL (%zu bytes needed)", need);
  if ((uintptr_t)workspace & 255) return fail(RPD_ERR_UNSUPPORTED, "workspace must be 256-byte aligned");
  if (workspace_bytes < need)
    return fail(RPD_ERR_WORKSPACE_TOO_SMALL, "workspace has %zu bytes, %zu needed", workspace_bytes, need);

  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  rpd::Launch a{};
  a.K = p->K;
  a.B = p->B;
  a.L = p->L;
  a.d = p->d;
  a.V = p->V;
  a.hidden = p->hidden;
  a.w_u = p->w_u;
  a.mask = p->mask;
  a.max_masked = (int)cap;
  a.n_masked = reinterpret_cast<int32_t*>(ws);
  a.dev_status = reinterpret_cast<int32_t*>(ws + 4);
  a.rows = reinterpret_cast<int32_t*>(ws + kHeaderBytes);
  a.partials = reinterpret_cast<float4*>(ws + kHeaderBytes + align256((size_t)((long long)p->B * p->L) * 4));
  a.norm_weight = p->norm_weight;
  a.norm_eps = p->norm_eps;
  a.norm_final = p->norm_final;
  // the normalized rows sit at the end, the lazy state before them (the
  // partials are sized for the largest plan)
  a.xrows = p->norm_weight ? ws + (need - norm_bytes(p, cap)) : nullptr;
  {
    char* lz = ws + (need - norm_bytes(p, cap) - lazy_bytes(cap));
    const size_t a4 = align256((size_t)cap * 4);
    a.lazy.rowoff = reinterpret_cast<long long*>(lz);
    lz += align256((size_t)cap * 8);
    int32_t** ints[] = {&a.lazy.act, &a.lazy.y, &a.lazy.k, &a.lazy.alive, &a.lazy.depth};
    for (int32_t** q4 : ints) {
      *q4 = reinterpret_cast<int32_t*>(lz);
      lz += a4;
    }
    float** floats[] = {&a.lazy.c, &a.lazy.h, &a.lazy.pmax};
    for (float** q4 : floats) {
      *q4 = reinterpret_cast<float*>(lz);
      lz += a4;
    }
    a.lazy.m = reinterpret_cast<int32_t*>(ws + 12);
    a.lazy.tier = reinterpret_cast<int32_t*>(ws + 16);
  }
  a.rowoff = nullptr;
  const bool lazy = (q->flags & RPD_PARAM_LAZY) != 0;
  fill_common(a, q, o);

  auto mark = [&](int k) -> hipError_t {
    if (k < n_events && events[k]) return hipEventRecord(static_cast<hipEvent_t>(events[k]), s);
    return hipSuccess;
  };
  // with a known bound the plan comes first, and small canvases are
  // compacted inside the projection kernel
  a.fused_compact = false;
  if (p->max_masked >= 0) {
    a.plan = rpd::plan_projection(p->dtype, (long long)p->K * a.max_masked, p->V);
    a.fused_compact = !lazy && rpd::compact_fused(a);
  }
  hipError_t e = mark(0);
  if (e == hipSuccess && !a.fused_compact) e = rpd::launch_compact(a, lazy, s);
  if (e != hipSuccess) return fail(RPD_ERR_HIP, "compaction: %s", hipGetErrorString(e));
  if (p->max_masked < 0) {
    int32_t n = 0;
    e = hipMemcpyAsync(&n, a.n_masked, sizeof n, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail(RPD_ERR_HIP, "reading the masked count: %s", hipGetErrorString(e));
    a.max_masked = n;
    a.plan = rpd::plan_projection(p->dtype, (long long)p->K * a.max_masked, p->V);
  }
  if (lazy) {
    e = run_lazy(a, p->dtype, s, mark);
  } else if ((e = mark(1)) == hipSuccess && (!a.xrows || (e = rpd::launch_norm_rows(a, s)) == hipSuccess) &&
             (e = rpd::launch_projection(a, s)) == hipSuccess && (e = mark(2)) == hipSuccess &&
             (e = rpd::launch_reduce_score(a, s)) == hipSuccess && (e = mark(3)) == hipSuccess &&
             (e = rpd::launch_commit(a, s)) == hipSuccess) {
    e = mark(4);
  }
  if (e != hipSuccess) return fail(RPD_ERR_HIP, "launch: %s", hipGetErrorString(e));
  return RPD_OK;
}

rpd_status rpd_score_commit(const rpd_problem* p, const rpd_params* q, const rpd_outputs* o, void* workspace,
                            size_t workspace_bytes, void* stream) {
  return score_commit_impl(p, q, o, workspace, workspace_bytes, stream, nullptr, 0);
}

rpd_status rpd_score_commit_timed(const rpd_problem* p, const rpd_params* q, const rpd_outputs* o,
                                  void* workspace, size_t workspace_bytes, void* stream, void* const* events,
                                  int32_t n_events) {
  return score_commit_impl(p, q, o, workspace, workspace_bytes, stream, events, n_events);
}

rpd_status rpd_score_commit_noalloc(const rpd_problem* p, const rpd_params* q, const rpd_outputs* o,
                                    void* stream) {
  g_err[0] = '\0';
  if (!p) return fail(RPD_ERR_NULL_POINTER, "problem is NULL");
  // the size first: a problem beyond the array is refused before any HIP call
  const size_t need = rpd_workspace_size(p);
  if (need > RPD_NOALLOC_SCRATCH_BYTES)
    return fail(RPD_ERR_WORKSPACE_TOO_SMALL,
                "the problem needs %zu workspace bytes; rpd_score_commit_noalloc has %zu (use rpd_score_commit with a "
                "workspace of that size)", need, (size_t)RPD_NOALLOC_SCRATCH_BYTES);
  // an invalid shape or dtype (need 0) is reported by the validation in score_commit_impl, which checks
  // them before the workspace
  void* ws = nullptr;
  if (need > 0) {
    const hipError_t e = scratch_address(&ws);
    if (e != hipSuccess) return fail(RPD_ERR_HIP, "looking up the scratch array: %s", hipGetErrorString(e));
  }
  return score_commit_impl(p, q, o, ws, RPD_NOALLOC_SCRATCH_BYTES, stream, nullptr, 0);
}

rpd_status rpd_apply_commit(int32_t B, int32_t L, uint8_t* mask, int32_t* canvas, const uint8_t* commit,
                            const int32_t* token, int32_t* progress, int32_t progress_len, int32_t* step,
                            void* stream) {
  g_err[0] = '\0';
  if (!mask || !canvas || !commit || !token) return fail(RPD_ERR_NULL_POINTER, "mask, canvas, commit and token are required");
  if (step && !progress) return fail(RPD_ERR_NULL_POINTER, "step needs progress (the call counter)");
  if (B < 1 || L < 1 || (long long)B * L > kMaxBL)
    return fail(RPD_ERR_BAD_SHAPE, "need B,L>=1, B*L<=2^24 (got B=%d L=%d)", B, L);
  if (progress && progress_len < 0) return fail(RPD_ERR_BAD_PARAM, "progress_len must be >= 0");
  const hipError_t e = rpd::launch_apply_commit((long long)B * L, mask, canvas, commit, token, progress,
                                                progress ? progress_len : 0, step, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(RPD_ERR_HIP, "launch: %s", hipGetErrorString(e));
  return RPD_OK;
}

rpd_status rpd_gate_commit(int32_t K, int32_t B, int32_t L, const uint8_t* mask, const int32_t* layer_argmax,
                           const float* layer_conf, const float* layer_entropy, const rpd_params* q,
                           const rpd_outputs* o, void* stream) {
  g_err[0] = '\0';
  if (!mask || !layer_argmax || !layer_conf || !layer_entropy)
    return fail(RPD_ERR_NULL_POINTER, "mask and the three per-layer inputs are required");
  if (K < 1 || K > kMaxK || B < 1 || L < 1 || (long long)B * L > kMaxBL)
    return fail(RPD_ERR_BAD_SHAPE, "need 1<=K<=%d, B,L>=1, B*L<=2^24 (got K=%d B=%d L=%d)", kMaxK, K, B, L);
  rpd_status st = check_params(q);
  if (st != RPD_OK) return st;
  st = check_outputs(o);
  if (st != RPD_OK) return st;
  rpd::Launch a{};
  a.K = K;
  a.B = B;
  a.L = L;
  a.mask = mask;
  fill_common(a, q, o);
  a.layer_argmax = nullptr;
  a.layer_conf = nullptr;
  a.layer_entropy = nullptr;
  a.user_status = nullptr;
  hipError_t e =
      rpd::launch_gate_commit(a, layer_argmax, layer_conf, layer_entropy, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(RPD_ERR_HIP, "launch: %s", hipGetErrorString(e));
  return RPD_OK;
}

const char* rpd_status_string(rpd_status s) {
  switch (s) {
    case RPD_OK: return "ok";
    case RPD_ERR_NULL_POINTER: return "null pointer";
    case RPD_ERR_BAD_SHAPE: return "bad shape";
    case RPD_ERR_BAD_PARAM: return "bad parameter";
    case RPD_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case RPD_ERR_UNSUPPORTED: return "unsupported";
    case RPD_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

const char* rpd_last_error(void) { return g_err; }

int32_t rpd_abi_version(void) { return RPD_ABI_VERSION; }

}  // extern "C"
