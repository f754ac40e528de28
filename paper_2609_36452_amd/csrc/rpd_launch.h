// Internal interface between the C ABI (rpd_api.cpp), the projection plan
// (proj_plan.cpp) and the gfx950 kernels (proj_*.hip, score_commit.hip).
// Not installed; no torch or HIP types beyond hipStream_t.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rpd {

// Projection kernel shapes. A "row" is one (masked position, layer) pair:
// row r = p*K + l for compacted masked position p. A "vocab tile" is a
// contiguous range of W_U rows; tile t covers [t*V/NVT, (t+1)*V/NVT).
enum ProjVariant {
  PROJ_BF16_S32 = 0,    // <= 32 rows: W_U streamed through wave-private LDS, hidden rows shared
  PROJ_BF16_S64 = 1,    // <= 64 rows, same kernel family
  PROJ_F32 = 3,         // fp32 inputs: vector ALU, 16 rows x 64 vocab
  PROJ_BF16_BIG = 4,    // MFMA-bound: 256 x 256 tiles, both operands staged through LDS
  PROJ_BF16_BIG192 = 6, // the same kernel with 256 x 192 tiles (where they pad the rows less)
  PROJ_BF16_BIG128 = 7, // the same kernel with 256 x 128 tiles, for 65..128 rows
};

// tile of the large-row variant: vocabulary rows x projected rows
constexpr int kBigTileVocab = 256, kBigTileRows = 256;
// vocabulary rows of one workgroup of the streaming variants (all of them)
constexpr int kStreamTileVocab = 256;
// most projected rows a streaming variant takes; above, the MFMA tiles are
// faster (256 x 128 measured 7-12% faster than 128-row streaming at 68-128
// rows, 256 x 192 3-8% faster than 192-row streaming at 132-192 rows,
// 256 x 256 7-9% faster than 256-row streaming at 224 and 256; at 48 and 64
// rows the 64-row streaming form is 11% faster than 256 x 128)
constexpr int kStreamMaxRows = 64;
// rows of the smaller MFMA tiles
constexpr int kBigTileRowsSmall = 192, kBigTileRowsMid = 128;
// largest bound on a lazy pass's rows below which the host reads no count back
constexpr int kLazyGateRows = 256;
// largest canvas (B * L) whose compaction the streaming projection does itself
constexpr int kFusedCompactMax = 2048;

struct ProjPlan {
  ProjVariant variant;
  int rows_per_tile;   // TR
  int vocab_cap;       // max vocab rows one tile can hold
  int nvt;             // number of vocab tiles
  int nrt;             // number of row tiles (for the row bound)
  int per_xcd;         // workgroups per XCD slot in the launch
  int split_rows;      // 1: XCDs own row tiles; 0: XCDs own vocab tiles
  int grid;            // workgroups launched
};

// the shape plan for `rows_cap` rows (K * max masked positions)
ProjPlan plan_projection(int dtype, long long rows_cap, int V);

// per-position state of the lazy layerwise projection (lazy.hip)
struct LazyState {
  int32_t* act;        // [cap] compacted positions listed for the current pass
  long long* rowoff;   // [cap] element offsets into hidden of their rows
  int32_t* y;          // [cap] final-layer token
  float* c;            // [cap] final-layer top probability
  float* h;            // [cap] final-layer entropy
  int32_t* k;          // [cap] agreement suffix length so far
  float* pmax;         // [cap] peak top probability over the suffix
  int32_t* alive;      // [cap] 1 while the walk continues
  int32_t* depth;      // [cap] layers projected
  int32_t* m;          // [1] rows in the current pass
  int32_t* tier;       // [3] the same count in its size class (<= 64, <= 128, above), 0 in the others
};

struct LazyScoreArgs {
  int K, B, L;
  float theta_h, theta_c, theta_s, w;
  int k_max;
  int walk_all;        // every position with a finite confidence walked (else only the band)
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

struct Launch {
  int K, B, L, d, V;
  const void* hidden;
  const void* w_u;
  const uint8_t* mask;
  int max_masked;        // bound used for the launches (>= 0)
  // workspace pieces
  int32_t* n_masked;     // [1] device count (clamped to max_masked)
  int32_t* dev_status;   // [1] internal status word
  bool fused_compact;    // the projection kernel does the compaction (no launch_compact)
  int32_t* rows;         // [max_masked] compacted b*L+i
  float4* partials;      // [K*max_masked][nvt]
  // final normalization (norm_weight NULL: none): the projection then reads
  // projected row r at xrows + r * d (normalized, compacted) instead of
  // gathering it from hidden
  const void* norm_weight;
  float norm_eps;
  int norm_final;
  void* xrows;
  // explicit row list (lazy passes): projected row r is hidden + rowoff[r]
  // (with K == 1 and n_masked pointing at the row count); NULL: gathered
  const long long* rowoff;
  int pass_layer;        // the layer of an explicit row list (normalization)
  LazyState lazy;
  ProjPlan plan;
  // params
  float theta_h, theta_c, theta_s, w, beta;
  int k_max, window;
  int block;             // 0: full RPD; > 0: RPD-block
  float logit_scale;     // multiplies every logit before the softmax statistics
  bool lazy_all;         // lazy projection: every masked position walks its layers (RPD_PARAM_LAZY_ALL)
  // outputs
  uint8_t* commit; int32_t* token; float* entropy; float* confidence;
  int32_t* persistence; float* drop; float* stability; uint8_t* flags;
  float* upstream_entropy; int32_t* n_commit;
  int32_t* layer_argmax; float* layer_conf; float* layer_entropy;
  int32_t* user_status;
};

// enqueue, in this order: compaction, projection, reduction + scoring,
// commitment (the last three use a.plan and a.max_masked)
// lazy_list: also list the first lazy pass (a.lazy: act, rowoff, m, tier)
hipError_t launch_compact(const Launch& a, bool lazy_list, hipStream_t s);
hipError_t launch_projection(const Launch& a, hipStream_t s);
hipError_t launch_reduce_score(const Launch& a, hipStream_t s);
hipError_t launch_commit(const Launch& a, hipStream_t s);

// lazy layerwise projection: list the rows of layer l still walking,
// reduce a pass over layer l, score from the per-position state
hipError_t launch_lazy_next(const Launch& a, int l, hipStream_t s);
// class_plans: the plans for rows <= 64, <= 128 and above, when the pass
// ran once per size class (NULL: a.plan)
hipError_t launch_lazy_reduce(const Launch& a, int l, int m_cap, const ProjPlan* class_plans, hipStream_t s);
hipError_t launch_lazy_score(const Launch& a, hipStream_t s);
// the projection does the compaction itself (needs a.plan and a.max_masked
// >= 0): the call then launches no compaction kernel
bool compact_fused(const Launch& a);

// the projection variants, dispatched by launch_projection on a.plan.variant
// the final normalization of the compacted rows into a.xrows (before the projection)
hipError_t launch_norm_rows(const Launch& a, hipStream_t s);
hipError_t launch_proj_stream(const Launch& a, hipStream_t s);  // PROJ_BF16_S32, PROJ_BF16_S64
hipError_t launch_proj_big(const Launch& a, hipStream_t s);     // PROJ_BF16_BIG
hipError_t launch_proj_f32(const Launch& a, hipStream_t s);     // PROJ_F32

// end of an iteration: fill the canvas with the committed tokens, unmask them
hipError_t launch_apply_commit(long long BL, uint8_t* mask, int32_t* canvas, const uint8_t* commit,
                               const int32_t* token, int32_t* progress, int progress_len, int32_t* step,
                               hipStream_t s);

// scoring + commitment from caller-supplied per-layer statistics
hipError_t launch_gate_commit(const Launch& a, const int32_t* layer_argmax, const float* layer_conf,
                              const float* layer_entropy, hipStream_t s);

}  // namespace rpd
