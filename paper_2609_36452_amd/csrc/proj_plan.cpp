// Host side of the projection: the tile plan for a row bound, and the
// dispatch to the kernel variant it names.
#include "rpd_launch.h"

namespace rpd {

ProjPlan plan_projection(int dtype, long long rows_cap, int V) {
  ProjPlan p{};
  if (rows_cap < 1) rows_cap = 1;
  if (dtype == 1) {   // fp32
    p.variant = PROJ_F32;
    p.rows_per_tile = 16;
    p.vocab_cap = 64;
    p.nvt = (V + 63) / 64;
    p.nrt = (int)((rows_cap + 15) / 16);
    p.split_rows = 0;
    p.per_xcd = 0;
    p.grid = p.nvt * p.nrt;
    return p;
  }
  if (rows_cap <= kStreamMaxRows) {
    // HBM-bound: one row tile holding every projected row, so W_U is read
    // once; a multiple of 256 equal vocabulary tiles, so every CU streams the
    // same share
    p.variant = rows_cap <= 32 ? PROJ_BF16_S32 : PROJ_BF16_S64;
    p.rows_per_tile = rows_cap <= 32 ? 32 : 64;
    p.vocab_cap = kStreamTileVocab;
    int nvt = (V + p.vocab_cap - 1) / p.vocab_cap;
    nvt = ((nvt + 255) / 256) * 256;
    p.nvt = nvt < V ? nvt : V;
  } else if (rows_cap <= kBigTileRowsMid) {
    // one MFMA tile of 256 vocabulary rows x 128 projected rows per vocabulary tile
    p.variant = PROJ_BF16_BIG128;
    p.rows_per_tile = kBigTileRowsMid;
    p.vocab_cap = kBigTileVocab;
    p.nvt = (V + p.vocab_cap - 1) / p.vocab_cap;
  } else {
    // MFMA tiles of 256 vocabulary rows x 256 or 192 projected rows, whichever
    // pads the rows less (ties to 256)
    const long long pad256 = (rows_cap + kBigTileRows - 1) / kBigTileRows * kBigTileRows;
    const long long pad192 = (rows_cap + kBigTileRowsSmall - 1) / kBigTileRowsSmall * kBigTileRowsSmall;
    p.variant = pad192 < pad256 ? PROJ_BF16_BIG192 : PROJ_BF16_BIG;
    p.rows_per_tile = pad192 < pad256 ? kBigTileRowsSmall : kBigTileRows;
    p.vocab_cap = kBigTileVocab;
    p.nvt = (V + p.vocab_cap - 1) / p.vocab_cap;
  }
  p.nrt = (int)((rows_cap + p.rows_per_tile - 1) / p.rows_per_tile);
  p.split_rows = p.nrt >= 8 ? 1 : 0;
  p.per_xcd = p.split_rows ? ((p.nrt + 7) / 8) * p.nvt : ((p.nvt + 7) / 8) * p.nrt;
  p.grid = 8 * p.per_xcd;
  return p;
}

hipError_t launch_projection(const Launch& a, hipStream_t s) {
  if (a.max_masked <= 0) return hipSuccess;
  switch (a.plan.variant) {
    case PROJ_BF16_S32:
    case PROJ_BF16_S64: return launch_proj_stream(a, s);
    case PROJ_BF16_BIG:
    case PROJ_BF16_BIG192:
    case PROJ_BF16_BIG128: return launch_proj_big(a, s);
    case PROJ_F32: return launch_proj_f32(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace rpd
