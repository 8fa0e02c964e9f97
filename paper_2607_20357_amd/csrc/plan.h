// Host planner: turns sequence lengths and the controller masks into the
// work descriptors each kernel launch reads.  Host-only code.
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/svl.h"
#include "plan_types.h"

namespace svl {

struct GemmLaunch {
  int64_t groups_off = 0;   // byte offset of the group array in the plan image
                            // (MmGroup on the 16-bit MFMA path, GemmGroup on the
                            // float32 path)
  int64_t tiles_off = 0;    // 16-bit MFMA path: byte offset of the MmTile table
  int32_t ngroups = 0;
  int32_t ntiles = 0;
  int32_t nb = 0;           // 16-bit MFMA path: kernel block count (tiles hold <= nb)
  int32_t waves = 8;        // 16-bit MFMA path: waves per workgroup (8, or 4 for wide
                            // residual-add launches)
  int32_t nsplit = 1;       // > 1: split-K pieces written as float32 partial slices
  int32_t nitems = 0;       // split QKV / gate-up launches: finish kernel work items
  int32_t nblocks = 0;      // 16-bit path: the groups' 16-column blocks (each group's
                            // first block in MmGroup::pad0); shared row-vector
                            // launches: the segments' blocks
  // shared row-vector launch (decode of a batch), nsegs > 0
  int64_t segs_off = 0, uses_off = 0, cmasks_off = 0;
  int32_t nsegs = 0, max_uses = 0;
};

struct AttnLaunch {
  int64_t groups_off = 0, heads_off = 0, kvheads_off = 0;
  int32_t ngroups = 0, ntiles = 0;
  int32_t max_kv_cnt = 0;   // most active K/V heads of a group (cache append grid)
  int32_t bq = ATTN_BQ;     // query rows per workgroup (ATTN_BQ or ATTN_BQ_SHORT)
};

// A residual / RMSNorm launch: adds pending split-K partials (nsplit slices)
// into the residual rows flagged for it, and writes the normed rows flagged
// for it.
struct NormLaunch {
  int64_t segs_off = 0;
  int32_t nsegs = 0, nrows = 0;
  int32_t ngroups8 = 0;     // sum over segments of ceil(nrows / 8)
  bool rows8 = false;       // 16-bit output through the 8-row-group kernel
  int32_t nsplit = 0;       // partial slices to add (0: none pending)
  bool write_out = false;   // some segment writes normed rows
};

struct LayerPlan {
  NormLaunch norm_attn, norm_ffn;
  GemmLaunch qkv, o, gu, down;
  AttnLaunch attn;
  int64_t chunks_off = 0;   // byte offset of this layer's KChunk table
};

// The plan image is copied verbatim to the start of the workspace.  Its
// header holds keep[B] and cu_seqlens[B+1] (device copies for the select and
// gather kernels).
struct Plan {
  std::vector<uint8_t> image;
  std::vector<LayerPlan> layers;
  NormLaunch final_norm;          // adds the last layer's pending partials
  int64_t keep_off = 0, cu_off = 0;
  // per activation row (padded space): its RoPE position inside its sample
  // (padding rows: 0), read by QKV tiles that span several samples
  int64_t rowpos_off = 0;
  int32_t max_seq = 0;            // most rows of one sample in this call
  int32_t max_pos = 0;            // positions the RoPE table covers: max of pos_base + rows
  int32_t padded_rows = 0;        // rows of the activation buffers
};

struct LayerMasks {
  const uint8_t* layer_on;   // [B]
  const uint8_t* head_mask;  // [B][A], row stride head_stride
  int64_t head_stride;
  const uint8_t* ffn_mask;   // [B][G] with row stride ffn_stride, or nullptr
  int64_t ffn_stride;
};

// Rows of a sample up to which the 16-bit MFMA GEMMs count a sample as
// skinny (one M tile): the output and down projections then split K so the
// launch still covers the CUs.
constexpr int32_t kSkinnyRows = MFMA_BM;
// Workgroups a launch aims for (one per CU).
constexpr int32_t kTargetTiles = 256;
// Norm launches of at least this many rows (16-bit output) use the 8-row
// group kernel (whole packed lines per store) instead of one row per
// workgroup (more workgroups for short launches: at 208 rows the 8-row
// kernel's 26 workgroups take 29.5 us against 11.1; from 1024 rows it is
// faster, 18.7 -> 12.6 us per launch on a ragged batch of 8).
constexpr int32_t kNormRows8 = 1024;

// Builds the plan for `nlayers` layers.  seqlens/keep host [B]; masks[l]
// gives layer l's masks.  Returns false with a message on inconsistency.
// pos_base (host [B] or nullptr = all 0): positions already cached per sample
// (decode); the rows of sample b are positions pos_base[b] .. + seqlens[b]-1.
bool build_plan(const svl_config& cfg, int32_t B, const int32_t* keep, const int32_t* seqlens,
                int32_t nlayers, const LayerMasks* masks, Plan* plan, std::string* err,
                const int32_t* pos_base = nullptr);

// Upper bound of the plan image for any masks (B samples, R packed rows).
int64_t plan_bytes_bound(const svl_config& cfg, int32_t B, int32_t R, int32_t nlayers);

// Upper bound of the padded activation rows for B samples and R packed rows.
inline int64_t padded_rows_bound(const svl_config& cfg, int32_t B, int32_t R) {
  return cfg.dtype == SVL_BF16 ? (int64_t)R + 15 * (int64_t)B : (int64_t)R;
}

// Floats of split-K partial slices the workspace holds: (split pieces x
// rows) up to min(8 x padded rows, MFMA_PARTIAL_ROWS), each as wide as the
// widest split output (d_model for the output / down projections, the Q/K/V
// width, or gate + up = 2 d_ffn).  The planner splits a launch only while its
// slices fit.
inline int64_t partial_floats_bound(const svl_config& cfg, int32_t B, int32_t R) {
  if (cfg.dtype != SVL_BF16) return 0;
  int64_t r = padded_rows_bound(cfg, B, R) * MFMA_MAX_SPLIT;
  if (r > MFMA_PARTIAL_ROWS) r = MFMA_PARTIAL_ROWS;
  int64_t w = cfg.d_model;
  const int64_t qkv = (int64_t)(cfg.n_heads + 2 * cfg.n_kv_heads) * cfg.head_dim;
  if (qkv > w) w = qkv;
  if (2 * (int64_t)cfg.d_ffn > w) w = 2 * (int64_t)cfg.d_ffn;
  return r * w;
}

}  // namespace svl
