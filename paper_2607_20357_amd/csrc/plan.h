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
  int64_t groups_off = 0;   // byte offset of the GemmGroup array in the plan image
  int32_t ngroups = 0;
  int32_t ntiles = 0;
  int32_t bn = 0;           // weight rows per tile (bf16 kernels: 32, 64 or 128)
};

struct AttnLaunch {
  int64_t groups_off = 0, heads_off = 0;
  int32_t ngroups = 0, ntiles = 0;
};

struct NormLaunch {
  int64_t segs_off = 0;
  int32_t nsegs = 0, nrows = 0;
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
  int64_t keep_off = 0, cu_off = 0;
  int32_t max_seq = 0;            // longest sequence (RoPE table rows)
};

struct LayerMasks {
  const uint8_t* layer_on;   // [B]
  const uint8_t* head_mask;  // [B][A], row stride head_stride
  int64_t head_stride;
  const uint8_t* ffn_mask;   // [B][G] with row stride ffn_stride, or nullptr
  int64_t ffn_stride;
};

// Rows of a sample up to which the bf16 GEMMs use their narrow tiles.
constexpr int32_t kSkinnyRows = 256;

// Builds the plan for `nlayers` layers.  seqlens/keep host [B]; masks(l)
// gives layer l's masks.  Returns false with a message on inconsistency.
bool build_plan(const svl_config& cfg, int32_t B, const int32_t* keep, const int32_t* seqlens,
                int32_t nlayers, const LayerMasks* masks, Plan* plan, std::string* err);

// Upper bound of the plan image for any masks.
int64_t plan_bytes_bound(const svl_config& cfg, int32_t B, int32_t nlayers);

}  // namespace svl
