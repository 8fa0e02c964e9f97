// Threshold counts -> keep counts and masks under a compute budget: the
// deterministic budget projection applied at inference (Sec. 3.3), with the
// estimated prefill cost of Eq. (8).  Host-only code.
#pragma once

#include <stdint.h>

#include "../../include/svl.h"

namespace svl {

// One sample's projection.  n_pos: tokens with a positive logit; masks of the
// sample (layer_on [L], head_on [L][A], ffn_on [L][G] or nullptr,
// gate_logits [L][units] or nullptr) are updated in place.  units: gate units
// per layer, n_groups (layer-head controller: a unit is head group j and FFN
// slice j) or 1 (layer controller: a unit is the whole layer).  budget is
// finite and > 0.  Returns the number of visual tokens to keep.
int32_t project_budget_sample(const svl_config& cfg, int32_t n_vision, int32_t n_text,
                              int32_t n_pos, float budget, int64_t vocab, int32_t prefix,
                              uint8_t* layer_on, uint8_t* head_on, uint8_t* ffn_on,
                              const float* gate_logits, int32_t units);

}  // namespace svl
