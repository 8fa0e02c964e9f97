// Plan descriptors and tile sizes shared by the host planner and the
// kernels (plain C++, no HIP types).
#pragma once

#include <stdint.h>

namespace svl {

// ---------------------------------------------------------------------------
// Plan descriptors (built on the host, copied once per call into the
// workspace, read by the kernels).

// A run of packed rows belonging to one sample.
struct Seg {
  int32_t row0;    // first packed row
  int32_t nrows;   // rows in the run
  int32_t prefix;  // sum of nrows of the earlier runs in the same list
  int32_t pos0;    // RoPE position of the first row (0: a whole sample)
};

// One (sample, output-column range) pair of a GEMM launch.  Its tiles are
// ceil(nrows/BM) x ceil((n1-n0)/BNO), enumerated M tile fastest, starting at
// tile index tile0 of the launch (BNO: output columns per tile).
struct GemmGroup {
  int32_t row0, nrows;  // rows of A (and of the output) in the packed space
  int32_t n0, n1;       // output columns [n0, n1)
  int32_t kc_off;       // first entry of this group's K chunks in the chunk table
  int32_t kc_cnt;       // number of K chunks
  int32_t tile0;        // first tile index of the group
  int32_t pad0;
};

// One sample of an attention launch: one workgroup per (active head, q tile).
struct AttnGroup {
  int32_t row0, S;      // packed rows of the sample, sequence length
  int32_t h_off, h_cnt; // active query heads: head_table[h_off .. h_off+h_cnt)
  int32_t nqt;          // query tiles
  int32_t tile0;        // first workgroup index of the group
  int32_t pad0, pad1;
};

// K chunk: columns [k0, k0+len) of both operands.
struct KChunk {
  int32_t k0, len;
};

// ---------------------------------------------------------------------------
// Tile sizes (the planner and the kernels must agree).
// bf16: 128-row tiles; the tile width BN (weight rows per tile) is chosen per
// launch from {32, 64, 128} (gate/up tiles hold BN/2 channels).
constexpr int BF16_BM = 128, BF16_BK = 64;
constexpr int F32_BM = 64, F32_BN = 64, F32_BK = 16;
constexpr int F32_SWIGLU_CH = 32;
constexpr int ATTN_BQ = 64;          // query rows per attention workgroup

}  // namespace svl
