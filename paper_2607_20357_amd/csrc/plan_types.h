// Plan descriptors and tile sizes shared by the host planner and the
// kernels (plain C++, no HIP types).
#pragma once

#include <stdint.h>

namespace svl {

// ---------------------------------------------------------------------------
// Plan descriptors (built on the host, copied once per call into the
// workspace, read by the kernels).
//
// Row spaces.  The residual stream uses the caller's packed rows (sample b
// at rows cu[b] .. cu[b+1]-1).  On the 16-bit MFMA path the activation
// buffers of the workspace (normed input, Q/K/V, attention output, FFN
// hidden) give every sample a whole number of 16-row blocks: sample b starts
// at padded row pcu[b] = sum over earlier samples of round_up(S, 16).  On the
// float32 path both spaces coincide.

// Rows of one sample handled by a residual / RMSNorm launch.
enum NormFlags : int32_t {
  NORM_ADD_PARTIALS = 1,   // resid += the split-K partial slices, written back
  NORM_WRITE_OUT = 2,      // write the normed rows
};
struct NormSeg {
  int32_t row0;    // first residual row
  int32_t prow0;   // first activation row (padded space)
  int32_t nrows;
  int32_t prefix;  // sum of nrows of the earlier segments of the launch
  int32_t flags;   // NormFlags
  int32_t gprefix; // sum of ceil(nrows / 8) of the earlier segments (8-row groups)
  int32_t pad1, pad2;
};

// One (sample, output-column range) pair of a GEMM launch.  Its tiles are
// nsplit x ceil(nrows/BM) x ceil((n1-n0)/BNO), enumerated split fastest, then
// M tile, then N tile, starting at tile index tile0 of the launch (BNO:
// output columns per tile).
struct GemmGroup {
  int32_t arow0;        // first row of A (activation row space)
  int32_t orow0;        // first output row (residual rows for RESID / PARTIAL,
                        // activation rows otherwise)
  int32_t nrows;
  int32_t n0, n1;       // output columns [n0, n1)
  int32_t kc_off;       // first entry of this group's K chunks in the chunk table
  int32_t kc_cnt;       // number of K chunks
  int32_t nsplit;       // split-K pieces (PARTIAL epilogue only)
  int32_t tile0;        // first tile index of the group
  int32_t pad0, pad1, pad2;
};

// 16-bit MFMA GEMM.  The output columns of a group are cut into 16-column
// blocks.  A block of a PLAIN launch (output / down projection) holds 16
// consecutive columns.  A block of a PAIRED launch holds 8 columns and their
// 8 partners, so a lane (column i of the block) and lane ^ 8 hold both
// members of a pair: for QKV the rotary pair (dim, dim + d/2) of a head, 8
// blocks (d = 128) or 4 blocks (d = 64) per head; for gate/up the gate and
// the up row of the same FFN channel, 8 channels per block.
struct MmGroup {
  int32_t arow0;        // first packed row of A (multiple of 16)
  int32_t orow0;        // first output row (residual rows for RESID / PARTIAL)
  int32_t nrows;
  int32_t wsel;         // weight matrix (QKV: 0 query, 1 key, 2 value; else 0)
  int32_t wrow0;        // weight row of the group's first column (QKV: first
                        // head * d; gate/up: first channel; PLAIN: 0)
  int32_t ocol0;        // output column of the group's first column
  int32_t kc_off;       // first entry of the group's K chunks in the chunk table
  int32_t kc_cnt;
  int32_t rope;         // QKV: rotate (query and key groups)
  int32_t nblocks;      // 16-column blocks
  int32_t fitem0;       // split paired launches: first finish work item of the group
  int32_t kdense;       // >= 0: the group's chunk c starts at column kdense + 64 c
  int32_t pos_base;     // QKV: RoPE position of the group's first row
  int32_t pad0, pad1, pad2;
};

// One workgroup of a 16-bit MFMA GEMM launch: rows [m0, m0 + 256) of its
// group, blocks [b0, b0 + nblk), K chunks [kc0, kc0 + kcn) of the group's
// list; a split-K piece stores its float32 result in partial slice `slice`.
// The record carries the group fields the GEMM reads, resolved for the tile,
// so a workgroup starts from this one 64-byte load.
struct MmTile {
  int32_t arow;     // first packed row of A: group arow0 + m0 (multiple of 16)
  int32_t orow;     // first output row: group orow0 + m0
  int32_t mcnt;     // rows of the tile (1 .. 256)
  int32_t pos0;     // position in the sample of the first row: m0 (RoPE); -1:
                    // the rows span several samples (per-row position table)
  int32_t wsel, wrow0, ocol0, rope;   // as in the group
  int32_t chunk0;   // first entry of the tile's K chunks in the chunk table
  int32_t kcn;      // K chunks
  int32_t kdense;   // >= 0: chunk c starts at column kdense + 64 c (the chunk
                    // table is not read); -1: read it
  int32_t b0, nblk; // 16-column blocks [b0, b0 + nblk) of the group
  int32_t slice;    // split-K piece
  int32_t group;    // group index (planner checks)
  int32_t pad0;
};
static_assert(sizeof(MmTile) == 64, "one 64-byte record per workgroup");

// Decode row-vector launches of a batch: a segment is a run of 16-column
// weight blocks (same block layout as the groups: QKV blocks pair rotary
// dims, gate/up blocks pair gate and up channels) together with the samples
// (uses) whose masks include those blocks, so each weight block is streamed
// once for all of them.  Output / down projection segments multiply the
// union of their samples' active K chunks; a chunk's use mask says which
// samples it belongs to.
constexpr int DEC_MAX_USES = 8;
struct DecUse {
  int32_t arow;     // the sample's activation row
  int32_t orow;     // its output row (activation row, or residual row for RESID)
  int32_t pos;      // RoPE position of its new token
  int32_t pad;
};
struct DecSeg {
  int32_t blk0, nblk;          // launch blocks [blk0, blk0 + nblk)
  int32_t wsel, wrow0, ocol0, rope;   // as in MmGroup
  int32_t nuse, use_off;       // uses [use_off, use_off + nuse) of the use table
  int32_t kc_off, kc_cnt;      // K chunks (the layer's chunk table)
  int32_t kdense;              // >= 0: chunk c starts at kdense + 64 c
  int32_t mask_off;            // >= 0: per-chunk use masks (bit u: use u); -1: every use
};

// One sample of an attention launch: one workgroup per (active head, q tile).
// With a KV cache, the sample's rows are positions pos_base .. pos_base+S-1
// of its cached sequence (prefill: pos_base = 0; decode: S = 1 new row).
struct AttnGroup {
  int32_t row0, S;      // first activation row of the sample, rows in this call
  int32_t h_off, h_cnt; // active query heads: head_table[h_off .. h_off+h_cnt)
  int32_t nqt;          // query tiles
  int32_t tile0;        // first workgroup index of the group
  int32_t sample;       // batch index (cache addressing)
  int32_t pos_base;     // cached positions before this call's rows
  int32_t kv_off, kv_cnt;   // active K/V heads: kvhead_table[kv_off .. kv_off+kv_cnt)
  int32_t pad0, pad1;
};

// K chunk: columns [k0, k0+len) of both operands.
struct KChunk {
  int32_t k0, len;
};

// ---------------------------------------------------------------------------
// Tile sizes (the planner and the kernels must agree).
// 16-bit MFMA path: 256-row tiles (8 waves x 32 rows) of up to
// MFMA_MAX_NB 16-column blocks (the kernel is instantiated for a few block
// counts, the planner picks one per launch); K walks in chunks of 64.
constexpr int MFMA_BM = 256, MFMA_BK = 64;
constexpr int MFMA_MAX_SPLIT = 8;
constexpr int MFMA_MAX_NB = 8;
constexpr int MFMA_PARTIAL_ROWS = 4096;   // split pieces x rows the partial buffer holds
constexpr int F32_BM = 64, F32_BN = 64, F32_BK = 16;
constexpr int F32_SWIGLU_CH = 32;
constexpr int ATTN_BQ = 64;          // query rows per attention workgroup
constexpr int ATTN_BQ_SHORT = 32;    // 16-bit path, launches too short to fill the chip

// Fragment-packed activation layout (16-bit MFMA path).  A matrix with K
// columns (K % 64 == 0) is stored as blocks of 16 rows x 64 columns, 2 KB
// each, block (row/16, k/64) at block index (row/16) * (K/64) + k/64.  Inside
// a block, the element (r, k) sits at
//   ((k / 8) % 2) * 512 + (((k / 16) % 4) * 16 + r % 16) * 8 + k % 8,
// i.e. the first halves of the MFMA fragments of all 64 lanes, then the
// second halves: one 16-byte load per lane reads 1 KB contiguously.
inline constexpr int64_t packed_index(int64_t r, int64_t k, int64_t K) {
  return ((r >> 4) * (K >> 6) + (k >> 6)) * 1024 + ((k >> 3) & 1) * 512 +
         (((k >> 4) & 3) * 16 + (r & 15)) * 8 + (k & 7);
}

}  // namespace svl
