// Internal declarations of libsvl: plan descriptors shared by the host
// planner and the kernels, kernel launchers, and small device helpers.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>
#include <stdint.h>

#include "../../include/svl.h"
#include "plan_types.h"

namespace svl {

enum Epilogue : int32_t {
  EPI_STORE = 0,    // out[row][col] = acc (float32 path)
  EPI_RESID = 1,    // resid[row][col] += acc (float32)
  EPI_SWIGLU = 2,   // out[row][ch] = silu(gate) * up, gate/up tiles paired
  EPI_QKV = 3,      // store, with RoPE applied to query / key columns
  EPI_PARTIAL = 4,  // split-K piece p: partial[p][row][col] = acc (float32)
};

struct GemmArgs {
  const GemmGroup* groups;
  int32_t ngroups, ntiles;
  const KChunk* chunks;
  const void* A;       // activations [rows][lda]
  int32_t lda;
  const void* W0;      // weight row sources ([out][in] layout, row stride ldw)
  const void* W1;
  const void* W2;
  int32_t ldw;
  int32_t nb1, nb2;    // EPI_STORE: columns < nb1 -> W0, < nb2 -> W1, else W2
  void* out;           // output / residual, row stride ldo
  int32_t ldo;
  const float2* rope;  // EPI_QKV: (cos, sin)[pos][head_dim/2]
  int32_t head_dim;    // EPI_QKV: 64 or 128
  int32_t rope_cols;   // EPI_QKV: columns < rope_cols are rotated (Q and K heads)
  float* partial;      // EPI_PARTIAL: split-K slices, slice p at partial + p * pslice
  int64_t pslice;
};

// 16-bit MFMA GEMM (tile table built by the planner).
struct MmArgs {
  const MmGroup* groups;
  const MmTile* tiles;
  int32_t ntiles;
  const KChunk* chunks;
  const void* A;         // fragment-packed activations, K = lda
  const void* A2;        // bf16 products of QKV / gate-up: the low bf16 parts of
                         // the same activations (A2 = bf16(x - A)), same layout,
                         // multiplied after A against the same weights; or nullptr
  int32_t lda;
  const void* W[3];      // bf16 weight matrices [rows][ldw] (gate/up: W[0] gate, W[1] up)
  int32_t w_rows[3];     // their row counts (load range)
  int32_t ldw;
  void* out;             // QKV: row-major 16-bit [rows][ldo]; SWIGLU: packed 16-bit,
                         // K = ldo; RESID: float32 residual [rows][ldo]
  int32_t ldo;
  const float2* rope;    // QKV: (cos, sin)[pos][head_dim/2]
  int32_t head_dim;
  float* partial;        // split-K slices: slice p at partial + p * pslice
  int64_t pslice;
  int32_t split;         // QKV / SWIGLU: > 1 stores raw float32 pieces (row stride
                         // pld; SWIGLU: gate columns, then up columns at pld / 2)
                         // for the finish kernel; PARTIAL: row stride ldo
  int32_t pld;
  int32_t ngroups;       // row-vector launches (decode): groups, and the blocks
  int32_t nblocks;       // of all groups (a group's first block in its pad0)
  const DecSeg* segs;    // shared row-vector launches (decode of a batch): segments,
  int32_t nsegs;         // their uses and per-chunk use masks; nblocks counts
  const DecUse* uses;    // the segments' blocks
  const int32_t* cmasks;
  int32_t max_uses;      // most uses of a segment
  const int32_t* rowpos; // per activation row: RoPE position in its sample (QKV
                         // tiles spanning samples: pos0 < 0)
};

// Finish of a split QKV / gate-up launch: sums the split slices in order,
// then RoPE (QKV) or silu(gate) * up (SWIGLU), rounded once to 16 bits.
struct FinishArgs {
  const MmGroup* groups;     // the GEMM launch's groups; pad0 = first work item
  int32_t ngroups, nitems;
  const float* partial;
  int64_t pslice;
  int32_t pld, nsplit;
  void* out;                 // QKV: row-major [rows][ldo]; SWIGLU: packed, K = ldo
  int32_t ldo;
  const float2* rope;
  int32_t head_dim;
};

struct AttnArgs {
  const AttnGroup* groups;
  int32_t ngroups, ntiles;
  const int32_t* head_table;
  const void* qkv;     // [rows][(A + 2 KV) d]: Q heads, then K heads, then V heads
  int32_t ldq;         // row stride of qkv
  int32_t n_heads, n_kv_heads;
  void* out;           // [rows][A d]: fragment-packed (16-bit) or row-major (float32)
  int32_t ldo;
  const float2* rope;  // (cos, sin)[pos][d/2]; used by kernels that rotate on load
  float scale;         // 1/sqrt(d)
  // KV cache of this layer (decode attention reads it, the append writes it):
  // [batch][n_kv_heads][2][max_len][d], activation type
  void* cache;
  int32_t max_len;
  const int32_t* kvhead_table;
  int32_t max_kv_cnt;
  int32_t bq;          // query rows per workgroup of the 16-bit prefill attention
};

constexpr int NORM_INLINE_SEGS = 8;
struct NormArgs {
  const NormSeg* segs;
  int32_t nsegs, nrows;
  // launches of up to NORM_INLINE_SEGS segments carry them here (read from
  // the kernel arguments, no dependent global load); longer ones read segs
  NormSeg inl[NORM_INLINE_SEGS];
  int32_t ngroups8;    // 8-row groups (row-group kernel grid)
  int32_t rows8;       // 1: the 8-row-group kernel (16-bit output)
  int32_t rowmajor;    // 1: 16-bit output row-major [rows][D] (decode), else packed
  float* x;            // residual [rows][D] (written back when partials are added)
  const float* partial;  // split-K slices to add: slice p at partial + p * pslice
  int32_t nsplit;
  int64_t pslice;
  const void* gain;    // [D], weight dtype
  void* out;           // normed rows: fragment-packed (16-bit) or row-major (float32)
  void* out2;          // bf16 packed output: the low parts bf16(x - out), or nullptr
  int32_t D;
  float eps;
};

// Small matrix-vector products of the compute controller:
// y[r][o] = act(sum_i W[o][i] x[r][i] + bias[o]) (+ add[row(r)][o]) for
// r < nvec, W [out][in] in the storage dtype (in % 8 == 0, rows 16-byte
// aligned), x / y / add float32.  add_cu: row(r) = add_cu[r+1] - 1 (the last
// packed row of sample r), else row(r) = r.
enum CtrlAct : int32_t { CTRL_ACT_NONE = 0, CTRL_ACT_GELU = 1 };
struct CtrlLinearArgs {
  const void* W;
  const void* bias;     // [out] or nullptr
  int32_t in, out, nvec, act;
  const float* x;
  int64_t ldx;
  const float* add;
  const int32_t* add_cu;
  int64_t ldadd;
  float* y;
  int64_t ldy;
};

// Row moves of the controlled prefill: new packing from the old one after
// the budget projection shortened the visual blocks.
struct CompactArgs {
  const float* src;          // old packed rows [old rows][D]
  float* dst;                // new packed rows [new rows][D]
  const int32_t* old_cu;     // [B+1]
  const int32_t* old_keep;   // [B]
  const int32_t* old_kidx;   // [B][N], ascending kept indices
  const int32_t* new_cu;
  const int32_t* new_keep;
  const int32_t* new_kidx;   // subset of old_kidx per sample
  int32_t B, N, D;
};

// Training-time budget term, per sample b (rows of N tokens / nl = (L-P) U
// units).  Cost constants: c1 = 8 D^2 + 6 D F, c2 = 4 D, lm = 2 D V,
// full = C_full; budget is the float32 budget's value.
struct BudgetLossArgs {
  const float* z;          // [B][N] token logits
  const float* xi_tok;     // [B][N] noise or nullptr
  const float* gl;         // [B][nl] gate logits
  const float* xi_gate;    // [B][nl] noise or nullptr
  int32_t N, T, L, P, U;
  double c1, c2, lm, full;
  double budget, margin, w_over, w_under, lam, tau_comp;
  uint8_t* tok_mask;       // [B][N]
  uint8_t* unit_mask;      // [B][nl]
  float* ratio;            // [B]
  float* loss;             // [B]
  float* grad_z;           // [B][N]
  float* grad_gate;        // [B][nl]
};

// ---------------------------------------------------------------------------
// Launchers (each returns hipSuccess or the launch error).
hipError_t launch_count_positive(const float* logits, int32_t B, int32_t N, int32_t* counts,
                                 hipStream_t st);
hipError_t launch_select(const float* scores, int32_t B, int32_t N, const int32_t* keep_dev,
                         int32_t* kept_idx, hipStream_t st);
hipError_t launch_gather(const int32_t* kept_idx, const int32_t* keep_dev, const int32_t* cu_dev,
                         int32_t B, int32_t N, int32_t T, int32_t D, int32_t total_rows,
                         const void* vision, const void* text, int32_t dtype, float* resid,
                         hipStream_t st);
// out_kind: 0 float32 row-major, 1 bf16 packed, 2 fp16 packed
hipError_t launch_resid_norm(const NormArgs& a, int32_t out_kind, hipStream_t st);
// waves: 8 (any epilogue and block count) or 4 (EPI_RESID with 4 blocks)
hipError_t launch_gemm_mfma(const MmArgs& a, int32_t epi, int32_t nb, int32_t waves, bool f16,
                            hipStream_t st);
hipError_t launch_finish(const FinishArgs& a, int32_t epi, bool f16, hipStream_t st);
// Decode: one-row groups, one workgroup per 16-column block (QKV, SWIGLU, RESID).
hipError_t launch_gemv_shared(const MmArgs& a, int32_t epi, bool f16, hipStream_t st);
hipError_t launch_gemv(const MmArgs& a, int32_t epi, bool f16, hipStream_t st);
hipError_t launch_gemm_f32(const GemmArgs& a, int32_t epi, hipStream_t st);
hipError_t launch_attn_mfma(const AttnArgs& a, int32_t head_dim, bool f16, hipStream_t st);
// KV cache: append this call's K / V rows; decode attention over the cache.
hipError_t launch_kv_append(const AttnArgs& a, int32_t head_dim, hipStream_t st);
hipError_t launch_attn_decode(const AttnArgs& a, int32_t head_dim, bool f16, hipStream_t st);
hipError_t launch_attn_f32(const AttnArgs& a, int32_t head_dim, hipStream_t st);
hipError_t launch_rope_table(float2* table, int32_t max_pos, int32_t head_dim, float theta,
                             hipStream_t st);
// Compute controller.
hipError_t launch_ctrl_stats(const float* z, int32_t B, int32_t N, int32_t* counts, double* kappa,
                             hipStream_t st);
hipError_t launch_pe(const double* xs, double x0, int32_t nvec, int32_t E, double scale,
                     double base, float* out, hipStream_t st);
hipError_t launch_ctrl_linear(const CtrlLinearArgs& a, bool bf16, hipStream_t st);
hipError_t launch_budget_rows(const float* eb, const int32_t* cu, int32_t B, int32_t D,
                              float* resid, hipStream_t st);
hipError_t launch_compact_rows(const CompactArgs& a, int32_t rows, hipStream_t st);
hipError_t launch_budget_loss(const BudgetLossArgs& a, int32_t B, hipStream_t st);
hipError_t launch_fill_i32(int32_t* p, int32_t value, int64_t n, hipStream_t st);
// *flag = SVL_STATUS_NONFINITE if one of x[0..n) (n % 4 == 0) is inf or NaN
hipError_t launch_nonfinite(const float* x, int64_t n, uint32_t* flag, hipStream_t st);

// Shared by the C-ABI sources: sets the per-thread message of svl_last_error
// and returns st; validates a config as every entry point does.
svl_status set_error(svl_status st, const char* msg);
svl_status validate_config(const svl_config* c);

}  // namespace svl
