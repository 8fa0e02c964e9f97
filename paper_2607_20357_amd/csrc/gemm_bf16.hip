// Masked grouped GEMM on bf16 MFMA (gfx950 v_mfma_f32_16x16x32_bf16).
//
//   C[rows, cols] = sum over the group's K chunks of A[rows, k] * W[cols, k]
//
// A is an activation matrix (packed rows, row-major), W a weight matrix in
// [out][in] layout.  A launch is a list of groups (one sample and one active
// column range each, or one sample and its active K chunks), so weight rows of
// inactive heads / FFN slices (QKV, gate/up) and weight columns of inactive
// heads / slices (output and down projections) are never read.
//
// Tile: 128 x 128 x 64, 256 threads = 4 waves in a 2 x 2 grid, each wave a
// 64 x 64 block of 16 x 16 MFMA tiles.  A and W tiles are staged through LDS
// (double-buffered; rows padded to 144 B so that the 16-lane fragment reads
// hit distinct banks), the next chunk's global loads are in flight while the
// current chunk is multiplied.
//
// Split-K: a group may be cut into nsplit K ranges.  Each piece stores its
// float32 partial tile to the workspace; the last piece to arrive (integer
// arrival counter) adds the pieces in split order, so the result does not
// depend on arrival order, and runs the epilogue.
//
// Epilogues:
//   QKV: store as bf16; query and key columns are first rotated by RoPE at
//     the row's position inside its sample (the float32 accumulators are
//     rotated, so Q and K are rounded to bf16 once).  Rotation pairs dims
//     (r, r + d/2) of a head; for d = 128 the tile's weight rows are
//     interleaved so that one lane holds both members of each pair;
//   RESID: add into the float32 residual (output and down projections);
//   SWIGLU: the tile's 128 weight rows are 64 gate rows and the 64 matching
//     up rows, interleaved so that one lane holds both the gate and the up
//     value of a channel, and silu(gate) * up is stored.
#include "svl_internal.h"
#include "device_util.h"

namespace svl {
namespace {

constexpr int BM = BF16_BM, BN = BF16_BN, BK = BF16_BK;
constexpr int LDS_STRIDE = BK + 8;   // bf16 elements per LDS row
constexpr int NT = 256;

template <int EPI>
__global__ __launch_bounds__(NT, 2) void gemm_bf16_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LDS_STRIDE];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * LDS_STRIDE];
  __shared__ int s_last;

  const int t = xcd_tile_index();
  if (t >= a.ntiles) return;
  const GemmGroup g = a.groups[find_group(a.groups, a.ngroups, t)];
  constexpr int BNO = (EPI == EPI_SWIGLU) ? BF16_SWIGLU_CH : BN;  // output columns per tile
  const int local = t - g.tile0;
  const int split = local % g.nsplit;
  const int rest = local / g.nsplit;
  const int nm = (g.nrows + BM - 1) / BM;
  const int mt = rest % nm, nt = rest / nm;
  const int mrow0 = g.row0 + mt * BM;
  const int mcnt = min(BM, g.nrows - mt * BM);
  const int n0 = g.n0 + nt * BNO;
  const int ncnt = min(BNO, g.n1 - n0);
  const int kc0 = g.kc_off + (g.kc_cnt * split) / g.nsplit;
  const int kc1 = g.kc_off + (g.kc_cnt * (split + 1)) / g.nsplit;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // Loader: thread covers 16-byte column chunk lc of rows lr + 32 i.
  const int lc = tid & 7, lr = tid >> 3;
  const uint16_t* Ab = static_cast<const uint16_t*>(a.A);
  const uint16_t* a_ptr[4];
  const uint16_t* b_ptr[4];
  bool a_ok[4], b_ok[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = lr + 32 * i;
    a_ok[i] = r < mcnt;
    a_ptr[i] = Ab + (size_t)(mrow0 + (a_ok[i] ? r : 0)) * a.lda + lc * 8;
    const uint16_t* src;
    int wrow;
    if constexpr (EPI == EPI_SWIGLU) {
      const int half = r >> 6, j = (r & 63) >> 4;
      const int ch = half * 32 + (j & 1) * 16 + (r & 15);
      b_ok[i] = ch < ncnt;
      src = static_cast<const uint16_t*>((j >> 1) ? a.W1 : a.W0);
      wrow = n0 + (b_ok[i] ? ch : 0);
    } else if constexpr (EPI == EPI_QKV) {
      // tile row r -> head dim: d = 128 interleaves the two rotation halves
      const int half = r >> 6, j = (r & 63) >> 4;
      const int tr = (a.head_dim == 128) ? (j >> 1) * 64 + half * 32 + (j & 1) * 16 + (r & 15) : r;
      b_ok[i] = tr < ncnt;
      const int col = n0 + (b_ok[i] ? tr : 0);
      if (n0 < a.nb1) { src = static_cast<const uint16_t*>(a.W0); wrow = col; }
      else if (n0 < a.nb2) { src = static_cast<const uint16_t*>(a.W1); wrow = col - a.nb1; }
      else { src = static_cast<const uint16_t*>(a.W2); wrow = col - a.nb2; }
    } else {
      b_ok[i] = r < ncnt;
      src = static_cast<const uint16_t*>(a.W0);
      wrow = n0 + (b_ok[i] ? r : 0);
    }
    b_ptr[i] = src + (size_t)wrow * a.ldw + lc * 8;
  }

  // Rows outside the tile read a valid row of the same group (row 0 of the
  // tile) and are zeroed in registers, so the loads carry no branches.
  uint4 ra[4], rb[4];
  auto gload = [&](int kc) {
    const int k0 = a.chunks[kc].k0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint4 va = *reinterpret_cast<const uint4*>(a_ptr[i] + k0);
      uint4 vb = *reinterpret_cast<const uint4*>(b_ptr[i] + k0);
      ra[i] = a_ok[i] ? va : make_uint4(0, 0, 0, 0);
      rb[i] = b_ok[i] ? vb : make_uint4(0, 0, 0, 0);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *reinterpret_cast<uint4*>(&As[buf][(lr + 32 * i) * LDS_STRIDE + lc * 8]) = ra[i];
      *reinterpret_cast<uint4*>(&Bs[buf][(lr + 32 * i) * LDS_STRIDE + lc * 8]) = rb[i];
    }
  };

  floatx4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int buf) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8_t af[4], bfr[4];
      const int koff = ks * 32 + (lane >> 4) * 8;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t*>(
            &As[buf][(wm * 64 + i * 16 + (lane & 15)) * LDS_STRIDE + koff]);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8_t*>(
            &Bs[buf][(wn * 64 + j * 16 + (lane & 15)) * LDS_STRIDE + koff]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
  };

  if (kc0 < kc1) {
    gload(kc0);
    lstore(0);
    __syncthreads();
    int buf = 0;
    for (int kc = kc0; kc < kc1; ++kc) {
      // the last iteration reloads its own chunk into the idle buffer
      gload(min(kc + 1, kc1 - 1));
      compute(buf);
      lstore(buf ^ 1);
      __syncthreads();
      buf ^= 1;
    }
  }

  if (g.nsplit > 1) {
    const int ctr = g.ctr0 + rest;
    float* base = a.partial + (size_t)ctr * g.nsplit * SPLITK_SLOT_FLOATS;
    floatx4* mine = reinterpret_cast<floatx4*>(base + (size_t)split * SPLITK_SLOT_FLOATS) + tid * 16;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) mine[i * 4 + j] = acc[i][j];
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = (atomicAdd(&a.counters[ctr], 1) == g.nsplit - 1);
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    floatx4 sum[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) sum[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < g.nsplit; ++s) {
      const floatx4* p = reinterpret_cast<const floatx4*>(base + (size_t)s * SPLITK_SLOT_FLOATS) + tid * 16;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) sum[i][j] += (s == split) ? acc[i][j] : p[i * 4 + j];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = sum[i][j];
    if (tid == 0) a.counters[ctr] = 0;
  }

  // Epilogue.  acc[i][j][r] is C[wm*64 + i*16 + 4*(lane/16) + r][wn*64 + j*16 + lane%16].
  const int rbase = wm * 64 + (lane >> 4) * 4;
  if constexpr (EPI == EPI_QKV) {
    uint16_t* out = static_cast<uint16_t*>(a.out);
    const bool rot = n0 < a.rope_cols;
    const int hd = a.head_dim, half = hd >> 1;
    // d = 128: this wave holds dims wn*32 + [0,32) (blocks 0,1) and the same
    // dims + 64 (blocks 2,3).  d = 64: this wave holds head wn of the tile,
    // dims [0,32) (blocks 0,1) and [32,64) (blocks 2,3).
    const int cbase = (hd == 128) ? wn * 32 : wn * 64;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rbase + i * 16 + r;
        const int rowc = min(row, mcnt - 1);
        const int pos = (mrow0 - g.row0) + rowc;
        uint16_t* orow = out + (size_t)(mrow0 + rowc) * a.ldo + n0;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int dim = j * 16 + (lane & 15) + ((hd == 128) ? wn * 32 : 0);  // in [0, d/2)
          const int c1 = (hd == 128) ? dim : cbase + dim;
          const int c2 = c1 + half;
          float v1 = acc[i][j][r], v2 = acc[i][j + 2][r];
          if (rot) {
            const float2 cs = a.rope[(size_t)pos * half + dim];
            const float o1 = v1 * cs.x - v2 * cs.y;
            const float o2 = v2 * cs.x + v1 * cs.y;
            v1 = o1;
            v2 = o2;
          }
          if (row < mcnt && c1 < ncnt) orow[c1] = f32_to_bf16_bits(v1);
          if (row < mcnt && c2 < ncnt) orow[c2] = f32_to_bf16_bits(v2);
        }
      }
  } else if constexpr (EPI == EPI_RESID) {
    float* out = static_cast<float*>(a.out);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rbase + i * 16 + r;
        float* orow = out + (size_t)(mrow0 + min(row, mcnt - 1)) * a.ldo + n0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int col = wn * 64 + j * 16 + (lane & 15);
          if (row < mcnt && col < ncnt) orow[col] += acc[i][j][r];
        }
      }
  } else {
    uint16_t* out = static_cast<uint16_t*>(a.out);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rbase + i * 16 + r;
        uint16_t* orow = out + (size_t)(mrow0 + min(row, mcnt - 1)) * a.ldo + n0;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int ch = wn * 32 + j * 16 + (lane & 15);
          const float gt = acc[i][j][r], up = acc[i][j + 2][r];
          if (row < mcnt && ch < ncnt) orow[ch] = f32_to_bf16_bits(gt / (1.0f + __expf(-gt)) * up);
        }
      }
  }
}

}  // namespace

hipError_t launch_gemm_bf16(const GemmArgs& a, int32_t epi, hipStream_t st) {
  if (a.ntiles <= 0) return hipSuccess;
  const unsigned grid = (unsigned)((a.ntiles + 7) / 8 * 8);
  switch (epi) {
    case EPI_QKV: gemm_bf16_kernel<EPI_QKV><<<grid, NT, 0, st>>>(a); break;
    case EPI_RESID: gemm_bf16_kernel<EPI_RESID><<<grid, NT, 0, st>>>(a); break;
    default: gemm_bf16_kernel<EPI_SWIGLU><<<grid, NT, 0, st>>>(a); break;
  }
  return hipGetLastError();
}

}  // namespace svl
