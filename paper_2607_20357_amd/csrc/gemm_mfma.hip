// Masked grouped GEMM on 16-bit MFMA (gfx950 v_mfma_f32_16x16x32_{f16,bf16}).
//
//   C[rows, cols] = sum over the group's K chunks of A[rows, k] * W[cols, k]
//
// A is an activation matrix (packed rows, row-major, fp16 or bf16), W a bf16
// weight matrix in [out][in] layout.  With fp16 activations each weight tile
// is widened bf16 -> fp16 on its way into LDS (exact inside fp16's range), so
// both operands of the fp16 MFMA carry 11-bit significands; with bf16
// activations the weights go through unchanged.  Accumulation is float32.
//
// A launch is a list of groups (one sample and one active column range each,
// or one sample and its active K chunks), so weight rows of inactive heads /
// FFN slices (QKV, gate/up) and weight columns of inactive heads / slices
// (output and down projections) are never read.
//
// Tile: 128 rows x BN weight rows x 64 k, 256 threads = 4 waves, each wave 32
// rows x BN columns of 16 x 16 MFMA blocks.  A and W tiles go through LDS
// (rows padded to 144 B so the 16-lane fragment reads hit distinct banks).
// Global loads run two chunks ahead of the MFMAs (two register stages, two
// LDS buffers); the loads are unconditional (rows outside the tile read a
// valid row and are masked to zero in registers) so the compiler can wait on
// exactly the older stage.
//
// Prefill shapes are skinny (a sample has a few hundred rows): every output
// column tile is computed by ceil(rows/128) workgroups with adjacent tile
// indices, which the XCD-aware numbering places on one XCD at about the same
// time, so each weight tile comes from HBM once and is shared through that
// XCD's L2.  Narrow N tiles (32 or 64 weight rows) give every launch enough
// workgroups for the 256 CUs without splitting K, so each output element is
// produced by exactly one workgroup (deterministic, no reduction).
//
// Epilogues:
//   QKV: store; query and key columns are first rotated by RoPE at the row's
//     position inside its sample (the float32 accumulators are rotated, so
//     Q and K are rounded once).  Rotation pairs dims (r, r + d/2) of a head;
//     the tile's weight rows are ordered so that one lane holds both members
//     of each pair (for d = 128 a 64-row tile holds dims t*32 + [0,32) and
//     64 + t*32 + [0,32), t = 0, 1);
//   RESID: add into the float32 residual (output and down projections);
//   SWIGLU: the tile's weight rows are BN/2 gate rows followed by the BN/2
//     matching up rows, so one lane holds the gate and the up value of a
//     channel, and silu(gate) * up is stored.
#include "svl_internal.h"
#include "device_util.h"

namespace svl {
namespace {

constexpr int BM = BF16_BM, BK = BF16_BK;
constexpr int LDS_STRIDE = BK + 8;   // 16-bit elements per LDS row
constexpr int NT = 256;
constexpr int MAX_CHUNKS = 1024;     // K chunks per group (K <= 65536)

// Raw buffer resource over [p, p + bytes): loads past the end return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint4 load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

template <bool F16>
__device__ __forceinline__ uint4 weight_to_act(const uint4& v) {
  if constexpr (F16) {
    return make_uint4(bf16x2_to_f16x2(v.x), bf16x2_to_f16x2(v.y), bf16x2_to_f16x2(v.z),
                      bf16x2_to_f16x2(v.w));
  } else {
    return v;
  }
}

template <int EPI, int BN, bool F16>
__global__ __launch_bounds__(NT, 2) void gemm_mfma_kernel(GemmArgs a) {
  constexpr int NB = BN / 16;                             // 16-column blocks per wave
  constexpr int BNO = (EPI == EPI_SWIGLU) ? BN / 2 : BN;  // output columns per tile
  constexpr int WLD = BN * 8 / NT;                        // 16-byte W loads per thread
  static_assert(WLD >= 1, "BN too small");
  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LDS_STRIDE];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * LDS_STRIDE];
  __shared__ int32_t s_k0[MAX_CHUNKS];   // the group's chunk offsets (LDS reads, no vmcnt waits)

  const int t = xcd_tile_index();
  if (t >= a.ntiles) return;
  const GemmGroup g = a.groups[find_group(a.groups, a.ngroups, t)];
  const int local = t - g.tile0;
  const int nm = (g.nrows + BM - 1) / BM;
  const int mt = local % nm, nt = local / nm;
  const int mrow0 = g.row0 + mt * BM;
  const int mcnt = min(BM, g.nrows - mt * BM);
  const int n0 = g.n0 + nt * BNO;
  const int ncnt = min(BNO, g.n1 - n0);
  const int kc0 = g.kc_off, nk = g.kc_cnt;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int c = tid; c < nk; c += NT) s_k0[c] = a.chunks[kc0 + c].k0;
  __syncthreads();

  // QKV: head base and which 32-dim quarter pair this tile holds (d = 128)
  int hbase = n0, quarter = 0;
  if constexpr (EPI == EPI_QKV) {
    if (a.head_dim == 128) {
      hbase = n0 - (n0 % 128);
      quarter = (n0 % 128) / 64;
    }
  }

  // Loader: A rows lr + 32 i (i < 4), W rows lr + 32 i (i < WLD), 16-byte
  // chunk lc.  Buffer loads: one resource per operand spans exactly the
  // tile's valid rows, so rows past the tile read as zero, the per-thread
  // byte offsets are fixed and the chunk offset is a scalar.
  const int lc = tid & 7, lr = tid >> 3;
  const uint16_t* Ab = static_cast<const uint16_t*>(a.A) + (size_t)mrow0 * a.lda;
  const __amdgpu_buffer_rsrc_t rsA = make_rsrc(Ab, (uint32_t)mcnt * a.lda * 2u);
  uint32_t voA[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) voA[i] = (uint32_t)(lr + 32 * i) * a.lda * 2u + lc * 16u;

  __amdgpu_buffer_rsrc_t rsB[WLD];
  uint32_t voB[WLD];
#pragma unroll
  for (int i = 0; i < WLD; ++i) {
    const int r = lr + 32 * i;     // tile row (weight row of the tile)
    const uint16_t* base;
    int nrows, row;
    if constexpr (EPI == EPI_SWIGLU) {
      // rows [0, BN/2) are gate channels n0.., rows [BN/2, BN) the same up
      // channels; lr < 32, so load i covers gate rows iff i < WLD/2
      base = static_cast<const uint16_t*>(i < WLD / 2 ? a.W0 : a.W1);
      row = r - (i < WLD / 2 ? 0 : BN / 2);
      nrows = ncnt;
    } else if constexpr (EPI == EPI_QKV) {
      int first;
      if (a.head_dim == 128) {
        first = hbase;
        row = (r < 32) ? quarter * 32 + r : 64 + quarter * 32 + (r - 32);
        nrows = 128;
      } else {
        first = n0;
        row = r;
        nrows = ncnt;
      }
      if (first < a.nb1) base = static_cast<const uint16_t*>(a.W0) + (size_t)first * a.ldw;
      else if (first < a.nb2) base = static_cast<const uint16_t*>(a.W1) + (size_t)(first - a.nb1) * a.ldw;
      else base = static_cast<const uint16_t*>(a.W2) + (size_t)(first - a.nb2) * a.ldw;
      base -= (size_t)n0 * a.ldw;   // re-added below for every epilogue
    } else {
      base = static_cast<const uint16_t*>(a.W0);
      row = r;
      nrows = ncnt;
    }
    rsB[i] = make_rsrc(base + (size_t)n0 * a.ldw, (uint32_t)nrows * a.ldw * 2u);
    voB[i] = (uint32_t)row * a.ldw * 2u + lc * 16u;
  }

  uint4 ra0[4], rb0[WLD], ra1[4], rb1[WLD];
  auto gload = [&](int c, uint4 (&ra)[4], uint4 (&rb)[WLD]) {
    const uint32_t so = (uint32_t)__builtin_amdgcn_readfirstlane(s_k0[c]) * 2u;
#pragma unroll
    for (int i = 0; i < 4; ++i) ra[i] = load16(rsA, voA[i], so);
#pragma unroll
    for (int i = 0; i < WLD; ++i) rb[i] = load16(rsB[i], voB[i], so);
  };
  auto lstore = [&](int buf, const uint4 (&ra)[4], const uint4 (&rb)[WLD]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<uint4*>(&As[buf][(lr + 32 * i) * LDS_STRIDE + lc * 8]) = ra[i];
#pragma unroll
    for (int i = 0; i < WLD; ++i)
      *reinterpret_cast<uint4*>(&Bs[buf][(lr + 32 * i) * LDS_STRIDE + lc * 8]) = weight_to_act<F16>(rb[i]);
  };

  floatx4 acc[2][NB];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int buf) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int koff = ks * 32 + (lane >> 4) * 8;
      uint4 af[2], bfr[NB];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[i] = *reinterpret_cast<const uint4*>(
            &As[buf][(wave * 32 + i * 16 + (lane & 15)) * LDS_STRIDE + koff]);
#pragma unroll
      for (int j = 0; j < NB; ++j)
        bfr[j] = *reinterpret_cast<const uint4*>(&Bs[buf][(j * 16 + (lane & 15)) * LDS_STRIDE + koff]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) acc[i][j] = mfma16x16x32<F16>(af[i], bfr[j], acc[i][j]);
    }
  };

  // Pipeline: chunk c lives in LDS buffer c & 1; chunks c+1 and c+2 are in
  // flight in the register stages.  The body is unrolled by two so the
  // register stages keep fixed roles; past the last chunk the loads repeat
  // the last chunk (cache hits, never used).
  if (nk > 0) {
    const int last = nk - 1;
    gload(0, ra0, rb0);
    gload(min(1, last), ra1, rb1);
    lstore(0, ra0, rb0);
    __syncthreads();
    for (int c = 0; c < nk; c += 2) {
      gload(min(c + 2, last), ra0, rb0);
      compute(0);
      lstore(1, ra1, rb1);
      __syncthreads();
      if (c + 1 >= nk) break;
      gload(min(c + 3, last), ra1, rb1);
      compute(1);
      lstore(0, ra0, rb0);
      __syncthreads();
    }
  }

  // Epilogue.  acc[i][j][r] is C[wave*32 + i*16 + 4*(lane/16) + r][j*16 + lane%16].
  const int rbase = wave * 32 + (lane >> 4) * 4;
  if constexpr (EPI == EPI_QKV) {
    static_assert(BN == 64, "QKV tiles are 64 weight rows");
    uint16_t* out = static_cast<uint16_t*>(a.out);
    const bool rot = n0 < a.rope_cols;
    const int half = a.head_dim >> 1;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rbase + i * 16 + r;
        const int rowc = min(row, mcnt - 1);
        const int pos = (mrow0 - g.row0) + rowc;
        uint16_t* orow = out + (size_t)(mrow0 + rowc) * a.ldo;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          // dims of this lane: dim (blocks 0, 1) and dim + d/2 (blocks 2, 3)
          const int dim = quarter * 32 + j * 16 + (lane & 15);
          const int c1 = hbase + dim;
          const int c2 = c1 + half;
          float v1 = acc[i][j][r], v2 = acc[i][j + 2][r];
          if (rot) {
            const float2 cs = a.rope[(size_t)pos * half + dim];
            const float o1 = v1 * cs.x - v2 * cs.y;
            const float o2 = v2 * cs.x + v1 * cs.y;
            v1 = o1;
            v2 = o2;
          }
          if (row < mcnt) {   // QKV tiles are always full (ranges are whole heads)
            orow[c1] = f32_to_act_bits<F16>(v1);
            orow[c2] = f32_to_act_bits<F16>(v2);
          }
        }
      }
  } else if constexpr (EPI == EPI_RESID) {
    float* out = static_cast<float*>(a.out);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rbase + i * 16 + r;
        float* orow = out + (size_t)(mrow0 + min(row, mcnt - 1)) * a.ldo + n0;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const int col = j * 16 + (lane & 15);
          if (row < mcnt && col < ncnt) orow[col] += acc[i][j][r];
        }
      }
  } else {
    uint16_t* out = static_cast<uint16_t*>(a.out);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rbase + i * 16 + r;
        uint16_t* orow = out + (size_t)(mrow0 + min(row, mcnt - 1)) * a.ldo + n0;
#pragma unroll
        for (int j = 0; j < NB / 2; ++j) {
          const int ch = j * 16 + (lane & 15);
          const float gt = acc[i][j][r], up = acc[i][j + NB / 2][r];
          if (row < mcnt && ch < ncnt)
            orow[ch] = f32_to_act_bits<F16>(gt / (1.0f + __expf(-gt)) * up);
        }
      }
  }
}

template <int EPI, int BN, bool F16>
hipError_t launch(const GemmArgs& a, hipStream_t st) {
  const unsigned grid = (unsigned)((a.ntiles + 7) / 8 * 8);
  gemm_mfma_kernel<EPI, BN, F16><<<grid, NT, 0, st>>>(a);
  return hipGetLastError();
}

template <bool F16>
hipError_t dispatch(const GemmArgs& a, int32_t epi, int32_t bn, hipStream_t st) {
  switch (epi) {
    case EPI_QKV:
      if (bn == 64) return launch<EPI_QKV, 64, F16>(a, st);
      break;
    case EPI_RESID:
      if (bn == 32) return launch<EPI_RESID, 32, F16>(a, st);
      if (bn == 64) return launch<EPI_RESID, 64, F16>(a, st);
      if (bn == 128) return launch<EPI_RESID, 128, F16>(a, st);
      break;
    case EPI_SWIGLU:
      if (bn == 64) return launch<EPI_SWIGLU, 64, F16>(a, st);
      if (bn == 128) return launch<EPI_SWIGLU, 128, F16>(a, st);
      break;
    default:
      break;
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gemm_mfma(const GemmArgs& a, int32_t epi, int32_t bn, bool f16, hipStream_t st) {
  if (a.ntiles <= 0) return hipSuccess;
  return f16 ? dispatch<true>(a, epi, bn, st) : dispatch<false>(a, epi, bn, st);
}

}  // namespace svl
