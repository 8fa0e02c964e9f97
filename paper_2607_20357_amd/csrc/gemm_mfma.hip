// Masked grouped GEMM on 16-bit MFMA (gfx950 v_mfma_f32_16x16x32_{f16,bf16}).
//
//   C[rows, cols] = sum over the group's K chunks of A[rows, k] * W[cols, k]
//
// A is an activation matrix in the fragment-packed layout (see plan_types.h:
// 16-row x 64-column blocks of 2 KB, fp16 or bf16); W a bf16 weight matrix
// in [out][in] layout.  With fp16 activations each weight tile is widened
// bf16 -> fp16 on its way into LDS (exact inside fp16's range), so both
// operands of the fp16 MFMA carry 11-bit significands; with bf16 activations
// the weights go through unchanged.  Accumulation is float32.
//
// A launch is a list of groups (one sample and one active column range each,
// or one sample and its active K chunks), so weight rows of inactive heads /
// FFN slices (QKV, gate/up) and weight columns of inactive heads / slices
// (output and down projections) are never read.
//
// Tile: 256 rows x BN weight rows, 512 threads = 8 waves, wave w owning rows
// 32w .. 32w+31 (two 16-row MFMA blocks) and all BN columns.  K advances in
// chunks of 64.  Per chunk:
//   * each wave loads its own A fragments straight from the packed layout
//     into registers (two 1 KB contiguous loads per 16-row block: every
//     cache line fully used, no LDS traffic for A);
//   * the BN weight rows are loaded cooperatively (16 bytes per thread and
//     row segment) and staged through LDS, where all eight waves read them;
// and NS = 3 chunks are in flight (register stages, one LDS buffer per
// stage); at most 128 VGPRs, so two workgroups share a CU.  A sample of up to 256 rows is one M tile, so each weight tile is
// streamed from HBM once.  Buffer loads: one resource per operand spans the
// tile's valid rows, so rows past the tile read as zero.
//
// Split-K (skinny output and down projections): a group may be cut into
// nsplit K ranges; piece p stores its float32 tile into partial slice p.  The
// next residual-finish kernel adds the slices in order, so no atomics or
// cross-workgroup synchronisation are needed and the sum order is fixed.
//
// Epilogues:
//   QKV: store row-major; query and key columns are first rotated by RoPE at
//     the row's position inside its sample (the float32 accumulators are
//     rotated, so Q and K are rounded once).  A tile holds BN/2 dims of the
//     first half of a head and the same dims of the second half, so one lane
//     holds both members (r, r + d/2) of each rotation pair;
//   RESID: add into the float32 residual;
//   PARTIAL: store the float32 split-K piece;
//   SWIGLU: the tile's weight rows are BN/2 gate rows followed by the BN/2
//     matching up rows, so one lane holds the gate and the up value of a
//     channel; silu(gate) * up is stored fragment-packed for the down GEMM.
#include <type_traits>

#include "svl_internal.h"
#include "device_util.h"

namespace svl {
namespace {

constexpr int BM = MFMA_BM, NWAVE = 8, NT = NWAVE * 64;
constexpr int LDS_STRIDE = MFMA_BK + 8;   // 16-bit elements per LDS row (144 B)
constexpr int MAX_CHUNKS = 1024;          // K chunks per group (K <= 65536)
constexpr int NS = 3;                     // chunks in flight

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
  constexpr int WLD = (BN * 8 + NT - 1) / NT;             // 16-byte W loads per thread
  constexpr int WROWS = NT / 8;                           // W rows one load round covers
  __shared__ __attribute__((aligned(16))) uint16_t Bs[NS][BN * LDS_STRIDE];
  __shared__ int32_t s_k0[MAX_CHUNKS];   // the piece's chunk offsets (LDS, no vmcnt waits)

  const int t = xcd_tile_index();
  if (t >= a.ntiles) return;
  const GemmGroup g = a.groups[find_group(a.groups, a.ngroups, t)];
  const int local = t - g.tile0;
  const int split = local % g.nsplit, rest = local / g.nsplit;
  const int nm = (g.nrows + BM - 1) / BM;
  const int mt = rest % nm, nt = rest / nm;
  const int mcnt = min(BM, g.nrows - mt * BM);
  const int n0 = g.n0 + nt * BNO;
  const int ncnt = min(BNO, g.n1 - n0);
  const int kb = g.kc_off + (g.kc_cnt * split) / g.nsplit;
  const int nk = g.kc_off + (g.kc_cnt * (split + 1)) / g.nsplit - kb;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int c = tid; c < nk; c += NT) s_k0[c] = a.chunks[kb + c].k0;

  // QKV: first dim (of the head's first half) this tile holds
  int hbase = n0, c0 = 0;
  if constexpr (EPI == EPI_QKV) {
    hbase = n0 - (n0 % a.head_dim);
    c0 = ((n0 - hbase) / BN) * (BN / 2);
  }

  // A: packed blocks of this tile's rows; wave w reads blocks 2w and 2w+1.
  const uint32_t kblocks = (uint32_t)(a.lda / 64);
  const uint32_t blk_bytes = kblocks * 2048u;   // one 16-row block over all of K
  const int rb0 = (g.arow0 + mt * BM) / 16;
  const __amdgpu_buffer_rsrc_t rsA =
      make_rsrc(static_cast<const uint16_t*>(a.A) + (size_t)rb0 * kblocks * 1024,
                (uint32_t)((mcnt + 15) / 16) * blk_bytes);
  uint32_t voA[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) voA[i] = (uint32_t)(2 * wave + i) * blk_bytes + lane * 16u;

  // W: tile rows lr + WROWS i, 16-byte segment lc of the chunk's 128 bytes.
  const int lc = tid & 7, lr = tid >> 3;
  __amdgpu_buffer_rsrc_t rsB[WLD];
  uint32_t voB[WLD];
#pragma unroll
  for (int i = 0; i < WLD; ++i) {
    const int r = lr + WROWS * i;     // tile row (weight row of the tile)
    const uint16_t* base;
    int nrows, row;
    if constexpr (EPI == EPI_SWIGLU) {
      // rows [0, BN/2) are gate channels n0.., rows [BN/2, BN) the same up
      // channels; the choice is uniform across a wave
      const int up = __builtin_amdgcn_readfirstlane(r >= BN / 2 ? 1 : 0);
      base = static_cast<const uint16_t*>(up ? a.W1 : a.W0) + (size_t)n0 * a.ldw;
      row = up ? r - BN / 2 : r;
      nrows = ncnt;
    } else if constexpr (EPI == EPI_QKV) {
      const int half = a.head_dim / 2;
      row = (r < BN / 2) ? c0 + r : half + c0 + (r - BN / 2);
      nrows = a.head_dim;
      if (hbase < a.nb1) base = static_cast<const uint16_t*>(a.W0) + (size_t)hbase * a.ldw;
      else if (hbase < a.nb2) base = static_cast<const uint16_t*>(a.W1) + (size_t)(hbase - a.nb1) * a.ldw;
      else base = static_cast<const uint16_t*>(a.W2) + (size_t)(hbase - a.nb2) * a.ldw;
    } else {
      base = static_cast<const uint16_t*>(a.W0) + (size_t)n0 * a.ldw;
      row = r;
      nrows = ncnt;
    }
    rsB[i] = make_rsrc(base, (uint32_t)nrows * a.ldw * 2u);
    // threads past the tile's rows read out of range (zero, no traffic)
    voB[i] = (r < BN) ? (uint32_t)row * a.ldw * 2u + lc * 16u : 0xfffffff0u;
  }
  __syncthreads();   // s_k0 ready

  // Register stages: stage s holds the A fragments and the W rows of chunk
  // c = s (mod NS).
  uint4 sa[NS][2][2], sb[NS][WLD];
  auto gload = [&](int c, uint4 (&ra)[2][2], uint4 (&rb)[WLD]) {
    const uint32_t k0 = (uint32_t)__builtin_amdgcn_readfirstlane(s_k0[c]);
    const uint32_t soA = k0 * 32u, soB = k0 * 2u;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      ra[i][0] = load16(rsA, voA[i], soA);
      ra[i][1] = load16(rsA, voA[i] + 1024u, soA);
    }
#pragma unroll
    for (int i = 0; i < WLD; ++i) rb[i] = load16(rsB[i], voB[i], soB);
  };
  auto wstore = [&](int buf, const uint4 (&rb)[WLD]) {
#pragma unroll
    for (int i = 0; i < WLD; ++i) {
      const int r = lr + WROWS * i;
      if (BN * 8 >= NT * (i + 1) || r < BN)
        *reinterpret_cast<uint4*>(&Bs[buf][r * LDS_STRIDE + lc * 8]) = weight_to_act<F16>(rb[i]);
    }
  };

  floatx4 acc[2][NB];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Inside a chunk, lane group q = lane / 16 holds k 16q + [0, 8) in the
  // first MFMA k-step and 16q + [8, 16) in the second, for both operands.
  auto compute = [&](int buf, const uint4 (&ra)[2][2]) {
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      uint4 bfr[NB];
#pragma unroll
      for (int j = 0; j < NB; ++j)
        bfr[j] = *reinterpret_cast<const uint4*>(
            &Bs[buf][(j * 16 + (lane & 15)) * LDS_STRIDE + (lane >> 4) * 16 + ks * 8]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) acc[i][j] = mfma16x16x32<F16>(ra[i][ks], bfr[j], acc[i][j]);
    }
  };

  // Pipeline: chunk c is multiplied from registers (A) and LDS buffer c % NS
  // (W) while chunks c+1 .. c+NS-1 are in flight; the W rows of chunk c+1 go
  // to LDS right after, and the freed stage is refilled with chunk c+NS.
  // Past the last chunk the loads repeat the last chunk (cache hits, unused).
  if (nk > 0) {
    const int last = nk - 1;
#pragma unroll
    for (int s = 0; s < NS; ++s) gload(min(s, last), sa[s], sb[s]);
    wstore(0, sb[0]);
    __syncthreads();
    auto step = [&](int cc, auto sc) {
      constexpr int s = decltype(sc)::value;
      compute(s, sa[s]);
      wstore((s + 1) % NS, sb[(s + 1) % NS]);
      __syncthreads();
      gload(min(cc + NS, last), sa[s], sb[s]);
    };
    // Whole groups of NS chunks: one exit, so the compiler waits on exactly
    // the oldest stage; then the remaining chunks.
    int c = 0;
    static_assert(NS == 3, "the step sequence below is written for three stages");
    for (; c + NS <= nk; c += NS) {
      step(c + 0, std::integral_constant<int, 0>{});
      step(c + 1, std::integral_constant<int, 1>{});
      step(c + 2, std::integral_constant<int, 2>{});
    }
    if (c + 0 < nk) step(c + 0, std::integral_constant<int, 0>{});
    if (c + 1 < nk) step(c + 1, std::integral_constant<int, 1>{});
  }

  // Epilogue.  acc[i][j][r] is C[wave*32 + i*16 + 4*(lane/16) + r][j*16 + lane%16]
  // of the tile; tile row m is row mt*BM + m of the group.
  const int rbase = wave * 32 + (lane >> 4) * 4;
  const int l16 = lane & 15;
  if constexpr (EPI == EPI_QKV) {
    uint16_t* out = static_cast<uint16_t*>(a.out);
    const bool rot = hbase < a.rope_cols;
    const int half = a.head_dim >> 1;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rbase + i * 16 + r;
        const int rowc = min(row, mcnt - 1);
        const int pos = mt * BM + rowc;
        uint16_t* orow = out + (size_t)(g.orow0 + pos) * a.ldo + hbase;
#pragma unroll
        for (int j = 0; j < NB / 2; ++j) {
          // this lane's dims: dim (block j) and dim + d/2 (block j + NB/2)
          const int dim = c0 + j * 16 + l16;
          float v1 = acc[i][j][r], v2 = acc[i][j + NB / 2][r];
          if (rot) {
            const float2 cs = a.rope[(size_t)pos * half + dim];
            const float o1 = v1 * cs.x - v2 * cs.y;
            const float o2 = v2 * cs.x + v1 * cs.y;
            v1 = o1;
            v2 = o2;
          }
          if (row < mcnt) {   // QKV tiles are always full (ranges are whole heads)
            orow[dim] = f32_to_act_bits<F16>(v1);
            orow[dim + half] = f32_to_act_bits<F16>(v2);
          }
        }
      }
  } else if constexpr (EPI == EPI_RESID || EPI == EPI_PARTIAL) {
    float* out = static_cast<float*>(EPI == EPI_PARTIAL ? a.partial + split * a.pslice : a.out);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rbase + i * 16 + r;
        float* orow = out + (size_t)(g.orow0 + mt * BM + min(row, mcnt - 1)) * a.ldo + n0;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const int col = j * 16 + l16;
          if (row < mcnt && col < ncnt) {
            if constexpr (EPI == EPI_RESID) orow[col] += acc[i][j][r];
            else orow[col] = acc[i][j][r];
          }
        }
      }
  } else {
    uint16_t* out = static_cast<uint16_t*>(a.out);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rbase + i * 16 + r;
        const int64_t prow = g.orow0 + mt * BM + min(row, mcnt - 1);
#pragma unroll
        for (int j = 0; j < NB / 2; ++j) {
          const int ch = j * 16 + l16;
          const float gt = acc[i][j][r], up = acc[i][j + NB / 2][r];
          if (row < mcnt && ch < ncnt)
            out[packed_index(prow, n0 + ch, a.ldo)] = f32_to_act_bits<F16>(gt / (1.0f + __expf(-gt)) * up);
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
      if (bn == 32) return launch<EPI_QKV, 32, F16>(a, st);
      if (bn == 64) return launch<EPI_QKV, 64, F16>(a, st);
      if (bn == 128) return launch<EPI_QKV, 128, F16>(a, st);
      break;
    case EPI_RESID:
      if (bn == 64) return launch<EPI_RESID, 64, F16>(a, st);
      break;
    case EPI_PARTIAL:
      if (bn == 64) return launch<EPI_PARTIAL, 64, F16>(a, st);
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
