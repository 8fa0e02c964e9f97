// Row-vector products of the decode step.
//
// In a decode step every GEMM group holds one row: the new token of one
// sample.  Such a launch is a list of 16-column weight blocks (the same
// blocks the MFMA tiles are cut into: QKV blocks pair 8 dims of a head with
// their rotary partners, gate/up blocks pair 8 gate channels with the same 8
// up channels), and its time is the time to stream the blocks' weight rows.
// Four workgroups per block, 4 waves each: a wave computes one column of the
// block, the dot product of one weight row with the sample's activation row
// over the group's K chunks; a workgroup holds two columns and their pair
// partners.  Activation rows are row-major in decode (the norm,
// the decode attention and this kernel's SwiGLU output write them so): a
// row of the fragment-packed layout would be spread over eight cache lines
// per 64 columns.  Lane l takes 8 consecutive columns of chunk
// 8 s + l / 8 in step s; four steps are loaded before they are used, so a
// wave keeps 4 KiB of its weight row in flight.  The lane sums are reduced
// in a fixed order and a workgroup's 4 results meet in LDS for the paired
// epilogues: RoPE on query / key columns, silu(gate) * up, or the residual
// add of the output and down projections (one writer per element).
#include "svl_internal.h"
#include "device_util.h"

namespace svl {
namespace {

constexpr int GV_WAVES = 4, GV_NT = GV_WAVES * 64, GV_U = 4;

// Workgroup x takes quarter q = x % 4 of block x / 4: columns 2q, 2q + 1 and
// their partners 2q + 8, 2q + 9 (wave w: column (w & 1) + 2q + 8 (w >> 1)).
constexpr int GV_MAX_CHUNKS = 1024;   // K chunks of a group (K <= 65536)

template <int EPI, bool F16>
__global__ __launch_bounds__(GV_NT) void gemv_kernel(MmArgs a) {
  __shared__ float s_v[GV_WAVES];
  __shared__ int32_t s_k0[GV_MAX_CHUNKS];   // a chunk-list group's offsets (no dependent loads)
  const int blk = blockIdx.x >> 2, quarter = blockIdx.x & 3;
  int lo = 0, hi = a.ngroups - 1;   // the group whose first block (pad0) is the largest <= blk
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.groups[mid].pad0 <= blk) lo = mid; else hi = mid - 1;
  }
  const MmGroup g = a.groups[lo];
  const int gb = blk - g.pad0;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ci = (wave & 1) + 2 * quarter + ((wave >> 1) ? 8 : 0);
  const int d = a.head_dim, hb = d >> 4, half = d >> 1;
  int m, row;
  if constexpr (EPI == EPI_QKV) {
    m = g.wsel;
    row = g.wrow0 + (gb / hb) * d + (gb % hb) * 8 + (ci & 7) + ((ci >> 3) ? half : 0);
  } else if constexpr (EPI == EPI_SWIGLU) {
    m = ci >> 3;   // gate rows, then up rows
    row = g.wrow0 + gb * 8 + (ci & 7);
  } else {
    m = 0;
    row = g.wrow0 + gb * 16 + ci;
  }
  const uint16_t* wr =
      static_cast<const uint16_t*>(m == 0 ? a.W[0] : (m == 1 ? a.W[1] : a.W[2])) + (size_t)row * a.ldw;
  const uint16_t* xr = static_cast<const uint16_t*>(a.A) + (size_t)g.arow0 * a.lda;
  const int nc = g.kc_cnt, cl = lane >> 3, off = (lane & 7) * 8;
  const bool dense = g.kdense >= 0;   // uniform across the workgroup
  if (!dense) {
    // chunk-list groups (output / down projections under head or FFN gates)
    // cover whole 64-column chunks: runs of heads (d in {64, 128}) and FFN
    // slices (a multiple of 64)
    for (int c = threadIdx.x; c < nc; c += GV_NT) s_k0[c] = a.chunks[g.kc_off + c].k0;
    __syncthreads();
  }
  float acc = 0.f;
  for (int s0 = 0; s0 < nc; s0 += 8 * GV_U) {
    uint4 wv[GV_U], xv[GV_U];
#pragma unroll
    for (int u = 0; u < GV_U; ++u) {
      const int c = s0 + 8 * u + cl;
      if (c < nc) {
        const int k = (dense ? g.kdense + MFMA_BK * c : s_k0[c]) + off;
        wv[u] = *reinterpret_cast<const uint4*>(wr + k);
        xv[u] = *reinterpret_cast<const uint4*>(xr + k);
      } else {
        wv[u] = make_uint4(0, 0, 0, 0);
        xv[u] = make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int u = 0; u < GV_U; ++u) {
      const uint32_t w4[4] = {wv[u].x, wv[u].y, wv[u].z, wv[u].w};
      const uint32_t x4[4] = {xv[u].x, xv[u].y, xv[u].z, xv[u].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc += bf16_bits_to_f32(w4[e] & 0xffffu) * act_bits_to_f32<F16>(x4[e] & 0xffffu);
        acc += bf16_bits_to_f32(w4[e] >> 16) * act_bits_to_f32<F16>(x4[e] >> 16);
      }
    }
  }
  acc = warp_sum(acc);
  if (lane == 0) s_v[wave] = acc;
  __syncthreads();
  if (lane != 0) return;
  float v = s_v[wave];
  if constexpr (EPI == EPI_QKV) {
    const int dim = (gb % hb) * 8 + (ci & 7);
    const int col = g.ocol0 + (gb / hb) * d + dim + ((ci >> 3) ? half : 0);
    if (g.rope) {
      // (x1, x2) -> (x1 cos - x2 sin, x2 cos + x1 sin); columns ci < 8 hold x1
      const float pv = s_v[wave ^ 2];
      const float2 cs = a.rope[(size_t)g.pos_base * half + dim];
      v = v * cs.x + ((ci < 8) ? -pv : pv) * cs.y;
    }
    static_cast<uint16_t*>(a.out)[(size_t)g.orow0 * a.ldo + col] = f32_to_act_bits<F16>(v);
  } else if constexpr (EPI == EPI_SWIGLU) {
    if (ci < 8) {
      const float up = s_v[wave + 2];
      const float h = v * __builtin_amdgcn_rcpf(1.0f + __expf(-v)) * up;
      static_cast<uint16_t*>(a.out)[(size_t)g.orow0 * a.ldo + g.ocol0 + gb * 8 + ci] =
          f32_to_act_bits<F16>(h);
    }
  } else {
    float* o = static_cast<float*>(a.out) + (size_t)g.orow0 * a.ldo + g.ocol0 + gb * 16 + ci;
    *o += v;
  }
}

// Shared row-vector products (decode of a batch) on MFMA.  One workgroup
// of 4 waves per 16-column block of a segment computes C[column][use] =
// sum_k W[column][k] x_use[k] for the segment's uses (at most 16; a segment
// holds at most DEC_MAX_USES) as one 16 x 16 x 32 MFMA per 32 k: the
// block's 16 weight rows are the A operand (lane l: row l % 16, k 8 (l / 16)
// .. +8, loaded straight from the weight matrix), the uses' activation rows
// the B operand (lane l: use l % 16, the same k), so each weight block is
// streamed once for every sample whose masks include it.  Uses past the
// segment's count, and a use's chunks outside its active heads or FFN slices
// (output / down projections: the chunk's use mask), enter as exact zeros
// (a select: the unwritten activation columns of inactive heads never reach
// the sum).  With fp16 activations the bf16 weights are widened to fp16
// (exact inside fp16's range), as in the prefill GEMMs.  Wave w takes a
// contiguous quarter of the segment's K chunks with four chunks in flight;
// the four partial sums meet in LDS and are added in wave order, then lane
// l holds rows 4 (l / 16) + r of use l % 16, and a column's pair partner
// (column ^ 8) sits in lane l ^ 32.
constexpr int GM_NT = 256, GM_CF = 4;

template <bool F16>
__device__ __forceinline__ uint4 weight_to_act_dec(const uint4& v) {
  if constexpr (F16) {
    return make_uint4(bf16x2_to_f16x2(v.x), bf16x2_to_f16x2(v.y), bf16x2_to_f16x2(v.z),
                      bf16x2_to_f16x2(v.w));
  } else {
    return v;
  }
}

template <int EPI, bool F16>
__global__ __launch_bounds__(GM_NT) void gemv_mfma_shared_kernel(MmArgs a) {
  __shared__ floatx4 s_acc[3][64];
  __shared__ int32_t s_k0[GV_MAX_CHUNKS];
  __shared__ int32_t s_m[GV_MAX_CHUNKS];
  const int blk = blockIdx.x;
  int lo = 0, hi = a.nsegs - 1;   // the segment whose first block is the largest <= blk
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.segs[mid].blk0 <= blk) lo = mid; else hi = mid - 1;
  }
  const DecSeg g = a.segs[lo];
  const int gb = blk - g.blk0;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int d = a.head_dim, hb = d >> 4, half = d >> 1;
  // A operand row of this lane: block column ci = lane % 16
  const int ci = lane & 15, kq = (lane >> 4) * 8;
  int m, row;
  if constexpr (EPI == EPI_QKV) {
    m = g.wsel;
    row = g.wrow0 + (gb / hb) * d + (gb % hb) * 8 + (ci & 7) + ((ci >> 3) ? half : 0);
  } else if constexpr (EPI == EPI_SWIGLU) {
    m = ci >> 3;   // gate rows, then up rows
    row = g.wrow0 + gb * 8 + (ci & 7);
  } else {
    m = 0;
    row = g.wrow0 + gb * 16 + ci;
  }
  const uint16_t* wr =
      static_cast<const uint16_t*>(m == 0 ? a.W[0] : (m == 1 ? a.W[1] : a.W[2])) + (size_t)row * a.ldw + kq;
  // B operand row of this lane: use ci (past the count: use 0's row, zeroed)
  const int nu = g.nuse;
  const bool uon = ci < nu;
  const uint16_t* xr = static_cast<const uint16_t*>(a.A) +
                       (size_t)a.uses[g.use_off + (uon ? ci : 0)].arow * a.lda + kq;
  const int nc = g.kc_cnt;
  const bool dense = g.kdense >= 0, masked = g.mask_off >= 0;   // uniform
  for (int c = threadIdx.x; c < nc; c += GM_NT) {
    s_k0[c] = dense ? g.kdense + MFMA_BK * c : a.chunks[g.kc_off + c].k0;
    s_m[c] = masked ? a.cmasks[g.mask_off + c] : -1;
  }
  __syncthreads();
  const int c0 = nc * wave / 4, c1 = nc * (wave + 1) / 4;
  floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int cb = c0; cb < c1; cb += GM_CF) {
    uint4 wv[GM_CF][2], xv[GM_CF][2];
    bool on[GM_CF];
#pragma unroll
    for (int t = 0; t < GM_CF; ++t) {
      const int c = min(cb + t, c1 - 1);   // past the range: the last chunk again, not added
      const int k = s_k0[c];
      on[t] = cb + t < c1 && uon && ((s_m[c] >> ci) & 1);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        wv[t][h] = *reinterpret_cast<const uint4*>(wr + k + 32 * h);
        xv[t][h] = *reinterpret_cast<const uint4*>(xr + k + 32 * h);
      }
    }
#pragma unroll
    for (int t = 0; t < GM_CF; ++t)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint4 z = make_uint4(0, 0, 0, 0);
        // a chunk past the range multiplies zero weights as well (no NaN
        // from a repeated chunk can enter)
        const uint4 wa = cb + t < c1 ? weight_to_act_dec<F16>(wv[t][h]) : z;
        acc = mfma16x16x32<F16>(wa, on[t] ? xv[t][h] : z, acc);
      }
  }
  if (wave > 0) s_acc[wave - 1][lane] = acc;
  __syncthreads();
  if (wave > 0) return;
#pragma unroll
  for (int w = 0; w < 3; ++w) {
    const floatx4 v = s_acc[w][lane];
    acc = floatx4{acc[0] + v[0], acc[1] + v[1], acc[2] + v[2], acc[3] + v[3]};
  }
  // lane holds C[column 4 (lane / 16) + r][use lane % 16]
  const int u = lane & 15;
  const bool store = u < nu;
  const DecUse us = a.uses[g.use_off + (store ? u : 0)];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int col_i = 4 * (lane >> 4) + r;   // block column
    float v = acc[r];
    const float pv = __shfl_xor(v, 32, 64);   // column col_i ^ 8
    if constexpr (EPI == EPI_QKV) {
      const int dim = (gb % hb) * 8 + (col_i & 7);
      const int col = g.ocol0 + (gb / hb) * d + dim + ((col_i >> 3) ? half : 0);
      if (g.rope) {
        const float2 cs = a.rope[(size_t)us.pos * half + dim];
        v = v * cs.x + ((col_i < 8) ? -pv : pv) * cs.y;
      }
      if (store) static_cast<uint16_t*>(a.out)[(size_t)us.orow * a.ldo + col] = f32_to_act_bits<F16>(v);
    } else if constexpr (EPI == EPI_SWIGLU) {
      if (store && col_i < 8) {
        const float h = v * __builtin_amdgcn_rcpf(1.0f + __expf(-v)) * pv;
        static_cast<uint16_t*>(a.out)[(size_t)us.orow * a.ldo + g.ocol0 + gb * 8 + col_i] =
            f32_to_act_bits<F16>(h);
      }
    } else {
      if (store) static_cast<float*>(a.out)[(size_t)us.orow * a.ldo + g.ocol0 + gb * 16 + col_i] += v;
    }
  }
}

template <bool F16>
hipError_t launch_shared(const MmArgs& a, int32_t epi, hipStream_t st) {
  switch (epi) {
    case EPI_QKV: gemv_mfma_shared_kernel<EPI_QKV, F16><<<a.nblocks, GM_NT, 0, st>>>(a); break;
    case EPI_SWIGLU: gemv_mfma_shared_kernel<EPI_SWIGLU, F16><<<a.nblocks, GM_NT, 0, st>>>(a); break;
    case EPI_RESID: gemv_mfma_shared_kernel<EPI_RESID, F16><<<a.nblocks, GM_NT, 0, st>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <bool F16>
hipError_t launch(const MmArgs& a, int32_t epi, hipStream_t st) {
  const unsigned grid = (unsigned)a.nblocks * 4;
  switch (epi) {
    case EPI_QKV: gemv_kernel<EPI_QKV, F16><<<grid, GV_NT, 0, st>>>(a); break;
    case EPI_SWIGLU: gemv_kernel<EPI_SWIGLU, F16><<<grid, GV_NT, 0, st>>>(a); break;
    case EPI_RESID: gemv_kernel<EPI_RESID, F16><<<grid, GV_NT, 0, st>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemv_shared(const MmArgs& a, int32_t epi, bool f16, hipStream_t st) {
  if (a.nblocks <= 0 || a.nsegs <= 0) return hipSuccess;
  if (a.lda / MFMA_BK > GV_MAX_CHUNKS || a.max_uses < 1 || a.max_uses > DEC_MAX_USES)
    return hipErrorInvalidValue;
  return f16 ? launch_shared<true>(a, epi, st) : launch_shared<false>(a, epi, st);
}

hipError_t launch_gemv(const MmArgs& a, int32_t epi, bool f16, hipStream_t st) {
  if (a.nblocks <= 0 || a.ngroups <= 0) return hipSuccess;
  if (a.lda / MFMA_BK > GV_MAX_CHUNKS) return hipErrorInvalidValue;
  return f16 ? launch<true>(a, epi, st) : launch<false>(a, epi, st);
}

}  // namespace svl
