// Float32 kernels of the masked GEMM and of the causal attention (the
// SVL_F32 path: small decoders checked at float32 accuracy).  Same plan
// descriptors and semantics as the bf16 MFMA kernels; plain FMA arithmetic.
//
// GEMM: 64 x 64 tiles, 256 threads with 4 x 4 outputs each, K walked in the
// group's chunks (any length) 16 columns at a time through LDS.
// Attention: one workgroup of 64 threads per (sample, active head, 64-row
// query tile), one query row per thread, 64-row K/V tiles in LDS, online
// softmax per 64-key block; RoPE applied to Q and K rows while loading.
#include "svl_internal.h"
#include "device_util.h"

namespace svl {
namespace {

constexpr int BM = F32_BM, BN = F32_BN, BK = F32_BK;

template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
  __shared__ float As[BK][BM + 4];
  __shared__ float Bs[BK][BN + 4];
  const int t = xcd_tile_index();
  if (t >= a.ntiles) return;
  const GemmGroup g = a.groups[find_group(a.groups, a.ngroups, t)];
  constexpr int BNO = (EPI == EPI_SWIGLU) ? F32_SWIGLU_CH : BN;
  const int local = t - g.tile0;
  const int nm = (g.nrows + BM - 1) / BM;
  const int mt = local % nm, nt = local / nm;
  const int arow0 = g.arow0 + mt * BM, orow0 = g.orow0 + mt * BM;
  const int mcnt = min(BM, g.nrows - mt * BM);
  const int n0 = g.n0 + nt * BNO;
  const int ncnt = min(BNO, g.n1 - n0);
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const float* A = static_cast<const float*>(a.A);

  // Weight row of tile column c (nullptr: outside the tile).
  auto wrow = [&](int c) -> const float* {
    if constexpr (EPI == EPI_SWIGLU) {
      const int ch = c & 31;
      if (ch >= ncnt) return nullptr;
      return static_cast<const float*>(c < 32 ? a.W0 : a.W1) + (size_t)(n0 + ch) * a.ldw;
    } else {
      if (c >= ncnt) return nullptr;
      const int col = n0 + c;
      if constexpr (EPI == EPI_STORE) {
        if (n0 < a.nb1) return static_cast<const float*>(a.W0) + (size_t)col * a.ldw;
        if (n0 < a.nb2) return static_cast<const float*>(a.W1) + (size_t)(col - a.nb1) * a.ldw;
        return static_cast<const float*>(a.W2) + (size_t)(col - a.nb2) * a.ldw;
      } else {
        return static_cast<const float*>(a.W0) + (size_t)col * a.ldw;
      }
    }
  };
  // Loader: element e of thread tid covers row (tid*4+e)/16, k (tid*4+e)%16.
  const int lrow = tid >> 2, lk = (tid & 3) * 4;
  const float* arow = lrow < mcnt ? A + (size_t)(arow0 + lrow) * a.lda : nullptr;
  const float* brow = wrow(lrow);
  // Output columns of this thread (tile columns).
  int cols[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
    cols[j] = (EPI == EPI_SWIGLU) ? ((j < 2) ? 2 * tx + j : 32 + 2 * tx + (j - 2)) : 4 * tx + j;

  float acc[4][4] = {};
  for (int kc = g.kc_off; kc < g.kc_off + g.kc_cnt; ++kc) {
    const KChunk ch = a.chunks[kc];
    for (int kk = 0; kk < ch.len; kk += BK) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int k = lk + e;
        const bool kin = kk + k < ch.len;
        As[k][lrow] = (arow && kin) ? arow[ch.k0 + kk + k] : 0.f;
        Bs[k][lrow] = (brow && kin) ? brow[ch.k0 + kk + k] : 0.f;
      }
      __syncthreads();
#pragma unroll
      for (int k = 0; k < BK; ++k) {
        float av[4], bv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) av[i] = As[k][ty * 4 + i];
#pragma unroll
        for (int j = 0; j < 4; ++j) bv[j] = Bs[k][cols[j]];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
      }
      __syncthreads();
    }
  }

#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = ty * 4 + i;
    if (row >= mcnt) continue;
    if constexpr (EPI == EPI_SWIGLU) {
      float* orow = static_cast<float*>(a.out) + (size_t)(orow0 + row) * a.ldo + n0;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int ch = cols[j];
        const float gt = acc[i][j], up = acc[i][j + 2];
        if (ch < ncnt) orow[ch] = gt / (1.0f + expf(-gt)) * up;
      }
    } else if constexpr (EPI == EPI_STORE) {
      float* orow = static_cast<float*>(a.out) + (size_t)(orow0 + row) * a.ldo + n0;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (cols[j] < ncnt) orow[cols[j]] = acc[i][j];
    } else {
      float* orow = static_cast<float*>(a.out) + (size_t)(orow0 + row) * a.ldo + n0;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (cols[j] < ncnt) orow[cols[j]] += acc[i][j];
    }
  }
}

template <int D>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a) {
  constexpr int BQ = ATTN_BQ, BKV = 64;
  __shared__ float Ks[BKV][D + 1];
  __shared__ float Vs[BKV][D + 1];
  const int t = blockIdx.x;
  if (t >= a.ntiles) return;
  const AttnGroup g = a.groups[find_group(a.groups, a.ngroups, t)];
  const int local = t - g.tile0;
  const int hs = local % g.h_cnt;
  const int qt = g.nqt - 1 - local / g.h_cnt;
  const int h = a.head_table[g.h_off + hs];
  const int kvh = h / (a.n_heads / a.n_kv_heads);
  const int S = g.S, q0 = qt * BQ, tid = threadIdx.x;
  const float* base = static_cast<const float*>(a.qkv) + (size_t)g.row0 * a.ldq;
  const int qcol = h * D, kcol = (a.n_heads + kvh) * D, vcol = (a.n_heads + a.n_kv_heads + kvh) * D;
  const int qi = q0 + tid;
  const bool qvalid = qi < S;
  constexpr int H = D / 2;

  float q[D], o[D];
  {
    const float* qp = base + (size_t)(qvalid ? qi : 0) * a.ldq + qcol;
    const float2* cs = a.rope + (size_t)(qvalid ? qi : 0) * H;
#pragma unroll
    for (int r = 0; r < H; ++r) {
      const float2 c = cs[r];
      const float x1 = qp[r], x2 = qp[r + H];
      q[r] = x1 * c.x - x2 * c.y;
      q[r + H] = x2 * c.x + x1 * c.y;
    }
#pragma unroll
    for (int d = 0; d < D; ++d) o[d] = 0.f;
  }
  float m_i = -1.0e30f, l_i = 0.f;
  const int kv_end = min(S, q0 + BQ);
  for (int kv0 = 0; kv0 < kv_end; kv0 += BKV) {
    __syncthreads();
    {
      const int kv = kv0 + tid;
      const bool ok = kv < S;
      const float* kp = base + (size_t)(ok ? kv : 0) * a.ldq + kcol;
      const float* vp = base + (size_t)(ok ? kv : 0) * a.ldq + vcol;
      const float2* cs = a.rope + (size_t)(ok ? kv : 0) * H;
      for (int r = 0; r < H; ++r) {
        const float2 c = cs[r];
        const float x1 = kp[r], x2 = kp[r + H];
        Ks[tid][r] = ok ? x1 * c.x - x2 * c.y : 0.f;
        Ks[tid][r + H] = ok ? x2 * c.x + x1 * c.y : 0.f;
      }
      for (int d = 0; d < D; ++d) Vs[tid][d] = ok ? vp[d] : 0.f;
    }
    __syncthreads();
    float s[BKV];
    float mt = -1.0e30f;
    for (int j = 0; j < BKV; ++j) {
      const int kv = kv0 + j;
      float dot = 0.f;
#pragma unroll
      for (int d = 0; d < D; ++d) dot = fmaf(q[d], Ks[j][d], dot);
      s[j] = (kv <= qi && kv < S) ? dot * a.scale : -1.0e30f;
      mt = fmaxf(mt, s[j]);
    }
    const float m_new = fmaxf(m_i, mt);
    const float alpha = expf(m_i - m_new);
    l_i *= alpha;
#pragma unroll
    for (int d = 0; d < D; ++d) o[d] *= alpha;
    for (int j = 0; j < BKV; ++j) {
      const int kv = kv0 + j;
      const float p = (kv <= qi && kv < S) ? expf(s[j] - m_new) : 0.f;
      l_i += p;
#pragma unroll
      for (int d = 0; d < D; ++d) o[d] = fmaf(p, Vs[j][d], o[d]);
    }
    m_i = m_new;
  }
  if (qvalid) {
    float* orow = static_cast<float*>(a.out) + (size_t)(g.row0 + qi) * a.ldo + h * D;
    const float inv = 1.0f / l_i;
#pragma unroll
    for (int d = 0; d < D; ++d) orow[d] = o[d] * inv;
  }
}

}  // namespace

hipError_t launch_gemm_f32(const GemmArgs& a, int32_t epi, hipStream_t st) {
  if (a.ntiles <= 0) return hipSuccess;
  const unsigned grid = (unsigned)((a.ntiles + 7) / 8 * 8);
  switch (epi) {
    case EPI_STORE: gemm_f32_kernel<EPI_STORE><<<grid, 256, 0, st>>>(a); break;
    case EPI_RESID: gemm_f32_kernel<EPI_RESID><<<grid, 256, 0, st>>>(a); break;
    default: gemm_f32_kernel<EPI_SWIGLU><<<grid, 256, 0, st>>>(a); break;
  }
  return hipGetLastError();
}

hipError_t launch_attn_f32(const AttnArgs& a, int32_t head_dim, hipStream_t st) {
  if (a.ntiles <= 0) return hipSuccess;
  switch (head_dim) {
    case 32: attn_f32_kernel<32><<<a.ntiles, 64, 0, st>>>(a); break;
    case 64: attn_f32_kernel<64><<<a.ntiles, 64, 0, st>>>(a); break;
    case 128: attn_f32_kernel<128><<<a.ntiles, 64, 0, st>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace svl
