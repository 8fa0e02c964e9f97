// Training-time masked decoder (Sec. 3.1 Eq. (6) with dropped tokens zeroed;
// Sec. 3.2 unit masks over head groups and FFN slices, or whole layers):
// float32 kernels for the static-shape forward and for its backward down to
// the token and gate logits.
//
// Rows: a batch of B samples of S = N + T rows each, row m = b S + i, RoPE
// position i.  Every head and FFN channel is computed; unit u of a layer
// scales the attention output of its heads and the SwiGLU output of its FFN
// slice (the matrix products read the scale with their A operand).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_util.h"
#include "train_internal.h"

namespace svl {
namespace {

constexpr int TNT = 256;

// ------------------------------------------------------------------ loads
template <class T>
__device__ __forceinline__ float4 ld4(const T* p, int64_t i);
template <>
__device__ __forceinline__ float4 ld4<float>(const float* p, int64_t i) {
  return *reinterpret_cast<const float4*>(p + i);
}
template <>
__device__ __forceinline__ float4 ld4<uint16_t>(const uint16_t* p, int64_t i) {
  const uint2 w = *reinterpret_cast<const uint2*>(p + i);
  return make_float4(__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u),
                     __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xffff0000u));
}

__device__ __forceinline__ float4 f4scale(float4 v, float s) {
  return make_float4(v.x * s, v.y * s, v.z * s, v.w * s);
}

// Sum over the 256 threads of a workgroup, the same order on every call.
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = warp_sum(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

// y (1 - y) / tau for y = sigma(v / tau), without cancellation on either side.
__device__ __forceinline__ float ste_factor(float v, float tau) {
  const float a = expf(-fabsf(v / tau));
  return a / ((1.0f + a) * (1.0f + a)) / tau;
}

// ------------------------------------------------------------------ masks
__global__ void train_masks_kernel(TrainMaskArgs a) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t nt = (int64_t)a.B * a.N;
  const int64_t per = (int64_t)(a.L - a.P) * a.U;
  const int64_t ng = (int64_t)a.B * per;
  const int64_t np = (int64_t)a.B * a.P * a.U;
  if (i < nt) {
    const float v = a.z[i] + (a.zn ? a.zn[i] : 0.0f);
    const bool on = v > 0.0f;
    a.tmask[i] = on ? 1 : 0;
    a.mtok[i] = on ? 1.0f : 0.0f;
    a.stet[i] = ste_factor(v, a.tau_tok);
    return;
  }
  i -= nt;
  if (i < ng) {
    const float v = a.g[i] + (a.gn ? a.gn[i] : 0.0f);
    const bool on = v > 0.0f;
    const int64_t b = i / per, r = i % per;
    a.umask[i] = on ? 1 : 0;
    a.mfull[b * a.L * a.U + (int64_t)a.P * a.U + r] = on ? 1.0f : 0.0f;
    a.steg[i] = ste_factor(v, a.tau_comp);
    return;
  }
  i -= ng;
  if (i < np) {
    const int64_t pp = (int64_t)a.P * a.U;
    a.mfull[(i / pp) * a.L * a.U + i % pp] = 1.0f;
  }
}

// X0 = [m_i v_i ; text] (Sec. 3.1, training: the sequence keeps its length).
template <class T>
__global__ void train_embed_kernel(const T* vision, const T* text, const float* mtok, int32_t B,
                                   int32_t N, int32_t Tn, int32_t D, float* X) {
  const int64_t D4 = D / 4, S = (int64_t)N + Tn;
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (int64_t)B * S * D4) return;
  const int64_t m = q / D4, c = (q % D4) * 4, b = m / S, i = m % S;
  float4 v;
  if (i < N) {
    v = f4scale(ld4(vision, (b * N + i) * D + c), mtok[b * N + i]);
  } else {
    v = ld4(text, (b * Tn + (i - N)) * D + c);
  }
  *reinterpret_cast<float4*>(X + m * D + c) = v;
}

// ------------------------------------------------------------------ RMSNorm
template <class T>
__global__ __launch_bounds__(TNT) void train_norm_kernel(const float* X, const T* gain, float eps,
                                                         int32_t D, float* U, float* r) {
  __shared__ float red[4];
  const int64_t m = blockIdx.x;
  const float* x = X + m * D;
  float ss = 0.0f;
  for (int c = threadIdx.x * 4; c < D; c += TNT * 4) {
    const float4 v = *reinterpret_cast<const float4*>(x + c);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = block_sum(ss, red);
  const float rr = 1.0f / sqrtf(ss / (float)D + eps);
  if (threadIdx.x == 0) r[m] = rr;
  for (int c = threadIdx.x * 4; c < D; c += TNT * 4) {
    const float4 v = *reinterpret_cast<const float4*>(x + c);
    const float4 g = ld4(gain, c);
    *reinterpret_cast<float4*>(U + m * D + c) =
        make_float4(v.x * rr * g.x, v.y * rr * g.y, v.z * rr * g.z, v.w * rr * g.w);
  }
}

// dX = dRes + r g dY - x r^3 (sum_k g_k dY_k x_k) / D  (dX may be dRes).
template <class T>
__global__ __launch_bounds__(TNT) void train_norm_bwd_kernel(const float* X, const T* gain,
                                                             const float* r, const float* dY,
                                                             const float* dRes, int32_t D,
                                                             float* dX) {
  __shared__ float red[4];
  const int64_t m = blockIdx.x;
  const float* x = X + m * D;
  const float* dy = dY + m * D;
  float dot = 0.0f;
  for (int c = threadIdx.x * 4; c < D; c += TNT * 4) {
    const float4 v = *reinterpret_cast<const float4*>(x + c);
    const float4 e = *reinterpret_cast<const float4*>(dy + c);
    const float4 g = ld4(gain, c);
    dot += g.x * e.x * v.x + g.y * e.y * v.y + g.z * e.z * v.z + g.w * e.w * v.w;
  }
  dot = block_sum(dot, red);
  const float rr = r[m];
  const float coef = rr * rr * rr * dot / (float)D;
  for (int c = threadIdx.x * 4; c < D; c += TNT * 4) {
    const float4 v = *reinterpret_cast<const float4*>(x + c);
    const float4 e = *reinterpret_cast<const float4*>(dy + c);
    const float4 g = ld4(gain, c);
    const float4 d0 = *reinterpret_cast<const float4*>(dRes + m * D + c);
    *reinterpret_cast<float4*>(dX + m * D + c) =
        make_float4(d0.x + rr * g.x * e.x - v.x * coef, d0.y + rr * g.y * e.y - v.y * coef,
                    d0.z + rr * g.z * e.z - v.z * coef, d0.w + rr * g.w * e.w - v.w * coef);
  }
}

// ------------------------------------------------------------------ matrix products
// C[M][N] = R + (s . A)[M][K] op(B): BL = 0 reads B as [N][K] (x W^T with
// W = [out][in]), BL = 1 as [K][N] (dY W).  64 x 64 output tiles over four
// waves (32 x 32 each, 2 x 2 blocks of v_mfma_f32_16x16x4_f32, float32 in
// and out); K in steps of 32 staged through LDS k-major, so a fragment is one
// 4-byte read per lane (K % 16 == 0: a last half step reads as zero); the
// next step's operands are in registers while the current one multiplies.  With ASC, A[m][k] is scaled by
// ascale[(m / S) astride + k / kg] (the unit masks).  blockIdx.z is the K
// piece: with more than one, each writes its own float32 slice (no R).
// LDS row stride (floats): measured over 68-96 on the headline-shape training
// step, 68 and 76 take 313 ms per step against 331 ms for 80 and 72 (fewer
// bank conflicts on the transposed stores and the fragment reads)
constexpr int GBM = 64, GBN = 64, GBK = 32, GLD = 68;

template <int BL, class TB, bool ASC>
__global__ __launch_bounds__(TNT) void train_gemm_kernel(TGemmArgs a) {
  __shared__ __attribute__((aligned(16))) float As[GBK][GLD];   // As[k][m]
  __shared__ __attribute__((aligned(16))) float Bs[GBK][GLD];   // Bs[k][n]
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wy = wave >> 1, wx = wave & 1;
  const int64_t m0 = (int64_t)blockIdx.y * GBM, n0 = (int64_t)blockIdx.x * GBN;
  const TB* B = static_cast<const TB*>(a.B);
  const int64_t k_lo = (int64_t)blockIdx.z * a.kpiece;   // this piece's K range
  const int64_t k_hi = k_lo + a.kpiece < a.K ? k_lo + a.kpiece : a.K;
  const bool split = gridDim.z > 1;
  float* C = split ? a.part + (int64_t)blockIdx.z * a.M * a.N : a.C;
  const int64_t ldc = split ? a.N : a.ldc;
  const float* R = split ? nullptr : a.R;

  // global -> register loads: A row ar, k ak..ak+3; B as [N][K] row bn, k bk..,
  // or as [K][N] row bk, n bn..
  const int ar = t >> 2, ak = (t & 3) * 4;
  const int64_t arow = m0 + ar;
  const bool aok = arow < a.M;
  int bn, bk;
  if constexpr (BL == 0) { bn = t >> 2; bk = (t & 3) * 4; }
  else { bk = t >> 4; bn = (t & 15) * 4; }
  const bool bok = n0 + bn < a.N;
  const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
  // the row's unit masks (its sample's), found once; a k's unit is a 32-bit
  // quotient (K < 2^31), the four k of a piece share it (kg % 4 == 0)
  const float* srow = nullptr;
  if constexpr (ASC) srow = a.ascale + (aok ? (arow / a.S) * a.astride : 0);
  auto load_a = [&](int64_t k0, float4 (&v)[2]) {
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      v[h2] = zero;
      if (aok && k0 + 16 * h2 < k_hi) {   // K % 32 == 16: the second half of the last step is 0
        v[h2] = *reinterpret_cast<const float4*>(a.A + arow * a.lda + k0 + 16 * h2 + ak);
        if constexpr (ASC)
          v[h2] = f4scale(v[h2], srow[(uint32_t)(k0 + 16 * h2 + ak) / (uint32_t)a.kg]);
      }
    }
  };
  auto load_b = [&](int64_t k0, float4 (&v)[2]) {
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      v[h2] = zero;
      if (bok && k0 + 16 * h2 < k_hi) {
        if constexpr (BL == 0) v[h2] = ld4(B, (n0 + bn) * a.ldb + k0 + 16 * h2 + bk);
        else v[h2] = ld4(B, (k0 + 16 * h2 + bk) * a.ldb + n0 + bn);
      }
    }
  };

  floatx4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  // fragment reads: lane l takes row (or column) 16 blk + l % 16 at k = l / 16
  const int fr = lane & 15, fk = lane >> 4;

  float4 av[2], bv[2];
  load_a(k_lo, av);
  load_b(k_lo, bv);
  for (int64_t k0 = k_lo; k0 < k_hi; k0 += GBK) {
    __syncthreads();   // the previous step's readers are done
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      const int kb = 16 * h2;
      As[kb + ak + 0][ar] = av[h2].x;
      As[kb + ak + 1][ar] = av[h2].y;
      As[kb + ak + 2][ar] = av[h2].z;
      As[kb + ak + 3][ar] = av[h2].w;
      if constexpr (BL == 0) {
        Bs[kb + bk + 0][bn] = bv[h2].x;
        Bs[kb + bk + 1][bn] = bv[h2].y;
        Bs[kb + bk + 2][bn] = bv[h2].z;
        Bs[kb + bk + 3][bn] = bv[h2].w;
      } else {
        *reinterpret_cast<float4*>(&Bs[kb + bk][bn]) = bv[h2];
      }
    }
    __syncthreads();
    if (k0 + GBK < k_hi) {
      load_a(k0 + GBK, av);
      load_b(k0 + GBK, bv);
    }
#pragma unroll
    for (int kk = 0; kk < GBK; kk += 4) {
      float fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) fa[i] = As[kk + fk][32 * wy + 16 * i + fr];
#pragma unroll
      for (int j = 0; j < 2; ++j) fb[j] = Bs[kk + fk][32 * wx + 16 * j + fr];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
  }

  // acc[i][j][r] = C[32 wy + 16 i + 4 (lane / 16) + r][32 wx + 16 j + lane % 16]
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int64_t col = n0 + 32 * wx + 16 * j + fr;
    if (col >= a.N) continue;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = m0 + 32 * wy + 16 * i + 4 * fk + r;
        if (row >= a.M) continue;
        float o = acc[i][j][r];
        if (R) o += R[row * a.ldr + col];
        C[row * ldc + col] = o;
      }
  }
}

// C = R + the K pieces' slices added in piece order, four columns per thread.
__global__ void train_splitk_reduce_kernel(const float* part, int32_t ns, int64_t M, int64_t N,
                                           const float* R, int64_t ldr, float* C, int64_t ldc) {
  const int64_t n4 = N / 4;
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= M * n4) return;
  const int64_t m = q / n4, c = (q % n4) * 4;
  float4 s = *reinterpret_cast<const float4*>(part + m * N + c);
  for (int z = 1; z < ns; ++z) {
    const float4 p = *reinterpret_cast<const float4*>(part + (z * M + m) * N + c);
    s.x += p.x; s.y += p.y; s.z += p.z; s.w += p.w;
  }
  if (R) {
    const float4 r = *reinterpret_cast<const float4*>(R + m * ldr + c);
    s.x = r.x + s.x; s.y = r.y + s.y; s.z = r.z + s.z; s.w = r.w + s.w;
  }
  *reinterpret_cast<float4*>(C + m * ldc + c) = s;
}

// ------------------------------------------------------------------ RoPE
// Rotates pairs (r, r + d/2) of nheads heads of X [M][ld] in place by the
// angle of the row's position (sgn = +1) or back (sgn = -1, the transpose).
__global__ void train_rope_kernel(float* X, int64_t ld, int32_t nheads, int32_t d, int32_t S,
                                  int64_t M, const float2* tab, float sgn) {
  const int half = d / 2;
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= M * nheads * half) return;
  const int64_t m = q / ((int64_t)nheads * half);
  const int rem = (int)(q % ((int64_t)nheads * half));
  const int h = rem / half, r = rem % half;
  const float2 cs = tab[(m % S) * half + r];
  const float s = sgn * cs.y;
  float* p = X + m * ld + (int64_t)h * d;
  const float a1 = p[r], a2 = p[r + half];
  p[r] = a1 * cs.x - a2 * s;
  p[r + half] = a2 * cs.x + a1 * s;
}

// ------------------------------------------------------------------ attention
// One workgroup: 64 rows (queries, or keys for the K/V gradient) of one head
// of one sample, four waves of 16 rows each on fp32 MFMA; the other
// operand's rows go through LDS 64 at a time.

// Forward: one workgroup = 64 query rows of one head against the key tiles
// up to its own, with an online softmax; writes O and the log-sum-exp of
// every row for the backward.
template <int HD>
struct FwdSmem {
  // one region in turn: Q^T of the query tile (scaled by 1/sqrt(d), read
  // once into registers), then per key tile K^T, then P^T (pt[key][query])
  // once every wave has its scores; 69 KB at d = 128, two workgroups per CU
  union {
    float qt[HD][68];
    float kt[HD][68];
    float pt[64][68];
  } u;
  float v[64][HD + 4];  // V rows of the key tile
};

template <int HD>
__global__ __launch_bounds__(TNT) void train_attn_fwd_kernel(TAttnArgs a) {
  // 64 queries x 64 keys per tile on v_mfma_f32_16x16x4_f32: wave w owns
  // queries 16 w .. 16 w + 15 against the tile's 64 keys (four 16 x 16
  // score blocks, A = the wave's Q fragments in registers, B = K^T), then
  // O += P V with P passed through the wave's own columns of P^T in LDS
  // (A operand) and V rows (B operand).  Lane l holds rows 4 (l / 16) + r, r < 4, of every
  // block, so a row's statistics stay in the 16 lanes that share l / 16.
  constexpr int NBO = HD / 16;   // 16-column blocks of the output
  constexpr int C4 = HD / 4;
  __shared__ __attribute__((aligned(16))) FwdSmem<HD> sm;
  const int qt = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int rep = a.A / a.KV, g = h / rep;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int64_t base = (int64_t)b * a.S;
  const int64_t ldq = (int64_t)a.A * HD, ldk = (int64_t)a.KV * HD;
  const int64_t q0 = (int64_t)qt * 64;

  for (int idx = t; idx < 64 * C4; idx += TNT) {
    const int r = idx / C4, c = (idx % C4) * 4;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (q0 + r < a.S) v = f4scale(*reinterpret_cast<const float4*>(a.Q + (base + q0 + r) * ldq + (int64_t)h * HD + c), a.scale);
    sm.u.qt[c + 0][r] = v.x;
    sm.u.qt[c + 1][r] = v.y;
    sm.u.qt[c + 2][r] = v.z;
    sm.u.qt[c + 3][r] = v.w;
  }
  __syncthreads();
  const int qw = 16 * wave;   // the wave's first query of the tile
  // the wave's A fragments of the score products: qf[i] = Q^T[4 i + lg][qw + lr]
  float qf[HD / 4];
#pragma unroll
  for (int i = 0; i < HD / 4; ++i) qf[i] = sm.u.qt[4 * i + lg][qw + lr];
  float mrow[4], lrow[4];
  floatx4 o[NBO];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    mrow[r] = -INFINITY;
    lrow[r] = 0.0f;
  }
#pragma unroll
  for (int n = 0; n < NBO; ++n) o[n] = floatx4{0.f, 0.f, 0.f, 0.f};
  // K / V of a key tile: thread pieces idx = t + TNT e (row idx / C4, 4
  // columns from (idx % C4) * 4), loaded into registers one tile ahead
  constexpr int KE = 64 * C4 / TNT;
  static_assert(64 * C4 % TNT == 0, "whole pieces per thread");
  float4 kreg[KE], vreg[KE];
  auto load_kv = [&](int64_t k0) {
#pragma unroll
    for (int e = 0; e < KE; ++e) {
      const int idx = t + TNT * e, r = idx / C4, c = (idx % C4) * 4;
      kreg[e] = make_float4(0.f, 0.f, 0.f, 0.f);
      vreg[e] = kreg[e];
      if (k0 + r < a.S) {
        const int64_t off = (base + k0 + r) * ldk + (int64_t)g * HD + c;
        kreg[e] = *reinterpret_cast<const float4*>(a.K + off);
        vreg[e] = *reinterpret_cast<const float4*>(a.V + off);
      }
    }
  };
  load_kv(0);
  for (int kt = 0; kt <= qt; ++kt) {
    const int64_t k0 = (int64_t)kt * 64;
    __syncthreads();   // the previous tile's readers (and the Q^T readers) are done
#pragma unroll
    for (int e = 0; e < KE; ++e) {
      const int idx = t + TNT * e, r = idx / C4, c = (idx % C4) * 4;
      sm.u.kt[c + 0][r] = kreg[e].x;
      sm.u.kt[c + 1][r] = kreg[e].y;
      sm.u.kt[c + 2][r] = kreg[e].z;
      sm.u.kt[c + 3][r] = kreg[e].w;
      *reinterpret_cast<float4*>(&sm.v[r][c]) = vreg[e];
    }
    __syncthreads();
    if (kt < qt) load_kv(k0 + 64);
    floatx4 sc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) sc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int d = 0; d < HD; d += 4) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        sc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(qf[d / 4], sm.u.kt[d + lg][16 * j + lr], sc[j],
                                                     0, 0, 0);
    }
    // sc[j][r] = score of query qw + 4 lg + r and key 16 j + lr of the tile
    float corr[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t qi = q0 + qw + 4 * lg + r;
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t kj = k0 + 16 * j + lr;
        if (kj > qi || kj >= a.S) sc[j][r] = -INFINITY;
        mx = fmaxf(mx, sc[j][r]);
      }
#pragma unroll
      for (int o2 = 1; o2 < 16; o2 <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o2, 64));
      const float mn = fmaxf(mrow[r], mx);
      // a row with no valid key so far keeps max -inf: its probabilities are 0
      const float mref = mn == -INFINITY ? 0.0f : mn;
      corr[r] = expf(mrow[r] - mref);
      float rs = 0.0f;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float p = expf(sc[j][r] - mref);
        sc[j][r] = p;
        rs += p;
      }
#pragma unroll
      for (int o2 = 1; o2 < 16; o2 <<= 1) rs += __shfl_xor(rs, o2, 64);
      lrow[r] = lrow[r] * corr[r] + rs;
      mrow[r] = mn;
    }
    // P^T: pt[key][query], the wave's own 16 query columns, in K^T's place
    // once every wave has read K^T
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *reinterpret_cast<float4*>(&sm.u.pt[16 * j + lr][qw + 4 * lg]) =
          make_float4(sc[j][0], sc[j][1], sc[j][2], sc[j][3]);
#pragma unroll
    for (int n = 0; n < NBO; ++n)
#pragma unroll
      for (int r = 0; r < 4; ++r) o[n][r] *= corr[r];
    // O += P V (the P^T writes above are the wave's own; LDS keeps a wave's order)
#pragma unroll 4
    for (int k = 0; k < 64; k += 4) {
      const float pa = sm.u.pt[k + lg][qw + lr];
#pragma unroll
      for (int n = 0; n < NBO; ++n)
        o[n] = __builtin_amdgcn_mfma_f32_16x16x4f32(pa, sm.v[k + lg][16 * n + lr], o[n], 0, 0, 0);
    }
  }
  // o[n][r] = O of query qw + 4 lg + r, column 16 n + lr
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t qi = q0 + qw + 4 * lg + r;
    if (qi >= a.S) continue;
    const float inv = 1.0f / lrow[r];
#pragma unroll
    for (int n = 0; n < NBO; ++n)
      a.out[(base + qi) * ldq + (int64_t)h * HD + 16 * n + lr] = o[n][r] * inv;
    if (lr == 0) a.lse[(base + qi) * a.A + h] = mrow[r] + logf(lrow[r]);
  }
}

// Loads rows [row0, row0 + 64) x columns [col0, col0 + HD) of a [M][ld]
// float matrix transposed into dst[HD][68] (rows past `rows_left` read 0),
// optionally scaled.
template <int HD>
__device__ __forceinline__ void load_t(float (*dst)[68], const float* src, int64_t row0, int64_t ld,
                                       int64_t col0, int64_t rows_left, float scale) {
  constexpr int C4 = HD / 4;
  for (int idx = threadIdx.x; idx < 64 * C4; idx += TNT) {
    const int r = idx / C4, c = (idx % C4) * 4;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r < rows_left) v = f4scale(*reinterpret_cast<const float4*>(src + (row0 + r) * ld + col0 + c), scale);
    dst[c + 0][r] = v.x;
    dst[c + 1][r] = v.y;
    dst[c + 2][r] = v.z;
    dst[c + 3][r] = v.w;
  }
}

// Query gradient: one workgroup = 64 query rows of one head.  Per key tile
// S = (Q scale) K^T and dP = dO V^T, dS = P (dP - D) with P = exp(S - lse),
// then dQ += dS K (scaled at the end).  D = dO . O per row is formed first
// and stored for the key / value gradient.
template <int HD>
struct DqSmem {
  // first the query tile's Q^T (scaled) in kt and dO^T in vt, read once into
  // registers; then per key tile K^T and V^T, and dS (ds[key][query]) in
  // V^T's place once every wave has its dP: 69 KB at d = 128, two
  // workgroups per CU
  float kt[HD][68];
  union {
    float vt[HD][68];
    float ds[64][68];
  } u;
};

template <int HD>
__global__ __launch_bounds__(TNT, 2) void train_attn_dq_kernel(TAttnArgs a) {   // 2 waves per SIMD
  // v_mfma_f32_16x16x4_f32: wave w owns queries 16 w .. 16 w + 15 of the
  // tile; S = (Q scale) K^T and dP = dO V^T as four 16 x 16 blocks each (A
  // the wave's Q / dO fragments in registers, B from K^T / V^T), then
  // dS = P (dP - D) through the wave's own columns of ds[key][query] into
  // dQ += dS K.  Lane l holds rows 4 (l / 16) + r, r < 4, of every block.
  constexpr int NBO = HD / 16;
  constexpr int CPT = HD / 16;   // columns per lane of the D reduction
  __shared__ __attribute__((aligned(16))) DqSmem<HD> sm;
  const int qt = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int rep = a.A / a.KV, g = h / rep;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int64_t base = (int64_t)b * a.S;
  const int64_t ldq = (int64_t)a.A * HD, ldk = (int64_t)a.KV * HD;
  const int64_t q0 = (int64_t)qt * 64;
  const int qw = 16 * wave;
  load_t<HD>(sm.kt, a.Q, base + q0, ldq, (int64_t)h * HD, a.S - q0, a.scale);
  load_t<HD>(sm.u.vt, a.dO, base + q0, ldq, (int64_t)h * HD, a.S - q0, 1.0f);
  __syncthreads();
  // the wave's A fragments: qf[i] = (Q scale)^T[4 i + lg][qw + lr], df[i] the same of dO
  float qf[HD / 4], df[HD / 4];
#pragma unroll
  for (int i = 0; i < HD / 4; ++i) {
    qf[i] = sm.kt[4 * i + lg][qw + lr];
    df[i] = sm.u.vt[4 * i + lg][qw + lr];
  }
  // D = dO . O and lse of the lane's four rows (each of the 16 lanes of a
  // row sums HD / 16 of its columns)
  float Dr[4], lse[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t qi = q0 + qw + 4 * lg + r;
    float d = 0.0f;
    if (qi < a.S) {
      const int64_t off = (base + qi) * ldq + (int64_t)h * HD + lr * CPT;
#pragma unroll
      for (int c = 0; c < CPT; ++c) d += a.dO[off + c] * a.O[off + c];
    }
#pragma unroll
    for (int o2 = 1; o2 < 16; o2 <<= 1) d += __shfl_xor(d, o2, 64);
    Dr[r] = d;
    lse[r] = qi < a.S ? a.lse[(base + qi) * a.A + h] : 0.0f;
    if (lr == 0 && qi < a.S) a.Dv[(base + qi) * a.A + h] = d;
  }
  floatx4 acc[NBO];
#pragma unroll
  for (int n = 0; n < NBO; ++n) acc[n] = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int kt = 0; kt <= qt; ++kt) {
    const int64_t k0 = (int64_t)kt * 64;
    __syncthreads();   // the previous tile's (and the query fragments') readers are done
    load_t<HD>(sm.kt, a.K, base + k0, ldk, (int64_t)g * HD, a.S - k0, 1.0f);
    load_t<HD>(sm.u.vt, a.V, base + k0, ldk, (int64_t)g * HD, a.S - k0, 1.0f);
    __syncthreads();
    floatx4 sc[4], dp[4];
#pragma unroll
    for (int jb = 0; jb < 4; ++jb) sc[jb] = dp[jb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int d = 0; d < HD; d += 4) {
#pragma unroll
      for (int jb = 0; jb < 4; ++jb) {
        sc[jb] = __builtin_amdgcn_mfma_f32_16x16x4f32(qf[d / 4], sm.kt[d + lg][16 * jb + lr], sc[jb],
                                                      0, 0, 0);
        dp[jb] = __builtin_amdgcn_mfma_f32_16x16x4f32(df[d / 4], sm.u.vt[d + lg][16 * jb + lr],
                                                      dp[jb], 0, 0, 0);
      }
    }
    __syncthreads();   // every wave has read V^T: dS goes in its place
    // dS of query qw + 4 lg + r and key 16 jb + lr, into ds[key][query]
#pragma unroll
    for (int jb = 0; jb < 4; ++jb) {
      float4 w;
      float* wv = reinterpret_cast<float*>(&w);
      const int64_t kj = k0 + 16 * jb + lr;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t qi = q0 + qw + 4 * lg + r;
        const float p = (kj <= qi && kj < a.S && qi < a.S) ? expf(sc[jb][r] - lse[r]) : 0.0f;
        wv[r] = p * (dp[jb][r] - Dr[r]);
      }
      *reinterpret_cast<float4*>(&sm.u.ds[16 * jb + lr][qw + 4 * lg]) = w;
    }
    // dQ[q][d] += sum_k dS[q][k] K[k][d] (the ds writes above are the wave's own)
#pragma unroll 4
    for (int k = 0; k < 64; k += 4) {
      const float pa = sm.u.ds[k + lg][qw + lr];
#pragma unroll
      for (int n = 0; n < NBO; ++n)
        acc[n] = __builtin_amdgcn_mfma_f32_16x16x4f32(pa, sm.kt[16 * n + lr][k + lg], acc[n], 0, 0, 0);
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t qi = q0 + qw + 4 * lg + r;
    if (qi >= a.S) continue;
#pragma unroll
    for (int n = 0; n < NBO; ++n)
      a.out[(base + qi) * ldq + (int64_t)h * HD + 16 * n + lr] = acc[n][r] * a.scale;
  }
}

// Key / value gradient: one workgroup = 64 key rows of one K/V head; for
// each query head of the group and each query tile at or after the key
// tile: S^T = K (Q scale)^T and dP^T = V dO^T, P^T = exp(S^T - lse), then dV += P^T dO and, through the
// same LDS block, dK += dS^T (Q scale) with dS^T = P^T (dP^T - D) (the
// scaled query tile carries the 1/sqrt(d) of dK).
template <int HD>
struct DkvSmem {
  float kt[HD][68];     // K^T of the workgroup's keys
  float vt[HD][68];     // V^T
  float qt[HD][68];     // Q^T of the query tile (scaled)
  float dot[HD][68];    // dO^T of the query tile
  float w[64][68];      // w[query][key]: P, then dS
  float lse[64], dv[64];
};

template <int HD>
__global__ __launch_bounds__(TNT) void train_attn_dkv_kernel(TAttnArgs a) {
  // v_mfma_f32_16x16x4_f32: wave w owns keys 16 w .. 16 w + 15 of the tile;
  // S^T = K (Q scale)^T and dP^T = V dO^T as four 16 x 16 blocks each, P^T
  // and then dS^T through the wave's own columns of w[query][key] into
  // dV += P^T dO and dK += dS^T (Q scale).
  constexpr int NBO = HD / 16;
  __shared__ __attribute__((aligned(16))) DkvSmem<HD> sm;
  const int kt = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int rep = a.A / a.KV;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int64_t base = (int64_t)b * a.S;
  const int64_t ldq = (int64_t)a.A * HD, ldk = (int64_t)a.KV * HD;
  const int64_t k0 = (int64_t)kt * 64;
  const int kw = 16 * wave;
  load_t<HD>(sm.kt, a.K, base + k0, ldk, (int64_t)g * HD, a.S - k0, 1.0f);
  load_t<HD>(sm.vt, a.V, base + k0, ldk, (int64_t)g * HD, a.S - k0, 1.0f);
  floatx4 gk[NBO], gv[NBO];
#pragma unroll
  for (int n = 0; n < NBO; ++n) gk[n] = gv[n] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int nqt = (int)((a.S + 63) / 64);
  for (int h = g * rep; h < (g + 1) * rep; ++h) {
    for (int qt = kt; qt < nqt; ++qt) {
      const int64_t q0 = (int64_t)qt * 64;
      __syncthreads();
      load_t<HD>(sm.qt, a.Q, base + q0, ldq, (int64_t)h * HD, a.S - q0, a.scale);
      load_t<HD>(sm.dot, a.dO, base + q0, ldq, (int64_t)h * HD, a.S - q0, 1.0f);
      if (t < 64) {
        const bool in = q0 + t < a.S;
        sm.lse[t] = in ? a.lse[(base + q0 + t) * a.A + h] : 0.0f;
        sm.dv[t] = in ? a.Dv[(base + q0 + t) * a.A + h] : 0.0f;
      }
      __syncthreads();
      floatx4 st[4], dpt[4];
#pragma unroll
      for (int jb = 0; jb < 4; ++jb) st[jb] = dpt[jb] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
      for (int d = 0; d < HD; d += 4) {
        const float ka = sm.kt[d + lg][kw + lr], va = sm.vt[d + lg][kw + lr];
#pragma unroll
        for (int jb = 0; jb < 4; ++jb) {
          st[jb] = __builtin_amdgcn_mfma_f32_16x16x4f32(ka, sm.qt[d + lg][16 * jb + lr], st[jb], 0, 0, 0);
          dpt[jb] = __builtin_amdgcn_mfma_f32_16x16x4f32(va, sm.dot[d + lg][16 * jb + lr], dpt[jb], 0, 0, 0);
        }
      }
      // P^T of key kw + 4 lg + r and query 16 jb + lr, into w[query][key]
      float4 pw[4];
#pragma unroll
      for (int jb = 0; jb < 4; ++jb) {
        const int qj = 16 * jb + lr;
        const int64_t q = q0 + qj;
        const float lq = sm.lse[qj];
        float* pv = reinterpret_cast<float*>(&pw[jb]);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t ki = k0 + kw + 4 * lg + r;
          pv[r] = (q >= ki && q < a.S && ki < a.S) ? expf(st[jb][r] - lq) : 0.0f;
        }
        *reinterpret_cast<float4*>(&sm.w[qj][kw + 4 * lg]) = pw[jb];
      }
      // dV[k][c] += sum_q P^T[k][q] dO[q][c]
#pragma unroll 4
      for (int qq = 0; qq < 64; qq += 4) {
        const float pa = sm.w[qq + lg][kw + lr];
#pragma unroll
        for (int n = 0; n < NBO; ++n)
          gv[n] = __builtin_amdgcn_mfma_f32_16x16x4f32(pa, sm.dot[16 * n + lr][qq + lg], gv[n], 0, 0, 0);
      }
      // dS^T = P^T (dP^T - D) over the same columns (after this wave's reads above)
#pragma unroll
      for (int jb = 0; jb < 4; ++jb) {
        const int qj = 16 * jb + lr;
        const float dq = sm.dv[qj];
        const float* pv = reinterpret_cast<const float*>(&pw[jb]);
        float4 w;
        float* wv = reinterpret_cast<float*>(&w);
#pragma unroll
        for (int r = 0; r < 4; ++r) wv[r] = pv[r] * (dpt[jb][r] - dq);
        *reinterpret_cast<float4*>(&sm.w[qj][kw + 4 * lg]) = w;
      }
      // dK[k][c] += sum_q dS^T[k][q] (Q scale)[q][c]
#pragma unroll 4
      for (int qq = 0; qq < 64; qq += 4) {
        const float sa = sm.w[qq + lg][kw + lr];
#pragma unroll
        for (int n = 0; n < NBO; ++n)
          gk[n] = __builtin_amdgcn_mfma_f32_16x16x4f32(sa, sm.qt[16 * n + lr][qq + lg], gk[n], 0, 0, 0);
      }
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t ki = k0 + kw + 4 * lg + r;
    if (ki >= a.S) continue;
#pragma unroll
    for (int n = 0; n < NBO; ++n) {
      const int64_t off = (base + ki) * ldk + (int64_t)g * HD + 16 * n + lr;
      a.dK[off] = gk[n][r];
      a.dV[off] = gv[n][r];
    }
  }
}

// ------------------------------------------------------------------ SwiGLU
__global__ void train_swiglu_kernel(const float* AG, const float* AE, int64_t n, float* H) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= n) return;
  const float x = AG[q];
  H[q] = x / (1.0f + expf(-x)) * AE[q];
}

// Per row: part[m][u] = sum over unit u's channels of dHm . H; then, with the
// unit's mask s, dH = s dHm and the gate / up gradients replace AG and AE.
__global__ __launch_bounds__(TNT) void train_swiglu_bwd_kernel(const float* dHm, float* AG,
                                                               float* AE, const float* H,
                                                               const float* mrow, int64_t mstride,
                                                               int32_t S, int32_t F, int32_t U,
                                                               float* part) {
  __shared__ float red[4];
  const int64_t m = blockIdx.x;
  const int64_t b = m / S;
  const int w = F / U;
  for (int u = 0; u < U; ++u) {
    const float s = mrow[b * mstride + u];
    float dot = 0.0f;
    for (int c = u * w + threadIdx.x; c < (u + 1) * w; c += TNT) {
      const int64_t q = m * F + c;
      const float dh = dHm[q];
      dot += dh * H[q];
      const float x = AG[q], e = AE[q];
      const float sg = 1.0f / (1.0f + expf(-x));
      const float dm = dh * s;
      AG[q] = dm * e * sg * (1.0f + x * (1.0f - sg));
      AE[q] = dm * x * sg;
    }
    dot = block_sum(dot, red);
    if (threadIdx.x == 0) part[m * U + u] = dot;
  }
}

// Per row: part[m][u] = sum over unit u's head columns of dOm . O; dOm *= s.
__global__ __launch_bounds__(TNT) void train_attn_mask_bwd_kernel(float* dOm, const float* O,
                                                                  const float* mrow,
                                                                  int64_t mstride, int32_t S,
                                                                  int32_t W, int32_t U,
                                                                  float* part) {
  __shared__ float red[4];
  const int64_t m = blockIdx.x;
  const int64_t b = m / S;
  const int w = W / U;
  for (int u = 0; u < U; ++u) {
    const float s = mrow[b * mstride + u];
    float dot = 0.0f;
    for (int c = u * w + threadIdx.x; c < (u + 1) * w; c += TNT) {
      const int64_t q = m * W + c;
      const float d = dOm[q];
      dot += d * O[q];
      dOm[q] = d * s;
    }
    dot = block_sum(dot, red);
    if (threadIdx.x == 0) part[m * U + u] = dot;
  }
}

// dM[b][l][u] = sum over the sample's rows of both partial sums, in float64: one
// workgroup per (b, u), each thread a stride of rows, then a fixed-order tree.
__global__ __launch_bounds__(TNT) void train_mask_reduce_kernel(const float* pa, const float* pf,
                                                                int32_t S, int32_t U, int32_t L,
                                                                int32_t l, float* dM) {
  __shared__ double red[TNT / 64];
  const int b = blockIdx.x / U, u = blockIdx.x % U;
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < S; i += TNT) {
    const int64_t r = ((int64_t)b * S + i) * U + u;
    s += (double)pa[r] + (double)pf[r];
  }
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0)
    dM[((int64_t)b * L + l) * U + u] = (float)((red[0] + red[1]) + (red[2] + red[3]));
}

// dL/dz_i = (dX0_i . v_i) y (1 - y) / tau_tok, one workgroup per vision token.
template <class T>
__global__ __launch_bounds__(TNT) void train_token_grad_kernel(const float* dX0, const T* vision,
                                                               const float* stet, int32_t N,
                                                               int32_t S, int32_t D,
                                                               float* grad) {
  __shared__ float red[4];
  const int64_t t = blockIdx.x;   // b N + i
  const int64_t b = t / N, i = t % N;
  const float* dx = dX0 + (b * S + i) * D;
  float dot = 0.0f;
  for (int c = threadIdx.x * 4; c < D; c += TNT * 4) {
    const float4 e = *reinterpret_cast<const float4*>(dx + c);
    const float4 v = ld4(vision, t * D + c);
    dot += e.x * v.x + e.y * v.y + e.z * v.z + e.w * v.w;
  }
  dot = block_sum(dot, red);
  if (threadIdx.x == 0) grad[t] = dot * stet[t];
}

__global__ void train_gate_grad_kernel(const float* dM, const float* steg, int32_t B, int32_t L,
                                       int32_t P, int32_t U, float* grad) {
  const int64_t per = (int64_t)(L - P) * U;
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= B * per) return;
  const int64_t b = q / per, r = q % per;
  grad[q] = dM[b * L * U + (int64_t)P * U + r] * steg[q];
}

unsigned blocks(int64_t n) { return (unsigned)((n + TNT - 1) / TNT); }

}  // namespace

hipError_t launch_train_masks(const TrainMaskArgs& a, hipStream_t st) {
  const int64_t n = (int64_t)a.B * a.N + (int64_t)a.B * (a.L - a.P) * a.U + (int64_t)a.B * a.P * a.U;
  if (n <= 0) return hipSuccess;
  train_masks_kernel<<<blocks(n), TNT, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_train_embed(const void* vision, const void* text, const float* mtok, int32_t B,
                              int32_t N, int32_t T, int32_t D, bool bf16, float* X,
                              hipStream_t st) {
  const int64_t n = (int64_t)B * (N + T) * (D / 4);
  if (n <= 0) return hipSuccess;
  if (bf16)
    train_embed_kernel<uint16_t><<<blocks(n), TNT, 0, st>>>(
        static_cast<const uint16_t*>(vision), static_cast<const uint16_t*>(text), mtok, B, N, T, D, X);
  else
    train_embed_kernel<float><<<blocks(n), TNT, 0, st>>>(static_cast<const float*>(vision),
                                                         static_cast<const float*>(text), mtok, B,
                                                         N, T, D, X);
  return hipGetLastError();
}

hipError_t launch_train_norm(const float* X, const void* gain, float eps, int64_t M, int32_t D,
                             bool bf16, float* U, float* r, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (bf16)
    train_norm_kernel<uint16_t><<<(unsigned)M, TNT, 0, st>>>(X, static_cast<const uint16_t*>(gain),
                                                             eps, D, U, r);
  else
    train_norm_kernel<float><<<(unsigned)M, TNT, 0, st>>>(X, static_cast<const float*>(gain), eps,
                                                          D, U, r);
  return hipGetLastError();
}

hipError_t launch_train_norm_bwd(const float* X, const void* gain, const float* r, const float* dY,
                                 const float* dRes, int64_t M, int32_t D, bool bf16, float* dX,
                                 hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (bf16)
    train_norm_bwd_kernel<uint16_t><<<(unsigned)M, TNT, 0, st>>>(
        X, static_cast<const uint16_t*>(gain), r, dY, dRes, D, dX);
  else
    train_norm_bwd_kernel<float><<<(unsigned)M, TNT, 0, st>>>(X, static_cast<const float*>(gain),
                                                              r, dY, dRes, D, dX);
  return hipGetLastError();
}

hipError_t launch_train_gemm(const TGemmArgs& a, int32_t bl, bool bf16, hipStream_t st) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  const int32_t ns = a.ksplit > 1 ? a.ksplit : 1;
  if (ns > 1 && (!a.part || a.kpiece % GBK || a.kpiece * (ns - 1) >= a.K || a.kpiece * ns < a.K))
    return hipErrorInvalidValue;
  TGemmArgs g = a;
  if (ns == 1) g.kpiece = a.K;
  const dim3 grid((unsigned)((a.N + GBN - 1) / GBN), (unsigned)((a.M + GBM - 1) / GBM),
                  (unsigned)ns);
  const bool asc = a.ascale != nullptr;
#define SVL_TGEMM(BLV, TB, ASCV) train_gemm_kernel<BLV, TB, ASCV><<<grid, TNT, 0, st>>>(g)
  if (bl == 0) {
    if (bf16) { if (asc) SVL_TGEMM(0, uint16_t, true); else SVL_TGEMM(0, uint16_t, false); }
    else { if (asc) SVL_TGEMM(0, float, true); else SVL_TGEMM(0, float, false); }
  } else {
    if (bf16) SVL_TGEMM(1, uint16_t, false);
    else SVL_TGEMM(1, float, false);
  }
#undef SVL_TGEMM
  if (ns == 1) return hipGetLastError();
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  train_splitk_reduce_kernel<<<blocks(a.M * (a.N / 4)), TNT, 0, st>>>(a.part, ns, a.M, a.N, a.R,
                                                                       a.ldr, a.C, a.ldc);
  return hipGetLastError();
}

hipError_t launch_train_rope(float* X, int64_t ld, int32_t nheads, int32_t d, int32_t S, int64_t M,
                             const float2* tab, float sgn, hipStream_t st) {
  const int64_t n = M * nheads * (d / 2);
  if (n <= 0) return hipSuccess;
  train_rope_kernel<<<blocks(n), TNT, 0, st>>>(X, ld, nheads, d, S, M, tab, sgn);
  return hipGetLastError();
}

hipError_t launch_train_attn(const TAttnArgs& a, int32_t head_dim, int32_t B, int32_t which,
                             hipStream_t st) {
  const unsigned tiles = (unsigned)((a.S + 63) / 64);
  if (tiles == 0 || B <= 0) return hipSuccess;
  const dim3 grid(tiles, (unsigned)(which == 2 ? a.KV : a.A), (unsigned)B);
#define SVL_TATTN(HD)                                                      \
  do {                                                                     \
    if (which == 0) train_attn_fwd_kernel<HD><<<grid, TNT, 0, st>>>(a);    \
    else if (which == 1) train_attn_dq_kernel<HD><<<grid, TNT, 0, st>>>(a); \
    else train_attn_dkv_kernel<HD><<<grid, TNT, 0, st>>>(a);               \
  } while (0)
  switch (head_dim) {
    case 32: SVL_TATTN(32); break;
    case 64: SVL_TATTN(64); break;
    case 128: SVL_TATTN(128); break;
    default: return hipErrorInvalidValue;
  }
#undef SVL_TATTN
  return hipGetLastError();
}

hipError_t launch_train_swiglu(const float* AG, const float* AE, int64_t n, float* H,
                               hipStream_t st) {
  if (n <= 0) return hipSuccess;
  train_swiglu_kernel<<<blocks(n), TNT, 0, st>>>(AG, AE, n, H);
  return hipGetLastError();
}

hipError_t launch_train_swiglu_bwd(const float* dHm, float* AG, float* AE, const float* H,
                                   const float* mrow, int64_t mstride, int32_t S, int64_t M,
                                   int32_t F, int32_t U, float* part, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  train_swiglu_bwd_kernel<<<(unsigned)M, TNT, 0, st>>>(dHm, AG, AE, H, mrow, mstride, S, F, U, part);
  return hipGetLastError();
}

hipError_t launch_train_attn_mask_bwd(float* dOm, const float* O, const float* mrow,
                                      int64_t mstride, int32_t S, int64_t M, int32_t W, int32_t U,
                                      float* part, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  train_attn_mask_bwd_kernel<<<(unsigned)M, TNT, 0, st>>>(dOm, O, mrow, mstride, S, W, U, part);
  return hipGetLastError();
}

hipError_t launch_train_mask_reduce(const float* pa, const float* pf, int32_t B, int32_t S,
                                    int32_t U, int32_t L, int32_t l, float* dM, hipStream_t st) {
  if (B * U <= 0) return hipSuccess;
  train_mask_reduce_kernel<<<(unsigned)(B * U), TNT, 0, st>>>(pa, pf, S, U, L, l, dM);
  return hipGetLastError();
}

hipError_t launch_train_token_grad(const float* dX0, const void* vision, const float* stet,
                                   int32_t B, int32_t N, int32_t S, int32_t D, bool bf16,
                                   float* grad, hipStream_t st) {
  const int64_t n = (int64_t)B * N;
  if (n <= 0) return hipSuccess;
  if (bf16)
    train_token_grad_kernel<uint16_t><<<(unsigned)n, TNT, 0, st>>>(
        dX0, static_cast<const uint16_t*>(vision), stet, N, S, D, grad);
  else
    train_token_grad_kernel<float><<<(unsigned)n, TNT, 0, st>>>(
        dX0, static_cast<const float*>(vision), stet, N, S, D, grad);
  return hipGetLastError();
}

hipError_t launch_train_gate_grad(const float* dM, const float* steg, int32_t B, int32_t L,
                                  int32_t P, int32_t U, float* grad, hipStream_t st) {
  const int64_t n = (int64_t)B * (L - P) * U;
  if (n <= 0) return hipSuccess;
  train_gate_grad_kernel<<<blocks(n), TNT, 0, st>>>(dM, steg, B, L, P, U, grad);
  return hipGetLastError();
}

}  // namespace svl
