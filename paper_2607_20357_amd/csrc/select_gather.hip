// Token selection (top-k by score, kept indices ascending) and the packing of
// kept vision rows and text rows into the float32 residual stream.
//
// Selection, one workgroup per sample:
//   1. every score is mapped to an unsigned key whose order is the required
//      order: larger score -> larger key, -0 and +0 -> one key, NaN -> 0
//      (below -inf, whose key is 0x007fffff);
//   2. a 4-pass radix select (8 bits per pass, 256-bin LDS histogram whose
//      suffix counts come from a parallel scan; keys kept in LDS for samples
//      of up to 16384 scores) finds the k-th largest key T and how many keys
//      equal to T are kept;
//   3. one ordered pass over the indices keeps key > T, and key == T while
//      fewer than the needed number of equal keys have been seen (ties go to
//      the lower index); wave ballots give the prefix counts, so the kept
//      indices come out in ascending order.
// Gather: one workgroup per packed row, 16-byte loads, exact widening of
// bf16 to float32.
#include "svl_internal.h"
#include "device_util.h"

namespace svl {
namespace {

constexpr int NT = 256;

__device__ __forceinline__ uint32_t score_key(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;  // NaN
  if (u == 0x80000000u) u = 0u;                      // -0 -> +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive count of `p` over the workgroup's threads in thread order, and
// the total.  Every thread of the workgroup must call it.
__device__ __forceinline__ int block_excl_count(bool p, int* s_wave, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const unsigned long long m = __ballot(p);
  const int below = __popcll(m & ((1ull << lane) - 1ull));
  if (lane == 0) s_wave[w] = __popcll(m);
  __syncthreads();
  int off = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) {
    off += (i < w) ? s_wave[i] : 0;
    tot += s_wave[i];
  }
  __syncthreads();
  *total = tot;
  return off + below;
}

// Keys of samples with at most this many scores stay in LDS across the passes.
constexpr int SEL_LDS_KEYS = 16384;

__global__ __launch_bounds__(NT) void select_kernel(const float* scores, int N, const int32_t* keep,
                                                    int32_t* kept_idx) {
  static_assert(NT == 256, "one thread per histogram bin");
  __shared__ uint32_t s_keys[SEL_LDS_KEYS];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t s_wsum[NT / 64];
  __shared__ uint32_t s_digit, s_remaining;
  __shared__ int s_wave[NT / 64];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const float* s = scores + (size_t)b * N;
  int32_t* out = kept_idx + (size_t)b * N;
  const int k = keep[b];
  const bool cached = N <= SEL_LDS_KEYS;
  auto key_at = [&](int i) { return cached ? s_keys[i] : score_key(s[i]); };

  if (k > 0 && k < N) {
    if (cached) {
      for (int i = tid; i < N; i += NT) s_keys[i] = score_key(s[i]);
      __syncthreads();
    }
    uint32_t prefix = 0, mask = 0, remaining = (uint32_t)k;
    for (int shift = 24; shift >= 0; shift -= 8) {
      hist[tid] = 0;
      __syncthreads();
      for (int i = tid; i < N; i += NT) {
        const uint32_t key = key_at(i);
        if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      // Suffix counts S(t) = number of candidate keys whose digit is >= t
      // (thread t holds bin t).  S(0) >= remaining > S(256) = 0, and S never
      // increases, so exactly one bin has S(t) >= remaining > S(t + 1): the
      // digit of the k-th largest key.
      const uint32_t h = hist[tid];
      uint32_t v = h;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t n = __shfl_down(v, o, 64);
        if (lane + o < 64) v += n;
      }
      if (lane == 0) s_wsum[w] = v;
      __syncthreads();
      uint32_t above = 0;
#pragma unroll
      for (int j = 0; j < NT / 64; ++j) above += j > w ? s_wsum[j] : 0u;
      const uint32_t S = v + above, S_next = S - h;
      if (S >= remaining && S_next < remaining) {
        s_digit = (uint32_t)tid;
        s_remaining = remaining - S_next;
      }
      __syncthreads();
      prefix |= s_digit << shift;
      mask |= 255u << shift;
      remaining = s_remaining;
      __syncthreads();
    }
    const uint32_t T = prefix;
    const int need_eq = (int)remaining;
    int eq_seen = 0, written = 0;
    for (int c0 = 0; c0 < N; c0 += NT) {
      const int i = c0 + tid;
      const uint32_t key = i < N ? key_at(i) : 0u;
      const bool gt = i < N && key > T;
      const bool eq = i < N && key == T;
      int eq_tot, keep_tot;
      const int eq_rank = eq_seen + block_excl_count(eq, s_wave, &eq_tot);
      const bool kp = gt || (eq && eq_rank < need_eq);
      const int pos = written + block_excl_count(kp, s_wave, &keep_tot);
      if (kp) out[pos] = i;
      eq_seen += eq_tot;
      written += keep_tot;
    }
  } else if (k == N) {
    for (int i = tid; i < N; i += NT) out[i] = i;
  }
  for (int i = k + tid; i < N; i += NT) out[i] = -1;
}

// Threshold count, one workgroup per sample: visual tokens with
// sigma(z) > 0.5, i.e. z > 0 (zero, -0 and NaN are not counted).
__global__ __launch_bounds__(NT) void count_positive_kernel(const float* logits, int N,
                                                            int32_t* counts) {
  __shared__ int s_wave[NT / 64];
  const int b = blockIdx.x, tid = threadIdx.x;
  const float* z = logits + (size_t)b * N;
  int n = 0;
  for (int i = tid; i < N; i += NT) n += z[i] > 0.0f ? 1 : 0;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) n += __shfl_xor(n, o, 64);
  if ((tid & 63) == 0) s_wave[tid >> 6] = n;
  __syncthreads();
  if (tid == 0) {
    int tot = 0;
#pragma unroll
    for (int i = 0; i < NT / 64; ++i) tot += s_wave[i];
    counts[b] = tot;
  }
}

template <bool BF16>
__global__ __launch_bounds__(NT) void gather_kernel(const int32_t* kept_idx, const int32_t* keep,
                                                    const int32_t* cu, int B, int N, int T, int D,
                                                    const void* vision, const void* text,
                                                    float* resid) {
  const int r = blockIdx.x;
  int lo = 0, hi = B - 1;   // sample b with cu[b] <= r < cu[b+1]
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu[mid] <= r) lo = mid; else hi = mid - 1;
  }
  const int b = lo, i = r - cu[b], k = keep[b];
  if (i >= k + T) return;   // rows past the text (the controlled prefill's budget token)
  size_t src_row;
  const void* src;
  if (i < k) {
    src = vision;
    src_row = (size_t)b * N + min(max(kept_idx[(size_t)b * N + i], 0), N - 1);
  }
  else { src = text; src_row = (size_t)b * T + (i - k); }
  float* dst = resid + (size_t)r * D;
  if constexpr (BF16) {
    const uint4* p = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(src) + src_row * D);
    const int n8 = D / 8;
    constexpr int PER = 4;   // every load of a batch in flight before the first store
    for (int c0 = threadIdx.x; c0 < n8; c0 += PER * NT) {
      uint4 v[PER];
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const int c = c0 + j * NT;
        v[j] = c < n8 ? p[c] : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const int c = c0 + j * NT;
        if (c >= n8) break;
        const float4 f0 = make_float4(bf16_bits_to_f32(v[j].x & 0xffffu), bf16_bits_to_f32(v[j].x >> 16),
                                      bf16_bits_to_f32(v[j].y & 0xffffu), bf16_bits_to_f32(v[j].y >> 16));
        const float4 f1 = make_float4(bf16_bits_to_f32(v[j].z & 0xffffu), bf16_bits_to_f32(v[j].z >> 16),
                                      bf16_bits_to_f32(v[j].w & 0xffffu), bf16_bits_to_f32(v[j].w >> 16));
        reinterpret_cast<float4*>(dst)[2 * c] = f0;
        reinterpret_cast<float4*>(dst)[2 * c + 1] = f1;
      }
    }
  } else {
    const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(src) + src_row * D);
    for (int c = threadIdx.x; c < D / 4; c += NT) reinterpret_cast<float4*>(dst)[c] = p[c];
  }
}

}  // namespace

hipError_t launch_select(const float* scores, int32_t B, int32_t N, const int32_t* keep_dev,
                         int32_t* kept_idx, hipStream_t st) {
  if (B <= 0 || N <= 0) return hipSuccess;
  select_kernel<<<B, NT, 0, st>>>(scores, N, keep_dev, kept_idx);
  return hipGetLastError();
}

hipError_t launch_count_positive(const float* logits, int32_t B, int32_t N, int32_t* counts,
                                 hipStream_t st) {
  if (B <= 0) return hipSuccess;
  count_positive_kernel<<<B, NT, 0, st>>>(logits, N, counts);
  return hipGetLastError();
}

hipError_t launch_gather(const int32_t* kept_idx, const int32_t* keep_dev, const int32_t* cu_dev,
                         int32_t B, int32_t N, int32_t T, int32_t D, int32_t total_rows,
                         const void* vision, const void* text, int32_t dtype, float* resid,
                         hipStream_t st) {
  if (total_rows <= 0) return hipSuccess;
  if (dtype == SVL_BF16)
    gather_kernel<true><<<total_rows, NT, 0, st>>>(kept_idx, keep_dev, cu_dev, B, N, T, D, vision,
                                                    text, resid);
  else
    gather_kernel<false><<<total_rows, NT, 0, st>>>(kept_idx, keep_dev, cu_dev, B, N, T, D, vision,
                                                     text, resid);
  return hipGetLastError();
}

}  // namespace svl
