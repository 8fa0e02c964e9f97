// Internal declarations of the training-time masked decoder: argument blocks
// of its kernels and their launchers (float32 compute, weights and hidden
// inputs in the storage dtype).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace svl {

// Straight-through masks of Eq. (6) for the tokens and the units.
struct TrainMaskArgs {
  const float* z;      // token logits [B][N]
  const float* zn;     // token noise or nullptr
  const float* g;      // gate logits [B][(L-P) U]
  const float* gn;     // gate noise or nullptr
  int32_t B, N, L, P, U;
  float tau_tok, tau_comp;
  uint8_t* tmask;      // [B][N] out: 1 iff z + xi > 0
  uint8_t* umask;      // [B][(L-P) U] out
  float* mtok;         // [B][N] the token masks as floats
  float* stet;         // [B][N] y (1 - y) / tau_tok
  float* mfull;        // [B][L][U] unit masks of every layer (prefix layers: 1)
  float* steg;         // [B][(L-P) U] y (1 - y) / tau_comp
};

// C = R + (s . A) op(B) (see train_gemm_kernel).
struct TGemmArgs {
  const float* A;
  int64_t lda;
  const void* B;       // weights, storage dtype
  int64_t ldb;
  float* C;
  int64_t ldc;
  const float* R;      // nullptr: no residual (may equal C)
  int64_t ldr;
  const float* ascale; // nullptr, or unit masks: row m, column k -> ascale[(m/S) astride + k/kg]
  int64_t astride;
  int32_t S, kg;
  int64_t M, N, K;     // K % 16 == 0, N % 4 == 0, kg % 4 == 0
  // split K: ksplit pieces of kpiece (a multiple of 32; the last one shorter)
  // write float32 slices [ksplit][M][N] at part, then C = R + their sum
  // (slices in order); ksplit = 1 writes C directly
  int32_t ksplit;
  int64_t kpiece;
  float* part;
};

// Attention of one layer over B samples of S rows (buffers [B S][heads d]).
struct TAttnArgs {
  const float *Q, *K, *V;   // rotated queries and keys, values
  const float* O;           // backward: the forward output (before the masks)
  const float* dO;          // backward: gradient of O (masks applied)
  float* out;               // forward: O; dq pass: dQ
  float* lse;               // [B S][A] log-sum-exp of each row's scores
  float* Dv;                // [B S][A] dO . O
  float *dK, *dV;           // dkv pass outputs
  int64_t S;
  int32_t A, KV;
  float scale;              // 1 / sqrt(d)
};

hipError_t launch_train_masks(const TrainMaskArgs& a, hipStream_t st);
hipError_t launch_train_embed(const void* vision, const void* text, const float* mtok, int32_t B,
                              int32_t N, int32_t T, int32_t D, bool bf16, float* X,
                              hipStream_t st);
hipError_t launch_train_norm(const float* X, const void* gain, float eps, int64_t M, int32_t D,
                             bool bf16, float* U, float* r, hipStream_t st);
hipError_t launch_train_norm_bwd(const float* X, const void* gain, const float* r, const float* dY,
                                 const float* dRes, int64_t M, int32_t D, bool bf16, float* dX,
                                 hipStream_t st);
// bl: 0 reads B as [N][K], 1 as [K][N] (ascale only with bl == 0)
hipError_t launch_train_gemm(const TGemmArgs& a, int32_t bl, bool bf16, hipStream_t st);
hipError_t launch_train_rope(float* X, int64_t ld, int32_t nheads, int32_t d, int32_t S, int64_t M,
                             const float2* tab, float sgn, hipStream_t st);
// which: 0 forward (O, lse), 1 query gradient (dQ, Dv), 2 key / value gradients
hipError_t launch_train_attn(const TAttnArgs& a, int32_t head_dim, int32_t B, int32_t which,
                             hipStream_t st);
hipError_t launch_train_swiglu(const float* AG, const float* AE, int64_t n, float* H,
                               hipStream_t st);
hipError_t launch_train_swiglu_bwd(const float* dHm, float* AG, float* AE, const float* H,
                                   const float* mrow, int64_t mstride, int32_t S, int64_t M,
                                   int32_t F, int32_t U, float* part, hipStream_t st);
hipError_t launch_train_attn_mask_bwd(float* dOm, const float* O, const float* mrow,
                                      int64_t mstride, int32_t S, int64_t M, int32_t W, int32_t U,
                                      float* part, hipStream_t st);
hipError_t launch_train_mask_reduce(const float* pa, const float* pf, int32_t B, int32_t S,
                                    int32_t U, int32_t L, int32_t l, float* dM, hipStream_t st);
hipError_t launch_train_token_grad(const float* dX0, const void* vision, const float* stet,
                                   int32_t B, int32_t N, int32_t S, int32_t D, bool bf16,
                                   float* grad, hipStream_t st);
hipError_t launch_train_gate_grad(const float* dM, const float* steg, int32_t B, int32_t L,
                                  int32_t P, int32_t U, float* grad, hipStream_t st);

}  // namespace svl
