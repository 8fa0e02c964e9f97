// C ABI of the training-time masked decoder: argument checks (all before
// anything is enqueued), workspace layout and the launch sequence of the
// forward and of the backward to the token and gate logits.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>

#include "../../include/svl.h"
#include "svl_internal.h"
#include "train_internal.h"

namespace svl {
namespace {

int64_t round256(int64_t x) { return (x + 255) & ~int64_t(255); }
bool is_aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

svl_status err(svl_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
svl_status err(svl_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  return set_error(st, buf);
}

// K pieces of a product of M x N over K: a launch of fewer than 1024 64 x 64
// tiles takes 2-4 pieces of at least 512 of K each, so that it holds about
// 1280 workgroups, five per CU (640 tiles leave half the CUs one workgroup
// short); ns = 1 keeps K whole.
struct KSplit {
  int32_t ns;
  int64_t kpiece;
};

KSplit k_split(int64_t M, int64_t N, int64_t K) {
  const int64_t tiles = ((N + 63) / 64) * ((M + 63) / 64);
  int64_t ns = 1;
  if (tiles < 1024) ns = std::min<int64_t>({4, K / 512, (1280 + tiles - 1) / tiles});
  if (ns < 2) return {1, K};
  const int64_t kp = ((K + ns - 1) / ns + 31) / 32 * 32;
  ns = (K + kp - 1) / kp;
  if (ns < 2) return {1, K};
  return {(int32_t)ns, kp};
}

// Byte offsets of the workspace regions (each 256-byte aligned).
struct TrainLayout {
  int64_t xs;                          // X_0 .. X_{L-1}, [L][M][D]
  int64_t mtok, stet, mfull, steg, dM; // masks and straight-through factors
  int64_t rope;                        // (cos, sin)[S][d/2]
  int64_t u, r1, q, k, v, o, lse, x1, u2, r2, ag, ae, hh;   // one layer's forward
  int64_t dxa, dxb, dx1, du, dh, dO, dq, dk, dv, dvec, pa, pf;  // its backward
  int64_t kpart, kpart_floats;         // the K pieces' slices of one product
  int64_t total;
};

TrainLayout train_layout(const svl_config& c, int32_t U, int32_t B, int32_t N, int32_t T) {
  const int64_t S = (int64_t)N + T, M = (int64_t)B * S, D = c.d_model, F = c.d_ffn;
  const int64_t A = c.n_heads, KV = c.n_kv_heads, d = c.head_dim, L = c.n_layers;
  TrainLayout t{};
  int64_t off = 0;
  auto take = [&](int64_t floats) {
    const int64_t at = off;
    off += round256(std::max<int64_t>(floats, 1) * 4);
    return at;
  };
  t.xs = take(L * M * D);
  t.mtok = take((int64_t)B * N);
  t.stet = take((int64_t)B * N);
  t.mfull = take((int64_t)B * L * U);
  t.steg = take((int64_t)B * L * U);
  t.dM = take((int64_t)B * L * U);
  t.rope = take(S * (d / 2) * 2);
  t.u = take(M * D);
  t.r1 = take(M);
  t.q = take(M * A * d);
  t.k = take(M * KV * d);
  t.v = take(M * KV * d);
  t.o = take(M * A * d);
  t.lse = take(M * A);
  t.x1 = take(M * D);
  t.u2 = take(M * D);
  t.r2 = take(M);
  t.ag = take(M * F);
  t.ae = take(M * F);
  t.hh = take(M * F);
  t.dxa = take(M * D);
  t.dxb = take(M * D);
  t.dx1 = take(M * D);
  t.du = take(M * D);
  t.dh = take(M * F);
  t.dO = take(M * A * d);
  t.dq = take(M * A * d);
  t.dk = take(M * KV * d);
  t.dv = take(M * KV * d);
  t.dvec = take(M * A);
  t.pa = take(M * U);
  t.pf = take(M * U);
  // every (N, K) the layer passes multiply
  const int64_t shapes[][2] = {{A * d, D}, {KV * d, D}, {D, A * d}, {D, KV * d}, {F, D}, {D, F}};
  for (const auto& nk : shapes) {
    const KSplit ks = k_split(M, nk[0], nk[1]);
    if (ks.ns > 1) t.kpart_floats = std::max(t.kpart_floats, ks.ns * M * nk[0]);
  }
  t.kpart = take(t.kpart_floats);
  t.total = off;
  return t;
}

svl_status check_train(const svl_config* cfg, const svl_train_params* p, int32_t B, int32_t N,
                       int32_t T) {
  svl_status s = validate_config(cfg);
  if (s != SVL_OK) return s;
  if (!p) return err(SVL_E_NULL, "train params are NULL");
  const svl_config& c = *cfg;
  if (!(std::isfinite(p->tau_tok) && p->tau_tok > 0.f) ||
      !(std::isfinite(p->tau_comp) && p->tau_comp > 0.f))
    return err(SVL_E_VALUE, "temperatures must be finite and > 0");
  if (p->prefix < 0 || p->prefix > c.n_layers) return err(SVL_E_VALUE, "prefix outside [0, n_layers]");
  if (p->units < 1) return err(SVL_E_VALUE, "units must be >= 1");
  if (c.n_heads % p->units || c.d_ffn % p->units)
    return err(SVL_E_SHAPE, "n_heads and d_ffn must be divisible by units");
  if ((c.d_ffn / p->units) % 4) return err(SVL_E_SHAPE, "d_ffn / units must be a multiple of 4");
  if (c.head_dim != 32 && c.head_dim != 64 && c.head_dim != 128)
    return err(SVL_E_SHAPE, "training path: head_dim must be 32, 64 or 128");
  if (c.d_model % 16 || c.d_ffn % 16)
    return err(SVL_E_SHAPE, "training path: d_model and d_ffn must be multiples of 16");
  if (B <= 0 || B > 65535) return err(SVL_E_SHAPE, "batch must be in [1, 65535]");
  if (N < 0 || T < 0 || (int64_t)N + T <= 0) return err(SVL_E_SHAPE, "need n_vision + n_text > 0");
  const int64_t M = (int64_t)B * ((int64_t)N + T);
  if (M > ((int64_t)65535 * 64)) return err(SVL_E_SHAPE, "too many rows (batch x sequence)");
  if ((int64_t)B * N > INT32_MAX || M > INT32_MAX) return err(SVL_E_SHAPE, "too many rows");
  return SVL_OK;
}

svl_status hip_err(hipError_t e, const char* where) {
  return err(SVL_E_HIP, "%s: %s", where, hipGetErrorString(e));
}

// Runs one training step once every argument has been checked.
struct TrainRun {
  const svl_config& c;
  const svl_layer_weights* W;
  int32_t B, N, T, P, U;
  int64_t S, M;
  bool bf16;
  uint8_t* ws;
  const TrainLayout& Lw;
  hipStream_t st;

  float* f(int64_t off) const { return reinterpret_cast<float*>(ws + off); }
  float* xs(int32_t l) const { return f(Lw.xs) + (int64_t)l * M * c.d_model; }

  hipError_t gemm(const float* A, int64_t lda, const void* Bw, int64_t ldb, float* C, int64_t ldc,
                  const float* R, int64_t N_, int64_t K, int32_t bl, const float* ascale,
                  int32_t kg) const {
    TGemmArgs g{};
    g.A = A;
    g.lda = lda;
    g.B = Bw;
    g.ldb = ldb;
    g.C = C;
    g.ldc = ldc;
    g.R = R;
    g.ldr = ldc;
    g.ascale = ascale;
    g.astride = (int64_t)c.n_layers * U;
    g.S = (int32_t)S;
    g.kg = kg;
    g.M = M;
    g.N = N_;
    g.K = K;
    const KSplit ks = k_split(M, N_, K);
    g.ksplit = 1;
    g.kpiece = K;
    if (ks.ns > 1 && ks.ns * M * N_ <= Lw.kpart_floats) {
      g.ksplit = ks.ns;
      g.kpiece = ks.kpiece;
      g.part = f(Lw.kpart);
    }
    return launch_train_gemm(g, bl, bf16, st);
  }

  TAttnArgs attn_args() const {
    TAttnArgs a{};
    a.Q = f(Lw.q);
    a.K = f(Lw.k);
    a.V = f(Lw.v);
    a.O = f(Lw.o);
    a.dO = nullptr;
    a.lse = f(Lw.lse);
    a.Dv = f(Lw.dvec);
    a.S = S;
    a.A = c.n_heads;
    a.KV = c.n_kv_heads;
    a.scale = (float)(1.0 / std::sqrt((double)c.head_dim));
    return a;
  }

  // Forward of layer l from X_l: fills the layer intermediates; with `out`,
  // also the down projection into out (X_{l+1}).
  hipError_t layer_forward(int32_t l, float* out) const {
    const svl_layer_weights& w = W[l];
    const int64_t D = c.d_model, F = c.d_ffn, A = c.n_heads, KV = c.n_kv_heads, d = c.head_dim;
    const float* ms = f(Lw.mfull) + (int64_t)l * U;
    const float2* tab = reinterpret_cast<const float2*>(ws + Lw.rope);
    hipError_t e;
    if ((e = launch_train_norm(xs(l), w.attn_norm, c.rms_eps, M, (int32_t)D, bf16, f(Lw.u),
                               f(Lw.r1), st)) != hipSuccess) return e;
    if ((e = gemm(f(Lw.u), D, w.wq, D, f(Lw.q), A * d, nullptr, A * d, D, 0, nullptr, 1)) != hipSuccess) return e;
    if ((e = gemm(f(Lw.u), D, w.wk, D, f(Lw.k), KV * d, nullptr, KV * d, D, 0, nullptr, 1)) != hipSuccess) return e;
    if ((e = gemm(f(Lw.u), D, w.wv, D, f(Lw.v), KV * d, nullptr, KV * d, D, 0, nullptr, 1)) != hipSuccess) return e;
    if ((e = launch_train_rope(f(Lw.q), A * d, (int32_t)A, (int32_t)d, (int32_t)S, M, tab, 1.f, st)) != hipSuccess) return e;
    if ((e = launch_train_rope(f(Lw.k), KV * d, (int32_t)KV, (int32_t)d, (int32_t)S, M, tab, 1.f, st)) != hipSuccess) return e;
    TAttnArgs a = attn_args();
    a.out = f(Lw.o);
    if ((e = launch_train_attn(a, (int32_t)d, B, 0, st)) != hipSuccess) return e;
    // X1 = X_l + (M . O) Wo^T
    if ((e = gemm(f(Lw.o), A * d, w.wo, A * d, f(Lw.x1), D, xs(l), D, A * d, 0, ms,
                  (int32_t)(A / U * d))) != hipSuccess) return e;
    if ((e = launch_train_norm(f(Lw.x1), w.ffn_norm, c.rms_eps, M, (int32_t)D, bf16, f(Lw.u2),
                               f(Lw.r2), st)) != hipSuccess) return e;
    if ((e = gemm(f(Lw.u2), D, w.w_gate, D, f(Lw.ag), F, nullptr, F, D, 0, nullptr, 1)) != hipSuccess) return e;
    if ((e = gemm(f(Lw.u2), D, w.w_up, D, f(Lw.ae), F, nullptr, F, D, 0, nullptr, 1)) != hipSuccess) return e;
    if ((e = launch_train_swiglu(f(Lw.ag), f(Lw.ae), M * F, f(Lw.hh), st)) != hipSuccess) return e;
    if (out) {
      // X_{l+1} = X1 + (M . H) Wd^T
      if ((e = gemm(f(Lw.hh), F, w.w_down, F, out, D, f(Lw.x1), D, F, 0, ms, (int32_t)(F / U))) != hipSuccess)
        return e;
    }
    return hipSuccess;
  }

  // Backward of layer l (its intermediates in the workspace): dX2 = dL/dX_{l+1}
  // in, dX = dL/dX_l out, and the layer's mask gradients into dM.
  hipError_t layer_backward(int32_t l, const float* dX2, float* dX) const {
    const svl_layer_weights& w = W[l];
    const int64_t D = c.d_model, F = c.d_ffn, A = c.n_heads, KV = c.n_kv_heads, d = c.head_dim;
    const float* ms = f(Lw.mfull) + (int64_t)l * U;
    const int64_t mstride = (int64_t)c.n_layers * U;
    const float2* tab = reinterpret_cast<const float2*>(ws + Lw.rope);
    hipError_t e;
    // FFN branch: dHm = dX2 Wd, then SwiGLU (gate / up gradients replace AG / AE)
    if ((e = gemm(dX2, D, w.w_down, F, f(Lw.dh), F, nullptr, F, D, 1, nullptr, 1)) != hipSuccess) return e;
    if ((e = launch_train_swiglu_bwd(f(Lw.dh), f(Lw.ag), f(Lw.ae), f(Lw.hh), ms, mstride,
                                     (int32_t)S, M, (int32_t)F, U, f(Lw.pf), st)) != hipSuccess) return e;
    if ((e = gemm(f(Lw.ag), F, w.w_gate, D, f(Lw.du), D, nullptr, D, F, 1, nullptr, 1)) != hipSuccess) return e;
    if ((e = gemm(f(Lw.ae), F, w.w_up, D, f(Lw.du), D, f(Lw.du), D, F, 1, nullptr, 1)) != hipSuccess) return e;
    if ((e = launch_train_norm_bwd(f(Lw.x1), w.ffn_norm, f(Lw.r2), f(Lw.du), dX2, M, (int32_t)D,
                                   bf16, f(Lw.dx1), st)) != hipSuccess) return e;
    // attention branch: dOm = dX1 Wo, scaled in place by the masks into dO
    float* dO = f(Lw.dO);
    float* dQ = f(Lw.dq);
    if ((e = gemm(f(Lw.dx1), D, w.wo, A * d, dO, A * d, nullptr, A * d, D, 1, nullptr, 1)) != hipSuccess) return e;
    if ((e = launch_train_attn_mask_bwd(dO, f(Lw.o), ms, mstride, (int32_t)S, M, (int32_t)(A * d),
                                        U, f(Lw.pa), st)) != hipSuccess) return e;
    TAttnArgs a = attn_args();
    a.dO = dO;
    a.out = dQ;
    if ((e = launch_train_attn(a, (int32_t)d, B, 1, st)) != hipSuccess) return e;
    a.dK = f(Lw.dk);
    a.dV = f(Lw.dv);
    if ((e = launch_train_attn(a, (int32_t)d, B, 2, st)) != hipSuccess) return e;
    if ((e = launch_train_rope(dQ, A * d, (int32_t)A, (int32_t)d, (int32_t)S, M, tab, -1.f, st)) != hipSuccess) return e;
    if ((e = launch_train_rope(f(Lw.dk), KV * d, (int32_t)KV, (int32_t)d, (int32_t)S, M, tab, -1.f, st)) != hipSuccess) return e;
    if ((e = gemm(dQ, A * d, w.wq, D, f(Lw.du), D, nullptr, D, A * d, 1, nullptr, 1)) != hipSuccess) return e;
    if ((e = gemm(f(Lw.dk), KV * d, w.wk, D, f(Lw.du), D, f(Lw.du), D, KV * d, 1, nullptr, 1)) != hipSuccess) return e;
    if ((e = gemm(f(Lw.dv), KV * d, w.wv, D, f(Lw.du), D, f(Lw.du), D, KV * d, 1, nullptr, 1)) != hipSuccess) return e;
    if ((e = launch_train_norm_bwd(xs(l), w.attn_norm, f(Lw.r1), f(Lw.du), f(Lw.dx1), M,
                                   (int32_t)D, bf16, dX, st)) != hipSuccess) return e;
    return launch_train_mask_reduce(f(Lw.pa), f(Lw.pf), B, (int32_t)S, U, c.n_layers, l, f(Lw.dM), st);
  }
};

}  // namespace
}  // namespace svl

using namespace svl;

extern "C" {

size_t svl_train_workspace_bytes(const svl_config* cfg, const svl_train_params* params,
                                 int32_t batch, int32_t n_vision, int32_t n_text) {
  if (check_train(cfg, params, batch, n_vision, n_text) != SVL_OK) return 0;
  return (size_t)train_layout(*cfg, params->units, batch, n_vision, n_text).total;
}

svl_status svl_train_step(const svl_config* cfg, const svl_layer_weights* layers,
                          const svl_train_params* params, int32_t batch, int32_t n_vision,
                          int32_t n_text, const float* logits, const float* token_noise,
                          const float* gate_logits, const float* gate_noise, const void* vision,
                          const void* text, const float* grad_hidden, float* hidden,
                          uint8_t* token_mask, uint8_t* unit_mask, float* grad_logits,
                          float* grad_gate, void* ws, size_t ws_bytes, void* stream) {
  svl_status s = check_train(cfg, params, batch, n_vision, n_text);
  if (s != SVL_OK) return s;
  const svl_config& c = *cfg;
  const int32_t B = batch, N = n_vision, T = n_text, P = params->prefix, U = params->units;
  const int64_t ngate = (int64_t)B * (c.n_layers - P) * U;
  if (!layers) return err(SVL_E_NULL, "layers is NULL");
  for (int32_t l = 0; l < c.n_layers; ++l) {
    const svl_layer_weights& w = layers[l];
    for (const void* p : {w.attn_norm, w.wq, w.wk, w.wv, w.wo, w.ffn_norm, w.w_gate, w.w_up, w.w_down}) {
      if (!p) return err(SVL_E_NULL, "layer %d: NULL weight pointer", l);
      if (!is_aligned16(p)) return err(SVL_E_ALIGN, "layer %d: weight pointers must be 16-byte aligned", l);
    }
  }
  if (!hidden) return err(SVL_E_NULL, "hidden is NULL");
  if (N > 0 && (!logits || !vision || !token_mask))
    return err(SVL_E_NULL, "logits, vision and token_mask are required when n_vision > 0");
  if (T > 0 && !text) return err(SVL_E_NULL, "text is required when n_text > 0");
  if (ngate > 0 && (!gate_logits || !unit_mask))
    return err(SVL_E_NULL, "gate_logits and unit_mask are required when layers are controlled");
  if (grad_hidden) {
    if (N > 0 && !grad_logits) return err(SVL_E_NULL, "grad_logits is required with grad_hidden");
    if (ngate > 0 && !grad_gate) return err(SVL_E_NULL, "grad_gate is required with grad_hidden");
  }
  for (const void* p : {(const void*)vision, text, (const void*)grad_hidden, (const void*)hidden}) {
    if (p && !is_aligned16(p)) return err(SVL_E_ALIGN, "device pointers must be 16-byte aligned");
  }
  if (!ws) return err(SVL_E_NULL, "workspace is NULL");
  if (!is_aligned16(ws)) return err(SVL_E_ALIGN, "workspace not 16-byte aligned");
  const TrainLayout Lw = train_layout(c, U, B, N, T);
  if ((int64_t)ws_bytes < Lw.total)
    return err(SVL_E_WORKSPACE, "workspace %zu bytes < %lld needed", ws_bytes, (long long)Lw.total);

  const bool bf16 = c.dtype == SVL_BF16;
  const int64_t S = (int64_t)N + T, M = (int64_t)B * S;
  hipStream_t st = static_cast<hipStream_t>(stream);
  TrainRun run{c, layers, B, N, T, P, U, S, M, bf16, static_cast<uint8_t*>(ws), Lw, st};
  hipError_t e;

  TrainMaskArgs ma{};
  ma.z = logits;
  ma.zn = token_noise;
  ma.g = gate_logits;
  ma.gn = gate_noise;
  ma.B = B;
  ma.N = N;
  ma.L = c.n_layers;
  ma.P = P;
  ma.U = U;
  ma.tau_tok = params->tau_tok;
  ma.tau_comp = params->tau_comp;
  ma.tmask = token_mask;
  ma.umask = unit_mask;
  ma.mtok = run.f(Lw.mtok);
  ma.stet = run.f(Lw.stet);
  ma.mfull = run.f(Lw.mfull);
  ma.steg = run.f(Lw.steg);
  if ((e = launch_train_masks(ma, st)) != hipSuccess) return hip_err(e, "masks");
  if ((e = launch_train_embed(vision, text, run.f(Lw.mtok), B, N, T, c.d_model, bf16, run.xs(0),
                              st)) != hipSuccess) return hip_err(e, "embed");
  if ((e = launch_rope_table(reinterpret_cast<float2*>(run.ws + Lw.rope), (int32_t)S, c.head_dim,
                             c.rope_theta, st)) != hipSuccess) return hip_err(e, "rope table");
  for (int32_t l = 0; l < c.n_layers; ++l) {
    float* out = l + 1 < c.n_layers ? run.xs(l + 1) : hidden;
    if ((e = run.layer_forward(l, out)) != hipSuccess) return hip_err(e, "forward");
  }
  if (!grad_hidden) return SVL_OK;

  const float* dcur = grad_hidden;
  float* bufs[2] = {run.f(Lw.dxa), run.f(Lw.dxb)};
  for (int32_t l = c.n_layers - 1; l >= 0; --l) {
    float* dnext = bufs[l & 1];
    if ((e = run.layer_forward(l, nullptr)) != hipSuccess) return hip_err(e, "recompute");
    if ((e = run.layer_backward(l, dcur, dnext)) != hipSuccess) return hip_err(e, "backward");
    dcur = dnext;
  }
  if ((e = launch_train_token_grad(dcur, vision, run.f(Lw.stet), B, N, (int32_t)S, c.d_model, bf16,
                                   grad_logits, st)) != hipSuccess) return hip_err(e, "token gradient");
  if ((e = launch_train_gate_grad(run.f(Lw.dM), run.f(Lw.steg), B, c.n_layers, P, U, grad_gate,
                                  st)) != hipSuccess) return hip_err(e, "gate gradient");
  return SVL_OK;
}

}  // extern "C"
