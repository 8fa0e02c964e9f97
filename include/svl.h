/*
 * svl.h -- C ABI of the budget-adapted MLLM prefill library (libsvl.so) for
 * AMD Instinct MI355X (gfx950).
 *
 * The library runs the inference-time prefill of SmartVL ("Look Less, Think
 * Faster: Joint Token-Compute Adaptation for Multimodal LLMs"): the token
 * controller's per-token scores and an integer keep budget select the vision
 * tokens to keep (Sec. 3.1 and Sec. 3.3 "Inference": the budget projection
 * discards the lowest-confidence tokens first); the kept tokens are packed
 * with the text tokens into one compressed, contiguous sequence per sample
 * (Sec. 3.1); then the LLaMA decoder layers run under the compute
 * controller's masks (Sec. 3.2): a layer with mask 0 is bypassed through its
 * residual, an inactive head contributes nothing, and head group j also gates
 * slice j of the FFN intermediate dimension.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Ownership.  The caller owns every buffer: weights, inputs, outputs and the
 *   workspace.  The library keeps no per-call state and allocates no device
 *   memory in these calls.  Host arrays (keep, masks, cu_seqlens) are read or
 *   written before the call returns.
 * Pointers.  "dev" pointers are HIP device pointers (16-byte aligned);
 *   "host" pointers are ordinary host memory.
 * Streams.  `stream` is a hipStream_t passed as void* (NULL: the null
 *   stream).  All device work is enqueued on it; device outputs are valid once
 *   the stream reaches that point.  No call synchronises the stream, except
 *   svl_count_positive and svl_prefill_controlled (host outputs that the
 *   host plans from) and svl_workspace_status (a host copy of a status
 *   word).
 * Dtypes.  `svl_config.dtype` selects the storage type of weights and of the
 *   vision / text hidden states: SVL_F32 (float) or SVL_BF16 (bfloat16).  The
 *   residual stream `resid` is always float32.  SVL_BF16 runs 16-bit MFMA
 *   matrix products (fp16 or bf16 inputs, see svl_compute) with float32
 *   accumulation.
 * Layouts.  Row-major throughout.  Linear weights use the [out][in] layout
 *   (y = x W^T).  The packed residual holds the samples one after another:
 *   rows cu_seqlens[b] .. cu_seqlens[b+1]-1 are sample b's sequence, kept
 *   vision tokens (ascending original index) followed by its text tokens.
 * Errors.  Every argument is validated before anything is enqueued, so an
 *   error leaves the stream untouched.  A non-zero svl_status is returned and
 *   svl_last_error() gives a message (per thread).  HIP launch errors are
 *   reported as SVL_E_HIP; faults inside kernels surface at the caller's
 *   next synchronisation.
 */
#ifndef SVL_H
#define SVL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SVL_ABI_VERSION 1

typedef enum {
  SVL_OK = 0,
  SVL_E_NULL = 1,       /* a required pointer is NULL */
  SVL_E_SHAPE = 2,      /* inconsistent or unsupported sizes */
  SVL_E_VALUE = 3,      /* a value out of range (keep budget, mask byte not 0/1) */
  SVL_E_WORKSPACE = 4,  /* workspace smaller than svl_workspace_bytes() */
  SVL_E_DTYPE = 5,      /* unknown dtype */
  SVL_E_HIP = 6,        /* HIP runtime error (no device, launch failure) */
  SVL_E_ALIGN = 7       /* a device pointer not 16-byte aligned */
} svl_status;

typedef enum { SVL_F32 = 0, SVL_BF16 = 1 } svl_dtype;

/* Type of the activations between kernels and of the matrix-product inputs
 * when the storage dtype is SVL_BF16 (ignored for SVL_F32, which computes in
 * float32).  SVL_COMPUTE_F16 widens each bf16 weight to fp16 inside the
 * matrix-product kernels (exact for magnitudes in [2^-14, 65504]; smaller
 * ones become fp16 subnormals, absolute error at most 2^-25) and keeps
 * activations in fp16 (11-bit significand): weights and activations must lie
 * inside the fp16 range.  SVL_COMPUTE_BF16 keeps bf16 activations (8-bit
 * significand, full bf16 range) and multiplies them by bf16 MFMA; the
 * RMS-normed rows enter the QKV and gate/up products of a prefill as two
 * bf16 terms, hi = bf16(x) and lo = bf16(x - hi), both multiplied by the
 * same weights (about 16 significant bits for those operands; twice the
 * products, and a workspace plane of the low terms).  Decode steps take the
 * hi terms only.  Both modes accumulate in float32 and keep the residual
 * stream in float32. */
typedef enum { SVL_COMPUTE_F16 = 0, SVL_COMPUTE_BF16 = 1 } svl_compute;

/* Decoder shape (LLaMA block: pre-RMSNorm, rotate-half RoPE, causal
 * attention with n_kv_heads K/V heads shared by n_heads/n_kv_heads query
 * heads each, SwiGLU FFN, no biases).  n_groups is the number of head
 * groups G of the layer-head controller (Sec. 3.2); FFN slice j is the
 * channel range [j*d_ffn/G, (j+1)*d_ffn/G).
 * Requirements: all sizes > 0; n_heads % n_kv_heads == 0; head_dim even;
 * d_ffn % n_groups == 0; for SVL_BF16 also d_model % 64 == 0,
 * head_dim in {64, 128}, d_ffn/n_groups % 64 == 0, d_model, d_ffn and
 * n_heads*head_dim at most 65536, and every weight matrix under 2 GiB
 * (SVL_E_SHAPE otherwise). */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ffn, n_groups;
  float rms_eps;     /* RMSNorm epsilon */
  float rope_theta;  /* RoPE base: pair (r, r+d/2) turns by p * theta^(-2r/d) */
  int32_t dtype;     /* svl_dtype: storage of weights and hidden inputs */
  int32_t compute;   /* svl_compute (SVL_BF16 storage only; 0 = SVL_COMPUTE_F16) */
} svl_config;

/* One layer's weights (dev, config dtype).  Shapes:
 *   attn_norm, ffn_norm [D];  wq [A*d][D];  wk, wv [KV*d][D];  wo [D][A*d];
 *   w_gate, w_up [F][D];  w_down [D][F]. */
typedef struct {
  const void *attn_norm, *wq, *wk, *wv, *wo, *ffn_norm, *w_gate, *w_up, *w_down;
} svl_layer_weights;

/* Batch description: B samples, each with n_vision scored vision tokens and
 * n_text text tokens; keep (host [B]) is each sample's keep budget k_b in
 * [0, n_vision].  Sample b's sequence length is S_b = k_b + n_text. */
typedef struct {
  int32_t batch, n_vision, n_text;
  const int32_t *keep;
} svl_batch;

/* Executed FLOPs (2 per multiply-add, matrix products only), by component:
 * q: query projection; kv: key and value projections; o: output projection;
 * attn: causal scores and probability-value products; ffn: gate, up, down. */
typedef struct {
  uint64_t q, kv, o, attn, ffn, total;
} svl_flops;

/* Token selection and packing (Sec. 3.1; Sec. 3.3 budget projection).
 * For each sample b: keeps the keep[b] highest scores of scores[b][:]
 * (ordering: larger score first, NaN below every number, -0 equal to +0,
 * equal scores -> lower index first), writes the kept indices in ascending
 * order to kept_idx[b][0..k_b) and -1 to kept_idx[b][k_b..N), and packs
 * [vision[b][kept] ; text[b]] into resid rows cu_seqlens[b]..cu_seqlens[b+1].
 *   scores   dev  float  [B][N]
 *   vision   dev  dtype  [B][N][D]
 *   text     dev  dtype  [B][T][D]
 *   kept_idx dev  int32  [B][N]       (out)
 *   resid    dev  float  [sum S_b][D] (out, widened exactly from dtype)
 *   cu_seqlens host int32 [B+1]       (out; cu_seqlens[0] = 0)
 *   ws/ws_bytes: workspace of at least svl_workspace_bytes(cfg, B, sum S_b). */
svl_status svl_select_tokens(const svl_config *cfg, const svl_batch *batch,
                             const float *scores, const void *vision, const void *text,
                             int32_t *kept_idx, float *resid, int32_t *cu_seqlens,
                             void *ws, size_t ws_bytes, void *stream);

/* One decoder layer on a packed residual (Sec. 3.2), in place.
 *   layer      index of the layer (informational; weights are passed directly)
 *   cu_seqlens host int32 [batch+1]: the packed rows of each sample
 *   layer_on   host uint8 [batch]: 0 = the layer is bypassed for the sample
 *   head_mask  host uint8 [batch][A]: query-head gates (0/1); a K/V head is
 *              computed iff one of its query heads is active
 *   ffn_mask   host uint8 [batch][G] or NULL (FFN ungated): FFN slice gates
 *   resid      dev float [cu_seqlens[batch]][D], updated in place
 * Positions for RoPE are 0..S_b-1 within each sample.  Rows of samples with
 * layer_on = 0 are not read or written. */
svl_status svl_layer_forward(const svl_config *cfg, int32_t layer, const svl_layer_weights *w,
                             int32_t batch, const int32_t *cu_seqlens, const uint8_t *layer_on,
                             const uint8_t *head_mask, const uint8_t *ffn_mask, float *resid,
                             void *ws, size_t ws_bytes, void *stream);

/* The whole budget-adapted prefill: svl_select_tokens followed by every
 * layer under the masks (Eq. (1) with the allocation given).
 *   layers     host array of cfg->n_layers svl_layer_weights
 *   layer_mask host uint8 [B][L];  head_mask host uint8 [B][L][A];
 *   ffn_mask   host uint8 [B][L][G] or NULL
 *   kept_idx, resid, cu_seqlens: as svl_select_tokens; resid holds the
 *   residual stream after the last layer (no final norm, no LM head)
 *   flops      host, may be NULL: executed FLOPs (same as svl_count_flops) */
svl_status svl_prefill(const svl_config *cfg, const svl_layer_weights *layers,
                       const svl_batch *batch, const float *scores, const void *vision,
                       const void *text, const uint8_t *layer_mask, const uint8_t *head_mask,
                       const uint8_t *ffn_mask, int32_t *kept_idx, float *resid,
                       int32_t *cu_seqlens, svl_flops *flops, void *ws, size_t ws_bytes,
                       void *stream);

/* Workspace bytes any of the calls above needs for `batch` samples and at
 * most `total_rows` packed rows (sum of S_b), for any masks.  0 on bad args. */
size_t svl_workspace_bytes(const svl_config *cfg, int32_t batch, int32_t total_rows);

/* Executed FLOPs for the given sequence lengths (host [B]) and masks, in
 * closed form (host only, no device work; only the shape rules that do
 * not depend on the kernels apply).  Per executed (sample, layer) with
 * H active query heads, K active K/V heads, C active FFN channels:
 *   q = 2 S D d H, kv = 4 S D d K, o = 2 S H d D, attn = 2 H d S (S+1),
 *   ffn = 6 S D C.
 * The paper's estimator Eq. (8) charges 4 D S^2 for a full score matrix; the
 * causal products charge only the triangle. */
svl_status svl_count_flops(const svl_config *cfg, int32_t batch, const int32_t *seqlens,
                           const uint8_t *layer_mask, const uint8_t *head_mask,
                           const uint8_t *ffn_mask, svl_flops *out);

/* ---- threshold selection and budget projection -------------------------
 * At inference the token controller keeps visual token i iff
 * sigma(z_i) > 0.5, i.e. iff its logit z_i > 0 (Sec. 3.1), and for a budget
 * b < 1 a deterministic projection brings the estimated prefill cost of
 * Eq. (8) within b * C_full, discarding the lowest-confidence visual tokens
 * first and reducing layers / heads only when that is not enough (Sec. 3.3
 * "Inference").  The two calls below give the keep counts and the masks that
 * svl_prefill then runs with, the logits serving as its scores (the kept
 * tokens are the keep[b] largest logits, which are all positive). */

/* Threshold counts: counts[b] = number of i with logits[b][i] > 0 (zero, -0
 * and NaN do not count).
 *   logits  dev float [batch][n_vision]
 *   counts  host int32 [batch] (out)
 *   ws/ws_bytes: device workspace of at least 4 * batch bytes.
 * Unlike the other calls, this one synchronises `stream`: the counts come
 * back to the host, which plans the prefill from them. */
svl_status svl_count_positive(int32_t batch, int32_t n_vision, const float *logits,
                              int32_t *counts, void *ws, size_t ws_bytes, void *stream);

/* Budget projection, host only (no device work).  Per sample, with S =
 * n_text + s, alpha_l = (active query heads of layer l) / A (0 for a skipped
 * layer) and
 *   C(s) = sum_l alpha_l [(8 D^2 + 6 D F) S + 4 D S^2] + 2 D V S    (Eq. (8)),
 * C_full = C with every alpha_l = 1 and s = n_vision:
 *   budget >= 1: keep[b] = counts[b], masks unchanged;
 *   otherwise keep[b] = the largest s <= counts[b] with C(s) <= budget * C_full;
 *   if even s = 0 does not fit, whole head groups (heads [j A/G, (j+1) A/G)
 *   and FFN slice j) of layers l >= prefix are switched off one at a time,
 *   lowest gate logit first (ties: the later layer, then the higher group;
 *   without gate logits: the later layer first, then the higher group), a
 *   layer left with no active head is skipped, until s = 0 fits, and keep[b]
 *   is then the largest s that fits with the reduced masks; if every
 *   eligible group is off and s = 0 still does not fit, keep[b] = 0.
 * C(s) <= budget * C_full is decided exactly (budget at its exact float
 * value, costs in integer arithmetic).
 *   counts      host int32 [batch]: threshold counts, each in [0, n_vision]
 *   budget      target fraction of C_full; finite and > 0 (else SVL_E_VALUE)
 *   vocab       V of the LM-head term, >= 0 (0 leaves the term out)
 *   prefix      P: layers 0..P-1 are never reduced, 0 <= P <= n_layers
 *   layer_mask  host uint8 [batch][L] (in/out); head_mask host uint8
 *               [batch][L][A] (in/out); ffn_mask host uint8 [batch][L][G]
 *               (in/out) or NULL (FFN ungated)
 *   gate_logits host float [batch][L][G] or NULL: the compute controller's
 *               group logits (finite)
 *   keep        host int32 [batch] (out) */
svl_status svl_budget_project(const svl_config *cfg, int32_t batch, int32_t n_vision,
                              int32_t n_text, const int32_t *counts, float budget, int64_t vocab,
                              int32_t prefix, uint8_t *layer_mask, uint8_t *head_mask,
                              uint8_t *ffn_mask, const float *gate_logits, int32_t *keep);

/* ---- compute controller and the controlled prefill ----------------------
 * The LLM-side compute controller (Sec. 3.2) decides, per sample, which
 * layers and head groups run after the P prefix layers:
 *   e_b = MLP_LLM(PE(b)), the budget token, is appended after the text
 *   tokens and runs through the prefix layers with the rest of the sequence;
 *   kappa = sum_i sigma(z_i) / N, the soft survival rate of the visual
 *   tokens, is encoded and added to the budget token's state after the
 *   prefix: h~ = h_b^(P) + MLP_kappa(PE(kappa)) (Eq. (7));
 *   the gating head's logits W_h h~ + c_h switch a unit on iff > 0 (sigma >
 *   0.5, Gumbel noise removed at inference).  Layer-head controller: one
 *   unit per (dynamic layer, head group j), gating heads [j A/G, (j+1) A/G)
 *   and FFN slice j, a layer with every group off is skipped; layer
 *   controller: one unit per dynamic layer (full capacity or bypassed).
 * PE(x) of width E: entry 2i = sin(x s w_i), entry 2i+1 = cos(x s w_i),
 * w_i = base^(-2i/E), s = pe_scale.  MLP: Linear(E -> H) + bias, GELU
 * (erf form), Linear(H -> D) + bias.  The controller's products run in
 * float32 (weights widened from the storage dtype); the encodings and
 * kappa in float64. */
typedef struct {
  int32_t prefix;     /* P: layers 0..P-1 run at full capacity, 0 <= P < n_layers */
  int32_t units;      /* gates per dynamic layer: n_groups (layer-head) or 1 (layer) */
  int32_t pe_dim;     /* E: encoding width, a multiple of 8 in [8, 65536] */
  int32_t hidden;     /* H: hidden width of both MLPs, a multiple of 8 in [8, 65536] */
  float pe_scale;     /* s: the encoded scalar is multiplied by s (finite) */
  float pe_base;      /* frequency base (finite, > 0; 10000 in the Transformer encoding) */
  /* dev, config dtype, [out][in] rows 16-byte aligned:
   *   llm_w1, kap_w1 [H][E];  llm_b1, kap_b1 [H];  llm_w2, kap_w2 [D][H];
   *   llm_b2, kap_b2 [D];  gate_w [(L-P)*units][D];  gate_b [(L-P)*units]. */
  const void *llm_w1, *llm_b1, *llm_w2, *llm_b2;
  const void *kap_w1, *kap_b1, *kap_w2, *kap_b2;
  const void *gate_w, *gate_b;
} svl_controller;

/* Workspace bytes of svl_prefill_controlled (0 on bad arguments). */
size_t svl_controlled_workspace_bytes(const svl_config *cfg, const svl_controller *ctrl,
                                      int32_t batch, int32_t n_vision, int32_t n_text);

/* The controlled prefill (Sec. 3.1-3.3 at inference), per sample b:
 *   1. threshold selection: the visual tokens with logits[b][i] > 0 (their
 *      count c_b) in ascending index order, then the text tokens, then the
 *      budget token: c_b + n_text + 1 rows;
 *   2. layers 0..P-1 at full capacity;
 *   3. the controller's gate logits and masks (above);
 *   4. budget < 1: the budget projection of svl_budget_project (counts c_b,
 *      the controller's masks, its gate logits as the confidence order, with
 *      units = whole layers for the layer controller); the visual tokens it
 *      discards (the lowest logits) leave the sequence here, the remaining
 *      rows keep their order and are numbered 0..S'-1 for RoPE from layer P
 *      on (Eq. (8)'s S counts text and visual tokens, not the budget token);
 *   5. layers P..L-1 under the final masks.
 * Arguments:
 *   logits     dev float [B][N]: the token controller's logits z
 *   vision     dev dtype [B][N][D];  text dev dtype [B][T][D]
 *   budget     b, finite and > 0 (>= 1: no projection); vocab: V of Eq. (8)
 *   kept_idx   dev int32 [B][N] (out): final kept tokens ascending, rest -1
 *   resid      dev float, room for B*(N+T+1) rows (out): the final packed
 *              sequences [kept vision ; text ; budget token] after layer L-1
 *   cu_seqlens host int32 [B+1] (out) of the final sequences
 *   keep       host int32 [B] (out): final visual tokens per sample
 *   layer_mask host uint8 [B][L], head_mask [B][L][A], ffn_mask [B][L][G]
 *              (out): the masks the layers ran with
 *   gate_logits host float [B][(L-P)*units] (out, may be NULL): the raw
 *              gate logits, layer-major
 *   flops      host (out, may be NULL): executed layer FLOPs (the prefix
 *              layers at the threshold lengths, the others at the final ones)
 *   ws/ws_bytes: at least svl_controlled_workspace_bytes(...).
 * Like svl_count_positive, this call synchronises `stream` twice: after
 * the threshold counts and after the gate logits, which the host needs to
 * plan the launches.  An error found after the first synchronisation (a HIP
 * error) leaves the outputs undefined. */
svl_status svl_prefill_controlled(const svl_config *cfg, const svl_layer_weights *layers,
                                  const svl_controller *ctrl, int32_t batch, int32_t n_vision,
                                  int32_t n_text, float budget, int64_t vocab,
                                  const float *logits, const void *vision, const void *text,
                                  int32_t *kept_idx, float *resid, int32_t *cu_seqlens,
                                  int32_t *keep, uint8_t *layer_mask, uint8_t *head_mask,
                                  uint8_t *ffn_mask, float *gate_logits, svl_flops *flops,
                                  void *ws, size_t ws_bytes, void *stream);

/* ---- training-time budget term -------------------------------------------
 * During training the controllers' decisions are Gumbel-sigmoid
 * straight-through masks (Eq. (6)): y = sigma((z + xi) / tau), mask =
 * 1[y > 0.5] in the forward pass, dy/dz in the backward pass.  The budget
 * term (Sec. 3.3) prices them with Eq. (8) at the soft visual count
 * S~ = sum_i sigma(z_i) (S = n_text + S~) and the layer activities
 * alpha_l = (units on) / U of the unit masks (prefix layers at 1):
 *   r = C^ / C_full,
 *   loss = lambda_t (w_over max(0, r - b)^2 + w_under max(0, (b - margin) - r))
 * (Eq. (9), the budget part of Eq. (10)).  svl_budget_loss gives, per sample,
 * the forward masks, r, the loss and its gradient with respect to the token
 * logits (through S~; the token masks act on the prediction loss only) and
 * to the gate logits (straight-through: dalpha_l/dg = (1/U) y (1 - y) /
 * tau_comp).  The hinge's derivative at its kink is taken as 0.  Sums run in
 * float64; outputs are float32. */
typedef struct {
  float budget;      /* b, finite and > 0 */
  float margin;      /* mu >= 0: zero-loss band [b - mu, b] */
  float w_over, w_under;  /* >= 0 */
  float lambda_t;    /* warm-up factor lambda(t) = min(1, t / T_warmup), >= 0 */
  float tau_tok;     /* token temperature (> 0; the decision z + xi > 0 does not depend on it) */
  float tau_comp;    /* compute temperature (> 0) */
  int32_t prefix;    /* P, 0 <= P < n_layers */
  int32_t units;     /* n_groups (layer-head controller) or 1 (layer controller) */
  int64_t vocab;     /* V of Eq. (8), >= 0 */
} svl_budget_loss_params;

/* Per sample b (all pointers dev):
 *   logits      float [B][N]: token logits z;  token_noise float [B][N] or NULL
 *   gate_logits float [B][(L-P) units];  gate_noise same or NULL
 *   token_mask  uint8 [B][N] (out): 1 iff z + xi > 0
 *   unit_mask   uint8 [B][(L-P) units] (out): 1 iff g + xi > 0
 *   ratio, loss float [B] (out);  grad_logits float [B][N] (out): dloss/dz;
 *   grad_gate   float [B][(L-P) units] (out): dloss/dg.
 * n_vision + n_text > 0.  Enqueued on `stream`; no workspace. */
svl_status svl_budget_loss(const svl_config *cfg, const svl_budget_loss_params *params,
                           int32_t batch, int32_t n_vision, int32_t n_text,
                           const float *logits, const float *token_noise,
                           const float *gate_logits, const float *gate_noise,
                           uint8_t *token_mask, uint8_t *unit_mask, float *ratio, float *loss,
                           float *grad_logits, float *grad_gate, void *stream);

/* ---- status of the last prefill on a workspace ---------------------------
 * With fp16 activations (SVL_COMPUTE_F16) a value outside fp16's range
 * becomes inf when it is converted, and the inf (or the NaN it produces)
 * reaches the output rows; the call itself still returns SVL_OK.  At its
 * end every svl_prefill, svl_prefill_cache and svl_prefill_controlled clears
 * a status word in the last four bytes of its workspace buffer
 * (ws + (ws_bytes & ~3) - 4) and sets it to SVL_STATUS_NONFINITE if any of
 * its output values (resid rows 0 .. sum S_b - 1, S_b the final lengths) is
 * inf or NaN, whatever the cause (fp16 overflow, or
 * non-finite inputs or weights).  svl_workspace_status copies that word to
 * *status (host) once `stream` has reached it: it synchronises the stream.
 * After other calls on the same buffer the word is undefined.
 * Errors: SVL_E_NULL (ws or status NULL), SVL_E_ALIGN, SVL_E_WORKSPACE
 * (ws_bytes < 256), SVL_E_HIP. */
#define SVL_STATUS_NONFINITE 1u
svl_status svl_workspace_status(const void *ws, size_t ws_bytes, uint32_t *status, void *stream);

/* ---- training-time masked decoder ----------------------------------------
 * The prediction side of a training step (Sec. 3.1 Eq. (6); Sec. 3.2).  The
 * sequences keep their length: sample b is S = N + T rows, its N vision
 * embeddings each multiplied by the forward value of its straight-through
 * token mask m_i = 1[z_i + xi_i > 0] (a dropped token becomes a zero row),
 * then its T text embeddings, at positions 0..S-1.  Every decoder layer
 * computes every head and every FFN channel; in the controlled layers
 * l >= P, unit u's mask M_lu = 1[g_lu + xi_lu > 0] multiplies the attention
 * output of the heads of group u (heads [u A/U, (u+1) A/U)) before the output
 * projection and the SwiGLU output of FFN slice u (channels [u F/U,
 * (u+1) F/U)) before the down projection.  U = n_groups is the layer-head
 * controller; U = 1 is the layer controller (M_l = 0 makes layer l the
 * identity).  Layers 0..P-1 run with every mask at 1.
 *
 * Given an upstream gradient G of the final hidden states (the prediction
 * loss, outside the library, as dL/dX_L), the call runs the backward of that
 * decoder, with the masks treated as numbers, and applies the straight-
 * through estimator:
 *   dL/dz_i  = (sum_d dL/dX0[i][d] v_i[d]) y_i (1 - y_i) / tau_tok,
 *   dL/dg_lu = dL/dM_lu y_lu (1 - y_lu) / tau_comp,
 * with y = sigma((logit + xi) / tau).  The budget term's gradient
 * (svl_budget_loss) is separate; the total gradient is the sum.
 *
 * Arithmetic: float32 throughout (weights and embeddings widened exactly
 * from the storage dtype; svl_config.compute is ignored); the forward of each
 * layer is recomputed from its stored input during the backward.
 * Requirements beyond the config's: head_dim in {32, 64, 128}; d_model and
 * d_ffn multiples of 16; n_heads and d_ffn divisible by units, d_ffn / units
 * a multiple of 4 (SVL_E_SHAPE otherwise). */
typedef struct {
  float tau_tok;     /* token temperature, finite and > 0 */
  float tau_comp;    /* compute temperature, finite and > 0 */
  int32_t prefix;    /* P, 0 <= P <= n_layers */
  int32_t units;     /* U >= 1 */
} svl_train_params;

/* Workspace bytes of svl_train_step for `batch` samples of n_vision + n_text
 * rows (0 on bad arguments): the input of every layer, one layer's forward
 * intermediates and its gradients, all float32. */
size_t svl_train_workspace_bytes(const svl_config *cfg, const svl_train_params *params,
                                 int32_t batch, int32_t n_vision, int32_t n_text);

/* One training step of the masked decoder (all pointers dev, row-major):
 *   logits       float [B][N] token logits z;  token_noise float [B][N] or NULL
 *   gate_logits  float [B][(L-P) U] (layer-major);  gate_noise same or NULL
 *   vision       dtype [B][N][D];  text dtype [B][T][D]
 *   grad_hidden  float [B][S][D]: dL/dX_L, or NULL for the forward only
 *   hidden       float [B][S][D] (out): X_L
 *   token_mask   uint8 [B][N] (out);  unit_mask uint8 [B][(L-P) U] (out)
 *   grad_logits  float [B][N] (out, when grad_hidden is given)
 *   grad_gate    float [B][(L-P) U] (out, when grad_hidden is given)
 *   ws/ws_bytes: at least svl_train_workspace_bytes(...).
 * Arrays with no elements (N = 0, or (L-P) U = 0) may be NULL.  Enqueued on
 * `stream`; nothing is synchronised. */
svl_status svl_train_step(const svl_config *cfg, const svl_layer_weights *layers,
                          const svl_train_params *params, int32_t batch, int32_t n_vision,
                          int32_t n_text, const float *logits, const float *token_noise,
                          const float *gate_logits, const float *gate_noise, const void *vision,
                          const void *text, const float *grad_hidden, float *hidden,
                          uint8_t *token_mask, uint8_t *unit_mask, float *grad_logits,
                          float *grad_gate, void *ws, size_t ws_bytes, void *stream);

/* ---- decode on the pruned and gated KV cache ----------------------------
 * After the prefill, tokens are generated one at a time; the paper leaves
 * this stage to future work (Sec. 5).  The cache holds only what the prefill
 * computed: the kept tokens' rows (the compressed sequence of Sec. 3.1) and,
 * per layer, only the active K/V heads of samples that run the layer
 * (Sec. 3.2).  A decode step runs the same decoder, under the sample's same
 * masks, on one new token per sample at position p = the sample's cached
 * length: its queries attend to the cached keys / values of positions 0..p-1
 * and to its own.  Its result equals the last row of a prefill over the
 * sequence extended by that token (causal attention).  16-bit path only
 * (SVL_BF16 storage; SVL_E_DTYPE otherwise).
 *
 * Cache layout (dev, activation type: fp16, or bf16 with SVL_COMPUTE_BF16):
 *   [n_layers][batch][n_kv_heads][2 (K, V)][max_len][head_dim], K rotated
 *   (RoPE at its position).  Entries of skipped layers and inactive heads
 *   are neither written nor read. */

/* Bytes of a cache for `batch` samples of up to `max_len` positions (0 on bad
 * arguments; max_len <= 32768). */
size_t svl_kv_cache_bytes(const svl_config *cfg, int32_t batch, int32_t max_len);

/* The whole prefill (as svl_prefill) that also writes every layer's K / V of
 * the executed rows into the cache at positions 0..S_b-1.  max_len >= every
 * S_b (else SVL_E_SHAPE). */
svl_status svl_prefill_cache(const svl_config *cfg, const svl_layer_weights *layers,
                             const svl_batch *batch, const float *scores, const void *vision,
                             const void *text, const uint8_t *layer_mask,
                             const uint8_t *head_mask, const uint8_t *ffn_mask,
                             int32_t *kept_idx, float *resid, int32_t *cu_seqlens,
                             void *kv_cache, int32_t max_len, void *ws, size_t ws_bytes,
                             void *stream);

/* Workspace bytes of svl_decode_step for `batch` samples and caches of up to
 * `max_len` positions (0 on bad arguments). */
size_t svl_decode_workspace_bytes(const svl_config *cfg, int32_t batch, int32_t max_len);

/* One decode step: sample b's new token at position cache_len[b].
 *   layers     host array of cfg->n_layers svl_layer_weights
 *   x          dev float [batch][D]: the new tokens' hidden states in, their
 *              residual after the last layer out (no final norm, no LM head)
 *   cache_len  host int32 [batch]: positions already cached, each < max_len;
 *              the step writes position cache_len[b] of every executed layer
 *              (the caller then advances cache_len)
 *   layer_mask, head_mask, ffn_mask: as svl_prefill (the sample's masks)
 *   kv_cache, max_len: as svl_prefill_cache
 *   ws/ws_bytes: at least svl_decode_workspace_bytes(cfg, batch, max_len). */
svl_status svl_decode_step(const svl_config *cfg, const svl_layer_weights *layers,
                           int32_t batch, float *x, const int32_t *cache_len,
                           const uint8_t *layer_mask, const uint8_t *head_mask,
                           const uint8_t *ffn_mask, void *kv_cache, int32_t max_len,
                           void *ws, size_t ws_bytes, void *stream);

/* Allocation-free decode step, for callers that cannot allocate device
 * memory between steps (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same computation, kernels and
 * results as svl_decode_step, with its workspace taken from a device array
 * of SVL_NOALLOC_SCRATCH_BYTES inside the library instead of a caller
 * buffer.  Arguments as svl_decode_step without ws / ws_bytes.
 *   - Calls no hipMalloc, hipFree or other allocating routine; the step's
 *     plan is copied from host memory with an ordinary stream copy.
 *   - The array exists once per GPU the library runs on and is held until
 *     the process ends.  Its device address on the current GPU is looked up
 *     on the first call there.
 *   - Every call on one GPU uses that GPU's array and leaves the last call's
 *     contents in it (nothing in it needs to start at zero): calls that
 *     overlap on one GPU (several host threads or streams) race and must be
 *     serialised by the caller.
 *   - A shape whose decode workspace (svl_decode_workspace_bytes) exceeds
 *     the array returns SVL_E_WORKSPACE before anything is enqueued. */
#define SVL_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
svl_status svl_decode_step_noalloc(const svl_config *cfg, const svl_layer_weights *layers,
                                   int32_t batch, float *x, const int32_t *cache_len,
                                   const uint8_t *layer_mask, const uint8_t *head_mask,
                                   const uint8_t *ffn_mask, void *kv_cache, int32_t max_len,
                                   void *stream);

/* Message for the last non-OK status returned on this thread. */
const char *svl_last_error(void);

/* SVL_ABI_VERSION of the built library. */
int32_t svl_abi_version(void);

/* ---- kernel timing (instrumentation for benchmarks) ----------------------
 * With timing on, every launch is bracketed by two hipEvents recorded on the
 * launch's stream; svl_timing_read() waits for the recorded events and
 * returns the summed kernel time (ms) and launch count of one kernel class,
 * then forgets them.  Timing adds event records between launches, so time
 * whole calls with timing off.
 * Kernel classes: 0 select, 1 gather, 2 rmsnorm, 3 qkv gemm, 4 attention
 * (prefill and decode), 5 o-proj gemm, 6 gate/up gemm, 7 down gemm, 8 rope
 * table, 9 split-K finish (QKV and gate/up launches whose K was split),
 * 10 KV-cache append, 11 compute controller (statistics, encodings, its
 * matrix-vector products, budget rows and row compaction) and the
 * training-time budget term. */
#define SVL_KCLASS_COUNT 12
svl_status svl_timing_enable(int32_t on);
svl_status svl_timing_read(int32_t kernel_class, double *total_ms, int64_t *launches);

#ifdef __cplusplus
}
#endif
#endif /* SVL_H */
