/*
 * phyai.h -- C ABI of the MI355X (gfx950) action-expert denoising library.
 *
 * The library runs the flow-matching action-expert loop of a pi0-style
 * vision-language-action policy (PhyAI, arXiv 2608.03682): a request's
 * action chunk x (H actions of A values) starts as noise and is refined by K
 * Euler steps, x <- x + (t_{k+1} - t_k) * v(x, t_k), where v is an L-layer
 * transformer over the action tokens that attends to a frozen prefix K/V
 * cache from the vision-language model (Section "Embodied Task Formulation",
 * "From Observation to Action"; Section "PhyAI Architecture", paragraphs
 * "Graph replay" and "Profiled operator selection").  The prefix state is
 * valid for one chunk: it is read, never written, and stays fixed across
 * the K steps.  Requests in a batch are independent (Section "Cloud
 * Batching").  The same library also runs the step before the loop: the
 * vision-language model's language part over the prefix tokens, which
 * produces that prefix K/V cache (phyai_prefill, on a handle of variant
 * PHYAI_VARIANT_PREFIX_LM), and the vision tower before it, which turns the
 * camera images into the image tokens at the head of that prefix
 * (phyai_encode_images, variant PHYAI_VARIANT_VISION).
 *
 * Every step runs in hand-written HIP kernels; the K-step loop is captured
 * in a HIP graph per (batch, steps) bucket and replayed.
 *
 * Conventions for every entry point:
 *   - Pointers documented "device" must be device memory of the current HIP
 *     device; "host" pointers are read before the call returns.
 *   - Arguments are validated on the host before anything is enqueued; a
 *     failing call enqueues nothing and leaves outputs untouched.
 *   - Return value: PHYAI_OK or a negative phyai_status; the text of the last
 *     error on the calling thread is returned by phyai_last_error().
 *   - A handle is not thread-safe: at most one call in flight per handle.
 *   - "stream" is a hipStream_t passed as void* (NULL = the null stream).
 */
#ifndef PHYAI_H
#define PHYAI_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PHYAI_OK = 0,
  PHYAI_EINVAL = -1,        /* bad argument, shape or missing tensor       */
  PHYAI_ENOMEM = -2,        /* device or host allocation failed            */
  PHYAI_EHIP = -3,          /* a HIP runtime call failed                   */
  PHYAI_EUNSUPPORTED = -4   /* valid but not implemented (shape, dtype)    */
} phyai_status;

typedef enum {
  PHYAI_VARIANT_PI0 = 0,    /* time mixed into action tokens by a 2-layer MLP; optional state token */
  PHYAI_VARIANT_PI05 = 1,   /* adaRMSNorm timestep conditioning in every norm                      */
  PHYAI_VARIANT_DIT = 2,    /* DiT head: adaLN-zero, alternating cross/self attention              */
  PHYAI_VARIANT_PREFIX_LM = 3, /* the VLM's language part over the prefix tokens, producing the prefix
                                  K/V cache the pi0 / pi0.5 experts read (see phyai_prefill)        */
  PHYAI_VARIANT_VISION = 4     /* the VLM's vision tower: image patches to the image tokens that open
                                  the prefix (see phyai_encode_images)                              */
} phyai_variant;

typedef enum {
  PHYAI_DTYPE_F32 = 0,
  PHYAI_DTYPE_BF16 = 1,     /* uint16 bit patterns of bfloat16                                     */
  PHYAI_DTYPE_FP8E4M3 = 2,  /* uint8 OCP e4m3fn codes with one float32 scale per output column     */
  PHYAI_DTYPE_FP4E2M1 = 3   /* 4-bit weights: OCP e2m1 codes, two per byte, with one power-of-two
                               float32 scale per group of 32 input rows and output column          */
} phyai_dtype;

/* Shape of one expert.  Derived sizes: M = horizon + state_token suffix
 * tokens per request.  weight_dtype F32 selects the fp32 path (all compute
 * in fp32); BF16, FP8E4M3 and FP4E2M1 select the bf16 MFMA path (fp32
 * accumulate, fp32 residual stream, norms, softmax and solver state).
 * FP4E2M1 is the 4-bit weight, 16-bit activation (W4A16) path of Section
 * "PhyAI Architecture", paragraph "Quantization": its GEMMs decode the
 * codes to bf16 on the fly and run the small-row kernels at every batch
 * size (it is meant for weight-streaming batches). */
typedef struct {
  int32_t variant;          /* phyai_variant                                                      */
  int32_t n_layers;         /* L                                                                  */
  int32_t d_model;          /* d (multiple of 256, at most 2048)                                  */
  int32_t n_q_heads;        /* query heads                                                        */
  int32_t n_kv_heads;       /* key/value heads (1 for MQA)                                        */
  int32_t head_dim;         /* 64, 128 or 256                                                     */
  int32_t d_mlp;            /* MLP width F (multiple of 64)                                       */
  int32_t horizon;          /* H action tokens per chunk                                          */
  int32_t action_dim;       /* A values per action (<= 64)                                        */
  int32_t max_steps;        /* largest K accepted by phyai_denoise                                */
  int32_t prefix_cap;       /* P_cap: prefix rows reserved per request in the prefix buffer        */
  int32_t max_batch;        /* largest B accepted by phyai_denoise                                */
  int32_t state_token;      /* 1: one state token is prepended (needs `state`)                   */
  int32_t rope;             /* 1: RoPE on suffix queries/keys at positions prefix_len + i          */
  int32_t weight_dtype;     /* phyai_dtype of the per-layer trunk linears                         */
  int32_t kv_dtype;         /* phyai_dtype of the prefix buffer (F32 or BF16)                     */
  int32_t d_feat;           /* DiT: width of the VLM feature tokens; 0 otherwise                  */
  int32_t time_dim;         /* width of the sinusoidal timestep embedding                         */
  float rms_eps;            /* norm epsilon (1e-6)                                                */
  float sin_min_period;     /* sinusoid periods run geometrically from min to max                 */
  float sin_max_period;
  float rope_base;          /* 10000                                                              */
  int32_t n_images;         /* VISION: images per request; 0 otherwise                           */
  int32_t n_patches;        /* VISION: patches (tokens) per image                                 */
  int32_t patch_dim;        /* VISION: values per patch (multiple of 64)                          */
  int32_t d_out;            /* VISION: width of the projected image tokens (multiple of 32)       */
} phyai_config;

/* PHYAI_VARIANT_PREFIX_LM uses n_layers, d_model, n_q_heads, n_kv_heads,
 * head_dim, d_mlp, prefix_cap (rows per request: the prefix tokens),
 * max_batch, rope (RoPE on queries and keys at positions 0 .. prefix_len-1),
 * weight_dtype, kv_dtype, rms_eps and rope_base; horizon, action_dim,
 * max_steps, time_dim and the sinusoid periods are ignored, state_token and
 * d_feat must be 0, prefix_cap >= 1.  Its blocks are the pi0 trunk's
 * (RMSNorm with gain (1 + w), fused QKV, GeGLU MLP, residual adds) with a
 * bidirectional mask over the valid prefix tokens.
 *
 * PHYAI_VARIANT_VISION uses n_layers, d_model, n_q_heads = n_kv_heads,
 * head_dim, d_mlp, max_batch (requests; max_batch * n_images <= 512),
 * weight_dtype, kv_dtype, rms_eps (the LayerNorm epsilon), n_images,
 * n_patches, patch_dim and d_out; rope, state_token and d_feat must be 0 and
 * the other fields are ignored.  Its blocks are a pre-norm vision
 * transformer's (LayerNorm with gain (1 + w) and bias, multi-head attention
 * with biased projections over the patches of one image, GELU MLP with
 * biases, residual adds), after a linear patch embedding plus a learned
 * position embedding and before a final LayerNorm and a linear projector to
 * d_out. */

/* One named parameter, stored [rows][cols] row-major on the host.  Linear
 * weights are [in][out] (y = x W + b); vectors have rows = 1.  dtype must be
 * the config's weight_dtype for the per-layer trunk linears
 * (wq, wk, wv, wo, w_gate, w_up, w_down; DiT and VISION: mlp_w1, mlp_w2) and F32 or BF16 (matching the path:
 * F32 for the fp32 path, BF16 otherwise) for every other tensor.  For
 * FP8E4M3, `scale` holds `cols` float32 scales (W_ij = code_ij * scale_j).
 * For FP4E2M1, `data` holds rows x cols/2 bytes (byte (i, j) = the codes of
 * columns 2j, low nibble, and 2j + 1, high nibble; cols even, rows a multiple
 * of 32) and `scale` holds (rows/32) x cols float32 powers of two in
 * 2^-126 .. 2^127 (W_ij = value(code_ij) * scale[i/32][j]); any other scale
 * is PHYAI_EINVAL. */
typedef struct {
  const char* name;         /* e.g. "in_w", "layers.3.wq" (see phyai_load_expert)               */
  int32_t dtype;            /* phyai_dtype                                                        */
  int32_t rows, cols;
  const void* data;         /* host                                                               */
  const float* scale;       /* host, FP8E4M3 and FP4E2M1 only                                     */
} phyai_tensor;

typedef struct phyai_expert phyai_expert;

/* Validate `cfg`, copy and repack every tensor into library-owned device
 * memory (MFMA operand order; the Q/K/V projections are fused into one
 * weight and gate/up into another, as in the paper's single QKV and single
 * gate+up GEMMs, Section "Optimization Methods", paragraph "Kernel fusion"),
 * allocate the working buffers for up to max_batch requests, and build the
 * timestep tables of the default schedule t_k = 1 - k/max_steps.
 *
 * Tensor names (L = n_layers, l = layer index):
 *   all:   in_w [A][d], in_b [1][d], out_w [d][A], out_b [1][A],
 *          layers.l.{wq [d][nq*dh], wk, wv [din][nkv*dh], wo [nq*dh][d]}
 *          (din = d_feat on even DiT layers, else d)
 *   state_token: state_w [A][d], state_b [1][d]
 *   PI0:   time_w1 [d+time_dim][d], time_b1, time_w2 [d][d], time_b2,
 *          layers.l.{attn_norm, mlp_norm} [1][d], final_norm [1][d],
 *          layers.l.{w_gate, w_up} [d][F], layers.l.w_down [F][d]
 *   PI05:  cond_w1 [time_dim][d], cond_b1, cond_w2 [d][d], cond_b2,
 *          layers.l.{attn_mod_w, mlp_mod_w} [d][2d] (+ _b [1][2d]),
 *          final_mod_w [d][2d], final_mod_b, gate/up/down as PI0
 *   DIT:   cond_w1 [time_dim][d], cond_b1, cond_w2, cond_b2, pos_emb [H][d],
 *          layers.l.ada_w [d][6d], ada_b [1][6d], layers.l.mlp_w1 [d][F],
 *          mlp_b1 [1][F], mlp_w2 [F][d], mlp_b2 [1][d],
 *          final_ada_w [d][2d], final_ada_b [1][2d]
 *   PREFIX_LM: layers.l.{attn_norm [1][d], wq, wk, wv} for every layer and
 *          layers.l.{wo, mlp_norm, w_gate, w_up, w_down} for every layer but
 *          the last (whose keys and values depend only on its input); no
 *          in/out, time or state tensors
 *   VISION: patch_w [patch_dim][d], patch_b [1][d], pos_emb [n_patches][d],
 *          layers.l.{ln1_w, ln1_b, ln2_w, ln2_b} [1][d],
 *          layers.l.{wq, wk, wv, wo} [d][d], layers.l.{bq, bk, bv, bo} [1][d],
 *          layers.l.mlp_w1 [d][F], mlp_b1 [1][F], mlp_w2 [F][d], mlp_b2 [1][d],
 *          post_ln_w, post_ln_b [1][d], proj_w [d][d_out], proj_b [1][d_out]
 * Host buffers may be freed after the call returns.  On failure *out is set
 * to NULL and nothing is leaked.  The call synchronises `stream`. */
int phyai_load_expert(const phyai_config* cfg, const phyai_tensor* tensors, int32_t n_tensors,
                      void* stream, phyai_expert** out);

/* Produce one action chunk per request (the K-step Euler loop).
 *
 * Operation: the policy map from an observation to an action chunk of
 * Section "Embodied Task Formulation", subsection "From Observation to
 * Action", for flow policies: x_0 = noise, x_{k+1} = x_k + (t_{k+1} - t_k)
 * v(x_k, t_k) for k < K, output x_K.  The vision-language prefix state is
 * computed once per chunk and stays fixed across the K steps while only the
 * action tokens change; the timestep tables are built before denoising; the
 * whole loop is captured once per shape bucket and replayed (Section "PhyAI
 * Architecture", subsection "Optimization Methods", paragraph "Graph
 * replay").  Requests of a batch are independent (Section "Cloud Batching").
 *
 *   prefix      device, read-only, caller-owned.  PI0/PI05: the frozen prefix
 *               K/V cache, [L][2][B][prefix_cap][n_kv*head_dim] (index 0 = K,
 *               1 = V; keys already rotated), dtype kv_dtype.  DIT: the VLM
 *               feature tokens [B][prefix_cap][d_feat], dtype kv_dtype.
 *               Rows at or beyond prefix_len[b] are never read.
 *   prefix_len  host [B], 0 <= prefix_len[b] <= prefix_cap (DIT: >= 1).
 *   noise       device float32 [B][H][A]: x at t_0.
 *   timesteps   host float32 [n_steps + 1]: t_0 .. t_K (any values; the
 *               default schedule runs from 1 to 0).  Tables that depend only
 *               on the schedule are rebuilt when it differs from the last.
 *   n_steps     K, 1 <= K <= max_steps.
 *   batch       B, 1 <= B <= max_batch.
 *   state       device float32 [B][A] when state_token = 1, else ignored.
 *   out_actions device float32 [B][H][A]: x at t_K.  May alias `noise`.
 *   stream      work is enqueued on it; the call returns after enqueueing
 *               (it waits on the host only for a schedule change that
 *               arrives while the previous change's table upload is still
 *               pending).
 *
 * Device pointers (prefix, noise, state, out_actions) must be 16-byte
 * aligned: the kernels read and write them with 16-byte accesses.  A
 * misaligned pointer fails with PHYAI_EINVAL before anything is enqueued.
 * The prefix validity scope is the call: the library keeps no reference to
 * it after the enqueued work ends.  Calls on one handle must be ordered on
 * the device (the same stream, or streams the caller orders): they share
 * the handle's working buffers and timestep tables.
 *
 * The first call for a (batch, n_steps) pair captures a HIP graph of the
 * whole loop (the graph bucket of paragraph "Graph replay"); later calls
 * replay it and allocate nothing.  Errors: PHYAI_EINVAL for a NULL handle or
 * argument, a size out of range, a prefix length outside 0..prefix_cap (DiT:
 * 1..prefix_cap), a non-finite timestep or a misaligned pointer; PHYAI_EHIP
 * if a HIP call fails (capture, instantiation, launch). */
int phyai_denoise(phyai_expert* e, const void* prefix, const int32_t* prefix_len,
                  const float* noise, const float* timesteps, int32_t n_steps, int32_t batch,
                  const float* state, float* out_actions, void* stream);

/* phyai_denoise for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same arguments, validation, kernels and results, with two differences.
 * It never allocates (no hipMalloc, hipFree or allocating library routine):
 * it launches the loop's kernels directly instead of capturing and
 * instantiating a graph, and the scratch those kernels need between launches
 * (split-K partial sums of the residual GEMMs, key-split attention partials)
 * lives in a static device array of 32 MiB, one per device, held until the
 * process ends.  A call that would need more (large batches with key-split
 * attention) fails with PHYAI_EINVAL before anything is enqueued.  Every call
 * on a device shares that device's array: calls that overlap on one device
 * race, so they must be ordered (one stream, or streams the caller orders),
 * whatever handle they use.  Nothing in the array needs to start at zero:
 * each call writes every partial before reading it. */
int phyai_denoise_static(phyai_expert* e, const void* prefix, const int32_t* prefix_len,
                         const float* noise, const float* timesteps, int32_t n_steps, int32_t batch,
                         const float* state, float* out_actions, void* stream);

/* Produce the frozen prefix K/V cache of a batch of requests from their
 * prefix token embeddings (handle of variant PHYAI_VARIANT_PREFIX_LM).
 *
 * Operation: the language-prefix phase of the pi-family, which the paper
 * times separately from the vision tower and the action expert (Section
 * "Evaluation", batch analysis of PI0.5) and whose per-layer K/V the action
 * expert reads unchanged at every denoising step (Section "PhyAI
 * Architecture", paragraph "Graph replay").  For every layer l and valid
 * prefix token t: the keys (rotated at position t when rope = 1) and values
 * of that layer's K/V projection, after layers 0 .. l-1 have run over all
 * valid tokens of the request with bidirectional attention.
 *
 *   embeds      device float32 [B][prefix_cap][d_model]: the prefix token
 *               embeddings (image tokens and text, already scaled), the
 *               input of layer 0.  Rows at or beyond prefix_len[b] are never
 *               read.
 *   prefix_len  host [B], 0 <= prefix_len[b] <= prefix_cap.
 *   kv_out      device, [L][2][B][prefix_cap][n_kv*head_dim] in kv_dtype
 *               (index 0 = K, 1 = V): exactly the `prefix` argument of
 *               phyai_denoise for an expert with the same n_layers, n_kv_heads,
 *               head_dim and prefix_cap.  Rows at or beyond prefix_len[b] are
 *               written as zeros.  Caller-owned.
 *   batch       B, 1 <= B <= max_batch.
 *   stream      work is enqueued on it; the call returns after enqueueing.
 *
 * embeds and kv_out must be 16-byte aligned.  Calls on one handle must be
 * ordered on the device (they share its working buffers).  Errors:
 * PHYAI_EINVAL for a NULL or non-prefix-LM handle, a NULL or misaligned
 * pointer, a batch or prefix length out of range; PHYAI_EHIP if a launch
 * fails.  The denoising entry points refuse a prefix-LM handle. */
int phyai_prefill(phyai_expert* e, const float* embeds, const int32_t* prefix_len, void* kv_out, int32_t batch,
                  void* stream);

/* Encode the camera images of a batch of requests into image tokens (handle
 * of variant PHYAI_VARIANT_VISION).
 *
 * Operation: the vision-tower phase of the pi-family, which the paper times
 * separately from the language prefix and the action expert (Section
 * "Evaluation", batch analysis of PI0.5); its tokens are the first rows of
 * the prefix embeddings that phyai_prefill takes.  Per image: h = patches
 * W_patch + b_patch + pos_emb; per block h += Attn(LN1(h)) W_o + b_o (every
 * patch attends to every patch of its own image, scale 1/sqrt(head_dim)),
 * h += GELU_tanh(LN2(h) W_1 + b_1) W_2 + b_2; tokens = LN_post(h) W_proj +
 * b_proj, with LN(x) = (x - mean) / sqrt(var + rms_eps) * (1 + w) + b.
 *
 *   patches     device float32 [B][n_images][n_patches][patch_dim]: the
 *               images already cut into patches and normalised.
 *   tokens_out  device float32 [B][out_rows][d_out]: rows 0 ..
 *               n_images*n_patches-1 of request b receive its image tokens,
 *               image-major; rows from n_images*n_patches on are not
 *               touched (so a prefix-embedding buffer [B][prefix_cap][d]
 *               with d = d_out can take the text embeddings there).
 *               Caller-owned.
 *   out_rows    rows per request in tokens_out, >= n_images*n_patches.
 *   batch       B requests, 1 <= B <= max_batch.
 *   stream      work is enqueued on it; the call returns after enqueueing.
 *
 * patches and tokens_out must be 16-byte aligned.  Calls on one handle must
 * be ordered on the device (they share its working buffers).  Errors:
 * PHYAI_EINVAL for a NULL or non-vision handle, a NULL or misaligned
 * pointer, a batch or out_rows out of range; PHYAI_EHIP if a launch fails.
 * The denoising entry points and phyai_prefill refuse a vision handle. */
int phyai_encode_images(phyai_expert* e, const float* patches, float* tokens_out, int32_t out_rows,
                        int32_t batch, void* stream);

/* Capture the graph of the K-step loop for the (batch, n_steps) bucket ahead
 * of the first phyai_denoise with that shape, so that the first prediction
 * does not pay for the capture (the runner captures the full loop in the
 * matching graph bucket once buffers and control flow are stable: Section
 * "PhyAI Architecture", paragraph "Graph replay").  The graph reads its
 * per-call pointers and prefix lengths from a device descriptor that
 * phyai_denoise writes, so one bucket serves every call of that shape.
 * `stream` is unused (capture runs on a private stream).  Errors:
 * PHYAI_EINVAL for a NULL handle or a size out of range; PHYAI_EHIP if
 * capture or instantiation fails.  Idempotent. */
int phyai_prepare(phyai_expert* e, int32_t batch, int32_t n_steps, void* stream);

/* Copy the residual stream h [B*M][d] (float32) left by the last
 * phyai_denoise call (after the final step's last layer, before the final
 * norm) into `dst` (device).  Diagnostic for layer-by-layer parity tests. */
int phyai_debug_hidden(phyai_expert* e, float* dst, int32_t batch, void* stream);

/* Measurement aid: enqueue `reps` passes over all L layers of one stage of
 * the transformer block, exactly as the graph launches it (step 0 of the
 * current schedule, the batch of the last phyai_denoise call), eagerly on
 * `stream`, so that a caller can time a single kernel with events.
 * Stages: 0 norm before attention, 1 QKV GEMM (+RoPE, KV write),
 * 2 attention (with key splits, the merge kernel too when the O projection
 * does not merge them), 3 O-projection GEMM + residual (at small batch it
 * merges the attention's key splits on the way in), 4 norm before the MLP,
 * 5 gate/up GEMM + GeGLU (DiT: MLP-in + GELU), 6 down GEMM + residual.  Requires a previous phyai_denoise on this handle (the stage
 * reads the buffers it left); it overwrites working buffers only, never the
 * caller's.  Loop semantics (Section "PhyAI Architecture", paragraph
 * "Kernel fusion", lists these fused operators). */
int phyai_profile_stage(phyai_expert* e, int32_t stage, int32_t reps, void* stream);

/* Decode `n` OCP e4m3fn codes (device uint8) to bfloat16 bit patterns (device
 * uint16) with the same conversion the GEMM kernels use when they expand fp8
 * weights (the W8A16 path of the paper's quantised GEMMs, paragraph
 * "Quantization").  Codes 0x7f/0xff (NaN) give a NaN pattern. */
int phyai_fp8_to_bf16(const uint8_t* codes, uint16_t* out, int64_t n, void* stream);

/* Free every device buffer and graph of the handle.  NULL is accepted. */
void phyai_free_expert(phyai_expert* e);

/* Thread-local text of the last error ("" if none). */
const char* phyai_last_error(void);

/* Library ABI version (major * 100 + minor). */
int phyai_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PHYAI_H */
