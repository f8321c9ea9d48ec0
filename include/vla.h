/*
 * vla.h - C ABI of the MI355X (gfx950) two-phase VLA inference library.
 *
 * The library runs the inference pipeline the paper characterises
 * (Section 2.1, "Vision-Language-Action Models", and its last paragraph on
 * the execution model): phase 1, a VLM (ViT patch encoder + language-model
 * prefill), turns a camera frame and an instruction into a per-layer KV
 * cache; phase 2, a flow-matching action expert, integrates a velocity field
 * with Euler steps to produce an action chunk, every step attending to that
 * cache. The VLM prefill of frame N+1 runs concurrently with the action phase
 * of frame N on a second stream (Section 2.1; Fig. "streamexec" (a)-(c) of
 * Section 2.4 name the serialized, naive two-stream and ideal schedules).
 *
 * Conventions
 *  - Every function returns 0 (VLA_OK) or a negative status; nothing aborts
 *    and no C++ exception crosses the ABI. vla_last_error() returns a
 *    thread-local message for the last failing call on this thread.
 *  - Pointers documented "device" are HIP device pointers on the model's
 *    device; "host" pointers are ordinary host memory. They are never mixed.
 *  - Streams are hipStream_t passed as void*; NULL means the null stream.
 *  - Objects made by *_create are owned by the library until *_destroy.
 *    All other buffers are owned by the caller and must stay alive until the
 *    asynchronous work that reads or writes them has completed.
 *  - One model runs one prefill and one denoise at a time (they use
 *    model-owned scratch memory per phase). A prefill (or denoise) called on
 *    another stream than the previous one first waits, on the device, for
 *    that call's work, so calls of one phase never overlap; a prefill and a
 *    denoise do overlap. Calls made while their stream is being captured into
 *    a graph are not ordered this way: captured calls of one phase on two
 *    streams race. vla_pipeline_run first waits on the host for the last
 *    standalone call of each phase.
 */
#ifndef VLA_H
#define VLA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---- */
#define VLA_OK 0
#define VLA_EINVAL (-1)       /* invalid argument or configuration            */
#define VLA_ENOMEM (-2)       /* device or host allocation failed             */
#define VLA_EHIP (-3)         /* a HIP runtime call failed (message has it)   */
#define VLA_EUNSUPPORTED (-4) /* valid request the library does not implement */
#define VLA_ESTATE (-5)       /* object in the wrong state (e.g. mismatched), */
                              /* or an internal error of the library          */

/* ---- number types ---- */
#define VLA_F32 0  /* every tensor and operand fp32                           */
#define VLA_BF16 1 /* bf16 weights, GEMM operands and KV cache; fp32 elsewhere */

/*
 * Model shape. The paper fixes no layer shapes (it names the model families,
 * Section 2.1); the fields below describe a SigLIP-style ViT, a Gemma-style
 * prefix LM with grouped (multi-query) attention, and a pi0-style action
 * expert that shares the LM's attention head layout.
 */
typedef struct vla_config {
  int32_t dtype;                                 /* VLA_F32 or VLA_BF16          */
  int32_t n_views, img_h, img_w, patch;          /* camera views, HWC image, patch */
  int32_t vit_dim, vit_heads, vit_mlp, vit_layers;
  int32_t lm_dim, lm_heads, lm_kv_heads, head_dim, lm_mlp, lm_layers;
  int32_t vocab, n_text, state_dim;              /* state_dim 0 = no state token */
  int32_t ex_dim, ex_mlp, ex_layers;             /* ex_layers must equal lm_layers */
  int32_t chunk_len, action_dim, n_steps;        /* action chunk H x A, Euler steps */
  int32_t head;     /* VLA_HEAD_PI0, VLA_HEAD_DIT or VLA_HEAD_COG                    */
  int32_t shuffle;  /* pixel-shuffle factor of the ViT grid before the projector (1: none) */
  int32_t ex_heads; /* DiT and cognition heads: attention heads (head dim ex_dim / ex_heads) */
  int32_t sampler;  /* VLA_SAMPLER_EULER or VLA_SAMPLER_DDIM (see below)              */
} vla_config;

/* Action-head families (Section 2.1): the pi0-style expert runs its own
 * decoder layers over [the LM's per-layer KV cache; its own K/V]
 * (ex_layers == lm_layers); the GR00T-style DiT (adaLN-conditioned, even
 * layers cross-attending to the LM's final normalised hidden states, odd
 * layers self-attending) reads per-frame cross K/V made from those features. */
#define VLA_HEAD_PI0 0
#define VLA_HEAD_DIT 1
/* VLA_HEAD_COG: the CogACT-style diffusion head (Section 2.1 names CogACT's
 * head as a 300M DiT fed by cognition features). A learned cognition token
 * is appended to the prefix (prefix + 1 rows), every LM layer runs, and the
 * token's final RMS-normalised output, projected to ex_dim (c = W_c f + b_c),
 * is the hand-off (one fp32 vector per context). The head runs ex_layers
 * pre-LN self-attention layers (ex_heads heads, no biases, GELU MLP of ex_mlp)
 * over [chunk_len action tokens; c; a time token], chunk_len <= 62; the final
 * LayerNorm and the out-projection of the action rows give the head output
 * (the noise estimate under VLA_SAMPLER_DDIM). */
#define VLA_HEAD_COG 2

/* Samplers of the action head (Section 2.1 names flow-matching and diffusion
 * heads). EULER: flow matching from noise at t = 1 to data at t = 0, the head
 * output read as a velocity, t_k = (N - k) / N and x += -(1/N) v. DDIM: the
 * head output read as the noise estimate; deterministic DDIM over a linear
 * beta schedule (1e-4 .. 0.02, 1000 training steps), timesteps
 * s_k = floor((N - k) 1000 / N) - 1, time input t_k = s_k / 1000, and
 * x <- a_k x + b_k eps with a_k = sqrt(abar_{k+1} / abar_k),
 * b_k = sqrt(1 - abar_{k+1}) - a_k sqrt(1 - abar_k) (abar after the last
 * step = 1). */
#define VLA_SAMPLER_EULER 0
#define VLA_SAMPLER_DDIM 1

typedef struct vla_model vla_model;
typedef struct vla_ctx vla_ctx;

/* One robot frame, all device pointers, read-only for the library. */
typedef struct vla_frame {
  const float* pixels;     /* fp32 [n_views, img_h, img_w, 3] (HWC), values as given */
  const int32_t* text_ids; /* int32 [n_text], each in [0, vocab)                     */
  const float* state;      /* fp32 [state_dim]; NULL when state_dim == 0             */
} vla_frame;

/* Pipeline schedules (Fig. "streamexec"): */
#define VLA_MODE_SERIAL 0     /* both phases of every frame on one stream           */
#define VLA_MODE_CONCURRENT 1 /* VLM and action streams, hardware dispatcher decides */
#define VLA_MODE_CU_MASKED 2  /* as CONCURRENT, each stream limited to a CU set      */
#define VLA_MODE_WG_CAPPED 3  /* as CONCURRENT, VLM grids capped per CU              */

typedef struct vla_sched {
  int32_t mode;       /* VLA_MODE_*                                                 */
  int32_t vlm_cus;    /* CU_MASKED: CUs for the VLM stream (multiple of 8)           */
  int32_t act_cus;    /* CU_MASKED: CUs for the action stream (multiple of 8); the  */
                      /*   two sets are disjoint and together at most the CU count   */
  int32_t vlm_wg_cap; /* WG_CAPPED: max VLM workgroups per CU in flight (>= 1)       */
  int32_t act_streams;/* action streams (0 or 1: one; at most 4). With k > 1 the     */
                      /*   action phases of k consecutive frames (different robots)  */
                      /*   run concurrently on k streams; not with VLA_MODE_SERIAL   */
  int32_t graphs;     /* 1: replay each phase as a captured HIP graph (captured on   */
                      /*   first use and cached per context / stream)                */
  int32_t vlm_streams;/* VLM streams (0 or 1: one; at most 2). With 2, the prefills  */
                      /*   of consecutive frames alternate between two streams and   */
                      /*   may overlap each other; not with VLA_MODE_SERIAL          */
  int32_t act_batch;  /* frames per action phase (0 or 1: one; at most 8). With     */
                      /*   k > 1, the action phases of k consecutive frames          */
                      /*   (different robots) run as one denoising loop that reads   */
                      /*   the weights once for all of them; it starts when their    */
                      /*   prefills are done. A final group of fewer than k frames   */
                      /*   runs with as many as remain. A frame's chunk does not     */
                      /*   depend on k >= 2 or on the group it lands in (every       */
                      /*   reduction is planned for 8 frames); it differs from the   */
                      /*   one-frame loop only in rounding order (see                */
                      /*   vla_pipeline_run). VLA_HEAD_PI0 models only.              */
  int32_t vlm_batch;  /* frames per VLM prefill (0 or 1: one; else 2, 4 or 8). With  */
                      /*   k > 1, the prefills of k consecutive frames (different    */
                      /*   robots) run as one pass: their views stacked for the ViT  */
                      /*   and their prefixes for the LM, so every weight is read    */
                      /*   once for all k; a final group of fewer than k frames runs */
                      /*   with as many as remain. Every frame's cache and chunk are */
                      /*   bit identical to its own run.                             */
  int32_t act_chunks; /* action chunks per VLM output (0 or 1: one; at most 64):     */
                      /*   asynchronous inference. Each frame's context feeds k      */
                      /*   action phases (items), each from its own noise; item i is */
                      /*   chunk i % k of frame i / k. act_batch then counts items.  */
} vla_sched;

typedef struct vla_timing {
  double wall_ms;       /* host wall time of the run, enqueue to final sync   */
  double frames_per_s;  /* R / wall time                                      */
  double actions_per_s; /* frames_per_s * chunk_len (chunk rows per second)   */
  double vlm_ms;        /* GPU time of the VLM phases (events), summed        */
  double act_ms;        /* GPU time of the action phases (events), summed     */
} vla_timing;

/* Fill *out with a named preset: "tiny" (fp32, 2+2+2 layers, chunk 8x7,
 * 4 steps), "pi0" (PaliGemma-3B-shaped VLM + pi0-shaped expert, bf16),
 * "pi0_3view" (pi0 with three camera views and 64 text tokens), "pi0_ddim"
 * (pi0 sampled with DDIM), "tiny_ddim", "gr00t" (GR00T-shaped VLA with its
 * DiT head, bf16), "tiny_dit", "cogact" (the PaliGemma-shaped VLM with the
 * cognition-token head: 24 layers of width 1024, 16 heads, MLP 4096, chunk
 * 16x7, 10 DDIM steps, bf16) or "tiny_cog" (fp32).
 * VLA_EINVAL for an unknown name or NULL pointers. */
int vla_preset(const char* name, vla_config* out);

/* Check a configuration without allocating (VLA_EINVAL with a message when
 * a shape rule fails: n_q % n_kv, ex_layers == lm_layers, patch divides the
 * image, head_dim a multiple of 32, MLP widths multiples of 16, ...). */
int vla_validate(const vla_config* cfg);

/* Create a model on the current HIP device: validate cfg, generate every
 * parameter from `seed` with the counter-based SplitMix64 generator (the
 * same published generator the test inputs use; bf16 configurations round
 * the fp32 master value to bf16, nearest-even), upload them and allocate the
 * per-phase scratch memory. Blocking. The library owns *out. */
int vla_create(const vla_config* cfg, uint64_t seed, vla_model** out);

/* Copy the model's configuration to *out (host). VLA_EINVAL for NULL
 * pointers. Lets a caller size the device buffers of the calls below. */
int vla_model_config(const vla_model* m, vla_config* out);

/* Free everything the model owns (waits for its streams). NULL is a no-op. */
int vla_destroy(vla_model* m);

/* Phase-1 -> phase-2 hand-off: the per-layer KV cache of the model's storage
 * type, in the layout the attention kernel reads (MFMA fragment order, keys
 * in blocks of 32; documented at vla_debug_attention_cache), prefix rounded
 * up to 32 keys per KV head; vla_ctx_export_kv returns it row-major.
 * Caller-owned via these two calls; destroy NULL is a no-op. */
int vla_ctx_create(vla_model* m, vla_ctx** out);
int vla_ctx_destroy(vla_ctx* c);

/* Phase 1 for one frame, enqueued on `stream`, asynchronous: ViT over each
 * view, projector, prefix [image; text * sqrt(lm_dim); state], LM prefill
 * writing every layer's K (after RoPE) and V into `ctx`. */
int vla_vlm_prefill(vla_model* m, const vla_frame* in, vla_ctx* ctx, void* stream);

/* Phase 2 for one frame, enqueued on `stream`, asynchronous: n_steps sampler
 * steps from x_0 = noise, each a full pass of the action head (pi0 expert:
 * over [ctx KV; its own KV]; DiT: over the ctx cross K/V) whose output
 * updates x in the output projection's epilogue: x <- x + dt v (Euler, t
 * from 1 to 0) or x <- a_k x + b_k eps (DDIM; see VLA_SAMPLER_DDIM). noise
 * and actions are device fp32 [chunk_len, action_dim] and may alias. Must be
 * ordered after the prefill that wrote ctx (same stream, or an event wait). */
int vla_action_denoise(vla_model* m, const vla_ctx* ctx, const float* noise, float* actions,
                       void* stream);

/* Run R frames through the two-stage pipeline and wait for it. frames:
 * host array of at least R vla_frame (device pointers inside); noise: device
 * fp32 [R * k, chunk_len, action_dim] with k = max(1, act_chunks), item i =
 * chunk i % k of frame i / k; actions: device fp32 of the same shape. The
 * library cannot check these lengths: shorter buffers are read and written
 * out of bounds (the Python binding checks tensors before the call). The VLM
 * prefill of a later prefill group overlaps the action phases of earlier
 * ones (a ring of model-owned contexts, allocated in blocks of 8, and events
 * between the streams) except in VLA_MODE_SERIAL. Results are bit-identical
 * across modes, stream counts, prefill batching and graph replay. Batched
 * action loops (act_batch >= 2) are bit-identical among themselves and
 * differ from one-item loops only in the GEMMs' rounding order: for Euler
 * both are within the chunk tolerance of the exact model; DDIM amplifies a
 * head-output difference by up to sum_k |b_k| prod_{j>k} |a_j| (about 160 for
 * 10 steps), so its batched and one-item chunks differ by that factor more.
 * t may be NULL (frames_per_s counts frames, actions_per_s counts chunk rows
 * of every item). Calls on one model are serialised. */
int vla_pipeline_run(vla_model* m, const vla_frame* frames, const float* noise, int32_t R,
                     const vla_sched* sched, float* actions, vla_timing* t);

/* Parameter inventory (host-side queries). Names follow the logical layout
 * [out, in] of each matrix, e.g. "lm.3.q.w". */
int vla_param_count(const vla_model* m, int32_t* count);
int vla_param_info(const vla_model* m, int32_t i, const char** name, int64_t* numel);

/* Copy one parameter, as the model stores it, to host fp32 in its logical
 * layout (bf16 values upcast exactly). host_dst: numel floats. Blocking. */
int vla_export_param(vla_model* m, const char* name, float* host_dst, int64_t numel);

/* Copy layer `layer` of a context's K and V cache to host fp32 buffers of
 * [prefix, lm_kv_heads * head_dim] each (logical head-dim order). Blocking. */
int vla_ctx_export_kv(vla_model* m, const vla_ctx* c, int32_t layer, float* host_k, float* host_v);

/* VLA_HEAD_DIT only: copy the cross K and V of even DiT layer `layer` (made
 * from the LM features in the prefill) to host fp32 buffers of [prefix,
 * ex_dim] each (head-major columns). Blocking. */
int vla_ctx_export_cross(vla_model* m, const vla_ctx* c, int32_t layer, float* host_k, float* host_v);

/* VLA_HEAD_COG only: copy a context's cognition vector (fp32 [ex_dim]) to
 * host_dst. Blocking. */
int vla_ctx_export_cog(vla_model* m, const vla_ctx* c, float* host_dst);

/* Test entry points for single kernels (same kernels and launch planner as
 * the phases). dtype VLA_F32 or VLA_BF16 selects the operand type of A and W
 * (bf16 passed as uint16 bit patterns). All pointers device.
 *  gemm:      C[M,N] (fp32) = A[M,K] W[N,K]^T + bias[N] (bias may be NULL);
 *             K a multiple of 8, lda/ldw >= K elements.
 *  attention: out[Sq, nq*hd] = softmax(q k^T / sqrt(hd)) v per query head,
 *             query head h reading KV head h / (nq / nkv); keys are
 *             [k0 (S0 rows); k1 (S1 rows)], values likewise; rows of q have
 *             nq*hd elements, rows of k/v nkv*hd (operand type); out in the
 *             operand type. k1/v1 may be NULL when S1 == 0.             */
int vla_debug_gemm(int32_t dtype, int32_t M, int32_t N, int32_t K, const void* A, int32_t lda,
                   const void* W, int32_t ldw, const float* bias, float* C, void* stream);
int vla_debug_attention(int32_t dtype, int32_t Sq, int32_t nq, int32_t nkv, int32_t hd,
                        const void* q, const void* k0, const void* v0, int32_t S0, const void* k1,
                        const void* v1, int32_t S1, void* out, void* stream);

/* Test entry point for the GEMM epilogues (the fused operations of every
 * phase), on the tiled kernel or the skinny one. A [M][K] and W [N][K] are
 * row-major device arrays of the operand type (dtype as in vla_debug_gemm;
 * K a multiple of 8) with W in its logical row order; with v = A W^T:
 *  BIAS       out fp32 [M][N] = v + bias
 *  T          out [M][N] = T(v + bias)            (T: round to the operand type)
 *  GELU       out [M][N] = T(gelu_tanh(v + bias))
 *  SWISH      out [M][N] = T(swish(v + bias))
 *  GEGLU      W = [gate (N/2 rows); up (N/2 rows)], N a multiple of 32:
 *             out [M][N/2] = T(gelu_tanh(v_gate) * v_up)
 *  QKV_ROPE   W = [q (nq hd rows); k (nkv hd); v (nkv hd)], hd a multiple of
 *             32: q_out [M][nq hd] and k_out [M][nkv hd] = T(RoPE(v_q or v_k,
 *             position pos0 + m)) (rotate-half pairs (i, i + hd/2), angle
 *             p 10000^(-2 i / hd)), v_out [M][nkv hd] = T(v_v); K and V pass
 *             through the KV-cache layout and are returned row-major
 *  QKV_PLAIN  as QKV_ROPE without the rotation (hd a multiple of 8)
 *  STEP       x fp32 [M][N] <- xs x + dt (v + bias); out [M][N] = T(new x)
 *  RESID_NORM resid fp32 [M][N] += v (split-K partials summed in split
 *             order); out [M][N] = T(RMSNorm(resid) * gain), N <= 2048
 * bias may be NULL; GEGLU and QKV take none. skinny = 1 runs the action
 * head's kernel (M <= 64): W is converted to MFMA fragment order and A to
 * the row-block operand layout, and operand-type outputs are written in that
 * layout and returned row-major. skinny = 0 runs the tiled kernel with the
 * tile the planner picks for M and N. plan_out (host, may be NULL) receives
 * the tile's rows and columns (0 and 32 for the skinny kernel) and the
 * split-K factor. Blocking; allocates temporaries. */
#define VLA_DEBUG_EPI_BIAS 0
#define VLA_DEBUG_EPI_T 1
#define VLA_DEBUG_EPI_GELU 2
#define VLA_DEBUG_EPI_SWISH 3
#define VLA_DEBUG_EPI_GEGLU 4
#define VLA_DEBUG_EPI_QKV_ROPE 5
#define VLA_DEBUG_EPI_QKV_PLAIN 6
#define VLA_DEBUG_EPI_STEP 7
#define VLA_DEBUG_EPI_RESID_NORM 8
typedef struct vla_debug_epi {
  int32_t kind;           /* VLA_DEBUG_EPI_*                                   */
  int32_t skinny;         /* 0: tiled kernel, 1: skinny kernel (M <= 64)       */
  const float* bias;      /* device fp32 [N] or NULL                           */
  void* out;              /* device, see above                                 */
  int32_t nq, nkv, hd, pos0; /* QKV_ROPE / QKV_PLAIN                           */
  void* q_out;            /* device, operand type                              */
  void* k_out;
  void* v_out;
  float* x;               /* STEP: device fp32 [M][N], updated                 */
  float xs, dt;           /* STEP coefficients                                 */
  float* resid;           /* RESID_NORM: device fp32 [M][N], updated           */
  const float* gain;      /* RESID_NORM: device fp32 [N]                       */
  int32_t* plan_out;      /* host int32[3] or NULL                             */
} vla_debug_epi;
int vla_debug_gemm_epi(int32_t dtype, int32_t M, int32_t N, int32_t K, const void* A, const void* W,
                       const vla_debug_epi* e, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops and harnesses that forbid hipMalloc): the GEMM of
 * vla_debug_gemm, same arguments, layouts, kernels, plan and result bits,
 * but it allocates nothing and never synchronises. Its split-K partials go
 * to a fixed device array of 2^21 floats (8 MiB) that every GPU the library
 * runs on holds until the process ends; a shape whose plan needs more
 * returns VLA_EUNSUPPORTED (the planner splits at most 256 64-wide tiles, so
 * no valid shape needs more than 2^20 floats). Every call on one GPU shares
 * that array and a later call overwrites it: calls whose executions overlap
 * on one GPU (two streams, or two host threads) race. Each call writes every
 * partial it reads, so nothing needs clearing between calls. All pointers
 * device; asynchronous on `stream`. */
int vla_gemm_noalloc(int32_t dtype, int32_t M, int32_t N, int32_t K, const void* A, int32_t lda,
                     const void* W, int32_t ldw, const float* bias, float* C, void* stream);

/* Test entry point for the attention kernel of the LM and the expert: as
 * vla_debug_attention (q and out row-major, out 16-byte aligned), but K and V
 * of each segment are in the KV-cache layout, with nb = ceil(S / 32) blocks
 * per KV head. With VEC = 8 (bf16) or 4 (fp32) elements per 16 bytes,
 * SW = 4 VEC, NS = ceil(hd / SW), NDT = ceil(hd / 16), PVS = 32 / SW, key
 * p = 32 b + kin (kin < 32) and head-dim index d of KV head j sit at
 *   K: ((((j nb + b) 2 + nt) NS + d / SW) 64 + 16 ((d % SW) / VEC) + i) VEC + d % VEC
 *      with (nt, i) = ((kin / 4) % 2, 4 (kin / 8) + kin % 4) for bf16 and
 *      (kin / 16, kin % 16) for fp32;
 *   V: ((((j nb + b) NDT + d / 16) PVS + kin / SW) 64 + 16 ((kin % SW) / VEC)
 *      + d % 16) VEC + kin % VEC.
 * Each 64 x VEC run is one MFMA operand load. V must be zero at keys
 * S .. 32 nb - 1; other unused positions are never read into the result.
 * fp32 needs hd <= 128. All pointers device. */
int vla_debug_attention_cache(int32_t dtype, int32_t Sq, int32_t nq, int32_t nkv, int32_t hd,
                              const void* q, const void* k0, const void* v0, int32_t S0, const void* k1,
                              const void* v1, int32_t S1, void* out, void* stream);

/* Test entry point for the row norm of every layer (the pre-norms of the
 * ViT, LM and expert layers: LayerNorm with biased variance, or RMSNorm;
 * epsilon 1e-6). For each of `rows` rows of d fp32 values x (device,
 * row-major, leading dimension ldx elements):
 *  - with splits > 0, x <- x + bias + colscale * (part[0] + ... +
 *    part[splits-1]) first, the partials summed in split order and the
 *    result written back to x (the residual update of a split-K GEMM);
 *    part is [splits][rows][d] fp32, contiguous; bias and colscale [d] may
 *    be NULL. With splits = 0, x is only read and bias and colscale are not
 *    used;
 *  - y = (x - mean) / sqrt(var + 1e-6) * g + shift (rms = 0, LayerNorm), or
 *    y = x / sqrt(mean(x^2) + 1e-6) * g (rms = 1; shift may still be given),
 *    with g = gain, or 1 + gain when gain_plus_one != 0; gain [d] required,
 *    shift [d] may be NULL;
 *  - out [rows][ldo] in the operand type of dtype (bf16 as uint16 bits).
 * d is a multiple of 4 in 4 .. 2048; ldx and ldo are multiples of 4 and at
 * least d; x, part, bias, colscale, gain and shift are 16-byte aligned, out
 * 16-byte (fp32) or 8-byte (bf16) aligned, else VLA_EINVAL. rows = 0 does
 * nothing and reads no pointer (they may be NULL). All pointers device;
 * asynchronous on `stream`. */
int vla_debug_norm(int32_t dtype, int32_t rows, int32_t d, float* x, int32_t ldx, const float* part,
                   int32_t splits, const float* bias, const float* colscale, const float* gain,
                   int32_t gain_plus_one, const float* shift, int32_t rms, void* out, int32_t ldo,
                   void* stream);

/* Kernel timer for measurement: while `tag` is set, every launch of the
 * kernels behind that call site (tags: "vit.patch", "vit.qkv", "vit.attn",
 * "vit.o", "vit.fc1", "vit.fc2", "proj", "state", "lm.qkv", "lm.attn", "lm.o",
 * "lm.gateup", "lm.down", "ex.in", "ex.time1", "ex.time2", "ex.qkv",
 * "ex.attn", "ex.o", "ex.gateup", "ex.down", "ex.out"; DiT head also
 * "dit.cross_kv", "ex.q", "ex.fc1", "ex.fc2") records a pair of
 * HIP events at the start and end of its main kernel (hipExtLaunchKernel
 * start/stop events, on the launching stream; a separate split-K reduce or
 * attention-combine kernel is not included). NULL or "" turns it off.
 * _read waits for the recorded events, returns the summed duration (ms) and
 * the number of bracketed launches since the last read, and resets both. */
int vla_kernel_timer(vla_model* m, const char* tag);
int vla_kernel_timer_read(vla_model* m, double* total_ms, int64_t* launches);

/* Measurement: workgroup residency log. _enable allocates room for
 * `capacity` records and points every instrumented kernel of the process at
 * it (capacity 0 turns logging off and frees the buffer); call it with no
 * work in flight. While on, the first lane of each workgroup appends a
 * record when the workgroup starts and when it ends; each record is 24
 * bytes: uint64 time (100 MHz constant clock), uint32 HW_ID register (CU,
 * shader array, shader engine, queue), uint32 XCC_ID register, uint32
 * kernel kind (1 GEMM, 2 split-K reduce, 3 skinny GEMM, 4 LDS attention,
 * 5 attention combine, 6 cache attention, 7 norm, 8 patchify, 9 embed,
 * 10 convert), uint32 end flag. _read waits for the device, copies up to
 * max_records records written since the last read to host_dst, sets *n to
 * the number copied and restarts the log; it returns VLA_ESTATE when the
 * log overflowed (records past the capacity are lost).
 * One log per process and device: the last model to enable it owns it. */
int vla_wavelog_enable(vla_model* m, int64_t capacity);
int vla_wavelog_read(vla_model* m, void* host_dst, int64_t max_records, int64_t* n);

/* Host-only: values start .. start+n-1 of the library's parameter generator
 * for (seed, name) with the given mean and std, as fp32 (before any bf16
 * rounding) into host_dst. Needs no GPU. */
int vla_debug_generate(uint64_t seed, const char* name, int64_t n, double mean, double stdv,
                       float* host_dst);

/* Host-only test entry point: the launch plan that the phases' GEMMs and
 * vla_debug_gemm_epi get for an M x N x K product. kind is a VLA_DEBUG_EPI_* epilogue
 * (RESID_NORM: split-K partials for a norm); skinny = 1 plans the action
 * head's kernel (M <= 64 rows per frame), 0 the tiled one. plan_m (0: M) is
 * the row count the split factor is planned for and plan_batch the most
 * frames of plan_m rows one launch may stack (the phases plan a batched
 * prefill for one frame's rows with plan_batch 8, and the batched action
 * loops for 8 frames' rows with plan_batch 1). out (host int32[4])
 * receives the tile's rows and columns (0 and 32 for the skinny kernel), the
 * split-K factor and the workgroup count; scratch_floats (host, may be NULL)
 * the fp32 partials the launch needs. Needs no GPU. */
int vla_debug_gemm_plan(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t kind, int32_t skinny,
                        int32_t plan_m, int32_t plan_batch, int32_t* out, int64_t* scratch_floats);

/* Message for the last non-zero status on this thread ("" if none). */
const char* vla_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* VLA_H */
