/*
 * dif.h - C ABI of the step-pruned video-DiT denoise step on MI355X (gfx950).
 *
 * Problem (Sec. 3.1, Sec. 3.2, Sec. 4.3 of "Dynamic-in-Few-Step"): a T = 4
 * step few-step sampler visits timesteps t_1 (most noise) .. t_4.  Step t_i
 * runs its own structure: binary gates g_{t_i} keep or remove whole blocks,
 * attention heads and FFN hidden channels, and a gate multiplies the output
 * of the component it controls (gating equation, Sec. 3.2).  The trained
 * network is exported to one dense network per step (Sec. 3.2), and the
 * inference engine keeps the union of all steps' parameters plus per-step
 * index tables, gathering each step's active parameters (Sec. 4.3).  Given
 * latent video tokens z_t, the timestep t, the text context c and the step
 * structure, one denoise step returns the model prediction v_t (Sec. 4.2
 * "predicted clean data ... computed from the model prediction v_t").
 *
 * Block internals are not given by the paper (it names a Wan2.1 DiT,
 * Sec. 5.1).  The library implements a Wan2.1-style block:
 *   x += gate1 * (SelfAttn(RoPE(RMSNorm_D(q)), RoPE(RMSNorm_D(k)), v) Wo^T + bo)
 *        with q,k,v projected from LN(x) * (1 + scale1) + shift1
 *   x += CrossAttn(RMSNorm_D(q_c), RMSNorm_D(k_c), v_c) Wco^T + bco
 *        with q_c from LN_affine(x), k_c, v_c from the text context
 *   x += gate2 * (GELU_tanh(LN(x)(1 + scale2) + shift2) W1^T + b1) W2^T + b2)
 * where (shift1, scale1, gate1, shift2, scale2, gate2) = layer modulation +
 * e0(t), RMSNorm_D spans the full width D with pruned channels counted as
 * zeros, and a pruned head / channel contributes nothing.
 *
 * Conventions
 *   - Every call returns dif_status: 0 on success, a negative DIF_E_* code
 *     on error.  No C++ exception and no abort ever crosses this ABI.  After
 *     an error, dif_last_error() returns a thread-local description.
 *   - Device pointers are HIP device addresses owned by the caller (the
 *     library never frees them).  Host pointers are read during the call
 *     only, unless stated.  The library allocates no device memory: plan
 *     memory and workspaces are caller-provided, sized by the *_bytes calls.
 *   - Kernel launches are asynchronous on the caller's hipStream_t (NULL =
 *     the default stream).  A fault inside a kernel surfaces at the caller's
 *     next synchronisation, or as DIF_E_HIP from a later call.
 *   - Matrices are row-major, nn.Linear layout [out_features, in_features].
 *     "dtype" storage is bfloat16 (DIF_BF16) or float32 (DIF_F32); norm,
 *     bias, gain and modulation vectors are always float32.
 *   - Calls on one model/plan from several host threads must be serialised
 *     by the caller; distinct plans may be used concurrently on distinct
 *     streams with distinct workspaces.
 */
#ifndef DIF_H_
#define DIF_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t dif_status;
#define DIF_OK 0
#define DIF_E_ARG (-1)          /* null pointer, bad enum, bad scalar       */
#define DIF_E_SHAPE (-2)        /* inconsistent or unsupported sizes        */
#define DIF_E_MASK (-3)         /* mask entry not 0/1, or wrong length      */
#define DIF_E_UNSUPPORTED (-4)  /* (dtype, head_dim) pair or device arch     */
#define DIF_E_WORKSPACE (-5)    /* plan memory / workspace too small or misaligned */
#define DIF_E_HIP (-6)          /* a HIP runtime call failed                */

typedef enum { DIF_BF16 = 0, DIF_F32 = 1 } dif_dtype;

/* Model hyper-parameters.  Supported (dtype, head_dim): (BF16,128), (F32,64),
 * (F32,128).  dim == n_heads * head_dim; dim % 64 == 0; dim <= 8192 (BF16)
 * or 4096 (F32); patch_dim % 64 == 0; freq_dim even; grid_* >= 1. */
typedef struct dif_config {
  int32_t dim;          /* D  */
  int32_t n_heads;      /* H  */
  int32_t head_dim;     /* dh */
  int32_t ffn_dim;      /* F  */
  int32_t n_layers;     /* N  */
  int32_t patch_dim;    /* Cp: latent features per token */
  int32_t freq_dim;     /* sinusoidal timestep features (256) */
  int32_t grid_f, grid_h, grid_w; /* latent token grid; L = f*h*w */
  int32_t max_text_len; /* upper bound on Lc accepted by the calls */
  int32_t dtype;        /* dif_dtype */
  float eps;            /* LayerNorm / RMSNorm epsilon (1e-6) */
  float rope_theta;     /* RoPE base (10000) */
} dif_config;

/* One block's parameters (device pointers, caller-owned, must outlive the
 * model and every plan built from it).  W* are [D, D] dtype unless stated. */
typedef struct dif_layer_weights {
  const float* mod;                     /* [6, D]: shift1 scale1 gate1 shift2 scale2 gate2 */
  const void* self_wq; const void* self_wk; const void* self_wv; const void* self_wo;
  const float* self_bq; const float* self_bk; const float* self_bv; const float* self_bo; /* [D] */
  const float* self_gq; const float* self_gk;   /* RMSNorm gains [D] */
  const float* norm3_w; const float* norm3_b;   /* cross-attention LayerNorm affine [D] */
  const void* cross_wq; const void* cross_wk; const void* cross_wv; const void* cross_wo;
  const float* cross_bq; const float* cross_bk; const float* cross_bv; const float* cross_bo;
  const float* cross_gq; const float* cross_gk;
  const void* ffn_w1;   /* [F, D] */
  const float* ffn_b1;  /* [F]    */
  const void* ffn_w2;   /* [D, F] */
  const float* ffn_b2;  /* [D]    */
} dif_layer_weights;

/* The union-of-all-steps parameter set theta_union (Sec. 4.3). */
typedef struct dif_weights {
  const void* patch_w;  const float* patch_b;  /* [D, Cp], [D]           */
  const void* t_w1;     const float* t_b1;     /* [D, freq_dim], [D]     */
  const void* t_w2;     const float* t_b2;     /* [D, D], [D]            */
  const void* t_w3;     const float* t_b3;     /* [6D, D], [6D]          */
  const float* head_mod;                       /* [2, D]: shift, scale   */
  const void* head_w;   const float* head_b;   /* [Cp, D], [Cp]          */
  const dif_layer_weights* layers;             /* host array [n_layers], copied */
} dif_weights;

/* One step's structure g_t (Sec. 3.2: gate tensors [T, N_block], [T, N_head],
 * [T, N_channel], here one step's slice per layer).  Host memory, entries 0
 * or 1.  Self- and cross-attention heads are gated independently. */
typedef struct dif_step_masks {
  const uint8_t* block_keep;      /* [n_layers]            */
  const uint8_t* self_head_keep;  /* [n_layers * n_heads]  */
  const uint8_t* cross_head_keep; /* [n_layers * n_heads]  */
  const uint8_t* ffn_keep;        /* [n_layers * ffn_dim]  */
} dif_step_masks;

/* Kept widths of one layer in a plan (for FLOP accounting and tests). */
typedef struct dif_layer_info {
  int32_t block_keep;
  int32_t self_heads;   /* h   */
  int32_t cross_heads;  /* h_c */
  int32_t ffn_channels; /* f   */
  int32_t ffn_padded;   /* FFN width the GEMMs run: compact plans f rounded up
                           to 64; indexed plans 16-byte channel chunks holding
                           a kept channel, rounded up to 64 */
} dif_layer_info;

/* How a plan presents step t's active parameters to the kernels. */
#define DIF_PLAN_COMPACT 0 /* gathered once into contiguous per-step weights */
#define DIF_PLAN_INDEXED 1 /* read in place from theta_union through I_t    */

typedef struct dif_model dif_model;
typedef struct dif_plan dif_plan;
typedef struct ihipStream_t* dif_stream; /* == hipStream_t */

/* Description of the last error on the calling thread ("" if none). */
const char* dif_last_error(void);

/* Host-only validation (no HIP call): DIF_OK, DIF_E_ARG, DIF_E_SHAPE or
 * DIF_E_UNSUPPORTED for the config; DIF_E_MASK for masks. */
dif_status dif_validate_config(const dif_config* cfg);
dif_status dif_validate_masks(const dif_config* cfg, const dif_step_masks* masks);

/* Record the model: validates cfg and that every weight pointer is non-null,
 * copies the layer array, checks the current device is gfx950 (else
 * DIF_E_UNSUPPORTED).  No device memory is allocated or copied. */
dif_status dif_model_create(const dif_config* cfg, const dif_weights* w, dif_model** out);
dif_status dif_model_destroy(dif_model* model);

/* Bytes of device plan memory dif_plan_step needs for these masks. */
dif_status dif_plan_bytes(const dif_model* model, const dif_step_masks* masks, size_t* bytes);

/* Build the per-step index tables I_t and gather step t's active parameters
 * into contiguous per-layer weights (Sec. 4.3; the "dense format" of
 * Sec. 3.2): kept q/k/v rows concatenated as one [3a, D] matrix, kept Wo
 * columns [D, a], the same for cross-attention, kept W1 rows / b1 entries
 * and W2 columns zero-padded to a multiple of 64 channels.  Kept indices
 * are in ascending order.  `step` is the structure's index in the sampler
 * (0-based, < 4096), kept for the caller's bookkeeping.
 *
 * t_s is the timestep the structure belongs to: the sampler pairs step i's
 * structure g_{t_i} with its timestep t_i (Sec. 3.1 fixes the T = 4
 * timesteps, Sec. 3.2 gives each of them its own gates).  The plan stores
 * t_s, and dif_step_forward / dif_step_forward_cached / dif_rollout /
 * dif_rollout_cached return DIF_E_ARG for any other timestep (exact float
 * comparison) unless the plan was built with DIF_PLAN_ANY_T.  t_s must be
 * finite (DIF_E_ARG) unless DIF_PLAN_ANY_T is set, where it is ignored.
 *
 * plan_mem: caller device memory of >= dif_plan_bytes bytes, 256-byte
 * aligned, which must stay valid until dif_plan_destroy.  The gather
 * kernels and a small table upload are enqueued on `stream`; the host index
 * tables are owned by the plan.  Errors: DIF_E_ARG, DIF_E_MASK,
 * DIF_E_WORKSPACE (too small / misaligned), DIF_E_HIP. */
dif_status dif_plan_step(const dif_model* model, int32_t step, float t_s,
                         const dif_step_masks* masks, void* plan_mem, size_t plan_bytes,
                         dif_stream stream, dif_plan** out);

/* Plan flags of dif_plan_step_ex. */
#define DIF_PLAN_ANY_T 1 /* the plan runs at any timestep (t_s is not checked) */

/* Plan of either kind (DIF_PLAN_COMPACT with flags 0 is dif_plan_step).
 *
 * DIF_PLAN_INDEXED keeps only theta_union and the index tables I_t, as the
 * paper's inference engine does (Sec. 4.3, Fig. 2(c)): the GEMMs gather
 * kept q/k/v, cross-q/k/v and W1 rows (and their biases and QK-norm gains)
 * by row index, and read the kept columns of Wo, cross-Wo and W2 as
 * 16-byte chunks through a chunk table, so no weight is copied and plan
 * memory is the tables plus the RoPE table (kilobytes per layer).  FFN
 * channels are taken in chunks of 16 bytes (8 bf16 / 4 float32 channels,
 * the paper's C = 8 chunks at bf16; App. A): a chunk with any kept channel
 * is run whole with its dropped channels zeroed, so the result equals the
 * compact plan's (exactly, when every chunk is wholly kept or dropped, as
 * with C = 8 gates).  Requires ffn_dim % 8 == 0 and ffn_dim <= 65536
 * (bf16) / 32768 (float32), else DIF_E_UNSUPPORTED.  The union weights
 * must stay valid and unchanged while the plan is used.  flags: 0 or
 * DIF_PLAN_ANY_T (other bits: DIF_E_ARG).  Other arguments, ownership and
 * errors as dif_plan_step; an unknown kind is DIF_E_ARG. */
dif_status dif_plan_bytes_ex(const dif_model* model, const dif_step_masks* masks, int32_t kind,
                             size_t* bytes);
dif_status dif_plan_step_ex(const dif_model* model, int32_t step, float t_s,
                            const dif_step_masks* masks, int32_t kind, int32_t flags,
                            void* plan_mem, size_t plan_bytes, dif_stream stream, dif_plan** out);

/* The timestep a plan is bound to and its flags (host only). */
dif_status dif_plan_timestep(const dif_plan* plan, float* t_s, int32_t* flags);

/* Frees the plan's host metadata only (plan_mem stays the caller's).  The
 * caller must synchronise `stream` before freeing plan_mem. */
dif_status dif_plan_destroy(dif_plan* plan);
dif_status dif_plan_layer_info(const dif_plan* plan, int32_t layer, dif_layer_info* out);

/* Bytes of device workspace dif_block_forward / dif_step_forward need for
 * B samples of L video tokens and Lc text tokens. */
dif_status dif_workspace_bytes(const dif_model* model, int32_t B, int32_t L, int32_t Lc,
                               size_t* bytes);

/* Timestep embedding: e [D] and e0 [6, D] (float32 device outputs) for
 * timestep t.  Uses the workspace's scratch. */
dif_status dif_time_embed(const dif_model* model, float t, float* e_out, float* e0_out,
                          void* ws, size_t ws_bytes, dif_stream stream);

/* One block (layer `layer`) of the plan's step structure, in place on the
 * residual stream x [B, L, D] (dtype).  ctx [B, Lc, D] (dtype) text tokens,
 * e0 [6, D] float32 step modulation (B samples share the step, Sec. 2.2:
 * routing that depends only on the step allows plain batching).  L must
 * equal grid_f*grid_h*grid_w (the RoPE grid); 1 <= Lc <= max_text_len.
 * A block whose gate is 0 leaves x unchanged and launches nothing. */
dif_status dif_block_forward(const dif_plan* plan, int32_t layer, void* x, const void* ctx,
                             const float* e0, int32_t B, int32_t L, int32_t Lc,
                             void* ws, size_t ws_bytes, dif_stream stream);

/* One denoise step: model prediction v [B, L, Cp] (float32) for latents
 * z [B, L, Cp] (float32) at timestep t under the plan's structure:
 * timestep embedding, patch embedding, the N blocks, output head.  t must
 * be the plan's t_s unless the plan has DIF_PLAN_ANY_T (DIF_E_ARG). */
dif_status dif_step_forward(const dif_plan* plan, const float* z, float t, const void* ctx,
                            int32_t B, int32_t L, int32_t Lc, float* v_out,
                            void* ws, size_t ws_bytes, dif_stream stream);

/* Cross-attention text cache.  The text keys and values of every layer
 * depend on the context and the layer only, not on the timestep or the
 * step's structure (Sec. 3.2 routes by step; the context is fixed over the
 * few-step chain of Sec. 4.2), so they can be projected once per context
 * for all heads and shared by the steps of a rollout.  Each step then takes
 * its kept heads from the cache and applies its key RMSNorm (over all D
 * channels, pruned ones counting as zero, as without the cache), with
 * results identical to the calls that take ctx.
 *
 * dif_text_cache_bytes: device bytes of the cache for B samples of Lc text
 * tokens (per layer B*Lc*D keys and B*D*round_up(Lc, 64) transposed values
 * in the model dtype, plus one B*Lc*D staging buffer).
 * dif_text_cache_build: fills `cache` (caller-owned device memory, 256-byte
 * aligned, cache_bytes >= the size above) from ctx [B, Lc, D] (dtype),
 * enqueued on `stream`; 4*B*Lc*D*D*n_layers flops.  The cache stays valid
 * while the model's weights and the context are unchanged.
 * Errors: DIF_E_ARG (null model / ctx / cache, misaligned cache),
 * DIF_E_SHAPE (B < 1, Lc outside [1, max_text_len]), DIF_E_WORKSPACE (cache
 * too small), DIF_E_HIP. */
dif_status dif_text_cache_bytes(const dif_model* model, int32_t B, int32_t Lc, size_t* bytes);
dif_status dif_text_cache_build(const dif_model* model, const void* ctx, int32_t B, int32_t Lc,
                                void* cache, size_t cache_bytes, dif_stream stream);

/* dif_block_forward / dif_step_forward reading the text keys and values from
 * a cache built for the same model, B and Lc (which the library cannot check:
 * a cache of another model or context gives that model's / context's
 * result).  Same results, bit for bit, as the calls with that context.
 * Errors: those of the calls with a context, and DIF_E_ARG / DIF_E_WORKSPACE
 * for a null, misaligned or too small cache. */
dif_status dif_block_forward_cached(const dif_plan* plan, int32_t layer, void* x, const void* cache,
                                    size_t cache_bytes, const float* e0, int32_t B, int32_t L,
                                    int32_t Lc, void* ws, size_t ws_bytes, dif_stream stream);
dif_status dif_step_forward_cached(const dif_plan* plan, const float* z, float t, const void* cache,
                                   size_t cache_bytes, int32_t B, int32_t L, int32_t Lc,
                                   float* v_out, void* ws, size_t ws_bytes, dif_stream stream);

/* Euler update between sampler steps, in place: z += (sigma_to - sigma_from) * v,
 * n float32 elements. */
dif_status dif_euler(float* z, const float* v, float sigma_from, float sigma_to, int64_t n,
                     dif_stream stream);

/* Clean-estimate and re-noise update between sampler steps (the student's
 * single-step clean prediction and the re-noising of Sec. 3.1 / Sec. 4.2,
 * with sigma = 1 - tau), in place on n float32 elements:
 *   x_hat = z - sigma_from * v;   z = (1 - sigma_to) * x_hat + sigma_to * eps.
 * eps (device, n float32, caller-drawn noise) may be null only when
 * sigma_to == 0, which leaves z = x_hat.  Errors: DIF_E_ARG (null z / v,
 * non-finite sigma_from, sigma_to outside [0, 1], eps missing), DIF_E_SHAPE
 * (n < 0), DIF_E_HIP. */
dif_status dif_renoise(float* z, const float* v, float sigma_from, float sigma_to, const float* eps,
                       int64_t n, dif_stream stream);

#define DIF_SAMPLER_EULER 0   /* z += (sigma_{s+1} - sigma_s) v                         */
#define DIF_SAMPLER_RENOISE 1 /* x_hat = z - sigma_s v; z = (1 - sigma_{s+1}) x_hat + sigma_{s+1} eps_s */

/* The student applied step after step from its current state to the last
 * step (the output rollout of Sec. 4.2 and Fig. 2(b)): for i < n_steps,
 * v = step(plans[i], z, timesteps[i]) then the sampler update from
 * sigma = timesteps[i] / 1000 to timesteps[i+1] / 1000 (0 after the last).
 * The last update of either sampler leaves the clean estimate z - sigma v.
 * Start mid-chain by passing the remaining plans and timesteps.  eps[i]
 * (device, B*L*patch_dim float32) is the re-noise of transition i, needed
 * for i < n_steps - 1 with DIF_SAMPLER_RENOISE (eps itself may be null for
 * DIF_SAMPLER_EULER).  z [B, L, Cp] float32 in place; v_scratch: device
 * float32 of the same size; ctx, ws, ws_bytes, B, L, Lc as for
 * dif_step_forward.  Everything is enqueued on `stream`.  Errors: those of
 * dif_step_forward and dif_renoise, DIF_E_ARG for null plans / timesteps,
 * unknown sampler, plans of different models. */
dif_status dif_rollout(const dif_plan* const* plans, const float* timesteps, int32_t n_steps,
                       int32_t sampler, float* z, const float* const* eps, const void* ctx,
                       int32_t B, int32_t L, int32_t Lc, float* v_scratch, void* ws,
                       size_t ws_bytes, dif_stream stream);

/* dif_rollout with the text keys and values read from a cache built by
 * dif_text_cache_build for the same model, B and Lc: every step shares the
 * one projection of the context.  Errors: those of dif_rollout and of
 * dif_step_forward_cached. */
dif_status dif_rollout_cached(const dif_plan* const* plans, const float* timesteps, int32_t n_steps,
                              int32_t sampler, float* z, const float* const* eps, const void* cache,
                              size_t cache_bytes, int32_t B, int32_t L, int32_t Lc,
                              float* v_scratch, void* ws, size_t ws_bytes, dif_stream stream);

/* Hard gates of one step from its continuous masks (Sec. 4.1): block gate
 * 1 iff m_block[l] > 0; a head is kept iff the mean of its head_dim mask
 * values is > 0 (summed in double, in index order); FFN channels form
 * consecutive chunks of `chunk` (the paper uses C = 8) and chunk c of layer
 * l is kept iff m_ffn[l * (ffn_dim / chunk) + c] > 0.  Comparisons are
 * strict, so 0 (and NaN) prunes.  Host memory, no HIP call:
 *   m_block [n_layers], m_self / m_cross [n_layers * dim] (head h owns
 *   entries h*head_dim ..), m_ffn [n_layers * ffn_dim / chunk] float32 in;
 *   block_keep [n_layers], self_head_keep / cross_head_keep
 *   [n_layers * n_heads], ffn_keep [n_layers * ffn_dim] uint8 out — the
 *   dif_step_masks arrays of that step.
 * Errors: those of dif_validate_config, DIF_E_ARG (null), DIF_E_SHAPE
 * (chunk < 1 or ffn_dim not a multiple of chunk). */
dif_status dif_hard_gates(const dif_config* cfg, int32_t chunk, const float* m_block,
                          const float* m_self, const float* m_cross, const float* m_ffn,
                          uint8_t* block_keep, uint8_t* self_head_keep, uint8_t* cross_head_keep,
                          uint8_t* ffn_keep);

/* FFN channel reordering before chunking (App. A): sorts layer `layer`'s
 * hidden channels by decreasing L2 norm of their weights — W1 row, b1 entry
 * and W2 column, norms in double, ties in index order — and writes the
 * permuted W1 rows to w1_out [ffn_dim, dim], b1 to b1_out [ffn_dim] and W2
 * columns to w2_out [dim, ffn_dim] (device, caller-owned, model dtype /
 * float32), and the permutation to perm_out [ffn_dim] (host: channel i of
 * the outputs is channel perm_out[i] of the model).  Permuting the three
 * together leaves the block's function unchanged, so the outputs can stand
 * in for the layer's FFN weights in a new model.  scratch: device memory of
 * >= ffn_dim * 12 bytes, 8-byte aligned.  The model's weights are only
 * read.  The call synchronises `stream` (the sort runs on the host).
 * Errors: DIF_E_ARG (null, layer out of range), DIF_E_WORKSPACE, DIF_E_HIP. */
dif_status dif_ffn_reorder(const dif_model* model, int32_t layer, void* w1_out, float* b1_out,
                           void* w2_out, int32_t* perm_out, void* scratch, size_t scratch_bytes,
                           dif_stream stream);

/* ------------------------------------------------------------------------
 * Operator-level entry points: the hot kernels on their own, for tests and
 * benchmarks of a single kernel.
 * ---------------------------------------------------------------------- */

/* Epilogues of dif_gemm: C = A B^T (+ bias) then
 *   DIF_EPI_STORE:    C = acc + bias
 *   DIF_EPI_GELU:     C = GELU_tanh(acc + bias)
 *   DIF_EPI_RESIDUAL: C += (gate0 + gate1) * (acc + bias), gate* per column
 *                     (gate0 == NULL: gate 1)  */
typedef enum { DIF_EPI_STORE = 0, DIF_EPI_GELU = 1, DIF_EPI_RESIDUAL = 2 } dif_epilogue;

/* C[M, N] (out_dtype) = epilogue(A[M, K] B[N, K]^T), A and B in `dtype`,
 * float32 accumulation.  K % 64 == 0 for BF16, K % 32 == 0 for F32; K may
 * be 0 (acc = 0).  Leading dimensions in elements: lda >= K and ldb >= K,
 * multiples of 16 bytes; ldc >= N (rows of 4-element-aligned C take the
 * vector path); 256 rows of A, B or C must span less than 2 GiB
 * (DIF_E_SHAPE otherwise).  bias [N] float32 or NULL.  out_dtype = dtype
 * or DIF_F32. */
dif_status dif_gemm(int32_t dtype, int32_t out_dtype, const void* A, int64_t lda,
                    const void* B, int64_t ldb, void* C, int64_t ldc,
                    int32_t M, int32_t N, int32_t K, int32_t epilogue, const float* bias,
                    const float* gate0, const float* gate1, dif_stream stream);

/* Flash attention, bidirectional, scale 1/sqrt(head_dim):
 * O[b, i, h*dh:(h+1)*dh] = softmax_j(Q_bih . K_bjh / sqrt(dh)) V_bjh.
 * Q: row (b*Lq + i), column h*dh, row stride ldq.  K: row (b*Lk + j),
 * row stride ldk.  V is given transposed: Vt[(b*n_heads + h)*dh + d][j],
 * row stride ldvt >= Lk (ldvt a multiple of 16 bytes).  O like Q with
 * stride ldo.  1 <= Lk; head_dim 128 (BF16) or 64/128 (F32). */
dif_status dif_attention(int32_t dtype, int32_t head_dim, const void* Q, int64_t ldq,
                         const void* K, int64_t ldk, const void* Vt, int64_t ldvt,
                         void* O, int64_t ldo, int32_t B, int32_t Lq, int32_t Lk,
                         int32_t n_heads, dif_stream stream);

/* Flags of dif_attention_ex. */
#define DIF_ATTN_Q_PRESCALED 1 /* Q already holds q * log2(e) / sqrt(head_dim) */

/* Bytes of the split workspace dif_attention_ex may use (any Lq, Lk, B,
 * n_heads).  DIF_E_UNSUPPORTED for a head_dim other than 64 / 128. */
dif_status dif_attention_split_bytes(int32_t head_dim, size_t* bytes);

/* dif_attention as the blocks launch it, for operator tests and
 * benchmarks of that exact launch: the attention of the block's
 * self-attention (softmax(Q K^T / sqrt(dh)) V, bidirectional, Sec. 3.2's
 * pruned structure only changes n_heads).
 *   flags & DIF_ATTN_Q_PRESCALED: Q holds the queries already multiplied by
 *     log2(e)/sqrt(head_dim) (the block's QK-norm writes them so); the
 *     kernel then takes its scores as base-2 exponents directly.  The result
 *     is softmax(Q K^T ln 2) V for the given Q.  Other flag bits: DIF_E_ARG.
 *   split_ws (device, >= dif_attention_split_bytes, 256-byte aligned) or
 *     NULL: with a workspace, when the last round of workgroups on this
 *     device would run at most half full, those work items run as two key
 *     halves each whose partial sums a second kernel merges (as the blocks
 *     do for bfloat16 with Lk >= 4096).  The result equals the unsplit
 *     launch's up to float rounding.  Calls sharing a workspace must not
 *     overlap.
 * Every other argument, layout and error as dif_attention; DIF_E_WORKSPACE
 * for a too small or misaligned split_ws; DIF_E_HIP if the device's compute
 * unit count cannot be read. */
dif_status dif_attention_ex(int32_t dtype, int32_t head_dim, int32_t flags, const void* Q,
                            int64_t ldq, const void* K, int64_t ldk, const void* Vt, int64_t ldvt,
                            void* O, int64_t ldo, int32_t B, int32_t Lq, int32_t Lk,
                            int32_t n_heads, void* split_ws, size_t split_ws_bytes,
                            dif_stream stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation):
 * dif_attention_ex with its key-split workspace taken from a buffer the
 * library keeps in static device memory, so the call allocates nothing.
 * The buffer is DIF_ATTN_STATIC_SCRATCH_BYTES (32.5 MiB) on every device
 * the library runs on, held until the process ends; it covers every problem
 * size (the split needs a fixed-size workspace, at most that, for head_dim
 * 64 and 128).  Every call on one device shares the buffer and leaves its
 * contents behind (each launch writes every entry it reads, nothing needs
 * clearing): calls that overlap on one device -- concurrent streams or host
 * threads -- race, and the caller must serialise them.  Arguments, results
 * and errors as dif_attention_ex with split_ws = the library's buffer;
 * DIF_E_HIP if its device address cannot be obtained. */
#define DIF_ATTN_STATIC_SCRATCH_BYTES ((size_t)34078720)
dif_status dif_attention_ex_static(int32_t dtype, int32_t head_dim, int32_t flags, const void* Q,
                                   int64_t ldq, const void* K, int64_t ldk, const void* Vt,
                                   int64_t ldvt, void* O, int64_t ldo, int32_t B, int32_t Lq,
                                   int32_t Lk, int32_t n_heads, dif_stream stream);

/* The matrix cores' sustained rate, for the roofline's context: launches
 * (on `stream`, asynchronously) a kernel that keeps every CU's matrix units
 * issuing one bf16 MFMA shape -- `shape` 0: v_mfma_f32_32x32x16_bf16 (the
 * attention kernels'), 1: v_mfma_f32_16x16x32_bf16 (the bf16 GEMM's) -- on
 * random operands, `iters` x 262144 FLOPs per wave (8 or 16 MFMAs; iters
 * rounded up to a multiple of 4; 300000 take about 0.1 s), two workgroups
 * of four waves per CU, with no memory traffic, and sets *flops to the FLOPs
 * it performs.  Time it with events on the same stream:
 * FLOPs / time is the rate the chip holds under its power limit with
 * nothing but MFMAs to do.  `shape` 2 measures the softmax's exponential
 * the same way: eight workgroups of four waves per CU, every lane
 * evaluating `iters` x 16 v_exp_f32 (sixteen independent chains
 * x <- 2^-x; 300000 take about 0.15 s), and *flops is set to the number of
 * exponentials.  `sink` is a device float the kernel may
 * write (it never does for any realistic result; it keeps the work from
 * being optimised away).  Errors: DIF_E_ARG for a shape other than 0, 1 or
 * 2, iters outside 1 .. 10^7 (a launch of a few seconds at most) or a null
 * pointer, DIF_E_UNSUPPORTED off gfx950. */
dif_status dif_mfma_probe(int32_t shape, int32_t iters, float* sink, double* flops,
                          dif_stream stream);

/* ------------------------------------------------------------------------
 * Kernel timing: while enabled, every kernel the library launches is
 * bracketed by HIP events on its stream, grouped by kind, with the kind's
 * algorithmic FLOPs and bytes.  dif_profile_collect synchronises on the
 * recorded events and returns, per kind, launches / total ms / FLOPs /
 * bytes.  Kinds are listed by dif_profile_kind_name(i) for i < DIF_PROF_KINDS.
 * ---------------------------------------------------------------------- */
#define DIF_PROF_KINDS 16
dif_status dif_profile_enable(int32_t on);
dif_status dif_profile_reset(void);
const char* dif_profile_kind_name(int32_t kind);
dif_status dif_profile_collect(int64_t* launches, double* total_ms, double* flops,
                               double* bytes); /* each an array of DIF_PROF_KINDS */

#ifdef __cplusplus
}
#endif
#endif /* DIF_H_ */
