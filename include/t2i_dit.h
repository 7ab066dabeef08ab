/*
 * t2i_dit.h -- C ABI of the MI355X (gfx950) diffusion-transformer denoising step.
 *
 * ServerlessT2I (Sec. 4, Fig. "Flux function" and Fig. "workflow definition")
 * treats the base diffusion model as a stateless model function: it loads its
 * bf16 weights once, then each call takes `latents` and `prompt_embeds` and
 * returns `noise_pred`; an orchestrator loop calls it once per denoising step
 * and applies `denoise(noise_pred, latents)`.  The paper calls this inference
 * compute-bound (Sec. 3.1) and requires identical results under fixed seeds
 * (Sec. 4, "Function-as-a-Service Paradigm"; Sec. 8.1 checks that its system
 * produces the same images as the unmodified models).  This library is that
 * model function and its loop:
 *
 *   t2i_dit_init    load: bind the caller's device weights and workspace
 *   t2i_dit_step    one model evaluation (+ guidance, + optional Euler update)
 *   t2i_dit_sample  the whole denoising loop, with the optional step-skip cache
 *   t2i_cache_check the cache-skip decision of one step
 *
 * Conventions for every call:
 *   - Device pointers are HIP device memory owned by the caller; host pointers
 *     are ordinary host memory.  Each argument says which it is.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Launches are asynchronous on it; calls return before the GPU finishes,
 *     except where a call says it synchronises.
 *   - Every call validates all arguments before launching anything, returns a
 *     t2i_status and never aborts or throws; a failed call writes nothing.
 *     t2i_last_error() gives a message for the last failure on a handle.
 *   - A handle is used from one host thread and one stream at a time.  The
 *     library keeps no global mutable state; distinct handles are independent.
 *   - Identical inputs give bitwise-identical outputs (all reductions have a
 *     fixed order).
 */
#ifndef T2I_DIT_H
#define T2I_DIT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  T2I_OK = 0,
  T2I_ERR_INVALID_ARG = 1,   /* NULL pointer, bad enum, struct_size mismatch */
  T2I_ERR_SHAPE = 2,         /* sizes inconsistent with the config or limits */
  T2I_ERR_UNSUPPORTED = 3,   /* valid but not implemented for this configuration */
  T2I_ERR_WORKSPACE = 4,     /* workspace or cache state too small */
  T2I_ERR_OUT_OF_MEMORY = 5, /* host allocation failed */
  T2I_ERR_DEVICE = 6         /* a HIP call failed; t2i_last_error has its text */
} t2i_status;

typedef enum { T2I_F32 = 0, T2I_BF16 = 1 } t2i_dtype;
typedef enum { T2I_ARCH_CROSS_DIT = 0, T2I_ARCH_MMDIT = 1 } t2i_arch;
typedef enum { T2I_CACHE_ACCUMULATE = 0, T2I_CACHE_PER_STEP = 1 } t2i_cache_mode;

/* Most sequences one call may carry: requests times guidance branches. */
#define T2I_MAX_SEQ 64
/* Most requests one call may carry. */
#define T2I_MAX_REQ 32
#define T2I_MAX_CONTROL 64     /* entries of one t2i_control */

/*
 * Model shape.  `dtype` is the type of weights, text embeddings and of the
 * GEMM / attention operands; accumulation, the residual stream, LayerNorm,
 * softmax, modulation, the final layer and the sampler are always fp32.
 *
 * Architecture readings (the paper names the model families -- Flux, SD3.5,
 * Z-Image, Sec. 8.1 -- but fixes no architecture):
 *   T2I_ARCH_CROSS_DIT  adaLN-Zero DiT blocks: self-attention, cross-attention
 *                       to projected text (ungated, query from the raw
 *                       residual), MLP with tanh-GELU; fixed 2D sin-cos
 *                       position embedding.
 *   T2I_ARCH_MMDIT      joint attention over [text; image] with per-stream
 *                       weights and 2D RoPE on image queries and keys.
 */
typedef struct t2i_dit_config {
  uint32_t struct_size;      /* = sizeof(t2i_dit_config) */
  int32_t arch;              /* t2i_arch */
  int32_t dtype;             /* t2i_dtype */
  int32_t latent_channels;   /* C */
  int32_t patch;             /* p: tokens are p x p latent patches */
  int32_t hidden;            /* D, multiple of 64 */
  int32_t heads;             /* H, heads * head_dim == hidden */
  int32_t head_dim;          /* d, multiple of 8, <= 128 */
  int32_t depth;             /* number of blocks */
  int32_t mlp_hidden;        /* F, multiple of 64 */
  int32_t text_dim;          /* width of prompt_embeds, multiple of 64 */
  int32_t text_tokens;       /* tokens per prompt (>= 1) */
  int32_t freq_dim;          /* sinusoidal timestep width (even) */
  int32_t max_tokens;        /* most image tokens one call carries, summed over
                                requests and guidance branches; bf16 models
                                need 4*(rows+64)*hidden < 2^31, rows being
                                max_tokens plus the MMDiT text rows (the
                                attention's 32-bit byte offsets) */
  int32_t max_requests;      /* most requests per call, <= T2I_MAX_REQ */
  int32_t max_steps;         /* most steps of one t2i_dit_sample call */
  float ln_eps;              /* LayerNorm epsilon */
  float t_scale;             /* timestep multiplier before the sinusoid */
} t2i_dit_config;

typedef struct t2i_dit t2i_dit;  /* opaque handle, owned by the library */

/*
 * Weight table: the per-layer parameter lookup of the model function
 * (Sec. 5.3, "Layer Lookup Table").  t2i_dit_weight_count gives its length and
 * t2i_dit_weight_desc the name, shape (up to 4 dims, unused dims 0) and dtype
 * of entry i.  Linear weights are [out, in] row-major (the input dimension is
 * contiguous).  Returns 0 / T2I_ERR_* on a bad config or index.
 */
size_t t2i_dit_weight_count(const t2i_dit_config* cfg);
t2i_status t2i_dit_weight_desc(const t2i_dit_config* cfg, size_t i,
                               char name[64], int64_t shape[4], int32_t* dtype);

/* Device workspace the handle needs, in bytes (0 on a bad config). */
size_t t2i_dit_workspace_bytes(const t2i_dit_config* cfg);

/*
 * Device bytes of the cache-skip state for a request mix: n_req requests with
 * tokens_per_req[r] image tokens each (host array) and `branches` guidance
 * branches (1, or 2 under classifier-free guidance).
 */
size_t t2i_cache_state_bytes(const t2i_dit_config* cfg, int32_t n_req,
                             const int32_t* tokens_per_req, int32_t branches);

/*
 * Create a handle (the model function's load_model).
 *   weights   host array of t2i_dit_weight_count(cfg) device pointers, each to
 *             a tensor of the shape and dtype t2i_dit_weight_desc gives.
 *             Borrowed: they must stay valid and unchanged for the handle's
 *             life (t2i_dit_rebind_weights replaces them).
 *   workspace device buffer of ws_bytes >= t2i_dit_workspace_bytes(cfg),
 *             256-byte aligned, borrowed for the handle's life.
 * Touches no device memory; `stream` is unused and may be NULL.
 */
t2i_status t2i_dit_init(const t2i_dit_config* cfg, const void* const* weights,
                        void* workspace, size_t ws_bytes, void* stream,
                        t2i_dit** out);

/*
 * Create a handle that needs no workspace from the caller and allocates no
 * device memory: for callers that cannot allocate (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc).  Same as
 * t2i_dit_init, except that the workspace is a static device array of
 * T2I_STATIC_WORKSPACE_BYTES held by the library on every device it runs
 * on, until the process ends.
 *   Returns T2I_ERR_WORKSPACE when t2i_dit_workspace_bytes(cfg) exceeds
 *   T2I_STATIC_WORKSPACE_BYTES (small models and request mixes only: e.g.
 *   tiny models, or a 2-block 1152-wide DiT at 256 px), T2I_ERR_DEVICE when
 *   the array's device address cannot be obtained on the current device.
 *   The array belongs to the device that is current at this call.
 * Every handle created this way on one device shares that device's array:
 * calls on such handles (step, sample, cache check) that overlap in time race
 * on it, so serialise them (one stream, or events between streams).  The
 * array keeps the last call's contents; no call depends on them.
 */
#define T2I_STATIC_WORKSPACE_BYTES ((size_t)64 << 20)
t2i_status t2i_dit_init_static(const t2i_dit_config* cfg, const void* const* weights,
                               void* stream, t2i_dit** out);

/* Replace the weight pointers (same shapes and dtypes) of a live handle;
 * every block becomes resident (queued loads are waited for first). */
t2i_status t2i_dit_rebind_weights(t2i_dit* h, const void* const* weights,
                                  void* stream);

/*
 * Callback input of a step: the `control_outputs` input the paper's model
 * function declares with callback=True (Sec. 4, Fig. "Flux function";
 * Sec. 5, "Efficient and flexible data fetching"), consumed partway through
 * the forward pass -- the single-GPU half of ControlNet parallelization.
 * Entry i adds residuals[i], an fp32 [rows, hidden] device tensor in the
 * image-stream row order of hidden_out (branch-major, then request), to the
 * residual stream right after block blocks[i].  When ready != NULL and
 * ready[i] != NULL (a hipEvent_t recorded by the producer, possibly on
 * another stream), the step's stream waits on that event only at that point,
 * so the producer overlaps with the blocks before it.  blocks[] is strictly
 * increasing; entries at or past the last block that runs are rejected.
 * Requests whose blocks are skipped by the cache reuse their residual and get
 * no control input.  All pointers are borrowed for the duration of the call.
 */
typedef struct t2i_control {
  uint32_t struct_size;           /* = sizeof(t2i_control) */
  int32_t n;                      /* 1 .. T2I_MAX_CONTROL */
  const int32_t* blocks;          /* host [n] */
  const float* const* residuals;  /* host [n] of device pointers */
  void* const* ready;             /* host [n] of hipEvent_t (entries may be NULL), or NULL */
} t2i_control;

/*
 * One model evaluation for a batch of requests (the model function's
 * `execute`), with classifier-free guidance and an optional Euler update.
 *
 * Request r has a latent of [C, lat_h[r], lat_w[r]] fp32 (both multiples of
 * p); the latents of all requests are packed back to back in `latents`.
 * Under guidance (guidance != 1) every request runs a conditional branch on its
 * text and an unconditional branch on all-zero text embeddings, and
 * v = v_u + guidance * (v_c - v_u).
 */
typedef struct t2i_step_args {
  uint32_t struct_size;        /* = sizeof(t2i_step_args) */
  int32_t n_req;               /* 1 .. max_requests */
  const int32_t* lat_h;        /* host [n_req] */
  const int32_t* lat_w;        /* host [n_req] */
  const double* t;             /* host [n_req] model time of each request */
  const double* t_next;        /* host [n_req], or NULL: no Euler update;
                                  else latents += (t_next - t) * v in place */
  float* latents;              /* device, packed fp32 latents */
  const void* prompt_embeds;   /* device [n_req, text_tokens, text_dim], dtype */
  float guidance;              /* 1 = no guidance */
  float* noise_pred;           /* device, packed like latents, or NULL */
  int32_t n_blocks;            /* < 0: all blocks; else run only the first
                                  n_blocks (diagnostics; then the final layer
                                  reads the partial residual stream) */
  float* hidden_out;           /* device or NULL: receives the residual stream
                                  after the blocks, fp32 [rows, hidden], rows
                                  ordered branch-major then request; MMDiT
                                  appends the text stream after the image */
  const uint8_t* skip;         /* host [n_req] or NULL: 1 = reuse the cached
                                  residual instead of running the blocks */
  void* cache_state;           /* device or NULL: when given, computed requests
                                  store their residual for later skips */
  size_t cache_state_bytes;
  const t2i_control* control_outputs; /* callback input (see t2i_control), or NULL */
} t2i_step_args;

t2i_status t2i_dit_step(t2i_dit* h, const t2i_step_args* args, void* stream);

/*
 * Cache-skip decision of step `step` of an n_steps loop (reading of the
 * step-skip cache the paper names: the relative L1 change of block 0's
 * modulated input between consecutive steps, accumulated until it reaches
 * tau, first and last steps always computed).  Computes m_k from the current
 * latents, d_k = sum|m_k - m_{k-1}| / sum|m_{k-1}| per request with fp64
 * sums in a fixed order, updates the accumulator, stores m_k.  A check at
 * step 0 resets the request's state.  Synchronises `stream` once to return
 * the decisions in host memory.
 */
typedef struct t2i_cache_args {
  uint32_t struct_size;        /* = sizeof(t2i_cache_args) */
  int32_t n_req;
  const int32_t* lat_h;        /* host [n_req] */
  const int32_t* lat_w;        /* host [n_req] */
  const double* t;             /* host [n_req] */
  const float* latents;        /* device, packed fp32 latents */
  int32_t step, n_steps;       /* 0 <= step < n_steps */
  double tau;                  /* <= 0: never skip */
  int32_t mode;                /* t2i_cache_mode */
  int32_t branches;            /* 1, or 2 under guidance */
  void* cache_state;           /* device, t2i_cache_state_bytes() */
  size_t cache_state_bytes;
  double* rel_l1;              /* host [n_req] out: d_k (NaN at step 0) */
  uint8_t* skip;               /* host [n_req] out: 1 = skip the blocks */
} t2i_cache_args;

t2i_status t2i_cache_check(t2i_dit* h, const t2i_cache_args* args, void* stream);

/*
 * The denoising loop: for k = start_step .. n_steps-1, optionally a cache
 * check, then one step with the Euler update from t_k to t_{k+1}.
 * Conditioning (timestep embeddings and every block's modulation for every
 * step) and the text projections are computed once per call.
 */
typedef struct t2i_sample_args {
  uint32_t struct_size;        /* = sizeof(t2i_sample_args) */
  int32_t n_req;
  const int32_t* lat_h;        /* host [n_req] */
  const int32_t* lat_w;        /* host [n_req] */
  int32_t n_steps;             /* 1 .. max_steps */
  int32_t start_step;          /* resume point, 0 .. n_steps-1 */
  const double* timesteps;     /* host [(n_steps+1) * n_req], row k holds t_k
                                  of every request; NULL = t_k = 1 - k/n_steps */
  float* latents;              /* device, updated in place */
  const void* prompt_embeds;   /* device [n_req, text_tokens, text_dim] */
  float guidance;
  double cache_tau;            /* <= 0 disables the cache */
  int32_t cache_mode;          /* t2i_cache_mode */
  void* cache_state;           /* device, needed when cache_tau > 0 */
  size_t cache_state_bytes;
  uint8_t* skip_log;           /* host [n_steps * n_req] or NULL */
  double* rel_l1_log;          /* host [n_steps * n_req] or NULL */
} t2i_sample_args;

/* Synchronises `stream` once per step when cache_tau > 0, else never. */
t2i_status t2i_dit_sample(t2i_dit* h, const t2i_sample_args* args, void* stream);

/*
 * Layer residency: first-layers caching with progressive loading (Sec. 5.1,
 * "Caching the first layers", Eq. 1-2) over the weight table as a layer
 * lookup table (Sec. 5.3, "model weight virtualization").
 *
 * A block's weights are its t2i_dit_weight_desc entries [first_index + b *
 * n_tensors, first_index + (b + 1) * n_tensors).  Packed, tensor j of a block
 * sits at byte offsets[j] (256-byte aligned) of a block_bytes record.  The
 * host tier is the caller's page-locked host copy of every block, packed
 * [depth][block_bytes]; the arena is a device buffer of the same shape that
 * the library loads evicted blocks into (block b at b * block_bytes).
 *
 * A block is resident (its table entries point at device weights: the
 * caller's from init / rebind, or its arena record after a load), loading
 * (a copy into its arena record is queued, with an event recorded after it)
 * or evicted (its entries are unbound).  Eviction goes in reverse layer
 * order and loading in layer order, so the resident and loading blocks
 * always form a prefix.  A step or sample whose blocks include an evicted one
 * fails with T2I_ERR_INVALID_ARG before launching anything.  A loading block
 * is waited for on the call's stream only right before its first use: its
 * modulation rows and (cross-DiT) text K/V are then computed there instead of
 * up front, with the same kernels and arguments, so results are bitwise
 * those of a resident model.
 */

/* Bytes of one packed block; fills *first_index, *n_tensors and, when
 * offsets != NULL, offsets[n_tensors].  Returns 0 on a bad config. */
size_t t2i_dit_block_layout(const t2i_dit_config* cfg, int32_t* first_index,
                            int32_t* n_tensors, size_t* offsets);

/*
 * Register the host tier.  host_blocks: page-locked host memory (hipHostMalloc)
 * of depth * block_bytes bytes; arena: device memory, 256-byte aligned, of
 * arena_bytes >= depth * block_bytes.  Both are borrowed for the handle's life
 * (or until the next t2i_dit_host_tier).  Pageable host memory is rejected
 * (T2I_ERR_INVALID_ARG): copies from it would not overlap with compute.
 * Waits for loads still queued from an earlier registration.
 */
t2i_status t2i_dit_host_tier(t2i_dit* h, const void* host_blocks, void* arena,
                             size_t arena_bytes);

/*
 * Evict blocks [keep, depth), last block first (Sec. 5.3, elastic weight
 * eviction: reverse layer order keeps the first layers that let loading
 * overlap inference).  Needs a host tier.  Waits for queued loads of those
 * blocks to finish.  Frees nothing: the device memory the evicted blocks
 * were bound to goes back to its owner, who may reuse it once the work
 * queued on it (earlier steps) has completed.
 */
t2i_status t2i_dit_evict(t2i_dit* h, int32_t keep);

/*
 * Queue the load of every evicted block, in layer order, on copy_stream (a
 * hipStream_t as void*; use a stream other than the compute stream to
 * overlap): one host-to-device copy of block_bytes into the block's arena
 * record, then an event.  The blocks' table entries are rebound to the arena
 * at once, and later calls wait on the events.  *n_loaded (may be NULL)
 * receives the number of blocks queued.
 */
t2i_status t2i_dit_load_async(t2i_dit* h, void* copy_stream, int32_t* n_loaded);

/*
 * Prefix length to keep resident (Eq. 2): the fewest first layers of L
 * uniform layers (copy time t_load and inference time t_comp per layer, any
 * one unit) whose resident copy lets the copies of the others finish while
 * inference runs, so that the latency is L * t_comp.  Equals Eq. 2 when
 * t_load >= t_comp (the case the paper considers); otherwise 1, since with
 * nothing resident the first layer's copy always delays inference.  Returns
 * -1 when L < 1 or a time is not finite and positive.
 */
int32_t t2i_first_layers(int32_t L, double t_load, double t_comp);

/* Per-block state, host [depth]: 0 resident, 1 loading, 2 evicted.  A loading
 * block whose copy has finished is reported (and kept) as resident. */
t2i_status t2i_dit_block_state(t2i_dit* h, int32_t* state);

/*
 * Kernel timing (tracing aid).  When a class's bit is set in `class_mask`,
 * every launch of that class on a handle's calls is bracketed by two HIP
 * events recorded on the call's stream.  t2i_dit_profile resets the counters
 * (mask 0 disables timing); t2i_dit_profile_read synchronises on the last
 * recorded event and returns the summed device time and the launch count.
 */
typedef enum {
  T2I_K_GEMM_QKV = 0, T2I_K_ATTN_SELF = 1, T2I_K_GEMM_O = 2, T2I_K_GEMM_XQ = 3,
  T2I_K_ATTN_CROSS = 4, T2I_K_GEMM_XO = 5, T2I_K_LN = 6, T2I_K_GEMM_FC1 = 7,
  T2I_K_GEMM_FC2 = 8,
  T2I_K_EMBED = 9,    /* patch + position embedding of a step */
  T2I_K_FINAL = 10,   /* final layer + guidance + Euler update */
  T2I_K_CACHE = 11,   /* cache-skip signal and decision */
  T2I_K_COUNT = 12
} t2i_kernel_class;

t2i_status t2i_dit_profile(t2i_dit* h, uint32_t class_mask);
t2i_status t2i_dit_profile_read(t2i_dit* h, int32_t kernel_class, double* total_ms,
                                int64_t* launches);

void t2i_dit_destroy(t2i_dit* h);
const char* t2i_status_str(t2i_status s);
const char* t2i_last_error(const t2i_dit* h);

#ifdef __cplusplus
}
#endif
#endif /* T2I_DIT_H */
