/*
 * ebrl.h -- C ABI of the generation-stage policy forward on one MI355X.
 *
 * The paper's generation stage ingests each environment's observation and
 * produces its next action chunk (Section 2.1, "Embodied Models", and the
 * generation stage of Section 2.2): a vision-language backbone fuses image
 * patches and instruction tokens into a KV cache that an action head reads.
 * Batches are groups of environments that become ready together (Section
 * 4.2.2, intra-rollout simulation-generation pipeline), so every call takes
 * a ragged set of env ids.  The paper's per-stage GPU quota s (Section 4.3.1,
 * the GPU-CPU resource pool's (s, m) descriptor) maps to a stream whose
 * compute-unit mask covers a share of the chip; its memory budget m maps to
 * the KV-pool byte budget given at creation.
 *
 * Conventions for every call below:
 *  - Status: 0 (EBRL_OK) or a negative ebrl_status.  No exceptions cross the
 *    ABI.  ebrl_last_error() returns a per-policy message for the last
 *    failure.  A HIP runtime error is sticky: the policy then answers
 *    EBRL_E_HIP to every call until it is destroyed.
 *  - Memory: pointers documented "device" must point to memory on the
 *    policy's device; "host" pointers are ordinary CPU memory that is read
 *    before the call returns.  The caller owns all argument buffers; the
 *    library owns the weights, the paged KV pool and its scratch.
 *  - Asynchrony: compute is enqueued on the bound stream (ebrl_policy_bind_stream;
 *    default: the null stream) and the call returns after enqueueing.
 *    Device outputs are valid once that stream is synchronised.  Device
 *    inputs must stay unchanged until then.
 *  - Threading: one host thread per policy at a time.  Several policies may
 *    share a device on different streams.
 *  - Env ids: integers in [0, max_envs); a call's ids must be distinct.
 *    n == 0 is a no-op returning EBRL_OK.
 */
#ifndef EBRL_H
#define EBRL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ebrl_policy ebrl_policy;

typedef enum {
    EBRL_OK = 0,
    EBRL_E_INVALID = -1,      /* bad argument, shape, id, or unsupported preset */
    EBRL_E_OOM = -2,          /* device allocation or KV budget exhausted */
    EBRL_E_HIP = -3,          /* HIP runtime error (sticky) */
    EBRL_E_STATE = -4,        /* e.g. decode of an env that was never prefilled */
    EBRL_E_UNSUPPORTED = -5   /* call not available for this model (e.g. flow on an AR policy) */
} ebrl_status;

enum { EBRL_DTYPE_FP32 = 0, EBRL_DTYPE_BF16 = 1 };

/* Policy shape.  The paper names the model families (VLM backbone plus an
 * autoregressive or flow-matching action head, Section 2.1) but no sizes;
 * the presets are the five benchmark workloads' models. */
typedef struct ebrl_config {
    int32_t dtype;            /* EBRL_DTYPE_FP32: all fp32; EBRL_DTYPE_BF16: bf16
                                 weights, KV and GEMM operands, fp32 accumulate,
                                 softmax, residual stream, norms and logits */
    /* vision: n_cams cameras of img x img x 3 float32 pixels, square patches */
    int32_t n_cams, img, patch;
    /* optional ViT encoder before the decoder (0 layers = patch embedding
       straight into the decoder width) */
    int32_t vit_layers, vit_d, vit_heads, vit_mlp;
    /* decoder backbone */
    int32_t layers, d, q_heads, kv_heads, head_dim, mlp, vocab, n_lang;
    /* autoregressive action head (action_logits = 0: none) */
    int32_t action_logits, n_action_tokens, n_bins;
    /* flow-matching action expert (exp_layers = 0: none); adim <= 64 */
    int32_t exp_layers, exp_d, exp_heads, exp_mlp, chunk, adim, n_steps;
    /* capacity */
    int32_t max_envs;         /* env ids live in [0, max_envs); also max n per call */
    int32_t max_seq;          /* longest prefix T_e accepted by ebrl_prefill */
    int64_t kv_budget_bytes;  /* KV pool size; 0 = enough for every env at max_seq */
    double init_std;          /* weight init N(0, init_std^2); presets use 0.02 */
    /* world action model (Section 2.1): the expert also denoises frame_tokens
       latent future-frame tokens of frame_dim channels per env jointly with
       the action chunk (0 = actions only); frame_dim <= 64 */
    int32_t frame_tokens, frame_dim;
} ebrl_config;

/* Observation batch for ebrl_prefill.  Env i's prefix is its image tokens
 * (camera 0 patches in raster order, then camera 1, ...) followed by
 * lang_len[i] language tokens: T_i = (images ? n_cams * (img/patch)^2 : 0)
 * + lang_len[i] (ViT models emit one decoder token per patch). */
typedef struct ebrl_obs_batch {
    const float* images;      /* device float32 NHWC [n, n_cams, img, img, 3], or NULL
                                 for language-only prefixes */
    const int32_t* lang_ids;  /* device int32 [n, lang_stride], ids in [0, vocab) */
    const int32_t* lang_len;  /* host int32 [n], or NULL = n_lang for every env */
    int32_t lang_stride;      /* row stride of lang_ids in elements (>= every lang_len) */
} ebrl_obs_batch;

/* Paper: Section 2.1 names the model families; Section 6.1 the models the
 * workloads stand in for (no sizes are given, the presets are readings).
 * Fill *out with preset 1..5 (1 tiny fp32 VLA, 2 small bf16 VLA, 3 7B-class
 * bf16 VLA with ViT, 4 flow-matching expert on a GQA backbone, 5 world
 * action model: preset 4's backbone and expert denoising two future frames
 * of 7 x 7 latent tokens (32 channels) with the action chunk); capacity
 * fields get the workload's batch size and prefix length.  Returns
 * EBRL_E_INVALID for any other preset. */
int ebrl_config_preset(int32_t preset, ebrl_config* out);

/* Paper: Section 2.1 (the policy the generation stage runs); the KV budget
 * is the memory share m of a GPU-CPU resource pool (Section 4.3.1).
 * Create a policy on the current HIP device: validates *config, generates
 * the seeded random-init weights (Philox4x32-10 + Box-Muller, N(0, std^2),
 * bf16 by nearest-even rounding of the fp32 value), uploads them and
 * allocates the paged KV pool (16-token blocks) and scratch.  *out receives
 * the handle, or NULL on failure. */
int ebrl_policy_create(const ebrl_config* config, uint64_t seed, ebrl_policy** out);

/* Synchronises the bound stream and frees everything the policy owns. */
void ebrl_policy_destroy(ebrl_policy* p);

/* Paper: Section 4.3.1 (per-stage GPU quota s) and Section 5 (quotas fixed
 * when a worker is launched).
 * Create a stream restricted to the compute units whose bits are set in
 * cu_mask (n_words 32-bit words, bit k of word w = CU 32*w + k in the
 * runtime's enumeration) on `device`: the stand-in for the paper's per-stage
 * SM quota.  *out_stream receives a hipStream_t. */
int ebrl_stream_create_cu_masked(int32_t device, const uint32_t* cu_mask, uint32_t n_words,
                                 void** out_stream);
int ebrl_stream_destroy(void* stream);

/* Paper: Section 4.3.1 (the generation stage runs inside its quota).
 * All later calls on p enqueue on `stream` (a hipStream_t on p's device;
 * NULL = the null stream).  For a stream made by
 * ebrl_stream_create_cu_masked (and not yet destroyed) the GEMMs size their
 * tiles for the CUs its mask selects; results are bitwise the same on any
 * stream. */
int ebrl_policy_bind_stream(ebrl_policy* p, void* stream);

/* Paper: Section 2.1 (the backbone fuses observations into the KV cache the
 * action head consumes) and Section 4.2.2 (ragged groups of environments).
 * Encode n environments' observations into their KV caches (all decoder
 * layers) and remember each env's final-normed last prefix row for the
 * action head.  env_ids: host int32 [n].  Re-prefilling an env replaces its
 * cache.  Errors: EBRL_E_INVALID for bad ids/lengths/shapes or T_i >
 * max_seq, EBRL_E_OOM when the KV budget cannot hold the prefixes. */
int ebrl_prefill(ebrl_policy* p, const ebrl_obs_batch* obs, const int32_t* env_ids, int32_t n);

/* Paper: Section 2.1 (the action head produces the action from the cache),
 * Section 2.2 (generation produces each env's next action) and Section
 * 4.2.2 (ragged groups).
 * Autoregressive action decode for n prefilled envs: token t0 = argmax of
 * the 256-bin logits of the last prefix row, then six decode steps, each
 * feeding the previous token's action embedding at the next position.
 * Ties in the argmax go to the lowest bin.  Bin b maps to -1 + (2b+1)/256.
 * env_ids: host int32 [n].  out_tokens: device int32 [n, n_action_tokens];
 * out_actions: device float32 [n, n_action_tokens]; out_margin: device
 * float32 [n, n_action_tokens] (top-1 minus top-2 logit) or NULL.  The
 * action tokens' KV goes to scratch past the prefix, so repeated calls are
 * idempotent.  EBRL_E_STATE if an env has no prefix;
 * EBRL_E_UNSUPPORTED without an action head. */
int ebrl_decode_actions(ebrl_policy* p, const int32_t* env_ids, int32_t n, int32_t* out_tokens,
                        float* out_actions, float* out_margin);

/* Seeded noise streams (Philox4x32-10 counter word 3) of the denoising calls. */
#define EBRL_NOISE_STREAM_ACTIONS 3u
#define EBRL_NOISE_STREAM_FRAMES 4u

/* Paper: Section 2.1 (an action head that iteratively denoises the action
 * chunk from the backbone's cache) and Section 3.1 (the lightweight
 * denoising steps of generation).
 * Flow-matching action-chunk denoising for n prefilled envs: from
 * x_0 = noise, ten Euler steps x_{k+1} = x_k - v(x_k, tau_k)/10 with
 * tau_k = 1 - k/10, where v is the action expert attending to the env's
 * backbone KV cache layer by layer plus its own chunk tokens.
 * noise: device float32 [n, chunk, adim], or NULL to draw it on the device:
 * env e's chunk, flattened, takes element pairs (2j, 2j + 1) from
 * Philox4x32-10 with key (low, high word of the policy seed) and counter
 * (j, c_e, e, EBRL_NOISE_STREAM_ACTIONS), Box-Muller on u = (x + 1/2) 2^-32
 * of the first two output words in double, rounded to float; c_e counts
 * env e's earlier calls with NULL noise (0 after ebrl_policy_create), so an
 * env's noise does not depend on the other envs of a call.
 * out_actions: device float32 [n, chunk, adim] (may alias noise).
 * EBRL_E_UNSUPPORTED without an expert or for a world action model
 * (frame_tokens > 0: use ebrl_wam_denoise), EBRL_E_STATE for an env with
 * no prefix, EBRL_E_INVALID for a NULL out_actions. */
int ebrl_flow_denoise(ebrl_policy* p, const int32_t* env_ids, int32_t n, const float* noise,
                      float* out_actions);

/* Paper: Section 2.1 (world action models) and Section 6.1 (the DreamZero
 * workload).
 * World-action-model denoising (Section 2.1: a diffusion transformer that
 * jointly denoises latent future frames and the action chunk, each modality
 * with its own decoder): the same Euler schedule as ebrl_flow_denoise over
 * frame_tokens + chunk tokens per env -- frame latents at positions T_e ..
 * T_e + frame_tokens - 1, then the actions -- that attend to each other
 * without a mask and to the env's backbone cache.  Frame tokens enter
 * through W_fin [exp_d, frame_dim] and leave through the final norm and
 * W_fout [frame_dim, exp_d]; actions as in ebrl_flow_denoise.
 * frame_noise / out_frames: device float32 [n, frame_tokens, frame_dim];
 * action_noise / out_actions: device float32 [n, chunk, adim] (outputs may
 * alias their noise).  A NULL noise pointer draws that noise on the device
 * as ebrl_flow_denoise does, frames on EBRL_NOISE_STREAM_FRAMES; the env's
 * call count advances once per call that draws either.
 * EBRL_E_UNSUPPORTED unless frame_tokens > 0. */
int ebrl_wam_denoise(ebrl_policy* p, const int32_t* env_ids, int32_t n, const float* frame_noise,
                     const float* action_noise, float* out_frames, float* out_actions);

/* Message describing the last failure on p (never NULL; "" if none).
 * With p == NULL: the last failure of ebrl_policy_create on this thread. */
const char* ebrl_last_error(const ebrl_policy* p);

/* ---------------------------------------------------------------------
 * Inspection, for tests and the benchmark.  These synchronise the bound
 * stream and copy to host memory.
 * ------------------------------------------------------------------- */

enum {
    EBRL_STATE_H_LAST_PRE = 0,  /* float32 [d]: env's last prefix row before the final norm */
    EBRL_STATE_H_LAST = 1,      /* float32 [d]: the same row after the final RMSNorm */
    EBRL_STATE_K = 2,           /* KV dtype [T_e, kv_heads, head_dim]: layer's post-rotary keys */
    EBRL_STATE_V = 3,           /* KV dtype [T_e, kv_heads, head_dim]: layer's values */
    EBRL_STATE_FLOW_V0 = 4,     /* float32 [chunk, adim]: velocity at tau = 1 of the env's
                                   latest flow call */
    EBRL_STATE_PREFIX_LEN = 5,  /* int32 [1]: T_e, or 0 if the env has no prefix */
    EBRL_STATE_GRAPHS = 6       /* int32 [1]: HIP graphs the policy holds (decode graphs are kept per
                                   batch-size class, denoise graphs per batch size; env_id is
                                   ignored but must be in range) */
};

/* Copy one piece of env `env_id`'s state to host memory `out` (capacity
 * `bytes`); `layer` selects the decoder layer for K/V.  EBRL_E_INVALID if
 * `bytes` is too small or the indices are out of range. */
int ebrl_read_state(ebrl_policy* p, int32_t what, int32_t env_id, int32_t layer, void* out,
                    int64_t bytes);

/* Host-side weight generator, no device needed: tensor `tensor_id` with
 * `count` elements in its logical [out, in] row-major order, as stored
 * (bf16 bit patterns when bf16 != 0, else float32).  Tensor ids:
 * 1 patch embedding, 2 language embedding, 3 action-token embedding,
 * 4 action logits, 5 ViT position embedding, 6 ViT projector, 7 expert
 * action-in, 8/9 expert time-MLP, 10 expert action-out, 11 frame-latent
 * in, 12 frame-latent out; layer l of the
 * decoder / ViT / expert uses base 1000 / 2000 / 3000 + 16 l plus
 * 0 q, 1 k, 2 v, 3 o, 4 gate, 5 up, 6 down. */
int ebrl_generate_weight_host(uint64_t seed, uint32_t tensor_id, int64_t count, double std,
                              int32_t bf16, void* out);

/* Read back / overwrite a resident weight tensor in its logical [out, in]
 * layout and storage dtype (bytes must equal its size).  Writing lets tests
 * install special weights (zeros, one-hot).  EBRL_E_INVALID for an unknown
 * id or a size mismatch. */
int ebrl_read_weight(ebrl_policy* p, uint32_t tensor_id, void* out, int64_t bytes);
int ebrl_write_weight(ebrl_policy* p, uint32_t tensor_id, const void* in, int64_t bytes);

/* Per-kernel timing for roofline reports.  While enabled, every launch of
 * a kernel class whose bit (1 << class) is set in class_mask is bracketed by
 * HIP events on the bound stream, and its algorithmic FLOP and HBM bytes are
 * accumulated.  class_mask = 0 disables timing. */
enum {
    EBRL_K_GEMM = 0,            /* bf16/fp32 GEMMs of prefill, ViT and flow expert (M > 256) */
    EBRL_K_GEMM_SKINNY = 1,     /* decode GEMMs (M <= 256) */
    EBRL_K_ATTN_PREFILL = 2,    /* flash attention (prefill, ViT, flow) */
    EBRL_K_ATTN_DECODE = 3,     /* paged decode attention (split + combine) */
    EBRL_K_OTHER = 4,           /* norms, rotary/KV write, gathers, logits, flow update */
    EBRL_K_COUNT = 5
};
int ebrl_profile_enable(ebrl_policy* p, int32_t class_mask);
/* Totals since enable (and resets them when reset != 0).  Synchronises. */
int ebrl_profile_read(ebrl_policy* p, int32_t kernel_class, int64_t* launches, double* total_ms,
                      double* flop, double* bytes, int32_t reset);

#ifdef __cplusplus
}
#endif
#endif /* EBRL_H */
