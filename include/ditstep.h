/*
 * ditstep.h -- C ABI of the MI355X (gfx950) K-seed DiT denoise-step library.
 *
 * One denoising step of a diffusion transformer, run for the K seeds of a
 * prompt group (the rollout / seed-exploration unit of GRPO-style DiT RL
 * post-training: K samples per prompt from distinct seeds, Spotlight paper
 * section 2.1 and Fig. "fig:grpo"; every step is one forward pass of the DiT
 * backbone, section 2.1), followed by the flow-matching sampler update
 * (FlowGRPO backbone, section 5) and the per-prompt-group reward statistics
 * with seed ordering used for top/bottom seed selection (sigma_g of section
 * 4.3.2; top-k/bottom-k selection of section 5 "Dynamic Exploration").
 *
 * Conventions for every entry point
 *   - Tensors are caller-owned DEVICE pointers (hipMalloc / torch on the GPU)
 *     unless stated otherwise; the library never frees them and performs no
 *     device allocation on the hot path. Scratch memory comes from a
 *     caller-provided workspace whose size the *_workspace_bytes() calls give.
 *   - Every call is asynchronous on `stream` (a hipStream_t; NULL = the null
 *     stream), except group_reward_stats, which synchronises `stream` once
 *     to check its small input for NaN (group_reward_stats_async checks on the
 *     device instead).
 *   - Arguments are validated before any launch; on any error nothing is
 *     written, the status says why and dit_last_error_message() (per host
 *     thread) gives detail. Launch failures return DIT_ERR_HIP.
 *   - Layouts are row-major with the last index contiguous. Linear weights
 *     are stored [out][in] (both GEMM operands K-contiguous); biases [out].
 *   - Element types: DIT_BF16 = bfloat16 storage with fp32 accumulation and
 *     fp32 epilogue math; DIT_F32 = fp32 throughout. temb, the latent, the
 *     velocity, noise and rewards are always fp32.
 *   - Thread safety: no mutable global state besides the per-thread error
 *     text, per-device caches filled once (atomics: the device's compute
 *     unit count and the kernels' LDS limits) and the fixed scratch array of
 *     dit_timestep_embed_noalloc (one per GPU; overlapping calls of that entry
 *     point on one GPU race); calls on different streams with disjoint
 *     buffers may overlap, also on their first call.
 */
#ifndef DITSTEP_H
#define DITSTEP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DIT_ABI_VERSION 1

typedef enum {
  DIT_OK = 0,
  DIT_ERR_INVALID_ARG = 1,  /* NULL required pointer, negative size, k_select > n, ... */
  DIT_ERR_SHAPE = 2,        /* inconsistent shape (hidden != heads*head_dim, n_img != grid_h*grid_w, ...) */
  DIT_ERR_DOMAIN = 3,       /* flow_step: noise_level > 0 with t outside (0,1), or t_next > t, ... */
  DIT_ERR_NAN = 4,          /* group_reward_stats: a reward is NaN or infinite */
  DIT_ERR_UNSUPPORTED = 5,  /* valid but not implemented (head_dim not 64/128, hidden > 4096, ...) */
  DIT_ERR_HIP = 6,          /* a HIP runtime call or kernel launch failed */
  DIT_ERR_WORKSPACE = 7     /* workspace NULL, misaligned (256 B) or smaller than required */
} dit_status;

typedef enum { DIT_F32 = 0, DIT_BF16 = 1 } dit_dtype;

typedef void* dit_stream; /* hipStream_t */

/* Shape of one dual-stream MMDiT block (image stream + text stream, joint
 * attention). Sequence order inside the block is [text ; image]. */
typedef struct {
  int32_t hidden;      /* D = heads * head_dim, multiple of 64, <= 4096 */
  int32_t heads;       /* H */
  int32_t head_dim;    /* d, 64 or 128 */
  int32_t mlp_hidden;  /* F (4*D in the configurations used), multiple of 64 */
  int32_t n_img;       /* N_i image tokens = grid_h * grid_w */
  int32_t n_txt;       /* N_t text tokens (>= 0) */
  int32_t grid_h;      /* latent token grid (rows) */
  int32_t grid_w;      /* latent token grid (columns) */
  int32_t rope;        /* nonzero: 2D axial RoPE on image-token q and k */
  float ln_eps;        /* LayerNorm epsilon (1e-6) */
  float rope_theta;    /* RoPE base (1e4) */
  int32_t dtype;       /* dit_dtype of weights and activations */
} dit_block_config;

/* Weights of one block; index 0 = image stream, 1 = text stream. Element
 * type = config dtype. Shapes ([out][in]):
 *   mod_w [6D][D], mod_b [6D]   adaLN modulation, chunks in the order
 *                               shift1, scale1, gate1, shift2, scale2, gate2
 *   qkv_w [3D][D], qkv_b [3D]   rows [0,D) -> q, [D,2D) -> k, [2D,3D) -> v;
 *                               head j owns columns [j*d, (j+1)*d) of each
 *   out_w [D][D],  out_b [D]
 *   mlp1_w [F][D], mlp1_b [F]
 *   mlp2_w [D][F], mlp2_b [D] */
typedef struct {
  const void* mod_w[2];
  const void* mod_b[2];
  const void* qkv_w[2];
  const void* qkv_b[2];
  const void* out_w[2];
  const void* out_b[2];
  const void* mlp1_w[2];
  const void* mlp1_b[2];
  const void* mlp2_w[2];
  const void* mlp2_b[2];
} dit_block_weights;

/* Weights around the block stack for a full step (element type = config dtype):
 *   t1_w [D][256], t1_b [D], t2_w [D][D], t2_b [D]   timestep MLP
 *   in_w [D][C],   in_b [D]                          patch embedding, C = latent_dim
 *   fmod_w [2D][D], fmod_b [2D]                      final modulation (shift_f, scale_f)
 *   fout_w [C][D], fout_b [C]                        velocity head */
typedef struct {
  const void* t1_w;
  const void* t1_b;
  const void* t2_w;
  const void* t2_b;
  const void* in_w;
  const void* in_b;
  const void* fmod_w;
  const void* fmod_b;
  const void* fout_w;
  const void* fout_b;
} dit_step_weights;

/* ------------------------------------------------------------------ */
/* library                                                              */
/* ------------------------------------------------------------------ */
int32_t dit_abi_version(void);
const char* dit_status_string(dit_status s);
/* Detail of the last non-OK status returned on the calling host thread. */
const char* dit_last_error_message(void);

/* ------------------------------------------------------------------ */
/* one MMDiT block (the DiT forward pass is a stack of these)           */
/* ------------------------------------------------------------------ */
/* Bytes of workspace dit_block_forward / dit_block_mlp need for `batch`. */
size_t dit_block_workspace_bytes(const dit_block_config* cfg, int32_t batch);

/* One dual-stream MMDiT block, in place on both residual streams.
 * Source: every denoising step of the rollout is one full forward pass of the DiT
 * backbone, run for the K seeds of a prompt group (section 2.1, "Diffusion Models and
 * DiT RL Post-Training"); the backbone is Qwen-Image, a 20B MMDiT (section 6.1, "Model
 * Setup"). The paper does not restate the block, so its internals below (adaLN
 * modulation, joint attention, GELU-tanh MLP) are the dual-stream MMDiT reading, and
 * the sizes are those of the workloads the paper runs (512x512 and 1280x1280 images).
 *   temb  [B][D] fp32        per-sample conditioning vector
 *   x_img [B][N_i][D]        image residual stream (in/out), config dtype
 *   x_txt [B][N_t][D]        text residual stream (in/out), config dtype
 * Per stream s: (shift1..gate2) = W_mod SiLU(temb) + b_mod;
 *   h = LN(x)(1+scale1)+shift1; q,k,v = W_qkv h + b_qkv; RoPE on image q,k;
 *   o = softmax(q k^T / sqrt(d)) v over all S = N_t + N_i tokens, per head;
 *   x += gate1 * (W_o o + b_o); h2 = LN(x)(1+scale2)+shift2;
 *   x += gate2 * (W_2 GELU_tanh(W_1 h2 + b_1) + b_2).
 * workspace: device, 256-byte aligned, >= dit_block_workspace_bytes(). */
dit_status dit_block_forward(const dit_block_config* cfg, const dit_block_weights* w, int32_t batch,
                             const float* temb, void* x_img, void* x_txt,
                             void* workspace, size_t workspace_bytes, dit_stream stream);

/* Only the MLP half of dit_block_forward (modulation, then
 * x += gate2 * MLP(LN(x)(1+scale2)+shift2) on both streams). This is the
 * per-token part a sequence-parallel rank runs on its own token slice. */
dit_status dit_block_mlp(const dit_block_config* cfg, const dit_block_weights* w, int32_t batch,
                         const float* temb, void* x_img, void* x_txt,
                         void* workspace, size_t workspace_bytes, dit_stream stream);

/* Joint non-causal multi-head attention, o = softmax(q k^T * scale) v per
 * (sample, head), every query attending to all `seq` keys.
 * Source: the attention inside each block of the DiT forward pass (section 2.1); at
 * 1280x1280 the paper splits it over a sequence-parallel group (sections 2.1 and 4.4,
 * SP=2 in section 6.1), and one rank's share is a subset of the heads over the whole
 * sequence, which is what the head stride here addresses. Text and image tokens form one
 * sequence with no mask (the joint attention of an MMDiT; the paper does not restate it).
 * q, k, v: element (b, s, h, e) at base + b*qkv_stride_b + s*qkv_stride_s +
 *   h*qkv_stride_h + e (strides in ELEMENTS, e contiguous), so q/k/v may be
 *   slices of one packed [B][S][3][H][d] buffer.
 * o: element (b, s, h, e) at o + b*o_stride_b + s*o_stride_s + h*o_stride_h + e.
 * head_dim: 64 or 128. scale: usually 1/sqrt(head_dim). dtype: DIT_BF16
 * (bf16 MFMA, fp32 softmax) or DIT_F32. Pointers and strides must keep
 * 16-byte alignment of every (b, s, h) row. */
dit_status joint_attention(const void* q, const void* k, const void* v, void* o,
                           int32_t batch, int32_t heads, int32_t seq, int32_t head_dim,
                           int64_t qkv_stride_b, int64_t qkv_stride_s, int64_t qkv_stride_h,
                           int64_t o_stride_b, int64_t o_stride_s, int64_t o_stride_h,
                           float scale, int32_t dtype, dit_stream stream);

/* ------------------------------------------------------------------ */
/* sampler and reward statistics                                        */
/* ------------------------------------------------------------------ */
/* One flow-matching sampler step on n fp32 elements, in place on x.
 * h = t_next - t (<= 0; noise at t = 1, data at t = 0).
 *   noise_level == 0: x' = x + h v                              (Euler ODE)
 *   noise_level  > 0: sigma = a sqrt(t/(1-t)),
 *     x' = x + h (v + sigma^2/(2t) (x + (1-t) v)) + sigma sqrt(-h) noise  (SDE)
 * noise may be NULL iff noise_level == 0. Errors: DIT_ERR_DOMAIN if
 * noise_level < 0, t_next > t, t or t_next not finite, or noise_level > 0
 * with t outside (0,1) or t_next < 0. n == 0 is a no-op. */
dit_status flow_step(float* x, const float* v, const float* noise, int64_t n,
                     float t, float t_next, float noise_level, dit_stream stream);

/* Log-density of x_next under the SDE step's Gaussian transition from x (the per-sample
 * likelihood behind FlowGRPO's policy ratio; FlowGRPO is the paper's algorithm backbone,
 * section 5). With h = t_next - t and sigma = a sqrt(t/(1-t)) as in flow_step,
 *   mean = x + h (v + sigma^2/(2t) (x + (1-t) v)),  var = sigma^2 (-h),
 *   logp[b] = -sum_i (x_next - mean)^2 / (2 var) - n/2 log(2 pi var)
 * summed over the n_per_sample elements of sample b (rows of [batch][n_per_sample]
 * fp32 device arrays x, v, x_next). Output logp [batch] fp64 on the device; the sum is
 * taken in fp64 in a fixed order (one workgroup per sample), so it is deterministic.
 * Errors: DIT_ERR_DOMAIN unless noise_level > 0, 0 < t < 1 and t_next < t (the ODE step
 * has no density); DIT_ERR_INVALID_ARG for NULL pointers or negative sizes. batch == 0 or
 * n_per_sample == 0 writes zeros (n == 0) or nothing (batch == 0). */
dit_status flow_logprob(const float* x, const float* v, const float* x_next, int32_t batch,
                        int64_t n_per_sample, float t, float t_next, float noise_level, double* logp,
                        dit_stream stream);

/* Per prompt-group statistics over rewards [G][n] fp32 (row g = the n seeds
 * of prompt group g):
 *   mean[g] = sum_j r / n; std[g] = sqrt(sum_j (r - mean)^2 / n) (population);
 *   adv[g][j] = (r - mean) / (std + adv_eps);
 *   order[g][:] = seed indices by descending reward, ties by ascending index;
 *   selected[g][:] = order[g][0 : ceil(k/2)] then order[g][n - floor(k/2) : n].
 * Outputs (device): mean, std [G] fp32; adv [G][n] fp32; order [G][n] int32;
 * selected [G][k_select] int32. Any output may be NULL (skipped).
 * 1 <= n <= 4096; 0 <= k_select <= n. A NaN/Inf reward returns DIT_ERR_NAN
 * and writes nothing (the call synchronises `stream` to check). */
dit_status group_reward_stats(const float* rewards, int32_t groups, int32_t n, float adv_eps,
                              int32_t k_select, float* mean, float* std, float* adv,
                              int32_t* order, int32_t* selected, dit_stream stream);

/* group_reward_stats without the host synchronisation, for callers that keep the stream
 * asynchronous (a step loop, HIP graph capture): the finiteness check runs on the device. A
 * one-workgroup pass over the G x n rewards writes *status (device int32) = DIT_OK, or
 * DIT_ERR_NAN when any reward is NaN or infinite; the statistics kernel then writes its outputs
 * only when *status is DIT_OK, so on bad input nothing but *status is written. The caller reads
 * *status after synchronising. Same outputs, bit for bit, as group_reward_stats on finite input.
 * Arguments are validated on the host as there (DIT_ERR_INVALID_ARG, also for status NULL);
 * groups == 0 writes nothing, not even *status. */
dit_status group_reward_stats_async(const float* rewards, int32_t groups, int32_t n, float adv_eps,
                                    int32_t k_select, float* mean, float* std, float* adv,
                                    int32_t* order, int32_t* selected, int32_t* status,
                                    dit_stream stream);

/* ------------------------------------------------------------------ */
/* full denoise step                                                    */
/* ------------------------------------------------------------------ */
/* temb [B][D] fp32 = W_2 SiLU(W_1 e(t) + b_1) + b_2 with
 * e(t) = [cos(1000 t f_j) ; sin(1000 t f_j)], f_j = 10000^(-j/128), j < 128.
 * t: device [B] fp32. */
dit_status dit_timestep_embed(const dit_block_config* cfg, const dit_step_weights* w, int32_t batch,
                              const float* t, float* temb, void* workspace, size_t workspace_bytes,
                              dit_stream stream);

/* dit_timestep_embed for callers that cannot allocate (code under HIP graph capture, serving
 * loops and harnesses that forbid device allocation, callers with no workspace to hand): the
 * same kernels and result, with their scratch (the sinusoid, the hidden layer and the GEMV's
 * split input) in a fixed device array the library holds, DIT_TIMESTEP_SCRATCH_BYTES per GPU,
 * instead of a caller workspace. The call allocates nothing (no hipMalloc, no events).
 * DIT_ERR_UNSUPPORTED when batch and hidden need more than that array (the need is
 * batch * (256 + 2 hidden) * 4 bytes plus 64 * hidden bytes, each part rounded up to 256 bytes:
 * at hidden 3072, up to 156 samples). Every call on a GPU shares that GPU's array: calls that
 * overlap on one GPU (other streams, other host threads) race and must be serialised by the
 * caller. Nothing in the array needs to start at zero. */
#define DIT_TIMESTEP_SCRATCH_BYTES (4u << 20)
dit_status dit_timestep_embed_noalloc(const dit_block_config* cfg, const dit_step_weights* w, int32_t batch,
                                      const float* t, float* temb, dit_stream stream);

/* x_img [B][N_i][D] (config dtype) = W_in latent + b_in; latent [B][N_i][C] fp32. */
dit_status dit_patch_embed(const dit_block_config* cfg, const dit_step_weights* w, int32_t batch,
                           int32_t latent_dim, const float* latent, void* x_img,
                           void* workspace, size_t workspace_bytes, dit_stream stream);

/* v [B][N_i][C] fp32 = W_out (LN(x_img)(1+scale_f)+shift_f) + b_out,
 * (shift_f, scale_f) = W_f SiLU(temb) + b_f. */
dit_status dit_final_layer(const dit_block_config* cfg, const dit_step_weights* w, int32_t batch,
                           int32_t latent_dim, const float* temb, const void* x_img, float* v,
                           void* workspace, size_t workspace_bytes, dit_stream stream);

/* Workspace for dit_denoise_step (includes the residual streams and the adaLN modulation of up to
 * 8 blocks, which the step computes 8 blocks per GEMV launch). */
size_t dit_denoise_workspace_bytes(const dit_block_config* cfg, int32_t batch, int32_t latent_dim);

/* One K-seed denoise step: temb(t) -> patch embedding -> n_blocks blocks ->
 * velocity -> flow_step(t -> t_next, noise_level) in place on latent.
 *   t, t_next  the step's timestep and the next one (all K seeds share t)
 *   latent  [B][N_i][C] fp32 (in/out); x_txt [B][N_t][D] text hidden input
 *           (config dtype, read only); noise [B][N_i][C] fp32 (NULL iff
 *           noise_level == 0); v_out [B][N_i][C] fp32 velocity (may be NULL).
 *   blocks  host array of n_blocks weight sets. */
dit_status dit_denoise_step(const dit_block_config* cfg, const dit_step_weights* sw,
                            const dit_block_weights* blocks, int32_t n_blocks, int32_t batch,
                            int32_t latent_dim, float t, float t_next,
                            float noise_level, float* latent, const void* x_txt, const float* noise,
                            float* v_out, void* workspace, size_t workspace_bytes, dit_stream stream);

/* ------------------------------------------------------------------ */
/* TeaCache gate (fewer effective denoising steps, section 4.3.1)       */
/* ------------------------------------------------------------------ */
/* The exploration planner's effective step count s comes from TeaCache: the block stack's
 * output residual is cached and reused on steps whose block input barely moved. Here:
 *   h    = block 0's modulated image input LN(x_img)(1 + scale1) + shift1, [B][N_i][D];
 *   rel  = sum |h - h_prev| / sum |h_prev| over the whole batch (the K seeds of a batch
 *          run or skip together);
 *   acc += poly(rel), poly = coef[0] rel^(n-1) + ... + coef[n-1] (identity when n_coef == 0);
 *   the step reuses the residual while acc < threshold, else runs the blocks and acc = 0.
 * The first step of a state (no h_prev or no residual yet) and any step with force != 0
 * (e.g. the last) run the blocks and reset acc. Initialise a state with
 * dit_teacache_init; the caller owns it (host memory). */
typedef struct {
  double threshold;
  int32_t n_coef;          /* 0..8 */
  double coef[8];          /* rescale polynomial, highest power first */
  double accumulated;
  int32_t has_prev;        /* the cache holds h of an earlier step */
  int32_t has_residual;    /* the cache holds the residual of an earlier computed step */
} dit_teacache_state;

/* threshold >= 0, 0 <= n_coef <= 8 (coef may be NULL when n_coef == 0). */
dit_status dit_teacache_init(dit_teacache_state* st, double threshold, const double* coef, int32_t n_coef);
/* The gate alone (host): *run_blocks = 1 to run the blocks, 0 to reuse the residual; rel is
 * ignored when the state has no previous input or force != 0. */
dit_status dit_teacache_gate(dit_teacache_state* st, double rel, int32_t force, int32_t* run_blocks);
/* Device cache for one state: h_prev [B][N_i][D] (config dtype), residual [B][N_i][D] fp32 and
 * reduction scratch. 0 for an invalid config. */
size_t dit_teacache_cache_bytes(const dit_block_config* cfg, int32_t batch);
/* dit_denoise_step with the gate in front of the block stack (same arguments and workspace,
 * n_blocks >= 1). Computes h, updates the cache's h_prev, and either runs the blocks (then
 * stores the residual x_out - x_in) or adds the stored residual to the patch-embedded input.
 * *ran_blocks (may be NULL) receives the decision and *rel (may be NULL) the distance (NaN on
 * a step without a previous input). The decision needs the distance on the host, so the call
 * synchronises `stream` once. DIT_ERR_WORKSPACE if cache_bytes is too small. */
dit_status dit_denoise_step_teacache(const dit_block_config* cfg, const dit_step_weights* sw,
                                     const dit_block_weights* blocks, int32_t n_blocks, int32_t batch,
                                     int32_t latent_dim, float t, float t_next, float noise_level,
                                     float* latent, const void* x_txt, const float* noise, float* v_out,
                                     dit_teacache_state* state, int32_t force, void* cache,
                                     size_t cache_bytes, int32_t* ran_blocks, double* rel,
                                     void* workspace, size_t workspace_bytes, dit_stream stream);

/* ------------------------------------------------------------------ */
/* kernel timing (benchmark instrumentation)                            */
/* ------------------------------------------------------------------ */
/* One kernel class (a family of launches: "gemm_mlp_up_gelu", "attention",
 * ...) accumulated between dit_profile_begin and dit_profile_end. flops and
 * bytes are ALGORITHMIC totals over those launches (2*M*N*K per GEMM,
 * 4*B*H*S^2*d per attention, bytes each memory-bound kernel must move). */
typedef struct {
  char name[40];
  int32_t launches;
  double total_ms;   /* sum of per-launch durations, hipEvent pairs on the launch stream */
  double flops;
  double bytes;
} dit_kernel_stat;

/* Start recording: every library launch from now on is bracketed by a pair
 * of hipEvents on its stream. Process-wide; not for concurrent callers. */
dit_status dit_profile_begin(void);
/* Stop recording, wait for the recorded events, and write up to `capacity`
 * per-class totals (host array) plus their number to *count. */
dit_status dit_profile_end(dit_kernel_stat* stats, int32_t capacity, int32_t* count);

#ifdef __cplusplus
}
#endif
#endif /* DITSTEP_H */
