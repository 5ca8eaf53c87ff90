/*
 * ff.h -- C ABI of the MI355X (gfx950) Flow-GRPO rollout library (libff.so).
 *
 * The library computes one data-parallel rollout step of a flow-matching
 * transformer as in Flow-Factory (arXiv 2602.12529):
 *   v = v_theta(x_t, c, t)                       -> ff_dit_forward
 *   x_{t+dt} by the Flow-GRPO SDE (Sec. 3.1, Eq. 1) -> ff_sde_step
 *   log-probability of the Gaussian transition    -> ff_sde_step / ff_logprob
 *   group-normalised advantages (Sec. 2.3)        -> ff_group_advantage
 *
 * Conventions shared by every entry point
 *   - Every pointer argument named as device memory must point to memory of
 *     the current HIP device; host pointers are marked "host".
 *   - The caller owns every buffer.  The library never allocates device
 *     memory: scratch space comes from the caller's `workspace`, whose size
 *     is given by the matching *_workspace_size call.  Workspace contents do
 *     not need to be initialised and are clobbered.
 *   - All work is enqueued asynchronously on `stream` (a hipStream_t; NULL is
 *     the legacy default stream).  Outputs are valid once the stream has
 *     been synchronised.  Arguments are validated on the host before any
 *     launch: a call that returns an error has enqueued nothing.
 *   - Return value: FF_OK (0) or a negative ff_status.  ff_last_error()
 *     returns a thread-local description of the last failure.
 *   - Tensors are dense, row-major, last index fastest.  Floating-point
 *     tensors are float32 (FF_F32) or bfloat16 (FF_BF16, stored as 16-bit
 *     words) as selected by the call's dtype.  Device pointers to float
 *     tensors must be 16-byte aligned.
 */
#ifndef FF_H
#define FF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FF_OK = 0,
  FF_EINVAL = -1,       /* null pointer, bad shape, bad dtype, misalignment */
  FF_EDOMAIN = -2,      /* time/noise arguments outside the SDE's domain     */
  FF_EWORKSPACE = -3,   /* workspace missing or smaller than required        */
  FF_EHIP = -4,         /* HIP runtime or launch error                       */
  FF_EUNSUPPORTED = -5  /* valid request outside the implemented limits      */
} ff_status;

typedef enum { FF_F32 = 0, FF_BF16 = 1 } ff_dtype;

/* Thread-local message describing the last non-OK return on this thread. */
const char* ff_last_error(void);
/* Library version string, e.g. "ff 0.1 gfx950". */
const char* ff_version(void);

/* ------------------------------------------------------------------------
 * SDE step and transition log-probability (Sec. 3.1, Eq. 1; Table 1)
 *
 * Time runs from t = 1 (noise) to t = 0 (data); a step goes from t to
 * t_next < t, so dt = t_next - t < 0.  With sigma = sigma_t of the chosen
 * schedule (Table 1), for every element of x, v, eps:
 *   mean   = x + [v + sigma^2/(2t) (x + (1-t) v)] dt
 *   x_next = mean + sigma sqrt(|dt|) eps
 * sigma = 0 is the deterministic ODE step x_next = x + v dt.
 *
 * The per-sample log-probability is the Gaussian density of the stored
 * x_next (after rounding to dtype) under N(mean, sigma^2 |dt| I), summed over
 * the D elements of the sample:
 *   logp[b] = -sum_d (x_next - mean)^2 / (2 sigma^2 |dt|)
 *             - D log(sigma sqrt(|dt|)) - (D/2) log(2 pi)
 * The element arithmetic is float32; the sum is accumulated in float64 in a
 * fixed order (the result is bitwise reproducible run to run), and the
 * recomputation by ff_logprob on the same tensors returns identical bits.
 * ------------------------------------------------------------------------ */

/* Workspace bytes needed by ff_sde_step / ff_logprob for a [B, D] batch. */
int ff_sde_workspace_size(int64_t B, int64_t D, size_t* bytes /* host, out */);

/* x, v, eps: device [B, D] of dtype.  x_next: device [B, D] of dtype; may not
 * alias x, v or eps.  logp: device float64 [B], or NULL to skip the
 * log-probability.  Domain: 0 <= t_next < t <= 1, sigma >= 0 finite, t > 0;
 * sigma = 0 requires logp == NULL (an ODE step has no density) -> FF_EDOMAIN.
 * B = 0 is a no-op returning FF_OK.  D = 0 (empty samples) reads no tensor and writes only
 * logp[b] = 0 when logp is given: the log-density above with no terms. */
int ff_sde_step(const void* x, const void* v, const void* eps, void* x_next, double* logp,
                int64_t B, int64_t D, double t, double t_next, double sigma, int32_t dtype,
                void* workspace, size_t ws_bytes, void* stream);

/* ff_sde_step for callers that cannot allocate device memory or pass a workspace (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation): the same step and
 * log-probability, bit for bit, with the log-probability's per-block partial sums kept in a
 * library-owned device array of 81920 doubles (640 KiB per device, held until the process ends,
 * its address looked up once per device on the first call there).  Arguments, domain and
 * errors as ff_sde_step, without the workspace.  No call allocates (no hipMalloc, no events, no
 * library allocation).  Every call on one device shares that array: calls that overlap on one
 * device (concurrent streams, other host threads) race and must be serialised by the caller.
 * The partial sums are all written before they are read, so nothing needs clearing between
 * calls.  B * blocks-per-sample above 81920 -> FF_EUNSUPPORTED (never reached for B <= 65535). */
int ff_sde_step_noalloc(const void* x, const void* v, const void* eps, void* x_next, double* logp,
                        int64_t B, int64_t D, double t, double t_next, double sigma, int32_t dtype,
                        void* stream);

/* Recomputes logp[b] for stored (x, v, x_next) exactly as ff_sde_step does (D = 0: logp[b] = 0).
 * sigma must be > 0 (FF_EDOMAIN otherwise). */
int ff_logprob(const void* x, const void* v, const void* x_next, double* logp,
               int64_t B, int64_t D, double t, double t_next, double sigma, int32_t dtype,
               void* workspace, size_t ws_bytes, void* stream);

/* The SDE step with the noise drawn on the device instead of read from memory
 * (Sec. 3.1: eps ~ N(0, I)), from the counter-based generator Philox4x32-10
 * (Salmon et al., SC 2011): element d of sample b takes word d % 4 of the block
 * with counter (d / 4 low word, d / 4 high word, b, step) under the key
 * (seed low, seed high), and each pair of words gives two normals by the
 * Box-Muller transform with u = (w + 1/2) 2^-32 (float32).  Same arguments,
 * domain, logp semantics and workspace as ff_sde_step; x_next may not alias
 * x or v.  The step reads 2 tensors and writes 1 instead of reading 3. */
int ff_sde_step_philox(const void* x, const void* v, void* x_next, double* logp, int64_t B, int64_t D,
                       double t, double t_next, double sigma, uint64_t seed, uint32_t step, int32_t dtype,
                       void* workspace, size_t ws_bytes, void* stream);

/* The noise ff_sde_step_philox uses, materialised: eps device [B, D] of dtype. */
int ff_philox_normal(void* eps, int64_t B, int64_t D, uint64_t seed, uint32_t step, int32_t dtype,
                     void* stream);

/* Raw Philox4x32-10 words: out device uint32 [n, 4], block i with counter
 * ((ctr_base + i) low word, (ctr_base + i) high word, c2, c3) and key (key low,
 * key high).  For checking the generator against its known-answer vectors. */
int ff_philox4x32(uint32_t* out, int64_t n, uint64_t ctr_base, uint32_t c2, uint32_t c3, uint64_t key,
                  void* stream);

/* ------------------------------------------------------------------------
 * Group-normalised advantages with multi-reward aggregation (Sec. 2.3)
 *
 * rewards: device float32 [N, K]; weights: device float32 [K];
 * group_id: device int32 [N], values in [0, n_groups).
 * mode 0 (weighted sum): r~ = sum_k w_k r_k;  adv = (r~ - mean_g) / (std_g + eps)
 * mode 1 (GDPO-style):   adv = sum_k w_k (r_k - mean_{g,k}) / (std_{g,k} + eps)
 * std is the population standard deviation of the group (ddof 0); statistics
 * are float64 and summed in sample order.  adv: device float32 [N].
 * group_count: device int32 [n_groups] receiving the group sizes, or NULL.
 * A sample whose group id is out of range gets adv = NaN and is counted in
 * no group.  Limits: 1 <= K <= 16, n_groups * K <= 4096, N <= 2^20 (FF_EUNSUPPORTED).
 * ------------------------------------------------------------------------ */
int ff_group_advantage(const float* rewards, const float* weights, const int32_t* group_id,
                       int64_t N, int32_t K, int32_t n_groups, int32_t mode, float eps,
                       float* adv, int32_t* group_count, void* stream);

/* ------------------------------------------------------------------------
 * DiT velocity field v_theta(x_t, c, t) (Eq. 1 / Eq. 2 notation)
 *
 * The paper names FLUX.1-dev, Qwen-Image and WAN as backbones but gives no
 * architecture; the implemented blocks are:
 *   dual-stream (MMDiT) block: per stream s in {txt, img},
 *     (sh1,sc1,g1,sh2,sc2,g2) = split6(W_mod,s SiLU(c) + b)
 *     QKV from Norm(X_s)(1+sc1)+sh1; per-head RMSNorm * w on Q, K; RoPE on
 *     image tokens; softmax(QK^T/sqrt(d))V over the joint [txt; img]
 *     sequence; X_s += g1 (O_s W_o^T + b);
 *     X_s += g2 (GELU_tanh((Norm(X_s)(1+sc2)+sh2) W_1^T + b) W_2^T + b)
 *   single-stream block on [txt; img]: (sh,sc,g) = split3(W_mod SiLU(c) + b);
 *     [QKV | U] = Mod(X) W_1^T + b; X += g ([O | GELU_tanh(U)] W_2^T + b)
 *   WAN block: LayerNorm modulation from E_block + e(t), full-width QK
 *     RMSNorm, 3D RoPE self-attention, cross-attention to the text context,
 *     GELU_tanh FFN.
 * Norm is RMSNorm (x / sqrt(mean x^2 + eps)) or LayerNorm without affine.
 * RoPE rotates adjacent pairs (2i, 2i+1); the head dimension is split into
 * three bands of widths rope_axes over the token's (frame, row, col) grid
 * position; pair i of band a turns by pos_a * rope_theta^(-2i/rope_axes[a]).
 * Text tokens have position 0 (no rotation).
 *
 * Size limits (FF_EUNSUPPORTED beyond them, checked on the host before any
 * allocation or launch): at most 4096 blocks of each kind; hidden <= 65536,
 * heads <= 1024, mlp_hidden <= 262144, in_channels, txt_dim, pooled_dim <=
 * 65536; per forward each grid axis <= 2^20, n_txt <= 2^20, n_prompts <=
 * 65535, and N_img, B (N_img + n_txt) and n_prompts n_txt <= 2^27 token rows.
 * No C++ exception leaves an entry point (a failed host allocation returns
 * FF_EUNSUPPORTED).
 * ------------------------------------------------------------------------ */

enum { FF_MODEL_MMDIT = 0, FF_MODEL_WAN = 1 };
enum { FF_IO_LATENT = 0, FF_IO_HIDDEN = 1 };
enum { FF_NORM_RMS = 0, FF_NORM_LN = 1 };

typedef struct ff_dit_config {
  int32_t model;        /* FF_MODEL_*                                            */
  int32_t io_mode;      /* FF_IO_LATENT: x is a latent [B,N_img,C], v is [B,N_img,C];
                           FF_IO_HIDDEN: block stack only, x is the image hidden
                           [B,N_img,H] and v is the stack's image-stream output   */
  int32_t dtype;        /* FF_F32 or FF_BF16: weights, activations, x and v       */
  int32_t n_dual;       /* dual-stream blocks                                     */
  int32_t n_single;     /* single-stream blocks (after the dual ones)             */
  int32_t n_wan;        /* WAN blocks (model == FF_MODEL_WAN)                     */
  int32_t hidden;       /* H = heads * head_dim                                   */
  int32_t heads;
  int32_t head_dim;     /* d: even; bf16 attention requires d == 128              */
  int32_t mlp_hidden;   /* F                                                      */
  int32_t in_channels;  /* C (latent channels per token)                          */
  int32_t txt_dim;      /* width of the cached prompt embeddings (LATENT mode)    */
  int32_t pooled_dim;   /* pooled-text width (MMDiT, LATENT), 0 = none            */
  int32_t norm_kind;    /* FF_NORM_RMS or FF_NORM_LN for the modulated norms      */
  int32_t rope_axes[3]; /* band widths, even, summing to head_dim                 */
  double rope_theta;
  double norm_eps;
} ff_dit_config;

typedef struct ff_dit ff_dit;

/* Number of parameter tensors of the model described by cfg. */
int ff_dit_num_tensors(const ff_dit_config* cfg, int64_t* n /* host, out */);

/* Name (NUL-terminated, at most name_cap bytes incl. NUL) and shape of
 * parameter tensor i.  Linear layers are "<prefix>.w" [out, in] (nn.Linear
 * layout) and "<prefix>.b" [out]; 1-D tensors report shape1 = 0. */
int ff_dit_tensor_info(const ff_dit_config* cfg, int64_t i, char* name, size_t name_cap,
                       int64_t* shape0, int64_t* shape1);

/* Creates a model handle.  tensors[i] is the device pointer of tensor i in
 * ff_dit_tensor_info order, of cfg->dtype, 16-byte aligned.  The handle keeps
 * the pointers (caller-owned, must outlive the handle) and a host copy of cfg. */
int ff_dit_create(const ff_dit_config* cfg, const void* const* tensors, int64_t n_tensors,
                  ff_dit** out);
int ff_dit_destroy(ff_dit* m);

/* Workspace bytes for a forward of B samples with grid (frames,rows,cols),
 * n_txt text tokens and n_prompts prompts. */
int ff_dit_workspace_size(const ff_dit* m, int64_t B, const int32_t grid[3] /* host */,
                          int64_t n_txt, int64_t n_prompts, size_t* bytes /* host, out */);

/* One velocity evaluation for B samples.
 * LATENT mode:
 *   x         device [B, N_img, C]           latent at time t
 *   txt       device [n_prompts, n_txt, txt_dim]  cached prompt embeddings
 *   txt_index device int32 [B], prompt row of each sample (NULL: identity,
 *             requires n_prompts == B); values outside [0, n_prompts) -> the
 *             sample's text is zero
 *   cond      device [n_prompts, pooled_dim] pooled text, or NULL when
 *             pooled_dim == 0
 *   t         device float32 [B] times in [0, 1]
 *   v_out     device [B, N_img, C]
 *   txt_out   must be NULL
 * HIDDEN mode (block stack only):
 *   x         device [B, N_img, H] image-stream hidden
 *   txt       device [B, n_txt, H] text-stream hidden (n_prompts == B, txt_index NULL)
 *   cond      device [B, H] conditioning vector c
 *   t         ignored (may be NULL)
 *   v_out     device [B, N_img, H] image-stream output
 *   txt_out   device [B, n_txt, H] text-stream output, or NULL to discard
 * grid: host int32[3] (frames, rows, cols), N_img = product.
 * v_out and txt_out may not alias any input. */
int ff_dit_forward(const ff_dit* m, const void* x, const void* txt, const int32_t* txt_index,
                   int64_t n_prompts, const void* cond, const float* t, const int32_t grid[3],
                   int64_t B, int64_t n_txt, void* v_out, void* txt_out,
                   void* workspace, size_t ws_bytes, void* stream);

/* WAN models only (others: FF_EUNSUPPORTED).  The cross-attention keys and values of every WAN block
 * depend on the text context alone, which stays fixed along a trajectory (the condition c of
 * Sec. 3.1), so a rollout computes them once:
 *   ff_dit_context_size     bytes of the per-block store for B samples and n_txt text tokens
 *   ff_dit_prepare_context  fills `context` (device, caller-owned, 16-byte aligned) from txt,
 *                           txt_index and n_prompts as ff_dit_forward takes them; the workspace is
 *                           sized by ff_dit_workspace_size for the same B, grid, n_txt, n_prompts
 *   ff_dit_forward_ctx      ff_dit_forward with the text path replaced by that store: the same
 *                           results as ff_dit_forward on the text the store was prepared from;
 *                           any workspace sized by ff_dit_workspace_size for B, grid, n_txt serves
 * Layout of the store: for block i, K [B, heads, n_txt, d] then V (bf16: transposed to
 * [B, heads, d, n_txt]; float32: [B, heads, n_txt, d]), each padded to 256 bytes.  Errors as for
 * ff_dit_forward; a store or workspace too small -> FF_EWORKSPACE. */
int ff_dit_context_size(const ff_dit* m, int64_t B, int64_t n_txt, size_t* bytes /* host, out */);
int ff_dit_prepare_context(const ff_dit* m, const void* txt, const int32_t* txt_index, int64_t n_prompts,
                           const int32_t grid[3] /* host */, int64_t B, int64_t n_txt, void* context,
                           size_t context_bytes, void* workspace, size_t ws_bytes, void* stream);
int ff_dit_forward_ctx(const ff_dit* m, const void* x, const void* context, size_t context_bytes, const float* t,
                       const int32_t grid[3] /* host */, int64_t B, int64_t n_txt, void* v_out,
                       void* workspace, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Kernel timing.  When enabled, every kernel the library launches is
 * bracketed by HIP events on its stream; ff_profile_read synchronises those
 * events and returns per-kernel-name totals (launch count, summed duration
 * and the algorithmic flops and bytes of those launches).
 * ------------------------------------------------------------------------ */
int ff_profile_enable(int32_t on);
/* Restricts the timing to launches of one kernel name (the string is copied; NULL or "" times
 * every kernel again), so that a timed run pays for the events of that kernel only. */
int ff_profile_filter(const char* name);
int ff_profile_reset(void);
int ff_profile_count(int32_t* n /* host, out: distinct kernel names */);
int ff_profile_read(int32_t i, char* name, size_t name_cap, int64_t* launches, double* total_ms,
                    double* flops, double* bytes);

#ifdef __cplusplus
}
#endif
#endif /* FF_H */
