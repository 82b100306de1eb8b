/*
 * orch.h -- C ABI of the MI355X (gfx950) patch-parallel DiT denoising step.
 *
 * One device's share of a patch-parallel denoising step (Algorithm 1: "one-step
 * inference on p_i with buffer", then the buffer update; patch parallelism
 * with stale activation reuse, §II-B): a DiT denoiser evaluated on an elastic
 * band of latent token rows, whose attention reads the whole image's keys and
 * values -- fresh for the band, stale from a buffer for every other row --
 * followed by classifier-free guidance and the scheduler update of §I with the
 * eps coefficient of Lemma 1 (Eq. (1)).
 *
 * Conventions for every entry point:
 *   - Returns ORCH_OK (0) or a negative orch_status; orch_last_error() gives a
 *     thread-local message for the last failure on the calling thread.
 *   - Arguments are validated on the host before anything is launched: an
 *     error return means nothing was written.
 *   - Device pointers are HIP device addresses owned by the caller; the
 *     library owns its weights and workspace.  Kernels are enqueued on
 *     `hip_stream` (a hipStream_t; NULL = the default stream) and the call
 *     returns without synchronising.  An asynchronous device fault surfaces as
 *     ORCH_EHIP on a later call.
 *   - A context is used by one host thread and one stream at a time.
 *   - Element types: ORCH_F32 = IEEE float32; ORCH_BF16 = bfloat16 stored as
 *     16-bit words.  Rounding to bf16 is round-to-nearest-even.
 */
#ifndef ORCH_H
#define ORCH_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ORCH_OK = 0,
  ORCH_EINVAL = -1,     /* bad argument, shape or blob                        */
  ORCH_ENOWEIGHTS = -2, /* step called before orch_load_dit_weights            */
  ORCH_EHIP = -3,       /* a HIP runtime call or kernel launch failed          */
  ORCH_ENOMEM = -4      /* device allocation failed                            */
} orch_status;

enum { ORCH_F32 = 0, ORCH_BF16 = 1 };

/* DiT shape and sampler constants.  hidden = heads * head_dim, head_dim in
 * {32, 64, 72, 80, 96, 128}; hidden % 128 == 0; latent % patch == 0;
 * patch == 2; cfg_batch in {1, 2}; T = number of DDPM steps of the
 * linear-beta schedule beta = linspace(beta_start, beta_end, T). */
typedef struct {
  int n_blocks, hidden, heads, mlp_hidden;
  int in_ch, out_ch, patch, latent;
  int num_classes, freq_dim, cfg_batch, dtype;
  int T;
  double beta_start, beta_end;
} orch_dit_config;

typedef struct orch_ctx orch_ctx;

/* Create a context on the current HIP device.  Allocates the workspace for a
 * band of every row (so any band fits).  *out is set on success. */
int orch_create(const orch_dit_config* cfg, orch_ctx** out);

/* Release the context and its device memory.  NULL is ignored. */
void orch_destroy(orch_ctx* ctx);

/* Load the weight blob (host memory, `nbytes` bytes) and copy it to the
 * device.  Blob format: 256-byte header (magic "ORCHDIT1", u32 version 1,
 * u32 dtype, u32 n_blocks, hidden, heads, mlp_hidden, in_ch, out_ch, patch,
 * grid, num_classes, freq_dim, n_tensors) followed by the tensors in the
 * fixed DiT order, each 256-byte aligned, linear weights [out][in].  The
 * header must match the context's config.  Synchronous. */
int orch_load_dit_weights(orch_ctx* ctx, const void* host_blob, size_t nbytes);

/* Bytes of the stale K/V buffer: n_blocks * cfg_batch * 2 * N_kv * hidden
 * elements, N_kv = (latent/patch)^2.  Layout per (block l, branch b), at
 * element offset (l * cfg_batch + b) * 2 * N_kv * hidden: K as
 * [heads][N_kv][head_dim], then V transposed as [heads][head_dim][N_kv].
 * Token index n = row * (latent/patch) + column.
 * Why not token-major [N_kv][hidden] for K and V: the attention kernel reads
 * a tile of 64 consecutive keys of one head; head-major K makes that tile one
 * contiguous run, and V^T makes its values contiguous 128-byte runs per
 * channel, the row layout of the PV product's MFMA operand.  A band of token
 * rows is still a set of contiguous runs (one per head for K, one per head
 * and channel for V^T), so the refresh and a transfer of a band to a peer
 * need no packing. */
size_t orch_stale_kv_bytes(const orch_ctx* ctx);

/* One executed denoising step of one device (Algorithm 1; §I update with
 * Lemma 1's coefficient).
 *   x_full      device fp32 [in_ch][latent][latent]: the current sample x_t.
 *   row_begin,  the band of token rows [row_begin, row_end),
 *   row_end     0 <= row_begin < row_end <= latent/patch.
 *   t, t_prev   source and target timesteps, 0 <= t < T, -1 <= t_prev < t;
 *               t_prev = -1 means alpha_bar = 1 (the final step).
 *   labels      host int[cfg_batch], each in [0, num_classes]; with guidance
 *               labels[0] is the class and labels[1] the null label
 *               (num_classes).
 *   cfg_scale   guidance scale g: eps = eps_u + g (eps_c - eps_u); unused
 *               when cfg_batch == 1.
 *   stale_kv    device, orch_stale_kv_bytes() bytes in the config dtype.
 *               Read for every token outside the band.  Not written unless
 *               refresh != 0, and then only the band's tokens, which receive
 *               this step's fresh K/V (Algorithm 1, buffer update).
 *   z, eta      eta == 0: deterministic DDIM, z unused (may be NULL).
 *               eta > 0: z device fp32 [in_ch][latent][latent] noise, added
 *               with the eta-DDIM coefficient.
 *   out_eps     device fp32 [cfg_batch][out_ch][2r][latent] or NULL: the
 *               unguided eps of every branch for the band (r = row_end -
 *               row_begin, 2r = r * patch latent rows).
 *   out_x_patch device fp32: the band of x_{t_prev}.  Either a separate
 *               [in_ch][r*patch][latent] array, or exactly the band of x_full
 *               (x_full + row_begin*patch*latent): the band is then updated
 *               in place, in x_full's layout (channel stride latent*latent;
 *               the step reads x_full before it writes the band).  Any other
 *               overlap with x_full, stale_kv or out_eps is an error.
 * Errors: ORCH_EINVAL for a bad band, timestep, label, NULL pointer or
 * overlap; ORCH_ENOWEIGHTS before weights are loaded; ORCH_EHIP. */
int orch_patch_denoise_step(orch_ctx* ctx, const float* x_full, int row_begin, int row_end,
                            int t, int t_prev, const int* labels, float cfg_scale,
                            void* stale_kv, int refresh, const float* z, float eta,
                            float* out_eps, float* out_x_patch, void* hip_stream);

/* Algorithm 1 on n_bands virtual devices, run one after another on this GPU:
 * the whole sampler from x_{t_grid[0]} to the final latent, in place.
 *   latent      device fp32 [in_ch][latent][latent]: the initial noise in,
 *               the sample out.
 *   row_splits  host [n_bands + 1]: device i owns token rows
 *               [row_splits[i], row_splits[i+1]); 0 = row_splits[0] < ... <
 *               row_splits[n_bands] = latent / patch.
 *   tiers       host [n_bands]: 0 = every grid step, 1 = the reduced tier of
 *               Eq. (2) (steps of two grid intervals after the warm-up).
 *   t_grid      host [steps + 1]: strictly decreasing timesteps below T,
 *               t_grid[steps] = -1.
 *   warmup      1 <= warmup <= steps.
 *   kv_a, kv_b  device, orch_stale_kv_bytes() each: the K/V buffer of the
 *               last exchange and the one being filled; both are
 *               overwritten.
 * Warm-up steps are full-image steps (synchronous exchange): the buffer then
 * holds every token's K/V of that step.  After the warm-up the grid is
 * covered in sync intervals of two steps (one if a single step is left): each
 * device reads the buffer of the interval's start for the other devices'
 * tokens (its own are fresh); a tier-0 device runs t_m -> t_{m+1}, exchanging
 * that step's K/V, then t_{m+1} -> t_{m+2} without exchange (Algorithm 1:
 * no buffer update on odd offsets); a tier-1 device runs t_m -> t_{m+2} and
 * exchanges.  At the interval's end the exchanged K/V become the buffer and
 * the bands form the latent.  DDIM (eta = 0).  Errors: ORCH_EINVAL,
 * ORCH_ENOWEIGHTS, ORCH_EHIP. */
int orch_sample_patch_parallel(orch_ctx* ctx, float* latent, int n_bands, const int* row_splits,
                               const int* tiers, const int* t_grid, int steps, int warmup,
                               const int* labels, float cfg_scale, void* kv_a, void* kv_b,
                               void* hip_stream);

/* The fused guidance + scheduler update of §I, elementwise over n floats:
 *   eps = eps_uncond ? eps_uncond + g (eps_cond - eps_uncond) : eps_cond
 *   out = a x - b eps + c z          (z may be NULL when c == 0)
 * All pointers are device fp32 arrays of n elements; out may equal x.
 * With eps_uncond == NULL this is the plain update of one eps; the two-eps
 * form fuses classifier-free guidance into the same pass over memory (no
 * separate guided-eps array is written and read back). */
int orch_scheduler_update(const float* x, const float* eps_cond, const float* eps_uncond,
                          float cfg_scale, const float* z, double a, double b, double c,
                          float* out, size_t n, void* hip_stream);

/* Host only: coefficients (a, b, c) of the update for t -> t_prev under the
 * config's schedule: alpha = sqrt(abar), sigma = sqrt(1 - abar),
 * a = alpha_p / alpha_s, b = alpha_p sigma_s / alpha_s - sqrt(1 - abar_p - c^2)
 * (Lemma 1's sigma_p (e^h - 1) when eta = 0), c = eta-DDIM noise scale. */
int orch_schedule_coefficients(const orch_dit_config* cfg, int t, int t_prev, double eta,
                               double out_abc[3]);

/* Host only: the device plan of the method for n devices of effective speed
 * speed[i] > 0 (for example c_i (1 - rho_i): capability times idle share).
 * Temporal adaptation (Eq. (2)): with v_max = max speed, device i keeps
 * m_base steps when a*v_max < speed[i], the reduced tier
 * ceil((m_base + m_warmup) / 2) when b*v_max < speed[i] <= a*v_max (m_warmup
 * single steps, then the rest of the grid in steps of two intervals), and is
 * excluded (0 steps, 0 rows) otherwise; 0 < b < a < 1 (the evaluation of
 * §V-A uses a = 0.75, b = 0.25).  Spatial adaptation (Eq. (3)): device i gets
 * the share (v_i/M_i) / sum_j (v_j/M_j) of total_rows token rows, rounded to
 * whole rows by largest remainders (ties to the lower index), so the rows sum
 * to total_rows; a device whose share rounds to no rows gets 0 steps.
 * steps_out and rows_out are host arrays of n ints.  Errors: ORCH_EINVAL. */
int orch_plan_devices(const double* speed, int n, int m_base, int m_warmup, double a, double b,
                      int total_rows, int* steps_out, int* rows_out);

/* ---- convolutional (U-Net) band block -------------------------------------
 * The first half of a U-Net ResNet block, GroupNorm -> SiLU -> 3x3
 * convolution (stride 1, zero padding 1, + bias), on a band of rows of one
 * device's patch, with stale activation reuse (§II-B): a 3x3 convolution at
 * the band's edge rows reads one row beyond each edge (halo rows, from the
 * stale buffer of the convolution's input; zero outside the map), and the
 * GroupNorm statistics of the whole map combine the band's fresh per-row
 * partial sums with the stale partial sums of every other row.  GroupNorm has
 * a per-channel affine (gamma, beta) and the biased variance
 * (sum x^2)/N - mean^2 over the group's N elements of the whole map.
 * Layouts are pixel-major (NHWC). */
typedef struct {
  int height, width;        /* feature map rows and columns                     */
  int channels, groups;     /* C % 64 == 0, C % groups == 0, groups <= 256       */
  int out_channels;         /* % 64 == 0                                         */
  float eps;                /* GroupNorm epsilon, > 0                            */
} orch_unet_conv_shape;

/* Workspace bytes of orch_unet_conv_band for a band of band_rows rows.  The
 * need is not monotonic in the height: a call with few convolution tiles
 * splits its k-tiles over more workgroups and needs room for their fp32
 * partial sums, so a shorter band can need more than the whole map; a
 * caller that reuses one workspace sizes it for every height it calls
 * with. */
size_t orch_unet_conv_workspace_bytes(const orch_unet_conv_shape* shape, int band_rows);

/* GroupNorm -> SiLU -> conv3x3 on rows [row_begin, row_end) of the map.
 *   x_band      device fp32 [r][W][C]: the block input on the band's rows.
 *   gamma, beta device fp32 [C].
 *   weight      device bf16 [C_out][3][3][C] (tap (dy, dx) reads input row
 *               y + dy - 1, column x + dx - 1).
 *   bias        device fp32 [C_out].
 *   stale_act   device bf16 [H][W][C]: the convolution input of an earlier
 *               step; rows row_begin - 1 and row_end are read (when inside
 *               the map).  May be NULL for a band of every row without
 *               refresh.
 *   stale_sums  device fp32 [H][groups][2]: (sum, sum of squares) of x per
 *               row and group of an earlier step; every row outside the band
 *               is read.  May be NULL as stale_act.
 *   refresh     != 0: the band's rows of stale_act receive this step's
 *               activations (bf16) and of stale_sums its partial sums; other
 *               rows are never written.
 *   out         device fp32 [r][W][C_out].
 *   workspace   device, >= orch_unet_conv_workspace_bytes(shape, r) bytes.
 * Device pointers 16-byte aligned.  Errors: ORCH_EINVAL (shape, band, NULL
 * pointer, alignment, workspace too small, a map of (height + 2) x (width +
 * 2) x channels or a weight of 9 x channels x out_channels reaching 2 GiB in
 * bf16: the kernels index them with 32-bit offsets), ORCH_EHIP. */
int orch_unet_conv_band(const orch_unet_conv_shape* shape, int row_begin, int row_end,
                        const float* x_band, const float* gamma, const float* beta,
                        const void* weight, const float* bias, void* stale_act,
                        float* stale_sums, int refresh, float* out, void* workspace,
                        size_t workspace_bytes, void* hip_stream);

/* Host only: effective speeds for orch_plan_devices from inference time
 * profiles (§V-A: speeds derived from historical inference times).  Device
 * i has n_points[i] measured (band height, step time) pairs, taken in order
 * from rows[] and ms[] (device 0's first).  Its times are fitted by least
 * squares as t = alpha + beta * rows (a fixed per-step cost, the overhead
 * that makes small patches inefficient, plus a per-row cost) and its speed is
 * the rows per unit time at the reference band height:
 * speed_out[i] = ref_rows / (alpha + beta * ref_rows).  With a single point,
 * or one distinct height, alpha = 0.  Scaling a device's times by k divides
 * its speed by k.  Errors: ORCH_EINVAL (no points, rows < 1, a time not
 * finite and > 0, a non-positive fitted time at ref_rows). */
int orch_speeds_from_profiles(int n, const int* n_points, const int* rows, const double* ms,
                              int ref_rows, double* speed_out);

/* Thread-local message describing the last error ("" if none). */
const char* orch_last_error(void);

/* ---- per-kernel timing (measurement) -------------------------------------
 * When enabled, every kernel launch of orch_patch_denoise_step is bracketed
 * by a pair of HIP events on the caller's stream (the kernels themselves are
 * unchanged).  orch_kernel_times synchronises on the recorded events, adds
 * their elapsed times per kernel class into total_ms[class] and the launch
 * counts into launches[class] (arrays of ORCH_KCLASS_COUNT entries, may be
 * NULL), and clears the record.  Enabling allocates the event pool; disabling
 * releases it. */
enum {
  ORCH_KCLASS_CONDITIONING = 0, ORCH_KCLASS_PATCH_EMBED, ORCH_KCLASS_LAYERNORM,
  ORCH_KCLASS_QKV, ORCH_KCLASS_ATTENTION, ORCH_KCLASS_PROJ, ORCH_KCLASS_FC1,
  ORCH_KCLASS_FC2, ORCH_KCLASS_FINAL, ORCH_KCLASS_UPDATE, ORCH_KCLASS_COUNT
};
int orch_set_kernel_timing(orch_ctx* ctx, int enable);

/* Work split of the step's kernels (default on).  On: GEMMs with too few
 * output tiles to fill the GPU split K over more workgroups, and attention
 * cuts query tiles between workgroups, whenever the context's workspace
 * allows (faster for short bands; the summation order then depends on the
 * band's height).  Off: every GEMM runs unsplit and every attention query
 * tile stays in one workgroup, so each output's summation order is fixed by
 * the token alone: bands stitched from a buffer holding the full step's K/V
 * reproduce the all-rows step bit for bit.  Takes effect at the next step. */
int orch_set_work_split(orch_ctx* ctx, int enable);
int orch_kernel_times(orch_ctx* ctx, double* total_ms, long long* launches);

/* ---- kernel-level entry points ------------------------------------------
 * The kernels of the step, callable one at a time on caller buffers (same
 * launch configuration the step uses).  `dtype` is ORCH_F32 or ORCH_BF16 and
 * applies to every non-fp32 operand named "T" below. */

/* adaLN LayerNorm: out[m][:] = LN(x[m][:]) * (1 + scale[b][:]) + shift[b][:],
 * b = m / rows_per_batch; LN over `hidden` without affine, eps 1e-6, biased
 * variance, fp32 statistics.  x fp32 [rows][hidden]; shift, scale fp32 rows
 * of a [B][mod_stride] array; out T [rows][hidden]. */
int orch_op_layernorm_modulate(const float* x, int rows, int hidden, int rows_per_batch,
                               const float* shift, const float* scale, int mod_stride,
                               void* out, int dtype, void* hip_stream);

enum { ORCH_EPI_STORE = 0, ORCH_EPI_GELU = 1, ORCH_EPI_RESIDUAL = 2 };

/* y = A W^T + bias with A T [M][K], W T [N][K], bias fp32 [N], fp32
 * accumulation.  epilogue STORE: out T [M][N] = y.  GELU: out T = GELU_tanh(y).
 * RESIDUAL: out fp32 [M][N] += gate[b][n] * y, gate fp32 rows of a
 * [B][gate_stride] array, b = m / rows_per_batch.
 * workspace: device memory of at least orch_linear_workspace_bytes() bytes
 * (16-byte aligned) lets a GEMM with too few output tiles to fill the GPU
 * split K over more workgroups (fp32 partials, then a reduction that applies
 * the epilogue); NULL (or fewer bytes) runs unsplit.  The result does not
 * depend on the split beyond rounding. */
int orch_op_linear(const void* A, int M, int K, const void* W, int N, const float* bias,
                   int epilogue, const float* gate, int gate_stride, int rows_per_batch,
                   void* out, void* workspace, size_t workspace_bytes, int dtype,
                   void* hip_stream);

/* Workspace bytes orch_op_linear can use for this shape (0: never splits). */
size_t orch_linear_workspace_bytes(int M, int N, int K, int dtype);

/* The QKV projection with its scatter epilogue.  A T [B*n_tok][K], W T
 * [3H][K], bias fp32 [3H].  Q goes to q_out T [B][heads][n_tok][d]; K and V
 * of token i of branch b go to kv_out + b * kv_branch_stride, K at
 * [heads][kv_tokens][d] and V at offset kv_tokens*H as [heads][d][kv_tokens],
 * both at token index tok_offset + i. */
int orch_op_qkv_projection(const void* A, int B, int n_tok, int K, const void* W,
                           const float* bias, int hidden, int heads, void* q_out,
                           void* kv_out, size_t kv_branch_stride, int kv_tokens, int tok_offset,
                           int dtype, void* hip_stream);

/* Attention of a band's queries over the whole image (§II-B, stale K/V):
 * for branch b, head j: O = softmax(Q K^T / sqrt(d)) V.  q T [B][heads][n_q][d].
 * Keys/values of token n come from `kv_fresh` when fresh_begin <= n <
 * fresh_begin + n_fresh (fresh token n - fresh_begin; K [heads][n_fresh][d],
 * V at offset n_fresh*H as [heads][d][n_fresh], branch stride
 * fresh_branch_stride) and from `kv_stale` otherwise (buffer layout, branch
 * stride stale_branch_stride).  n_fresh may be 0.  out T [B][n_q][H].
 * workspace: device memory of at least orch_attention_workspace_bytes() bytes
 * lets short bands split the keys over more workgroups; NULL (or fewer
 * bytes) runs unsplit.  The result does not depend on the split beyond
 * rounding. */
int orch_op_attention(const void* q, const void* kv_stale, size_t stale_branch_stride,
                      const void* kv_fresh, size_t fresh_branch_stride, int fresh_begin,
                      int n_fresh, int B, int heads, int n_q, int n_kv, int head_dim, void* out,
                      void* workspace, size_t workspace_bytes, int dtype, void* hip_stream);

/* Workspace bytes orch_op_attention can use for this shape (0: never splits). */
size_t orch_attention_workspace_bytes(int B, int heads, int n_q, int n_kv, int head_dim,
                                      int dtype);

/* orch_op_attention for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same arguments without the workspace, the same kernels
 * and work plan (query tiles cut between workgroups where that pays).  The
 * cut tiles' parts go to a static device array of 20 MiB per GPU, held until
 * the process ends, which covers every shape of the work plan (at most 512
 * workgroups, head_dim <= 72); a shape needing more returns ORCH_EINVAL.
 * Calls nothing that allocates.  Every call on one GPU shares that GPU's
 * array: calls that overlap on one GPU (concurrent streams or threads) race.
 * Errors as orch_op_attention. */
int orch_op_attention_noalloc(const void* q, const void* kv_stale, size_t stale_branch_stride,
                              const void* kv_fresh, size_t fresh_branch_stride, int fresh_begin,
                              int n_fresh, int B, int heads, int n_q, int n_kv, int head_dim,
                              void* out, int dtype, void* hip_stream);

/* Conditioning of the loaded model: out fp32 [cfg_batch][6*H*n_blocks + 2*H],
 * the adaLN vectors of every block followed by the final layer's
 * (shift, scale), for timestep t and host labels[cfg_batch]. */
int orch_op_conditioning(orch_ctx* ctx, int t, const int* labels, float* out, void* hip_stream);

/* Patch embedding of the band's tokens plus the position table:
 * out fp32 [cfg_batch][r*R][H] (identical rows for every branch). */
int orch_op_patch_embed(orch_ctx* ctx, const float* x_full, int row_begin, int row_end,
                        float* out, void* hip_stream);

/* Final layer of the loaded model on h fp32 [cfg_batch][r*R][H] with the
 * final (shift, scale) of `mod` (the conditioning output): out_eps fp32
 * [cfg_batch][out_ch][r*patch][latent]. */
int orch_op_final_layer(orch_ctx* ctx, const float* h, int row_begin, int row_end,
                        const float* mod, float* out_eps, void* hip_stream);

#ifdef __cplusplus
}
#endif
#endif /* ORCH_H */
