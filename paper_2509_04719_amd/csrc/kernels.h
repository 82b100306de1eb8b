// Internal launchers of the gfx950 kernels.  All take device pointers and
// enqueue on `stream`; they return the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

namespace orch {

enum Dtype { kF32 = 0, kBF16 = 1 };
// kEpiPartial (internal): a k-split's fp32 partial sums, reduced by a second
// kernel that applies the caller's epilogue
enum Epi { kEpiStore = 0, kEpiGelu = 1, kEpiResidual = 2, kEpiQkv = 3, kEpiPartial = 4 };

// Epilogue parameters of the projection GEMMs.
struct EpiParams {
  void* out;                  // STORE / GELU: T [M][N]; RESIDUAL: fp32 [M][N]
  const float* bias;          // fp32 [N]
  const float* gate;          // RESIDUAL: fp32 [B][gate_stride]
  int gate_stride;
  int rows_per_batch;         // rows of one guidance branch
  // QKV scatter
  void* q;                    // T [B][heads][n_tok][d]
  void* kv;                   // T, branch b at kv + b*kv_branch_stride
  size_t kv_branch_stride;    // elements
  int kv_tokens;              // token extent of the K/V destination
  int tok_offset;             // destination token of the first row
  int heads, hidden, head_dim;
  unsigned hd_magic;          // set by the launcher: ceil(2^32 / head_dim)
  float q_scale = 1.0f;       // Q is written as (acc + bias) * q_scale, then rounded
  // optional fp32 workspace: lets a GEMM with too few output tiles to fill
  // the machine split K (partials [splits][M][N], then a reduction)
  float* ws = nullptr;
  size_t ws_elems = 0;
};

// Workspace elements (fp32) the GEMM's k-split takes for this shape (0: no split).
size_t gemm_split_workspace_elems(int M, int N, int K, int dtype);

// y = A W^T (+ epilogue).  A T [M][K], W T [N][K].
hipError_t launch_gemm(const void* A, const void* W, int M, int N, int K, int epi,
                       const EpiParams& ep, int dtype, hipStream_t stream);

// True when the MFMA GEMM handles this shape (bf16, N % 128 == 0, K % 64 == 0).
bool gemm_uses_mfma(int N, int K, int dtype);

hipError_t launch_layernorm_modulate(const float* x, int rows, int hidden, int rows_per_batch,
                                     const float* shift, const float* scale, int mod_stride,
                                     void* out, int dtype, hipStream_t stream);

struct AttnParams {
  const void* q;              // T [B][heads][n_q][d]
  const void* kv_stale;       // T buffer layout, branch stride stale_bs
  size_t stale_bs;
  const void* kv_fresh;       // T, branch stride fresh_bs; may be null when n_fresh == 0
  size_t fresh_bs;
  int fresh_begin, n_fresh;
  // layout of the fresh buffer: token extent (K [heads][fresh_n][d], V^T at
  // fresh_n*H as [heads][d][fresh_n]) and the index of token fresh_begin in
  // it: (n_fresh, 0) for a compact band buffer, (n_kv, fresh_begin) when the
  // fresh K/V sit in a buffer of the stale layout
  int fresh_n, fresh_off;
  int B, heads, n_q, n_kv, d;
  void* out;                  // T [B][n_q][heads*d]
  // workspace (optional) for query tiles cut between workgroups, see
  // attention_workspace_bytes
  void* ws;
  size_t ws_bytes;
  // set by the launcher: workgroup w takes work units [w * per, (w+1) * per)
  // of (branch, head, 128-query tile, 64-key tile); parts of cut tiles go to
  // part_o bf16 [2 * workers][128][d] (O_s / l_s) and part_ml float2
  // [2 * workers][128] (max, sum), slot 2w for w's first tile, 2w + 1 for
  // its last
  int per, workers;
  void* part_o;
  float2* part_ml;
  // 1: q already carries log2(e)/sqrt(d) (the step's QKV epilogue applies it
  // before rounding); 0: the kernels apply it
  int q_scaled = 0;
};

// Workspace bytes that let the attention cut query tiles between workgroups
// for this shape (0: tiles stay whole).
size_t attention_workspace_bytes(int B, int heads, int n_q, int n_kv, int d, int dtype);
hipError_t launch_attention(const AttnParams& p, int dtype, hipStream_t stream);
bool attention_uses_mfma(int d, int n_kv, int dtype);

// Conditioning.  temb: fp32 [H] scratch; sc: fp32 [B][H] SiLU(c);
// mod: fp32 [B][n_mod].
struct CondParams {
  const void* w_t1; const float* b_t1;     // [H][freq], [H]
  const void* w_t2; const float* b_t2;     // [H][H], [H]
  const void* table;                        // [(classes+1)][H]
  // w_ada: [n_mod][H] held in 64-row groups, element (n, c) at
  // adaln_group_index(n, c, H, element size) (rows past n_mod zero)
  const void* w_ada; const float* b_ada;   // [n_mod], biases
  int hidden, freq_dim, n_mod, B;
  int labels[2];
  float t;
  float* t1;                                // fp32 [H] scratch
  float* sc;                                // fp32 [B][H]
  float* mod;                               // fp32 [B][n_mod]
};
hipError_t launch_conditioning(const CondParams& p, int dtype, hipStream_t stream);
size_t adaln_group_index(size_t row, size_t col, int H, int esize);

struct PatchEmbedParams {
  const float* x;        // fp32 [C][latent][latent]
  const float* w;        // fp32 [C*p*p][H] (transposed)
  const float* b;        // fp32 [H]
  const float* pos;      // fp32 [N_kv][H]
  float* h;              // fp32 [B][n_tok][H]
  int C, latent, patch, grid, hidden, row_begin, n_rows, B;
};
hipError_t launch_patch_embed(const PatchEmbedParams& p, hipStream_t stream);

struct FinalParams {
  const void* u;         // T [B][n_tok][H] (already LN-modulated)
  const void* w;         // T [p*p*Co][H]
  const float* b;        // fp32 [p*p*Co]
  float* eps;            // fp32 [B][Co][n_rows*p][latent]
  int B, n_tok, hidden, out_ch, patch, grid, n_rows;
};
hipError_t launch_final_linear(const FinalParams& p, int dtype, hipStream_t stream);

// out = a x - b (eu + g (ec - eu)) + c z over a [rows][cols] region; x has
// row stride ldx, z row stride ldz, the rest row stride cols.  eu, z nullable.
// out row r at out + r * ldo (rows = channels of a band, or one flat row)
hipError_t launch_update(const float* x, int ldx, const float* ec, const float* eu, float g,
                         const float* z, int ldz, float a, float b, float c, float* out, int ldo,
                         int rows, size_t cols, hipStream_t stream);

// U-Net band block: GroupNorm -> SiLU -> 3x3 convolution with stale halo
// rows and stale group statistics (pixel-major layouts).
struct UNetConvParams {
  const float* x;             // fp32 [rows][W][C]: the band's block input
  const float* gamma;         // fp32 [C]
  const float* beta;          // fp32 [C]
  const void* weight;         // bf16 [C_out][3][3][C]
  const float* bias;          // fp32 [C_out]
  void* stale_act;            // bf16 [H][W][C]: convolution input of an earlier step
  float* stale_sums;          // fp32 [H][G][2]: per-row (sum, sum of squares)
  float* out;                 // fp32 [rows][W][C_out]
  int H, W, C, G, C_out, row_begin, row_end, refresh;
  float eps;
  // set by the launcher: workspace parts, and where the band's activations go
  float* fresh_sums;          // fp32 [rows][G][2]
  void* act_pad;              // bf16 [rows + 2][W + 2][C]: the band's activations, zero-bordered,
                              // with the stale rows above and below
  float* partial;             // split launch: fp32 [splits][rows * W][C_out]
};
size_t unet_conv_workspace_bytes(int W, int C, int G, int C_out, int rows);
// Largest padded activation tile (bytes) the kernels index with 32-bit offsets.
constexpr size_t kUNetMaxTileBytes = (size_t)1 << 31;
hipError_t launch_unet_conv(const UNetConvParams& p, void* workspace, hipStream_t stream);

}  // namespace orch
