// Token-local and per-step kernels of the DiT band step:
//   adaLN LayerNorm (LN without affine, then x(1 + scale) + shift),
//   conditioning (sinusoidal timestep MLP + label table -> adaLN vectors of
//   every block in one weight-streaming GEMV),
//   patch embedding of the band rows (+ the fixed position table),
//   final linear + unpatchify,
//   guidance + the scheduler update of §I (Lemma 1's eps coefficient).
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace orch {

// ---------------------------------------------------------------------------
// adaLN LayerNorm: one wave per row, the row held in registers as float2
// (hidden % 128 == 0, hidden <= 2048), two-pass mean / variance in fp32.
template <typename T>
__global__ __launch_bounds__(256) void ln_mod_kernel(const float* __restrict__ x, int rows, int H,
                                                     int rpb, const float* __restrict__ shift,
                                                     const float* __restrict__ scale,
                                                     int mod_stride, T* __restrict__ out) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const int nv = H >> 7;
  const float2* xr = reinterpret_cast<const float2*>(x + (size_t)row * H);
  float2 v[16];
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i)
    if (i < nv) {
      v[i] = xr[lane + 64 * i];
      s += v[i].x + v[i].y;
    }
  const float mean = wave_sum(s) / (float)H;
  float s2 = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i)
    if (i < nv) {
      const float a = v[i].x - mean, c = v[i].y - mean;
      s2 += a * a + c * c;
    }
  const float var = wave_sum(s2) / (float)H;
  const float rstd = 1.0f / sqrtf(var + 1e-6f);
  const int b = row / rpb;
  const float* sh = shift + (size_t)b * mod_stride;
  const float* sc = scale + (size_t)b * mod_stride;
  T* o = out + (size_t)row * H;
#pragma unroll
  for (int i = 0; i < 16; ++i)
    if (i < nv) {
      const int col = 2 * (lane + 64 * i);
      o[col] = from_f<T>((v[i].x - mean) * rstd * (1.0f + sc[col]) + sh[col]);
      o[col + 1] = from_f<T>((v[i].y - mean) * rstd * (1.0f + sc[col + 1]) + sh[col + 1]);
    }
}

hipError_t launch_layernorm_modulate(const float* x, int rows, int hidden, int rpb,
                                     const float* shift, const float* scale, int mod_stride,
                                     void* out, int dtype, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (hidden % 128 != 0 || hidden > 2048) return hipErrorInvalidValue;
  dim3 grid(ceil_div(rows, 4));
  if (dtype == kBF16)
    hipLaunchKernelGGL(ln_mod_kernel<bf16>, grid, dim3(256), 0, s, x, rows, hidden, rpb, shift,
                       scale, mod_stride, reinterpret_cast<bf16*>(out));
  else
    hipLaunchKernelGGL(ln_mod_kernel<float>, grid, dim3(256), 0, s, x, rows, hidden, rpb, shift,
                       scale, mod_stride, reinterpret_cast<float*>(out));
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Conditioning.
// t1[n] = SiLU(W1[n] . sinusoid(t) + b1[n]); sinusoid = [cos(t f_i), sin(t f_i)],
// f_i = 10000^(-i/half), evaluated in double.  One wave per output row.
template <typename T>
__global__ __launch_bounds__(256) void temb1_kernel(const T* __restrict__ w1,
                                                    const float* __restrict__ b1, float t, int H,
                                                    int freq, float* __restrict__ t1) {
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (n >= H) return;
  const int half = freq / 2;
  float acc = 0.0f;
  for (int k = lane; k < freq; k += 64) {
    const int i = k < half ? k : k - half;
    const double f = exp(-9.210340371976184 * (double)i / (double)half);  // ln(10000)
    const double a = (double)t * f;
    const float e = (float)(k < half ? cos(a) : sin(a));
    acc = fmaf(to_f<T>(w1[(size_t)n * freq + k]), e, acc);
  }
  acc = wave_sum(acc);
  if (lane == 0) t1[n] = silu_f(acc + b1[n]);
}

// sc[b][n] = SiLU(W2[n] . t1 + b2[n] + table[label_b][n]).
template <typename T>
__global__ __launch_bounds__(256) void temb2_kernel(const T* __restrict__ w2,
                                                    const float* __restrict__ b2,
                                                    const float* __restrict__ t1,
                                                    const T* __restrict__ table, int H, int B,
                                                    int lab0, int lab1, float* __restrict__ sc) {
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (n >= H) return;
  float acc = 0.0f;
  for (int k = lane; k < H; k += 64) acc = fmaf(to_f<T>(w2[(size_t)n * H + k]), t1[k], acc);
  acc = wave_sum(acc) + b2[n];
  if (lane == 0) {
    sc[n] = silu_f(acc + to_f<T>(table[(size_t)lab0 * H + n]));
    if (B > 1) sc[H + n] = silu_f(acc + to_f<T>(table[(size_t)lab1 * H + n]));
  }
}

// mod[b][n] = W_ada[n] . sc[b] + b_ada[n] for every adaLN row of every block:
// streams the whole adaLN weight once.  Each lane keeps its 8-element slices
// of sc in registers and the wave walks rows grid-stride.
template <typename T>
__global__ __launch_bounds__(256) void adaln_gemv_kernel(const T* __restrict__ w,
                                                         const float* __restrict__ bias,
                                                         const float* __restrict__ sc, int H,
                                                         int n_rows, int B,
                                                         float* __restrict__ mod) {
  const int lane = threadIdx.x & 63;
  const int wave_id = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int n_waves = gridDim.x * 4;
  const int nck = H / 8;  // 8-element chunks per row
  float xs[2][4][8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int ck = lane + 64 * j;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      xs[0][j][e] = ck < nck ? sc[ck * 8 + e] : 0.0f;
      xs[1][j][e] = (ck < nck && B > 1) ? sc[H + ck * 8 + e] : 0.0f;
    }
  }
  for (int n = wave_id; n < n_rows; n += n_waves) {
    const T* wr = w + (size_t)n * H;
    float a0 = 0.0f, a1 = 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int ck = lane + 64 * j;
      if (ck < nck) {
        float wv[8];
        if constexpr (sizeof(T) == 2) {
          const bf16x8 q = *reinterpret_cast<const bf16x8*>(wr + ck * 8);
#pragma unroll
          for (int e = 0; e < 8; ++e) wv[e] = (float)q[e];
        } else {
          const float4 q0 = *reinterpret_cast<const float4*>(wr + ck * 8);
          const float4 q1 = *reinterpret_cast<const float4*>(wr + ck * 8 + 4);
          wv[0] = q0.x; wv[1] = q0.y; wv[2] = q0.z; wv[3] = q0.w;
          wv[4] = q1.x; wv[5] = q1.y; wv[6] = q1.z; wv[7] = q1.w;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          a0 = fmaf(wv[e], xs[0][j][e], a0);
          a1 = fmaf(wv[e], xs[1][j][e], a1);
        }
      }
    }
    a0 = wave_sum(a0);
    if (B > 1) a1 = wave_sum(a1);
    if (lane == 0) {
      mod[n] = a0 + bias[n];
      if (B > 1) mod[(size_t)n_rows + n] = a1 + bias[n];
    }
  }
}

template <typename T>
static hipError_t launch_cond_t(const CondParams& p, hipStream_t s) {
  hipLaunchKernelGGL(temb1_kernel<T>, dim3(ceil_div(p.hidden, 4)), dim3(256), 0, s,
                     reinterpret_cast<const T*>(p.w_t1), p.b_t1, p.t, p.hidden, p.freq_dim, p.t1);
  hipLaunchKernelGGL(temb2_kernel<T>, dim3(ceil_div(p.hidden, 4)), dim3(256), 0, s,
                     reinterpret_cast<const T*>(p.w_t2), p.b_t2, p.t1,
                     reinterpret_cast<const T*>(p.table), p.hidden, p.B, p.labels[0],
                     p.labels[1], p.sc);
  const int blocks = min(2048, ceil_div(p.n_mod, 4));
  hipLaunchKernelGGL(adaln_gemv_kernel<T>, dim3(blocks), dim3(256), 0, s,
                     reinterpret_cast<const T*>(p.w_ada), p.b_ada, p.sc, p.hidden, p.n_mod, p.B,
                     p.mod);
  return hipGetLastError();
}

hipError_t launch_conditioning(const CondParams& p, int dtype, hipStream_t s) {
  if (p.hidden % 8 != 0 || p.hidden > 2048 || p.B < 1 || p.B > 2) return hipErrorInvalidValue;
  return dtype == kBF16 ? launch_cond_t<bf16>(p, s) : launch_cond_t<float>(p, s);
}

// ---------------------------------------------------------------------------
// Patch embedding of the band: h[b][tok][n] = W[n] . patch(tok) + bias[n]
// + pos[global tok][n], patch vector ordered (channel, dy, dx).
__global__ __launch_bounds__(128) void patch_embed_kernel(PatchEmbedParams p) {
  const int tok = blockIdx.x;                    // band-local token
  const int n = blockIdx.y * 128 + threadIdx.x;  // output feature
  if (n >= p.hidden) return;
  const int i = tok / p.grid, j = tok - (tok / p.grid) * p.grid;
  const int gi = p.row_begin + i;
  const int pd = p.C * p.patch * p.patch;
  const float* wr = p.w + (size_t)n * pd;
  float acc = p.b[n];
  int k = 0;
  for (int c = 0; c < p.C; ++c)
    for (int dy = 0; dy < p.patch; ++dy)
      for (int dx = 0; dx < p.patch; ++dx, ++k) {
        const float xv = p.x[((size_t)c * p.latent + gi * p.patch + dy) * p.latent + j * p.patch + dx];
        acc = fmaf(wr[k], xv, acc);
      }
  acc += p.pos[((size_t)gi * p.grid + j) * p.hidden + n];
  const int n_tok = p.n_rows * p.grid;
  for (int b = 0; b < p.B; ++b) p.h[((size_t)b * n_tok + tok) * p.hidden + n] = acc;
}

hipError_t launch_patch_embed(const PatchEmbedParams& p, hipStream_t s) {
  const int n_tok = p.n_rows * p.grid;
  if (n_tok <= 0) return hipSuccess;
  hipLaunchKernelGGL(patch_embed_kernel, dim3(n_tok, ceil_div(p.hidden, 128)), dim3(128), 0, s, p);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Final linear + unpatchify: one wave per (branch, token); output vector
// ordered (dy, dx, channel) -> eps[b][c][i*p + dy][j*p + dx].
template <typename T, int NO>
__global__ __launch_bounds__(256) void final_linear_kernel(FinalParams p) {
  const int wid = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (wid >= p.B * p.n_tok) return;
  const int b = wid / p.n_tok, tok = wid - b * p.n_tok;
  const T* u = reinterpret_cast<const T*>(p.u) + (size_t)wid * p.hidden;
  const T* w = reinterpret_cast<const T*>(p.w);
  float acc[NO];
#pragma unroll
  for (int o = 0; o < NO; ++o) acc[o] = 0.0f;
  for (int k = lane; k < p.hidden; k += 64) {
    const float uv = to_f<T>(u[k]);
#pragma unroll
    for (int o = 0; o < NO; ++o) acc[o] = fmaf(to_f<T>(w[(size_t)o * p.hidden + k]), uv, acc[o]);
  }
#pragma unroll
  for (int o = 0; o < NO; ++o) acc[o] = wave_sum(acc[o]);
  if (lane < NO) {
    float v = 0.0f;
#pragma unroll
    for (int o = 0; o < NO; ++o)
      if (o == lane) v = acc[o];
    v += p.b[lane];
    const int pp = p.patch;
    const int c = lane % p.out_ch;
    const int dxy = lane / p.out_ch;
    const int dy = dxy / pp, dx = dxy - (dxy / pp) * pp;
    const int i = tok / p.grid, j = tok - (tok / p.grid) * p.grid;
    const int rows = p.n_rows * pp, W = p.grid * pp;
    p.eps[(((size_t)b * p.out_ch + c) * rows + i * pp + dy) * W + j * pp + dx] = v;
  }
}

hipError_t launch_final_linear(const FinalParams& p, int dtype, hipStream_t s) {
  const int total = p.B * p.n_tok;
  if (total <= 0) return hipSuccess;
  if (p.out_ch * p.patch * p.patch != 16) return hipErrorInvalidValue;
  dim3 grid(ceil_div(total, 4));
  if (dtype == kBF16)
    hipLaunchKernelGGL((final_linear_kernel<bf16, 16>), grid, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL((final_linear_kernel<float, 16>), grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Guidance + scheduler update: out = a x - b (eu + g (ec - eu)) + c z.
__global__ __launch_bounds__(256) void update_vec4_kernel(const float* __restrict__ x, int ldx,
                                                          const float* __restrict__ ec,
                                                          const float* __restrict__ eu, float g,
                                                          const float* __restrict__ z, int ldz,
                                                          float a, float b, float c,
                                                          float* __restrict__ out, int rows,
                                                          size_t cols4) {
  const size_t total = (size_t)rows * cols4;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (size_t)gridDim.x * 256) {
    const size_t r = i / cols4, q = i - r * cols4;
    const float4 xv = reinterpret_cast<const float4*>(x + r * (size_t)ldx)[q];
    const float4 cv = reinterpret_cast<const float4*>(ec + r * cols4 * 4)[q];
    float4 e = cv;
    if (eu) {
      const float4 uv = reinterpret_cast<const float4*>(eu + r * cols4 * 4)[q];
      e.x = uv.x + g * (cv.x - uv.x);
      e.y = uv.y + g * (cv.y - uv.y);
      e.z = uv.z + g * (cv.z - uv.z);
      e.w = uv.w + g * (cv.w - uv.w);
    }
    float4 o;
    o.x = a * xv.x - b * e.x;
    o.y = a * xv.y - b * e.y;
    o.z = a * xv.z - b * e.z;
    o.w = a * xv.w - b * e.w;
    if (z) {
      const float4 zv = reinterpret_cast<const float4*>(z + r * (size_t)ldz)[q];
      o.x += c * zv.x;
      o.y += c * zv.y;
      o.z += c * zv.z;
      o.w += c * zv.w;
    }
    reinterpret_cast<float4*>(out + r * cols4 * 4)[q] = o;
  }
}

__global__ __launch_bounds__(256) void update_scalar_kernel(const float* __restrict__ x, int ldx,
                                                            const float* __restrict__ ec,
                                                            const float* __restrict__ eu, float g,
                                                            const float* __restrict__ z, int ldz,
                                                            float a, float b, float c,
                                                            float* __restrict__ out, int rows,
                                                            size_t cols) {
  const size_t total = (size_t)rows * cols;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (size_t)gridDim.x * 256) {
    const size_t r = i / cols, q = i - r * cols;
    float e = ec[r * cols + q];
    if (eu) {
      const float u = eu[r * cols + q];
      e = u + g * (e - u);
    }
    float o = a * x[r * (size_t)ldx + q] - b * e;
    if (z) o += c * z[r * (size_t)ldz + q];
    out[r * cols + q] = o;
  }
}

static bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

hipError_t launch_update(const float* x, int ldx, const float* ec, const float* eu, float g,
                         const float* z, int ldz, float a, float b, float c, float* out, int rows,
                         size_t cols, hipStream_t s) {
  const size_t total = (size_t)rows * cols;
  if (total == 0) return hipSuccess;
  const bool vec = cols % 4 == 0 && ldx % 4 == 0 && (!z || ldz % 4 == 0) && al16(x) && al16(ec) &&
                   (!eu || al16(eu)) && (!z || al16(z)) && al16(out);
  const size_t work = vec ? total / 4 : total;
  const int blocks = (int)std::min<size_t>((work + 255) / 256, 8192);
  if (vec)
    hipLaunchKernelGGL(update_vec4_kernel, dim3(blocks), dim3(256), 0, s, x, ldx, ec, eu, g, z,
                       ldz, a, b, c, out, rows, cols / 4);
  else
    hipLaunchKernelGGL(update_scalar_kernel, dim3(blocks), dim3(256), 0, s, x, ldx, ec, eu, g, z,
                       ldz, a, b, c, out, rows, cols);
  return hipGetLastError();
}

}  // namespace orch
