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
// (hidden % 128 == 0, hidden <= 2048).  The statistics are shifted sums
// sum(x - x0), sum((x - x0)^2) with x0 the row's first element (stable
// against a large mean), reduced together in one pass; shift and scale are
// loaded with the row, and the output is written as packed pairs.
template <typename T> struct Pair;
template <> struct Pair<float> { typedef float type __attribute__((ext_vector_type(2))); };
template <> struct Pair<bf16> { typedef __bf16 type __attribute__((ext_vector_type(2))); };

template <typename T>
__global__ __launch_bounds__(256) void ln_mod_kernel(const float* __restrict__ x, int rows, int H,
                                                     int rpb, const float* __restrict__ shift,
                                                     const float* __restrict__ scale,
                                                     int mod_stride, T* __restrict__ out) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const int nv = H >> 7;
  const int b = row / rpb;
  const float2* xr = reinterpret_cast<const float2*>(x + (size_t)row * H);
  const float2* shr = reinterpret_cast<const float2*>(shift + (size_t)b * mod_stride);
  const float2* scr = reinterpret_cast<const float2*>(scale + (size_t)b * mod_stride);
  float2 v[16], sh[16], sc[16];
#pragma unroll
  for (int i = 0; i < 16; ++i)
    if (i < nv) {
      v[i] = xr[lane + 64 * i];
      sh[i] = shr[lane + 64 * i];
      sc[i] = scr[lane + 64 * i];
    }
  const float x0 = __shfl(v[0].x, 0, kWave);
  float s1 = 0.0f, s2 = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i)
    if (i < nv) {
      const float a = v[i].x - x0, c = v[i].y - x0;
      s1 += a + c;
      s2 += a * a + c * c;
    }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    s1 += __shfl_xor(s1, o, kWave);
    s2 += __shfl_xor(s2, o, kWave);
  }
  const float inv_h = 1.0f / (float)H;
  const float dmean = s1 * inv_h;
  const float var = fmaxf(s2 * inv_h - dmean * dmean, 0.0f);
  const float mean = x0 + dmean;
  const float rstd = 1.0f / sqrtf(var + 1e-6f);
  typedef typename Pair<T>::type P;
  P* o = reinterpret_cast<P*>(out + (size_t)row * H);
#pragma unroll
  for (int i = 0; i < 16; ++i)
    if (i < nv) {
      P w;
      w[0] = from_f<T>((v[i].x - mean) * rstd * (1.0f + sc[i].x) + sh[i].x);
      w[1] = from_f<T>((v[i].y - mean) * rstd * (1.0f + sc[i].y) + sh[i].y);
      o[lane + 64 * i] = w;
    }
}

// The same for a compile-time row length: two rows per wave (32 lanes each),
// 16-byte loads, NV float4 per lane (H = 128 NV).
template <typename T, int NV>
__global__ __launch_bounds__(256) void ln_mod_fixed_kernel(const float* __restrict__ x, int rows,
                                                           int rpb, const float* __restrict__ shift,
                                                           const float* __restrict__ scale,
                                                           int mod_stride, T* __restrict__ out) {
  constexpr int H = 128 * NV;
  const int row = blockIdx.x * 8 + (threadIdx.x >> 5);
  const int lane = threadIdx.x & 31;
  if (row >= rows) return;
  const int b = row / rpb;
  const float4* xr = reinterpret_cast<const float4*>(x + (size_t)row * H);
  const float4* shr = reinterpret_cast<const float4*>(shift + (size_t)b * mod_stride);
  const float4* scr = reinterpret_cast<const float4*>(scale + (size_t)b * mod_stride);
  float4 v[NV], sh[NV], sc[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = xr[lane + 32 * i];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    sh[i] = shr[lane + 32 * i];
    sc[i] = scr[lane + 32 * i];
  }
  const float x0 = __shfl(v[0].x, 0, 32);
  float s1 = 0.0f, s2 = 0.0f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const float a = v[i].x - x0, c = v[i].y - x0, d = v[i].z - x0, e = v[i].w - x0;
    s1 += (a + c) + (d + e);
    s2 += (a * a + c * c) + (d * d + e * e);
  }
#pragma unroll
  for (int o = 16; o > 0; o >>= 1) {
    s1 += __shfl_xor(s1, o, 32);
    s2 += __shfl_xor(s2, o, 32);
  }
  constexpr float inv_h = 1.0f / (float)H;
  const float dmean = s1 * inv_h;
  const float var = fmaxf(s2 * inv_h - dmean * dmean, 0.0f);
  const float mean = x0 + dmean;
  const float rstd = 1.0f / sqrtf(var + 1e-6f);
  typedef T Q __attribute__((ext_vector_type(4)));
  Q* o = reinterpret_cast<Q*>(out + (size_t)row * H);
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    Q w;
    w[0] = from_f<T>((v[i].x - mean) * rstd * (1.0f + sc[i].x) + sh[i].x);
    w[1] = from_f<T>((v[i].y - mean) * rstd * (1.0f + sc[i].y) + sh[i].y);
    w[2] = from_f<T>((v[i].z - mean) * rstd * (1.0f + sc[i].z) + sh[i].z);
    w[3] = from_f<T>((v[i].w - mean) * rstd * (1.0f + sc[i].w) + sh[i].w);
    o[lane + 32 * i] = w;
  }
}

template <typename T>
static void launch_ln_t(const float* x, int rows, int hidden, int rpb, const float* shift,
                        const float* scale, int mod_stride, T* out, hipStream_t s) {
  const bool al = ((uintptr_t)shift % 16 == 0) && ((uintptr_t)scale % 16 == 0) && mod_stride % 4 == 0;
  if (al && hidden == 1152) {
    hipLaunchKernelGGL((ln_mod_fixed_kernel<T, 9>), dim3(ceil_div(rows, 8)), dim3(256), 0, s, x,
                       rows, rpb, shift, scale, mod_stride, out);
  } else if (al && hidden == 384) {
    hipLaunchKernelGGL((ln_mod_fixed_kernel<T, 3>), dim3(ceil_div(rows, 8)), dim3(256), 0, s, x,
                       rows, rpb, shift, scale, mod_stride, out);
  } else {
    hipLaunchKernelGGL(ln_mod_kernel<T>, dim3(ceil_div(rows, 4)), dim3(256), 0, s, x, rows,
                       hidden, rpb, shift, scale, mod_stride, out);
  }
}

hipError_t launch_layernorm_modulate(const float* x, int rows, int hidden, int rpb,
                                     const float* shift, const float* scale, int mod_stride,
                                     void* out, int dtype, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (hidden % 128 != 0 || hidden > 2048) return hipErrorInvalidValue;
  if (dtype == kBF16)
    launch_ln_t<bf16>(x, rows, hidden, rpb, shift, scale, mod_stride, reinterpret_cast<bf16*>(out), s);
  else
    launch_ln_t<float>(x, rows, hidden, rpb, shift, scale, mod_stride, reinterpret_cast<float*>(out), s);
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
// streams the whole adaLN weight once.  One lane per row: the weight is held
// in 64-row groups, 16-byte chunk k of the group's rows stored contiguously
// ([group][chunk][64 rows][16 B], see adaln_group_index), so a wave's load
// of chunk k is one contiguous KiB and no dot product crosses lanes.  sc
// (both guidance branches) sits in LDS and is read as a broadcast.
constexpr int kAdaGroup = 64;

template <typename T>
__global__ __launch_bounds__(256) void adaln_gemv_kernel(const T* __restrict__ w,
                                                         const float* __restrict__ bias,
                                                         const float* __restrict__ sc, int H,
                                                         int n_rows, int B,
                                                         float* __restrict__ mod) {
  constexpr int CH = 16 / sizeof(T);   // elements per 16-byte chunk
  constexpr int U = 8;                 // chunks in flight per lane
  __shared__ float4 xs[2 * 2048 / 4];  // sc[b][H], H <= 2048
  const int nck = H / CH;
  for (int i = threadIdx.x; i < 2 * H / 4; i += 256) {
    const int b = i / (H / 4);
    xs[i] = b < B ? reinterpret_cast<const float4*>(sc)[i] : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int group = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int n = group * kAdaGroup + lane;
  if (group * kAdaGroup >= n_rows) return;
  const uint4* wg = reinterpret_cast<const uint4*>(w) + (size_t)group * nck * kAdaGroup + lane;
  float a0 = 0.0f, a1 = 0.0f;
  for (int k0 = 0; k0 < nck; k0 += U) {
    uint4 q[U];
#pragma unroll
    for (int u = 0; u < U; ++u) q[u] = k0 + u < nck ? wg[(size_t)(k0 + u) * kAdaGroup] : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = k0 + u;
      if (k < nck) {
        float wv[CH];
        if constexpr (sizeof(T) == 2) {
          const unsigned wd[4] = {q[u].x, q[u].y, q[u].z, q[u].w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            wv[2 * e] = __uint_as_float(wd[e] << 16);
            wv[2 * e + 1] = __uint_as_float(wd[e] & 0xFFFF0000u);
          }
        } else {
          wv[0] = __uint_as_float(q[u].x); wv[1] = __uint_as_float(q[u].y);
          wv[2] = __uint_as_float(q[u].z); wv[3] = __uint_as_float(q[u].w);
        }
#pragma unroll
        for (int e4 = 0; e4 < CH / 4; ++e4) {
          const float4 x0 = xs[(k * CH) / 4 + e4], x1 = xs[H / 4 + (k * CH) / 4 + e4];
          a0 = fmaf(wv[4 * e4 + 0], x0.x, a0); a1 = fmaf(wv[4 * e4 + 0], x1.x, a1);
          a0 = fmaf(wv[4 * e4 + 1], x0.y, a0); a1 = fmaf(wv[4 * e4 + 1], x1.y, a1);
          a0 = fmaf(wv[4 * e4 + 2], x0.z, a0); a1 = fmaf(wv[4 * e4 + 2], x1.z, a1);
          a0 = fmaf(wv[4 * e4 + 3], x0.w, a0); a1 = fmaf(wv[4 * e4 + 3], x1.w, a1);
        }
      }
    }
  }
  if (n < n_rows) {
    mod[n] = a0 + bias[n];
    if (B > 1) mod[(size_t)n_rows + n] = a1 + bias[n];
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
  const int blocks = ceil_div(ceil_div(p.n_mod, kAdaGroup), 4);
  hipLaunchKernelGGL(adaln_gemv_kernel<T>, dim3(blocks), dim3(256), 0, s,
                     reinterpret_cast<const T*>(p.w_ada), p.b_ada, p.sc, p.hidden, p.n_mod, p.B,
                     p.mod);
  return hipGetLastError();
}

size_t adaln_group_index(size_t row, size_t col, int H, int esize) {
  const size_t ch = 16 / esize, nck = H / ch;
  const size_t g = row / kAdaGroup, l = row % kAdaGroup, k = col / ch;
  return ((g * nck + k) * kAdaGroup + l) * ch + col % ch;
}

hipError_t launch_conditioning(const CondParams& p, int dtype, hipStream_t s) {
  if (p.hidden % 8 != 0 || p.hidden > 2048 || p.B < 1 || p.B > 2) return hipErrorInvalidValue;
  return dtype == kBF16 ? launch_cond_t<bf16>(p, s) : launch_cond_t<float>(p, s);
}

// ---------------------------------------------------------------------------
// Patch embedding of the band: h[b][tok][n] = W[n] . patch(tok) + bias[n]
// + pos[global tok][n], patch vector ordered (channel, dy, dx).  The weight is
// held transposed, wt[k][n], so a block's threads read it coalesced.
constexpr int kPatchTok = 4;  // tokens per thread

// (patch 2, 4 channels: a 16-element patch vector, index k = c*4 + dy*2 + dx)
__global__ __launch_bounds__(128) void patch_embed_kernel(PatchEmbedParams p) {
  const int n = blockIdx.y * 128 + threadIdx.x;  // output feature
  if (n >= p.hidden) return;
  float wk[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) wk[k] = p.w[(size_t)k * p.hidden + n];
  const float bias = p.b[n];
  const int n_tok = p.n_rows * p.grid;
  for (int u = 0; u < kPatchTok; ++u) {
    const int tok = blockIdx.x * kPatchTok + u;    // band-local token
    if (tok >= n_tok) break;
    const int i = tok / p.grid, j = tok - (tok / p.grid) * p.grid;
    const int gi = p.row_begin + i;
    float acc = bias;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int c = k >> 2, dy = (k >> 1) & 1, dx = k & 1;
      acc = fmaf(wk[k], p.x[((size_t)c * p.latent + gi * 2 + dy) * p.latent + j * 2 + dx], acc);
    }
    acc += p.pos[((size_t)gi * p.grid + j) * p.hidden + n];
    for (int b = 0; b < p.B; ++b) p.h[((size_t)b * n_tok + tok) * p.hidden + n] = acc;
  }
}

hipError_t launch_patch_embed(const PatchEmbedParams& p, hipStream_t s) {
  const int n_tok = p.n_rows * p.grid;
  if (n_tok <= 0) return hipSuccess;
  if (p.patch != 2 || p.C != 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(patch_embed_kernel, dim3(ceil_div(n_tok, kPatchTok), ceil_div(p.hidden, 128)),
                     dim3(128), 0, s, p);
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
// out may be x itself (each element is read before it is written, by the
// same thread), so neither carries __restrict__.
__global__ __launch_bounds__(256) void update_vec4_kernel(const float* x, int ldx,
                                                          const float* __restrict__ ec,
                                                          const float* __restrict__ eu, float g,
                                                          const float* __restrict__ z, int ldz,
                                                          float a, float b, float c,
                                                          float* out, int ldo,
                                                          int rows, size_t cols4) {
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
    reinterpret_cast<float4*>(out + r * (size_t)ldo)[q] = o;
  }
}

__global__ __launch_bounds__(256) void update_scalar_kernel(const float* x, int ldx,
                                                            const float* __restrict__ ec,
                                                            const float* __restrict__ eu, float g,
                                                            const float* __restrict__ z, int ldz,
                                                            float a, float b, float c,
                                                            float* out, int ldo,
                                                            int rows, size_t cols) {
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
    out[r * (size_t)ldo + q] = o;
  }
}

static bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

hipError_t launch_update(const float* x, int ldx, const float* ec, const float* eu, float g,
                         const float* z, int ldz, float a, float b, float c, float* out, int ldo,
                         int rows, size_t cols, hipStream_t s) {
  const size_t total = (size_t)rows * cols;
  if (total == 0) return hipSuccess;
  const bool vec = cols % 4 == 0 && ldx % 4 == 0 && ldo % 4 == 0 && (!z || ldz % 4 == 0) &&
                   al16(x) && al16(ec) && (!eu || al16(eu)) && (!z || al16(z)) && al16(out);
  const size_t work = vec ? total / 4 : total;
  const int blocks = (int)std::min<size_t>((work + 255) / 256, 8192);
  if (vec)
    hipLaunchKernelGGL(update_vec4_kernel, dim3(blocks), dim3(256), 0, s, x, ldx, ec, eu, g, z,
                       ldz, a, b, c, out, ldo, rows, cols / 4);
  else
    hipLaunchKernelGGL(update_scalar_kernel, dim3(blocks), dim3(256), 0, s, x, ldx, ec, eu, g, z,
                       ldz, a, b, c, out, ldo, rows, cols);
  return hipGetLastError();
}

}  // namespace orch
