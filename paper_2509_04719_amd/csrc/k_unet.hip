// The first half of a U-Net ResNet block on a band of rows, with stale
// activations (patch parallelism, §II-B): GroupNorm -> SiLU -> 3x3
// convolution.  The group statistics combine the band's fresh per-row
// partial sums with the stale partial sums of every other row; the
// convolution's halo rows come from the stale buffer of its input.
//
// Four launches:
//   1. per-row partial sums (sum, sum of squares) of every channel group of
//      the band's rows (one workgroup per row);
//   2. the group statistics (mean, 1/sqrt(var + eps)) from every row's sums
//      (one workgroup, float64 sums);
//   3. SiLU(GroupNorm(x)) of the band, rounded to bf16, into the buffer's
//      band rows (refresh) or the workspace;
//   4. the 3x3 convolution as an implicit GEMM on bf16 MFMAs: M = band
//      pixels, N = output channels, K = 9 taps x input channels, fp32
//      accumulation, bias added in the epilogue.
// Layouts are pixel-major (NHWC), so a tap's input channels for one pixel are
// one contiguous run and a 32-channel k-tile of a pixel is 64 bytes.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace orch {

// ---------------------------------------------------------------------------
// 1. Partial sums of one band row.  A thread owns one channel quad and walks
// a share of the row's pixels; the shares meet in LDS and are added in a
// fixed order (the sums are bitwise reproducible), then per group.
__global__ __launch_bounds__(256) void gn_row_sums_kernel(UNetConvParams p) {
  extern __shared__ float s_part[];          // [per][C][2]
  const int y = blockIdx.x;
  const int C = p.C, W = p.W, Q = C / 4;
  // Q <= 256: 256 / Q pixel shares, one quad per thread; wider rows: one
  // share, a thread takes quads tid, tid + 256, ...
  const int per = Q <= 256 ? 256 / Q : 1;
  const int p0 = Q <= 256 ? threadIdx.x / Q : 0;
  const float4* row = reinterpret_cast<const float4*>(p.x + (size_t)y * W * C);
  if (p0 < per) {
    for (int q = Q <= 256 ? threadIdx.x % Q : threadIdx.x; q < Q; q += Q <= 256 ? Q : 256) {
      float s[4] = {0, 0, 0, 0}, ss[4] = {0, 0, 0, 0};
      for (int x = p0; x < W; x += per) {
        const float4 v = row[(size_t)x * Q + q];
        s[0] += v.x; s[1] += v.y; s[2] += v.z; s[3] += v.w;
        ss[0] += v.x * v.x; ss[1] += v.y * v.y; ss[2] += v.z * v.z; ss[3] += v.w * v.w;
      }
      float* dst = s_part + (size_t)p0 * 2 * C + 8 * q;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        dst[2 * k] = s[k];
        dst[2 * k + 1] = ss[k];
      }
    }
  }
  __syncthreads();
  const int cg = C / p.G;
  for (int g = threadIdx.x; g < p.G; g += 256) {
    float a = 0.0f, b = 0.0f;
    for (int c = g * cg; c < (g + 1) * cg; ++c)
      for (int k = 0; k < per; ++k) {
        a += s_part[(size_t)k * 2 * C + 2 * c];
        b += s_part[(size_t)k * 2 * C + 2 * c + 1];
      }
    float2 v = make_float2(a, b);
    reinterpret_cast<float2*>(p.fresh_sums)[(size_t)y * p.G + g] = v;
    if (p.refresh) reinterpret_cast<float2*>(p.stale_sums)[(size_t)(p.row_begin + y) * p.G + g] = v;
  }
}

// 2. Group statistics over the whole map: band rows from the fresh sums,
// every other row from the stale sums.
__global__ __launch_bounds__(256) void gn_stats_kernel(UNetConvParams p) {
  const int g = threadIdx.x;
  if (g >= p.G) return;
  double s = 0.0, q = 0.0;
  const float2* st = reinterpret_cast<const float2*>(p.stale_sums);
  const float2* fr = reinterpret_cast<const float2*>(p.fresh_sums);
  for (int y = 0; y < p.H; ++y) {
    const bool band = y >= p.row_begin && y < p.row_end;
    const float2 v = band ? fr[(size_t)(y - p.row_begin) * p.G + g] : st[(size_t)y * p.G + g];
    s += v.x;
    q += v.y;
  }
  const double n = (double)p.H * p.W * (p.C / p.G);
  const double mean = s / n;
  const double var = q / n - mean * mean;
  reinterpret_cast<float2*>(p.stats)[g] =
      make_float2((float)mean, (float)(1.0 / sqrt(var + (double)p.eps)));
}

// 3. act = SiLU((x - mean) rstd gamma + beta) in bf16, four channels a thread.
__global__ __launch_bounds__(256) void gn_silu_kernel(UNetConvParams p) {
  const size_t n4 = (size_t)(p.row_end - p.row_begin) * p.W * p.C / 4;
  const int Q = p.C / 4, cg = p.C / p.G;
  const float2* stats = reinterpret_cast<const float2*>(p.stats);
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (size_t)gridDim.x * 256) {
    const int c0 = (int)(i % Q) * 4;
    const float4 v = reinterpret_cast<const float4*>(p.x)[i];
    const float4 gm = reinterpret_cast<const float4*>(p.gamma)[c0 / 4];
    const float4 bt = reinterpret_cast<const float4*>(p.beta)[c0 / 4];
    const float xv[4] = {v.x, v.y, v.z, v.w}, gv[4] = {gm.x, gm.y, gm.z, gm.w},
                bv[4] = {bt.x, bt.y, bt.z, bt.w};
    bf16x4 o;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float2 sr = stats[(c0 + k) / cg];
      o[k] = (bf16)silu_f((xv[k] - sr.x) * sr.y * gv[k] + bv[k]);
    }
    reinterpret_cast<bf16x4*>(p.act_band)[i] = o;
  }
}

// ---------------------------------------------------------------------------
// 4. The convolution.  Workgroup tile: 128 band pixels x 64 output channels,
// four waves of 32 pixels each; k-tiles of one tap x 32 input channels, staged
// through registers into double-buffered LDS (rows of 32 channels padded to
// 40, so the 16-byte fragment reads of 16 rows land on distinct banks).  The
// MFMAs take the weight rows as the first operand, so a lane ends with four
// consecutive output channels of one pixel: one 16-byte store each.
namespace conv {
constexpr int BM = 128, BN = 64, BK = 32, LDR = BK + 8;
}

__global__ __launch_bounds__(256) void conv3x3_mfma_kernel(UNetConvParams p) {
  using namespace conv;
  __shared__ __attribute__((aligned(16))) bf16 sA[2][BM][LDR];
  __shared__ __attribute__((aligned(16))) bf16 sB[2][BN][LDR];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rows = p.row_end - p.row_begin;
  const int M = rows * p.W;
  const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
  const int C = p.C, W = p.W;
  const int kc = C / BK, KT = 9 * kc;
  const bf16* act_band = reinterpret_cast<const bf16*>(p.act_band);
  const bf16* stale = reinterpret_cast<const bf16*>(p.stale_act);
  const bf16* wgt = reinterpret_cast<const bf16*>(p.weight);

  // loader roles: A chunks j = tid + 256 e (row j / 4, 16-byte chunk j % 4),
  // B chunk tid (row tid / 4, chunk tid % 4)
  int ay[2], ax[2];
  bool aon[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int m = m0 + ((tid + 256 * e) >> 2);
    aon[e] = m < M;
    const int mm = aon[e] ? m : 0;
    ay[e] = p.row_begin + mm / W;
    ax[e] = mm % W;
  }
  const int ach = (tid & 3) * 8;               // channel offset of this thread's chunks
  const int brow = tid >> 2;
  uint4 ra[2], rw;

  auto load = [&](int kt) {
    const int tap = kt / kc, c0 = (kt - tap * kc) * BK;
    const int dy = tap / 3 - 1, dx = tap % 3 - 1;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int sy = ay[e] + dy, sx = ax[e] + dx;
      ra[e] = make_uint4(0, 0, 0, 0);
      if (aon[e] && sx >= 0 && sx < W && sy >= 0 && sy < p.H) {
        const bf16* src = (sy >= p.row_begin && sy < p.row_end)
                              ? act_band + ((size_t)(sy - p.row_begin) * W + sx) * C
                              : stale + ((size_t)sy * W + sx) * C;
        ra[e] = *reinterpret_cast<const uint4*>(src + c0 + ach);
      }
    }
    rw = *reinterpret_cast<const uint4*>(wgt + ((size_t)(n0 + brow) * 9 + tap) * C + c0 + ach);
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int e = 0; e < 2; ++e)
      *reinterpret_cast<uint4*>(&sA[buf][(tid + 256 * e) >> 2][ach]) = ra[e];
    *reinterpret_cast<uint4*>(&sB[buf][brow][ach]) = rw;
  };

  f32x16 acc[2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.0f;

  load(0);
  store(0);
  __syncthreads();
  const int frow = lane & 31, fk = 8 * (lane >> 5);
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT) load(kt + 1);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const bf16x8 fa = *reinterpret_cast<const bf16x8*>(&sA[cur][32 * wave + frow][16 * ks + fk]);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const bf16x8 fw = *reinterpret_cast<const bf16x8*>(&sB[cur][32 * j + frow][16 * ks + fk]);
        acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw, fa, acc[j], 0, 0, 0);
      }
    }
    if (kt + 1 < KT) store(cur ^ 1);
    __syncthreads();
  }

  // epilogue: lane holds pixel m0 + 32 wave + (lane & 31), channels
  // n0 + 32 j + 8 g + 4 (lane >> 5) + 0..3 in acc[j][4 g .. 4 g + 3]
  const int m = m0 + 32 * wave + frow;
  if (m >= M) return;
  float* orow = p.out + (size_t)m * p.C_out;
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int co = n0 + 32 * j + 8 * g + 4 * (lane >> 5);
      const float4 b = *reinterpret_cast<const float4*>(p.bias + co);
      float4 o;
      o.x = acc[j][4 * g + 0] + b.x;
      o.y = acc[j][4 * g + 1] + b.y;
      o.z = acc[j][4 * g + 2] + b.z;
      o.w = acc[j][4 * g + 3] + b.w;
      *reinterpret_cast<float4*>(orow + co) = o;
    }
}

// ---------------------------------------------------------------------------
size_t unet_conv_workspace_bytes(int W, int C, int G, int rows) {
  auto al = [](size_t b) { return (b + 255) / 256 * 256; };
  return al((size_t)rows * G * 2 * sizeof(float)) + al((size_t)G * 2 * sizeof(float)) +
         al((size_t)rows * W * C * sizeof(bf16));
}

hipError_t launch_unet_conv(const UNetConvParams& p0, void* ws, hipStream_t s) {
  UNetConvParams p = p0;
  const int rows = p.row_end - p.row_begin;
  auto al = [](size_t b) { return (b + 255) / 256 * 256; };
  char* w = reinterpret_cast<char*>(ws);
  p.fresh_sums = reinterpret_cast<float*>(w);
  w += al((size_t)rows * p.G * 2 * sizeof(float));
  p.stats = reinterpret_cast<float*>(w);
  w += al((size_t)p.G * 2 * sizeof(float));
  // the band's activations: straight into the buffer's band rows on a refresh
  p.act_band = p.refresh ? reinterpret_cast<char*>(p.stale_act) + (size_t)p.row_begin * p.W * p.C * sizeof(bf16)
                         : reinterpret_cast<void*>(w);
  const int q4 = p.C / 4, shares = q4 <= 256 ? 256 / q4 : 1;
  hipLaunchKernelGGL(gn_row_sums_kernel, dim3(rows), dim3(256), (size_t)shares * 2 * p.C * sizeof(float), s, p);
  hipLaunchKernelGGL(gn_stats_kernel, dim3(1), dim3(256), 0, s, p);
  const size_t n4 = (size_t)rows * p.W * p.C / 4;
  const int blocks = (int)std::min<size_t>((n4 + 255) / 256, 4096);
  hipLaunchKernelGGL(gn_silu_kernel, dim3(blocks), dim3(256), 0, s, p);
  dim3 grid(ceil_div(rows * p.W, conv::BM), p.C_out / conv::BN);
  hipLaunchKernelGGL(conv3x3_mfma_kernel, grid, dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace orch
