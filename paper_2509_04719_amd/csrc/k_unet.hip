// The first half of a U-Net ResNet block on a band of rows, with stale
// activations (patch parallelism, §II-B): GroupNorm -> SiLU -> 3x3
// convolution.  The group statistics combine the band's fresh per-row
// partial sums with the stale partial sums of every other row; the
// convolution's halo rows come from the stale buffer of its input.
//
// Three launches (four when the convolution splits its k-tiles):
//   1. per-row partial sums (sum, sum of squares) of every channel group of
//      the band's rows (one workgroup per row);
//   2. the group statistics (mean, 1/sqrt(var + eps)) from every row's sums
//      (float64 sums, taken by every workgroup of this launch), then
//      SiLU(GroupNorm(x)) of the band, rounded to bf16, into the buffer's
//      band rows (refresh) or the workspace;
//   3. the 3x3 convolution as an implicit GEMM on bf16 MFMAs: M = band
//      pixels, N = output channels, K = 9 taps x input channels, fp32
//      accumulation, bias added in the epilogue.
// Layouts are pixel-major (NHWC), so a tap's input channels for one pixel are
// one contiguous run and a 32-channel k-tile of a pixel is 64 bytes.
#include <algorithm>
#include <numeric>

#include "common.h"
#include "kernels.h"

namespace orch {

// ---------------------------------------------------------------------------
// 1. Partial sums of one band row.  A thread owns one channel quad and walks
// a share of the row's pixels (1024 threads: about a dozen shares, so each
// thread has a few independent loads in flight); the shares meet in LDS and
// are added in a fixed order (the sums are bitwise reproducible), then per
// group.
constexpr int kRowSumThreads = 1024;

__global__ __launch_bounds__(kRowSumThreads) void gn_row_sums_kernel(UNetConvParams p) {
  extern __shared__ float s_part[];          // [shares][C][2]
  const int y = blockIdx.x;
  const int C = p.C, W = p.W, Q = C / 4;
  // Q <= threads: threads / Q pixel shares, one quad per thread; wider rows:
  // one share, a thread takes quads tid, tid + threads, ...
  const int per = Q <= kRowSumThreads ? kRowSumThreads / Q : 1;
  const int p0 = Q <= kRowSumThreads ? threadIdx.x / Q : 0;
  const float4* row = reinterpret_cast<const float4*>(p.x + (size_t)y * W * C);
  if (p0 < per) {
    for (int q = Q <= kRowSumThreads ? threadIdx.x % Q : threadIdx.x; q < Q;
         q += Q <= kRowSumThreads ? Q : kRowSumThreads) {
      float s[4] = {0, 0, 0, 0}, ss[4] = {0, 0, 0, 0};
#pragma unroll 4
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
  // channel totals over the shares (in share order) into share 0's slots,
  // then group totals over the channels (in channel order)
  for (int i = threadIdx.x; i < 2 * C; i += kRowSumThreads) {
    float a = s_part[i];
    for (int k = 1; k < per; ++k) a += s_part[(size_t)k * 2 * C + i];
    s_part[i] = a;
  }
  __syncthreads();
  const int cg = C / p.G;
  for (int g = threadIdx.x; g < p.G; g += kRowSumThreads) {
    float a = 0.0f, b = 0.0f;
    for (int c = g * cg; c < (g + 1) * cg; ++c) {
      a += s_part[2 * c];
      b += s_part[2 * c + 1];
    }
    float2 v = make_float2(a, b);
    reinterpret_cast<float2*>(p.fresh_sums)[(size_t)y * p.G + g] = v;
    if (p.refresh) reinterpret_cast<float2*>(p.stale_sums)[(size_t)(p.row_begin + y) * p.G + g] = v;
  }
}

// 2a. Group statistics over the whole map: band rows from the fresh sums,
// every other row from the stale sums.  256 / G threads per group each add
// a stride of the rows (independent loads), then the group's shares are
// added in a fixed order, in float64.  Every workgroup of the GroupNorm +
// SiLU kernel takes them itself into LDS (the same order in each, so the
// same bits), which spares their own launch.
__device__ void group_stats(const UNetConvParams& p, float2* stats_lds) {
  __shared__ double red[256][2];
  const int t = threadIdx.x;
  const int per = 256 / p.G;                  // G <= 256
  const int g = t % p.G, part = t / p.G;
  const float2* st = reinterpret_cast<const float2*>(p.stale_sums);
  const float2* fr = reinterpret_cast<const float2*>(p.fresh_sums);
  double s = 0.0, q = 0.0;
  if (part < per) {
#pragma unroll 4
    for (int y = part; y < p.H; y += per) {
      const bool band = y >= p.row_begin && y < p.row_end;
      const float2 v = band ? fr[(size_t)(y - p.row_begin) * p.G + g] : st[(size_t)y * p.G + g];
      s += v.x;
      q += v.y;
    }
  }
  red[t][0] = s;
  red[t][1] = q;
  __syncthreads();
  if (t < p.G) {
    s = 0.0;
    q = 0.0;
    for (int k = 0; k < per; ++k) {
      s += red[k * p.G + t][0];
      q += red[k * p.G + t][1];
    }
    const double n = (double)p.H * p.W * (p.C / p.G);
    const double mean = s / n;
    const double var = q / n - mean * mean;
    stats_lds[t] = make_float2((float)mean, (float)(1.0 / sqrt(var + (double)p.eps)));
  }
  __syncthreads();
}

// 2b. act = SiLU((x - mean) rstd gamma + beta) in bf16, four channels a thread
// (256 threads a workgroup, the statistics first).  The launch's thread count
// is a multiple of the row's C / 4 channel quads, so a thread keeps one quad
// for all its elements and folds its statistics and affine into one
// multiply-add per channel.  Workgroup 0 also clears the convolution's zero
// page (read for taps outside the map).
constexpr int kSiluBlocks = 512;

__global__ __launch_bounds__(256) void gn_silu_kernel(UNetConvParams p) {
  __shared__ float2 stats[256];
  if (blockIdx.x == 0 && threadIdx.x < 64) reinterpret_cast<float*>(p.zero_page)[threadIdx.x] = 0.0f;
  group_stats(p, stats);
  const size_t n4 = (size_t)(p.row_end - p.row_begin) * p.W * p.C / 4;
  const size_t first = (size_t)blockIdx.x * 256 + threadIdx.x, stride = (size_t)gridDim.x * 256;
  const int Q = p.C / 4, cg = p.C / p.G;
  const int c0 = (int)(first % Q) * 4;
  const float4 gm = reinterpret_cast<const float4*>(p.gamma)[c0 / 4];
  const float4 bt = reinterpret_cast<const float4*>(p.beta)[c0 / 4];
  const float gv[4] = {gm.x, gm.y, gm.z, gm.w}, bv[4] = {bt.x, bt.y, bt.z, bt.w};
  float mul[4], add[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float2 sr = stats[(c0 + k) / cg];
    mul[k] = sr.y * gv[k];
    add[k] = bv[k] - sr.x * mul[k];
  }
  for (size_t i = first; i < n4; i += stride) {
    const float4 v = reinterpret_cast<const float4*>(p.x)[i];
    const float xv[4] = {v.x, v.y, v.z, v.w};
    bf16x4 o;
#pragma unroll
    for (int k = 0; k < 4; ++k) o[k] = (bf16)silu_f(fmaf(xv[k], mul[k], add[k]));
    reinterpret_cast<bf16x4*>(p.act_band)[i] = o;
  }
}

// ---------------------------------------------------------------------------
// 3. The convolution as an implicit GEMM.  Workgroup tile: 128 band pixels x
// 64 output channels, four waves of 32 pixels (or x 128 channels, eight
// waves, see below); k-tiles of one tap x 64 input channels (128-byte rows),
// loaded straight into LDS (16 bytes per lane, no register staging) into a
// ring of stages, one barrier per k-tile.  A
// lane of a wave-level load fills LDS row (lane / 8) of its 8-row slab at
// physical chunk lane % 8, holding logical chunk (lane % 8) ^ ((row / 2) % 8):
// the fragment reads (16 rows at one logical chunk) then hit distinct banks.
// The A rows are gathered per tap: the pixel shifted by (dy - 1, dx - 1),
// read from the band's activations, the stale buffer (halo rows) or a zero
// page (outside the map).  The MFMAs take the weight rows as the first
// operand, so a lane ends with four consecutive output channels of one pixel.
// Launches with few tiles split their k-tiles (tap, channel chunk) in even
// ranges over more workgroups; the fp32 partial sums are added in order by a
// second kernel, which adds the bias.  Output widths divisible by 128 take
// 128-channel tiles on eight waves (one workgroup per CU, four stages).
namespace conv {
constexpr int BM = 128, BK = 64;
constexpr int ROWB = 2 * BK;                         // bytes per LDS row
// BN output channels per workgroup over NW waves (each 32 pixels x 64
// channels), a ring of S stages
template <int BN_, int NW_, int S_>
struct Geo {
  static constexpr int BN = BN_, NW = NW_, S = S_;
  static constexpr int STAGE = (BM + BN) * ROWB;
  static constexpr int LA = BM * ROWB / (NW * 1024);  // A loads per lane per k-tile
  static constexpr int LB = BN * ROWB / (NW * 1024);  // B loads per lane per k-tile
  static constexpr int LPT = LA + LB;
  static constexpr int WPC = 160 * 1024 / (S * STAGE);  // workgroups per CU (LDS)
  static_assert(NW * 64 == 4 * BN, "four waves of 32 pixels per 64 channels");
  static_assert(LA * NW * 1024 == BM * ROWB && LB * NW * 1024 == BN * ROWB, "whole wave-level loads");
  static_assert(S >= 2 && S <= 4 && (S - 1) * LPT < 64, "ring depth");
};
// 64 channels: 24 KB stages, three, two workgroups of four waves per CU;
// 128 channels (output widths divisible by 128): 32 KB stages, four, one
// workgroup of eight waves per CU, a third fewer operand bytes per MAC
using Narrow = Geo<64, 4, 3>;
using Wide = Geo<128, 8, 4>;
}

template <int LPTn>
__device__ __forceinline__ void conv_wait(int tiles_after) {
  if (tiles_after >= 3) wait_vmcnt<3 * LPTn>();
  else if (tiles_after == 2) wait_vmcnt<2 * LPTn>();
  else if (tiles_after == 1) wait_vmcnt<LPTn>();
  else wait_vmcnt<0>();
}

template <class G>
__global__ __launch_bounds__(64 * G::NW) void conv3x3_mfma_kernel(UNetConvParams p, int splits) {
  using namespace conv;
  constexpr int BN = G::BN, NW = G::NW, S = G::S, STAGE = G::STAGE, LA = G::LA, LB = G::LB, LPT = G::LPT;
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // wave's 32 pixels (wm) and 64 output channels (wn) of the tile
  const int wm = wave % 4, wn = wave / 4;
  const int rows = p.row_end - p.row_begin;
  const int M = rows * p.W;
  const int tiles_n = p.C_out / BN;
  const int tiles = ceil_div(M, BM) * tiles_n;
  const int split = __builtin_amdgcn_readfirstlane((int)blockIdx.x / tiles);
  const int tile = blockIdx.x - split * tiles;
  const int m0 = (tile / tiles_n) * BM, n0 = (tile % tiles_n) * BN;
  const int C = p.C, W = p.W;
  const int kc = C / BK;                               // channel chunks per tap
  // this split's k-tiles [kt0, kt0 + KT) of the 9 kc (tap, channel chunk) ones
  const int kt0 = split * 9 * kc / splits, KT = (split + 1) * 9 * kc / splits - kt0;
  const char* act_band = reinterpret_cast<const char*>(p.act_band);
  const char* stale = reinterpret_cast<const char*>(p.stale_act);
  const char* zero = reinterpret_cast<const char*>(p.zero_page);
  const char* wgt = reinterpret_cast<const char*>(p.weight);

  // this lane's load slots: A rows 8 (i NW + wave) + lane / 8 (pixel of the
  // tile), B rows likewise (output channel); logical chunk of the slot
  const int lrow = lane >> 3, pc = lane & 7;
  int ay[LA], ax[LA], alc[LA];
  bool aon[LA];
#pragma unroll
  for (int i = 0; i < LA; ++i) {
    const int r = 8 * (i * NW + wave) + lrow;
    const int m = m0 + r;
    aon[i] = m < M;
    const int mm = aon[i] ? m : 0;
    ay[i] = p.row_begin + mm / W;
    ax[i] = mm % W;
    alc[i] = pc ^ ((r >> 1) & 7);
  }
  size_t boff[LB];
#pragma unroll
  for (int i = 0; i < LB; ++i) {
    const int r = 8 * (i * NW + wave) + lrow;
    boff[i] = ((size_t)(n0 + r) * 9 * C + (size_t)(pc ^ ((r >> 1) & 7)) * 8) * 2;
  }

  auto issue = [&](int kt, int st) {
    const int g = kt0 + kt, tap = g / kc, c0 = (g % kc) * BK;
    const int dy = tap / 3 - 1, dx = tap % 3 - 1;
    char* base = smem + st * STAGE;
#pragma unroll
    for (int i = 0; i < LA; ++i) {
      const int sy = ay[i] + dy, sx = ax[i] + dx;
      const char* src = zero;
      if (aon[i] && sx >= 0 && sx < W && sy >= 0 && sy < p.H) {
        src = (sy >= p.row_begin && sy < p.row_end)
                  ? act_band + (((size_t)(sy - p.row_begin) * W + sx) * C + c0 + alc[i] * 8) * 2
                  : stale + (((size_t)sy * W + sx) * C + c0 + alc[i] * 8) * 2;
      }
      __builtin_amdgcn_global_load_lds((const ORCH_GLB void*)src,
                                       (ORCH_LDS void*)(base + (i * NW + wave) * 1024), 16, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < LB; ++i) {
      const char* src = wgt + boff[i] + ((size_t)tap * C + c0) * 2;
      __builtin_amdgcn_global_load_lds((const ORCH_GLB void*)src,
                                       (ORCH_LDS void*)(base + BM * ROWB + (i * NW + wave) * 1024), 16, 0, 0);
    }
  };

  f32x16 acc[2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.0f;

  // fragment reads: A row 32 wave + (lane & 31), B rows 32 j + (lane & 31),
  // logical chunk 2 kk + (lane >> 5)
  const int frow = lane & 31, h = lane >> 5;
  const int arow = (32 * wm + frow) * ROWB, brow = BM * ROWB + (64 * wn + frow) * ROWB;
  int koff[BK / 16];
#pragma unroll
  for (int kk = 0; kk < BK / 16; ++kk) koff[kk] = ((2 * kk + h) ^ ((frow >> 1) & 7)) * 16;

  const int pro = min(S - 1, KT);
  for (int t = 0; t < pro; ++t) issue(t, t);
  for (int kt = 0; kt < KT; ++kt) {
    conv_wait<LPT>(min(KT, kt + S - 1) - (kt + 1));
    lds_barrier();
    if (kt + S - 1 < KT) issue(kt + S - 1, (kt + S - 1) % S);
    const char* base = smem + (kt % S) * STAGE;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const bf16x8 fa = *reinterpret_cast<const bf16x8*>(base + arow + koff[kk]);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const bf16x8 fw = *reinterpret_cast<const bf16x8*>(base + brow + j * 32 * ROWB + koff[kk]);
        acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw, fa, acc[j], 0, 0, 0);
      }
    }
  }

  // epilogue: lane holds pixel m0 + 32 wm + (lane & 31), channels
  // n0 + 64 wn + 32 j + 8 g + 4 (lane >> 5) + 0..3 in acc[j][4 g .. 4 g + 3]
  const int m = m0 + 32 * wm + frow;
  if (m >= M) return;
  float* orow = splits > 1 ? p.partial + ((size_t)split * M + m) * p.C_out : p.out + (size_t)m * p.C_out;
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int co = n0 + 64 * wn + 32 * j + 8 * g + 4 * h;
      float4 b = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      if (splits == 1) b = *reinterpret_cast<const float4*>(p.bias + co);
      float4 o;
      o.x = acc[j][4 * g + 0] + b.x;
      o.y = acc[j][4 * g + 1] + b.y;
      o.z = acc[j][4 * g + 2] + b.z;
      o.w = acc[j][4 * g + 3] + b.w;
      *reinterpret_cast<float4*>(orow + co) = o;
    }
}

// The split launch's partial sums, added in split order, plus the bias.
__global__ __launch_bounds__(256) void conv_split_reduce_kernel(UNetConvParams p, int splits) {
  const size_t n4 = (size_t)(p.row_end - p.row_begin) * p.W * p.C_out / 4;
  const int q4 = p.C_out / 4;
  const float4* part = reinterpret_cast<const float4*>(p.partial);
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (size_t)gridDim.x * 256) {
    float4 v = reinterpret_cast<const float4*>(p.bias)[i % q4];
    for (int sp = 0; sp < splits; ++sp) {
      const float4 a = part[(size_t)sp * n4 + i];
      v.x += a.x; v.y += a.y; v.z += a.z; v.w += a.w;
    }
    reinterpret_cast<float4*>(p.out)[i] = v;
  }
}

// ---------------------------------------------------------------------------
// K splits of a launch: the 9 C / 64 k-tiles (tap, channel chunk) cut into
// 1, 3, 9 or 16 even ranges over more workgroups, at least four k-tiles
// each, the count with the least estimated time.  The estimate (fitted to
// measurements of the three SDXL-sized stages on MI355X): rounds of
// workgroups over the slots (256 CUs, two narrow workgroups or one wide per
// CU) x k-tiles per workgroup x 0.8 us, plus, when split, the fp32
// partials' round trip at 0.5 us per MB and 3 us for the reduction kernel,
// which adds them in order.
static bool conv_wide(int C_out) { return C_out % conv::Wide::BN == 0; }

static int conv_splits(int M, int C, int C_out) {
  const bool wide = conv_wide(C_out);
  const int tiles = ceil_div(M, conv::BM) * (C_out / (wide ? conv::Wide::BN : conv::Narrow::BN));
  const int slots = 256 * (wide ? conv::Wide::WPC : conv::Narrow::WPC);
  const int kts = 9 * (C / conv::BK);
  const double mb = (double)M * C_out * sizeof(float) / 1e6;
  int best = 1;
  double best_us = 0.0;
  for (const int s : {1, 3, 9, 16}) {
    if (s > 1 && kts < 4 * s) break;
    const double us = ceil_div(tiles * s, slots) * ceil_div(kts, s) * 0.8 + (s > 1 ? s * mb * 0.5 + 3.0 : 0.0);
    if (s == 1 || us < best_us) {
      best = s;
      best_us = us;
    }
  }
  return best;
}

template <class G>
static void launch_conv(const UNetConvParams& p, int M, int sp, hipStream_t s) {
  auto kern = conv3x3_mfma_kernel<G>;
  static bool attr = [&] {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                              G::S * G::STAGE);
    return true;
  }();
  (void)attr;
  const int tiles = ceil_div(M, conv::BM) * (p.C_out / G::BN);
  hipLaunchKernelGGL(kern, dim3(tiles * sp), dim3(64 * G::NW), G::S * G::STAGE, s, p, sp);
}

static size_t al256(size_t b) { return (b + 255) / 256 * 256; }

size_t unet_conv_workspace_bytes(int W, int C, int G, int C_out, int rows) {
  const int M = rows * W;
  const int sp = conv_splits(M, C, C_out);
  return al256((size_t)rows * G * 2 * sizeof(float)) +
         al256((size_t)rows * W * C * sizeof(bf16)) + 256 /* zero page */ +
         (sp > 1 ? al256((size_t)sp * M * C_out * sizeof(float)) : 0);
}

hipError_t launch_unet_conv(const UNetConvParams& p0, void* ws, hipStream_t s) {
  UNetConvParams p = p0;
  const int rows = p.row_end - p.row_begin;
  const int M = rows * p.W;
  const int sp = conv_splits(M, p.C, p.C_out);
  char* w = reinterpret_cast<char*>(ws);
  p.fresh_sums = reinterpret_cast<float*>(w);
  w += al256((size_t)rows * p.G * 2 * sizeof(float));
  void* act_ws = w;
  w += al256((size_t)rows * p.W * p.C * sizeof(bf16));
  p.zero_page = w;
  w += 256;
  p.partial = sp > 1 ? reinterpret_cast<float*>(w) : nullptr;
  // the band's activations: straight into the buffer's band rows on a refresh
  p.act_band = p.refresh ? reinterpret_cast<char*>(p.stale_act) + (size_t)p.row_begin * p.W * p.C * sizeof(bf16)
                         : act_ws;
  const int q4 = p.C / 4, shares = q4 <= kRowSumThreads ? kRowSumThreads / q4 : 1;
  hipLaunchKernelGGL(gn_row_sums_kernel, dim3(rows), dim3(kRowSumThreads),
                     (size_t)shares * 2 * p.C * sizeof(float), s, p);
  // workgroups: enough for the band (at most kSiluBlocks), a multiple of
  // Q / gcd(Q, 256) so that 256 * blocks is a multiple of the C / 4 quads
  const size_t n4 = (size_t)rows * p.W * p.C / 4;
  const int nq = p.C / 4, unit = nq / std::gcd(nq, 256);
  int blocks = (int)std::min<size_t>((n4 + 255) / 256, kSiluBlocks);
  blocks = std::max(unit, blocks / unit * unit);
  hipLaunchKernelGGL(gn_silu_kernel, dim3(blocks), dim3(256), 0, s, p);
  if (conv_wide(p.C_out))
    launch_conv<conv::Wide>(p, M, sp, s);
  else
    launch_conv<conv::Narrow>(p, M, sp, s);
  if (sp > 1) {
    const size_t o4 = (size_t)M * p.C_out / 4;
    hipLaunchKernelGGL(conv_split_reduce_kernel, dim3((int)std::min<size_t>((o4 + 255) / 256, 4096)),
                       dim3(256), 0, s, p, sp);
  }
  return hipGetLastError();
}

}  // namespace orch
