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
//      SiLU(GroupNorm(x)) of the band, rounded to bf16, into a zero-bordered
//      tile of the band (one more row above and below, from the stale buffer
//      or zero outside the map, and a zero column on each side) and, on a
//      refresh, into the buffer's band rows;
//   3. the 3x3 convolution as an implicit GEMM on bf16 MFMAs over the tile:
//      M = band pixels, N = output channels, K = 9 taps x input channels,
//      fp32 accumulation, bias added in the epilogue.
// Layouts are pixel-major (NHWC), so a tap's input channels for one pixel are
// one contiguous run and a 64-channel k-tile of a pixel is 128 bytes.
#include <algorithm>
#include <numeric>
#include <type_traits>

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
constexpr int kRowSumBatch = 12;

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
      // up to kRowSumBatch pixels' loads in flight, then their sums in pixel order
      for (int x0 = p0; x0 < W; x0 += kRowSumBatch * per) {
        float4 v[kRowSumBatch];
#pragma unroll
        for (int i = 0; i < kRowSumBatch; ++i)
          if (x0 + i * per < W) v[i] = row[(size_t)(x0 + i * per) * Q + q];
#pragma unroll
        for (int i = 0; i < kRowSumBatch; ++i)
          if (x0 + i * per < W) {
            s[0] += v[i].x; s[1] += v[i].y; s[2] += v[i].z; s[3] += v[i].w;
            ss[0] += v[i].x * v[i].x; ss[1] += v[i].y * v[i].y; ss[2] += v[i].z * v[i].z; ss[3] += v[i].w * v[i].w;
          }
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
// multiply-add per channel.  The result goes to the interior of the padded
// tile [rows + 2][W + 2][C] (pixel (y, x) of the band at tile row y + 1,
// column x + 1) and, on a refresh, to the band rows of the stale buffer.  The
// tile's border follows: its first and last rows are the stale rows above
// and below the band (zero outside the map), its first and last columns zero.
constexpr int kSiluBlocks = 512;

__global__ __launch_bounds__(256) void gn_silu_kernel(UNetConvParams p) {
  __shared__ float2 stats[256];
  group_stats(p, stats);
  const int rows = p.row_end - p.row_begin, W = p.W, Q = p.C / 4, cg = p.C / p.G;
  // every index below fits 32 bits: the launcher keeps the tile under 2^31 bytes
  const unsigned n4 = (unsigned)rows * W * Q;
  const unsigned first = blockIdx.x * 256u + threadIdx.x, stride = gridDim.x * 256u;
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
  bf16x4* tile = reinterpret_cast<bf16x4*>(p.act_pad);
  bf16x4* band = p.refresh ? reinterpret_cast<bf16x4*>(p.stale_act) + (size_t)p.row_begin * W * Q : nullptr;
  const float inv_w = 1.0f / (float)W;
  for (unsigned i = first; i < n4; i += stride) {
    const float4 v = reinterpret_cast<const float4*>(p.x)[i];
    const float xv[4] = {v.x, v.y, v.z, v.w};
    bf16x4 o;
#pragma unroll
    for (int k = 0; k < 4; ++k) o[k] = (bf16)silu_f(fmaf(xv[k], mul[k], add[k]));
    // band pixel px = (y, x) -> tile pixel (y + 1) (W + 2) + x + 1 = px + 2 y + W + 3
    const int px = (int)(i / Q);
    int y = (int)(((float)px + 0.5f) * inv_w);
    y -= y * W > px;
    y += (y + 1) * W <= px;
    tile[(unsigned)(px + 2 * y + W + 3) * Q + (i - (unsigned)px * Q)] = o;
    if (band) band[i] = o;
  }
  // border: 2 (W + 2) Q quads of the halo rows, then 2 rows Q of the side columns
  const unsigned halo = 2u * (W + 2) * Q, nb = halo + 2u * rows * Q;
  const bf16x4* stale = reinterpret_cast<const bf16x4*>(p.stale_act);
  for (unsigned i = first; i < nb; i += stride) {
    bf16x4 o;
#pragma unroll
    for (int k = 0; k < 4; ++k) o[k] = (bf16)0.0f;
    unsigned dst;
    if (i < halo) {
      const unsigned below = i / ((W + 2) * Q);
      const unsigned r = i - below * (W + 2) * Q;
      const int col = (int)(r / Q), q = (int)(r % Q);
      const int sy = below ? p.row_end : p.row_begin - 1;
      if (col >= 1 && col <= W && sy >= 0 && sy < p.H) o = stale[((size_t)sy * W + col - 1) * Q + q];
      dst = ((below ? rows + 1 : 0) * (W + 2) + col) * Q + q;
    } else {
      const unsigned r = i - halo;
      const int y = (int)(r / (2 * Q)), side = (int)(r / Q) & 1, q = (int)(r % Q);
      dst = ((unsigned)(y + 1) * (W + 2) + (side ? W + 1 : 0)) * Q + q;
    }
    tile[dst] = o;
  }
}

// ---------------------------------------------------------------------------
// 3. The convolution as an implicit GEMM over the padded tile.  Workgroup
// tile: 128 band pixels x BN output channels on WM x WN waves; k-tiles of one
// tap x 64 input channels (128-byte rows), loaded straight into LDS (16 bytes
// per lane, no register staging) into a ring of stages, one barrier per
// k-tile.  In the padded tile the tap (dy, dx) of every pixel is the pixel's
// own address plus one uniform offset, so a lane's source is a constant
// per-lane offset plus a scalar per k-tile, for the weights as for the
// activations, and a load costs no vector arithmetic.  A wave-level load
// fills one 8-row slab: lane l writes row l / 8 at physical chunk l % 8,
// holding logical chunk (l % 8) ^ ((row / 2) % 8), so the fragment reads (16
// rows at one logical chunk) hit distinct banks.  The MFMAs take the weight
// rows as the first operand, so a lane ends with four consecutive output
// channels of one pixel.  The main loop's emission order is fixed with
// scheduling fences: each MFMA, then its share of the next k-step's fragment
// reads, then its share of the next tile's loads.  The epilogue stages each
// wave's block in LDS and writes whole runs of a pixel's channels.  Launches
// with few tiles split their k-tiles (tap, channel chunk) in even ranges over
// more workgroups; the fp32 partial sums are added in order by a second
// kernel, which adds the bias.
namespace conv {
constexpr int BM = 128, BK = 64;
constexpr int ROWB = 2 * BK;                         // bytes per LDS row
// BN output channels per workgroup on WM x WN waves (wave tile TM pixels x
// TN channels), MF x MF MFMA blocks (32: v_mfma_f32_32x32x16_bf16, 16:
// v_mfma_f32_16x16x32_bf16), a ring of S stages
template <int BN_, int WM_, int WN_, int S_, int MF_>
struct Geo {
  static constexpr int BN = BN_, WM = WM_, WN = WN_, NW = WM_ * WN_, S = S_, MF = MF_;
  static constexpr int TM = BM / WM, TN = BN / WN;
  static constexpr int FM = TM / MF, FN = TN / MF;     // MFMA blocks per wave
  static constexpr int KK = BK / (MF == 32 ? 16 : 32); // MFMA k-steps per k-tile
  static constexpr int STAGE = (BM + BN) * ROWB;
  static constexpr int SLABS_A = BM / 8, SLABS = (BM + BN) / 8;
  static constexpr int LPT = (SLABS + NW - 1) / NW;    // loads per lane per k-tile
  static constexpr int LPK = (LPT + KK - 1) / KK;      // loads issued per k-step
  static constexpr int WPC = 160 * 1024 / (S * STAGE);  // workgroups per CU (LDS)
  static constexpr int SROW = TN + 4;                  // epilogue strip row (floats)
  static constexpr int CPR = TN / 4;                   // 16-byte chunks of a strip row
  static_assert(MF == 32 || MF == 16, "MFMA shape");
  static_assert(TM % MF == 0 && TN % MF == 0 && BN % 8 == 0, "wave tile");
  static_assert(SLABS_A % NW == 0, "A slabs evenly over the waves");
  static_assert(LPT * NW - SLABS <= SLABS_A, "spare slots re-load A slabs");
  static_assert(S >= 2 && S <= 4 && (S - 1) * LPT < 64, "ring depth");
  static_assert(NW * TM * SROW * 4 <= S * STAGE, "epilogue strips fit the ring");
  static_assert(CPR <= 64, "strip row");
};
// 64 channels: 24 KB stages, three, two workgroups of four waves per CU;
// 128 channels (output widths divisible by 128): 32 KB stages, four, one
// workgroup of eight waves per CU, a third fewer operand bytes per MAC;
// 160 channels (widths divisible by 160 and not by 128, such as 320):
// 36 KB stages, four, one workgroup of eight waves of 32 pixels x 80
// channels on 16x16x32 MFMAs, so a 320-wide map is two tiles across
using Narrow = Geo<64, 4, 1, 3, 32>;
using Wide = Geo<128, 4, 2, 4, 32>;
using Mid = Geo<160, 4, 2, 4, 16>;
}

template <class G>
__global__ __launch_bounds__(64 * G::NW) void conv3x3_mfma_kernel(UNetConvParams p, int splits) {
  using namespace conv;
  constexpr int NW = G::NW, S = G::S, STAGE = G::STAGE, LPT = G::LPT, LPK = G::LPK, KK = G::KK;
  constexpr int MF = G::MF, FM = G::FM, FN = G::FN, TM = G::TM, TN = G::TN, SROW = G::SROW, CPR = G::CPR;
  using Acc = std::conditional_t<MF == 32, f32x16, f32x4>;
  constexpr int AR = MF == 32 ? 16 : 4;                // accumulator registers
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % G::WM, wn = wave / G::WM;
  const int rows = p.row_end - p.row_begin;
  const int M = rows * p.W;
  const int tiles_n = p.C_out / G::BN;
  const int tiles = ceil_div(M, BM) * tiles_n;
  const int split = __builtin_amdgcn_readfirstlane((int)blockIdx.x / tiles);
  const int tile = blockIdx.x - split * tiles;
  const int m0 = (tile / tiles_n) * BM, n0 = (tile % tiles_n) * G::BN;
  const int C = p.C, W = p.W, WP = p.W + 2;
  const int kc = C / BK;                               // channel chunks per tap
  // this split's k-tiles [kt0, kt0 + KT) of the 9 kc (tap, channel chunk) ones
  const int kt0 = split * 9 * kc / splits, KT = (split + 1) * 9 * kc / splits - kt0;
  const char* gA = reinterpret_cast<const char*>(p.act_pad);
  const char* gW = reinterpret_cast<const char*>(p.weight);

  // load j of a k-tile fills slab s = j NW + wave: A (pixel) slabs first,
  // then B (output channel) slabs; slots past the last slab re-load A slab
  // s - SLABS (the same bytes to the same place).  Byte offsets of tap
  // (0, 0), channel chunk 0; rows past M re-read pixel M - 1.
  const int lrow = lane >> 3, pc = lane & 7;
  unsigned off[LPT];
  int dsto[LPT];
  bool isa[LPT];
#pragma unroll
  for (int j = 0; j < LPT; ++j) {
    int sl = j * NW + wave;
    if (sl >= G::SLABS) sl -= G::SLABS;
    isa[j] = sl < G::SLABS_A;
    const int r = 8 * (isa[j] ? sl : sl - G::SLABS_A) + lrow;
    const unsigned lc = (unsigned)(pc ^ ((r >> 1) & 7)) * 16u;
    dsto[j] = sl * 1024;
    if (isa[j]) {
      const int m = min(m0 + r, M - 1), y = m / W;
      off[j] = (unsigned)((y + 1) * WP + (m - y * W) + 1) * (unsigned)C * 2u + lc;
    } else {
      off[j] = (unsigned)(n0 + r) * (unsigned)(9 * C) * 2u + lc;
    }
  }
  // scalar offsets of k-tile g: the tap's shift in the padded tile plus the
  // channel chunk (A); g 128-byte k-tiles into each weight row (B)
  auto a_shift = [&](int g) -> int {
    const int tap = g / kc, dy = tap / 3 - 1, dx = tap % 3 - 1;
    return ((dy * WP + dx) * C + (g - tap * kc) * BK) * 2;
  };
  auto dma = [&](auto jc, int g, int ashift, int st) {
    constexpr int j = decltype(jc)::value;
    const char* src = (isa[j] ? gA + ashift : gW + g * ROWB) + off[j];
    __builtin_amdgcn_global_load_lds((const ORCH_GLB void*)src, (ORCH_LDS void*)(smem + st * STAGE + dsto[j]),
                                     16, 0, 0);
  };

  Acc acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < AR; ++r) acc[i][j][r] = 0.0f;

  // fragment reads: row (lane & (MF - 1)) of an MF-row block, logical chunk
  // (KS / 8) kk + lane / MF for the KS-deep k-step; block rows start at
  // multiples of 16, so the row's swizzle depends on the lane alone
  const int frow = lane & (MF - 1), fh = lane / MF;
  const int arow = (TM * wm + frow) * ROWB, brow = BM * ROWB + (TN * wn + frow) * ROWB;
  int koff[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) koff[kk] = (((64 / MF) * kk + fh) ^ ((frow >> 1) & 7)) * 16;

  // the MFMAs of stage st; with ISSUE, k-tile ig's loads into stage ist go
  // between them: MFMA e of k-step kk, its share of k-step kk + 1's
  // fragment reads, its share of the loads
  auto compute = [&](int st, auto issue_c, int ig, int ist) {
    constexpr bool ISSUE = decltype(issue_c)::value;
    constexpr int NM = FM * FN, ND = FM + FN;
    const char* base = smem + st * STAGE;
    const int ash = ISSUE ? a_shift(ig) : 0;
    bf16x8 fa[2][FM], fb[2][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) fa[0][i] = *reinterpret_cast<const bf16x8*>(base + arow + i * MF * ROWB + koff[0]);
#pragma unroll
    for (int j = 0; j < FN; ++j) fb[0][j] = *reinterpret_cast<const bf16x8*>(base + brow + j * MF * ROWB + koff[0]);
    __builtin_amdgcn_sched_barrier(0);
    static_for<0, KK>([&](auto kkc) {
      constexpr int kk = decltype(kkc)::value;
      constexpr int cur = kk & 1, nk = kk + 1 < KK ? kk + 1 : kk;
      constexpr int nd = kk + 1 < KK ? ND : 0;
      constexpr int l0 = cmin(kk * LPK, LPT), nl = ISSUE ? cmin(kk * LPK + LPK, LPT) - l0 : 0;
      static_for<0, NM>([&](auto ec) {
        constexpr int e = decltype(ec)::value;
        constexpr int i = e / FN, j = e % FN;
        if constexpr (MF == 32)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[cur][j], fa[cur][i], acc[i][j], 0, 0, 0);
        else
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[cur][j], fa[cur][i], acc[i][j], 0, 0, 0);
        static_for<e * nd / NM, (e + 1) * nd / NM>([&](auto dc) {
          constexpr int d = decltype(dc)::value;
          if constexpr (d < FM)
            fa[cur ^ 1][d] = *reinterpret_cast<const bf16x8*>(base + arow + d * MF * ROWB + koff[nk]);
          else
            fb[cur ^ 1][d - FM] = *reinterpret_cast<const bf16x8*>(base + brow + (d - FM) * MF * ROWB + koff[nk]);
        });
        static_for<l0 + e * nl / NM, l0 + (e + 1) * nl / NM>([&](auto jc) { dma(jc, ig, ash, ist); });
        __builtin_amdgcn_sched_barrier(0);
      });
    });
  };

  // prologue: k-tiles 0 .. S - 2 (KT >= S - 1: at least four k-tiles a split)
#pragma unroll
  for (int t = 0; t < S - 1; ++t) {
    const int ash = a_shift(kt0 + t);
    static_for<0, LPT>([&](auto jc) { dma(jc, kt0 + t, ash, t); });
  }
  int kt = 0;
  for (; kt + S - 1 < KT; ++kt) {
    wait_vmcnt<(S - 2) * LPT>();
    lds_barrier();
    compute(kt % S, std::true_type{}, kt0 + kt + S - 1, (kt + S - 1) % S);
  }
  // drain: the last S - 1 k-tiles, nothing more to issue
  static_for<0, S - 2>([&](auto rc) {
    wait_vmcnt<(S - 2 - decltype(rc)::value) * LPT>();
    lds_barrier();
    compute(kt % S, std::false_type{}, 0, 0);
    ++kt;
  });
  wait_vmcnt<0>();
  lds_barrier();
  compute(kt % S, std::false_type{}, 0, 0);

  // epilogue: through a per-wave strip [TM pixels][TN channels] in LDS.  With
  // 32x32 blocks a lane holds pixel 32 i + (lane & 31), channels 32 j + 8 g +
  // 4 (lane >> 5) + 0..3 in acc[i][j][4 g .. 4 g + 3]; with 16x16 blocks
  // pixel 16 i + (lane & 15), channels 16 j + 4 (lane >> 4) + 0..3.  Each
  // pixel's TN channels then leave as TN / 4 lanes x 16 bytes.
  lds_barrier();
  float* strip = reinterpret_cast<float*>(smem) + wave * TM * SROW;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int g = 0; g < AR / 4; ++g)
        *reinterpret_cast<float4*>(strip + (MF * i + frow) * SROW + MF * j + 8 * g + 4 * fh) =
            make_float4(acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the strip is written
  constexpr int RPI = 64 / CPR;        // strip rows per store instruction
  const int q = lane % CPR, rl = lane / CPR, co = n0 + TN * wn + 4 * q;
  float4 b = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  if (splits == 1 && rl < RPI) b = *reinterpret_cast<const float4*>(p.bias + co);
  float* obase = splits > 1 ? p.partial + (size_t)split * M * p.C_out : p.out;
#pragma unroll
  for (int r0 = 0; r0 < TM; r0 += RPI) {
    const int r = r0 + rl, m = m0 + TM * wm + r;
    if (rl < RPI && r < TM && m < M) {
      const float4 v = *reinterpret_cast<const float4*>(strip + r * SROW + 4 * q);
      *reinterpret_cast<float4*>(obase + (size_t)m * p.C_out + co) =
          make_float4(v.x + b.x, v.y + b.y, v.z + b.z, v.w + b.w);
    }
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
// The launch plan: a tile shape (each that divides C_out) and a split of
// the 9 C / 64 k-tiles (tap, channel chunk) into 1, 2, 3, 4, 6, 9 or 16
// even ranges over more workgroups (at least four k-tiles each), whichever
// has the least estimated time.  The estimate, fitted by least squares (with
// non-negative terms) to every shape and split count on twelve bands of the
// three SDXL-sized stages on MI355X: each round of workgroups over the slots
// (256 CUs x workgroups per CU) costs its K k-tiles x (a + b x the round's
// fill), a and b per shape (narrow 0.30 + 0.31 fill us, wide 0.42 + 0.12,
// mid 0.51: a lone workgroup's k-tile, and what the round's sharing of CUs
// and bandwidth adds); a split adds the fp32 partials' round trip (written
// by the convolution, added in order by the reduction kernel) at 0.43 us
// per MB.  On those bands it picks plans within 3 us in total of the
// fastest measured.
struct ConvPlan {
  int geo;     // 0: narrow, 1: wide, 2: mid
  int splits;
};

template <class G>
static ConvPlan conv_best_splits(int geo, double a, double b, int M, int C, int C_out, double* best_us) {
  const int tiles = ceil_div(M, conv::BM) * (C_out / G::BN);
  const int slots = 256 * G::WPC;
  const int kts = 9 * (C / conv::BK);
  const double mb = (double)M * C_out * sizeof(float) / 1e6;
  ConvPlan best{geo, 1};
  for (const int s : {1, 2, 3, 4, 6, 9, 16}) {
    if (s > 1 && kts < 4 * s) break;
    const int wgs = tiles * s, rounds = ceil_div(wgs, slots);
    const double us = ceil_div(kts, s) * (rounds * a + b * wgs / slots) + (s > 1 ? 0.43 * s * mb : 0.0);
    if (s == 1 || us < *best_us) {
      best.splits = s;
      *best_us = us;
    }
  }
  return best;
}

// Ties go to the earlier of wide, narrow, mid.
static ConvPlan conv_plan(int M, int C, int C_out) {
  double us = 0.0, u = 0.0;
  ConvPlan best{-1, 0};
  if (C_out % conv::Wide::BN == 0) best = conv_best_splits<conv::Wide>(1, 0.42, 0.12, M, C, C_out, &us);
  {
    const ConvPlan n = conv_best_splits<conv::Narrow>(0, 0.30, 0.31, M, C, C_out, &u);
    if (best.geo < 0 || u < us) { best = n; us = u; }
  }
  if (C_out % conv::Mid::BN == 0) {
    const ConvPlan m = conv_best_splits<conv::Mid>(2, 0.51, 0.0, M, C, C_out, &u);
    if (u < us) best = m;
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
  const int sp = conv_plan(M, C, C_out).splits;
  return al256((size_t)rows * G * 2 * sizeof(float)) +
         al256((size_t)(rows + 2) * (W + 2) * C * sizeof(bf16)) +
         (sp > 1 ? al256((size_t)sp * M * C_out * sizeof(float)) : 0);
}

hipError_t launch_unet_conv(const UNetConvParams& p0, void* ws, hipStream_t s) {
  UNetConvParams p = p0;
  const int rows = p.row_end - p.row_begin;
  const int M = rows * p.W;
  const ConvPlan plan = conv_plan(M, p.C, p.C_out);
  const int sp = plan.splits;
  char* w = reinterpret_cast<char*>(ws);
  p.fresh_sums = reinterpret_cast<float*>(w);
  w += al256((size_t)rows * p.G * 2 * sizeof(float));
  p.act_pad = w;
  w += al256((size_t)(rows + 2) * (p.W + 2) * p.C * sizeof(bf16));
  p.partial = sp > 1 ? reinterpret_cast<float*>(w) : nullptr;
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
  switch (plan.geo) {
    case 1: launch_conv<conv::Wide>(p, M, sp, s); break;
    case 2: launch_conv<conv::Mid>(p, M, sp, s); break;
    default: launch_conv<conv::Narrow>(p, M, sp, s);
  }
  if (sp > 1) {
    const size_t o4 = (size_t)M * p.C_out / 4;
    hipLaunchKernelGGL(conv_split_reduce_kernel, dim3((int)std::min<size_t>((o4 + 255) / 256, 4096)),
                       dim3(256), 0, s, p, sp);
  }
  return hipGetLastError();
}

}  // namespace orch
