// Projection GEMMs of the DiT block: y = A W^T + bias with fused epilogues
// (plain store, GELU, gated residual add into the fp32 residual stream, and
// the QKV scatter into the head-major Q buffer and the K / V^T buffer).
//
// bf16 path: MFMA tiles fed by direct-to-LDS loads (described at the kernel).
// fp32 path (and shapes the MFMA tiling does not cover): a 64x64 SIMT tile
// with 4x4 outputs per thread.
#include <cstdlib>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace orch {

// ---------------------------------------------------------------------------
// Epilogue.  A lane owns one output column n and, per call, four consecutive
// rows m..m+3 (the 32x32 MFMA accumulator layout).  Everything that depends
// on the column only is computed once per column in `Col`.
template <typename T, int EPI>
struct Epilogue {
  const EpiParams& ep;
  int M, N;

  struct Col {
    bool on;
    float bias;
    // QKV: destination of (branch 0, token 0), strides, factor (Q: q_scale)
    T* base;
    size_t bstride;
    int tstride;
    float mul = 1.0f;
    // RESIDUAL: gate pointer of branch 0
    const float* gate;
  };

  __device__ __forceinline__ int branch_of(int m) const {
    int b = 0;
    while (m >= (b + 1) * ep.rows_per_batch) ++b;
    return b;
  }

  __device__ __forceinline__ Col column(int n) const {
    Col c{};
    c.on = n < N;
    if (!c.on) return c;
    c.bias = ep.bias[n];
    if (EPI == kEpiResidual) c.gate = ep.gate + n;
    if (EPI == kEpiQkv) {
      const int which = n / ep.hidden;
      const int nn = n - which * ep.hidden;
      const int head = nn / ep.head_dim;
      const int dd = nn - head * ep.head_dim;
      const size_t ntot = (size_t)ep.kv_tokens;
      if (which == 0) {
        c.mul = ep.q_scale;
        c.base = reinterpret_cast<T*>(ep.q) + (size_t)head * ep.rows_per_batch * ep.head_dim + dd;
        c.bstride = (size_t)ep.heads * ep.rows_per_batch * ep.head_dim;
        c.tstride = ep.head_dim;
      } else if (which == 1) {
        c.base = reinterpret_cast<T*>(ep.kv) + ((size_t)head * ntot + ep.tok_offset) * ep.head_dim + dd;
        c.bstride = ep.kv_branch_stride;
        c.tstride = ep.head_dim;
      } else {
        c.base = reinterpret_cast<T*>(ep.kv) + ntot * ep.hidden +
                 ((size_t)head * ep.head_dim + dd) * ntot + ep.tok_offset;
        c.bstride = ep.kv_branch_stride;
        c.tstride = 1;
      }
    }
    return c;
  }

  __device__ __forceinline__ void store4(const Col& c, int m, int n, const float* v) const {
    if (!c.on) return;
    if (EPI == kEpiStore || EPI == kEpiGelu) {
      T* out = reinterpret_cast<T*>(ep.out) + n;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (m + r < M) {
          float y = v[r] + c.bias;
          if (EPI == kEpiGelu) y = gelu_fast(y);
          out[(size_t)(m + r) * N] = from_f<T>(y);
        }
      }
    } else if (EPI == kEpiResidual) {
      float* h = reinterpret_cast<float*>(ep.out) + n;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int mm = m + r;
        if (mm < M) h[(size_t)mm * N] += c.gate[(size_t)branch_of(mm) * ep.gate_stride] * (v[r] + c.bias);
      }
    } else {  // kEpiQkv
      const int b = branch_of(m);
      const int tok = m - b * ep.rows_per_batch;
      if (m + 3 < M && tok + 3 < ep.rows_per_batch) {
        T* dst = c.base + b * c.bstride + (size_t)tok * c.tstride;
        if (sizeof(T) == 2 && c.tstride == 1 && ((uintptr_t)dst & 7) == 0) {
          bf16x4 w;
#pragma unroll
          for (int r = 0; r < 4; ++r) w[r] = (bf16)((v[r] + c.bias) * c.mul);
          *reinterpret_cast<bf16x4*>(dst) = w;
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) dst[(size_t)r * c.tstride] = from_f<T>((v[r] + c.bias) * c.mul);
        }
      } else {
        for (int r = 0; r < 4; ++r) {
          const int mm = m + r;
          if (mm >= M) break;
          const int bb = branch_of(mm);
          const int tk = mm - bb * ep.rows_per_batch;
          c.base[bb * c.bstride + (size_t)tk * c.tstride] = from_f<T>((v[r] + c.bias) * c.mul);
        }
      }
    }
  }

  // GELU (tanh form) with tanh(u) = 1 - 2 / (exp(2u) + 1) on the fast exp;
  // used where the result is rounded to bf16.
  __device__ __forceinline__ static float gelu_fast(float x) {
    if (sizeof(T) == 4) return gelu_tanh_f(x);
    const float u = 0.7978845608028654f * (x + 0.044715f * x * x * x);
    const float e = __expf(2.0f * u);
    const float th = 1.0f - 2.0f * __builtin_amdgcn_rcpf(e + 1.0f);
    return 0.5f * x * (1.0f + th);
  }
};

// ---------------------------------------------------------------------------
// Epilogue of the MFMA GEMM.  The MFMAs produce transposed 32x32 blocks, so a
// lane holds C[m][n..n+3] (m = lane % 32 of the block, n = 8g + 4(lane / 32)).
// Each wave stages one 32-row strip of its tile at a time in a private LDS
// area (row stride TN + 4 floats, so the 16-byte writes of 16 rows land in
// distinct banks), then walks the strip in chunks along n: every global load
// and store is 16 bytes wide and a row's chunks are contiguous.  The QKV
// scatter writes Q and K rows the same way and walks V^T columns (8 tokens of
// one channel per lane).
template <int FM, int FN, int EPI>
struct StripEpilogue {
  static constexpr int TN = 32 * FN;
  static constexpr int LS = TN + 4;
  static constexpr int BYTES = 32 * LS * 4;  // LDS per wave

  const EpiParams& ep;
  int M, N;
  int split;   // kEpiPartial: this workgroup's k-split

  __device__ __forceinline__ int branch_of(int m) const {
    int b = 0;
    while (m >= (b + 1) * ep.rows_per_batch) ++b;
    return b;
  }

  // GELU, tanh form, as y * sigmoid(2u): 0.5 (1 + tanh(u)) = 1 / (1 + e^(-2u)),
  // u = sqrt(2/pi) (y + 0.044715 y^3), with e^(-2u) = exp2(y (c0 + c1 y^2))
  __device__ __forceinline__ static float act(float y) {
    if (EPI != kEpiGelu) return y;
    constexpr float c0 = -2.0f * 0.7978845608028654f * 1.4426950408889634f;
    constexpr float c1 = c0 * 0.044715f;
    const float e = __builtin_amdgcn_exp2f(y * fmaf(c1, y * y, c0));
    return y * __builtin_amdgcn_rcpf(1.0f + e);
  }

  // Operands of the epilogue loaded before the main loop, so their latency
  // hides behind the MFMAs: the bias of each store chunk, and for the gated
  // residual of one-strip tiles the fp32 h and gate rows as well.
  static constexpr int SIT = 32 * (TN / 8) / 64;       // store chunks per lane per strip
  static constexpr int RIT = 32 * (TN / 4) / 64;       // residual chunks per lane per strip
  static constexpr bool PRE_H = EPI == kEpiResidual && FM == 1 && RIT <= 8;
  // 8-channel bias chunks: one per store chunk, or a single one when every
  // chunk of a lane falls on the same columns (64 a multiple of TN / 8)
  static constexpr bool BIAS8 = EPI == kEpiStore || EPI == kEpiGelu || EPI == kEpiQkv;
  static constexpr int NB = (64 % (TN / 8) == 0) ? 1 : SIT;
  struct Pre {
    f32x4 b[BIAS8 ? NB : 1][2];
    float vb[EPI == kEpiQkv ? TN / 16 : 1];
    f32x4 h[PRE_H ? RIT : 1], g[PRE_H ? RIT : 1], rb[PRE_H ? RIT : 1];
  };

  __device__ __forceinline__ void prefetch(Pre& pre, int lane, int m0, int n0) const {
    if constexpr (BIAS8) {
      constexpr int CH = TN / 8;
#pragma unroll
      for (int q = 0; q < NB; ++q) {
        const int n = n0 + ((q * 64 + lane) % CH) * 8;
        pre.b[q][0] = *reinterpret_cast<const f32x4*>(ep.bias + n);
        pre.b[q][1] = *reinterpret_cast<const f32x4*>(ep.bias + n + 4);
      }
    }
    if constexpr (EPI == kEpiQkv) {
#pragma unroll
      for (int q = 0; q < TN / 16; ++q) pre.vb[q] = ep.bias[n0 + q * 16 + (lane >> 2)];
    }
    if constexpr (PRE_H) {
      constexpr int CH = TN / 4;
      const float* hb = reinterpret_cast<const float*>(ep.out);
#pragma unroll
      for (int q = 0; q < RIT; ++q) {
        const int f = q * 64 + lane, m = m0 + f / CH, n = n0 + (f % CH) * 4;
        const bool in = m < M;
        const int mm = in ? m : M - 1;
        pre.h[q] = *reinterpret_cast<const f32x4*>(hb + (size_t)mm * N + n);
        pre.g[q] = *reinterpret_cast<const f32x4*>(ep.gate + (size_t)branch_of(mm) * ep.gate_stride + n);
        pre.rb[q] = *reinterpret_cast<const f32x4*>(ep.bias + n);
      }
    }
  }

  // rows [mr, mr + 32) x columns [n0, n0 + TN) of C, staged in strip
  __device__ __forceinline__ void rows_store(const float* strip, int lane, int mr, int n0,
                                             const Pre& pre) const {
    constexpr int CH = TN / 8, IT = 32 * CH / 64;
    bf16* out = reinterpret_cast<bf16*>(ep.out);
#pragma unroll
    for (int q = 0; q < IT; ++q) {
      const int f = q * 64 + lane, row = f / CH, c = f % CH;
      const int m = mr + row, n = n0 + c * 8;
      const f32x4 x0 = *reinterpret_cast<const f32x4*>(strip + row * LS + c * 8);
      const f32x4 x1 = *reinterpret_cast<const f32x4*>(strip + row * LS + c * 8 + 4);
      if (m < M) {
        const f32x4 b0 = pre.b[NB == 1 ? 0 : q][0];
        const f32x4 b1 = pre.b[NB == 1 ? 0 : q][1];
        bf16x8 o;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          o[r] = from_f<bf16>(act(x0[r] + b0[r]));
          o[4 + r] = from_f<bf16>(act(x1[r] + b1[r]));
        }
        *reinterpret_cast<bf16x8*>(out + (size_t)m * N + n) = o;
      }
    }
  }

  __device__ __forceinline__ void rows_residual(const float* strip, int lane, int mr, int n0,
                                                const Pre& pre) const {
    constexpr int CH = TN / 4, IT = 32 * CH / 64;
    float* hb = reinterpret_cast<float*>(ep.out);
    f32x4 x[IT], hv[IT];
    // all loads first (or prefetched): the stores below may alias them as far
    // as the compiler knows, so this keeps at most one round trip per strip
#pragma unroll
    for (int q = 0; q < IT; ++q) {
      const int f = q * 64 + lane, row = f / CH, c = f % CH;
      const int m = mr + row, n = n0 + c * 4;
      x[q] = *reinterpret_cast<const f32x4*>(strip + row * LS + c * 4);
      if constexpr (PRE_H) hv[q] = pre.h[q];
      else hv[q] = m < M ? *reinterpret_cast<const f32x4*>(hb + (size_t)m * N + n) : f32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int q = 0; q < IT; ++q) {
      const int f = q * 64 + lane, row = f / CH, c = f % CH;
      const int m = mr + row, n = n0 + c * 4;
      if (m < M) {
        f32x4 g, b;
        if constexpr (PRE_H) {
          g = pre.g[q];
          b = pre.rb[q];
        } else {
          g = *reinterpret_cast<const f32x4*>(ep.gate + (size_t)branch_of(m) * ep.gate_stride + n);
          b = *reinterpret_cast<const f32x4*>(ep.bias + n);
        }
        f32x4 y;
#pragma unroll
        for (int r = 0; r < 4; ++r) y[r] = hv[q][r] + g[r] * (x[q][r] + b[r]);
        *reinterpret_cast<f32x4*>(hb + (size_t)m * N + n) = y;
      }
    }
  }

  __device__ __forceinline__ void rows_qkv(const float* strip, int lane, int mr, int n0,
                                           const Pre& pre) const {
    const int hd = ep.head_dim, hidden = ep.hidden, rpb = ep.rows_per_batch;
    const size_t ntot = (size_t)ep.kv_tokens;
    bf16* qb = reinterpret_cast<bf16*>(ep.q);
    bf16* kvb = reinterpret_cast<bf16*>(ep.kv);
    // Q and K: 8 channels of one head per lane (head_dim % 8 == 0)
    if (n0 < 2 * hidden) {
      constexpr int CH = TN / 8, IT = 32 * CH / 64;
#pragma unroll
      for (int q = 0; q < IT; ++q) {
        const int f = q * 64 + lane, row = f / CH, c = f % CH;
        const int m = mr + row, n = n0 + c * 8;
        if (m >= M || n >= 2 * hidden) continue;
        const f32x4 x0 = *reinterpret_cast<const f32x4*>(strip + row * LS + c * 8);
        const f32x4 x1 = *reinterpret_cast<const f32x4*>(strip + row * LS + c * 8 + 4);
        const f32x4 b0 = pre.b[NB == 1 ? 0 : q][0];
        const f32x4 b1 = pre.b[NB == 1 ? 0 : q][1];
        const int b = branch_of(m), tok = m - b * rpb;
        const int which = n >= hidden, nn = n - which * hidden;
        const float mul = which ? 1.0f : ep.q_scale;
        const int head = (int)__umulhi((unsigned)nn, ep.hd_magic), dd = nn - head * hd;
        bf16* dst = which == 0 ? qb + (((size_t)b * ep.heads + head) * rpb + tok) * hd + dd
                               : kvb + b * ep.kv_branch_stride + ((size_t)head * ntot + ep.tok_offset + tok) * hd + dd;
        bf16x8 o;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          o[r] = from_f<bf16>((x0[r] + b0[r]) * mul);
          o[4 + r] = from_f<bf16>((x1[r] + b1[r]) * mul);
        }
        *reinterpret_cast<bf16x8*>(dst) = o;
      }
    }
    // V^T [head][d][token]: 8 consecutive tokens of one channel per lane;
    // four lanes cover the strip's 32 tokens (64 contiguous bytes).  Token
    // groups 2 and 3 read their tokens rotated by four (8 LS = 32 mod 64 banks
    // would put them on the banks of groups 0 and 1; 4 LS = 16 mod 64 moves
    // them to the free ones), then swap the halves back.
    static_assert((4 * LS) % 64 == 16, "conflict-free V^T reads");
    if (n0 + TN > 2 * hidden) {
      constexpr int IT = TN * 4 / 64;
#pragma unroll
      for (int q = 0; q < IT; ++q) {
        const int col = q * 16 + (lane >> 2), grp = lane & 3;
        const int n = n0 + col;
        if (n < 2 * hidden) continue;
        const int rot = (grp >> 1) * 4;
        float v[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const float x = strip[(grp * 8 + ((t + rot) & 7)) * LS + col];   // token t ^ rot
          v[t] = x;
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const float a = v[t], b = v[t + 4];
          v[t] = rot ? b : a;
          v[t + 4] = rot ? a : b;
        }
        const float bias = pre.vb[q];
        const int nn = n - 2 * hidden, head = (int)__umulhi((unsigned)nn, ep.hd_magic), dd = nn - head * hd;
        bf16* vt = kvb + ntot * hidden + ((size_t)head * hd + dd) * ntot + ep.tok_offset;
        const int m = mr + grp * 8;
        const int b = m < M ? branch_of(m) : 0, tok = m - b * rpb;
        bf16* dst = vt + b * ep.kv_branch_stride + tok;
        if (m + 7 < M && tok + 7 < rpb && ((uintptr_t)dst & 15) == 0) {
          bf16x8 o;
#pragma unroll
          for (int t = 0; t < 8; ++t) o[t] = from_f<bf16>(v[t] + bias);
          *reinterpret_cast<bf16x8*>(dst) = o;
        } else {
#pragma unroll
          for (int t = 0; t < 8; ++t) {
            const int mm = m + t;
            if (mm < M) {
              const int bb = branch_of(mm);
              vt[bb * ep.kv_branch_stride + (mm - bb * rpb)] = from_f<bf16>(v[t] + bias);
            }
          }
        }
      }
    }
  }

  // a k-split's partial sums, fp32 rows of ws[split]
  __device__ __forceinline__ void rows_partial(const float* strip, int lane, int mr, int n0) const {
    constexpr int CH = TN / 4, IT = 32 * CH / 64;
    float* wb = ep.ws + (size_t)split * M * N;
#pragma unroll
    for (int q = 0; q < IT; ++q) {
      const int f = q * 64 + lane, row = f / CH, c = f % CH;
      const int m = mr + row, n = n0 + c * 4;
      if (m < M)
        *reinterpret_cast<f32x4*>(wb + (size_t)m * N + n) = *reinterpret_cast<const f32x4*>(strip + row * LS + c * 4);
    }
  }

  // the wave's tile: rows [m0, m0 + 32 FM), columns [n0, n0 + TN)
  __device__ __forceinline__ void run(const f32x16 (&acc)[FM][FN], float* strip, int lane, int m0,
                                      int n0, const Pre& pre) const {
    const int lr = lane & 31, h = lane >> 5;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g)
          *reinterpret_cast<f32x4*>(strip + lr * LS + j * 32 + 8 * g + 4 * h) =
              f32x4{acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
      if constexpr (EPI == kEpiStore || EPI == kEpiGelu) rows_store(strip, lane, m0 + 32 * i, n0, pre);
      else if constexpr (EPI == kEpiResidual) rows_residual(strip, lane, m0 + 32 * i, n0, pre);
      else if constexpr (EPI == kEpiPartial) rows_partial(strip, lane, m0 + 32 * i, n0);
      else rows_qkv(strip, lane, m0 + 32 * i, n0, pre);
    }
  }
};

// ---------------------------------------------------------------------------
// bf16 MFMA GEMM.
//
// BM x BN x BK block tile over WM x WN waves; each wave owns a (BM/WM) x
// (BN/WN) block of v_mfma_f32_32x32x16_bf16 accumulators in fp32.  Operands go
// global -> LDS with the direct-to-LDS load (16 bytes per lane, 1 KB per wave
// instruction, no register staging) into a ring of S stages.  LDS rows are
// 2*BK bytes, unpadded; the 16-byte chunks of row r are XOR-swizzled by
// (r / Q) % CPR so that a fragment read (16 lanes = 16 rows at one logical
// chunk) touches 64 distinct banks.  One barrier per k-tile; the loads of
// tile kt+S-1 are interleaved with the MFMAs of tile kt.
// Compile-time layout of one configuration.
template <int BM, int BN, int BK, int WM, int WN, int S>
struct GemmGeo {
  static constexpr int NW = WM * WN;
  static constexpr int TM = BM / WM, TN = BN / WN;  // wave tile
  static constexpr int FM = TM / 32, FN = TN / 32;  // 32x32 blocks per wave
  static constexpr int CPR = BK / 8;                // 16-byte chunks per row
  static constexpr int RPL = 1024 / (2 * BK);       // rows per wave-level load
  static constexpr int Q = 128 / BK;                // rows per 256-byte bank sweep
  static constexpr int IA = BM / (NW * RPL), IB = BN / (NW * RPL);
  static constexpr int LPT = IA + IB;               // loads per lane per k-tile
  static constexpr int STAGE = (BM + BN) * BK * 2;  // bytes per stage
  static constexpr int KK = BK / 16;                // MFMA k-steps per k-tile
  // next-tile loads issued per k-step: all in the first with two stages (they
  // get one tile of compute to land), else spread over the k-steps
  static constexpr int LPK = S == 2 ? LPT : (LPT + KK - 1) / KK;
  static_assert(NW == 4 || NW == 8, "four or eight waves");
  static_assert(BK == 32 || BK == 64, "k-tile");
  static_assert(FM >= 1 && FN >= 1 && TM % 32 == 0 && TN % 32 == 0, "wave tile");
  static_assert(BM % (NW * RPL) == 0 && BN % (NW * RPL) == 0, "rows per wave");
  static_assert(S >= 2 && S <= 8 && LPT * (S - 1) < 64, "pipeline depth");
  static_assert(S * STAGE <= 160 * 1024, "LDS");
};

template <int BM, int BN, int BK, int WM, int WN, int S, int EPI>
__global__ __launch_bounds__(64 * WM * WN) void gemm_bf16_kernel(const bf16* __restrict__ A,
                                                        const bf16* __restrict__ W, int M, int N,
                                                        int K, int ldk, int tiles_m, int tiles_n,
                                                        EpiParams ep) {
  using G = GemmGeo<BM, BN, BK, WM, WN, S>;
  constexpr int FM = G::FM, FN = G::FN, KK = G::KK, IA = G::IA, LPT = G::LPT, LPK = G::LPK;

  extern __shared__ __attribute__((aligned(1024))) char smem[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;

  // K is this workgroup's k extent, ldk the row stride of A and W: with a
  // k-split, workgroup b takes split b / T, keys [split K, (split + 1) K).
  // Tile order inside a split: XCD-major, then groups of 8 tile rows,
  // column-major inside.
  const int T = tiles_m * tiles_n;
  const int split = __builtin_amdgcn_readfirstlane(blockIdx.x / T);
  int pid = blockIdx.x - split * T;
  const int per = T / 8;
  if (pid < per * 8) pid = (pid & 7) * per + (pid >> 3);
  constexpr int GROUP = 8;
  const int gid = pid / (GROUP * tiles_n);
  const int first_m = gid * GROUP;
  const int gsz = min(tiles_m - first_m, GROUP);
  const int tile_m = first_m + (pid % (GROUP * tiles_n)) % gsz;
  const int tile_n = (pid % (GROUP * tiles_n)) / gsz;
  const int m0 = tile_m * BM, n0 = tile_n * BN;

  // byte offset of this lane's source chunk in each wave-level load: load j
  // covers tile rows (j * NW + wave) * RPL .. + RPL - 1 (A rows first, then
  // W rows); A rows past M re-read row M - 1
  const int prow = lane / G::CPR;
  const int pchunk = lane % G::CPR;
  unsigned off[LPT];
#pragma unroll
  for (int j = 0; j < LPT; ++j) {
    const int i = j < IA ? j : j - IA;
    const int r = (i * G::NW + wave) * G::RPL + prow;
    const int lchunk = pchunk ^ ((r / G::Q) % G::CPR);
    const unsigned row = j < IA ? (unsigned)min(m0 + r, M - 1) : (unsigned)(n0 + r);
    off[j] = (row * (unsigned)ldk + lchunk * 8) * 2u;
  }
  const char* gA = reinterpret_cast<const char*>(A + (size_t)split * K);
  const char* gW = reinterpret_cast<const char*>(W + (size_t)split * K);

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // fragment read offsets: row = wave tile row + lrow, logical chunk 2 kk + h
  const int lrow = lane & 31;
  const int h = lane >> 5;
  int koff[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) koff[kk] = ((2 * kk + h) ^ ((lrow / G::Q) % G::CPR)) * 16;
  const int arow = (wm * G::TM + lrow) * BK * 2;
  const int brow = BM * BK * 2 + (wn * G::TN + lrow) * BK * 2;

  const int KT = K / BK;  // >= S - 1 (checked by the launcher)

  // load j of k-tile kt into stage st
  auto dma = [&](auto jc, int kt_, int st_) {
    constexpr int j = decltype(jc)::value;
    constexpr int i = j < IA ? j : j - IA;
    constexpr int part = j < IA ? 0 : BM * BK * 2;
    char* dst = smem + st_ * G::STAGE + part + (i * G::NW + wave) * G::RPL * BK * 2;
    const char* src = (j < IA ? gA : gW) + (unsigned)kt_ * (BK * 2) + off[j];
    __builtin_amdgcn_global_load_lds((const ORCH_GLB void*)src, (ORCH_LDS void*)dst, 16, 0, 0);
  };

  // the MFMAs of stage st; with issue, the loads of tile ikt into stage ist
  // go between them.  Emission order is fixed slot by slot (a scheduling
  // fence after each): MFMA e of k-step kk, then its share of the reads of
  // k-step kk+1's fragments, then its share of the next tile's loads.
  auto compute = [&](int st, auto issue_c, int ikt, int ist) {
    constexpr bool ISSUE = decltype(issue_c)::value;
    constexpr int NM = FM * FN, ND = FM + FN;
    const char* base = smem + st * G::STAGE;
    bf16x8 a[2][FM], b[2][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
      a[0][i] = *reinterpret_cast<const bf16x8*>(base + arow + i * 32 * BK * 2 + koff[0]);
#pragma unroll
    for (int j = 0; j < FN; ++j)
      b[0][j] = *reinterpret_cast<const bf16x8*>(base + brow + j * 32 * BK * 2 + koff[0]);
    __builtin_amdgcn_sched_barrier(0);
    static_for<0, KK>([&](auto kkc) {
      constexpr int kk = decltype(kkc)::value;
      constexpr int cur = kk & 1;
      constexpr int nd = kk + 1 < KK ? ND : 0;
      constexpr int l0 = cmin(kk * LPK, LPT), nl = ISSUE ? cmin(kk * LPK + LPK, LPT) - l0 : 0;
      static_for<0, NM>([&](auto ec) {
        constexpr int e = decltype(ec)::value;
        constexpr int i = e / FN, j = e % FN;
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[cur][j], a[cur][i], acc[i][j], 0, 0, 0);
        static_for<e * nd / NM, (e + 1) * nd / NM>([&](auto dc) {
          constexpr int d = decltype(dc)::value;
          if constexpr (d < FM)
            a[cur ^ 1][d] = *reinterpret_cast<const bf16x8*>(base + arow + d * 32 * BK * 2 + koff[kk + 1]);
          else
            b[cur ^ 1][d - FM] =
                *reinterpret_cast<const bf16x8*>(base + brow + (d - FM) * 32 * BK * 2 + koff[kk + 1]);
        });
        static_for<l0 + e * nl / NM, l0 + (e + 1) * nl / NM>([&](auto jc) { dma(jc, ikt, ist); });
        __builtin_amdgcn_sched_barrier(0);
      });
    });
  };

  // epilogue operands first: the oldest loads, covered by the main loop
  using E = StripEpilogue<FM, FN, EPI>;
  const E epi{ep, M, N, split};
  typename E::Pre pre;
  epi.prefetch(pre, lane, m0 + wm * G::TM, n0 + wn * G::TN);

#pragma unroll
  for (int s = 0; s < S - 1; ++s) static_for<0, LPT>([&](auto jc) { dma(jc, s, s); });
  int kt = 0;
  for (; kt + S - 1 < KT; ++kt) {
    wait_vmcnt<(S - 2) * LPT>();
    lds_barrier();
    compute(kt % S, std::true_type{}, kt + S - 1, (kt + S - 1) % S);
  }
  // drain: the last S-1 tiles, nothing more to issue
  static_for<0, S - 2>([&](auto rc) {
    wait_vmcnt<(S - 2 - decltype(rc)::value) * LPT>();
    lds_barrier();
    compute(kt % S, std::false_type{}, 0, 0);
    ++kt;
  });
  wait_vmcnt<0>(); lds_barrier(); compute(kt % S, std::false_type{}, 0, 0);

  // epilogue: the stage buffers become per-wave staging strips
  static_assert(G::NW * E::BYTES <= S * G::STAGE, "epilogue staging fits the stage buffers");
  lds_barrier();
  epi.run(acc, reinterpret_cast<float*>(smem + wave * E::BYTES), lane, m0 + wm * G::TM, n0 + wn * G::TN,
          pre);
}

// ---------------------------------------------------------------------------
// SIMT GEMM (fp32, and fallback shapes)
namespace simt_gemm {
constexpr int BM = 64, BN = 64, BK = 16;
}

template <typename T, int EPI>
__global__ __launch_bounds__(256) void gemm_simt_kernel(const T* __restrict__ A,
                                                        const T* __restrict__ W, int M, int N,
                                                        int K, EpiParams ep) {
  using namespace simt_gemm;
  __shared__ float sA[BK][BM + 4];
  __shared__ float sB[BK][BN + 4];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;

  for (int k0 = 0; k0 < K; k0 += BK) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      int idx = tid + 256 * e;
      int r = idx >> 4, kk = idx & 15;
      int gk = k0 + kk;
      int gm = m0 + r, gn = n0 + r;
      sA[kk][r] = (gm < M && gk < K) ? to_f<T>(A[(size_t)gm * K + gk]) : 0.f;
      sB[kk][r] = (gn < N && gk < K) ? to_f<T>(W[(size_t)gn * K + gk]) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = sA[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = sB[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  const Epilogue<T, EPI> epi{ep, M, N};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n = n0 + tx * 4 + j;
    float v[4] = {acc[0][j], acc[1][j], acc[2][j], acc[3][j]};
    epi.store4(epi.column(n), m0 + ty * 4, n, v);
  }
}

// ---------------------------------------------------------------------------
// Tile selection.  ORCH_GEMM_TILE=<index> forces a configuration (tuning).
struct TileCfg {
  int bm, bn, bk, waves, stages;
  float eff;  // measured relative throughput of the shape on a full machine
};
static const TileCfg kTiles[] = {
    {256, 256, 64, 8, 2, 0.80f},
    {256, 192, 64, 8, 2, 1.00f},
    {128, 128, 64, 8, 4, 0.75f},
    {128, 64, 64, 4, 2, 0.30f},  // fallback: any N % 64 == 0, K % 64 == 0
};
constexpr int kNumTiles = sizeof(kTiles) / sizeof(kTiles[0]);
constexpr int kFallbackTile = kNumTiles - 1;

static int forced_tile() {
  const char* s = getenv("ORCH_GEMM_TILE");
  return s ? atoi(s) : -1;
}

static bool tile_fits(const TileCfg& t, int N, int K) {
  return N % t.bn == 0 && K % t.bk == 0 && K / t.bk >= t.stages - 1;
}

// Pick the configuration with the least estimated time: whole rounds of tiles
// over the 256 CUs times the tile area, divided by the tile's relative
// throughput per CU.  The throughputs were measured on the DiT-XL projection
// shapes (K = 1152 and 4608, M from 768 to 8192): the 256x192 tile is the
// fastest per CU, the 256x256 one wins when it fills the machine in one round
// where 256x192 needs two, and the 128x128 one when 256-row tiles would leave
// most CUs idle.
static int pick_tile(int M, int N, int K) {
  const int f = forced_tile();
  if (f >= 0 && f < kNumTiles && tile_fits(kTiles[f], N, K)) return f;
  int best = kFallbackTile;
  float best_cost = 0.0f;
  for (int c = 0; c < kNumTiles; ++c) {
    const TileCfg& t = kTiles[c];
    if (!tile_fits(t, N, K)) continue;
    const int tiles = ceil_div(M, t.bm) * (N / t.bn);
    const float cost = (float)ceil_div(tiles, 256) * t.bm * t.bn / t.eff;
    if (best_cost == 0.0f || cost < best_cost) {
      best = c;
      best_cost = cost;
    }
  }
  return best;
}

bool gemm_uses_mfma(int N, int K, int dtype) {
  return dtype == kBF16 && N % 64 == 0 && K % 64 == 0;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// The MFMA kernel moves 16-byte chunks of every operand and output; shapes
// or pointers that do not allow that take the SIMT kernel.
static bool mfma_path_ok(const void* A, const void* W, int N, int K, int epi, const EpiParams& ep,
                         int dtype) {
  if (!gemm_uses_mfma(N, K, dtype) || !aligned16(A) || !aligned16(W) || !aligned16(ep.bias))
    return false;
  if (epi == kEpiResidual) return aligned16(ep.out) && aligned16(ep.gate) && ep.gate_stride % 4 == 0;
  if (epi == kEpiQkv)
    return aligned16(ep.q) && aligned16(ep.kv) && ep.head_dim % 8 == 0 && ep.kv_branch_stride % 8 == 0 &&
           ep.hidden < 65536;
  return aligned16(ep.out);
}

template <int BM, int BN, int BK, int WM, int WN, int S, int EPI>
static void launch_tile(const void* A, const void* W, int M, int N, int K, const EpiParams& ep0,
                        hipStream_t s, int splits = 1) {
  const int tm = ceil_div(M, BM), tn = N / BN;
  constexpr int lds = S * GemmGeo<BM, BN, BK, WM, WN, S>::STAGE;
  EpiParams ep = ep0;
  // head = umulhi(channel, ceil(2^32 / head_dim)): exact for channels < 2^16
  if (EPI == kEpiQkv) ep.hd_magic = (unsigned)((0x100000000ull + ep.head_dim - 1) / ep.head_dim);
  auto kern = gemm_bf16_kernel<BM, BN, BK, WM, WN, S, EPI>;
  static bool attr = [&] {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                              hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    return true;
  }();
  (void)attr;
  hipLaunchKernelGGL(kern, dim3(tm * tn * splits), dim3(64 * WM * WN), lds, s,
                     reinterpret_cast<const bf16*>(A), reinterpret_cast<const bf16*>(W), M, N,
                     K / splits, K, tm, tn, ep);
}

// Sum of the k-splits' partials, then the caller's epilogue (bias, GELU,
// gated residual or the QKV scatter): four rows of one column per thread, the
// splits added in order.
template <typename T, int EPI>
__global__ __launch_bounds__(256) void gemm_split_reduce_kernel(int splits, int M, int N,
                                                                EpiParams ep) {
  const int n = blockIdx.x * 256 + threadIdx.x;
  const int m = blockIdx.y * 4;
  if (n >= N) return;
  const Epilogue<T, EPI> epi{ep, M, N};
  float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int sp = 0; sp < splits; ++sp) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (m + r < M) v[r] += ep.ws[((size_t)sp * M + m + r) * N + n];
  }
  epi.store4(epi.column(n), m, n, v);
}

// K-split of a GEMM whose tiles leave most of the machine idle (at most 128
// tiles for 256 CUs): splits s with s * tiles <= 256, at least 8 k-tiles per
// split, s dividing the k-tiles and the partials fitting the workspace.
// (Splits that take more than one round, e.g. 144 tiles in three splits, or
// 378 in two, measured slower than no split: the partials' round trip
// through HBM costs more than the idle CUs.)
static int split_plan(int M, int N, int K, const TileCfg& t, size_t ws_elems) {
  const int tiles = ceil_div(M, t.bm) * (N / t.bn);
  const int kt = K / t.bk;
  if (tiles > 128) return 1;
  int sp = cmin(256 / tiles, kt / 8);
  while (sp > 1 && (kt % sp != 0 || (size_t)sp * M * N > ws_elems)) --sp;
  return sp;
}

template <int EPI>
static void launch_tile_cfg(int c, const void* A, const void* W, int M, int N, int K,
                            const EpiParams& ep, hipStream_t s, int splits) {
  switch (c) {
    case 0: launch_tile<256, 256, 64, 2, 4, 2, EPI>(A, W, M, N, K, ep, s, splits); break;
    case 1: launch_tile<256, 192, 64, 4, 2, 2, EPI>(A, W, M, N, K, ep, s, splits); break;
    case 2: launch_tile<128, 128, 64, 4, 2, 4, EPI>(A, W, M, N, K, ep, s, splits); break;
    default: launch_tile<128, 64, 64, 2, 2, 2, EPI>(A, W, M, N, K, ep, s, splits); break;
  }
}

template <int EPI>
static hipError_t launch_gemm_epi(const void* A, const void* W, int M, int N, int K,
                                  const EpiParams& ep, int dtype, hipStream_t s) {
  if (M <= 0 || N <= 0 || K <= 0) return hipSuccess;
  if (mfma_path_ok(A, W, N, K, EPI, ep, dtype)) {
    const int c = pick_tile(M, N, K);
    const int sp = ep.ws && aligned16(ep.ws) ? split_plan(M, N, K, kTiles[c], ep.ws_elems) : 1;
    if (sp > 1) {
      launch_tile_cfg<kEpiPartial>(c, A, W, M, N, K, ep, s, sp);
      hipLaunchKernelGGL((gemm_split_reduce_kernel<bf16, EPI>), dim3(ceil_div(N, 256), ceil_div(M, 4)),
                         dim3(256), 0, s, sp, M, N, ep);
    } else {
      launch_tile_cfg<EPI>(c, A, W, M, N, K, ep, s, 1);
    }
  } else {
    dim3 grid(ceil_div(N, simt_gemm::BN), ceil_div(M, simt_gemm::BM));
    if (dtype == kBF16)
      hipLaunchKernelGGL((gemm_simt_kernel<bf16, EPI>), grid, dim3(256), 0, s,
                         reinterpret_cast<const bf16*>(A), reinterpret_cast<const bf16*>(W), M,
                         N, K, ep);
    else
      hipLaunchKernelGGL((gemm_simt_kernel<float, EPI>), grid, dim3(256), 0, s,
                         reinterpret_cast<const float*>(A), reinterpret_cast<const float*>(W),
                         M, N, K, ep);
  }
  return hipGetLastError();
}

size_t gemm_split_workspace_elems(int M, int N, int K, int dtype) {
  if (M <= 0 || !gemm_uses_mfma(N, K, dtype)) return 0;
  const int c = pick_tile(M, N, K);
  if (!tile_fits(kTiles[c], N, K)) return 0;
  const int sp = split_plan(M, N, K, kTiles[c], (size_t)-1);
  return sp > 1 ? (size_t)sp * M * N : 0;
}

hipError_t launch_gemm(const void* A, const void* W, int M, int N, int K, int epi,
                       const EpiParams& ep, int dtype, hipStream_t s) {
  switch (epi) {
    case kEpiStore: return launch_gemm_epi<kEpiStore>(A, W, M, N, K, ep, dtype, s);
    case kEpiGelu: return launch_gemm_epi<kEpiGelu>(A, W, M, N, K, ep, dtype, s);
    case kEpiResidual: return launch_gemm_epi<kEpiResidual>(A, W, M, N, K, ep, dtype, s);
    case kEpiQkv: return launch_gemm_epi<kEpiQkv>(A, W, M, N, K, ep, dtype, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace orch
