// Projection GEMMs of the DiT block: y = A W^T + bias with fused epilogues
// (plain store, GELU, gated residual add into the fp32 residual stream, and
// the QKV scatter into the head-major Q buffer and the K / V^T buffer).
//
// bf16 path: BM x BN x 64 tiles, WM x WN waves, each wave a (BM/WM) x (BN/WN)
// block of v_mfma_f32_32x32x16_bf16 with fp32 accumulation; operands staged
// global -> registers -> padded LDS rows (144 B, conflict-free 16-byte reads),
// double buffered, one barrier per k-tile.  fp32 path (and shapes the MFMA
// tiling does not cover): a 64x64 SIMT tile with 4x4 outputs per thread.
#include <cstdlib>

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
    // QKV: destination of (branch 0, token 0) and strides
    T* base;
    size_t bstride;
    int tstride;
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
          for (int r = 0; r < 4; ++r) w[r] = (bf16)(v[r] + c.bias);
          *reinterpret_cast<bf16x4*>(dst) = w;
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) dst[(size_t)r * c.tstride] = from_f<T>(v[r] + c.bias);
        }
      } else {
        for (int r = 0; r < 4; ++r) {
          const int mm = m + r;
          if (mm >= M) break;
          const int bb = branch_of(mm);
          const int tk = mm - bb * ep.rows_per_batch;
          c.base[bb * c.bstride + (size_t)tk * c.tstride] = from_f<T>(v[r] + c.bias);
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
// bf16 MFMA GEMM
constexpr int kBK = 64;
constexpr int kLdsStride = kBK + 8;  // bf16 per LDS row: 144 B

template <int BM, int BN, int WM, int WN, int EPI>
__global__ __launch_bounds__(64 * WM * WN) void gemm_bf16_mfma_kernel(
    const bf16* __restrict__ A, const bf16* __restrict__ W, int M, int N, int K, EpiParams ep) {
  constexpr int NT = 64 * WM * WN;           // threads
  constexpr int TM = BM / WM, TN = BN / WN;  // wave tile
  constexpr int FM = TM / 32, FN = TN / 32;  // 32x32 blocks per wave
  constexpr int CH_A = BM * (kBK / 8);       // 16-byte chunks per tile
  constexpr int CH_B = BN * (kBK / 8);
  constexpr int LA = (CH_A + NT - 1) / NT;
  constexpr int LB = (CH_B + NT - 1) / NT;
  static_assert(CH_A % NT == 0 && CH_B % NT == 0, "tile must split evenly over threads");

  __shared__ __attribute__((aligned(16))) bf16 sA[2][BM * kLdsStride];
  __shared__ __attribute__((aligned(16))) bf16 sB[2][BN * kLdsStride];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int m0 = blockIdx.y * BM;
  const int n0 = blockIdx.x * BN;

  // this thread's global chunks: chunk c = tid + NT*i -> row c/8, k-chunk c%8
  const bf16* pa[LA];
  const bf16* pb[LB];
  int la[LA], lb[LB];
#pragma unroll
  for (int i = 0; i < LA; ++i) {
    const int c = tid + NT * i;
    const int r = c >> 3, kc = c & 7;
    pa[i] = A + (size_t)min(m0 + r, M - 1) * K + kc * 8;
    la[i] = r * kLdsStride + kc * 8;
  }
#pragma unroll
  for (int i = 0; i < LB; ++i) {
    const int c = tid + NT * i;
    const int r = c >> 3, kc = c & 7;
    pb[i] = W + (size_t)(n0 + r) * K + kc * 8;
    lb[i] = r * kLdsStride + kc * 8;
  }

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int KT = K / kBK;
  uint4 ra[LA], rb[LB];
#pragma unroll
  for (int i = 0; i < LA; ++i) ra[i] = *reinterpret_cast<const uint4*>(pa[i]);
#pragma unroll
  for (int i = 0; i < LB; ++i) rb[i] = *reinterpret_cast<const uint4*>(pb[i]);
#pragma unroll
  for (int i = 0; i < LA; ++i) *reinterpret_cast<uint4*>(&sA[0][la[i]]) = ra[i];
#pragma unroll
  for (int i = 0; i < LB; ++i) *reinterpret_cast<uint4*>(&sB[0][lb[i]]) = rb[i];
  __syncthreads();

  const int lrow = lane & 31;
  const int lk = (lane >> 5) * 8;
  const bf16* sa_base = &sA[0][(wm * TM + lrow) * kLdsStride + lk];
  const bf16* sb_base = &sB[0][(wn * TN + lrow) * kLdsStride + lk];

  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    // prefetch the next k-tile (the last iteration re-reads the last tile;
    // it is not stored)
    const int knext = (kt + 1 < KT ? kt + 1 : kt) * kBK;
#pragma unroll
    for (int i = 0; i < LA; ++i) ra[i] = *reinterpret_cast<const uint4*>(pa[i] + knext);
#pragma unroll
    for (int i = 0; i < LB; ++i) rb[i] = *reinterpret_cast<const uint4*>(pb[i] + knext);

    const bf16* sa = sa_base + buf * (BM * kLdsStride);
    const bf16* sb = sb_base + buf * (BN * kLdsStride);
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      bf16x8 a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        a[i] = *reinterpret_cast<const bf16x8*>(sa + i * 32 * kLdsStride + kk * 16);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        b[j] = *reinterpret_cast<const bf16x8*>(sb + j * 32 * kLdsStride + kk * 16);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < KT) {
      bf16* da = &sA[buf ^ 1][0];
      bf16* db = &sB[buf ^ 1][0];
#pragma unroll
      for (int i = 0; i < LA; ++i) *reinterpret_cast<uint4*>(da + la[i]) = ra[i];
#pragma unroll
      for (int i = 0; i < LB; ++i) *reinterpret_cast<uint4*>(db + lb[i]) = rb[i];
    }
    __syncthreads();
  }

  // accumulator layout of a 32x32 MFMA block: lane holds column lane%32,
  // register r holds row 8*(r/4) + 4*(lane/32) + r%4.
  const Epilogue<bf16, EPI> epi{ep, M, N};
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const int n = n0 + wn * TN + j * 32 + (lane & 31);
    const typename Epilogue<bf16, EPI>::Col col = epi.column(n);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int m = m0 + wm * TM + i * 32 + 8 * g + 4 * (lane >> 5);
        float v[4] = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                      acc[i][j][4 * g + 3]};
        epi.store4(col, m, n, v);
      }
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA GEMM with direct-to-LDS loads (global_load_lds_dwordx4) into an
// S-stage ring of BK-wide k-tiles.  LDS rows hold BK bf16 without padding and
// are swizzled for the 64-bank LDS, whose ds_read_b128 serves 16 lanes per
// cycle: with Q = 256 B / row bytes rows per bank sweep, the 16-byte chunk c
// of row r is stored at chunk c ^ ((r / Q) mod (BK / 8)), so the 16 rows one
// read cycle touches land on 16 distinct 4-bank groups.  Each wave-level
// load writes 1 KB (1024 / (2 BK) rows) of a stage; a manual vmcnt wait plus
// s_barrier publishes a stage, so up to S-1 k-tiles are in flight while one
// is consumed.  Operand fragments are double buffered across the 16-deep
// k-steps so LDS reads overlap the MFMAs.  Tiles are visited in XCD-major,
// row-grouped order so workgroups sharing an XCD's L2 share operand rows.

#define ORCH_LDS __attribute__((address_space(3)))
#define ORCH_GLB __attribute__((address_space(1)))

// s_waitcnt with vmcnt = n and the other counters left free (gfx9 encoding).
template <int n>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14));
}

__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int BM, int BN, int BK, int WM, int WN, int S, bool SCHED, int EPI>
__global__ __launch_bounds__(64 * WM * WN) void gemm_bf16_dma_kernel(const bf16* __restrict__ A,
                                                            const bf16* __restrict__ W, int M,
                                                            int N, int K, int tiles_m, int tiles_n,
                                                            EpiParams ep) {
  constexpr int NW = WM * WN;
  static_assert(NW == 4 || NW == 8, "four or eight waves");
  static_assert(BK == 32 || BK == 64, "k-tile");
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int CPR = BK / 8;                // 16-byte chunks per row
  constexpr int RPL = 1024 / (2 * BK);       // rows per wave-level load
  constexpr int Q = 128 / BK;                // rows per 256-byte bank sweep
  static_assert(BM % (NW * RPL) == 0 && BN % (NW * RPL) == 0, "rows per wave");
  constexpr int IA = BM / (NW * RPL), IB = BN / (NW * RPL);
  constexpr int LPT = IA + IB;               // loads per thread per stage
  constexpr int STAGE = (BM + BN) * BK;      // bf16 elements per stage
  constexpr int KK = BK / 16;
  static_assert(S >= 2 && LPT * (S - 1) < 64, "pipeline depth");

  extern __shared__ __attribute__((aligned(1024))) bf16 smem[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  // tile order: XCD-major, then groups of 8 tile rows, column-major inside
  int pid = blockIdx.x;
  const int T = tiles_m * tiles_n;
  const int per = T / 8;
  if (pid < per * 8) pid = (pid & 7) * per + (pid >> 3);
  constexpr int GROUP = 8;
  const int gid = pid / (GROUP * tiles_n);
  const int first_m = gid * GROUP;
  const int gsz = min(tiles_m - first_m, GROUP);
  const int tile_m = first_m + (pid % (GROUP * tiles_n)) % gsz;
  const int tile_n = (pid % (GROUP * tiles_n)) / gsz;
  const int m0 = tile_m * BM, n0 = tile_n * BN;

  // this lane's source chunk of each wave-level load
  const int prow = lane / CPR;          // row inside the 1 KB block
  const int pchunk = lane % CPR;        // physical chunk it fills
  const bf16* srcA[IA];
  const bf16* srcB[IB];
#pragma unroll
  for (int i = 0; i < IA; ++i) {
    const int r = (i * NW + wave) * RPL + prow;
    const int lchunk = pchunk ^ ((r / Q) % CPR);
    srcA[i] = A + (size_t)min(m0 + r, M - 1) * K + lchunk * 8;
  }
#pragma unroll
  for (int i = 0; i < IB; ++i) {
    const int r = (i * NW + wave) * RPL + prow;
    const int lchunk = pchunk ^ ((r / Q) % CPR);
    srcB[i] = W + (size_t)(n0 + r) * K + lchunk * 8;
  }

  auto issue = [&](int kt, int st) {
    bf16* sa = smem + st * STAGE;
    bf16* sb = sa + BM * BK;
    const int ko = kt * BK;
#pragma unroll
    for (int i = 0; i < IA; ++i)
      __builtin_amdgcn_global_load_lds((const ORCH_GLB void*)(srcA[i] + ko),
                                       (ORCH_LDS void*)(sa + (i * NW + wave) * RPL * BK), 16, 0, 0);
#pragma unroll
    for (int i = 0; i < IB; ++i)
      __builtin_amdgcn_global_load_lds((const ORCH_GLB void*)(srcB[i] + ko),
                                       (ORCH_LDS void*)(sb + (i * NW + wave) * RPL * BK), 16, 0, 0);
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // operand read offsets: row r = (wave tile row) + lrow; logical chunk 2 kk + h
  const int lrow = lane & 31;
  const int h = lane >> 5;
  int koff[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) koff[kk] = ((2 * kk + h) ^ ((lrow / Q) % CPR)) * 8;
  const int arow = (wm * TM + lrow) * BK;
  const int brow = BM * BK + (wn * TN + lrow) * BK;

  auto compute = [&](int st) {
    const bf16* base = smem + st * STAGE;
    bf16x8 a[2][FM], b[2][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
      a[0][i] = *reinterpret_cast<const bf16x8*>(base + arow + i * 32 * BK + koff[0]);
#pragma unroll
    for (int j = 0; j < FN; ++j)
      b[0][j] = *reinterpret_cast<const bf16x8*>(base + brow + j * 32 * BK + koff[0]);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      const int cur = kk & 1;
      if (kk + 1 < KK) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
          a[cur ^ 1][i] = *reinterpret_cast<const bf16x8*>(base + arow + i * 32 * BK + koff[kk + 1]);
#pragma unroll
        for (int j = 0; j < FN; ++j)
          b[cur ^ 1][j] = *reinterpret_cast<const bf16x8*>(base + brow + j * 32 * BK + koff[kk + 1]);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[cur][i], b[cur][j], acc[i][j], 0, 0, 0);
    }
    if constexpr (SCHED) {
      // reads of k-step 0, then per k-step: one MFMA, one read of the next
      // k-step's fragments, ... (masks: 0x8 MFMA, 0x100 DS read)
      __builtin_amdgcn_sched_group_barrier(0x100, FM + FN, 0);
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        if (kk + 1 < KK) {
#pragma unroll
          for (int e = 0; e < FM + FN; ++e) {
            __builtin_amdgcn_sched_group_barrier(0x8, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
          if (FM * FN > FM + FN) __builtin_amdgcn_sched_group_barrier(0x8, FM * FN - FM - FN, 0);
        } else {
          __builtin_amdgcn_sched_group_barrier(0x8, FM * FN, 0);
        }
      }
    }
  };

  const int KT = K / BK;  // >= S - 1 (checked by the launcher)
#pragma unroll
  for (int s = 0; s < S - 1; ++s) issue(s, s);
  int kt = 0;
  for (; kt + S - 1 < KT; ++kt) {
    wait_vmcnt<(S - 2) * LPT>();
    lds_barrier();
    issue(kt + S - 1, (kt + S - 1) % S);
    compute(kt % S);
  }
  // drain: the last S-1 tiles, nothing more to issue
  if constexpr (S >= 5) {
    wait_vmcnt<3 * LPT>(); lds_barrier(); compute(kt % S); ++kt;
  }
  if constexpr (S >= 4) {
    wait_vmcnt<2 * LPT>(); lds_barrier(); compute(kt % S); ++kt;
  }
  if constexpr (S >= 3) {
    wait_vmcnt<LPT>(); lds_barrier(); compute(kt % S); ++kt;
  }
  wait_vmcnt<0>(); lds_barrier(); compute(kt % S);

  const Epilogue<bf16, EPI> epi{ep, M, N};
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const int n = n0 + wn * TN + j * 32 + lrow;
    const typename Epilogue<bf16, EPI>::Col col = epi.column(n);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int m = m0 + wm * TM + i * 32 + 8 * g + 4 * h;
        float v[4] = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                      acc[i][j][4 * g + 3]};
        epi.store4(col, m, n, v);
      }
  }
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
  int bm, bn, bk, stages;  // stages 0: register-staged kernel
};
static const TileCfg kTiles[] = {
    {128, 128, 64, 0}, {256, 128, 64, 0}, {128, 64, 64, 0},      // register staged
    {128, 128, 64, 3}, {256, 128, 64, 3}, {256, 192, 64, 2},     // LDS DMA, 4 waves
    {128, 128, 64, 3}, {256, 128, 64, 3}, {256, 192, 64, 2},     //   + sched groups
    {256, 128, 64, 3}, {256, 192, 64, 2}, {256, 128, 32, 5},     // 8 waves + sched
    {128, 128, 64, 4}, {256, 64, 64, 4},                         // 8 waves + sched
};
constexpr int kNumTiles = sizeof(kTiles) / sizeof(kTiles[0]);

static int forced_tile() {
  const char* s = getenv("ORCH_GEMM_TILE");
  return s ? atoi(s) : -1;
}

static bool tile_fits(const TileCfg& t, int N, int K) {
  if (N % t.bn || K % t.bk) return false;
  if (t.stages && K / t.bk < t.stages - 1) return false;
  return true;
}

// Pick the configuration with the least estimated time per CU: whole rounds
// of tiles over the 256 CUs times the tile area, divided by the measured
// relative efficiency of the tile shape.
static int pick_tile(int M, int N, int K) {
  const int f = forced_tile();
  if (f >= 0 && f < kNumTiles && tile_fits(kTiles[f], N, K)) return f;
  struct Cand { int idx; float eff; };
  static const Cand cands[] = {{10, 1.0f}, {9, 0.85f}, {12, 0.75f}};
  int best = -1;
  float best_cost = 0.0f;
  for (const Cand& c : cands) {
    const TileCfg& t = kTiles[c.idx];
    if (!tile_fits(t, N, K)) continue;
    const int tiles = ceil_div(M, t.bm) * (N / t.bn);
    const float cost = (float)ceil_div(tiles, 256) * t.bm * t.bn / c.eff;
    if (best < 0 || cost < best_cost) {
      best = c.idx;
      best_cost = cost;
    }
  }
  if (best >= 0) return best;
  if (N % 128 == 0) return 0;
  return 2;
}

bool gemm_uses_mfma(int N, int K, int dtype) {
  return dtype == kBF16 && N % 64 == 0 && K % kBK == 0;
}

template <int BM, int BN, int WM, int WN, int EPI>
static void launch_cfg(const void* A, const void* W, int M, int N, int K, const EpiParams& ep,
                       hipStream_t s) {
  dim3 grid(N / BN, ceil_div(M, BM));
  hipLaunchKernelGGL((gemm_bf16_mfma_kernel<BM, BN, WM, WN, EPI>), grid, dim3(64 * WM * WN), 0, s,
                     reinterpret_cast<const bf16*>(A), reinterpret_cast<const bf16*>(W), M, N, K,
                     ep);
}

template <int BM, int BN, int BK, int WM, int WN, int S, bool SCHED, int EPI>
static void launch_dma(const void* A, const void* W, int M, int N, int K, const EpiParams& ep,
                       hipStream_t s) {
  const int tm = ceil_div(M, BM), tn = N / BN;
  const size_t lds = (size_t)S * (BM + BN) * BK * sizeof(bf16);
  auto kern = gemm_bf16_dma_kernel<BM, BN, BK, WM, WN, S, SCHED, EPI>;
  static bool attr = [&] {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    return true;
  }();
  (void)attr;
  hipLaunchKernelGGL(kern, dim3(tm * tn), dim3(64 * WM * WN), lds, s, reinterpret_cast<const bf16*>(A),
                     reinterpret_cast<const bf16*>(W), M, N, K, tm, tn, ep);
}

template <int EPI>
static hipError_t launch_gemm_epi(const void* A, const void* W, int M, int N, int K,
                                  const EpiParams& ep, int dtype, hipStream_t s) {
  if (M <= 0 || N <= 0 || K <= 0) return hipSuccess;
  if (gemm_uses_mfma(N, K, dtype)) {
    switch (pick_tile(M, N, K)) {
      case 0: launch_cfg<128, 128, 2, 2, EPI>(A, W, M, N, K, ep, s); break;
      case 1: launch_cfg<256, 128, 2, 2, EPI>(A, W, M, N, K, ep, s); break;
      case 2: launch_cfg<128, 64, 2, 2, EPI>(A, W, M, N, K, ep, s); break;
      case 3: launch_dma<128, 128, 64, 2, 2, 3, false, EPI>(A, W, M, N, K, ep, s); break;
      case 4: launch_dma<256, 128, 64, 2, 2, 3, false, EPI>(A, W, M, N, K, ep, s); break;
      case 5: launch_dma<256, 192, 64, 2, 2, 2, false, EPI>(A, W, M, N, K, ep, s); break;
      case 6: launch_dma<128, 128, 64, 2, 2, 3, true, EPI>(A, W, M, N, K, ep, s); break;
      case 7: launch_dma<256, 128, 64, 2, 2, 3, true, EPI>(A, W, M, N, K, ep, s); break;
      case 8: launch_dma<256, 192, 64, 2, 2, 2, true, EPI>(A, W, M, N, K, ep, s); break;
      case 9: launch_dma<256, 128, 64, 4, 2, 3, true, EPI>(A, W, M, N, K, ep, s); break;
      case 10: launch_dma<256, 192, 64, 4, 2, 2, true, EPI>(A, W, M, N, K, ep, s); break;
      case 11: launch_dma<256, 128, 32, 4, 2, 5, true, EPI>(A, W, M, N, K, ep, s); break;
      case 12: launch_dma<128, 128, 64, 4, 2, 4, true, EPI>(A, W, M, N, K, ep, s); break;
      case 13: launch_dma<256, 64, 64, 4, 2, 4, true, EPI>(A, W, M, N, K, ep, s); break;
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
