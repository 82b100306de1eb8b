// Projection GEMMs of the DiT block: y = A W^T + bias with fused epilogues
// (plain store, GELU, gated residual add into the fp32 residual stream, and
// the QKV scatter into the head-major Q buffer and the K / V^T buffer).
//
// bf16 path: 128x128x64 tiles, 256 threads (2x2 waves of 64x64), operands
// staged through padded, double-buffered LDS, v_mfma_f32_32x32x16_bf16 with
// fp32 accumulation.  fp32 path (and shapes the MFMA tiling does not cover):
// a 64x64 SIMT tile with 4x4 outputs per thread.
#include "common.h"
#include "kernels.h"

namespace orch {

// ---------------------------------------------------------------------------
// epilogue: one output element (m, n) with accumulator v (bias not yet added)
template <typename T, int EPI>
__device__ __forceinline__ void epilogue_store(const EpiParams& ep, int M, int N, int m, int n,
                                               float v) {
  if (m >= M || n >= N) return;
  v += ep.bias[n];
  if (EPI == kEpiStore) {
    reinterpret_cast<T*>(ep.out)[(size_t)m * N + n] = from_f<T>(v);
  } else if (EPI == kEpiGelu) {
    reinterpret_cast<T*>(ep.out)[(size_t)m * N + n] = from_f<T>(gelu_tanh_f(v));
  } else if (EPI == kEpiResidual) {
    const int b = m / ep.rows_per_batch;
    float* h = reinterpret_cast<float*>(ep.out) + (size_t)m * N + n;
    *h += ep.gate[(size_t)b * ep.gate_stride + n] * v;
  } else {  // kEpiQkv
    const int b = m / ep.rows_per_batch;
    const int tok = m - b * ep.rows_per_batch;
    const int which = n / ep.hidden;
    const int nn = n - which * ep.hidden;
    const int head = nn / ep.head_dim;
    const int dd = nn - head * ep.head_dim;
    const T val = from_f<T>(v);
    if (which == 0) {
      T* q = reinterpret_cast<T*>(ep.q);
      q[(((size_t)b * ep.heads + head) * ep.rows_per_batch + tok) * ep.head_dim + dd] = val;
    } else {
      T* kv = reinterpret_cast<T*>(ep.kv) + (size_t)b * ep.kv_branch_stride;
      const size_t ntot = (size_t)ep.kv_tokens;
      const size_t pos = (size_t)ep.tok_offset + tok;
      if (which == 1) {
        kv[((size_t)head * ntot + pos) * ep.head_dim + dd] = val;
      } else {
        T* vt = kv + ntot * ep.hidden;
        vt[((size_t)head * ep.head_dim + dd) * ntot + pos] = val;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA GEMM
namespace mfma_gemm {
constexpr int BM = 128, BN = 128, BK = 64;
constexpr int LDS_STRIDE = BK + 8;  // bf16 elements per LDS row (144 B: conflict-free b128 reads)
constexpr int THREADS = 256;
}  // namespace mfma_gemm

template <int EPI>
__global__ __launch_bounds__(256) void gemm_bf16_mfma_kernel(const bf16* __restrict__ A,
                                                             const bf16* __restrict__ W, int M,
                                                             int N, int K, EpiParams ep) {
  using namespace mfma_gemm;
  __shared__ __attribute__((aligned(16))) bf16 sA[2][BM * LDS_STRIDE];
  __shared__ __attribute__((aligned(16))) bf16 sB[2][BN * LDS_STRIDE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * BM;
  const int n0 = blockIdx.x * BN;

  // global -> register staging: 1024 chunks of 16 B per operand tile,
  // chunk c = tid + 256 i: row c / 8, k-chunk c % 8.
  uint4 ra[4], rb[4];
  const int kc = tid & 7;
  const int row_base = tid >> 3;  // 0..31

  auto load_tile = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int r = row_base + 32 * i;
      int gm = min(m0 + r, M - 1);
      ra[i] = *reinterpret_cast<const uint4*>(A + (size_t)gm * K + k0 + kc * 8);
      int gn = n0 + r;  // N % BN == 0
      rb[i] = *reinterpret_cast<const uint4*>(W + (size_t)gn * K + k0 + kc * 8);
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int r = row_base + 32 * i;
      *reinterpret_cast<uint4*>(&sA[buf][r * LDS_STRIDE + kc * 8]) = ra[i];
      *reinterpret_cast<uint4*>(&sB[buf][r * LDS_STRIDE + kc * 8]) = rb[i];
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int KT = K / BK;
  load_tile(0);
  store_tile(0);
  __syncthreads();

  const int lrow = lane & 31;
  const int lk = (lane >> 5) * 8;
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) load_tile((kt + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        a[i] = *reinterpret_cast<const bf16x8*>(
            &sA[buf][(wm * 64 + i * 32 + lrow) * LDS_STRIDE + kk * 16 + lk]);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        b[j] = *reinterpret_cast<const bf16x8*>(
            &sB[buf][(wn * 64 + j * 32 + lrow) * LDS_STRIDE + kk * 16 + lk]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < KT) store_tile(buf ^ 1);
    __syncthreads();
  }

  // accumulator layout of a 32x32 MFMA block: lane holds column lane%32,
  // register r holds row 8*(r/4) + 4*(lane/32) + r%4.
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int m = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        int n = n0 + wn * 64 + j * 32 + (lane & 31);
        epilogue_store<bf16, EPI>(ep, M, N, m, n, acc[i][j][r]);
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
    // 64 rows x 16 k per operand = 1024 elements, 4 per thread
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
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      epilogue_store<T, EPI>(ep, M, N, m0 + ty * 4 + i, n0 + tx * 4 + j, acc[i][j]);
}

// ---------------------------------------------------------------------------
bool gemm_uses_mfma(int N, int K, int dtype) {
  return dtype == kBF16 && N % mfma_gemm::BN == 0 && K % mfma_gemm::BK == 0;
}

template <int EPI>
static hipError_t launch_gemm_epi(const void* A, const void* W, int M, int N, int K,
                                  const EpiParams& ep, int dtype, hipStream_t s) {
  if (M <= 0 || N <= 0 || K <= 0) return hipSuccess;
  if (gemm_uses_mfma(N, K, dtype)) {
    dim3 grid(N / mfma_gemm::BN, ceil_div(M, mfma_gemm::BM));
    hipLaunchKernelGGL(gemm_bf16_mfma_kernel<EPI>, grid, dim3(256), 0, s,
                       reinterpret_cast<const bf16*>(A), reinterpret_cast<const bf16*>(W), M, N,
                       K, ep);
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
