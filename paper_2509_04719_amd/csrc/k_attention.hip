// Attention of a band's queries over the keys/values of the whole image,
// fresh for the band's tokens and stale (from the buffer) for all others
// (patch parallelism with stale activations, §II-B; Algorithm 1).
//
// bf16 path: a flash-style kernel on v_mfma_f32_32x32x16_bf16.  Each
// workgroup owns 128 queries of one (branch, head); each wave 32 of them.
// Scores are formed transposed, S^T = K Q^T, so that a lane owns one query
// column: the running max / sum of the online softmax stay in-lane, and the
// probabilities it holds are directly the B operand of O^T = V^T P^T.  K
// tiles ([64 keys][d]) and V^T tiles ([d][64 keys]) are staged through
// double-buffered LDS; the V^T layout of the buffer makes both tile loads
// contiguous 16-byte rows.
//
// fp32 path (and unsupported shapes): one thread per query, online softmax.
#include "common.h"
#include "kernels.h"

namespace orch {

namespace mfma_attn {
constexpr int BQ = 128, BKV = 64;
}

template <int D>
__global__ __launch_bounds__(256) void attn_bf16_mfma_kernel(AttnParams p) {
  using namespace mfma_attn;
  constexpr int DP = (D + 15) / 16 * 16;         // QK^T contraction, padded to 16
  constexpr int NC = DP / 16;
  constexpr int DV = (D + 31) / 32 * 32;         // rows of O^T, padded to 32
  constexpr int NT = DV / 32;
  constexpr int KS = (DP % 64 == 0) ? DP + 8 : DP;  // LDS row stride of K tiles
  constexpr int VS = BKV + 8;                        // LDS row stride of V^T tiles
  constexpr int KCH = D / 8;                         // 16-byte chunks per K row
  constexpr int K_CHUNKS = BKV * KCH;
  constexpr int V_CHUNKS = D * (BKV / 8);
  constexpr int K_IT = (K_CHUNKS + 255) / 256;
  constexpr int V_IT = (V_CHUNKS + 255) / 256;

  __shared__ __attribute__((aligned(16))) bf16 sK[2][BKV * KS];
  __shared__ __attribute__((aligned(16))) bf16 sV[2][DV * VS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int h = lane >> 5;
  const int lc = lane & 31;
  const int b = blockIdx.z;
  const int head = blockIdx.y;
  const int q0 = blockIdx.x * BQ;
  const int H = p.heads * D;

  const bf16* qbase = reinterpret_cast<const bf16*>(p.q) + ((size_t)b * p.heads + head) * p.n_q * D;
  const bf16* ks = reinterpret_cast<const bf16*>(p.kv_stale) + b * p.stale_bs +
                   (size_t)head * p.n_kv * D;
  const bf16* vs = reinterpret_cast<const bf16*>(p.kv_stale) + b * p.stale_bs +
                   (size_t)p.n_kv * H + (size_t)head * D * p.n_kv;
  const bf16* kf = nullptr;
  const bf16* vf = nullptr;
  if (p.n_fresh > 0) {
    kf = reinterpret_cast<const bf16*>(p.kv_fresh) + b * p.fresh_bs + (size_t)head * p.n_fresh * D;
    vf = reinterpret_cast<const bf16*>(p.kv_fresh) + b * p.fresh_bs + (size_t)p.n_fresh * H +
         (size_t)head * D * p.n_fresh;
  }

  // zero the padding columns of K and rows of V^T once (never overwritten)
  for (int i = tid; i < 2 * BKV * (KS - D); i += 256) {
    int buf = i / (BKV * (KS - D));
    int rem = i - buf * BKV * (KS - D);
    int r = rem / (KS - D), c = D + rem % (KS - D);
    sK[buf][r * KS + c] = (bf16)0.0f;
  }
  for (int i = tid; i < 2 * (DV - D) * VS; i += 256) {
    int buf = i / ((DV - D) * VS);
    int rem = i - buf * (DV - D) * VS;
    sV[buf][D * VS + rem] = (bf16)0.0f;
  }

  // this lane's query (B operand of S^T = K Q^T): Q[q][c*16 + 8h .. +8]
  const int qrow = min(q0 + wave * 32 + lc, p.n_q - 1);
  bf16x8 qf[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int d0 = c * 16 + h * 8;
    if (d0 < D) {
      qf[c] = *reinterpret_cast<const bf16x8*>(qbase + (size_t)qrow * D + d0);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) qf[c][e] = (bf16)0.0f;
    }
  }

  uint4 rk[K_IT], rv[V_IT];
  auto load_kv = [&](int n0) {
#pragma unroll
    for (int i = 0; i < K_IT; ++i) {
      int c = tid + 256 * i;
      if (c < K_CHUNKS) {
        int r = c / KCH, cc = c - r * KCH;
        int n = n0 + r;
        int f = n - p.fresh_begin;
        const bf16* src = ((unsigned)f < (unsigned)p.n_fresh) ? kf + (size_t)f * D : ks + (size_t)n * D;
        rk[i] = *reinterpret_cast<const uint4*>(src + cc * 8);
      }
    }
#pragma unroll
    for (int i = 0; i < V_IT; ++i) {
      int c = tid + 256 * i;
      if (c < V_CHUNKS) {
        int d = c >> 3, kc = c & 7;
        int n = n0 + kc * 8;
        int f = n - p.fresh_begin;
        const bf16* src = ((unsigned)f < (unsigned)p.n_fresh) ? vf + (size_t)d * p.n_fresh + f
                                                              : vs + (size_t)d * p.n_kv + n;
        rv[i] = *reinterpret_cast<const uint4*>(src);
      }
    }
  };
  auto store_kv = [&](int buf) {
#pragma unroll
    for (int i = 0; i < K_IT; ++i) {
      int c = tid + 256 * i;
      if (c < K_CHUNKS) {
        int r = c / KCH, cc = c - r * KCH;
        *reinterpret_cast<uint4*>(&sK[buf][r * KS + cc * 8]) = rk[i];
      }
    }
#pragma unroll
    for (int i = 0; i < V_IT; ++i) {
      int c = tid + 256 * i;
      if (c < V_CHUNKS) {
        int d = c >> 3, kc = c & 7;
        *reinterpret_cast<uint4*>(&sV[buf][d * VS + kc * 8]) = rv[i];
      }
    }
  };

  const float scale = 1.4426950408889634f / sqrtf((float)D);  // log2(e) / sqrt(d)
  float m_run = -1e30f, l_run = 0.0f;
  f32x16 o[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[t][r] = 0.0f;

  const int NIT = p.n_kv / BKV;
  load_kv(0);
  store_kv(0);
  __syncthreads();

  for (int it = 0; it < NIT; ++it) {
    const int buf = it & 1;
    if (it + 1 < NIT) load_kv((it + 1) * BKV);

    // S^T for keys [32 sub, 32 sub + 32) x this wave's 32 queries
    f32x16 s[2];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[sub][r] = 0.0f;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        bf16x8 a = *reinterpret_cast<const bf16x8*>(&sK[buf][(sub * 32 + lc) * KS + c * 16 + h * 8]);
        s[sub] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[c], s[sub], 0, 0, 0);
      }
    }
    // online softmax over this lane's query column
    float mx = s[0][0];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[sub][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    const float m_new = fmaxf(m_run, mx * scale);
    const float alpha = exp2f(m_run - m_new);
    m_run = m_new;
    float psum = 0.0f;
    bf16x8 pf[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int sub = c >> 1;
      const int g0 = 2 * (c & 1);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int r = 4 * (g0 + (e >> 2)) + (e & 3);
        const float pv = exp2f(fmaf(s[sub][r], scale, -m_new));
        psum += pv;
        pf[c][e] = (bf16)pv;
      }
    }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[t][r] *= alpha;

    // O^T += V^T P^T
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const bf16* vrow = &sV[buf][(t * 32 + lc) * VS + c * 16 + 4 * h];
        bf16x4 lo = *reinterpret_cast<const bf16x4*>(vrow);
        bf16x4 hi = *reinterpret_cast<const bf16x4*>(vrow + 8);
        bf16x8 a;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          a[e] = lo[e];
          a[e + 4] = hi[e];
        }
        o[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[c], o[t], 0, 0, 0);
      }
    }
    if (it + 1 < NIT) store_kv(buf ^ 1);
    __syncthreads();
  }

  const float l = l_run + __shfl_xor(l_run, 32, kWave);
  const float inv = 1.0f / l;
  const int q = q0 + wave * 32 + lc;
  if (q < p.n_q) {
    bf16* orow = reinterpret_cast<bf16*>(p.out) + ((size_t)b * p.n_q + q) * H + head * D;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d = t * 32 + 8 * g + 4 * h;
        if (d < D) {
          bf16x4 v;
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = (bf16)(o[t][4 * g + j] * inv);
          *reinterpret_cast<bf16x4*>(orow + d) = v;
        }
      }
  }
}

// ---------------------------------------------------------------------------
// SIMT attention: one thread per (branch, head, query).
template <typename T, int D>
__global__ __launch_bounds__(64) void attn_simt_kernel(AttnParams p) {
  const int q = blockIdx.x * 64 + threadIdx.x;
  const int head = blockIdx.y;
  const int b = blockIdx.z;
  if (q >= p.n_q) return;
  const int H = p.heads * D;
  const T* qv = reinterpret_cast<const T*>(p.q) + (((size_t)b * p.heads + head) * p.n_q + q) * D;
  const T* ks = reinterpret_cast<const T*>(p.kv_stale) + b * p.stale_bs + (size_t)head * p.n_kv * D;
  const T* vs = reinterpret_cast<const T*>(p.kv_stale) + b * p.stale_bs + (size_t)p.n_kv * H +
                (size_t)head * D * p.n_kv;
  const T* kf = nullptr;
  const T* vf = nullptr;
  if (p.n_fresh > 0) {
    kf = reinterpret_cast<const T*>(p.kv_fresh) + b * p.fresh_bs + (size_t)head * p.n_fresh * D;
    vf = reinterpret_cast<const T*>(p.kv_fresh) + b * p.fresh_bs + (size_t)p.n_fresh * H +
         (size_t)head * D * p.n_fresh;
  }
  float qr[D], acc[D];
  const float scale = 1.0f / sqrtf((float)D);
#pragma unroll
  for (int d = 0; d < D; ++d) {
    qr[d] = to_f<T>(qv[d]) * scale;
    acc[d] = 0.0f;
  }
  float m = -INFINITY, l = 0.0f;
  for (int n = 0; n < p.n_kv; ++n) {
    const int f = n - p.fresh_begin;
    const bool fresh = (unsigned)f < (unsigned)p.n_fresh;
    const T* kr = fresh ? kf + (size_t)f * D : ks + (size_t)n * D;
    float s = 0.0f;
#pragma unroll
    for (int d = 0; d < D; ++d) s = fmaf(qr[d], to_f<T>(kr[d]), s);
    const float mn = fmaxf(m, s);
    const float a = expf(m - mn);
    const float e = expf(s - mn);
    l = l * a + e;
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const float v = fresh ? to_f<T>(vf[(size_t)d * p.n_fresh + f]) : to_f<T>(vs[(size_t)d * p.n_kv + n]);
      acc[d] = fmaf(acc[d], a, e * v);
    }
    m = mn;
  }
  T* o = reinterpret_cast<T*>(p.out) + ((size_t)b * p.n_q + q) * H + head * D;
  const float inv = 1.0f / l;
#pragma unroll
  for (int d = 0; d < D; ++d) o[d] = from_f<T>(acc[d] * inv);
}

// ---------------------------------------------------------------------------
bool attention_uses_mfma(int d, int n_kv, int dtype) {
  return dtype == kBF16 && (d == 64 || d == 72) && n_kv % mfma_attn::BKV == 0;
}

template <typename T>
static hipError_t launch_simt(const AttnParams& p, hipStream_t s) {
  dim3 grid(ceil_div(p.n_q, 64), p.heads, p.B);
  switch (p.d) {
    case 32: hipLaunchKernelGGL((attn_simt_kernel<T, 32>), grid, dim3(64), 0, s, p); break;
    case 64: hipLaunchKernelGGL((attn_simt_kernel<T, 64>), grid, dim3(64), 0, s, p); break;
    case 72: hipLaunchKernelGGL((attn_simt_kernel<T, 72>), grid, dim3(64), 0, s, p); break;
    case 80: hipLaunchKernelGGL((attn_simt_kernel<T, 80>), grid, dim3(64), 0, s, p); break;
    case 96: hipLaunchKernelGGL((attn_simt_kernel<T, 96>), grid, dim3(64), 0, s, p); break;
    case 128: hipLaunchKernelGGL((attn_simt_kernel<T, 128>), grid, dim3(64), 0, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attention(const AttnParams& p, int dtype, hipStream_t s) {
  if (p.n_q <= 0) return hipSuccess;
  const bool aligned = (p.fresh_begin % 8 == 0) && (p.n_fresh % 8 == 0);
  if (attention_uses_mfma(p.d, p.n_kv, dtype) && aligned) {
    dim3 grid(ceil_div(p.n_q, mfma_attn::BQ), p.heads, p.B);
    if (p.d == 64)
      hipLaunchKernelGGL(attn_bf16_mfma_kernel<64>, grid, dim3(256), 0, s, p);
    else
      hipLaunchKernelGGL(attn_bf16_mfma_kernel<72>, grid, dim3(256), 0, s, p);
    return hipGetLastError();
  }
  if (dtype == kBF16) return launch_simt<bf16>(p, s);
  return launch_simt<float>(p, s);
}

}  // namespace orch
